"""Intensity descriptors and the CU-split planner (host logic, no GPU).

The quantisation and the descriptor arithmetic follow the paper's offline
profiling pass (section on profile metadata, table of intensity fields):
fraction of peak on the matrix, ALU and DRAM pipelines, quantised to 0..15.
The planner's cases below are worked by hand."""
import csv
import math

import pytest

from paper_2609_22335_amd import intensity as I


def test_quantize_levels():
    assert I.quantize(0.0) == 0
    assert I.quantize(-0.1) == 0
    assert I.quantize(float("nan")) == 0
    assert I.quantize(1.0) == 15
    assert I.quantize(3.0) == 15
    assert I.quantize(0.5) == 8          # 7.5 rounds half up
    assert I.quantize(1 / 30 - 1e-9) == 0  # just below level 1's lower edge (0.5 / 15)
    assert I.quantize(1 / 30 + 1e-9) == 1
    assert I.quantize(7 / 15) == 7
    levels = [I.quantize(i / 1000) for i in range(1001)]
    assert levels == sorted(levels) and set(levels) == set(range(16))


def _write(path, header, rows):
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)


TRACE_H = ["Kernel_Name", "Grid_Size_X", "Workgroup_Size_X", "Start_Timestamp", "End_Timestamp"]
CTR_H = ["Kernel_Name", "Grid_Size", "Workgroup_Size", "Counter_Name", "Counter_Value"]


def test_descriptor_arithmetic(tmp_path):
    # kernel A: 256 workgroups of 256 threads, 10 us per launch; kernel B:
    # 8 workgroups of 64 threads, 2 us
    _write(tmp_path / "t1.csv", TRACE_H, [["A", 65536, 256, 0, 10_000], ["B", 512, 64, 0, 2_000],
                                          ["S", 64, 64, 0, 1_000]])
    _write(tmp_path / "t3.csv", TRACE_H, [["A", 65536, 256, 0, 10_000]] * 3 + [["B", 512, 64, 0, 2_000]] * 7 +
           [["S", 64, 64, 0, 1_000]])
    small, large = I.read_trace(str(tmp_path / "t1.csv")), I.read_trace(str(tmp_path / "t3.csv"))
    counts = I.frame_counts(small, large, 2)
    assert counts == {("A", 256, 256): 1.0, ("B", 8, 64): 3.0}  # set-up kernel S cancels
    # A: 12.5 GFLOP of bf16 MFMA in 10 us = 1.25 PFLOP/s = half of peak;
    # B: 0.3146 GFLOP of fp32 VALU in 2 us = 157.3 TFLOP/s = all of peak
    alu_rows = [["A", 65536, 256, "SQ_INSTS_VALU_MFMA_MOPS_BF16", 12.5e9 / 512],
                ["A", 65536, 256, "SQ_INSTS_VALU_FLOPS_FP32", 0],
                ["B", 512, 64, "SQ_INSTS_VALU_MFMA_MOPS_BF16", 0],
                ["B", 512, 64, "SQ_INSTS_VALU_FLOPS_FP32", 157.3e12 * 2e-6 * 0.75],
                ["B", 512, 64, "SQ_INSTS_VALU_FLOPS_FP32_TRANS", 157.3e12 * 2e-6 * 0.25]]
    _write(tmp_path / "alu.csv", CTR_H, alu_rows)
    # DRAM: A moves 20 MB in 10 us = 2 TB/s = 0.25 of 8 TB/s (counted KiB
    # are half the true fetched bytes, scale 2; writes counted 1:1)
    _write(tmp_path / "fe.csv", CTR_H, [["A", 65536, 256, "FETCH_SIZE", 8e6 / 1024 / 2], ["B", 512, 64, "FETCH_SIZE", 0]])
    _write(tmp_path / "wr.csv", CTR_H, [["A", 65536, 256, "WRITE_SIZE", 12e6 / 1024], ["B", 512, 64, "WRITE_SIZE", 0]])
    d = I.descriptors(large, I.read_counters(str(tmp_path / "alu.csv")), I.read_counters(str(tmp_path / "fe.csv")),
                      I.read_counters(str(tmp_path / "wr.csv")), 2.0, 1.0, counts, "vlm")
    by = {x["kernel"]: x for x in d}
    assert by["A"]["frac"] == pytest.approx([0.5, 0.0, 0.25])
    assert by["A"]["tau"] == [8, 0, 4]
    assert by["B"]["frac"] == pytest.approx([0.0, 1.0, 0.0])
    assert by["B"]["tau"] == [0, 15, 0]
    assert by["A"]["us"] == pytest.approx(10.0) and by["B"]["launches_per_frame"] == 3.0
    assert d[0]["kernel"] == "A"  # ordered by time per frame (10 us vs 6 us)


def test_copy_scale(tmp_path):
    _write(tmp_path / "c.csv", CTR_H, [["void at::elementwise_copy", 1 << 20, 256, "FETCH_SIZE", 131072],
                                       ["other", 4, 64, "FETCH_SIZE", 10]])
    c = I.read_counters(str(tmp_path / "c.csv"))
    assert I.copy_scale(c, "FETCH_SIZE", 262144.0) == pytest.approx(2.0)
    with pytest.raises(ValueError):
        I.copy_scale(c, "WRITE_SIZE", 1.0)


def _d(phase, wgs, us, lpf=1.0, mem=0.1):
    return {"kernel": f"{phase}{wgs}", "workgroups": wgs, "wg_threads": 256, "phase": phase,
            "launches_per_frame": lpf, "us": us, "frac": [0.0, 0.0, mem], "tau": [0, 0, I.quantize(mem)]}


def test_planner_worked_case():
    # VLM: one 256-workgroup kernel, 1 ms alone; action: one 32-workgroup
    # kernel, 0.5 ms alone. On c VLM CUs the VLM takes 256 / c ms, the
    # action 0.5 * max(1, 32 / (256 - c)) ms:
    #   c = 224: max(1.143, 0.5) = 1.143;  c = 232: max(1.103, 0.667) = 1.103
    #   c = 240: max(1.067, 1.0)  = 1.067;  c = 248: max(1.032, 2.0)   = 2.0
    desc = [_d("vlm", 256, 1000.0), _d("action", 32, 500.0)]
    assert I.phase_time(desc, "vlm", 128) == pytest.approx(2e-3)
    assert I.phase_time(desc, "action", 128) == pytest.approx(0.5e-3)
    assert I.phase_time(desc, "action", 16) == pytest.approx(1e-3)
    p = I.plan_cu_split(desc)
    assert (p["vlm_cus"], p["act_cus"]) == (240, 16)
    assert p["per_frame_s"] == pytest.approx(256 / 240 * 1e-3)
    assert p["hbm_share"] == pytest.approx(0.2)


def test_planner_hbm_share_and_weights():
    # two launches per frame of the action kernel count twice; DRAM
    # fractions 0.7 (VLM) and 0.6 (action, time-weighted) exceed 1 together
    # by 0.3: without a calibration that share of the shorter phase does not
    # overlap
    desc = [_d("vlm", 64, 100.0, mem=0.7), _d("action", 8, 50.0, lpf=2.0, mem=0.9), _d("action", 8, 100.0, mem=0.3)]
    assert I.mem_level(desc, "action") == pytest.approx((100 * 0.9 + 100 * 0.3) / 200)
    p = I.predict_split(desc, 128)
    assert p["vlm_s"] == pytest.approx(100e-6) and p["action_s"] == pytest.approx(200e-6)
    assert p["per_frame_s"] == pytest.approx(200e-6 + 0.3 * 100e-6)
    assert math.isclose(p["hbm_share"], 1.3)


def test_kernel_time_bandwidth_limit():
    # a kernel at 40% of HBM peak on 256 CUs: with rho = 0.8 its CUs deliver
    # at most 0.8 * C / 256 of the peak, so on 64 CUs it stretches by
    # 0.4 * 256 / (0.8 * 64) = 2 (its 8 workgroups still fit)
    d = _d("action", 8, 10.0, mem=0.4)
    assert I.kernel_time(d, 256, 0.8) == pytest.approx(10e-6)
    assert I.kernel_time(d, 64, 0.8) == pytest.approx(20e-6)
    assert I.kernel_time(d, 64, 0.0) == pytest.approx(10e-6)
    # the slot limit wins where it is larger: 64 workgroups at 1 per CU on 16 CUs
    assert I.kernel_time(_d("vlm", 64, 10.0, mem=0.1), 16, 0.8) == pytest.approx(40e-6)


def test_fit_calibration_recovers_the_model():
    # frames/s generated by the model itself with rho = 0.5, kappa = 0.4 are
    # fitted back exactly, and the planner then picks the generated optimum
    # (the action kernels' bandwidth term binds on every split, so rho is
    # identifiable)
    desc = [_d("vlm", 512, 100.0, mem=0.3), _d("action", 64, 60.0, lpf=3.0, mem=0.6),
            _d("action", 25, 20.0, lpf=2.0, mem=0.05)]
    cal = {"rho": 0.5, "kappa": 0.4}
    meas = {v: 1.0 / I.predict_split(desc, v, cal=cal)["per_frame_s"] for v in (224, 192, 160, 128, 96)}
    fit = I.fit_calibration(desc, meas)
    assert fit["rho"] == pytest.approx(0.5) and fit["kappa"] == pytest.approx(0.4)
    assert fit["max_rel_err"] < 1e-9
    best = I.plan_cu_split(desc, cal=fit)
    assert best["vlm_cus"] == I.plan_cu_split(desc, cal=cal)["vlm_cus"]


def test_trace_stats_table_row(tmp_path):
    # the paper's micro-kernel table: median cycles and the shares below 5K,
    # 10K, 25K and 50K cycles; at 2 GHz, 1 us = 2000 cycles
    from paper_2609_22335_amd import trace_stats as T
    rows = [["k_a", 256, 256, 0, 1_000], ["k_b", 256, 256, 0, 3_000], ["k_c", 256, 256, 0, 6_000],
            ["k_d", 256, 256, 0, 20_000], ["k_unfrag", 256, 256, 0, 1]]
    _write(tmp_path / "t.csv", TRACE_H, rows)
    d = T.durations_ns(str(tmp_path / "t.csv"))
    assert d == [1000, 3000, 6000, 20000]  # the weight re-layout is skipped
    r = T.table_row(d, 2.0)
    # cycles 2000, 6000, 12000, 40000: median (6000 + 12000) / 2
    assert r["kernels"] == 4 and r["median_cyc"] == 9000
    assert (r["lt5k_pct"], r["lt10k_pct"], r["lt25k_pct"], r["lt50k_pct"]) == (25.0, 50.0, 75.0, 100.0)
    assert T.table_row([4999 / 2.0], 2.0)["lt5k_pct"] == 100.0  # strictly below the bound
    assert T.table_row([5000 / 2.0], 2.0)["lt5k_pct"] == 0.0
    with pytest.raises(ValueError):
        T.table_row([], 2.0)


def test_measured_splits_of_the_main_and_further_workloads(tmp_path):
    # the main workload's cu_V_A schedules, or those of the further workload
    # named <preset>_R<R> (exactly: "pi0_R8_async" is not the pi0 workload)
    import json
    from paper_2609_22335_amd import profile_intensity as PI
    det = {"modes": {"serial": {"frames_per_s": 1.0}, "cu_192_64": {"frames_per_s": 2.0},
                     "cu_160_96": {"frames_per_s": 3.0}, "cu_160_96_lanes2": {"frames_per_s": 9.0}},
           "other_workloads": {"pi0_R8_async": {"modes": {"cu_224_32": {"frames_per_s": 7.0}}},
                               "pi0_3view_R32": {"modes": {"cu_224_32": {"frames_per_s": 4.0},
                                                           "cu_192_64": {"frames_per_s": 5.0}}}}}
    p = tmp_path / "detail.json"
    p.write_text(json.dumps(det))
    assert PI.measured_splits(str(p)) == {192: 2.0, 160: 3.0}
    assert PI.measured_splits(str(p), "pi0") == {192: 2.0, 160: 3.0}
    assert PI.measured_splits(str(p), "pi0_3view") == {224: 4.0, 192: 5.0}


def test_refit_stores_the_calibration_and_plan(tmp_path):
    # splits generated by the model itself (rho 0.5, kappa 0.4) are fitted
    # back and stored in the descriptor file with the split the calibrated
    # planner picks, as the bench's cu_auto schedule reads them
    import json
    from paper_2609_22335_amd import profile_intensity as PI
    desc = [_d("vlm", 512, 100.0, mem=0.3), _d("action", 64, 60.0, lpf=3.0, mem=0.6),
            _d("action", 25, 20.0, lpf=2.0, mem=0.05)]
    cal = {"rho": 0.5, "kappa": 0.4}
    fps = {v: 1.0 / I.predict_split(desc, v, cal=cal)["per_frame_s"] for v in (224, 192, 160)}
    path = tmp_path / "intensity.json"
    I.save(str(path), desc, {"preset": "x"})
    det = tmp_path / "detail.json"
    det.write_text(json.dumps({"modes": {}, "other_workloads": {
        "x_R32": {"modes": {f"cu_{v}_{256 - v}": {"frames_per_s": f} for v, f in fps.items()}}}}))
    PI.refit("x", str(path), str(det))
    got = I.load_calibration(str(path))
    assert got["rho"] == pytest.approx(0.5) and got["kappa"] == pytest.approx(0.4)
    meta = json.load(open(path))["meta"]
    assert meta["preset"] == "x"
    assert meta["cu_split_plan"]["vlm_cus"] == I.plan_cu_split(desc, cal=cal)["vlm_cus"]

