"""Host logic of bench.py (no GPU): the algorithmic work behind the roofline
figure and the per-CU residency measure, on hand-worked cases."""
import importlib.util
import os

import numpy as np
import pytest

import synth

_ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
_spec = importlib.util.spec_from_file_location("bench_host", os.path.join(_ROOT, "bench.py"))
B = importlib.util.module_from_spec(_spec)
_spec.loader.exec_module(B)


def test_kernel_work_lm_gateup_eight_frames():
    # 8 stacked frames of the 305-token prefix: M = 2440, N = 2 x 16384 (gate
    # and up), K = 2048. Weights 2 N K, activations 2 M K, bf16 GeGLU output
    # 2 M (N / 2): 134,217,728 + 9,994,240 + 79,953,920 bytes
    cfg = synth.PRESETS["pi0"]
    byts, flops = B.kernel_work(cfg, "lm.gateup", vlm_frames=8)
    assert byts == 224_165_888
    assert flops == 2.0 * 2440 * 32768 * 2048 == 327_491_256_320


def test_kernel_work_expert_one_frame():
    cfg = synth.PRESETS["pi0"]
    # gate/up of one 50-row chunk: 16,777,216 + 102,400 + 409,600 bytes
    byts, flops = B.kernel_work(cfg, "ex.gateup")
    assert byts == 17_289_216 and flops == 2.0 * 50 * 8192 * 1024
    # a residual epilogue reads and writes the fp32 residual: 8 bytes per output
    byts, flops = B.kernel_work(cfg, "ex.down")
    assert byts == 2 * 1024 * 4096 + 2 * 50 * 4096 + 8 * 50 * 1024
    assert flops == 2.0 * 50 * 1024 * 4096
    # a batched loop of 8 stacks the rows; the weights count once
    b8, f8 = B.kernel_work(cfg, "ex.down", act_frames=8)
    assert b8 == 2 * 1024 * 4096 + 8 * (2 * 50 * 4096 + 8 * 50 * 1024) and f8 == 8 * flops


def _hw(cu, queue):
    """A hardware-id word with CU index cu (< 16, shader engine and array 0)
    on queue `queue` (< 8)."""
    return (cu & 15) << 8 | (queue & 7) << 24


def _records(wgs):
    """Workgroup start and end records from (cu, queue, kind, start, end)."""
    hw, kind, t, end = [], [], [], []
    for cu, q, k, t0, t1 in wgs:
        for tt, e in ((t0, 0), (t1, 1)):
            hw.append(_hw(cu, q))
            kind.append(k)
            t.append(tt)
            end.append(e)
    n = len(hw)
    return {"hwid": np.array(hw, np.uint32), "xcc": np.zeros(n, np.uint32), "kind": np.array(kind),
            "t": np.array(t, np.int64), "end": np.array(end)}


def test_cu_residency_hand_worked():
    # queue 1 runs a ViT-attention workgroup (kind 4), so it is a prefill
    # queue; queue 2 is the action phase's. CU 0: prefill 0-100, action
    # 50-150; CU 1: action 0-40, then action 40-60 (starts as the first ends)
    rec = _records([(0, 1, 4, 0, 100), (0, 2, 6, 50, 150), (1, 2, 6, 0, 40), (1, 2, 6, 40, 60)])
    r = B.cu_residency(rec)
    # default window: where both phases have records, [max of the first
    # records, min of the last] = [0, 100]; 2 CUs x 100 ticks
    assert r["cus"] == 2 and r["vlm_queues"] == 1
    assert r["window_ms"] == pytest.approx(100 * 1e-5)
    # busy: CU 0 all 100, CU 1 0-60 (no gap at 40) -> 160 / 200
    assert r["busy_frac"] == pytest.approx(0.8)
    # both phases: CU 0 50-100 -> 50 / 200
    assert r["both_phases_frac"] == pytest.approx(0.25)
    # an explicit window [0, 200]: busy 150 + 60, both 50, over 400
    r = B.cu_residency(rec, window=(0, 200))
    assert r["busy_frac"] == pytest.approx(210 / 400)
    assert r["both_phases_frac"] == pytest.approx(50 / 400)


def test_cu_residency_one_phase():
    # only action workgroups: no prefill queue; the window is the whole log
    rec = _records([(0, 2, 6, 10, 30), (3, 2, 6, 20, 50)])
    r = B.cu_residency(rec)
    assert r["vlm_queues"] == 0 and r["cus"] == 2
    assert r["busy_frac"] == pytest.approx((20 + 30) / (2 * 40))
    assert r["both_phases_frac"] == 0.0
