"""Per-kernel intensity descriptors on MI355X and a CU-split planner that
reads them.

The paper's offline phase (its section on profile metadata and the table of
intensity fields) profiles every kernel of a model once, in isolation, with
hardware counters, and keeps for each one the fraction of peak it reaches on
three pipelines -- matrix units, vector ALU (fp32 FLOP/s) and DRAM -- as
4-bit levels 0..15 (tau_TC, tau_ALU, tau_MEM), stored in a file. On MI355X the
matrix pipeline is MFMA, the counters come from rocprofv3, and a kernel is a
launch configuration (kernel symbol, grid, workgroup size), the unit the
paper also counts ("unique launch configurations").

Counters per dispatch (rocprofv3, each pass its own run):
  MFMA FLOPs   = 512 * (SQ_INSTS_VALU_MFMA_MOPS_BF16 + SQ_INSTS_VALU_MFMA_MOPS_F32)
  fp32 FLOPs   = SQ_INSTS_VALU_FLOPS_FP32 + SQ_INSTS_VALU_FLOPS_FP32_TRANS
  DRAM bytes   = FETCH_SIZE * f + WRITE_SIZE * w (KiB), f and w scaling a
                 plain device copy of known size to its true bytes
and durations from a kernel trace of the same workload without counters.

The hardware dispatcher the paper changes is not programmable here; what the
host controls is which CUs each phase's stream may use (CU masks) and how
many workgroups a VLM grid has. plan_cu_split predicts, from the descriptors,
the per-frame time of the two-phase pipeline for every split of the CUs and
returns the best one.

This module is pure Python (no GPU): the profiling driver in
profile_intensity.py produces its inputs.
"""
from __future__ import annotations

import csv
import json
import math
from collections import defaultdict
from typing import Dict, Iterable, List, Optional, Tuple

# MI355X peaks (dense): MFMA bf16 2.5 PFLOP/s, fp32 matrix and vector fp32
# 157.3 TFLOP/s, HBM3E 8 TB/s
PEAK_MFMA_BF16 = 2.5e15
PEAK_MFMA_F32 = 157.3e12
PEAK_VALU_F32 = 157.3e12
PEAK_HBM = 8.0e12
NUM_CUS = 256
LEVELS = 15

Key = Tuple[str, int, int]  # (kernel symbol, workgroups, threads per workgroup)


def quantize(frac: float) -> int:
    """Fraction of peak -> 4-bit level 0..15: round(15 * frac), clamped to
    [0, 15] (a fraction above 1, possible from counter noise, is level 15)."""
    if not frac > 0.0:  # also catches NaN
        return 0
    return min(LEVELS, int(math.floor(LEVELS * frac + 0.5)))


def _key(row: dict) -> Key:
    if "Grid_Size" in row:  # counter collection rows
        grid, wg = int(row["Grid_Size"]), int(row["Workgroup_Size"])
    else:  # kernel trace rows
        grid, wg = int(row["Grid_Size_X"]), int(row["Workgroup_Size_X"])
    return (row["Kernel_Name"], grid // max(wg, 1), wg)


def read_trace(path: str) -> Dict[Key, List[float]]:
    """Kernel trace CSV -> durations in seconds per launch configuration."""
    out: Dict[Key, List[float]] = defaultdict(list)
    with open(path, newline="") as f:
        for r in csv.DictReader(f):
            out[_key(r)].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9)
    return dict(out)


# rocprofv3's VGPR_Count on gfx950 is half the registers per lane the
# kernel allocates (VGPRs and AGPRs together), and its Accum_VGPR_Count is 0:
# compared with the compiler's resource report of the same code objects
# (141 -> 72, 249 -> 128, 359 -> 180, 142 -> 72), so the count is doubled.
TRACE_VGPR_SCALE = 2


def read_resources(path: str) -> Dict[Key, Tuple[int, int, int]]:
    """Kernel trace CSV -> (LDS bytes, VGPRs, AGPRs) per workgroup / wave of
    each launch configuration (registers per lane as allocated)."""
    out = {}
    with open(path, newline="") as f:
        for r in csv.DictReader(f):
            out.setdefault(_key(r), (int(r.get("LDS_Block_Size") or 0),
                                     TRACE_VGPR_SCALE * int(r.get("VGPR_Count") or 0),
                                     TRACE_VGPR_SCALE * int(r.get("Accum_VGPR_Count") or 0)))
    return out


# CDNA4 compute unit: 4 SIMDs, 512 VGPRs (arch + accumulation) per lane per
# SIMD, at most 8 waves per SIMD, 160 KB of LDS
CU_SIMDS, SIMD_REGS, SIMD_WAVES, CU_LDS = 4, 512, 8, 160 * 1024


def reg_share(wg_threads: int, vgpr: int, agpr: int) -> float:
    """Share of a CU's register file one workgroup holds: its waves times the
    registers per lane (VGPRs + AGPRs, allocated in granules of 8), over the
    4 SIMDs x 512 registers per lane."""
    waves = max(1, -(-wg_threads // 64))
    regs = -(-(vgpr + agpr) // 8) * 8
    return waves * regs / float(CU_SIMDS * SIMD_REGS)


def wgs_per_cu(wg_threads: int, lds: int, vgpr: int, agpr: int) -> int:
    """Workgroups of one launch configuration that fit on a CU at once."""
    waves = max(1, -(-wg_threads // 64))
    regs = max(8, -(-(vgpr + agpr) // 8) * 8)
    per_simd = min(SIMD_WAVES, SIMD_REGS // regs)
    by_regs = (per_simd * CU_SIMDS) // waves if waves <= CU_SIMDS else per_simd // -(-waves // CU_SIMDS)
    by_lds = CU_LDS // lds if lds > 0 else by_regs
    return max(1, min(by_regs, by_lds))


def read_counters(path: str) -> Dict[Key, Dict[str, float]]:
    """Counter collection CSV -> per launch configuration, the mean over its
    dispatches of each counter (one row per dispatch and counter)."""
    per: Dict[Key, Dict[str, List[float]]] = defaultdict(lambda: defaultdict(list))
    with open(path, newline="") as f:
        for r in csv.DictReader(f):
            per[_key(r)][r["Counter_Name"]].append(float(r["Counter_Value"]))
    return {k: {c: sum(v) / len(v) for c, v in cs.items()} for k, cs in per.items()}


def copy_scale(counters: Dict[Key, Dict[str, float]], counter: str, true_kib: float) -> float:
    """Scale factor true / counted for `counter` from the largest copy-like
    kernel of a calibration run that moved `true_kib` KiB each way."""
    best = None
    for k, cs in counters.items():
        name = k[0].lower()
        if counter in cs and ("copy" in name or "elementwise" in name):
            if best is None or cs[counter] > best:
                best = cs[counter]
    if not best:
        raise ValueError(f"no copy kernel with {counter} in the calibration run")
    return true_kib / best


def frame_counts(small: Dict[Key, List[float]], large: Dict[Key, List[float]], extra_frames: int) -> Dict[Key, float]:
    """Launches per frame of each configuration from two traces of the same
    workload that differ by `extra_frames` frames: whatever runs once per
    workload (model and context set-up, a prefill before the action loops)
    cancels."""
    out = {}
    for k, v in large.items():
        n = (len(v) - len(small.get(k, ()))) / extra_frames
        if n > 0:
            out[k] = n
    return out


def descriptors(trace: Dict[Key, List[float]], alu: Dict[Key, Dict[str, float]],
                fetch: Dict[Key, Dict[str, float]], write: Dict[Key, Dict[str, float]],
                fetch_scale: float, write_scale: float, counts: Dict[Key, float], phase: str,
                res: Optional[Dict[Key, Tuple[int, int, int]]] = None) -> List[dict]:
    """One descriptor per launch configuration with a per-frame count and a
    sample in the trace and in every counter pass."""
    out = []
    for k, lpf in counts.items():
        if k not in trace or k not in alu or k not in fetch or k not in write:
            continue
        durs = trace[k]
        t = sum(durs) / len(durs)
        if t <= 0:
            continue
        c = alu[k]
        tc_frac = (512.0 * c.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0) / t / PEAK_MFMA_BF16 +
                   512.0 * c.get("SQ_INSTS_VALU_MFMA_MOPS_F32", 0.0) / t / PEAK_MFMA_F32)
        alu_frac = (c.get("SQ_INSTS_VALU_FLOPS_FP32", 0.0) + c.get("SQ_INSTS_VALU_FLOPS_FP32_TRANS", 0.0)) / t / PEAK_VALU_F32
        mem_bytes = 1024.0 * (fetch[k].get("FETCH_SIZE", 0.0) * fetch_scale + write[k].get("WRITE_SIZE", 0.0) * write_scale)
        mem_frac = mem_bytes / t / PEAK_HBM
        lds, vgpr, agpr = (res or {}).get(k, (0, 0, 0))
        out.append({
            "kernel": k[0], "workgroups": k[1], "wg_threads": k[2], "phase": phase,
            "vgpr": vgpr, "agpr": agpr, "lds": lds,
            "wgs_per_cu": wgs_per_cu(k[2], lds, vgpr, agpr) if vgpr else 1,
            "launches_per_frame": lpf, "us": t * 1e6,
            "frac": [tc_frac, alu_frac, mem_frac],
            "tau": [quantize(tc_frac), quantize(alu_frac), quantize(mem_frac)],
        })
    out.sort(key=lambda d: -d["us"] * d["launches_per_frame"])
    return out


def save(path: str, desc: List[dict], meta: dict) -> None:
    with open(path, "w") as f:
        json.dump({"meta": meta, "descriptors": desc}, f, indent=1)


def load(path: str) -> List[dict]:
    with open(path) as f:
        return json.load(f)["descriptors"]


# ---------------------------------------------------------------------------
# CU-split planner
# ---------------------------------------------------------------------------

def kernel_time(d: dict, cus: int, rho: float = 0.0, num_cus: int = NUM_CUS) -> float:
    """Predicted time (s) of one launch configuration's launches per frame on
    `cus` CUs, alone. Two limits stretch its isolated time t:
      * workgroup slots: t * min(G, num_cus o) / (cus o) when its G
        workgroups (o per CU) no longer fit at once;
      * bandwidth per CU: a kernel that reached a fraction f of HBM peak on
        all CUs gets at most rho * cus / num_cus of the peak on `cus` CUs
        (rho: how far a CU can pull above its even share), so
        t * f num_cus / (rho cus) when that is larger (rho = 0: no limit)."""
    o = max(1, d.get("wgs_per_cu", 1))
    had = min(d["workgroups"], num_cus * o)
    slot = max(1.0, had / (cus * o))
    bw = max(1.0, d["frac"][2] * num_cus / (rho * cus)) if rho > 0 else 1.0
    return d["launches_per_frame"] * d["us"] * 1e-6 * max(slot, bw)


def phase_time(desc: Iterable[dict], phase: str, cus: int, num_cus: int = NUM_CUS, rho: float = 0.0) -> float:
    """Predicted time (s) of one frame's kernels of `phase` alone on `cus`
    CUs (the sum of kernel_time)."""
    return sum(kernel_time(d, cus, rho, num_cus) for d in desc if d["phase"] == phase)


def mem_level(desc: Iterable[dict], phase: str) -> float:
    """Time-weighted mean DRAM fraction of a phase's kernels."""
    w = s = 0.0
    for d in desc:
        if d["phase"] == phase:
            dt = d["launches_per_frame"] * d["us"]
            w += dt
            s += dt * d["frac"][2]
    return s / w if w else 0.0


def predict_split(desc: List[dict], vlm_cus: int, num_cus: int = NUM_CUS, cal: Optional[dict] = None) -> dict:
    """Per-frame time of the pipelined two-phase schedule (prefill of frame
    r + 1 beside the actions of frame r) with the VLM stream on vlm_cus CUs
    and the action stream on the rest.

    Each phase's time alone on its CUs is phase_time (with the calibrated
    rho); running beside each other, the longer phase sets the period and a
    share kappa of the shorter one does not overlap (it contends for the
    shared HBM, L2 and MALL the CU sets do not partition):
        period = max(t_v, t_a) + kappa min(t_v, t_a).
    Without a calibration rho = 0 and kappa = max(0, hbm_v + hbm_a - 1)
    (the phases' summed mean HBM fractions beyond 1)."""
    act_cus = num_cus - vlm_cus
    share = mem_level(desc, "vlm") + mem_level(desc, "action")
    rho = cal["rho"] if cal else 0.0
    kappa = cal["kappa"] if cal else max(0.0, share - 1.0)
    tv = phase_time(desc, "vlm", vlm_cus, num_cus, rho)
    ta = phase_time(desc, "action", act_cus, num_cus, rho)
    per_frame = max(tv, ta) + kappa * min(tv, ta)
    return {"vlm_cus": vlm_cus, "act_cus": act_cus, "vlm_s": tv, "action_s": ta,
            "hbm_share": share, "per_frame_s": per_frame}


def fit_calibration(desc: List[dict], measured: Dict[int, float], num_cus: int = NUM_CUS) -> dict:
    """(rho, kappa) minimising the largest relative error of predicted
    against measured frames/s over the measured splits ({vlm_cus: frames/s}
    of the pipelined schedule); grid search, rho in (0, 3], kappa in [0, 1]."""
    best = None
    for i in range(1, 61):
        rho = 0.05 * i
        tv = {v: phase_time(desc, "vlm", v, num_cus, rho) for v in measured}
        ta = {v: phase_time(desc, "action", num_cus - v, num_cus, rho) for v in measured}
        for j in range(0, 101):
            kappa = 0.01 * j
            err = max(abs(1.0 / (max(tv[v], ta[v]) + kappa * min(tv[v], ta[v])) / fps - 1.0)
                      for v, fps in measured.items())
            if best is None or err < best["max_rel_err"] - 1e-12:
                best = {"rho": rho, "kappa": kappa, "max_rel_err": err}
    best["measured_fps"] = {str(v): f for v, f in measured.items()}
    return best


def plan_cu_split(desc: List[dict], num_cus: int = NUM_CUS, step: int = 8, cal: Optional[dict] = None) -> dict:
    """The split (multiples of `step`, both phases at least `step` CUs) with
    the smallest predicted per-frame time; ties go to more VLM CUs."""
    best = None
    for v in range(num_cus - step, step - 1, -step):
        p = predict_split(desc, v, num_cus, cal)
        if best is None or p["per_frame_s"] < best["per_frame_s"] * (1 - 1e-12):
            best = p
    return best


def load_calibration(path: str) -> Optional[dict]:
    with open(path) as f:
        return json.load(f)["meta"].get("calibration")
