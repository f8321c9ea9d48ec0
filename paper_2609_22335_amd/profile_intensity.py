"""Offline profiling pass: intensity descriptors of every kernel of a preset.

    python paper_2609_22335_amd/profile_intensity.py --preset pi0 \
        --out profiles/intensity_pi0.json --work intensity_work/pi0

Runs on a machine with the GPU and rocprofv3. Each phase of one frame runs
on its own (the VLM prefill of frames, or the action loop of one frame over a
prefilled context), on one stream with nothing beside it, so every kernel
runs in isolation, as the paper's offline pass requires. rocprofv3 runs as a
child process, one pass per counter group (a pass holds at most 8 SQ and 4
TCC counters): a kernel trace for durations, then MFMA / fp32 VALU counters,
then FETCH_SIZE, then WRITE_SIZE; a plain device copy of known size scales
the two byte counters. Launches per frame come from the difference of two
traces that differ by two frames. The descriptors (intensity.py) go to
`--out`, followed by the CU split that intensity.plan_cu_split picks for the
one-frame pipeline; with `--fit` the planner is first calibrated on the
measured CU splits of a bench.py run (intensity.fit_calibration).

With `--run vlm|action|copy` the script is the profiled workload itself.
"""
from __future__ import annotations

import argparse
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
sys.path.insert(0, ROOT)
sys.path.insert(0, HERE)

# pure Python, imported on its own: the driver process never loads the GPU
# library (the profiled workloads are child processes)
import intensity  # noqa: E402

ALU_COUNTERS = ["SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_INSTS_VALU_MFMA_MOPS_F32", "SQ_INSTS_VALU_FLOPS_FP32",
                "SQ_INSTS_VALU_FLOPS_FP32_TRANS", "SQ_INSTS_VALU_ADD_F32", "SQ_INSTS_VALU_MUL_F32",
                "SQ_INSTS_VALU_FMA_F32", "SQ_INSTS_VALU_TRANS_F32"]
COPY_MIB = 256
SMALL, LARGE = 1, 3  # frames of the two traces


def run_workload(kind: str, preset: str, frames: int) -> None:
    import numpy as np
    import torch
    import paper_2609_22335_amd as V
    import synth
    if kind == "copy":
        n = COPY_MIB << 20
        x = torch.empty(n, dtype=torch.uint8, device="cuda")
        y = torch.empty_like(x)
        for _ in range(3):
            y.copy_(x)
        torch.cuda.synchronize()
        return
    cfg = V.vla_preset(preset)
    m = V.vla_create(cfg, 0)
    c = V.vla_ctx_create(m)
    fr = synth.make_frame(cfg, 0, 0)
    pix = torch.from_numpy(fr["pixels"]).cuda()
    ids = torch.from_numpy(fr["ids"]).cuda()
    st = torch.from_numpy(fr["state"]).cuda() if fr["state"].size else None
    frame = V.make_frame(pix, ids, st)
    noise = torch.from_numpy(np.ascontiguousarray(fr["noise"])).cuda()
    out = torch.empty_like(noise)
    if kind == "vlm":
        for _ in range(frames):
            V.vla_vlm_prefill(m, frame, c)
            torch.cuda.synchronize()
    else:
        V.vla_vlm_prefill(m, frame, c)
        torch.cuda.synchronize()
        for _ in range(frames):
            V.vla_action_denoise(m, c, noise, out)
            torch.cuda.synchronize()
    V.vla_ctx_destroy(c)
    V.vla_destroy(m)


def rocprof(work: str, name: str, args, pmc=None, timeout=240) -> str:
    """One rocprofv3 pass over `args` (a workload command line); returns the
    output folder."""
    d = os.path.join(work, name)
    cmd = ["timeout", "-s", "KILL", str(timeout), "rocprofv3"]
    if pmc:
        cmd += ["--pmc", *pmc]
    cmd += ["--kernel-trace", "-f", "csv", "-d", d, "-o", "run", "--", sys.executable, *args]
    print("[intensity]", name, flush=True)
    with open(os.path.join(work, name + ".log"), "w") as log:
        subprocess.run(cmd, check=True, stdout=log, stderr=subprocess.STDOUT, cwd="/tmp",
                       env=dict(os.environ, TMPDIR="/tmp"))
    return d


def measured_splits(path: str, preset: str = "") -> dict:
    """{VLM CUs: frames/s} of the CU-split schedules (cu_V_A) in a bench.py
    detail file: those of the further workload named <preset>_R<R> when the
    file holds one, else those of its main workload."""
    import json
    import re
    d = json.load(open(path))
    modes = d["modes"]
    for name, w in (d.get("other_workloads") or {}).items():
        if preset and re.fullmatch(re.escape(preset) + r"_R\d+", name):
            modes = w["modes"]
            break
    out = {}
    for name, r in modes.items():
        parts = name.split("_")
        if len(parts) == 3 and parts[0] == "cu" and parts[1].isdigit() and parts[2].isdigit():
            out[int(parts[1])] = r["frames_per_s"]
    return out


def profile(preset: str, out: str, work: str, collect: bool = True, fit: str = "") -> None:
    """Run the passes (collect) and build the descriptor file from their
    outputs under `work`; with collect=False only the second part. With
    `fit` (a bench.py detail file holding cu_V_A schedules of the same
    preset), the planner's calibration is fitted to those measured splits
    and stored with the descriptors."""
    out, work = os.path.abspath(out), os.path.abspath(work)  # the passes run in /tmp
    os.makedirs(work, exist_ok=True)
    me = os.path.abspath(__file__)
    wl = lambda kind, n: [me, "--run", kind, "--preset", preset, "--frames", str(n)]  # noqa: E731
    passes = [("copy_FETCH_SIZE", wl("copy", 0), ["FETCH_SIZE"]), ("copy_WRITE_SIZE", wl("copy", 0), ["WRITE_SIZE"])]
    for phase in ("vlm", "action"):
        passes += [(f"{phase}_trace_{SMALL}", wl(phase, SMALL), None), (f"{phase}_trace_{LARGE}", wl(phase, LARGE), None),
                   (f"{phase}_alu", wl(phase, LARGE), ALU_COUNTERS), (f"{phase}_fetch", wl(phase, LARGE), ["FETCH_SIZE"]),
                   (f"{phase}_write", wl(phase, LARGE), ["WRITE_SIZE"])]
    if collect:
        for name, args, pmc in passes:
            rocprof(work, name, args, pmc)
    csvf = lambda name, what: os.path.join(work, name, f"run_{what}.csv")  # noqa: E731
    calib = {c: intensity.copy_scale(intensity.read_counters(csvf(f"copy_{c}", "counter_collection")), c,
                                     COPY_MIB * 1024.0) for c in ("FETCH_SIZE", "WRITE_SIZE")}
    desc = []
    for phase in ("vlm", "action"):
        small = intensity.read_trace(csvf(f"{phase}_trace_{SMALL}", "kernel_trace"))
        large = intensity.read_trace(csvf(f"{phase}_trace_{LARGE}", "kernel_trace"))
        res = intensity.read_resources(csvf(f"{phase}_trace_{LARGE}", "kernel_trace"))
        counts = intensity.frame_counts(small, large, LARGE - SMALL)
        alu, fetch, write = (intensity.read_counters(csvf(f"{phase}_{p}", "counter_collection"))
                             for p in ("alu", "fetch", "write"))
        desc += intensity.descriptors(large, alu, fetch, write, calib["FETCH_SIZE"], calib["WRITE_SIZE"], counts, phase,
                                      res)
    cal = intensity.fit_calibration(desc, measured_splits(fit, preset)) if fit else None
    plan = intensity.plan_cu_split(desc, cal=cal)
    meta = {"preset": preset, "calibration": cal, "peaks": {"mfma_bf16": intensity.PEAK_MFMA_BF16, "mfma_f32": intensity.PEAK_MFMA_F32,
                                        "valu_f32": intensity.PEAK_VALU_F32, "hbm": intensity.PEAK_HBM},
            "counters": ALU_COUNTERS + ["FETCH_SIZE", "WRITE_SIZE"], "byte_scale": calib,
            "frames": [SMALL, LARGE], "cu_split_plan": plan}
    intensity.save(out, desc, meta)
    print(f"[intensity] {len(desc)} launch configurations -> {out}; planned CU split VLM/action "
          f"{plan['vlm_cus']}/{plan['act_cus']}, predicted {1.0 / plan['per_frame_s']:.1f} frames/s", flush=True)


def refit(preset: str, path: str, fit: str) -> None:
    """Fit the planner's calibration of an existing descriptor file to the
    measured CU splits of a bench.py detail file and store it, with the split
    the calibrated planner then picks, in the file (CPU only)."""
    import json
    d = json.load(open(path))
    desc, meta = d["descriptors"], d["meta"]
    cal = intensity.fit_calibration(desc, measured_splits(fit, preset))
    plan = intensity.plan_cu_split(desc, cal=cal)
    meta["calibration"], meta["cu_split_plan"] = cal, plan
    intensity.save(path, desc, meta)
    print(f"[intensity] {path}: rho {cal['rho']:.2f}, kappa {cal['kappa']:.2f}, largest error "
          f"{100 * cal['max_rel_err']:.1f}% over {len(cal['measured_fps'])} splits; planned CU split VLM/action "
          f"{plan['vlm_cus']}/{plan['act_cus']}, predicted {1.0 / plan['per_frame_s']:.1f} frames/s", flush=True)


def main() -> None:
    ap = argparse.ArgumentParser()
    ap.add_argument("--preset", default="pi0")
    ap.add_argument("--out", default="intensity.json")
    ap.add_argument("--work", default="intensity_work")
    ap.add_argument("--run", choices=["vlm", "action", "copy"], help="be the profiled workload")
    ap.add_argument("--frames", type=int, default=LARGE)
    ap.add_argument("--build-only", action="store_true", help="only build the file from the passes under --work")
    ap.add_argument("--fit", default="", help="bench.py detail file with cu_V_A schedules: fit the planner to them")
    ap.add_argument("--fit-only", action="store_true", help="only fit the descriptor file --out to --fit (CPU)")
    a = ap.parse_args()
    if a.run:
        run_workload(a.run, a.preset, a.frames)
    elif a.fit_only:
        if not a.fit:
            ap.error("--fit-only needs --fit")
        refit(a.preset, a.out, a.fit)
    else:
        profile(a.preset, a.out, a.work, collect=not a.build_only, fit=a.fit)


if __name__ == "__main__":
    main()
