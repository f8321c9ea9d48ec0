#!/usr/bin/env python
"""Benchmark of the two-phase VLA hot path on one MI355X.

Workload: the PaliGemma-3B-shaped VLM (27-layer ViT, d=1152, 256 patches of
a 224x224 image; 18-layer LM, d=2048, 8 query heads / 1 KV head of 256,
GeGLU 16384, prefix 256 image + 48 text + 1 state token) with a pi0-shaped
flow-matching expert (18 layers, d=1024, GeGLU 4096, chunk 50x32, 10 Euler
steps), bf16, R=8 independent robot request streams (a new seeded frame per
stream). One step = vla_pipeline_run over the R frames. Inputs are resident
in HBM before the timed region.

Schedules (``--modes``): the paper's serialized and naive two-stream ones,
CU masks, VLM workgroup caps, HIP graphs, several action lanes, and batched
prefills / action loops (several robots' frames through one pass). In a
schedule whose prefills come in two or more groups (one-frame prefills, or
groups smaller than R) a later group's prefill runs while an earlier
group's action loop runs on another stream; with one prefill group of all R
frames the action loops start after it. A cross-step schedule (``xs_``
prefix) runs the timed steps as one pipeline over steps x R frames (robot
r's frame of step j at index j R + r), so step j + 1's prefills overlap step
j's action loops, as R robots streaming frames would; every step's chunks
are checked to equal the first step's.

`value` is the frames/s of the schedule named by ``--mode`` (fixed in
advance, not the fastest measured one); the line also gives its speedup over
the one-frame serialized schedule and over the serialized schedule with the
same batching, and `best_overlapped`: the fastest schedule in which the two
phases overlap, with the per-CU residency of both phases measured from the
kernels' workgroup logs.

Output: the last stdout line is a compact JSON headline (a few KB): metric,
value, roofline of the dominant kernel (timed live with HIP events on its own
stream), the fp64 CPU oracle timed on this host as a baseline. Every
schedule's numbers, the residency logs and the further workloads
(``--extra``) go to ``--detail`` (a JSON file) and to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "VLA frames/sec & actions/sec at R robot streams; MFMA util; speedup vs serialized"
HBM_PEAK_GBS = 8000.0      # MI355X HBM3E, GB/s
BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA, TFLOP/s


def kernel_work(cfg, tag, vlm_frames=1, act_frames=1):
    """Algorithmic bytes and flops of one launch of a tagged kernel: weights,
    the A operand and the output (plus the fp32 residual read and write for
    residual epilogues) each moved once; flops = 2 M N K. A batched prefill
    stacks vlm_frames frames' rows into M, a batched action loop act_frames."""
    import synth
    d = synth.derived(cfg)
    H, P = cfg["chunk_len"] * act_frames, d["prefix"] * vlm_frames
    vit_rows = cfg["n_views"] * d["tokens_per_view"] * vlm_frames  # ViT rows (before any pixel shuffle)
    qd, kvd = cfg["lm_heads"] * cfg["head_dim"], cfg["lm_kv_heads"] * cfg["head_dim"]
    shapes = {  # tag: (M, N, K, output bytes per element, residual?)
        "ex.gateup": (H, 2 * cfg["ex_mlp"], cfg["ex_dim"], 2, False),
        "ex.down": (H, cfg["ex_dim"], cfg["ex_mlp"], 4, True),
        "ex.qkv": (H, qd + 2 * kvd, cfg["ex_dim"], 2, False),
        "ex.o": (H, cfg["ex_dim"], qd, 4, True),
        "lm.gateup": (P, 2 * cfg["lm_mlp"], cfg["lm_dim"], 2, False),
        "lm.down": (P, cfg["lm_dim"], cfg["lm_mlp"], 4, True),
        "lm.qkv": (P, qd + 2 * kvd, cfg["lm_dim"], 2, False),
        "lm.o": (P, cfg["lm_dim"], qd, 4, True),
        "vit.fc1": (vit_rows, cfg["vit_mlp"], cfg["vit_dim"], 2, False),
        "vit.fc2": (vit_rows, cfg["vit_dim"], cfg["vit_mlp"], 4, True),
    }
    M, N, K, ob, resid = shapes[tag]
    nout = N // 2 if tag.endswith("gateup") else N
    byts = 2 * N * K + 2 * M * K + (8 if resid else ob) * M * nout
    return byts, 2.0 * M * N * K


def cu_residency(rec, window=None):
    """Per-CU residency from workgroup start/end records (vla_wavelog_read).

    CU = (XCC, shader engine, shader array, CU) from the hardware-id
    registers; the phase of a record is that of its hardware queue (the
    VLM's queues are those that ran a kernel kind only the prefill has:
    ViT attention and its combine, patchify, text embedding). Returns the
    mean over CUs of the fraction of the window in which the CU hosts at
    least one workgroup, and in which it hosts workgroups of both phases."""
    import numpy as np
    hw = rec["hwid"].astype(np.int64)
    cu = rec["xcc"].astype(np.int64) * 256 + ((hw >> 13) & 7) * 32 + ((hw >> 12) & 1) * 16 + ((hw >> 8) & 15)
    queue = ((hw >> 30) & 3) * 64 + ((hw >> 6) & 3) * 8 + ((hw >> 24) & 7)
    vlm_q = np.unique(queue[np.isin(rec["kind"], (4, 5, 8, 9))])  # ViT attention, combine, patchify, embed
    is_vlm = np.isin(queue, vlm_q)
    t = rec["t"].astype(np.int64)
    d = np.where(rec["end"] == 1, -1, 1)
    if window is None:
        if is_vlm.any() and (~is_vlm).any():
            lo = max(t[is_vlm].min(), t[~is_vlm].min())
            hi = min(t[is_vlm].max(), t[~is_vlm].max())
        else:
            lo, hi = t.min(), t.max()
    else:
        lo, hi = window
    order = np.lexsort((d, t, cu))  # ends before starts at equal times
    cu, t, dv, da = cu[order], t[order], (d * is_vlm)[order], (d * ~is_vlm)[order]
    cv, ca = np.cumsum(dv), np.cumsum(da)
    # restart the running counts at each CU boundary
    first = np.r_[True, cu[1:] != cu[:-1]]
    seg = np.cumsum(first) - 1
    base_v = (cv - dv)[first][seg]
    base_a = (ca - da)[first][seg]
    nv, na = cv - base_v, ca - base_a
    nxt = np.r_[t[1:], t[-1]]
    same = np.r_[cu[1:] == cu[:-1], False]
    dur = np.clip(np.minimum(nxt, hi) - np.maximum(t, lo), 0, None) * same
    ncu = len(np.unique(cu))
    span = max(hi - lo, 1)
    busy = float(((nv + na) > 0) @ dur) / (span * ncu)
    both = float(((nv > 0) & (na > 0)) @ dur) / (span * ncu)
    return {"cus": int(ncu), "window_ms": float(span) * 1e-5, "busy_frac": float(busy),
            "both_phases_frac": float(both), "vlm_queues": int(len(vlm_q))}


def cpu_baseline(cfg, seed):
    """The fp64 oracle on one frame of the same workload (full VLM prefill
    and the 10-step denoising of that frame); frames/s = 1 / its time."""
    import numpy as np
    import synth
    from oracle import vla_oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:  # threadpoolctl missing: report the host CPU count
        threads = os.cpu_count() or 1
    print("[bench] cpu baseline: generating oracle parameters", file=sys.stderr, flush=True)
    P = synth.make_params(cfg, seed)
    fr = synth.make_frame(cfg, seed, 0)
    print("[bench] cpu baseline: timing oracle forward of frame 0", file=sys.stderr, flush=True)
    t0 = time.perf_counter()
    chunk = O.forward(P, cfg, fr)
    dt = time.perf_counter() - t0
    del P
    return {"value": 1.0 / dt, "unit": "frames/s", "cores": int(threads), "kind": "oracle",
            "sample": f"frame 0 of the workload: full VLM prefill + {cfg['n_steps']}-step action "
                      f"denoising, fp64 NumPy, {dt:.1f} s", "seconds": dt, "blas_threads": int(threads),
            "os_cpu_count": os.cpu_count()}, chunk


def measured_traffic(preset, R, kernel, schedule):
    """HBM bytes per launch of `kernel` from the committed counter record
    (FETCH_SIZE + WRITE_SIZE, each scaled by a plain copy's reading), or
    None when the record is for another workload or schedule, or the kernel
    source has changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"{kernel.replace('.', '_')}_{preset}_R{R}_{schedule}_traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if kernel_source_digest() != rec["kernels_code_sha256"]:
        return None
    return rec["traffic_bytes_per_launch"]


def kernel_source_digest():
    """sha256 of the kernel source with comments and whitespace removed: any
    code change (in any kernel) changes it, a comment edit does not."""
    import hashlib
    import re
    src = open(os.path.join(ROOT, "paper_2609_22335_amd", "csrc", "kernels.hip")).read()
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    return hashlib.sha256(" ".join(src.split()).encode()).hexdigest()


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--R", type=int, default=8, help="robot request streams (frames per step)")
    ap.add_argument("--mode", default="xs_vb8_ab8_lanes2_graph",
                    help="schedule reported as `value` (auto: the fastest measured one)")
    ap.add_argument("--modes", default="serial,concurrent,cu_masked,wg_capped,serial_graph,"
                                       "concurrent_graph,lanes2_graph,lanes3_graph,batch2_graph,"
                                       "batch2_lanes2_graph,batch4_graph,batch4_lanes2_graph,batch8_graph,"
                                       "vb2_ab2_graph,vb2_ab2_lanes2_graph,vb2_ab4_graph,vb4_ab4_graph,"
                                       "vb4_ab2_lanes2_graph,vb4_ab4_lanes2_graph,vb8_ab8_graph,"
                                       "vb8_ab4_lanes2_graph,vb4_ab4_v2_lanes2_graph,"
                                       "vb8_ab8_lanes2_graph,serial_vb8_ab4_graph,serial_vb4_ab4_graph,"
                                       "serial_vb8_ab8_graph,cu_160_96,cu_auto,xs_lanes2_graph,"
                                       "xs_vb4_ab4_lanes2_graph,xs_vb8_ab4_graph,xs_vb8_ab4_lanes2_graph,"
                                       "xs_vb8_ab8_lanes2_graph")
    ap.add_argument("--detail", default=os.path.join(ROOT, "bench_detail.json"),
                    help="JSON file for every schedule's numbers, residency logs and further workloads")
    ap.add_argument("--split", default="192,64", help="CU split VLM,action for cu_masked")
    ap.add_argument("--wg-cap", type=int, default=2, help="VLM workgroups per CU for wg_capped")
    ap.add_argument("--kernel", default="auto",
                    help="tag of the kernel timed for the roofline (auto: of the candidate tags, the one "
                         "with the most stream time in the reported schedule: summed launch time divided "
                         "by the number of concurrent streams of its phase)")
    ap.add_argument("--preset", default="pi0")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--extra", default="gr00t:8:serial,concurrent,cu_masked,lanes2_graph,v2_lanes2_graph,"
                                       "vb4_ab1_lanes2_graph,vb8_ab1_lanes4_graph,vb4_ab1_v2_lanes2_graph,"
                                       "xs_vb8_ab1_lanes4_graph;"
                                       "pi0_3view:32:serial,concurrent,cu_224_32,cu_192_64,cu_160_96,"
                                       "wg_cap1,wg_cap2,lanes2_graph,cu_160_96_lanes2,batch4_lanes2_graph,"
                                       "batch8_lanes2_graph,vb4_ab4_lanes2_graph,vb8_ab4_lanes2_graph,"
                                       "vb8_ab8_lanes2_graph,xs_vb8_ab8_lanes2_graph;"
                                       "pi0:8:async2_serial,async2_lanes2_graph,async2_vb8_ab4_lanes2_graph,"
                                       "async2_vb8_ab8_lanes2_graph,async4_serial,async4_vb8_ab8_lanes2_graph,"
                                       "xs_async2_vb8_ab8_lanes2_graph;"
                                       "pi0_ddim:8:serial,vb8_ab8_graph,vb8_ab4_lanes2_graph,xs_vb8_ab8_lanes2_graph;"
                                       "cogact:8:serial,concurrent,lanes2_graph,vb8_ab1_lanes2_graph,"
                                       "vb8_ab1_lanes4_graph,xs_vb8_ab1_lanes2_graph,xs_vb8_ab1_lanes4_graph",
                    help="further workloads, ';'-separated preset:R:schedule,schedule,...")
    ap.add_argument("--extra-steps", type=int, default=5)
    ap.add_argument("--residency", type=int, default=8_000_000,
                    help="capacity of the workgroup residency log (0: skip the residency runs)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB five times (the reference "
                         "kernel for scaling the HBM byte counters) and exit")
    args = ap.parse_args()
    if args.calibrate_copy:
        import torch
        n = args.calibrate_copy << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "launches": 5}), flush=True)
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "bench.py measures one GPU; the R robot streams of a "
                                   "multi-GPU deployment shard across GPUs with no exchange step; "
                                   "run with --gpus 1"}), flush=True)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2609_22335_amd as V
    import synth

    torch.cuda.set_device(0)
    cfg = V.vla_preset(args.preset)
    seed, R = 0, args.R
    modes = [m for m in args.modes.split(",") if m]
    if args.mode != "auto" and args.mode not in modes:
        modes.append(args.mode)
    vlm_cus, act_cus = (int(x) for x in args.split.split(","))

    # schedules: the paper's serialized and naive two-stream ones, the two
    # MI355X levers (CU masks, workgroup caps), graph replay, and several
    # action streams for the independent robots' action phases
    kw = {"serial": dict(mode="serial"), "concurrent": dict(mode="concurrent"),
          "cu_masked": dict(mode="cu_masked", vlm_cus=vlm_cus, act_cus=act_cus),
          "wg_capped": dict(mode="wg_capped", vlm_wg_cap=args.wg_cap),
          "serial_graph": dict(mode="serial", graphs=True),
          "concurrent_graph": dict(mode="concurrent", graphs=True),
          "cu_masked_graph": dict(mode="cu_masked", vlm_cus=vlm_cus, act_cus=act_cus, graphs=True),
          "lanes2_graph": dict(mode="concurrent", act_streams=2, graphs=True),
          "lanes3_graph": dict(mode="concurrent", act_streams=3, graphs=True),
          "lanes4_graph": dict(mode="concurrent", act_streams=4, graphs=True),
          "v2_lanes2_graph": dict(mode="concurrent", vlm_streams=2, act_streams=2, graphs=True),
          "v2_lanes3_graph": dict(mode="concurrent", vlm_streams=2, act_streams=3, graphs=True),
          "v2_lanes4_graph": dict(mode="concurrent", vlm_streams=2, act_streams=4, graphs=True),
          # two robots' action phases as one loop that reads the weights once
          "batch2_graph": dict(mode="concurrent", act_batch=2, graphs=True),
          "batch2_lanes2_graph": dict(mode="concurrent", act_batch=2, act_streams=2, graphs=True),
          "batch2_v2_graph": dict(mode="concurrent", act_batch=2, vlm_streams=2, graphs=True)}
    for v_ in (2, 4, 8):  # several robots' prefills as one pass, with action groups
        for a_ in (1, 2, 3, 4, 8):
            kw[f"vb{v_}_ab{a_}_graph"] = dict(mode="concurrent", vlm_batch=v_, act_batch=a_, graphs=True)
            kw[f"vb{v_}_ab{a_}_lanes2_graph"] = dict(mode="concurrent", vlm_batch=v_, act_batch=a_,
                                                     act_streams=2, graphs=True)
            kw[f"vb{v_}_ab{a_}_cu_192_64"] = dict(mode="cu_masked", vlm_cus=192, act_cus=64, vlm_batch=v_,
                                                  act_batch=a_, graphs=True)
            for l_ in (3, 4):
                kw[f"vb{v_}_ab{a_}_lanes{l_}_graph"] = dict(mode="concurrent", vlm_batch=v_, act_batch=a_,
                                                           act_streams=l_, graphs=True)
            kw[f"vb{v_}_ab{a_}_v2_lanes2_graph"] = dict(mode="concurrent", vlm_batch=v_, act_batch=a_,
                                                        vlm_streams=2, act_streams=2, graphs=True)
            for c_ in (1, 2, 3):  # VLM workgroups capped at c_ per CU
                kw[f"vb{v_}_ab{a_}_lanes2_cap{c_}_graph"] = dict(mode="wg_capped", vlm_wg_cap=c_, vlm_batch=v_,
                                                                act_batch=a_, act_streams=2, graphs=True)
            for cv_, ca_ in ((224, 32), (192, 64)):  # disjoint CU sets
                kw[f"vb{v_}_ab{a_}_lanes2_cu_{cv_}_{ca_}_graph"] = dict(
                    mode="cu_masked", vlm_cus=cv_, act_cus=ca_, vlm_batch=v_, act_batch=a_, act_streams=2,
                    graphs=True)
    # asynchronous inference: k action chunks per VLM output
    for k_ in (2, 4):
        kw[f"async{k_}_serial"] = dict(mode="serial", act_chunks=k_)
        kw[f"async{k_}_lanes2_graph"] = dict(mode="concurrent", act_streams=2, graphs=True, act_chunks=k_)
        kw[f"async{k_}_vb8_ab4_lanes2_graph"] = dict(mode="concurrent", vlm_batch=8, act_batch=4, act_streams=2,
                                                   graphs=True, act_chunks=k_)
        kw[f"async{k_}_vb8_ab8_lanes2_graph"] = dict(mode="concurrent", vlm_batch=8, act_batch=8, act_streams=2,
                                                   graphs=True, act_chunks=k_)
    for b_ in (4, 8):  # larger groups of robots per action loop
        kw[f"batch{b_}_graph"] = dict(mode="concurrent", act_batch=b_, graphs=True)
        kw[f"batch{b_}_lanes2_graph"] = dict(mode="concurrent", act_batch=b_, act_streams=2, graphs=True)
        kw[f"batch{b_}_v2_graph"] = dict(mode="concurrent", act_batch=b_, vlm_streams=2, graphs=True)
    for a_, b_ in ((224, 32), (192, 64), (160, 96), (128, 128), (96, 160)):  # CU-split sweep entries
        kw[f"cu_{a_}_{b_}"] = dict(mode="cu_masked", vlm_cus=a_, act_cus=b_)
        kw[f"cu_{a_}_{b_}_lanes2"] = dict(mode="cu_masked", vlm_cus=a_, act_cus=b_, act_streams=2, graphs=True)
        kw[f"cu_{a_}_{b_}_lanes3"] = dict(mode="cu_masked", vlm_cus=a_, act_cus=b_, act_streams=3, graphs=True)
    for c_ in (1, 2, 4):
        kw[f"wg_cap{c_}"] = dict(mode="wg_capped", vlm_wg_cap=c_)
    # cu_auto: the CU split the calibrated planner picks from the preset's
    # intensity descriptors (profiles/intensity_<preset>.json)
    auto_plan = None
    ipath = os.path.join(ROOT, "profiles", f"intensity_{args.preset}.json")
    if os.path.exists(ipath):
        from paper_2609_22335_amd import intensity as IN
        auto_plan = IN.plan_cu_split(IN.load(ipath), cal=IN.load_calibration(ipath))
        kw["cu_auto"] = dict(mode="cu_masked", vlm_cus=auto_plan["vlm_cus"], act_cus=auto_plan["act_cus"])
    elif "cu_auto" in modes:
        modes.remove("cu_auto")
    # serialized with batching: one stream, groups as in the batched schedules
    # (the same outputs bit for bit), the baseline of their concurrency gain
    for v_ in (1, 2, 4, 8):
        for a_ in (1, 2, 4, 8):
            kw[f"serial_vb{v_}_ab{a_}_graph"] = dict(mode="serial", vlm_batch=v_, act_batch=a_, graphs=True)
    # cross-step schedules (xs_<schedule>): the timed steps run as one pipeline
    # over steps x R frames (robot r's frame of step j at index j R + r), so
    # the prefills of step j + 1 run beside the action loops of step j: the
    # steady state of R robots streaming frames under asynchronous inference
    for name_ in list(kw):
        kw["xs_" + name_] = dict(kw[name_], xsteps=True)

    def lib_args(a):
        return {k: v for k, v in a.items() if k != "xsteps"}

    def measure(preset, R, modes, steps, warmup):
        """vla_pipeline_run over R seeded frames of `preset` in each schedule."""
        cfg = V.vla_preset(preset)
        print(f"[bench] creating {preset} model (seed {seed})", file=sys.stderr, flush=True)
        m = V.vla_create(cfg, seed)
        frames_np = [synth.make_frame(cfg, seed, r) for r in range(R)]
        dev = []
        for f in frames_np:
            pix = torch.from_numpy(f["pixels"]).cuda()
            ids = torch.from_numpy(f["ids"]).cuda()
            st = torch.from_numpy(f["state"]).cuda() if f["state"].size else None
            dev.append((pix, ids, st))
        cframes = [V.make_frame(p, i, s) for p, i, s in dev]
        noise = torch.from_numpy(np.stack([f["noise"] for f in frames_np])).cuda().contiguous()
        actions = torch.empty_like(noise)
        chunk_bufs = {1: (noise, actions)}  # k chunks per frame -> (noise, actions) [R k, H, A]

        def bufs(k):
            if k not in chunk_bufs:
                nk = np.stack([synth.chunk_noise(cfg, seed, r, j) for r in range(R) for j in range(k)])
                nt = torch.from_numpy(nk).cuda().contiguous()
                chunk_bufs[k] = (nt, torch.empty_like(nt))
            return chunk_bufs[k]
        xs_bufs = {}

        def xbufs(k, n):
            # noise and outputs of n steps: the same R frames' noise per step
            if (k, n) not in xs_bufs:
                nz = bufs(k)[0]
                nx = nz.repeat(n, 1, 1).contiguous()
                xs_bufs[(k, n)] = (nx, torch.empty_like(nx))
            return xs_bufs[(k, n)]
        results, outputs = {}, {}
        for mode in modes:
            a = kw[mode]
            kc = a.get("act_chunks", 1)
            noise, actions = bufs(kc)
            if a.get("xsteps"):
                # one call over all steps' frames; the warm-up call has as
                # many frames, so every graph the timed call replays is
                # captured before it
                print(f"[bench] {preset} mode {mode}: {steps} steps of R={R} as one pipeline (warm-up: the "
                      f"same)", file=sys.stderr, flush=True)
                nx, ax = xbufs(kc, steps)
                fx = cframes * steps
                V.vla_pipeline_run(m, fx, nx, R * steps, actions=ax, **lib_args(a))
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                t = V.vla_pipeline_run(m, fx, nx, R * steps, actions=ax, **lib_args(a))
                torch.cuda.synchronize()
                el = time.perf_counter() - t0
                lib_ms = [t["wall_ms"] / steps]
                per_frame = R * steps
                out_all = ax.cpu().numpy().reshape(steps, R * kc, *ax.shape[1:])
                outputs[mode] = out_all[0].copy()
                steps_same = all(np.array_equal(out_all[j], out_all[0]) for j in range(1, steps))
            else:
                print(f"[bench] {preset} mode {mode}: {warmup} warmup + {steps} timed steps of R={R}",
                      file=sys.stderr, flush=True)
                for _ in range(warmup):
                    V.vla_pipeline_run(m, cframes, noise, R, actions=actions, **a)
                torch.cuda.synchronize()
                lib_ms = []
                t0 = time.perf_counter()
                for _ in range(steps):
                    t = V.vla_pipeline_run(m, cframes, noise, R, actions=actions, **a)
                    lib_ms.append(t["wall_ms"])
                torch.cuda.synchronize()
                el = time.perf_counter() - t0
                per_frame = R
                outputs[mode] = actions.cpu().numpy().copy()
                steps_same = None
            fps = steps * R / el
            results[mode] = {"frames_per_s": fps, "actions_per_s": fps * kc * cfg["chunk_len"],
                             "chunks_per_frame": kc,
                             "ms_per_step": 1e3 * el / steps,
                             "median_step_ms": float(np.median(lib_ms)), "min_step_ms": float(np.min(lib_ms)),
                             "vlm_ms_per_frame": t["vlm_ms"] / per_frame,
                             "action_ms_per_frame": t["act_ms"] / per_frame}
            if steps_same is not None:
                results[mode]["steps_identical"] = steps_same
        # speedup over the serialized schedule with as many chunks per frame
        for mode in results:
            kc = kw[mode].get("act_chunks", 1)
            ser = results.get("serial" if kc == 1 else f"async{kc}_serial", {}).get("frames_per_s")
            results[mode]["speedup_vs_serialized"] = (results[mode]["frames_per_s"] / ser) if ser else None
        # Batched action loops (groups of >= 2 frames) run tiled GEMMs over
        # the stacked rows: identical among themselves, within the oracle
        # tolerance of the one-frame path; every other schedule is identical
        # to the one-frame path.
        def grp(mode):
            b, kc = kw[mode].get("act_batch", 1), kw[mode].get("act_chunks", 1)
            g_ = "batched" if b > 1 and (R * kc) % b != 1 else "one_frame"
            return g_ if kc == 1 else f"{g_}_{kc}_chunks"
        identical = {}
        for g_ in sorted({grp(m0) for m0 in outputs}):
            ms_ = [m0 for m0 in outputs if grp(m0) == g_]
            identical[g_] = all(np.array_equal(outputs[m0], outputs[ms_[0]]) for m0 in ms_)
        a_, b_ = [[outputs[m0] for m0 in outputs if grp(m0) == g_] for g_ in ("one_frame", "batched")]
        if a_ and b_:
            identical["max_abs_diff_batched_vs_one_frame"] = float(np.abs(a_[0] - b_[0]).max())
        xs_ = [m0 for m0 in results if "steps_identical" in results[m0]]
        if xs_:  # cross-step schedules: every step's chunks equal the first step's
            identical["cross_step_every_step"] = all(results[m0]["steps_identical"] for m0 in xs_)
        noise, actions = chunk_bufs[1]
        return cfg, m, results, outputs, identical, (cframes, noise, actions)

    cfg, m, results, outputs, identical, (cframes, noise, actions) = measure(
        args.preset, R, modes, args.steps, args.warmup)
    if args.mode == "auto":
        args.mode = max(results, key=lambda k: results[k]["frames_per_s"])

    def n_prefill_groups(name):
        return -(-R // max(1, kw[name].get("vlm_batch", 1)))

    def overlaps(name):
        """Both phases can run at once: two streams, and a later prefill group
        exists to run beside an earlier group's action loop (in a cross-step
        schedule the next step's prefills)."""
        return kw[name].get("mode") != "serial" and (n_prefill_groups(name) >= 2 or kw[name].get("xsteps", False))

    def run_once(name, nxs=4):
        """One pipeline run of a schedule outside the timed steps (a
        cross-step schedule over nxs steps' frames)."""
        a = kw[name]
        if a.get("xsteps"):
            kc = a.get("act_chunks", 1)
            nz = noise.repeat(nxs, 1, 1).contiguous() if kc == 1 else None
            if nz is None:
                raise SystemExit("cross-step schedules with several chunks per frame are not logged")
            return V.vla_pipeline_run(m, cframes * nxs, nz, R * nxs, actions=torch.empty_like(nz), **lib_args(a))
        return V.vla_pipeline_run(m, cframes, noise, R, actions=actions, **a)

    def same_batching_serial(name):
        a = kw[name]
        if a.get("mode") == "serial":
            return name if a.get("vlm_batch", 1) > 1 or a.get("act_batch", 1) > 1 else "serial"
        v_, b_ = max(1, a.get("vlm_batch", 1)), max(1, a.get("act_batch", 1))
        if v_ == 1 and b_ == 1:
            return "serial"
        return f"serial_vb{v_}_ab{b_}_graph"

    cands = [k for k in results if overlaps(k) and kw[k].get("act_chunks", 1) == 1]
    best_ovl = max(cands, key=lambda k: results[k]["frames_per_s"]) if cands else None

    # per-CU residency (workgroup start/end log): one logged pipeline run per
    # schedule (not part of the timed steps), the serialized one first
    residency = {}
    if args.residency:
        print("[bench] residency logs", file=sys.stderr, flush=True)
        V.vla_wavelog_enable(m, args.residency)
        logged = ["serial", "concurrent", "cu_masked", "wg_capped", "lanes2_graph", best_ovl, args.mode]
        for name in dict.fromkeys(x for x in logged if x and x in kw):
            V.vla_wavelog_read(m, 0)
            run_once(name)
            rec, n = V.vla_wavelog_read(m, args.residency)
            full = cu_residency(rec, window=(int(rec["t"].min()), int(rec["t"].max())))
            ovl = cu_residency(rec)
            residency[name] = {"whole_run": full, "overlap_window": ovl, "records": int(n)}
            print(f"[bench] residency {name}: busy {full['busy_frac']:.3f} whole run; overlap window "
                  f"{ovl['window_ms']:.2f} ms, busy {ovl['busy_frac']:.3f}, both phases "
                  f"{ovl['both_phases_frac']:.3f}", file=sys.stderr, flush=True)
        V.vla_wavelog_enable(m, 0)

    # dominant kernel of the reported schedule, timed live with HIP events
    # on its own stream (the timer replays the schedule without graphs; the
    # kernels and their grids are the same)
    sargs = kw[args.mode]
    tags = [args.kernel] if args.kernel != "auto" else ["lm.gateup", "lm.down", "ex.gateup", "ex.down", "vit.fc1"]
    timed = {}
    for tag in tags:
        print(f"[bench] kernel timer on {tag} in {args.mode}", file=sys.stderr, flush=True)
        V.vla_kernel_timer(m, tag)
        if sargs.get("xsteps"):
            run_once(args.mode, args.steps)
        else:
            for _ in range(args.steps):
                V.vla_pipeline_run(m, cframes, noise, R, actions=actions, **sargs)
        timed[tag] = V.vla_kernel_timer_read(m)
        V.vla_kernel_timer(m, None)
    # dominant: the most stream time; launches of concurrent lanes of one
    # phase overlap, so a tag's summed launch time counts once per stream
    def lanes_of(tag):
        return max(1, sargs.get("vlm_streams" if tag.startswith(("lm.", "vit.")) else "act_streams", 1))
    ran = [k for k in timed if timed[k][1] > 0]
    if not ran:
        raise SystemExit(f"none of the timed kernels ({', '.join(tags)}) runs in {args.preset}")
    kernel = max(ran, key=lambda k: timed[k][0] / lanes_of(k))
    tot_ms, launches = timed[kernel]
    avg_s = tot_ms * 1e-3 / max(launches, 1)
    vfr, afr = max(1, sargs.get("vlm_batch", 1)), max(1, sargs.get("act_batch", 1))
    byts, flops = kernel_work(cfg, kernel, vfr if kernel.startswith(("lm.", "vit.")) else 1,
                              afr if kernel.startswith("ex.") else 1)
    hbm_bound = flops / byts < BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)
    if hbm_bound:
        ach, peak, unit = byts / avg_s / 1e9, HBM_PEAK_GBS, "GB/s"
    else:
        ach, peak, unit = flops / avg_s / 1e12, BF16_PEAK_TFLOPS, "TFLOP/s"
    roofline = {"bound": "hbm" if hbm_bound else "mfma", "achieved": ach, "peak": peak, "unit": unit,
                "frac": ach / peak, "traffic": measured_traffic(args.preset, R, kernel, args.mode),
                "kernel": kernel, "schedule": args.mode, "avg_us": avg_s * 1e6, "launches": launches,
                "algorithmic_bytes": byts, "flops": flops}
    if sargs.get("xsteps") and args.mode[3:] in kw:
        # In a cross-step schedule the prefill shares the CUs with the previous
        # step's action loop, so the kernel's launches there stretch with what
        # runs beside them: a fraction of peak is then no measure of the
        # kernel. The roofline is the same kernel timed in the per-step
        # schedule of the same batching, where a step's prefill has the chip to
        # itself (rocprofv3's kernel trace of this command sees that rate in
        # both: the tracing removes the cross-stream overlap); the shared rate
        # is kept beside it.
        base = args.mode[3:]
        V.vla_kernel_timer(m, kernel)
        for _ in range(args.steps):
            V.vla_pipeline_run(m, cframes, noise, R, actions=actions, **kw[base])
        b_ms, b_n = V.vla_kernel_timer_read(m)
        V.vla_kernel_timer(m, None)
        b_s = b_ms * 1e-3 / max(b_n, 1)
        b_ach = (byts / b_s / 1e9) if hbm_bound else (flops / b_s / 1e12)
        shared = {"schedule": args.mode, "avg_us": avg_s * 1e6, "achieved": ach, "frac": ach / peak,
                  "launches": launches}
        roofline.update({"achieved": b_ach, "frac": b_ach / peak, "avg_us": b_s * 1e6, "launches": b_n,
                         "schedule": base, "in_reported_schedule": shared})
    roofline_detail = dict(roofline, gpu_ms_per_step_by_tag={k: v[0] / args.steps for k, v in timed.items()},
                           stream_ms_per_step_by_tag={k: v[0] / args.steps / lanes_of(k) for k, v in timed.items()})
    outs = outputs[args.mode]
    V.vla_destroy(m)
    del cframes, noise, actions

    # further workloads of the same pipeline: preset:R:schedules (a short
    # summary each; the first config above is the headline)
    others = {}
    for spec in [x for x in args.extra.split(";") if x]:
        preset, r_, sched = spec.split(":")
        ms_ = sched.split(",")
        ocfg, om, ores, _, oid, _ = measure(preset, int(r_), ms_, args.extra_steps, 1)
        V.vla_destroy(om)
        kmax = max(kw[m0].get("act_chunks", 1) for m0 in ms_)
        # asynchronous workloads differ in chunks per frame: best by actions/s
        best = max(ores, key=lambda k: ores[k]["actions_per_s" if kmax > 1 else "frames_per_s"])
        name = f"{preset}_R{r_}" + ("_async" if kmax > 1 else "")
        others[name] = {
            "workload": f"{preset}, R={r_} robot request streams"
                        + (", asynchronous inference (several action chunks per VLM output)" if kmax > 1 else ""),
            "best_schedule": best,
            "frames_per_s": ores[best]["frames_per_s"], "actions_per_s": ores[best]["actions_per_s"],
            "speedup_vs_serialized": ores[best]["speedup_vs_serialized"],
            "chunk": [ocfg["chunk_len"], ocfg["action_dim"]], "euler_steps": ocfg["n_steps"],
            "prefix_tokens": synth.derived(ocfg)["prefix"], "steps": args.extra_steps,
            "outputs_identical_across_modes": oid, "modes": ores}
        print(f"[bench] {name}: best {best} {ores[best]['frames_per_s']:.1f} frames/s "
              f"({ores[best]['speedup_vs_serialized'] or 0:.2f}x serialized)", file=sys.stderr, flush=True)

    main_r = results[args.mode]
    ser_same = same_batching_serial(args.mode)
    sp_same = (main_r["frames_per_s"] / results[ser_same]["frames_per_s"]) if ser_same in results else None
    a_ = kw[args.mode]
    streams = 1 if a_.get("mode") == "serial" else max(1, a_.get("vlm_streams", 1)) + max(1, a_.get("act_streams", 1))
    cpu = None
    if not args.no_cpu_baseline:
        cb, chunk = cpu_baseline(cfg, seed)
        cb["max_abs_err_gpu_vs_oracle_frame0"] = float(np.abs(outs[0].astype(np.float64) - chunk).max())
        cpu = cb

    def short_res(name):
        r_ = residency.get(name)
        if not r_:
            return None
        return {"busy_whole_run": round(r_["whole_run"]["busy_frac"], 4),
                "overlap_window_ms": round(r_["overlap_window"]["window_ms"], 3),
                "busy_in_overlap": round(r_["overlap_window"]["busy_frac"], 4),
                "both_phases_in_overlap": round(r_["overlap_window"]["both_phases_frac"], 4)}

    def rnd(x, n=4):
        return None if x is None else round(float(x), n)

    headline = {
        "metric": METRIC, "value": rnd(main_r["frames_per_s"], 3), "unit": "frames/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": rnd(main_r["ms_per_step"], 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded frames and weights of the stated shapes)",
        "config": {"workload": f"{args.preset}-shaped VLA (PaliGemma-3B-shaped VLM + pi0-shaped expert, "
                               f"chunk {cfg['chunk_len']}x{cfg['action_dim']}, {cfg['n_steps']} Euler steps), "
                               f"R={R} robot request streams",
                   "schedule": args.mode, "R": R, "global_batch": R,
                   "parallelism": f"1 GPU, {streams} HIP stream{'s' if streams > 1 else ''}"},
        "actions_per_s": rnd(main_r["actions_per_s"], 1),
        "speedup_vs_serialized": rnd(main_r["speedup_vs_serialized"]),
        "serialized_frames_per_s": rnd(results.get("serial", {}).get("frames_per_s"), 3),
        "speedup_vs_serialized_same_batching": rnd(sp_same),
        "serialized_same_batching": ser_same if ser_same in results else None,
        "best_overlapped": None if best_ovl is None else {
            "schedule": best_ovl, "frames_per_s": rnd(results[best_ovl]["frames_per_s"], 3),
            "speedup_vs_serialized": rnd(results[best_ovl]["speedup_vs_serialized"]),
            "speedup_vs_serialized_same_batching": rnd(
                results[best_ovl]["frames_per_s"] / results[same_batching_serial(best_ovl)]["frames_per_s"]
                if same_batching_serial(best_ovl) in results else None),
            "residency": short_res(best_ovl)},
        "naive_concurrent": None if "concurrent" not in results else {
            "frames_per_s": rnd(results["concurrent"]["frames_per_s"], 3),
            "speedup_vs_serialized": rnd(results["concurrent"]["speedup_vs_serialized"]),
            "residency": short_res("concurrent")},
        "serialized_residency": short_res("serial"),
        # context only: the paper's dispatcher gains are simulated on other
        # GPUs, over its baseline dispatch of the same concurrent kernels;
        # the closest figure here is a schedule change at the same per-frame
        # work (two action lanes with graphs against two plain streams)
        "paper_context": {
            "simulated_gain_max": 0.28, "simulated_gain_mean": 0.205,
            "over": "baseline CTA dispatch of the concurrent phases, simulated RTX 4090 / 5090",
            "lanes2_graph_vs_concurrent": rnd(results["lanes2_graph"]["frames_per_s"] /
                                              results["concurrent"]["frames_per_s"])
            if "lanes2_graph" in results and "concurrent" in results else None},
        "cu_auto": None if (auto_plan is None or "cu_auto" not in results) else {
            "split": f"{auto_plan['vlm_cus']}/{auto_plan['act_cus']}",
            "predicted_frames_per_s": rnd(1.0 / auto_plan["per_frame_s"], 2),
            "frames_per_s": rnd(results["cu_auto"]["frames_per_s"], 3)},
        "outputs_identical_across_modes": identical,
        "roofline": {k: (rnd(v, 5) if isinstance(v, float) else
                         {k2: (rnd(v2, 5) if isinstance(v2, float) else v2) for k2, v2 in v.items()}
                         if isinstance(v, dict) else v) for k, v in roofline.items()},
        "mfma_util_dominant_kernel": rnd(roofline["frac"]) if roofline["bound"] == "mfma" else None,
        "cpu_baseline": None if cpu is None else {
            "value": rnd(cpu["value"], 6), "unit": cpu["unit"], "cores": cpu["cores"], "kind": "oracle",
            "sample": cpu["sample"], "seconds": rnd(cpu["seconds"], 2), "blas_threads": cpu["blas_threads"],
            "os_cpu_count": cpu["os_cpu_count"],
            "max_abs_err_gpu_vs_oracle_frame0": rnd(cpu["max_abs_err_gpu_vs_oracle_frame0"], 6)},
        "detail_file": os.path.relpath(args.detail, ROOT),
    }
    detail = {"headline": headline, "modes": results, "schedule_args": {k: kw[k] for k in results},
              "roofline": roofline_detail, "cu_residency": residency, "other_workloads": others,
              "cpu_baseline": cpu}
    try:
        os.makedirs(os.path.dirname(os.path.abspath(args.detail)), exist_ok=True)
        with open(args.detail, "w") as f:
            json.dump(detail, f, indent=1)
    except OSError as e:
        print(f"[bench] could not write {args.detail}: {e}", file=sys.stderr, flush=True)
    for name, r_ in results.items():
        print(f"[bench] {name}: {r_['frames_per_s']:.2f} frames/s, {r_['speedup_vs_serialized'] or 0:.3f}x "
              f"serialized", file=sys.stderr, flush=True)
    print(json.dumps(headline), flush=True)


if __name__ == "__main__":
    main()
