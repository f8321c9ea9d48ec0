"""Host-side discrete-event simulator of workgroup dispatch for the two-phase
pipeline: the in-order baseline and the paper's two-phase admission
(Algorithm 1, with its GRID and REG scoring variants), driven by the
per-launch-configuration descriptors of intensity.py.

Model (what the paper's Algorithm 1 needs, and no more):
* N compute units (the paper's SMs). A kernel k has G_k workgroups (CTAs),
  at most o_k of them fit on one CU (occupancy), and each runs for
  w_k = T_k / ceil(G_k / (N o_k)) seconds when the kernel runs alone (T_k:
  its isolated time). A resident workgroup takes 1 / o_k of a CU.
* Streams run their kernels in order; a kernel is launched when the previous
  kernel of its stream has finished, and a stream may also wait for a kernel
  of another stream (the action loop of frame r waits for the prefill of
  frame r).
* Per CU j, utilisation registers U_TC[j], U_ALU[j], U_MEM[j] hold the sum of
  the tau fields of the resident workgroups (8-bit, saturating at 255).
* Admission on CU j is repeated until nothing more fits; each decision
  admits one workgroup:
    - baseline: the earliest-launched kernel with workgroups left is the only
      candidate; a later kernel waits until it has issued all of them
      (head-of-line blocking);
    - two-phase (Algorithm 1): phase 1 admits one workgroup of the first
      kernel, in dispatcher order, that has workgroups left, none resident on
      CU j and room on it; otherwise phase 2 admits one of the fitting kernel
      with the largest score s = sum_r (U_max - U_r[j]) tau_r(k), the first
      seen winning ties (strict comparison). GRID scales s by
      G_k / (c_k(j) + 1), REG by 1 / (c_k(j) R_k + 1), with c_k(j) the
      kernel's workgroups resident on CU j and R_k its registers per
      workgroup, as a share of the CU's register file (from the traced VGPR
      and AGPR counts).
* Contention: a workgroup's progress rate on CU j is 1 / max(1, U_r[j] / 15)
  over the pipelines r it uses (tau_r > 0): a pipeline asked for more than
  one kernel's full level slows everyone on it in proportion. With one
  kernel resident at its isolated occupancy the rate is 1 (sum of tau over a
  CU of one kernel is about its level).

Readings (the paper leaves them open): U_max = 255 (the registers' 8-bit
range); R_k in units of a CU's register file (a raw register count would
make any resident kernel's REG score vanish); the dispatcher order is the kernels' launch order; the per-CU sum of
levels that saturates a pipeline is 15 (one kernel at full level), and a
kernel's tau is split evenly over its resident workgroups on a CU
(tau_r / o_k per workgroup).
"""
from __future__ import annotations

import heapq
import math
from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence, Tuple

try:  # as a module of the package, or as a script next to intensity.py
    from .intensity import reg_share
except ImportError:
    from intensity import reg_share

U_MAX = 255
LEVEL = 15


@dataclass
class Kernel:
    name: str
    workgroups: int
    occupancy: int          # workgroups that fit on one CU
    wg_seconds: float       # run time of one workgroup alone
    tau: Tuple[int, int, int] = (0, 0, 0)
    regs: float = 0.0       # R_k of the REG variant: the workgroup's share of a CU's registers


@dataclass
class Launch:
    kernel: Kernel
    stream: int
    after: Optional[Tuple[int, int]] = None  # (stream, launch index) that must finish first


@dataclass
class _Run:
    launch: Launch
    order: int              # dispatcher order (launch time, then stream)
    pending: int
    running: int = 0


@dataclass
class _WG:
    run: _Run
    cu: int
    left: float             # seconds of isolated work left
    last: float             # time of the last rate update
    rate: float
    gen: int = 0
    rid: int = -1           # the run it belongs to


def wg_seconds(isolated_s: float, workgroups: int, occupancy: int, num_cus: int) -> float:
    """Per-workgroup time of a kernel that runs `isolated_s` alone."""
    rounds = max(1, math.ceil(workgroups / (num_cus * max(1, occupancy))))
    return isolated_s / rounds


class Sim:
    def __init__(self, num_cus: int, policy: str = "baseline"):
        assert policy in ("baseline", "two_phase", "grid", "reg")
        self.N, self.policy = num_cus, policy
        self.used = [0.0] * num_cus                       # occupied fraction of each CU
        self.U = [[0, 0, 0] for _ in range(num_cus)]      # utilisation registers
        self.resident: List[Dict[int, int]] = [dict() for _ in range(num_cus)]  # run id -> count
        self.wgs: List[List[_WG]] = [[] for _ in range(num_cus)]
        self.admitted = 0

    # -- utilisation registers ------------------------------------------------
    def _add(self, j: int, k: Kernel, sign: int) -> None:
        for r in range(3):
            self.U[j][r] = min(U_MAX, max(0, self.U[j][r] + sign * k.tau[r]))

    def _fits(self, j: int, run: _Run) -> bool:
        return run.pending > 0 and self.used[j] + 1.0 / run.launch.kernel.occupancy <= 1.0 + 1e-9

    def _score(self, j: int, run: _Run, rid: int) -> float:
        k = run.launch.kernel
        s = sum((U_MAX - self.U[j][r]) * k.tau[r] for r in range(3))
        c = self.resident[j].get(rid, 0)
        if self.policy == "grid":
            s *= k.workgroups / (c + 1)
        elif self.policy == "reg":
            s /= c * k.regs + 1
        return s

    def choose(self, j: int, active: Sequence[Tuple[int, _Run]]) -> Optional[int]:
        """One admission decision on CU j over the active kernels (run id,
        run) in dispatcher order; returns the run id to admit or None.

        Baseline: only the oldest kernel with workgroups left may dispatch.
        Two-phase policy (Section 3, Algorithm 1): a kernel with no workgroup
        on this CU yet goes first, so every co-runner gets a foothold;
        otherwise the kernel whose intensity best fills the CU's idle
        pipelines, by the score of _score (the first one on a tie)."""
        if self.policy == "baseline":
            oldest = next((run for _, run in active if run.pending > 0), None)
            if oldest is None or not self._fits(j, oldest):
                return None
            return next(rid for rid, run in active if run is oldest)
        fitting = [(rid, run) for rid, run in active if self._fits(j, run)]
        if not fitting:
            return None
        newcomer = next((rid for rid, _ in fitting if self.resident[j].get(rid, 0) == 0), None)
        if newcomer is not None:
            return newcomer
        scores = [self._score(j, run, rid) for rid, run in fitting]
        return fitting[scores.index(max(scores))][0]

    # -- contention ----------------------------------------------------------
    def _rate(self, j: int, k: Kernel) -> float:
        worst = 1.0
        for r in range(3):
            if k.tau[r] > 0:
                worst = max(worst, self._load(j, r) / LEVEL)
        return 1.0 / worst

    def _load(self, j: int, r: int) -> float:
        # tau_r of each kernel spread over its workgroups at full occupancy
        return sum(w.run.launch.kernel.tau[r] / w.run.launch.kernel.occupancy for w in self.wgs[j])


def simulate(launches: Sequence[Launch], num_cus: int, policy: str = "baseline") -> dict:
    """Run the launches; returns the makespan, per-launch finish times and
    the number of admitted workgroups."""
    sim = Sim(num_cus, policy)
    streams: Dict[int, List[int]] = {}
    for i, l in enumerate(launches):
        streams.setdefault(l.stream, []).append(i)
    glob = {(s, n): i for s, ids in streams.items() for n, i in enumerate(ids)}
    pos = {s: 0 for s in streams}          # next launch of each stream
    runs: Dict[int, _Run] = {}             # launched, not finished
    finished: Dict[int, float] = {}
    counter = [0, 0]                       # dispatcher order, event sequence
    events: List[Tuple[float, int, int, int, int]] = []  # (time, seq, cu, wg key, generation)
    live: Dict[int, _WG] = {}
    now = 0.0

    def try_launch(t: float) -> bool:
        started = False
        for s, ids in streams.items():
            while pos[s] < len(ids) and ids[pos[s]] not in runs:
                i = ids[pos[s]]
                dep = launches[i].after
                if dep is not None and glob[dep] not in finished:
                    break
                runs[i] = _Run(launches[i], counter[0], launches[i].kernel.workgroups)
                counter[0] += 1
                started = True
                if runs[i].pending > 0:
                    break
                finished[i] = t          # an empty grid finishes at once
                del runs[i]
                pos[s] += 1
        return started

    def reschedule(j: int, t: float) -> None:
        for w in sim.wgs[j]:
            w.left -= (t - w.last) * w.rate
            w.last = t
            w.rate = sim._rate(j, w.run.launch.kernel)
            w.gen += 1
            counter[1] += 1
            heapq.heappush(events, (t + max(0.0, w.left) / w.rate, counter[1], j, id(w), w.gen))

    def admit(t: float, cus) -> bool:
        """Admission cycles on the given CUs; True if some kernel issued its
        last workgroup (then other CUs may admit the next kernel)."""
        drained = False
        active = sorted(((i, r) for i, r in runs.items() if r.pending > 0), key=lambda x: x[1].order)
        if not active:
            return False
        for j in cus:
            changed = False
            while True:
                rid = sim.choose(j, active)
                if rid is None:
                    break
                run = runs[rid]
                k = run.launch.kernel
                run.pending -= 1
                run.running += 1
                drained |= run.pending == 0
                sim.used[j] += 1.0 / k.occupancy
                sim.resident[j][rid] = sim.resident[j].get(rid, 0) + 1
                sim._add(j, k, +1)
                w = _WG(run, j, k.wg_seconds, t, 1.0, 0, rid)
                sim.wgs[j].append(w)
                live[id(w)] = w
                sim.admitted += 1
                changed = True
            if changed:
                reschedule(j, t)
        return drained

    def admit_until_stable(t: float, cus) -> None:
        while admit(t, cus):
            cus = range(num_cus)

    try_launch(0.0)
    admit_until_stable(0.0, range(num_cus))
    while events:
        t, _, j, key, gen = heapq.heappop(events)
        w = live.get(key)
        if w is None or w.gen != gen:
            continue  # superseded by a later rate change
        now = t
        sim.wgs[j].remove(w)
        del live[key]
        run, rid, k = w.run, w.rid, w.run.launch.kernel
        run.running -= 1
        sim.used[j] -= 1.0 / k.occupancy
        sim.resident[j][rid] -= 1
        if sim.resident[j][rid] == 0:
            del sim.resident[j][rid]
        sim._add(j, k, -1)
        launched = False
        if run.pending == 0 and run.running == 0:
            finished[rid] = t
            del runs[rid]
            pos[run.launch.stream] += 1
            launched = try_launch(t)
        reschedule(j, t)
        admit_until_stable(t, range(num_cus) if launched else [j])
    return {"makespan": now, "finish": finished, "admitted": sim.admitted}


def from_descriptors(desc: Sequence[dict], num_cus: int, frames: int, limit: Optional[int] = None) -> List[Launch]:
    """Launch list of `frames` frames of the two-phase pipeline from
    intensity descriptors: stream 0 runs the prefills, stream 1 the action
    loops, the action loop of frame r after the prefill of frame r. Within a
    phase the configurations are interleaved in proportion to their launches
    per frame; `limit` keeps only the first launches of each phase (for short
    runs)."""
    def phase_seq(phase: str) -> List[Kernel]:
        items = []
        for d in desc:
            if d["phase"] != phase:
                continue
            n = int(round(d["launches_per_frame"]))
            o = max(1, int(d.get("wgs_per_cu", 1)))
            regs = reg_share(int(d.get("wg_threads", 256)), int(d.get("vgpr", 0)), int(d.get("agpr", 0)))
            k = Kernel(d["kernel"], int(d["workgroups"]), o,
                       wg_seconds(d["us"] * 1e-6, int(d["workgroups"]), o, num_cus), tuple(d["tau"]), regs)
            for i in range(n):
                items.append(((i + 0.5) / n, k))
        items.sort(key=lambda x: x[0])
        seq = [k for _, k in items]
        return seq[:limit] if limit else seq

    vlm, act = phase_seq("vlm"), phase_seq("action")
    out: List[Launch] = []
    n0 = 0
    for f in range(frames):
        for k in vlm:
            out.append(Launch(k, 0))
        last_vlm = n0 + len(vlm) - 1
        for i, k in enumerate(act):
            out.append(Launch(k, 1, after=(0, last_vlm) if i == 0 else None))
        n0 += len(vlm)
    return out


def main() -> None:
    """python paper_2609_22335_amd/cosched.py profiles/intensity_pi0.json [frames]
    prints a markdown table: the makespan of `frames` pipelined frames under
    each dispatch policy, and frames/s."""
    import json
    import sys
    path = sys.argv[1]
    frames = int(sys.argv[2]) if len(sys.argv) > 2 else 2
    with open(path) as f:
        desc = json.load(f)["descriptors"]
    L = from_descriptors(desc, NUM_CUS_DEFAULT, frames)
    print(f"| policy | makespan of {frames} frames (ms) | frames/s | workgroups |")
    print("|---|---|---|---|")
    for pol in ("baseline", "two_phase", "grid", "reg"):
        r = simulate(L, NUM_CUS_DEFAULT, pol)
        print(f"| {pol} | {r['makespan'] * 1e3:.3f} | {frames / r['makespan']:.1f} | {r['admitted']} |", flush=True)


NUM_CUS_DEFAULT = 256

if __name__ == "__main__":
    main()
