"""Dispatch simulator (host logic): hand-worked cases of the baseline and of
the two-phase admission (the paper's Algorithm 1) and its invariants."""
import pytest

from paper_2609_22335_amd import cosched as C


def K(name, wgs, occ, secs, tau=(0, 0, 0), regs=0):
    return C.Kernel(name, wgs, occ, secs, tau, regs)


def test_single_kernel_rounds():
    # 4 CUs x 2 slots = 8 at once; 16 workgroups of 1 s -> two rounds
    for pol in ("baseline", "two_phase", "grid", "reg"):
        r = C.simulate([C.Launch(K("a", 16, 2, 1.0, (4, 0, 4)), 0)], 4, pol)
        assert r["makespan"] == pytest.approx(2.0)
        assert r["admitted"] == 16


def test_stream_order_and_dependency():
    # stream 0: a (1 s) then b (1 s); stream 1: c after b; all fill the chip
    L = [C.Launch(K("a", 4, 1, 1.0), 0), C.Launch(K("b", 4, 1, 1.0), 0), C.Launch(K("c", 4, 1, 1.0), 1, after=(0, 1))]
    r = C.simulate(L, 4, "two_phase")
    assert r["finish"][0] == pytest.approx(1.0)
    assert r["finish"][1] == pytest.approx(2.0)
    assert r["finish"][2] == pytest.approx(3.0)


def test_head_of_line_blocking_removed():
    # A: 16 workgroups at two per CU (1 s each) on 2 CUs: 4 rounds. B (other
    # stream, launched right after A): 2 workgroups of 0.1 s at two per CU.
    a = K("A", 16, 2, 1.0, (10, 0, 0))
    b = K("B", 2, 2, 0.1, (0, 0, 10))
    L = [C.Launch(a, 0), C.Launch(b, 1)]
    base = C.simulate(L, 2, "baseline")
    two = C.simulate(L, 2, "two_phase")
    # baseline: A issues 4 per round (2 CUs x 2 slots), 4 rounds; its last
    # workgroups are admitted at t = 3, so B starts when a slot frees at 4
    assert base["finish"][1] == pytest.approx(4.1)
    # two-phase: B is unrepresented on each CU, so phase 1 admits it at t = 0
    # before A fills the CU (A is also unrepresented, but B comes after A in
    # dispatcher order: A takes the first slot, B the second)
    assert two["finish"][1] == pytest.approx(0.1)
    assert two["makespan"] <= base["makespan"] + 1e-9


def test_phase2_prefers_complementary_kernel():
    sim = C.Sim(1, "two_phase")
    tc = C._Run(C.Launch(K("tc", 8, 4, 1.0, (12, 0, 2)), 0), 0, 8)
    mem = C._Run(C.Launch(K("mem", 8, 4, 1.0, (1, 0, 12)), 1), 1, 8)
    # both already resident (phase 1 does not apply); the CU's MFMA register
    # is high, its memory register low
    sim.resident[0] = {0: 1, 1: 1}
    sim.U[0] = [200, 0, 20]
    sim.used[0] = 0.5
    # s(tc) = 55 * 12 + 255 * 0 + 235 * 2 = 1130; s(mem) = 55 * 1 + 235 * 12 = 2875
    assert sim._score(0, tc, 0) == 55 * 12 + 235 * 2
    assert sim.choose(0, [(0, tc), (1, mem)]) == 1
    # ties go to the first kernel in dispatcher order
    same = C._Run(C.Launch(K("same", 8, 4, 1.0, (1, 0, 12)), 1), 2, 8)
    sim.resident[0][2] = 1
    assert sim.choose(0, [(1, mem), (2, same)]) == 1
    # phase 1: an unrepresented kernel that fits wins regardless of score
    new = C._Run(C.Launch(K("new", 8, 4, 1.0, (15, 0, 0)), 1), 3, 8)
    assert sim.choose(0, [(0, tc), (1, mem), (3, new)]) == 3
    # nothing fits on a full CU
    sim.used[0] = 1.0
    assert sim.choose(0, [(0, tc), (1, mem), (3, new)]) is None


def test_grid_and_reg_scores():
    sim = C.Sim(1, "grid")
    r = C._Run(C.Launch(K("k", 64, 4, 1.0, (2, 0, 1), regs=100), 0), 0, 64)
    sim.resident[0] = {0: 3}
    base = (255 * 2 + 255 * 1)
    assert sim._score(0, r, 0) == pytest.approx(base * 64 / 4)
    sim.policy = "reg"
    assert sim._score(0, r, 0) == pytest.approx(base / (3 * 100 + 1))


def test_contention_slows_shared_pipeline():
    # one CU; a workgroup carries tau / occupancy of its kernel's level.
    # a and b (memory level 15, two per CU) side by side: load 7.5 + 7.5 = 15,
    # no slowdown
    a = K("a", 1, 2, 1.0, (0, 0, 15))
    b = K("b", 1, 2, 1.0, (0, 0, 15))
    r = C.simulate([C.Launch(a, 0), C.Launch(b, 1)], 1, "two_phase")
    assert r["makespan"] == pytest.approx(1.0)
    # b2 at level 30 (beyond the 4-bit range, to oversubscribe): load
    # 7.5 + 15 = 22.5, both run at rate 1 / 1.5 and end at 1.5 s
    b2 = K("b2", 1, 2, 1.0, (0, 0, 30))
    r = C.simulate([C.Launch(a, 0), C.Launch(b2, 1)], 1, "two_phase")
    assert r["makespan"] == pytest.approx(1.5)


def test_from_descriptors_pipeline():
    desc = [{"kernel": "v", "phase": "vlm", "workgroups": 8, "wgs_per_cu": 1, "launches_per_frame": 2, "us": 10.0,
             "tau": [4, 0, 2]},
            {"kernel": "x", "phase": "action", "workgroups": 2, "wgs_per_cu": 2, "launches_per_frame": 3, "us": 5.0,
             "tau": [0, 0, 3]}]
    L = C.from_descriptors(desc, 8, frames=2)
    assert len(L) == 2 * (2 + 3)
    assert [l.stream for l in L[:5]] == [0, 0, 1, 1, 1]
    assert L[2].after == (0, 1) and L[7].after == (0, 3)
    base = C.simulate(L, 8, "baseline")
    two = C.simulate(L, 8, "two_phase")
    assert base["admitted"] == two["admitted"] == 2 * (2 * 8 + 3 * 2)
    # between the critical path (two prefills of 20 us, then the last action
    # loop of 15 us) and the fully serialized run (2 x (20 + 15) us)
    for r in (base, two):
        assert 55e-6 - 1e-12 <= r["makespan"] <= 70e-6 + 1e-12
    assert two["makespan"] <= base["makespan"] + 1e-12
