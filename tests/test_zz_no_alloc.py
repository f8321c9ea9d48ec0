"""The allocation-free GEMM entry point (vla_gemm_noalloc) against the
allocating one (vla_debug_gemm) through the C ABI: the same kernels and
plan, so the same bits, on two calls in a row, the second with a smaller
input (its split-K partials reuse the fixed scratch the first call left
dirty); and both within the fp64 bound of the GEMM tests."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

RNG = np.random.default_rng(99)

# (dtype, [(M, N, K) first call, (M, N, K) second, smaller call])
CASES = [
    (1, [(50, 1024, 4096), (21, 136, 1024)]),  # bf16: 16 then 4 split-K partials
    (0, [(40, 100, 592), (7, 3, 16)]),          # fp32: 4 partials, then no split
    (1, [(305, 2048, 2048), (33, 128, 256)]),   # bf16 without split-K
]


@pytest.fixture(scope="module")
def V():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_22335_amd as V
    return V


@pytest.mark.parametrize("dtype,shapes", CASES, ids=["bf16-split", "f32-split", "bf16-plain"])
def test_noalloc_gemm_matches_allocating_entry_point(V, dtype, shapes):
    import gpu_util as g
    for M, N, K in shapes:
        g.say(f"gemm_noalloc dtype={dtype} M={M} N={N} K={K}")
        A = RNG.standard_normal((M, K))
        W = RNG.standard_normal((N, K)) * 0.05
        b = RNG.standard_normal(N).astype(np.float32)
        Ad, Wd, bd = g.operand_dev(A, dtype), g.operand_dev(W, dtype), g.to_dev(b)
        C0 = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        C1 = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        V.vla_debug_gemm(dtype, M, N, K, Ad, K, Wd, K, bd, C0)
        V.vla_gemm_noalloc(dtype, M, N, K, Ad, K, Wd, K, bd, C1)
        torch.cuda.synchronize()
        got, want = C1.cpu().numpy(), C0.cpu().numpy()
        assert np.array_equal(got, want), float(np.nanmax(np.abs(got - want)))
        a, w = g.operand_values(A, dtype), g.operand_values(W, dtype)
        ref = a @ w.T + b
        bound = 2 * K * 2.0 ** -24 * (np.abs(a) @ np.abs(w).T + np.abs(b)) + 1e-30
        assert np.all(np.abs(got - ref) <= bound)


def test_noalloc_gemm_rejects_bad_arguments(V):
    with pytest.raises(V.VlaError) as e:
        V.vla_gemm_noalloc(1, 4, 4, 7, 1, 8, 1, 8, None, 1)  # K not a multiple of 8
    assert e.value.code == -1
    with pytest.raises(V.VlaError) as e:
        V.vla_gemm_noalloc(1, 4, 4, 8, None, 8, None, 8, None, None)
    assert e.value.code == -1
