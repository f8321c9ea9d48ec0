"""GPU parity of the fused GEMM epilogues, kernel by kernel, through the C
ABI (vla_debug_gemm_epi), against the oracle's primitives in fp64.

Every epilogue the phases use (bias, operand-type store, GELU, swish,
GeGLU, RoPE + KV-cache store, plain QKV store, the Euler / DDIM state update
and the split-K residual add + RMSNorm) runs on the tiles that carry it in
the phases (32x64, 64x64, 128x128, 256x256 and the skinny kernel of the
action head) at the model's full N and K; the tile is asserted from the
planner's answer. Rows are sampled where M is large (the oracle computes
them one by one).

Bounds. With u = 2^-24, the GEMM value v = sum_k a_k w_k in fp32 has
|v - v_exact| <= delta = 2 K u sum_k |a_k w_k|. Each epilogue f turns that
into a sensitivity D (GELU' <= 1.13, swish' <= 1.1, GeGLU |up| 1.13 delta_g
+ |gelu(gate)| delta_u, RoPE delta_1 + delta_2, RMSNorm |g| (D_x / rms +
|x| max D_x / rms^2)); the stored value is rounded once to the operand type
(unit roundoff u_T = 2^-8 for bf16): |got - ref| <= u_T (|ref| + D) + D +
4e-6 (|ref| + D) (fp32 evaluation of tanh / exp / the rotation)."""
import numpy as np
import pytest
import torch

import synth
from oracle import vla_oracle as O

pytestmark = pytest.mark.gpu

RNG = np.random.default_rng(2024)
TILE = {"128": (128, 128), "64": (64, 64), "32": (32, 64), "256": (256, 256), "skinny": (0, 32)}


@pytest.fixture(scope="module")
def V():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_22335_amd as V
    return V


def _rows(M):
    if M <= 64:
        return np.arange(M)
    r = set([0, 1, M // 2, M - 1]) | set(RNG.choice(M, 28, replace=False).tolist())
    return np.array(sorted(r))


def _operands(g, dtype, M, N, K, wscale=0.05):
    A = RNG.standard_normal((M, K))
    W = RNG.standard_normal((N, K)) * wscale
    return g.operand_dev(A, dtype), g.operand_dev(W, dtype), g.operand_values(A, dtype), g.operand_values(W, dtype)


def _check(tag, got, ref, D, dtype, out_fp32=False):
    u = 2.0 ** -24 if (out_fp32 or dtype == 0) else 2.0 ** -8
    bound = u * (np.abs(ref) + D) + D + 4e-6 * (np.abs(ref) + D) + 1e-30
    err = np.abs(got - ref)
    worst = float((err / bound).max())
    print(f"[gpu] epilogue {tag}: max err {float(err.max()):.3e}, worst err / bound {worst:.3f}", flush=True)
    assert np.all(err <= bound), (tag, worst)


# name, dtype, M, N, K, path (tile), extra
CASES = [
    # GeGLU: the LM's gate/up (N = 2 x 16384, K = 2048) on every tile; the
    # expert's (N = 2 x 4096, K = 1024) on the skinny kernel; tiny in fp32
    ("geglu", 1, 20, 32768, 2048, "32", {}),
    ("geglu", 1, 100, 32768, 2048, "64", {}),
    ("geglu", 1, 305, 32768, 2048, "128", {}),
    ("geglu", 1, 2440, 32768, 2048, "256", {}),
    ("geglu", 1, 50, 8192, 1024, "skinny", {}),
    ("geglu", 0, 80, 2048, 256, "64", {}),
    ("geglu", 0, 8, 1024, 128, "skinny", {}),
    # RoPE + KV-cache store: the LM's q/k/v (8 query heads, 1 KV head of 256)
    # at prefix positions; 24 query heads to fill the 256 tile; the expert's
    # at action positions 305..354 on the skinny kernel; tiny in fp32
    ("qkv_rope", 1, 20, 2560, 2048, "32", dict(nq=8, nkv=1, hd=256, pos0=0)),
    ("qkv_rope", 1, 305, 2560, 2048, "64", dict(nq=8, nkv=1, hd=256, pos0=0)),
    ("qkv_rope", 1, 2440, 2560, 2048, "128", dict(nq=8, nkv=1, hd=256, pos0=0)),
    ("qkv_rope", 1, 2440, 6656, 2048, "256", dict(nq=24, nkv=1, hd=256, pos0=0)),
    ("qkv_rope", 1, 50, 2560, 1024, "skinny", dict(nq=8, nkv=1, hd=256, pos0=305)),
    ("qkv_rope", 0, 8, 384, 128, "skinny", dict(nq=4, nkv=1, hd=64, pos0=80)),
    ("qkv_rope", 0, 80, 384, 256, "64", dict(nq=4, nkv=1, hd=64, pos0=0)),
    # plain QKV store: the GR00T-shaped DiT's self-attention (32 heads of 48)
    # and its cross K/V from the 96 feature rows
    ("qkv_plain", 1, 16, 4608, 1536, "skinny", dict(nq=32, nkv=32, hd=48, pos0=0)),
    ("qkv_plain", 1, 96, 3072, 2048, "64", dict(nq=0, nkv=32, hd=48, pos0=0)),
    # GELU + bias: the ViT MLP (N = 4304, K = 1152) for 1, 4, 8 and 16 views
    # (8 views: a half-empty round of 256 tiles beats two of 128);
    # the DiT MLP (N = 6144, K = 1536) on the skinny kernel
    ("gelu", 1, 256, 4304, 1152, "64", {}),
    ("gelu", 1, 1024, 4304, 1152, "128", {}),
    ("gelu", 1, 2048, 4304, 1152, "256", {}),
    ("gelu", 1, 4096, 4304, 1152, "256", {}),
    ("gelu", 1, 16, 6144, 1536, "skinny", {}),
    # swish + bias: the expert's time MLP
    ("swish", 1, 50, 1024, 1024, "skinny", {}),
    ("swish", 1, 400, 1024, 1024, "64", {}),
    ("swish", 0, 8, 128, 128, "skinny", {}),
    # operand store + bias: the ViT's fused q/k/v; the action embedding
    ("t", 1, 256, 3456, 1152, "64", {}),
    ("t", 1, 50, 1024, 32, "skinny", {}),
    # Euler and DDIM state update + bias: the output projection
    ("step", 1, 50, 32, 1024, "skinny", dict(xs=1.0, dt=-0.1)),
    ("step", 1, 50, 32, 1024, "skinny", dict(xs=1.0526, dt=-0.3)),
    ("step", 1, 400, 32, 1024, "64", dict(xs=1.0, dt=-0.1)),
    ("step", 0, 8, 8, 128, "skinny", dict(xs=1.0, dt=-0.25)),
    # split-K partials + residual + RMSNorm: the LM's down projection
    # (K = 16384) and O projection, the expert's down and O projections; the
    # 256 tile's partials (two splits of a 32 x 8 grid of tiles)
    ("resid_norm", 1, 305, 2048, 16384, "64", {}),
    ("resid_norm", 1, 2440, 2048, 16384, "128", {}),
    ("resid_norm", 1, 8192, 2048, 1024, "256", {}),
    ("resid_norm", 1, 305, 2048, 2048, "64", {}),
    ("resid_norm", 1, 50, 1024, 4096, "skinny", {}),
    ("resid_norm", 1, 50, 1024, 2048, "skinny", {}),
    ("resid_norm", 0, 8, 128, 512, "skinny", {}),
]


def _id(c):
    return f"{c[0]}-{'bf16' if c[1] else 'f32'}-{c[2]}x{c[3]}x{c[4]}-{c[5]}"


@pytest.mark.parametrize("case", CASES, ids=[_id(c) for c in CASES])
def test_gemm_epilogue_vs_oracle(V, case):
    import gpu_util as g
    kind, dtype, M, N, K, path, ex = case
    g.say(f"gemm epilogue {_id(case)}")
    skinny = path == "skinny"
    Ad, Wd, a, w = _operands(g, dtype, M, N, K)
    rows = _rows(M)
    a_s = a[rows]
    v = a_s @ w.T
    delta = 2 * K * 2.0 ** -24 * (np.abs(a_s) @ np.abs(w).T)
    opt = torch.bfloat16 if dtype else torch.float32
    dev = lambda shape, t=opt: torch.full(shape, float("nan"), dtype=t, device="cuda")
    host = lambda t: t.float().cpu().numpy().astype(np.float64)[rows]
    if kind in ("t", "gelu", "swish", "step"):
        b = RNG.standard_normal(N).astype(np.float32)
        bd = g.to_dev(b)
        vb = v + b
        db = delta + 2.0 ** -24 * np.abs(b)
    if kind in ("t", "gelu", "swish"):
        out = dev((M, N))
        plan = V.vla_debug_gemm_epi(dtype, M, N, K, Ad, Wd, kind, skinny=skinny, bias=bd, out=out)
        f, L = {"t": (lambda z: z, 1.0), "gelu": (O.gelu_tanh, 1.13), "swish": (O.swish, 1.1)}[kind]
        _check(_id(case), host(out), f(vb), L * db, dtype)
    elif kind == "geglu":
        F = N // 2
        out = dev((M, F))
        plan = V.vla_debug_gemm_epi(dtype, M, N, K, Ad, Wd, kind, skinny=skinny, out=out)
        gate, up, dg, du = v[:, :F], v[:, F:], delta[:, :F], delta[:, F:]
        ref = O.gelu_tanh(gate) * up
        D = np.abs(up) * 1.13 * dg + np.abs(O.gelu_tanh(gate)) * du + 1.13 * dg * du
        _check(_id(case), host(out), ref, D, dtype)
    elif kind in ("qkv_rope", "qkv_plain"):
        nq, nkv, hd, pos0 = ex["nq"], ex["nkv"], ex["hd"], ex["pos0"]
        qo = dev((M, max(nq, 1) * hd))
        ko, vo = dev((M, nkv * hd)), dev((M, nkv * hd))
        plan = V.vla_debug_gemm_epi(dtype, M, N, K, Ad, Wd, kind, skinny=skinny, nq=nq, nkv=nkv, hd=hd, pos0=pos0,
                                    q_out=qo if nq else None, k_out=ko, v_out=vo)
        qc, kc = nq * hd, nkv * hd
        parts = [("q", 0, nq, qo), ("k", qc, nkv, ko)] if nq else [("k", qc, nkv, ko)]
        for name, c0, nh, t in parts:
            x = v[:, c0:c0 + nh * hd].reshape(len(rows), nh, hd)
            dx = delta[:, c0:c0 + nh * hd].reshape(len(rows), nh, hd)
            if kind == "qkv_rope":
                ref = O.rope(x, pos0 + rows)
                half = hd // 2
                dpair = dx[..., :half] + dx[..., half:] + 2.0 ** -21 * (np.abs(x[..., :half]) + np.abs(x[..., half:]))
                D = np.concatenate([dpair, dpair], -1)
            else:
                ref, D = x, dx
            _check(f"{_id(case)} {name}", host(t), ref.reshape(len(rows), -1), D.reshape(len(rows), -1), dtype)
        _check(f"{_id(case)} v", host(vo), v[:, qc + kc:], delta[:, qc + kc:], dtype)
    elif kind == "step":
        x0 = RNG.standard_normal((M, N)).astype(np.float32)
        xd = g.to_dev(x0)
        out = dev((M, N))
        plan = V.vla_debug_gemm_epi(dtype, M, N, K, Ad, Wd, kind, skinny=skinny, bias=bd, out=out, x=xd,
                                    xs=ex["xs"], dt=ex["dt"])
        xs, dt = float(np.float32(ex["xs"])), float(np.float32(ex["dt"]))
        ref = xs * x0.astype(np.float64)[rows] + dt * vb
        D = abs(dt) * db + 2.0 ** -22 * (np.abs(xs * x0.astype(np.float64)[rows]) + np.abs(dt * vb))
        _check(_id(case) + " x", xd.cpu().numpy().astype(np.float64)[rows], ref, D, dtype, out_fp32=True)
        _check(_id(case) + " x as operand", host(out), ref, D, dtype)
    elif kind == "resid_norm":
        r0 = RNG.standard_normal((M, N)).astype(np.float32)
        gain = (1 + 0.02 * RNG.standard_normal(N)).astype(np.float32)
        rd, gd = g.to_dev(r0), g.to_dev(gain)
        out = dev((M, N))
        plan = V.vla_debug_gemm_epi(dtype, M, N, K, Ad, Wd, kind, skinny=skinny, out=out, resid=rd, gain=gd)
        xr = r0.astype(np.float64)[rows] + v
        Dx = delta + 2.0 ** -23 * (np.abs(r0.astype(np.float64)[rows]) + np.abs(v))
        _check(_id(case) + " residual", rd.cpu().numpy().astype(np.float64)[rows], xr, Dx, dtype, out_fp32=True)
        ref = O.rms_norm(xr, gain.astype(np.float64))
        rms = np.sqrt((xr * xr).mean(1, keepdims=True) + 1e-6)
        D = np.abs(gain) * (Dx / rms + np.abs(xr) * Dx.max(1, keepdims=True) / rms ** 2)
        _check(_id(case) + " norm", host(out), ref, D, dtype)
    assert tuple(plan[:2]) == TILE[path], (plan, path)
    print(f"[gpu] epilogue {_id(case)}: tile {plan[0]}x{plan[1]}, {plan[2]} split(s)", flush=True)
