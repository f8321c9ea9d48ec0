"""Oracle: a plain, slow, fp64 CPU forward of the two-phase VLA.

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call or
run this module: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it. It shares no code with the HIP
library; the only common dependency is the seeded input generator ``synth``
(which holds none of the method's arithmetic).

What it computes (paper: Section 2.1 and Fig. "vla-arch"; the execution
model of Section 2.1, last paragraph, and Section 2.3): phase 1, a VLM,
encodes a camera frame and a language instruction into an intermediate
representation; for the pi-family models this hand-off is the LM's per-layer
KV cache. Phase 2, a flow-matching action head, integrates a velocity field
over a few Euler steps to produce an action chunk, every step attending to
that cache. The paper gives no layer equations, so the layer definitions
below are the readings this oracle fixes (SigLIP-style ViT, Gemma-style
prefix LM with multi-query attention, pi0-style action expert); each function
names the reading it follows.

Precision. Every intermediate is fp64. For bf16 configurations the model is
defined with bf16 storage at exactly these points, which this oracle applies
with ``_op`` (round to fp32, then to bf16, nearest-even):
  * weights (already bf16 when they come out of ``synth``);
  * every GEMM A-operand (norm outputs, attention outputs, GELU / GeGLU /
    swish outputs, patches, the state vector, x_t and the sinusoid phi(t));
  * attention Q, K, V after bias / RoPE (K and V are the bf16 KV cache).
Residual stream, norm statistics, softmax probabilities, velocities and the
Euler state stay exact (fp64 here). For fp32 configurations ``_op`` is the
identity and the oracle is the exact-arithmetic model.

Two action-head families (Section 2.1 names both flow-matching heads that
read the VLM's KV cache, as in pi0, and diffusion-transformer heads that read
the VLM's features): ``head == 0`` is the pi0-style expert sharing the LM
cache; ``head == 1`` is a GR00T-style DiT whose even layers cross-attend to
the LM's final normalised hidden states (the features) and whose odd layers
self-attend, conditioned on the flow time through adaLN. The DiT config also
pixel-shuffles the ViT grid 2x2 before the projector and runs every LM layer
(the features need the last layer's output). ``head == 2`` is a
CogACT-style diffusion head: a learned cognition token is appended to the
prefix, every LM layer runs, and the token's final normalised output,
projected to the head's width, conditions a DiT of self-attention layers in
context (with a time token); the head's output is the noise estimate of DDIM
steps.
"""
from __future__ import annotations

import math
from typing import Callable, Dict, List, Optional, Tuple

import numpy as np

F32, BF16 = 0, 1
EPS = 1e-6
ROPE_BASE = 10000.0
MIN_PERIOD, MAX_PERIOD = 4e-3, 4.0


# ---------------------------------------------------------------------------
# Number handling
# ---------------------------------------------------------------------------

def bf16(x: np.ndarray) -> np.ndarray:
    """fp64 -> fp32 (nearest) -> bf16 (nearest, ties to even), returned as fp64.

    Written from the bfloat16 definition (the top 16 bits of an IEEE binary32
    value) independently of ``synth.bf16_round``."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32)
    lower = u & np.uint32(0xFFFF)
    upper = u & np.uint32(0xFFFF0000)
    halfway = np.uint32(0x8000)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    round_up = (lower > halfway) | ((lower == halfway) & (lsb == 1))
    upper = upper + np.where(round_up, np.uint32(0x10000), np.uint32(0))
    return upper.astype(np.uint32).view(np.float32).astype(np.float64)


def _op(x: np.ndarray, cfg) -> np.ndarray:
    """A GEMM / attention operand as the model stores it (see module doc)."""
    if cfg["dtype"] == BF16:
        return bf16(x)
    return np.asarray(x, dtype=np.float64)


def _w(P, name) -> np.ndarray:
    return np.asarray(P[name], dtype=np.float64)


def linear(x: np.ndarray, w: np.ndarray, b: Optional[np.ndarray] = None) -> np.ndarray:
    """y = x W^T (+ b); weights are stored [out, in]."""
    y = x @ w.T
    if b is not None:
        y = y + b
    return y


# ---------------------------------------------------------------------------
# Primitives
# ---------------------------------------------------------------------------

def layer_norm(x, g, b, eps=EPS):
    """(x - mean) / sqrt(biased var + eps) * g + b over the last axis."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * g + b


def rms_norm(x, g, eps=EPS):
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    ms = (x * x).mean(axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def gelu_tanh(x):
    """0.5 x (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3)))."""
    return 0.5 * x * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (x + 0.044715 * x ** 3)))


def swish(x):
    """x * sigmoid(x)."""
    return x / (1.0 + np.exp(-x))


def softmax(s, axis=-1):
    """Row softmax with the row maximum subtracted."""
    e = np.exp(s - s.max(axis=axis, keepdims=True))
    return e / e.sum(axis=axis, keepdims=True)


def attention(q, k, v):
    """Unmasked scaled dot-product attention with grouped KV heads.

    q [Sq, nq, hd]; k, v [Skv, nkv, hd]; query head h reads KV head
    h // (nq / nkv) (nkv = 1 is multi-query attention); scale 1/sqrt(hd).
    Returns [Sq, nq, hd]."""
    sq, nq, hd = q.shape
    nkv = k.shape[1]
    assert nq % nkv == 0
    group = nq // nkv
    out = np.empty((sq, nq, hd), dtype=np.float64)
    scale = 1.0 / math.sqrt(hd)
    for h in range(nq):
        j = h // group
        s = (q[:, h, :] @ k[:, j, :].T) * scale
        out[:, h, :] = softmax(s) @ v[:, j, :]
    return out


def rope(x, positions):
    """Rotate-half rotary embedding: pair (i, i + hd/2) of every head is rotated
    by the angle pos * base^(-2i/hd). x [S, nh, hd], positions [S]."""
    hd = x.shape[-1]
    half = hd // 2
    inv = ROPE_BASE ** (-2.0 * np.arange(half, dtype=np.float64) / hd)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * inv[None, :]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def patchify(img, p):
    """Image [H, W, 3] (HWC) -> patches [(H/p)(W/p), 3 p^2]. Patch (i, j) in
    raster order; inside a patch, (row, column, channel) with channel fastest."""
    h, w, c = img.shape
    gh, gw = h // p, w // p
    t = img.reshape(gh, p, gw, p, c).transpose(0, 2, 1, 3, 4)
    return t.reshape(gh * gw, p * p * c)


def sinusoid(t, dim):
    """phi(t) = [sin(2 pi t / p_i)]_i ++ [cos(2 pi t / p_i)]_i, i < dim/2, with
    periods log-spaced from 4e-3 to 4: p_i = 4e-3 (4 / 4e-3)^(i / (dim/2 - 1))."""
    half = dim // 2
    frac = np.arange(half, dtype=np.float64) / max(half - 1, 1)
    period = MIN_PERIOD * (MAX_PERIOD / MIN_PERIOD) ** frac
    x = 2.0 * math.pi * float(t) / period
    return np.concatenate([np.sin(x), np.cos(x)])


def positions_sinusoid(n, dim):
    """Fixed token positions of the DiT: row p is [sin(p w_i)]_i ++ [cos(p w_i)]_i
    with w_i = 10000^(-i / (dim/2)), i < dim/2."""
    half = dim // 2
    w = ROPE_BASE ** (-np.arange(half, dtype=np.float64) / half)
    ang = np.arange(n, dtype=np.float64)[:, None] * w[None, :]
    return np.concatenate([np.sin(ang), np.cos(ang)], axis=1)


def pixel_shuffle(x, grid_h, grid_w, s):
    """Space-to-depth of a raster token grid: [gh gw, c] -> [(gh/s)(gw/s), s^2 c];
    coarse token (i, j) concatenates fine tokens (s i + dy, s j + dx) in
    (dy, dx) order, channels fastest."""
    c = x.shape[1]
    t = x.reshape(grid_h // s, s, grid_w // s, s, c).transpose(0, 2, 1, 3, 4)
    return t.reshape((grid_h // s) * (grid_w // s), s * s * c)


def flow_times(n_steps) -> Tuple[List[float], float]:
    """Euler schedule of the flow-matching head: noise sits at t = 1 and the
    data at t = 0; t_k = (N - k) / N and dt = -1 / N, each one fp32 division."""
    n = np.float32(n_steps)
    ts = [float(np.float32(n_steps - k) / n) for k in range(n_steps)]
    dt = float(np.float32(-1.0) / n)
    return ts, dt


def euler_integrate(x0, velocity: Callable[[np.ndarray, float], np.ndarray], n_steps):
    """x_{k+1} = x_k + dt * v(x_k, t_k), k = 0 .. N-1; returns x_N."""
    ts, dt = flow_times(n_steps)
    x = np.asarray(x0, dtype=np.float64)
    for k in range(n_steps):
        x = x + dt * velocity(x, ts[k])
    return x


DDIM_TRAIN_STEPS = 1000


def ddim_alpha_bar(train_steps: int = DDIM_TRAIN_STEPS) -> np.ndarray:
    """Cumulative products abar_s = prod_{i <= s} (1 - beta_i) of a linear beta
    schedule from 1e-4 to 0.02 over the training steps (the DDPM schedule)."""
    beta = np.linspace(1e-4, 0.02, train_steps, dtype=np.float64)
    return np.cumprod(1.0 - beta)


def ddim_schedule(n_steps: int) -> Tuple[List[float], List[int], np.ndarray]:
    """Deterministic DDIM sampling in N steps: timesteps s_k =
    floor((N - k) T / N) - 1 for k = 0 .. N-1 (T training steps), the head's
    time input t_k = s_k / T (one fp32 division, as the flow-matching times),
    and abar at each timestep followed by abar = 1 after the last step."""
    T = DDIM_TRAIN_STEPS
    s = [(n_steps - k) * T // n_steps - 1 for k in range(n_steps)]
    ts = [float(np.float32(sk) / np.float32(T)) for sk in s]
    ab = ddim_alpha_bar()
    abar = np.array([ab[sk] for sk in s] + [1.0])
    return ts, s, abar


def ddim_integrate(x0, eps: Callable[[np.ndarray, float], np.ndarray], n_steps):
    """DDIM (eta = 0): from x_k at abar_k, the clean estimate
    x0_hat = (x_k - sqrt(1 - abar_k) eps) / sqrt(abar_k) and
    x_{k+1} = sqrt(abar_{k+1}) x0_hat + sqrt(1 - abar_{k+1}) eps, with eps the
    head's output at (x_k, t_k); returns x_N."""
    ts, _, abar = ddim_schedule(n_steps)
    x = np.asarray(x0, dtype=np.float64)
    for k in range(n_steps):
        e = eps(x, ts[k])
        x0_hat = (x - np.sqrt(1.0 - abar[k]) * e) / np.sqrt(abar[k])
        x = np.sqrt(abar[k + 1]) * x0_hat + np.sqrt(1.0 - abar[k + 1]) * e
    return x


# ---------------------------------------------------------------------------
# Phase 1: VLM prefill
# ---------------------------------------------------------------------------

def vit_layer(P, cfg, l, x):
    """Pre-LN encoder layer: x += Attn(LN1 x); x += W2 GELU(W1 LN2 x + b1) + b2.
    Multi-head attention with biases on q, k, v and the output projection."""
    p = f"vit.{l}."
    t, d = x.shape
    nh = cfg["vit_heads"]
    hd = d // nh
    h = _op(layer_norm(x, _w(P, p + "ln1.g"), _w(P, p + "ln1.b")), cfg)
    q = _op(linear(h, _w(P, p + "q.w"), _w(P, p + "q.b")), cfg).reshape(t, nh, hd)
    k = _op(linear(h, _w(P, p + "k.w"), _w(P, p + "k.b")), cfg).reshape(t, nh, hd)
    v = _op(linear(h, _w(P, p + "v.w"), _w(P, p + "v.b")), cfg).reshape(t, nh, hd)
    a = _op(attention(q, k, v).reshape(t, d), cfg)
    x = x + linear(a, _w(P, p + "o.w"), _w(P, p + "o.b"))
    h2 = _op(layer_norm(x, _w(P, p + "ln2.g"), _w(P, p + "ln2.b")), cfg)
    f = _op(gelu_tanh(linear(h2, _w(P, p + "fc1.w"), _w(P, p + "fc1.b"))), cfg)
    return x + linear(f, _w(P, p + "fc2.w"), _w(P, p + "fc2.b"))


def vit_view(P, cfg, img):
    """One camera view: patch embedding (+ bias + learned position), the
    encoder layers, final LayerNorm. Returns [tokens_per_view, vit_dim]."""
    patches = _op(patchify(np.asarray(img, np.float64), cfg["patch"]), cfg)
    x = linear(patches, _w(P, "vit.patch.w"), _w(P, "vit.patch.b")) + _w(P, "vit.pos")
    for l in range(cfg["vit_layers"]):
        x = vit_layer(P, cfg, l, x)
    return layer_norm(x, _w(P, "vit.post.g"), _w(P, "vit.post.b"))


def image_tokens(P, cfg, pixels):
    """Views encoded independently, pixel-shuffled when the config asks for it,
    projected to the LM width, view-major."""
    outs = []
    gh, gw, s = cfg["img_h"] // cfg["patch"], cfg["img_w"] // cfg["patch"], cfg.get("shuffle", 1)
    for v in range(cfg["n_views"]):
        y = vit_view(P, cfg, pixels[v])
        if s > 1:
            y = pixel_shuffle(y, gh, gw, s)
        outs.append(linear(_op(y, cfg), _w(P, "proj.w"), _w(P, "proj.b")))
    return np.concatenate(outs, axis=0)


def prefix(P, cfg, frame, img=None):
    """LM input rows: [image tokens; E[ids] * sqrt(d_lm); W_s state + b_s];
    the cognition-token head appends its learned token row (unscaled)."""
    if img is None:
        img = image_tokens(P, cfg, frame["pixels"])
    rows = [img, _w(P, "lm.embed")[np.asarray(frame["ids"], dtype=np.int64)] * math.sqrt(cfg["lm_dim"])]
    if cfg["state_dim"] > 0:
        s = _op(np.asarray(frame["state"], np.float64)[None, :], cfg)
        rows.append(linear(s, _w(P, "state.w"), _w(P, "state.b")))
    if cfg.get("head", 0) == 2:
        rows.append(_w(P, "lm.cog"))
    return np.concatenate(rows, axis=0)


def geglu_mlp(P, cfg, p, x):
    """down(GELU(gate h) * up h) with h = RMSNorm2(x); no biases."""
    h = _op(rms_norm(x, _w(P, p + "rms2.g")), cfg)
    f = _op(gelu_tanh(linear(h, _w(P, p + "gate.w"))) * linear(h, _w(P, p + "up.w")), cfg)
    return linear(f, _w(P, p + "down.w"))


def qkv_rope(P, cfg, p, x, positions):
    """h = RMSNorm1(x); Q, K = RoPE(h W_q), RoPE(h W_k); V = h W_v (no biases)."""
    s = x.shape[0]
    nq, nkv, hd = cfg["lm_heads"], cfg["lm_kv_heads"], cfg["head_dim"]
    h = _op(rms_norm(x, _w(P, p + "rms1.g")), cfg)
    q = _op(rope(linear(h, _w(P, p + "q.w")).reshape(s, nq, hd), positions), cfg)
    k = _op(rope(linear(h, _w(P, p + "k.w")).reshape(s, nkv, hd), positions), cfg)
    v = _op(linear(h, _w(P, p + "v.w")).reshape(s, nkv, hd), cfg)
    return q, k, v


def decoder_layer(P, cfg, p, x, positions, past=None, kv_only=False):
    """One Gemma-style decoder layer with multi-query attention and no mask.

    Queries come from x; keys and values are [past K; own K], [past V; own V]
    (``past`` is None in the LM prefill and the LM cache layer in the action
    expert). Returns (x', K_own, V_own); with ``kv_only`` the attention output
    and MLP are skipped and x is returned unchanged."""
    s = x.shape[0]
    q, k, v = qkv_rope(P, cfg, p, x, positions)
    if kv_only:
        return x, k, v
    kall = k if past is None else np.concatenate([past[0], k], axis=0)
    vall = v if past is None else np.concatenate([past[1], v], axis=0)
    a = _op(attention(q, kall, vall).reshape(s, -1), cfg)
    x = x + linear(a, _w(P, p + "o.w"))
    x = x + geglu_mlp(P, cfg, p, x)
    return x, k, v


def lm_prefill(P, cfg, x0):
    """Prefix-LM prefill over the whole prefix (bidirectional, no mask),
    positions 0 .. P-1. Returns the KV cache: one (K_l, V_l) pair of
    [P, nkv, hd] per layer. The last layer's attention output and MLP do not
    reach the cache and are not computed."""
    x = np.asarray(x0, dtype=np.float64)
    pos = np.arange(x.shape[0])
    cache = []
    for l in range(cfg["lm_layers"]):
        last = l == cfg["lm_layers"] - 1
        x, k, v = decoder_layer(P, cfg, f"lm.{l}.", x, pos, kv_only=last)
        cache.append((k, v))
    return cache


def lm_features(P, cfg, x0):
    """Every LM layer over the prefix (positions 0 .. P-1, no mask), then the
    final RMSNorm: the features a DiT head reads. Returns (features, cache)."""
    x = np.asarray(x0, dtype=np.float64)
    pos = np.arange(x.shape[0])
    cache = []
    for l in range(cfg["lm_layers"]):
        x, k, v = decoder_layer(P, cfg, f"lm.{l}.", x, pos)
        cache.append((k, v))
    return rms_norm(x, _w(P, "lm.final.g")), cache


def dit_cross_kv(P, cfg, feats):
    """K, V of every cross-attention (even) DiT layer from the features, once
    per frame: [S, heads, hd] each, no biases."""
    s, nh = feats.shape[0], cfg["ex_heads"]
    hd = cfg["ex_dim"] // nh
    f = _op(feats, cfg)
    out = {}
    for l in range(0, cfg["ex_layers"], 2):
        p = f"ex.{l}."
        out[l] = (_op(linear(f, _w(P, p + "k.w")), cfg).reshape(s, nh, hd),
                  _op(linear(f, _w(P, p + "v.w")), cfg).reshape(s, nh, hd))
    return out


def vlm_prefill(P, cfg, frame, capture: Optional[dict] = None):
    """Phase 1. pi0 head: the per-layer KV cache. DiT head: the cross K/V of
    the DiT's even layers (from the LM features)."""
    img = image_tokens(P, cfg, frame["pixels"])
    x0 = prefix(P, cfg, frame, img)
    feats = None
    if cfg.get("head", 0) == 1:
        feats, cache = lm_features(P, cfg, x0)
        out = dit_cross_kv(P, cfg, feats)
    elif cfg.get("head", 0) == 2:
        feats, cache = lm_features(P, cfg, x0)
        out = cognition(P, cfg, feats)
    else:
        cache = lm_prefill(P, cfg, x0)
        out = cache
    if capture is not None:
        capture["image_tokens"] = img
        capture["prefix"] = x0
        capture["kv"] = cache
        if feats is not None:
            capture["features"] = feats
            capture["cog" if cfg.get("head", 0) == 2 else "cross_kv"] = out
    return out


def cognition(P, cfg, feats):
    """Hand-off of the cognition-token head (Section 2.1: CogACT's phase 1
    output is a cognition feature): the features' last row, the learned
    cognition token's final normalised output, projected to the head's width:
    c = W_c f + b_c, [ex_dim]."""
    f = _op(feats[-1:], cfg)
    return linear(f, _w(P, "cog.w"), _w(P, "cog.b"))[0]


# ---------------------------------------------------------------------------
# Phase 2: flow-matching action expert
# ---------------------------------------------------------------------------

def expert_velocity(P, cfg, cache, x, t):
    """v(x_t, t) of the pi0-style expert.

    a = W_in x + b_in; u = W_3 swish(W_2 [a; phi(t)] + b_2) + b_3; then per
    layer l: RMSNorm, Q/K/V with RoPE at positions P .. P+H-1, attention of the
    action queries over [K_l of the prefix; own K] and [V_l; own V] (no mask),
    output projection + residual, GeGLU MLP + residual; finally
    v = W_out RMSNorm_f(u) + b_out."""
    hlen = x.shape[0]
    npre = cache[0][0].shape[0]
    de = cfg["ex_dim"]
    a = _op(linear(_op(x, cfg), _w(P, "ex.in.w"), _w(P, "ex.in.b")), cfg)
    phi = _op(np.broadcast_to(sinusoid(t, de), (hlen, de)), cfg)
    hid = _op(swish(linear(np.concatenate([a, phi], axis=1), _w(P, "ex.time1.w"), _w(P, "ex.time1.b"))), cfg)
    u = linear(hid, _w(P, "ex.time2.w"), _w(P, "ex.time2.b"))
    pos = np.arange(npre, npre + hlen)
    for l in range(cfg["ex_layers"]):
        u, _, _ = decoder_layer(P, cfg, f"ex.{l}.", u, pos, past=cache[l])
    h = _op(rms_norm(u, _w(P, "ex.final.g")), cfg)
    return linear(h, _w(P, "ex.out.w"), _w(P, "ex.out.b"))


def dit_condition(P, cfg, t):
    """c = W_t2 swish(W_t1 phi_256(t) + b_t1) + b_t2 (the timestep embedder);
    returns the adaLN input swish(c) as stored for its GEMMs."""
    phi = _op(sinusoid(t, P["ex.time1.w"].shape[1])[None, :], cfg)
    hid = _op(swish(linear(phi, _w(P, "ex.time1.w"), _w(P, "ex.time1.b"))), cfg)
    c = linear(hid, _w(P, "ex.time2.w"), _w(P, "ex.time2.b"))
    return _op(swish(c), cfg)


def adaln(x, shift, scale):
    """LayerNorm without affine parameters, then x (1 + scale) + shift."""
    return layer_norm(x, 1.0 + scale, shift)


def dit_velocity(P, cfg, cross, x, t):
    """v(x_t, t) of the GR00T-style DiT head.

    X = W_a x + b_a + pos (fixed sinusoid positions); per layer l, from
    (shift1, scale1, gate1, shift2, scale2, gate2) = W_l swish(c) + b_l:
    X += gate1 * W_o MHA(adaLN(X; shift1, scale1)) -- cross-attention to the
    features' K/V on even layers, self-attention on odd ones, no mask, no
    biases -- then X += gate2 * W_2 GELU(W_1 adaLN(X; shift2, scale2)).
    Finally (shift, scale) = W_f swish(c) + b_f and v = W_out adaLN(X) + b_out."""
    hlen, de, nh = x.shape[0], cfg["ex_dim"], cfg["ex_heads"]
    hd = de // nh
    X = linear(_op(x, cfg), _w(P, "ex.in.w"), _w(P, "ex.in.b")) + positions_sinusoid(hlen, de)
    sc = dit_condition(P, cfg, t)
    for l in range(cfg["ex_layers"]):
        p = f"ex.{l}."
        mod = linear(sc, _w(P, p + "ada.w"), _w(P, p + "ada.b"))[0].reshape(6, de)
        sh1, sc1, g1, sh2, sc2, g2 = mod
        h = _op(adaln(X, sh1, sc1), cfg)
        q = _op(linear(h, _w(P, p + "q.w")), cfg).reshape(hlen, nh, hd)
        if l % 2 == 0:
            k, v = cross[l]
        else:
            k = _op(linear(h, _w(P, p + "k.w")), cfg).reshape(hlen, nh, hd)
            v = _op(linear(h, _w(P, p + "v.w")), cfg).reshape(hlen, nh, hd)
        a = _op(attention(q, k, v).reshape(hlen, de), cfg)
        X = X + g1 * linear(a, _w(P, p + "o.w"))
        h2 = _op(adaln(X, sh2, sc2), cfg)
        f = _op(gelu_tanh(linear(h2, _w(P, p + "fc1.w"))), cfg)
        X = X + g2 * linear(f, _w(P, p + "fc2.w"))
    sh, scl = linear(sc, _w(P, "ex.final.ada.w"), _w(P, "ex.final.ada.b"))[0].reshape(2, de)
    h = _op(adaln(X, sh, scl), cfg)
    return linear(h, _w(P, "ex.out.w"), _w(P, "ex.out.b"))


def cog_time_token(P, cfg, t):
    """The time token of the cognition-token head: W_t2 swish(W_t1 phi_256(t)
    + b_t1) + b_t2 (the DiT's timestep embedder without the final swish)."""
    phi = _op(sinusoid(t, P["ex.time1.w"].shape[1])[None, :], cfg)
    hid = _op(swish(linear(phi, _w(P, "ex.time1.w"), _w(P, "ex.time1.b"))), cfg)
    return linear(hid, _w(P, "ex.time2.w"), _w(P, "ex.time2.b"))[0]


def cog_velocity(P, cfg, cog, x, t):
    """Output of the cognition-token head (a DiT of self-attention layers,
    conditioned in context): the sequence [action tokens (W_a x + b_a + fixed
    sinusoid positions); the cognition vector; the time token] runs through
    pre-LN layers X += W_o MHA(LN1 X) (no mask, no biases), X += W_2 GELU(W_1
    LN2 X); the action rows' final LayerNorm, then W_out . + b_out. With the
    DDIM sampler this is the noise estimate."""
    hlen, de, nh = x.shape[0], cfg["ex_dim"], cfg["ex_heads"]
    hd = de // nh
    act = linear(_op(x, cfg), _w(P, "ex.in.w"), _w(P, "ex.in.b")) + positions_sinusoid(hlen, de)
    X = np.concatenate([act, np.asarray(cog, np.float64)[None, :], cog_time_token(P, cfg, t)[None, :]], axis=0)
    s = X.shape[0]
    for l in range(cfg["ex_layers"]):
        p = f"ex.{l}."
        h = _op(layer_norm(X, _w(P, p + "ln1.g"), _w(P, p + "ln1.b")), cfg)
        q = _op(linear(h, _w(P, p + "q.w")), cfg).reshape(s, nh, hd)
        k = _op(linear(h, _w(P, p + "k.w")), cfg).reshape(s, nh, hd)
        v = _op(linear(h, _w(P, p + "v.w")), cfg).reshape(s, nh, hd)
        a = _op(attention(q, k, v).reshape(s, de), cfg)
        X = X + linear(a, _w(P, p + "o.w"))
        h2 = _op(layer_norm(X, _w(P, p + "ln2.g"), _w(P, p + "ln2.b")), cfg)
        f = _op(gelu_tanh(linear(h2, _w(P, p + "fc1.w"))), cfg)
        X = X + linear(f, _w(P, p + "fc2.w"))
    h = _op(layer_norm(X[:hlen], _w(P, "ex.final.g"), _w(P, "ex.final.b")), cfg)
    return linear(h, _w(P, "ex.out.w"), _w(P, "ex.out.b"))


def action_denoise(P, cfg, cache, noise):
    """Euler integration of the head's velocity from x_0 = noise (t = 1) to
    t = 0, or DDIM steps with the head's output as the noise estimate
    (cfg["sampler"] == 1); returns the action chunk [chunk_len, action_dim].
    ``cache`` is the phase-1 hand-off (KV cache, the DiT's cross K/V, or the
    cognition vector)."""
    if cfg.get("head", 0) == 1:
        vel = lambda x, t: dit_velocity(P, cfg, cache, x, t)
    elif cfg.get("head", 0) == 2:
        vel = lambda x, t: cog_velocity(P, cfg, cache, x, t)
    else:
        vel = lambda x, t: expert_velocity(P, cfg, cache, x, t)
    if cfg.get("sampler", 0) == 1:
        return ddim_integrate(noise, vel, cfg["n_steps"])
    return euler_integrate(noise, vel, cfg["n_steps"])


def forward(P, cfg, frame, capture: Optional[dict] = None):
    """One frame through both phases: VLM prefill, then action denoising."""
    cache = vlm_prefill(P, cfg, frame, capture)
    return action_denoise(P, cfg, cache, frame["noise"])
