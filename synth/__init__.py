"""Seeded synthetic inputs for the two-phase VLA hot path.

This module is shared by the tests, the benchmark and the oracle. It holds none
of the method's arithmetic: only

* the counter-based random generator (SplitMix64, Steele, Lea & Flood,
  "Fast splittable pseudorandom number generators", OOPSLA 2014), read as
  "output i of the SplitMix64 stream whose state starts at s";
* the distributions built on it (an Irwin-Hall(4) stand-in for N(mu, sigma),
  24-bit uniforms, integer ids);
* the configuration presets (shapes only) and the parameter inventory
  (names, shapes, init distribution) of the VLA the paper characterises
  (two phases: a VLM that encodes a frame and an instruction, then an action
  head that turns its output into an action chunk; Section 2.1);
* the per-frame input recipe (pixels, text ids, robot state, noise).

The C-ABI library implements the same published generator on its own side;
the two agree bit for bit (checked by the tests), which is how the oracle and
the GPU path compute on identical weights without either feeding the other.

Definitions (all arithmetic on uint64 wraps modulo 2**64):

    GAMMA = 0x9E3779B97F4A7C15
    mix64(z):  z = (z ^ z>>30) * 0xBF58476D1CE4E5B9
               z = (z ^ z>>27) * 0x94D049BB133111EB
               return z ^ z>>31
    key(seed, name)   = mix64((seed ^ fnv1a64(name)) + GAMMA)
    draw(seed, name, i) = mix64(key + (i + 1) * GAMMA)      # i-th output

    normal:  S = sum of the four 16-bit fields of the draw (integer),
             z = ((S + 2) * 2**-16 - 2) * (sqrt(3) * sigma)   [fp64, in
             this order, one rounding per operation], value = fp32(mu + z).
             Irwin-Hall(4) has variance 4/12, hence the sqrt(3); the tails
             are truncated at +-2*sqrt(3)*sigma.
    uniform: u = (draw >> 40) * 2**-24, value = fp32(lo + (hi - lo) * u).
    ids:     draw mod vocab.
"""
from __future__ import annotations

import concurrent.futures as _cf
import math
import os
from typing import Dict, List, Tuple

import numpy as np

GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)
SQRT3 = 1.7320508075688772  # fp64 nearest to sqrt(3)
FRAME_SEED_STRIDE = 1000003

_CHUNK = 1 << 20


def fnv1a64(name: str) -> int:
    """64-bit FNV-1a of the UTF-8 bytes of ``name``."""
    h = 0xCBF29CE484222325
    for byte in name.encode("utf-8"):
        h ^= byte
        h = (h * 0x100000001B3) & 0xFFFFFFFFFFFFFFFF
    return h


def _mix64_inplace(z: np.ndarray) -> np.ndarray:
    z ^= z >> np.uint64(30)
    z *= _M1
    z ^= z >> np.uint64(27)
    z *= _M2
    z ^= z >> np.uint64(31)
    return z


def mix64(z) -> np.ndarray:
    """SplitMix64 output mixer on a uint64 array (copy)."""
    return _mix64_inplace(np.array(z, dtype=np.uint64, copy=True))


def stream_key(seed: int, name: str) -> int:
    x = np.array([(int(seed) ^ fnv1a64(name)) & 0xFFFFFFFFFFFFFFFF], dtype=np.uint64)
    with np.errstate(over="ignore"):
        x += GAMMA
        return int(_mix64_inplace(x)[0])


def _draws(key: int, start: int, count: int) -> np.ndarray:
    with np.errstate(over="ignore"):
        idx = np.arange(start + 1, start + count + 1, dtype=np.uint64)
        idx *= GAMMA
        idx += np.uint64(key)
        return _mix64_inplace(idx)


def draws(seed: int, name: str, count: int, start: int = 0) -> np.ndarray:
    """Raw 64-bit outputs ``start .. start+count-1`` of the named stream."""
    return _draws(stream_key(seed, name), start, count)


def _normal_chunk(key: int, start: int, count: int, mean: float, std: float) -> np.ndarray:
    h = _draws(key, start, count)
    mask = np.uint64(0xFFFF)
    s = (h & mask) + ((h >> np.uint64(16)) & mask) + ((h >> np.uint64(32)) & mask) + (h >> np.uint64(48))
    z = (s + np.uint64(2)).astype(np.float64)
    z *= 2.0 ** -16
    z -= 2.0
    z *= SQRT3 * std
    if mean != 0.0:
        z = mean + z
    return z.astype(np.float32)


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def _chunked(fn, key: int, count: int, *args) -> np.ndarray:
    if count <= _CHUNK:
        return fn(key, 0, count, *args)
    out = np.empty(count, dtype=np.float32)
    starts = list(range(0, count, _CHUNK))

    def work(s):
        n = min(_CHUNK, count - s)
        out[s:s + n] = fn(key, s, n, *args)

    with _cf.ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(work, starts))
    return out


def normal(seed: int, name: str, count: int, std: float, mean: float = 0.0) -> np.ndarray:
    """fp32 Irwin-Hall(4) stand-in for N(mean, std**2), element i from draw i."""
    return _chunked(_normal_chunk, stream_key(seed, name), int(count), float(mean), float(std))


def _uniform_chunk(key: int, start: int, count: int, lo: float, hi: float) -> np.ndarray:
    h = _draws(key, start, count)
    u = (h >> np.uint64(40)).astype(np.float64) * 2.0 ** -24
    return (lo + (hi - lo) * u).astype(np.float32)


def uniform(seed: int, name: str, count: int, lo: float, hi: float) -> np.ndarray:
    """fp32 U[lo, hi) from the top 24 bits of each draw."""
    return _chunked(_uniform_chunk, stream_key(seed, name), int(count), float(lo), float(hi))


def ids(seed: int, name: str, count: int, vocab: int) -> np.ndarray:
    """int32 ids, draw mod vocab."""
    h = draws(seed, name, int(count))
    return (h % np.uint64(vocab)).astype(np.int32)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bfloat16 (round to nearest, ties to even), returned
    as fp32. Used to turn generated fp32 master weights into the bf16 weights a
    bf16 model stores; finite inputs only."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    b = x.view(np.uint32).astype(np.uint64)
    b = (b + np.uint64(0x7FFF) + ((b >> np.uint64(16)) & np.uint64(1))) & np.uint64(0xFFFF0000)
    return b.astype(np.uint32).view(np.float32)


# --------------------------------------------------------------------------
# Configuration presets (shapes only)
# --------------------------------------------------------------------------

F32, BF16 = 0, 1

CONFIG_FIELDS = (
    "dtype", "n_views", "img_h", "img_w", "patch",
    "vit_dim", "vit_heads", "vit_mlp", "vit_layers",
    "lm_dim", "lm_heads", "lm_kv_heads", "head_dim", "lm_mlp", "lm_layers",
    "vocab", "n_text", "state_dim",
    "ex_dim", "ex_mlp", "ex_layers", "chunk_len", "action_dim", "n_steps",
    "head", "shuffle", "ex_heads", "sampler",
)

#: Action-head families: the pi0-style expert that shares the LM's KV cache,
#: and the GR00T-style DiT that cross-attends to the LM's final features.
HEAD_PI0, HEAD_DIT, HEAD_COG = 0, 1, 2
#: Samplers: flow-matching Euler steps, or deterministic DDIM steps with the
#: head's output read as the noise estimate.
SAMPLER_EULER, SAMPLER_DDIM = 0, 1


def _cfg(**kw) -> Dict[str, int]:
    kw = dict(dict(head=HEAD_PI0, shuffle=1, ex_heads=0, sampler=SAMPLER_EULER), **kw)
    missing = [f for f in CONFIG_FIELDS if f not in kw]
    assert not missing, missing
    return {f: int(kw[f]) for f in CONFIG_FIELDS}


#: Tiny fp32 VLA: 64 patches of 16x16x3, 2+2+2 layers, chunk 8x7, 4 Euler steps.
TINY = _cfg(dtype=F32, n_views=1, img_h=128, img_w=128, patch=16,
            vit_dim=256, vit_heads=4, vit_mlp=1024, vit_layers=2,
            lm_dim=256, lm_heads=4, lm_kv_heads=1, head_dim=64, lm_mlp=1024, lm_layers=2,
            vocab=1024, n_text=16, state_dim=0,
            ex_dim=128, ex_mlp=512, ex_layers=2, chunk_len=8, action_dim=7, n_steps=4)

#: PaliGemma-3B-shaped VLM + pi0-shaped action expert, bf16.
PI0 = _cfg(dtype=BF16, n_views=1, img_h=224, img_w=224, patch=14,
           vit_dim=1152, vit_heads=16, vit_mlp=4304, vit_layers=27,
           lm_dim=2048, lm_heads=8, lm_kv_heads=1, head_dim=256, lm_mlp=16384, lm_layers=18,
           vocab=1024, n_text=48, state_dim=32,
           ex_dim=1024, ex_mlp=4096, ex_layers=18, chunk_len=50, action_dim=32, n_steps=10)

#: Stress case: three camera views (768 image tokens) and 64 text tokens.
PI0_3VIEW = dict(PI0, n_views=3, n_text=64)

#: Small shapes for fast tests: ragged everywhere (M=21 prefix rows, K=192,
#: action dim 3), one layer per stack.
def micro(dtype: int = F32) -> Dict[str, int]:
    return _cfg(dtype=dtype, n_views=1, img_h=32, img_w=32, patch=8,
                vit_dim=64, vit_heads=2, vit_mlp=136, vit_layers=1,
                lm_dim=64, lm_heads=2, lm_kv_heads=1, head_dim=32, lm_mlp=128, lm_layers=1,
                vocab=1024, n_text=5, state_dim=3,
                ex_dim=32, ex_mlp=64, ex_layers=1, chunk_len=5, action_dim=3, n_steps=2)


#: GR00T-shaped VLA: the ViT on 448x448 with 28x28 patches (256 patches),
#: 2x2 pixel shuffle to 64 tokens, a 12-layer multi-head LM whose final
#: normalised hidden states are the features, and a 16-layer DiT action head
#: (even layers cross-attend to the features, odd layers self-attend; adaLN
#: timestep conditioning), chunk 16x32, 4 Euler steps.
GR00T = _cfg(dtype=BF16, n_views=1, img_h=448, img_w=448, patch=28,
             vit_dim=1152, vit_heads=16, vit_mlp=4304, vit_layers=27,
             lm_dim=2048, lm_heads=16, lm_kv_heads=16, head_dim=128, lm_mlp=8192, lm_layers=12,
             vocab=1024, n_text=32, state_dim=0,
             ex_dim=1536, ex_mlp=6144, ex_layers=16, chunk_len=16, action_dim=32, n_steps=4,
             head=HEAD_DIT, shuffle=2, ex_heads=32)


def micro_dit(dtype: int = F32) -> Dict[str, int]:
    """Smallest DiT-head model: 4x4 patches shuffled to 2x2 tokens, head dim 48."""
    return _cfg(dtype=dtype, n_views=1, img_h=32, img_w=32, patch=8,
                vit_dim=64, vit_heads=2, vit_mlp=136, vit_layers=1,
                lm_dim=64, lm_heads=2, lm_kv_heads=2, head_dim=32, lm_mlp=128, lm_layers=2,
                vocab=1024, n_text=5, state_dim=0,
                ex_dim=96, ex_mlp=192, ex_layers=2, chunk_len=5, action_dim=3, n_steps=2,
                head=HEAD_DIT, shuffle=2, ex_heads=2)


#: GR00T-shaped wiring at tiny sizes (fp32): 8x8 patches -> 16 tokens,
#: 4 DiT layers of width 192 (4 heads of 48).
TINY_DIT = _cfg(dtype=F32, n_views=1, img_h=128, img_w=128, patch=16,
                vit_dim=256, vit_heads=4, vit_mlp=1024, vit_layers=2,
                lm_dim=256, lm_heads=4, lm_kv_heads=4, head_dim=64, lm_mlp=1024, lm_layers=2,
                vocab=1024, n_text=16, state_dim=0,
                ex_dim=192, ex_mlp=768, ex_layers=4, chunk_len=8, action_dim=7, n_steps=4,
                head=HEAD_DIT, shuffle=2, ex_heads=4)

#: The pi0-shaped model sampled with DDIM steps instead of Euler steps (a
#: diffusion head of the same shapes).
TINY_DDIM = dict(TINY, sampler=SAMPLER_DDIM)
PI0_DDIM = dict(PI0, sampler=SAMPLER_DDIM)

#: CogACT-shaped VLA: the PaliGemma-shaped VLM with a learned cognition token
#: appended to the prefix (48 text tokens, no state; prefix 305), every LM
#: layer run; its final normalised output row, projected to the head's
#: width, conditions a 300M-parameter DiT-L-shaped diffusion head (24
#: self-attention layers, d = 1024, 16 heads of 64, MLP 4096) that predicts
#: the noise of a 16 x 7 chunk over 10 DDIM steps.
COGACT = _cfg(dtype=BF16, n_views=1, img_h=224, img_w=224, patch=14,
              vit_dim=1152, vit_heads=16, vit_mlp=4304, vit_layers=27,
              lm_dim=2048, lm_heads=8, lm_kv_heads=1, head_dim=256, lm_mlp=16384, lm_layers=18,
              vocab=1024, n_text=48, state_dim=0,
              ex_dim=1024, ex_mlp=4096, ex_layers=24, chunk_len=16, action_dim=7, n_steps=10,
              head=HEAD_COG, ex_heads=16, sampler=SAMPLER_DDIM)

#: The cognition-token head at tiny sizes (fp32).
TINY_COG = _cfg(dtype=F32, n_views=1, img_h=128, img_w=128, patch=16,
                vit_dim=256, vit_heads=4, vit_mlp=1024, vit_layers=2,
                lm_dim=256, lm_heads=4, lm_kv_heads=1, head_dim=64, lm_mlp=1024, lm_layers=2,
                vocab=1024, n_text=16, state_dim=0,
                ex_dim=128, ex_mlp=512, ex_layers=2, chunk_len=8, action_dim=7, n_steps=4,
                head=HEAD_COG, ex_heads=2, sampler=SAMPLER_DDIM)


def micro_cog(dtype: int = F32) -> Dict[str, int]:
    """Smallest cognition-token model: one LM layer, two head layers of width 64."""
    return _cfg(dtype=dtype, n_views=1, img_h=32, img_w=32, patch=8,
                vit_dim=64, vit_heads=2, vit_mlp=136, vit_layers=1,
                lm_dim=64, lm_heads=2, lm_kv_heads=1, head_dim=32, lm_mlp=128, lm_layers=1,
                vocab=1024, n_text=5, state_dim=0,
                ex_dim=64, ex_mlp=128, ex_layers=2, chunk_len=5, action_dim=3, n_steps=2,
                head=HEAD_COG, ex_heads=2, sampler=SAMPLER_DDIM)


PRESETS = {"tiny": TINY, "pi0": PI0, "pi0_3view": PI0_3VIEW, "gr00t": GR00T, "tiny_dit": TINY_DIT,
           "tiny_ddim": TINY_DDIM, "pi0_ddim": PI0_DDIM, "cogact": COGACT, "tiny_cog": TINY_COG}


def derived(cfg: Dict[str, int]) -> Dict[str, int]:
    """Sizes that follow from a config: patches per view, image tokens, prefix
    length P, key length of the expert's joint attention."""
    ph, pw = cfg["img_h"] // cfg["patch"], cfg["img_w"] // cfg["patch"]
    t_view = ph * pw
    n_img = cfg["n_views"] * t_view // cfg["shuffle"] ** 2
    prefix = n_img + cfg["n_text"] + (1 if cfg["state_dim"] > 0 else 0) + (1 if cfg["head"] == HEAD_COG else 0)
    return {"grid_h": ph, "grid_w": pw, "tokens_per_view": t_view, "n_img": n_img,
            "prefix": prefix, "patch_dim": 3 * cfg["patch"] ** 2,
            "kv_len": prefix + cfg["chunk_len"]}


# --------------------------------------------------------------------------
# Parameter inventory: (name, shape, mean, std). Matrices are [out, in].
# --------------------------------------------------------------------------

WEIGHT_STD = 0.02
DIT_TIME_DIM = 256  # width of the DiT's sinusoidal timestep embedding


def param_specs(cfg: Dict[str, int]) -> List[Tuple[str, Tuple[int, ...], float, float]]:
    d = derived(cfg)
    s = WEIGHT_STD
    dv, dl, de = cfg["vit_dim"], cfg["lm_dim"], cfg["ex_dim"]
    hd, nq, nkv = cfg["head_dim"], cfg["lm_heads"], cfg["lm_kv_heads"]
    out: List[Tuple[str, Tuple[int, ...], float, float]] = []

    def w(name, shape):
        out.append((name, tuple(shape), 0.0, s))

    def g(name, n):  # norm gain: 1 + N(0, s)
        out.append((name, (n,), 1.0, s))

    w("vit.patch.w", (dv, d["patch_dim"]))
    w("vit.patch.b", (dv,))
    w("vit.pos", (d["tokens_per_view"], dv))
    for l in range(cfg["vit_layers"]):
        p = f"vit.{l}."
        g(p + "ln1.g", dv); w(p + "ln1.b", (dv,))
        for m in "qkv":
            w(p + m + ".w", (dv, dv)); w(p + m + ".b", (dv,))
        w(p + "o.w", (dv, dv)); w(p + "o.b", (dv,))
        g(p + "ln2.g", dv); w(p + "ln2.b", (dv,))
        w(p + "fc1.w", (cfg["vit_mlp"], dv)); w(p + "fc1.b", (cfg["vit_mlp"],))
        w(p + "fc2.w", (dv, cfg["vit_mlp"])); w(p + "fc2.b", (dv,))
    g("vit.post.g", dv); w("vit.post.b", (dv,))
    w("proj.w", (dl, dv * cfg["shuffle"] ** 2)); w("proj.b", (dl,))
    w("lm.embed", (cfg["vocab"], dl))
    if cfg["state_dim"] > 0:
        w("state.w", (dl, cfg["state_dim"])); w("state.b", (dl,))
    for l in range(cfg["lm_layers"]):
        p = f"lm.{l}."
        g(p + "rms1.g", dl)
        w(p + "q.w", (nq * hd, dl)); w(p + "k.w", (nkv * hd, dl)); w(p + "v.w", (nkv * hd, dl))
        if l == cfg["lm_layers"] - 1 and cfg["head"] == HEAD_PI0:
            break  # the last layer's attention output and MLP never reach the KV cache
        w(p + "o.w", (dl, nq * hd))
        g(p + "rms2.g", dl)
        w(p + "gate.w", (cfg["lm_mlp"], dl)); w(p + "up.w", (cfg["lm_mlp"], dl))
        w(p + "down.w", (dl, cfg["lm_mlp"]))
    a = cfg["action_dim"]
    if cfg["head"] == HEAD_DIT:
        g("lm.final.g", dl)
        w("ex.in.w", (de, a)); w("ex.in.b", (de,))
        w("ex.time1.w", (de, DIT_TIME_DIM)); w("ex.time1.b", (de,))
        w("ex.time2.w", (de, de)); w("ex.time2.b", (de,))
        for l in range(cfg["ex_layers"]):
            p = f"ex.{l}."
            w(p + "ada.w", (6 * de, de)); w(p + "ada.b", (6 * de,))
            kv_in = dl if l % 2 == 0 else de  # even layers cross-attend to the features
            w(p + "q.w", (de, de)); w(p + "k.w", (de, kv_in)); w(p + "v.w", (de, kv_in))
            w(p + "o.w", (de, de))
            w(p + "fc1.w", (cfg["ex_mlp"], de)); w(p + "fc2.w", (de, cfg["ex_mlp"]))
        w("ex.final.ada.w", (2 * de, de)); w("ex.final.ada.b", (2 * de,))
        w("ex.out.w", (a, de)); w("ex.out.b", (a,))
        return out
    if cfg["head"] == HEAD_COG:
        g("lm.final.g", dl)
        w("lm.cog", (1, dl))  # the learned cognition token, appended to the prefix
        w("cog.w", (de, dl)); w("cog.b", (de,))
        w("ex.in.w", (de, a)); w("ex.in.b", (de,))
        w("ex.time1.w", (de, DIT_TIME_DIM)); w("ex.time1.b", (de,))
        w("ex.time2.w", (de, de)); w("ex.time2.b", (de,))
        for l in range(cfg["ex_layers"]):
            p = f"ex.{l}."
            g(p + "ln1.g", de); w(p + "ln1.b", (de,))
            w(p + "q.w", (de, de)); w(p + "k.w", (de, de)); w(p + "v.w", (de, de))
            w(p + "o.w", (de, de))
            g(p + "ln2.g", de); w(p + "ln2.b", (de,))
            w(p + "fc1.w", (cfg["ex_mlp"], de)); w(p + "fc2.w", (de, cfg["ex_mlp"]))
        g("ex.final.g", de); w("ex.final.b", (de,))
        w("ex.out.w", (a, de)); w("ex.out.b", (a,))
        return out
    w("ex.in.w", (de, a)); w("ex.in.b", (de,))
    w("ex.time1.w", (de, 2 * de)); w("ex.time1.b", (de,))
    w("ex.time2.w", (de, de)); w("ex.time2.b", (de,))
    for l in range(cfg["ex_layers"]):
        p = f"ex.{l}."
        g(p + "rms1.g", de)
        w(p + "q.w", (nq * hd, de)); w(p + "k.w", (nkv * hd, de)); w(p + "v.w", (nkv * hd, de))
        w(p + "o.w", (de, nq * hd))
        g(p + "rms2.g", de)
        w(p + "gate.w", (cfg["ex_mlp"], de)); w(p + "up.w", (cfg["ex_mlp"], de))
        w(p + "down.w", (de, cfg["ex_mlp"]))
    g("ex.final.g", de)
    w("ex.out.w", (a, de)); w("ex.out.b", (a,))
    return out


def param_count(cfg: Dict[str, int]) -> int:
    return sum(math.prod(shape) for _, shape, _, _ in param_specs(cfg))


def make_param(cfg: Dict[str, int], seed: int, spec) -> np.ndarray:
    """One parameter as the model stores it, upcast to fp32: the generated fp32
    master value, rounded to bf16 for bf16 configs."""
    name, shape, mean, std = spec
    v = normal(seed, name, math.prod(shape), std, mean).reshape(shape)
    if cfg["dtype"] == BF16:
        v = bf16_round(v)
    return v


def make_params(cfg: Dict[str, int], seed: int) -> Dict[str, np.ndarray]:
    return {spec[0]: make_param(cfg, seed, spec) for spec in param_specs(cfg)}


# --------------------------------------------------------------------------
# Per-frame inputs
# --------------------------------------------------------------------------

def frame_seed(seed: int, r: int) -> int:
    return (int(seed) + FRAME_SEED_STRIDE * (int(r) + 1)) & 0xFFFFFFFFFFFFFFFF


def make_frame(cfg: Dict[str, int], seed: int, r: int) -> Dict[str, np.ndarray]:
    """Inputs of frame ``r``: camera images (HWC fp32 in [-1, 1)), instruction
    ids, robot state (N(0, 1); absent when state_dim is 0) and the flow-matching
    start noise x_0 (N(0, 1), [chunk_len, action_dim])."""
    fs = frame_seed(seed, r)
    v, h, w_ = cfg["n_views"], cfg["img_h"], cfg["img_w"]
    fr = {
        "pixels": uniform(fs, "frame.pixels", v * h * w_ * 3, -1.0, 1.0).reshape(v, h, w_, 3),
        "ids": ids(fs, "frame.ids", cfg["n_text"], cfg["vocab"]),
        "noise": normal(fs, "frame.noise", cfg["chunk_len"] * cfg["action_dim"], 1.0).reshape(
            cfg["chunk_len"], cfg["action_dim"]),
    }
    fr["state"] = (normal(fs, "frame.state", cfg["state_dim"], 1.0) if cfg["state_dim"] > 0
                   else np.zeros(0, np.float32))
    return fr


def chunk_noise(cfg: Dict[str, int], seed: int, r: int, j: int) -> np.ndarray:
    """Start noise x_0 of action chunk ``j`` of frame ``r`` under asynchronous
    inference (several chunks from one VLM output): chunk 0 is the frame's own
    noise, chunk j > 0 an independent N(0, 1) draw of the same shape."""
    if j == 0:
        return make_frame(cfg, seed, r)["noise"]
    return normal(frame_seed(seed, r), f"frame.noise.{j}", cfg["chunk_len"] * cfg["action_dim"], 1.0).reshape(
        cfg["chunk_len"], cfg["action_dim"])
