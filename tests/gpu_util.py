"""Helpers for the GPU tests: device copies of seeded inputs and a model
handle that is always destroyed. PyTorch provides device memory only."""
from __future__ import annotations

import contextlib
import sys

import numpy as np
import torch

import paper_2609_22335_amd as V
import synth


def say(msg: str) -> None:
    """Name the case before a GPU step, flushed, so a failing run shows it."""
    print(f"[gpu] {msg}", flush=True)
    sys.stdout.flush()


def to_dev(x: np.ndarray, dtype=None) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(x))
    if dtype is not None:
        t = t.to(dtype)
    return t.to("cuda")


def bf16_dev(x: np.ndarray) -> torch.Tensor:
    """bf16 bit patterns (RNE from fp32) on the device."""
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16).to("cuda")


def operand_dev(x: np.ndarray, dtype: int) -> torch.Tensor:
    return bf16_dev(x) if dtype == V.VLA_BF16 else to_dev(x.astype(np.float32))


def operand_values(x: np.ndarray, dtype: int) -> np.ndarray:
    """The values an operand has after the conversion operand_dev makes."""
    if dtype == V.VLA_BF16:
        return synth.bf16_round(x.astype(np.float32)).astype(np.float64)
    return x.astype(np.float32).astype(np.float64)


class DevFrame:
    """Device copies of one frame's inputs, kept alive with the vla_frame."""

    def __init__(self, fr):
        self.pixels = to_dev(fr["pixels"].astype(np.float32))
        self.ids = to_dev(fr["ids"].astype(np.int32))
        self.state = to_dev(fr["state"].astype(np.float32)) if fr["state"].size else None
        self.noise = to_dev(fr["noise"].astype(np.float32))
        self.c = V.make_frame(self.pixels, self.ids, self.state)


@contextlib.contextmanager
def model(cfg, seed=0):
    m = V.vla_create(cfg, seed)
    try:
        yield m
    finally:
        torch.cuda.synchronize()
        V.vla_destroy(m)


@contextlib.contextmanager
def context(m):
    c = V.vla_ctx_create(m)
    try:
        yield c
    finally:
        torch.cuda.synchronize()
        V.vla_ctx_destroy(c)


def run_frame(m, cfg, fr, stream=0, cross=None):
    """Prefill + denoise of one frame on one stream; returns (chunk, ctx-kv
    list). For a DiT head, ``cross`` (a dict) receives the cross K/V of every
    even DiT layer; for the cognition-token head, its cognition vector under
    the key "cog"."""
    d = synth.derived(cfg)
    df = DevFrame(fr)
    out = torch.empty_like(df.noise)
    with context(m) as c:
        V.vla_vlm_prefill(m, df.c, c, stream)
        V.vla_action_denoise(m, c, df.noise, out, stream)
        torch.cuda.synchronize()
        n = d["prefix"] * cfg["lm_kv_heads"] * cfg["head_dim"]
        kv = [V.vla_ctx_export_kv(m, c, l, n) for l in range(cfg["lm_layers"])]
        if cross is not None and cfg.get("head", 0) == synth.HEAD_DIT:
            for l in range(0, cfg["ex_layers"], 2):
                cross[l] = V.vla_ctx_export_cross(m, c, l, d["prefix"] * cfg["ex_dim"])
        if cross is not None and cfg.get("head", 0) == synth.HEAD_COG:
            cross["cog"] = V.vla_ctx_export_cog(m, c, cfg["ex_dim"]).astype(np.float64)
    return out.cpu().numpy().astype(np.float64), kv
