"""Pins of the seeded input generator shared by the oracle and the tests."""
import math

import numpy as np
import pytest
import torch

import synth


def test_splitmix64_published_vectors():
    # The SplitMix64 stream started from state 0 (Steele, Lea & Flood 2014);
    # these first outputs are the published reference values of the generator.
    got = [int(x) for x in synth._draws(0, 0, 4)]
    assert got == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F, 0xF88BB8A8724C81EC]


def test_fnv1a64_published_vectors():
    # FNV-1a 64 of "" is the offset basis; of "a" is 0xaf63dc4c8601ec8c.
    assert synth.fnv1a64("") == 0xCBF29CE484222325
    assert synth.fnv1a64("a") == 0xAF63DC4C8601EC8C
    assert synth.fnv1a64("foobar") == 0x85944171F73967E8


def test_counter_based_streams_are_splittable():
    a = synth.draws(7, "x", 100)
    b = synth.draws(7, "x", 60, start=40)
    assert np.array_equal(a[40:], b)
    assert not np.array_equal(synth.draws(7, "y", 10), a[:10])
    assert not np.array_equal(synth.draws(8, "x", 10), a[:10])


def test_normal_is_irwin_hall4_grid_and_moments():
    n = 1 << 21
    v = synth.normal(3, "w", n, 0.02).astype(np.float64)
    # mean 0, std 0.02 within 4 sigma of the sampling error
    assert abs(v.mean()) < 4 * 0.02 / math.sqrt(n)
    assert abs(v.std() - 0.02) < 4 * 0.02 / math.sqrt(2 * n)
    assert np.abs(v).max() <= 2 * math.sqrt(3) * 0.02 * (1 + 1e-6)
    # brute force for a handful of elements from the raw draws
    h = synth.draws(3, "w", 8)
    for i in range(8):
        s = sum((int(h[i]) >> (16 * j)) & 0xFFFF for j in range(4))
        z = ((s + 2) * 2.0 ** -16 - 2.0) * (synth.SQRT3 * 0.02)
        assert np.float32(z) == np.float32(v[i])
    g = synth.normal(3, "g", 4096, 0.02, mean=1.0)
    assert abs(float(g.mean()) - 1.0) < 0.01


def test_chunked_generation_matches_single_chunk():
    n = synth._CHUNK + 12345
    v = synth.normal(11, "big", n, 0.5)
    head = synth._normal_chunk(synth.stream_key(11, "big"), 0, 1000, 0.0, 0.5)
    tail = synth._normal_chunk(synth.stream_key(11, "big"), n - 1000, 1000, 0.0, 0.5)
    assert np.array_equal(v[:1000], head) and np.array_equal(v[-1000:], tail)


def test_uniform_and_ids():
    u = synth.uniform(1, "u", 100000, -1.0, 1.0)
    assert u.min() >= -1.0 and u.max() < 1.0 and abs(float(u.mean())) < 0.02
    h = synth.draws(1, "u", 4)
    for i in range(4):
        assert u[i] == np.float32(-1.0 + 2.0 * ((int(h[i]) >> 40) / 2.0 ** 24))
    ii = synth.ids(1, "i", 5000, 1024)
    assert ii.dtype == np.int32 and ii.min() >= 0 and ii.max() < 1024
    assert len(np.unique(ii)) > 900


def test_bf16_round_matches_torch():
    x = np.concatenate([synth.normal(5, "b", 100000, 3.0),
                        np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -1.0 - 2 ** -8, 0.0, 65504.0], np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(synth.bf16_round(x), ref)


def test_param_inventory_shapes():
    cfg = synth.PI0
    specs = synth.param_specs(cfg)
    names = [s[0] for s in specs]
    assert len(names) == len(set(names))
    d = dict((s[0], s[1]) for s in specs)
    assert d["vit.patch.w"] == (1152, 588)
    assert d["lm.0.q.w"] == (2048, 2048) and d["lm.0.k.w"] == (256, 2048)
    assert d["ex.0.q.w"] == (2048, 1024) and d["ex.0.o.w"] == (1024, 2048)
    assert "lm.17.o.w" not in d and "lm.16.down.w" in d
    assert synth.derived(cfg)["prefix"] == 305 and synth.derived(cfg)["kv_len"] == 355
    assert synth.derived(synth.TINY)["prefix"] == 80
    assert synth.derived(synth.PI0_3VIEW)["prefix"] == 833
    # ~2.6e9 parameters for the PaliGemma-shaped VLM + pi0-shaped expert
    assert 2.5e9 < synth.param_count(cfg) < 2.7e9


def test_frame_recipe():
    cfg = synth.micro()
    f0, f0b, f1 = synth.make_frame(cfg, 0, 0), synth.make_frame(cfg, 0, 0), synth.make_frame(cfg, 0, 1)
    for k in f0:
        assert np.array_equal(f0[k], f0b[k])
    assert not np.array_equal(f0["pixels"], f1["pixels"])
    assert f0["pixels"].shape == (1, 32, 32, 3) and f0["noise"].shape == (5, 3)
    assert f0["state"].shape == (3,) and f0["ids"].shape == (5,)
    assert synth.make_frame(synth.TINY, 0, 0)["state"].shape == (0,)
