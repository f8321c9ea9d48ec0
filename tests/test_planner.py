"""The GEMM launch planner (host logic, no GPU), through vla_debug_gemm_plan.

Batched and one-frame runs give bit-identical caches and chunks because a
GEMM's split-K factor, and so each split's K range and the order in which
the partial sums are added, depends only on the rows it is planned for and
never on how many frames a launch stacks. These tests pin that invariant on
the shapes the presets run, and the measured planning rules."""
import pytest

import synth

V = pytest.importorskip("paper_2609_22335_amd")

BF16 = 1
BIAS, T, GELU, SWISH, GEGLU, QKV_ROPE, QKV_PLAIN, STEP, PART = range(9)


def plan(M, N, K, kind, plan_m=0, plan_batch=1, skinny=False):
    return V.vla_debug_gemm_plan(BF16, M, N, K, kind, skinny=skinny, plan_m=plan_m, plan_batch=plan_batch)


def _vlm_gemms(cfg):
    """(name, rows of one frame, N, K, kind) of the prefill's GEMMs."""
    dv, dl = cfg["vit_dim"], cfg["lm_dim"]
    views = cfg["n_views"]
    rows_v = views * (cfg["img_h"] // cfg["patch"]) * (cfg["img_w"] // cfg["patch"])
    prefix = rows_v // (cfg.get("pixel_shuffle", 1) ** 2 or 1) + cfg["n_text"]
    qkv_n = (cfg["lm_heads"] + 2 * cfg["lm_kv_heads"]) * cfg["head_dim"]
    qd = cfg["lm_heads"] * cfg["head_dim"]
    return [("vit.qkv", rows_v, 3 * dv, dv, T), ("vit.o", rows_v, dv, dv, PART),
            ("vit.fc1", rows_v, cfg["vit_mlp"], dv, GELU), ("vit.fc2", rows_v, dv, cfg["vit_mlp"], PART),
            ("lm.qkv", prefix, qkv_n, dl, QKV_ROPE), ("lm.o", prefix, dl, qd, PART),
            ("lm.gateup", prefix, 2 * cfg["lm_mlp"], dl, GEGLU), ("lm.down", prefix, dl, cfg["lm_mlp"], PART)]


@pytest.mark.parametrize("preset", ["pi0", "pi0_3view"])
def test_prefill_splits_do_not_depend_on_the_batch(preset):
    # a batched prefill of f frames stacks f x rows rows, planned for one
    # frame's rows with batches of up to 8: the same split count for every f
    cfg = getattr(synth, preset.upper())
    for name, rows, N, K, kind in _vlm_gemms(cfg):
        K8 = (K + 7) // 8 * 8
        splits = {f: plan(f * rows, N, K8, kind, plan_m=rows, plan_batch=8)["splits"] for f in range(1, 9)}
        assert len(set(splits.values())) == 1, (name, splits)


def test_action_loop_splits_do_not_depend_on_the_group():
    # the batched action loop's four expert GEMMs over f frames' rows are
    # planned for the largest group (8 frames)
    c = synth.PI0
    rows, de, mlp = c["chunk_len"] + 1, c["ex_dim"], c["ex_mlp"]
    qkv_n = (c["lm_heads"] + 2 * c["lm_kv_heads"]) * c["head_dim"]
    qd = c["lm_heads"] * c["head_dim"]
    for N, K, kind in ((qkv_n, de, QKV_ROPE), (de, qd, PART), (2 * mlp, de, GEGLU), (de, mlp, PART)):
        splits = {f: plan(f * rows, N, K, kind, plan_m=8 * rows)["splits"] for f in range(1, 9)}
        assert len(set(splits.values())) == 1, (N, K, splits)


def test_partial_scratch_is_splits_planes():
    # split-K partials: one fp32 M x N plane per split
    for M, N, K in ((305, 2048, 16384), (2440, 2048, 16384), (408, 1024, 4096), (2048, 1152, 4304)):
        p = plan(M, N, K, PART)
        assert p["scratch_floats"] == p["splits"] * M * N
    assert plan(2440, 2560, 2048, T)["scratch_floats"] == 0  # one split, no partials


def test_measured_rules():
    # the plans the measurements chose (batched pi0 prefill: 8 frames of the
    # one-frame rows; batched action loop: 8 frames of 51 rows)
    assert plan(2440, 2048, 16384, PART, 305, 8)["tile"] == (256, 256)
    assert plan(2440, 2048, 16384, PART, 305, 8)["splits"] == 3
    assert plan(2440, 2048, 2048, PART, 305, 8)["splits"] == 3  # LM O: one full round of 256 tiles
    assert plan(2440, 2048, 2048, PART, 305, 8)["tile"] == (256, 256)
    assert plan(2048, 1152, 4304, PART, 256, 8)["splits"] == 6  # ViT fc2
    assert plan(2048, 1152, 1152, PART, 256, 8)["splits"] == 1  # ViT O: short K, unsplit
    assert plan(408, 1024, 4096, PART, 408)["splits"] == 4       # expert down: two workgroups per CU at most
    assert plan(408, 1024, 2048, PART, 408)["splits"] == 4       # expert O
    assert plan(2440, 32768, 2048, GEGLU, 305, 8)["tile"] == (256, 256)


def test_256_tile_partials_make_one_full_round():
    # the 256 tile takes split-K partials only in one round of at least 7/8
    # of the 256 CUs (a second, partly empty round loses to the 128 tile)
    for M in range(1024, 8193, 256):
        for N, K in ((1152, 4304), (2048, 2048), (2048, 16384), (1024, 4096)):
            p = plan(M, N, K, PART, plan_m=M // 8, plan_batch=8)
            if p["tile"] == (256, 256) and p["splits"] > 1:
                assert 224 <= p["workgroups"] <= 256, (M, N, K, p)


def test_skinny_plan_and_errors():
    p = plan(50, 8192, 1024, GEGLU, skinny=True)
    assert p["tile"] == (0, 32) and p["workgroups"] == 256 * p["splits"]
    with pytest.raises(V.VlaError):
        plan(65, 8192, 1024, GEGLU, skinny=True)  # the skinny kernel takes at most 64 rows
    with pytest.raises(V.VlaError):
        plan(64, 64, 100, T)  # K a multiple of 8
    with pytest.raises(V.VlaError):
        plan(64, 64, 64, 9)  # unknown epilogue
