"""Pins of the oracle against what fixes it from outside: library routines,
closed forms, brute force on tiny inputs and invariants (CPU only).

The paper prints no worked example of the VLA forward, so no golden values
from it exist; every pin below is independent of the oracle's own code."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth
from oracle import vla_oracle as O

RNG = np.random.default_rng(1234)


def rnd(*shape, scale=1.0):
    return RNG.standard_normal(shape) * scale


def t64(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float64))


# ---------------------------------------------------------------- primitives

def test_layer_norm_vs_torch_and_properties():
    x, g, b = rnd(7, 33), rnd(33), rnd(33)
    ref = F.layer_norm(t64(x), (33,), t64(g), t64(b), eps=1e-6).numpy()
    assert np.allclose(O.layer_norm(x, g, b), ref, rtol=1e-12, atol=1e-12)
    y = O.layer_norm(x, np.ones(33), np.zeros(33))
    assert np.allclose(y.mean(-1), 0, atol=1e-12)
    assert np.allclose(y.var(-1), 1, atol=1e-5)
    assert np.allclose(O.layer_norm(3.5 * x, g, b), O.layer_norm(x, g, b), atol=1e-6)


def test_rms_norm_vs_torch_and_properties():
    x, g = rnd(5, 40), rnd(40)
    ref = F.rms_norm(t64(x), (40,), t64(g), eps=1e-6).numpy()
    assert np.allclose(O.rms_norm(x, g), ref, rtol=1e-12, atol=1e-12)
    y = O.rms_norm(x, np.ones(40))
    assert np.allclose(np.sqrt((y * y).mean(-1)), 1, atol=1e-5)
    assert np.allclose(O.rms_norm(0.25 * x, g), O.rms_norm(x, g), atol=1e-5)


def test_gelu_tanh():
    x = np.linspace(-6, 6, 1001)
    ref = F.gelu(t64(x), approximate="tanh").numpy()
    assert np.allclose(O.gelu_tanh(x), ref, rtol=1e-13, atol=1e-14)
    assert O.gelu_tanh(np.zeros(1))[0] == 0.0
    assert np.allclose(O.gelu_tanh(x) - O.gelu_tanh(-x), x, atol=1e-12)  # odd-part identity
    erf = F.gelu(t64(x)).numpy()
    assert np.abs(O.gelu_tanh(x) - erf).max() < 1e-3


def test_swish():
    x = np.linspace(-20, 20, 401)
    assert np.allclose(O.swish(x), F.silu(t64(x)).numpy(), rtol=1e-13, atol=1e-15)


def test_softmax_brute_force():
    s = rnd(3, 6, scale=4.0)
    for r in range(3):
        e = [math.exp(v) for v in s[r]]
        tot = sum(e)
        assert np.allclose(O.softmax(s)[r], [v / tot for v in e], rtol=1e-13)
    assert np.allclose(O.softmax(s + 100.0), O.softmax(s), rtol=1e-12)


def _attention_brute(q, k, v):
    sq, nq, hd = q.shape
    skv, nkv, _ = k.shape
    out = np.zeros_like(q)
    for i in range(sq):
        for h in range(nq):
            j = h * nkv // nq
            logits = [sum(q[i, h, d] * k[s, j, d] for d in range(hd)) / math.sqrt(hd) for s in range(skv)]
            m = max(logits)
            w = [math.exp(z - m) for z in logits]
            z = sum(w)
            for d in range(hd):
                out[i, h, d] = sum(w[s] * v[s, j, d] for s in range(skv)) / z
    return out


@pytest.mark.parametrize("nq,nkv", [(1, 1), (4, 1), (4, 2), (3, 3)])
def test_attention_brute_force(nq, nkv):
    q, k, v = rnd(3, nq, 4), rnd(5, nkv, 4), rnd(5, nkv, 4)
    assert np.allclose(O.attention(q, k, v), _attention_brute(q, k, v), rtol=1e-12, atol=1e-13)


def test_attention_vs_sdpa_gqa_and_invariants():
    q, k, v = rnd(9, 8, 16), rnd(13, 2, 16), rnd(13, 2, 16)
    ref = F.scaled_dot_product_attention(t64(q).transpose(0, 1), t64(k).transpose(0, 1),
                                         t64(v).transpose(0, 1), enable_gqa=True).transpose(0, 1).numpy()
    assert np.allclose(O.attention(q, k, v), ref, rtol=1e-11, atol=1e-12)
    # multi-query attention == multi-head attention with the KV head repeated
    k1, v1 = rnd(13, 1, 16), rnd(13, 1, 16)
    rep = O.attention(q, np.repeat(k1, 8, axis=1), np.repeat(v1, 8, axis=1))
    assert np.allclose(O.attention(q, k1, v1), rep, rtol=1e-13)
    # no mask: permuting the key/value rows changes nothing
    perm = RNG.permutation(13)
    assert np.allclose(O.attention(q, k[perm], v[perm]), O.attention(q, k, v), rtol=1e-12)
    # identical keys -> mean of the values
    kk = np.repeat(rnd(1, 2, 16), 13, axis=0)
    mean_v = np.repeat(v.mean(0)[None], 8 // 2, axis=1).reshape(1, 8, 16)
    got = O.attention(q, kk, v)
    assert np.allclose(got, np.broadcast_to(np.repeat(v.mean(0), 4, axis=0)[None], got.shape), rtol=1e-12)
    del mean_v
    # one dominant logit selects that value row
    kd = np.zeros((13, 1, 16)); kd[5, 0, :] = 1000.0
    qd = np.ones((2, 1, 16))
    assert np.allclose(O.attention(qd, kd, v[:, :1]), np.broadcast_to(v[5, :1], (2, 1, 16)))


def test_rope_complex_form_and_properties():
    x = rnd(6, 3, 8)
    pos = np.array([0, 1, 2, 7, 40, 300])
    y = O.rope(x, pos)
    half = 4
    z = x[..., :half] + 1j * x[..., half:]
    theta = 10000.0 ** (-np.arange(half) * 2.0 / 8)
    zr = z * np.exp(1j * pos[:, None, None] * theta[None, None, :])
    assert np.allclose(y, np.concatenate([zr.real, zr.imag], -1), rtol=1e-12, atol=1e-12)
    assert np.allclose(y[0], x[0])  # position 0 is the identity
    assert np.allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1))
    # scores depend on relative position only
    q, k = rnd(1, 1, 8), rnd(1, 1, 8)
    s1 = (O.rope(q, [5]) * O.rope(k, [2])).sum()
    s2 = (O.rope(q, [105]) * O.rope(k, [102])).sum()
    assert abs(s1 - s2) < 1e-9


def test_rope_vs_transformers():
    from transformers.models.gemma.modeling_gemma import apply_rotary_pos_emb
    hd = 16
    x = rnd(5, 2, hd)
    pos = np.arange(10, 15, dtype=np.float64)
    inv = 1.0 / (10000.0 ** (np.arange(0, hd, 2) / hd))
    emb = np.concatenate([pos[:, None] * inv, pos[:, None] * inv], -1)
    cos, sin = t64(np.cos(emb))[None], t64(np.sin(emb))[None]
    xt = t64(x).transpose(0, 1)[None]  # [1, heads, seq, hd]
    ref, _ = apply_rotary_pos_emb(xt, xt, cos, sin)
    assert np.allclose(O.rope(x, pos), ref[0].transpose(0, 1).numpy(), rtol=1e-12, atol=1e-12)


def test_patchify_brute_force():
    img = rnd(12, 8, 3)
    p = 4
    out = O.patchify(img, p)
    assert out.shape == (6, 48)
    for i in range(3):
        for j in range(2):
            t = i * 2 + j
            vec = [img[i * p + r, j * p + c, ch] for r in range(p) for c in range(p) for ch in range(3)]
            assert np.array_equal(out[t], vec)


def test_sinusoid_closed_form():
    d = 16
    phi0 = O.sinusoid(0.0, d)
    assert np.array_equal(phi0, np.r_[np.zeros(8), np.ones(8)])
    t = 0.3
    phi = O.sinusoid(t, d)
    assert np.isclose(phi[0], math.sin(2 * math.pi * t / 4e-3))
    assert np.isclose(phi[7], math.sin(2 * math.pi * t / 4.0))
    assert np.isclose(phi[8 + 7], math.cos(2 * math.pi * t / 4.0))
    assert np.allclose(phi[:8] ** 2 + phi[8:] ** 2, 1.0)


def test_flow_times():
    ts, dt = O.flow_times(10)
    assert np.float32(ts[1]) == np.float32(0.9) and ts[0] == 1.0 and len(ts) == 10
    assert np.float32(dt) == np.float32(-0.1)
    ts4, dt4 = O.flow_times(4)
    assert ts4 == [1.0, 0.75, 0.5, 0.25] and dt4 == -0.25


def test_euler_closed_forms():
    x0 = rnd(4, 3)
    _, dt = O.flow_times(10)
    lam = -0.7
    got = O.euler_integrate(x0, lambda x, t: lam * x, 10)
    assert np.allclose(got, (1 + lam * dt) ** 10 * x0, rtol=1e-13)
    b = rnd(4, 3)
    assert np.allclose(O.euler_integrate(x0, lambda x, t: b, 10), x0 + 10 * dt * b, rtol=1e-13)
    M = rnd(3, 3, scale=0.3)
    got = O.euler_integrate(x0, lambda x, t: x @ M.T, 5)
    _, dt5 = O.flow_times(5)
    A = np.linalg.matrix_power(np.eye(3) + dt5 * M, 5)
    assert np.allclose(got, x0 @ A.T, rtol=1e-12)
    # time dependence: v = t -> x_N = x_0 + dt * sum_k t_k
    ts, _ = O.flow_times(4)
    assert np.allclose(O.euler_integrate(x0, lambda x, t: np.full_like(x, t), 4), x0 - 0.25 * sum(ts))


def test_bf16_operand_rounding_vs_torch():
    x = rnd(10000, scale=5.0)
    ref = t64(x).to(torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(O.bf16(x), ref)
    assert np.array_equal(O.bf16(synth.normal(2, "q", 1000, 1.0)), synth.bf16_round(synth.normal(2, "q", 1000, 1.0)))


# ------------------------------------------------------- layers vs libraries

def _siglip_layer(cfg, P, l):
    from transformers import SiglipVisionConfig
    from transformers.models.siglip.modeling_siglip import SiglipEncoderLayer
    c = SiglipVisionConfig(hidden_size=cfg["vit_dim"], intermediate_size=cfg["vit_mlp"],
                           num_attention_heads=cfg["vit_heads"], layer_norm_eps=1e-6,
                           hidden_act="gelu_pytorch_tanh", attention_dropout=0.0)
    c._attn_implementation = "eager"
    m = SiglipEncoderLayer(c).double().eval()
    p = f"vit.{l}."
    sd = {
        "layer_norm1.weight": P[p + "ln1.g"], "layer_norm1.bias": P[p + "ln1.b"],
        "layer_norm2.weight": P[p + "ln2.g"], "layer_norm2.bias": P[p + "ln2.b"],
        "self_attn.q_proj.weight": P[p + "q.w"], "self_attn.q_proj.bias": P[p + "q.b"],
        "self_attn.k_proj.weight": P[p + "k.w"], "self_attn.k_proj.bias": P[p + "k.b"],
        "self_attn.v_proj.weight": P[p + "v.w"], "self_attn.v_proj.bias": P[p + "v.b"],
        "self_attn.out_proj.weight": P[p + "o.w"], "self_attn.out_proj.bias": P[p + "o.b"],
        "mlp.fc1.weight": P[p + "fc1.w"], "mlp.fc1.bias": P[p + "fc1.b"],
        "mlp.fc2.weight": P[p + "fc2.w"], "mlp.fc2.bias": P[p + "fc2.b"],
    }
    m.load_state_dict({k: t64(v) for k, v in sd.items()})
    return m


def _gemma_layer(cfg, P, prefix, l, dim, mlp):
    from transformers import GemmaConfig
    from transformers.models.gemma.modeling_gemma import GemmaDecoderLayer
    c = GemmaConfig(hidden_size=dim, intermediate_size=mlp, num_attention_heads=cfg["lm_heads"],
                    num_key_value_heads=cfg["lm_kv_heads"], head_dim=cfg["head_dim"], rms_norm_eps=1e-6,
                    hidden_activation="gelu_pytorch_tanh", attention_bias=False, vocab_size=cfg["vocab"])
    c._attn_implementation = "eager"
    m = GemmaDecoderLayer(c, layer_idx=l).double().eval()
    p = f"{prefix}.{l}."
    sd = {  # Gemma's RMSNorm scales by (1 + weight)
        "input_layernorm.weight": P[p + "rms1.g"] - 1.0,
        "post_attention_layernorm.weight": P[p + "rms2.g"] - 1.0,
        "self_attn.q_proj.weight": P[p + "q.w"], "self_attn.k_proj.weight": P[p + "k.w"],
        "self_attn.v_proj.weight": P[p + "v.w"], "self_attn.o_proj.weight": P[p + "o.w"],
        "mlp.gate_proj.weight": P[p + "gate.w"], "mlp.up_proj.weight": P[p + "up.w"],
        "mlp.down_proj.weight": P[p + "down.w"],
    }
    m.load_state_dict({k: t64(np.asarray(v, np.float64)) for k, v in sd.items()})
    return m


def _rope_tables(hd, pos):
    inv = 1.0 / (10000.0 ** (np.arange(0, hd, 2) / hd))
    ang = np.asarray(pos, np.float64)[:, None] * inv
    emb = np.concatenate([ang, ang], -1)
    return t64(np.cos(emb))[None], t64(np.sin(emb))[None]


def _cfg_params(cfg=None):
    cfg = cfg or synth.micro()
    return cfg, synth.make_params(cfg, 0)


def test_vit_layer_vs_siglip():
    cfg, P = _cfg_params()
    x = rnd(16, cfg["vit_dim"])
    ref = _siglip_layer(cfg, P, 0)(t64(x)[None], None)
    ref = (ref[0] if isinstance(ref, tuple) else ref)[0].detach().numpy()
    # transformers computes the softmax in fp32, hence 1e-7
    assert np.allclose(O.vit_layer(P, cfg, 0, x), ref, rtol=1e-7, atol=1e-7)


def test_lm_decoder_layer_vs_gemma():
    from transformers.cache_utils import DynamicCache
    cfg = dict(synth.micro(), lm_layers=2)
    P = synth.make_params(cfg, 0)
    x = rnd(21, cfg["lm_dim"])
    pos = np.arange(21)
    m = _gemma_layer(cfg, P, "lm", 0, cfg["lm_dim"], cfg["lm_mlp"])
    cache = DynamicCache()
    with torch.no_grad():
        ref = m(t64(x)[None], attention_mask=None, position_ids=torch.arange(21)[None],
                past_key_values=cache, use_cache=True, position_embeddings=_rope_tables(cfg["head_dim"], pos))
    ref = (ref[0] if isinstance(ref, tuple) else ref)[0].numpy()
    got, k, v = O.decoder_layer(P, cfg, "lm.0.", x, pos)
    # Gemma's RMSNorm runs in fp32, hence the tolerance
    assert np.allclose(got, ref, rtol=2e-5, atol=2e-5)
    assert np.allclose(k, cache.layers[0].keys[0].transpose(0, 1).numpy(), rtol=2e-5, atol=2e-5)
    assert np.allclose(v, cache.layers[0].values[0].transpose(0, 1).numpy(), rtol=2e-5, atol=2e-5)


def _expert_torch(cfg, P, kv, x, t):
    """The expert's velocity assembled from torch and transformers modules:
    in-proj, time MLP, Gemma decoder layers with the prefix K/V of `kv`
    ([(K, V)] per layer, [n, n_kv, hd]) in a DynamicCache at positions n..,
    final RMSNorm, out-proj."""
    from transformers.cache_utils import DynamicCache
    H, de, hd, L = cfg["chunk_len"], cfg["ex_dim"], cfg["head_dim"], cfg["ex_layers"]
    npre = kv[0][0].shape[0]
    lin = lambda w, b=None: (lambda z: F.linear(z, t64(P[w]), None if b is None else t64(P[b])))
    with torch.no_grad():
        a = lin("ex.in.w", "ex.in.b")(t64(x))
        phi = t64(O.sinusoid(t, de))[None].expand(H, de)
        u = lin("ex.time2.w", "ex.time2.b")(F.silu(lin("ex.time1.w", "ex.time1.b")(torch.cat([a, phi], 1))))
        cache = DynamicCache()
        for l in range(L):
            cache.update(t64(kv[l][0]).transpose(0, 1)[None], t64(kv[l][1]).transpose(0, 1)[None], l)
        pos = np.arange(npre, npre + H)
        h = u[None]
        for l in range(L):
            m = _gemma_layer(cfg, P, "ex", l, de, cfg["ex_mlp"])
            h = m(h, attention_mask=None, position_ids=torch.from_numpy(pos)[None], past_key_values=cache,
                  use_cache=True, position_embeddings=_rope_tables(hd, pos))
            h = h[0] if isinstance(h, tuple) else h
        return lin("ex.out.w", "ex.out.b")(F.rms_norm(h[0], (de,), t64(P["ex.final.g"]), eps=1e-6)).numpy()


def test_expert_velocity_vs_library_assembly():
    """The whole expert (in-proj, time MLP, decoder layers with the prefix KV in
    the cache at positions P.., final RMSNorm, out-proj) assembled from torch and
    transformers modules."""
    cfg = dict(synth.micro(), lm_layers=2, ex_layers=2)
    P = synth.make_params(cfg, 0)
    npre, H, A = 21, cfg["chunk_len"], cfg["action_dim"]
    nkv, hd = cfg["lm_kv_heads"], cfg["head_dim"]
    kv = [(rnd(npre, nkv, hd), rnd(npre, nkv, hd)) for _ in range(2)]
    x, t = rnd(H, A), 0.75
    got = O.expert_velocity(P, cfg, kv, x, t)
    assert np.allclose(got, _expert_torch(cfg, P, kv, x, t), rtol=2e-5, atol=2e-5)


def _prefill_torch(cfg, P, fr):
    """Phase 1 of one view from library modules (patches by unfold, SigLIP
    layers, post-LN, projector, text embedding x sqrt(d), state row, Gemma
    layers writing a DynamicCache; the last layer only projects K and V);
    returns [(K, V)] per LM layer as [n, n_kv, hd] arrays."""
    from transformers.cache_utils import DynamicCache
    from transformers.models.gemma.modeling_gemma import apply_rotary_pos_emb
    p, dl, L = cfg["patch"], cfg["lm_dim"], cfg["lm_layers"]
    with torch.no_grad():
        img = t64(fr["pixels"][0])
        gh, gw = cfg["img_h"] // p, cfg["img_w"] // p
        # unfold-based patch extraction, reordered to (row, col, channel)
        patches = img.permute(2, 0, 1).unfold(1, p, p).unfold(2, p, p)  # [3, gh, gw, p, p]
        patches = patches.permute(1, 2, 3, 4, 0).reshape(gh * gw, p * p * 3)
        x = F.linear(patches, t64(P["vit.patch.w"]), t64(P["vit.patch.b"])) + t64(P["vit.pos"])
        for l in range(cfg["vit_layers"]):
            y = _siglip_layer(cfg, P, l)(x[None], None)
            x = (y[0] if isinstance(y, tuple) else y)[0]
        x = F.layer_norm(x, (cfg["vit_dim"],), t64(P["vit.post.g"]), t64(P["vit.post.b"]), eps=1e-6)
        img_tok = F.linear(x, t64(P["proj.w"]), t64(P["proj.b"]))
        emb = torch.nn.Embedding(cfg["vocab"], dl).double()
        emb.weight.data = t64(P["lm.embed"])
        txt = emb(torch.from_numpy(fr["ids"].astype(np.int64))) * math.sqrt(dl)
        st = F.linear(t64(fr["state"])[None], t64(P["state.w"]), t64(P["state.b"]))
        h = torch.cat([img_tok, txt, st], 0)[None]
        n = h.shape[1]
        cos, sin = _rope_tables(cfg["head_dim"], np.arange(n))
        cache = DynamicCache()
        for l in range(L):
            if l == L - 1:  # the last layer has no MLP / o-proj weights: only its K, V matter
                q = F.rms_norm(h[0], (dl,), t64(P[f"lm.{l}.rms1.g"]), eps=1e-6)
                k = F.linear(q, t64(P[f"lm.{l}.k.w"])).reshape(n, cfg["lm_kv_heads"], -1)
                v = F.linear(q, t64(P[f"lm.{l}.v.w"])).reshape(n, cfg["lm_kv_heads"], -1)
                kt = k.transpose(0, 1)[None]
                kt, _ = apply_rotary_pos_emb(kt, kt, cos, sin)
                cache.update(kt, v.transpose(0, 1)[None], l)
                break
            m = _gemma_layer(cfg, P, "lm", l, dl, cfg["lm_mlp"])
            h = m(h, attention_mask=None, position_ids=torch.arange(n)[None], past_key_values=cache,
                  use_cache=True, position_embeddings=(cos, sin))
            h = h[0] if isinstance(h, tuple) else h
    return [(cache.layers[l].keys[0].transpose(0, 1).numpy(), cache.layers[l].values[0].transpose(0, 1).numpy())
            for l in range(L)]


def test_vlm_prefill_vs_library_assembly():
    """Phase 1 end to end (ViT from SigLIP layers, post-LN, projector, text
    embedding x sqrt(d), state row, Gemma layers writing the cache)."""
    cfg = dict(synth.micro(), vit_layers=2, lm_layers=2)
    P = synth.make_params(cfg, 0)
    fr = synth.make_frame(cfg, 0, 0)
    got = O.vlm_prefill(P, cfg, fr)
    ref = _prefill_torch(cfg, P, fr)
    for l in range(2):
        assert np.allclose(got[l][0], ref[l][0], rtol=5e-5, atol=5e-5)
        assert np.allclose(got[l][1], ref[l][1], rtol=5e-5, atol=5e-5)


def test_full_forward_vs_library_assembly():
    """Both phases end to end: the library prefill writes the cache, then the
    library expert is integrated from the noise at t = 1 to t = 0 in N Euler
    steps (flow-matching section of the paper's background: the action head
    integrates a learned velocity field), with t_k = (N - k) / N and
    dt = -1 / N each a single fp32 division (a reading of the schedule). The
    oracle's chunk must match, so a mistake in how the forward joins the two
    phases (the cache layers, the time schedule, the update's sign or step
    count) fails here."""
    cfg = dict(synth.micro(), vit_layers=2, lm_layers=3, ex_layers=3)
    P = synth.make_params(cfg, 0)
    fr = synth.make_frame(cfg, 0, 0)
    got = O.forward(P, cfg, fr)
    kv = _prefill_torch(cfg, P, fr)
    N = cfg["n_steps"]
    dt = float(np.float32(-1.0) / np.float32(N))
    x = fr["noise"].astype(np.float64)
    for k in range(N):
        t = float(np.float32(N - k) / np.float32(N))
        x = x + dt * _expert_torch(cfg, P, kv, x, t)
    assert N >= 2 and not np.allclose(x, fr["noise"], atol=1e-3)  # the loop moved the state
    # the two sides agree to ~3e-9; a step-count, time-shift, dt-sign or
    # cache-layer mistake moves the chunk by 1.8e-2 or more
    assert np.allclose(got, x, rtol=1e-6, atol=1e-6)


# ------------------------------------------------------------ model wiring

def test_zero_out_projection_gives_noise_minus_bias():
    cfg = synth.micro()
    P = synth.make_params(cfg, 0)
    P["ex.out.w"] = np.zeros_like(P["ex.out.w"])
    fr = synth.make_frame(cfg, 0, 0)
    chunk = O.forward(P, cfg, fr)
    _, dt = O.flow_times(cfg["n_steps"])
    b = P["ex.out.b"].astype(np.float64)
    assert np.allclose(chunk, fr["noise"].astype(np.float64) + cfg["n_steps"] * dt * b, rtol=0, atol=1e-12)
    assert np.allclose(chunk, fr["noise"] - P["ex.out.b"], atol=1e-6)


def test_vit_without_residual_branches_is_patch_embedding():
    cfg = synth.micro()
    P = synth.make_params(cfg, 0)
    for n in ("o.w", "o.b", "fc2.w", "fc2.b"):
        P["vit.0." + n] = np.zeros_like(P["vit.0." + n])
    img = synth.make_frame(cfg, 0, 0)["pixels"][0]
    emb = O.patchify(img.astype(np.float64), cfg["patch"]) @ P["vit.patch.w"].T.astype(np.float64)
    emb = emb + P["vit.patch.b"] + P["vit.pos"]
    want = O.layer_norm(emb, P["vit.post.g"], P["vit.post.b"])
    assert np.allclose(O.vit_view(P, cfg, img), want, rtol=1e-12, atol=1e-12)


def test_prefix_rows():
    cfg = synth.micro()
    P = synth.make_params(cfg, 0)
    fr = synth.make_frame(cfg, 0, 0)
    img = rnd(synth.derived(cfg)["n_img"], cfg["lm_dim"])
    x0 = O.prefix(P, cfg, fr, img)
    assert x0.shape == (synth.derived(cfg)["prefix"], cfg["lm_dim"])
    n = img.shape[0]
    for i, tok in enumerate(fr["ids"]):
        assert np.allclose(x0[n + i], P["lm.embed"][tok] * 8.0)  # sqrt(64)
    st = sum(P["state.w"][:, j].astype(np.float64) * fr["state"][j] for j in range(3)) + P["state.b"]
    assert np.allclose(x0[-1], st)


def test_bf16_config_differs_only_by_operand_rounding():
    """The bf16 model is the fp32 model with bf16 storage at the documented
    points; on the same (bf16-valued) weights the two chunks stay close."""
    c32, c16 = synth.micro(synth.F32), synth.micro(synth.BF16)
    P = synth.make_params(c16, 0)
    fr = synth.make_frame(c16, 0, 0)
    a, b = O.forward(P, c32, fr), O.forward(P, c16, fr)
    assert 0 < np.abs(a - b).max() < 2e-2


def test_multi_view_is_view_major_and_independent():
    cfg = dict(synth.micro(), n_views=2)
    P = synth.make_params(cfg, 0)
    fr = synth.make_frame(cfg, 0, 0)
    toks = O.image_tokens(P, cfg, fr["pixels"])
    single = dict(cfg, n_views=1)
    for v in range(2):
        want = O.image_tokens(P, single, fr["pixels"][v:v + 1])
        assert np.allclose(toks[v * 16:(v + 1) * 16], want, rtol=1e-13)


# ------------------------------------------------------------ DiT action head

def test_pixel_shuffle_hand_example_and_vs_torch():
    # 4x4 grid of one-channel tokens numbered in raster order: coarse token
    # (i, j) holds fine tokens (2i, 2j), (2i, 2j+1), (2i+1, 2j), (2i+1, 2j+1)
    x = np.arange(16, dtype=np.float64)[:, None]
    want = np.array([[0, 1, 4, 5], [2, 3, 6, 7], [8, 9, 12, 13], [10, 11, 14, 15]], dtype=np.float64)
    assert np.array_equal(O.pixel_shuffle(x, 4, 4, 2), want)
    assert np.array_equal(O.pixel_shuffle(x, 4, 4, 1), x)
    # channels fastest: torch's space-to-depth orders channels (c, dy, dx)
    gh, gw, c, s = 6, 4, 5, 2
    y = rnd(gh * gw, c)
    t = F.pixel_unshuffle(t64(y).T.reshape(1, c, gh, gw), s)[0]  # [c s s, gh/s, gw/s]
    t = t.reshape(c, s * s, gh // s, gw // s).permute(2, 3, 1, 0).reshape(-1, s * s * c)
    assert np.array_equal(O.pixel_shuffle(y, gh, gw, s), t.numpy())


def test_positions_sinusoid_closed_form():
    pos = O.positions_sinusoid(3, 4)  # w = [1, 10000^-1/2]
    w1 = 10000.0 ** -0.5
    want = np.array([[0, 0, 1, 1], [math.sin(1), math.sin(w1), math.cos(1), math.cos(w1)],
                     [math.sin(2), math.sin(2 * w1), math.cos(2), math.cos(2 * w1)]])
    assert np.allclose(pos, want, rtol=0, atol=1e-15)


def _dit_torch(P, cfg, cross, x, t):
    """The DiT velocity assembled from torch primitives: LayerNorm without
    affine, SDPA (multi-head), tanh-GELU, SiLU."""
    de, nh, H = cfg["ex_dim"], cfg["ex_heads"], x.shape[0]
    hd = de // nh
    lin = lambda z, w, b=None: F.linear(z, t64(P[w]), None if b is None else t64(P[b]))
    ln = lambda z, shift, scale: F.layer_norm(z, (de,), eps=1e-6) * (1 + scale) + shift
    half = de // 2
    ang = torch.arange(H, dtype=torch.float64)[:, None] * 10000.0 ** (-torch.arange(half, dtype=torch.float64) / half)
    X = lin(t64(x), "ex.in.w", "ex.in.b") + torch.cat([ang.sin(), ang.cos()], 1)
    phi = t64(O.sinusoid(t, 256))[None]
    c = lin(F.silu(lin(phi, "ex.time1.w", "ex.time1.b")), "ex.time2.w", "ex.time2.b")
    sc = F.silu(c)
    heads = lambda z: z.reshape(-1, nh, hd).transpose(0, 1)[None]
    for l in range(cfg["ex_layers"]):
        p = f"ex.{l}."
        sh1, sc1, g1, sh2, sc2, g2 = lin(sc, p + "ada.w", p + "ada.b")[0].reshape(6, de)
        h = ln(X, sh1, sc1)
        q = lin(h, p + "q.w")
        if l % 2 == 0:
            k, v = (t64(a).reshape(a.shape[0], de) for a in cross[l])
        else:
            k, v = lin(h, p + "k.w"), lin(h, p + "v.w")
        a = F.scaled_dot_product_attention(heads(q), heads(k), heads(v))[0].transpose(0, 1).reshape(H, de)
        X = X + g1 * lin(a, p + "o.w")
        X = X + g2 * lin(F.gelu(lin(ln(X, sh2, sc2), p + "fc1.w"), approximate="tanh"), p + "fc2.w")
    sh, scl = lin(sc, "ex.final.ada.w", "ex.final.ada.b")[0].reshape(2, de)
    return lin(ln(X, sh, scl), "ex.out.w", "ex.out.b").numpy()


def test_dit_velocity_vs_torch_assembly():
    cfg = dict(synth.micro_dit(), ex_layers=3)  # cross, self, cross
    P = synth.make_params(cfg, 0)
    de, nh = cfg["ex_dim"], cfg["ex_heads"]
    cross = {l: (rnd(9, nh, de // nh), rnd(9, nh, de // nh)) for l in (0, 2)}
    x, t = rnd(cfg["chunk_len"], cfg["action_dim"]), 0.5
    got = O.dit_velocity(P, cfg, cross, x, t)
    with torch.no_grad():
        ref = _dit_torch(P, cfg, cross, x, t)
    assert np.allclose(got, ref, rtol=1e-10, atol=1e-10)


def _zero_ada(P, cfg, bias_for=None):
    for l in range(cfg["ex_layers"]):
        P[f"ex.{l}.ada.w"] = np.zeros_like(P[f"ex.{l}.ada.w"])
        P[f"ex.{l}.ada.b"] = np.zeros_like(P[f"ex.{l}.ada.b"]) if bias_for is None else bias_for(l)
    P["ex.final.ada.w"] = np.zeros_like(P["ex.final.ada.w"])
    P["ex.final.ada.b"] = np.zeros_like(P["ex.final.ada.b"])


def test_dit_with_zero_gates_is_embedding_then_final_projection():
    """All adaLN outputs zero: every gated residual vanishes, so
    v = W_out LN(W_a x + b_a + pos) + b_out."""
    cfg = synth.micro_dit()
    P = synth.make_params(cfg, 0)
    _zero_ada(P, cfg)
    x = rnd(cfg["chunk_len"], cfg["action_dim"])
    cross = {0: (rnd(4, 2, 48), rnd(4, 2, 48))}
    X0 = x @ P["ex.in.w"].T.astype(np.float64) + P["ex.in.b"] + O.positions_sinusoid(x.shape[0], cfg["ex_dim"])
    mu = X0.mean(1, keepdims=True)
    xn = (X0 - mu) / np.sqrt(((X0 - mu) ** 2).mean(1, keepdims=True) + 1e-6)
    want = xn @ P["ex.out.w"].T.astype(np.float64) + P["ex.out.b"]
    assert np.allclose(O.dit_velocity(P, cfg, cross, x, 0.5), want, rtol=1e-12, atol=1e-12)


def test_dit_cross_attention_to_identical_features():
    """Identical feature rows make every cross-attention output the common V
    row (the softmax weights only mix equal rows); with gate1 = 1 and
    gate2 = 0 the layer adds exactly W_o (W_v f)."""
    cfg = dict(synth.micro_dit(), ex_layers=1)
    P = synth.make_params(cfg, 0)
    de = cfg["ex_dim"]
    _zero_ada(P, cfg, bias_for=lambda l: np.concatenate([np.zeros(2 * de), np.ones(de), np.zeros(3 * de)]))
    f = np.tile(rnd(1, cfg["lm_dim"]), (7, 1))
    cross = O.dit_cross_kv(P, cfg, f)
    x = rnd(cfg["chunk_len"], cfg["action_dim"])
    X0 = x @ P["ex.in.w"].T.astype(np.float64) + P["ex.in.b"] + O.positions_sinusoid(x.shape[0], de)
    vrow = f[0] @ P["ex.0.v.w"].T.astype(np.float64)
    X1 = X0 + vrow @ P["ex.0.o.w"].T.astype(np.float64)
    want = O.layer_norm(X1, np.ones(de), np.zeros(de)) @ P["ex.out.w"].T.astype(np.float64) + P["ex.out.b"]
    assert np.allclose(O.dit_velocity(P, cfg, cross, x, 0.25), want, rtol=1e-10, atol=1e-10)


def test_dit_zero_out_projection_gives_noise_minus_bias():
    cfg = synth.micro_dit()
    P = synth.make_params(cfg, 0)
    P["ex.out.w"] = np.zeros_like(P["ex.out.w"])
    fr = synth.make_frame(cfg, 0, 0)
    chunk = O.forward(P, cfg, fr)
    assert np.allclose(chunk, fr["noise"] - P["ex.out.b"], atol=1e-6)


def test_dit_phase1_hand_off():
    """Features are the final RMSNorm of the last LM layer (RMS just below 1
    before the gain); the hand-off holds the cross K/V of the even DiT layers only, and
    the shuffled ViT grid gives a quarter of the image tokens."""
    cfg = dict(synth.micro_dit(), ex_layers=4)
    P = synth.make_params(cfg, 0)
    fr = synth.make_frame(cfg, 0, 0)
    cap = {}
    out = O.vlm_prefill(P, cfg, fr, cap)
    d = synth.derived(cfg)
    assert cap["image_tokens"].shape == (d["n_img"], cfg["lm_dim"]) and d["n_img"] == 4
    f = cap["features"] / P["lm.final.g"]
    rms = np.sqrt((f ** 2).mean(1))  # m / (m + eps) with m the row's mean square
    assert np.all(rms <= 1.0) and np.all(rms > 0.99)
    assert sorted(out) == [0, 2]
    for l in (0, 2):
        assert out[l][0].shape == (d["prefix"], cfg["ex_heads"], cfg["ex_dim"] // cfg["ex_heads"])
    # the last LM layer now runs in full: the features differ from its input
    assert len(cap["kv"]) == cfg["lm_layers"]


def test_ddim_schedule_and_exact_recovery():
    """DDIM pins: the DDPM linear-beta abar (first value 1 - 1e-4, decreasing,
    abar_999 ~ 4.04e-5), the N = 10 timesteps 999, 899, ..., 99 and times
    s / 1000; and the defining property of deterministic DDIM: if the head
    returns the true noise eps of x_k = sqrt(abar_k) x0 + sqrt(1 - abar_k) eps,
    each step lands exactly on the next marginal, so N steps return x0."""
    ab = O.ddim_alpha_bar()
    assert ab[0] == 1 - 1e-4 and np.all(np.diff(ab) < 0)
    assert 4.0e-5 < ab[-1] < 4.1e-5
    ts, s, abar = O.ddim_schedule(10)
    assert s == [999 - 100 * k for k in range(10)]
    assert ts[0] == float(np.float32(0.999)) and ts[-1] == float(np.float32(0.099))
    assert abar[-1] == 1.0 and abar[0] == ab[999]
    rng = np.random.default_rng(3)
    x0, eps = rng.standard_normal((5, 3)), rng.standard_normal((5, 3))
    for n in (1, 4, 10):
        _, _, abar = O.ddim_schedule(n)
        xT = np.sqrt(abar[0]) * x0 + np.sqrt(1 - abar[0]) * eps
        got = O.ddim_integrate(xT, lambda x, t: eps, n)
        assert np.allclose(got, x0, rtol=0, atol=1e-9), n
    # one step from k = 0 lands on the k = 1 marginal
    _, _, abar = O.ddim_schedule(4)
    x1 = O.ddim_integrate(np.sqrt(abar[0]) * x0 + np.sqrt(1 - abar[0]) * eps, lambda x, t: eps, 1)
    # (a one-step run has abar_1 = 1: it returns x0; the four-step schedule's
    # second marginal follows from its own first step)
    assert np.allclose(x1, x0, atol=1e-9)
    seen = []
    O.ddim_integrate(np.sqrt(abar[0]) * x0 + np.sqrt(1 - abar[0]) * eps,
                     lambda x, t: (seen.append(x.copy()), eps)[1], 4)
    for k in range(4):
        assert np.allclose(seen[k], np.sqrt(abar[k]) * x0 + np.sqrt(1 - abar[k]) * eps, atol=1e-9), k


# ------------------------------------------- phase-1 hand-off of the DiT head

def test_lm_features_vs_gemma_stack():
    """The DiT's features: every LM layer runs in full (the last one's
    attention output and MLP included), then the final RMSNorm; assembled
    from transformers Gemma decoder layers (multi-head, 3 layers) and torch's
    RMSNorm, with every layer's K / V read back from the cache."""
    from transformers.cache_utils import DynamicCache
    cfg = dict(synth.micro_dit(), lm_layers=3)
    P = synth.make_params(cfg, 0)
    n, dl = 11, cfg["lm_dim"]
    x0 = rnd(n, dl)
    got, cache_o = O.lm_features(P, cfg, x0)
    pos = np.arange(n)
    with torch.no_grad():
        h = t64(x0)[None]
        cache = DynamicCache()
        for l in range(cfg["lm_layers"]):
            m = _gemma_layer(cfg, P, "lm", l, dl, cfg["lm_mlp"])
            h = m(h, attention_mask=None, position_ids=torch.arange(n)[None], past_key_values=cache,
                  use_cache=True, position_embeddings=_rope_tables(cfg["head_dim"], pos))
            h = h[0] if isinstance(h, tuple) else h
        ref = F.rms_norm(h[0], (dl,), t64(P["lm.final.g"]), eps=1e-6).numpy()
    # Gemma's RMSNorm runs in fp32, hence the tolerance
    assert np.allclose(got, ref, rtol=5e-5, atol=5e-5)
    assert len(cache_o) == cfg["lm_layers"]
    for l in range(cfg["lm_layers"]):
        assert np.allclose(cache_o[l][0], cache.layers[l].keys[0].transpose(0, 1).numpy(), rtol=5e-5, atol=5e-5)
        assert np.allclose(cache_o[l][1], cache.layers[l].values[0].transpose(0, 1).numpy(), rtol=5e-5, atol=5e-5)


def _dit_cross_torch(P, cfg, feats):
    """Cross K / V of the even DiT layers from the features with F.linear."""
    nh, hd = cfg["ex_heads"], cfg["ex_dim"] // cfg["ex_heads"]
    out = {}
    for l in range(0, cfg["ex_layers"], 2):
        k = F.linear(t64(feats), t64(P[f"ex.{l}.k.w"])).reshape(-1, nh, hd)
        v = F.linear(t64(feats), t64(P[f"ex.{l}.v.w"])).reshape(-1, nh, hd)
        out[l] = (k.numpy(), v.numpy())
    return out


def test_dit_cross_kv_vs_linear_and_velocity_from_features():
    """dit_cross_kv on distinct feature rows: K and V of every even layer
    against F.linear, and the DiT velocity fed with them against the torch
    assembly fed with K / V computed by torch from the same features (so a
    K projection that differs in any way changes the attention weights)."""
    cfg = dict(synth.micro_dit(), ex_layers=4)  # cross, self, cross, self
    P = synth.make_params(cfg, 0)
    feats = rnd(9, cfg["lm_dim"])
    got = O.dit_cross_kv(P, cfg, feats)
    want = _dit_cross_torch(P, cfg, feats)
    assert sorted(got) == [0, 2]
    for l in (0, 2):
        assert np.allclose(got[l][0], want[l][0], rtol=1e-12, atol=1e-12)
        assert np.allclose(got[l][1], want[l][1], rtol=1e-12, atol=1e-12)
    x, t = rnd(cfg["chunk_len"], cfg["action_dim"]), 0.75
    v_got = O.dit_velocity(P, cfg, got, x, t)
    with torch.no_grad():
        v_ref = _dit_torch(P, cfg, want, x, t)
    assert np.allclose(v_got, v_ref, rtol=1e-10, atol=1e-10)
    # the attention weights depend on K: a swapped projection moves the result
    swapped = {l: (want[l][1], want[l][0]) for l in want}
    with torch.no_grad():
        assert not np.allclose(_dit_torch(P, cfg, swapped, x, t), v_got, rtol=1e-6, atol=1e-6)


def test_image_tokens_with_pixel_shuffle_vs_torch_assembly():
    """Shuffled image tokens (the GR00T-shaped ViT): SigLIP layers, then the
    final LayerNorm on every fine token, then torch's space-to-depth
    (pixel_unshuffle, channels reordered to (dy, dx, c)), then the projector."""
    cfg = dict(synth.micro_dit(), vit_layers=2)
    P = synth.make_params(cfg, 0)
    fr = synth.make_frame(cfg, 0, 0)
    got = O.image_tokens(P, cfg, fr["pixels"])
    p, s = cfg["patch"], cfg["shuffle"]
    gh, gw = cfg["img_h"] // p, cfg["img_w"] // p
    ref = _image_tokens_torch(cfg, P, fr).numpy()
    assert s == 2 and got.shape == ((gh // s) * (gw // s), cfg["lm_dim"])
    # transformers computes the ViT softmax in fp32, hence 1e-7
    assert np.allclose(got, ref, rtol=1e-7, atol=1e-7)


def _image_tokens_torch(cfg, P, fr):
    """Image tokens of one view from library modules: patches by unfold,
    SigLIP layers, the final LayerNorm, space-to-depth by pixel_unshuffle
    (channels reordered to (dy, dx, c)) when the config shuffles, projector."""
    p, dv, s = cfg["patch"], cfg["vit_dim"], cfg.get("shuffle", 1)
    gh, gw = cfg["img_h"] // p, cfg["img_w"] // p
    with torch.no_grad():
        img = t64(fr["pixels"][0])
        patches = img.permute(2, 0, 1).unfold(1, p, p).unfold(2, p, p)
        patches = patches.permute(1, 2, 3, 4, 0).reshape(gh * gw, p * p * 3)
        x = F.linear(patches, t64(P["vit.patch.w"]), t64(P["vit.patch.b"])) + t64(P["vit.pos"])
        for l in range(cfg["vit_layers"]):
            y = _siglip_layer(cfg, P, l)(x[None], None)
            x = (y[0] if isinstance(y, tuple) else y)[0]
        x = F.layer_norm(x, (dv,), t64(P["vit.post.g"]), t64(P["vit.post.b"]), eps=1e-6)
        if s > 1:
            g = F.pixel_unshuffle(x.T.reshape(1, dv, gh, gw), s)[0]
            x = g.reshape(dv, s * s, gh // s, gw // s).permute(2, 3, 1, 0).reshape(-1, s * s * dv)
        return F.linear(x, t64(P["proj.w"]), t64(P["proj.b"]))


def _features_torch(cfg, P, fr):
    """Phase 1 of the feature heads from library modules: [image tokens; text
    embedding x sqrt(d); the state row if any; the learned cognition token for
    that head] through every LM layer as a transformers Gemma decoder layer,
    then torch's RMSNorm with the final gain."""
    from transformers.cache_utils import DynamicCache
    dl = cfg["lm_dim"]
    with torch.no_grad():
        rows = [_image_tokens_torch(cfg, P, fr)]
        emb = torch.nn.Embedding(cfg["vocab"], dl).double()
        emb.weight.data = t64(P["lm.embed"])
        rows.append(emb(torch.from_numpy(fr["ids"].astype(np.int64))) * math.sqrt(dl))
        if cfg["state_dim"] > 0:
            rows.append(F.linear(t64(fr["state"])[None], t64(P["state.w"]), t64(P["state.b"])))
        if cfg.get("head", 0) == 2:
            rows.append(t64(P["lm.cog"]))
        h = torch.cat(rows, 0)[None]
        n = h.shape[1]
        cache = DynamicCache()
        for l in range(cfg["lm_layers"]):
            m = _gemma_layer(cfg, P, "lm", l, dl, cfg["lm_mlp"])
            h = m(h, attention_mask=None, position_ids=torch.arange(n)[None], past_key_values=cache,
                  use_cache=True, position_embeddings=_rope_tables(cfg["head_dim"], np.arange(n)))
            h = h[0] if isinstance(h, tuple) else h
        return F.rms_norm(h[0], (dl,), t64(P["lm.final.g"]), eps=1e-6).numpy()


def _euler_reading(x0, velocity, N):
    """N Euler steps from t = 1: t_k = (N - k) / N and dt = -1 / N, each a
    single fp32 division (the flow-matching time reading)."""
    dt = float(np.float32(-1.0) / np.float32(N))
    x = np.asarray(x0, np.float64)
    for k in range(N):
        x = x + dt * velocity(x, float(np.float32(N - k) / np.float32(N)))
    return x


def _ddim_reading(x0, eps, N, T=1000):
    """Deterministic DDIM from its reading: the DDPM linear beta schedule
    (1e-4 .. 0.02 over T steps), timesteps s_k = floor((N - k) T / N) - 1 with
    the head's time input s_k / T as one fp32 division, and the update written
    as x <- a_k x + b_k eps with a_k = sqrt(abar_{k+1} / abar_k) and
    b_k = sqrt(1 - abar_{k+1}) - a_k sqrt(1 - abar_k), abar = 1 after the last
    step."""
    abar = np.cumprod(1.0 - np.linspace(1e-4, 0.02, T))
    s = [(N - k) * T // N - 1 for k in range(N)]
    ab = [abar[sk] for sk in s] + [1.0]
    x = np.asarray(x0, np.float64)
    for k in range(N):
        a = math.sqrt(ab[k + 1] / ab[k])
        b = math.sqrt(1.0 - ab[k + 1]) - a * math.sqrt(1.0 - ab[k])
        x = a * x + b * eps(x, float(np.float32(s[k]) / np.float32(T)))
    return x


def test_ddim_full_forward_vs_library_assembly():
    """The pi0-shaped model sampled with DDIM end to end: the library prefill
    and the library expert read as the noise estimate, the steps written in
    the a_k x + b_k eps form (the oracle takes the clean-estimate form; the two
    are equal algebraically). The chunk is ~1/sqrt(abar_0) times the noise, so
    the bound is relative to its magnitude."""
    cfg = dict(synth.micro(), vit_layers=2, lm_layers=2, ex_layers=2, sampler=1, n_steps=3)
    P = synth.make_params(cfg, 0)
    fr = synth.make_frame(cfg, 0, 0)
    got = O.forward(P, cfg, fr)
    kv = _prefill_torch(cfg, P, fr)
    want = _ddim_reading(fr["noise"], lambda x, t: _expert_torch(cfg, P, kv, x, t), cfg["n_steps"])
    scale = float(np.abs(want).max())
    assert scale > 10 * float(np.abs(fr["noise"]).max())  # the sampler scaled the state up
    assert float(np.abs(got - want).max()) <= DDIM_FWD_REL_TOL * scale


def test_dit_full_forward_vs_library_assembly():
    """The GR00T-shaped model end to end: library image tokens (2x2 shuffle),
    the Gemma feature stack, the cross K / V of the even DiT layers by
    F.linear, and the torch DiT integrated over N Euler steps; the oracle's
    chunk must match."""
    cfg = dict(synth.micro_dit(), vit_layers=2, lm_layers=2, ex_layers=4, n_steps=3)  # cross, self, cross, self
    P = synth.make_params(cfg, 0)
    fr = synth.make_frame(cfg, 0, 0)
    got = O.forward(P, cfg, fr)
    cross = _dit_cross_torch(P, cfg, _features_torch(cfg, P, fr))
    with torch.no_grad():
        want = _euler_reading(fr["noise"], lambda x, t: _dit_torch(P, cfg, cross, x, t), cfg["n_steps"])
    assert not np.allclose(want, fr["noise"], atol=1e-3)
    assert np.allclose(got, want, rtol=DIT_COG_FWD_TOL, atol=DIT_COG_FWD_TOL)


def test_cog_full_forward_vs_library_assembly():
    """The cognition-token head end to end (Euler sampler): the Gemma feature
    stack over the prefix ending in the learned token, the projection of its
    last row, and the torch head integrated over N Euler steps."""
    cfg = dict(synth.micro_cog(), vit_layers=2, lm_layers=2, sampler=0, n_steps=3)
    P = synth.make_params(cfg, 0)
    fr = synth.make_frame(cfg, 0, 0)
    got = O.forward(P, cfg, fr)
    feats = _features_torch(cfg, P, fr)
    with torch.no_grad():
        cog = F.linear(t64(feats[-1:]), t64(P["cog.w"]), t64(P["cog.b"]))[0].numpy()
        want = _euler_reading(fr["noise"], lambda x, t: _cog_torch(P, cfg, cog, x, t), cfg["n_steps"])
    assert not np.allclose(want, fr["noise"], atol=1e-3)
    assert np.allclose(got, want, rtol=DIT_COG_FWD_TOL, atol=DIT_COG_FWD_TOL)


# the oracle and the assemblies agree to 2e-12 (DiT) and 2e-10 (cognition
# head); shifted times, features without the final norm, another layer's
# cross K / V, the cognition hand-off from the first row or without its bias
# move the chunk by 3.7e-6 or more
DIT_COG_FWD_TOL = 1e-8
DDIM_FWD_REL_TOL = 1e-6


# ------------------------------------------------ cognition-token (CogACT) head

def _cog_torch(P, cfg, cog, x, t):
    """The cognition-token head assembled from torch modules: pre-LN
    nn.TransformerEncoderLayer (tanh-GELU, eps 1e-6, linear biases zero, the
    LayerNorms' own biases loaded), the time token from F.silu and F.linear,
    F.layer_norm and F.linear on the action rows."""
    de, nh, mlp, H = cfg["ex_dim"], cfg["ex_heads"], cfg["ex_mlp"], x.shape[0]
    lin = lambda z, w, b=None: F.linear(z, t64(P[w]), None if b is None else t64(P[b]))
    half = de // 2
    ang = torch.arange(H, dtype=torch.float64)[:, None] * 10000.0 ** (-torch.arange(half, dtype=torch.float64) / half)
    act = lin(t64(x), "ex.in.w", "ex.in.b") + torch.cat([ang.sin(), ang.cos()], 1)
    phi = t64(O.sinusoid(t, 256))[None]
    tt = lin(F.silu(lin(phi, "ex.time1.w", "ex.time1.b")), "ex.time2.w", "ex.time2.b")
    X = torch.cat([act, t64(cog)[None], tt], 0)[None]
    for l in range(cfg["ex_layers"]):
        p = f"ex.{l}."
        layer = torch.nn.TransformerEncoderLayer(de, nh, dim_feedforward=mlp, dropout=0.0,
                                                 activation=lambda z: F.gelu(z, approximate="tanh"),
                                                 layer_norm_eps=1e-6, batch_first=True, norm_first=True)
        layer = layer.double().eval()
        sd = layer.state_dict()
        sd["self_attn.in_proj_weight"] = torch.cat([t64(P[p + "q.w"]), t64(P[p + "k.w"]), t64(P[p + "v.w"])], 0)
        sd["self_attn.in_proj_bias"] = torch.zeros(3 * de, dtype=torch.float64)
        sd["self_attn.out_proj.weight"] = t64(P[p + "o.w"])
        sd["self_attn.out_proj.bias"] = torch.zeros(de, dtype=torch.float64)
        sd["linear1.weight"], sd["linear1.bias"] = t64(P[p + "fc1.w"]), torch.zeros(mlp, dtype=torch.float64)
        sd["linear2.weight"], sd["linear2.bias"] = t64(P[p + "fc2.w"]), torch.zeros(de, dtype=torch.float64)
        sd["norm1.weight"], sd["norm1.bias"] = t64(P[p + "ln1.g"]), t64(P[p + "ln1.b"])
        sd["norm2.weight"], sd["norm2.bias"] = t64(P[p + "ln2.g"]), t64(P[p + "ln2.b"])
        layer.load_state_dict(sd)
        X = layer(X)
    h = F.layer_norm(X[0, :H], (de,), t64(P["ex.final.g"]), t64(P["ex.final.b"]), eps=1e-6)
    return lin(h, "ex.out.w", "ex.out.b").numpy()


def test_cog_velocity_vs_torch_encoder_layers():
    cfg = dict(synth.micro_cog(), ex_layers=3)
    P = synth.make_params(cfg, 0)
    cog, x, t = rnd(cfg["ex_dim"]), rnd(cfg["chunk_len"], cfg["action_dim"]), 0.37
    got = O.cog_velocity(P, cfg, cog, x, t)
    with torch.no_grad():
        ref = _cog_torch(P, cfg, cog, x, t)
    assert np.allclose(got, ref, rtol=1e-10, atol=1e-10)
    # the conditioning rows matter: another cognition vector moves the output
    # (a constant shift would not: every LayerNorm removes it)
    assert not np.allclose(O.cog_velocity(P, cfg, cog + rnd(cfg["ex_dim"]), x, t), got, atol=1e-6)


def test_cog_hand_off_is_the_cognition_rows_projection():
    """Phase 1 of the cognition-token head: the prefix ends with the learned
    token (unscaled); the hand-off is W_c (final RMSNorm of a Gemma decoder
    stack's output at that last row) + b_c."""
    from transformers.cache_utils import DynamicCache
    cfg = dict(synth.micro_cog(), lm_layers=2)
    P = synth.make_params(cfg, 0)
    fr = synth.make_frame(cfg, 0, 0)
    cap = {}
    got = O.vlm_prefill(P, cfg, fr, cap)
    x0 = cap["prefix"]
    d = synth.derived(cfg)
    assert x0.shape[0] == d["prefix"] and np.array_equal(x0[-1], P["lm.cog"][0].astype(np.float64))
    n, dl = x0.shape[0], cfg["lm_dim"]
    with torch.no_grad():
        h = t64(x0)[None]
        cache = DynamicCache()
        for l in range(cfg["lm_layers"]):
            m = _gemma_layer(cfg, P, "lm", l, dl, cfg["lm_mlp"])
            h = m(h, attention_mask=None, position_ids=torch.arange(n)[None], past_key_values=cache,
                  use_cache=True, position_embeddings=_rope_tables(cfg["head_dim"], np.arange(n)))
            h = h[0] if isinstance(h, tuple) else h
        f = F.rms_norm(h[0, -1:], (dl,), t64(P["lm.final.g"]), eps=1e-6)
        ref = F.linear(f, t64(P["cog.w"]), t64(P["cog.b"]))[0].numpy()
    assert got.shape == (cfg["ex_dim"],)
    assert np.allclose(got, ref, rtol=5e-5, atol=5e-5)


def test_cog_zero_out_projection_recovers_x0_with_ddim():
    """With W_out = 0 the head's noise estimate is the constant b_out; DDIM
    started from x_T = sqrt(abar_0) x0 + sqrt(1 - abar_0) b_out lands exactly
    on x0 (deterministic DDIM recovers x0 when the estimate is the true
    noise), whatever the rest of the model computes."""
    cfg = synth.micro_cog()
    P = synth.make_params(cfg, 0)
    P["ex.out.w"] = np.zeros_like(P["ex.out.w"])
    fr = synth.make_frame(cfg, 0, 0)
    x0 = rnd(cfg["chunk_len"], cfg["action_dim"])
    _, _, abar = O.ddim_schedule(cfg["n_steps"])
    noise = np.sqrt(abar[0]) * x0 + np.sqrt(1 - abar[0]) * P["ex.out.b"].astype(np.float64)
    chunk = O.forward(P, cfg, dict(fr, noise=noise))
    assert np.allclose(chunk, x0, rtol=0, atol=1e-8)
