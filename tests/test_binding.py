"""CPU checks of the Python binding's argument checks: undersized, host,
wrongly typed or strided buffers and short frame lists are refused before
the library is called (the C entry points take raw pointers and cannot check
lengths)."""
import types

import pytest
import torch

import synth


class FakeDev:
    """Stands in for a device tensor (no GPU here): the attributes the
    binding's checks read."""

    def __init__(self, numel, dtype=torch.float32, is_cuda=True, contiguous=True):
        self._n, self.dtype, self.is_cuda, self._c = numel, dtype, is_cuda, contiguous

    def data_ptr(self):
        return 0x1000

    def numel(self):
        return self._n

    def is_contiguous(self):
        return self._c


@pytest.fixture
def V(monkeypatch):
    import paper_2609_22335_amd as V
    cfg = dict(synth.micro())
    monkeypatch.setattr(V, "vla_model_config", lambda m: cfg)

    def never(*a, **k):
        raise AssertionError("the library was called despite a bad argument")
    monkeypatch.setattr(V, "_lib", types.SimpleNamespace(vla_pipeline_run=never, vla_action_denoise=never,
                                                         vla_vlm_prefill=never, vla_last_error=lambda: b""))
    V.cfg = cfg
    return V


def _frame(V, cfg, **bad):
    n = cfg["n_views"] * cfg["img_h"] * cfg["img_w"] * 3
    pix = bad.get("pixels", FakeDev(n))
    ids = bad.get("ids", FakeDev(cfg["n_text"], torch.int32))
    st = bad.get("state", FakeDev(cfg["state_dim"]))
    return V.make_frame(pix, ids, st)


def test_pipeline_run_refuses_before_any_call(V):
    cfg = V.cfg
    R, k = 3, 2
    n = R * k * cfg["chunk_len"] * cfg["action_dim"]
    good = [_frame(V, cfg) for _ in range(R)]
    cases = [
        (good[:2], FakeDev(n), FakeDev(n), {}, "frames given"),
        (good, FakeDev(n - 1), FakeDev(n), {}, "noise holds"),
        (good, FakeDev(n), FakeDev(n // 2), {}, "actions holds"),
        (good, FakeDev(n, torch.float16), FakeDev(n), {}, "float32"),
        (good, FakeDev(n), FakeDev(n, is_cuda=False), {}, "device"),
        (good, FakeDev(n), FakeDev(n, contiguous=False), {}, "contiguous"),
        (good[:2] + [_frame(V, cfg, pixels=FakeDev(10))], FakeDev(n), FakeDev(n), {}, "frame 2 pixels"),
        (good[:2] + [_frame(V, cfg, ids=FakeDev(cfg["n_text"], torch.int64))], FakeDev(n), FakeDev(n), {},
         "text_ids"),
        (good, FakeDev(n), None, {}, "actions is None"),
    ]
    for frames, noise, actions, kw, msg in cases:
        with pytest.raises(V.VlaError) as e:
            V.vla_pipeline_run(1, frames, noise, R, mode="concurrent", actions=actions, act_chunks=k, **kw)
        assert e.value.code == -1 and msg in str(e.value), (msg, str(e.value))
    # one chunk per frame needs only R chunks: the same buffers pass the checks
    # and reach the (stubbed) library
    with pytest.raises(AssertionError, match="library was called"):
        V.vla_pipeline_run(1, good, FakeDev(n), R, actions=FakeDev(n))


def test_action_denoise_and_prefill_refuse_before_any_call(V):
    cfg = V.cfg
    n = cfg["chunk_len"] * cfg["action_dim"]
    for noise, out, msg in [(FakeDev(n - 1), FakeDev(n), "noise"), (FakeDev(n), FakeDev(n, torch.bfloat16), "actions"),
                            (FakeDev(n, is_cuda=False), FakeDev(n), "device")]:
        with pytest.raises(V.VlaError) as e:
            V.vla_action_denoise(1, 2, noise, out)
        assert msg in str(e.value)
    with pytest.raises(V.VlaError) as e:
        V.vla_vlm_prefill(1, _frame(V, cfg, state=FakeDev(cfg["state_dim"] - 1)), 2)
    assert "state" in str(e.value)
    with pytest.raises(AssertionError, match="library was called"):
        V.vla_action_denoise(1, 2, FakeDev(n), FakeDev(n))
