"""Host-side checks of the C ABI (no GPU compute): the library loads, exports
every entry point include/vla.h declares, validates configurations and
generates parameters bit-identically to the seeded generator."""
import ctypes
import os
import re

import numpy as np
import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _header_functions():
    src = open(os.path.join(ROOT, "include", "vla.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(vla_\w+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    import paper_2609_22335_amd as V
    lib = ctypes.CDLL(V.LIB_PATH)
    names = _header_functions()
    assert len(names) >= 17
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(V.exported_symbols())


def test_presets_match_shapes():
    import paper_2609_22335_amd as V
    assert V.vla_preset("tiny") == synth.TINY
    assert V.vla_preset("pi0") == synth.PI0
    assert V.vla_preset("pi0_3view") == synth.PI0_3VIEW
    assert V.vla_preset("gr00t") == synth.GR00T
    assert V.vla_preset("tiny_dit") == synth.TINY_DIT
    assert V.vla_preset("cogact") == synth.COGACT
    assert V.vla_preset("tiny_cog") == synth.TINY_COG
    assert V.vla_preset("pi0_ddim") == synth.PI0_DDIM
    assert V.vla_preset("tiny_ddim") == synth.TINY_DDIM
    with pytest.raises(V.VlaError) as e:
        V.vla_preset("nope")
    assert e.value.code == -1


@pytest.mark.parametrize("field,value,msg", [
    ("lm_kv_heads", 3, "lm_heads % lm_kv_heads"),
    ("ex_layers", 3, "ex_layers must equal lm_layers"),
    ("patch", 15, "patch must divide"),
    ("head_dim", 48, "head_dim"),
    ("lm_mlp", 1000, "multiples of 16"),
    ("dtype", 7, "dtype"),
    ("chunk_len", 0, "positive"),
])
def test_validate_rejects(field, value, msg):
    import paper_2609_22335_amd as V
    cfg = dict(synth.TINY, **{field: value})
    with pytest.raises(V.VlaError) as e:
        V.vla_validate(cfg)
    assert e.value.code == -1 and msg in str(e.value)
    V.vla_validate(synth.TINY)
    V.vla_validate(synth.PI0)
    V.vla_validate(synth.micro())
    V.vla_validate(synth.micro_cog())
    V.vla_validate(synth.COGACT)
    with pytest.raises(V.VlaError):
        V.vla_validate(dict(synth.micro_cog(), chunk_len=63))


@pytest.mark.parametrize("seed,name,mean", [(0, "lm.3.q.w", 0.0), (7, "vit.0.ln1.g", 1.0),
                                            (12345, "ex.out.b", 0.0)])
def test_library_generator_matches_seeded_generator(seed, name, mean):
    import paper_2609_22335_amd as V
    n = 1_500_000 if mean == 0.0 and seed == 0 else 5000
    a = V.vla_debug_generate(seed, name, n, mean, 0.02)
    b = synth.normal(seed, name, n, 0.02, mean)
    assert np.array_equal(a, b)


def test_null_arguments_are_errors_not_crashes():
    import paper_2609_22335_amd as V
    lib = V._lib
    assert lib.vla_create(None, 0, None) == -1
    assert lib.vla_destroy(None) == 0
    assert lib.vla_ctx_destroy(None) == 0
    assert lib.vla_vlm_prefill(None, None, None, None) == -1
    assert lib.vla_pipeline_run(None, None, None, 1, None, None, None) == -1
    assert "NULL" in V.vla_last_error() or "model" in V.vla_last_error()
    assert lib.vla_debug_gemm(0, 4, 4, 7, None, 8, None, 8, None, None, None) == -1


@pytest.mark.parametrize("struct", ["vla_config", "vla_frame", "vla_sched", "vla_timing", "vla_debug_epi"])
def test_binding_structs_match_header(struct):
    """The ctypes structures pass the header's fields in the header's order
    and types (a field added on one side only would shift every later one)."""
    import ctypes as C
    import paper_2609_22335_amd as V
    src = open(os.path.join(ROOT, "include", "vla.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    body = re.search(r"typedef struct " + struct + r"\s*\{(.*?)\}\s*" + struct + ";", src, flags=re.S).group(1)
    fields = []
    for t, names in re.findall(r"^\s*((?:const\s+)?\w+\s*\*?)\s*([\w\s,]+);", body, flags=re.M):
        fields += [(t.strip(), n.strip()) for n in names.split(",")]
    ctype = {"int32_t": C.c_int32, "double": C.c_double, "float": C.c_float}
    got = getattr(V, struct)._fields_
    assert [n for _, n in fields] == [n for n, _ in got], struct
    for (t, n), (gn, gt) in zip(fields, got):
        t = t.replace("const", "").strip()
        if t.endswith("*"):
            assert gt in (C.c_void_p,), (struct, n, gt)
        else:
            assert gt is ctype[t], (struct, n, t, gt)
