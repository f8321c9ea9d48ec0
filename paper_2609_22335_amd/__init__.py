"""Python binding of libvla.so, the MI355X two-phase VLA inference library.

Argument marshalling only: every function forwards to the C entry point of
the same name (see include/vla.h); every step of the computation runs in the
library's HIP kernels. Device buffers are passed as integer device pointers
(e.g. ``torch.Tensor.data_ptr()``) and streams as integer ``hipStream_t``
handles (``torch.cuda.current_stream().cuda_stream``).

Importing this module loads the library and raises if it is not built:
there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Iterable, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# the in-tree build; VLA_LIBRARY names another build of the same library
# (a tuning variant, say) to load instead
LIB_PATH = os.environ.get("VLA_LIBRARY") or os.path.join(_HERE, "libvla.so")

VLA_F32, VLA_BF16 = 0, 1
MODE_SERIAL, MODE_CONCURRENT, MODE_CU_MASKED, MODE_WG_CAPPED = 0, 1, 2, 3
MODES = {"serial": MODE_SERIAL, "concurrent": MODE_CONCURRENT, "cu_masked": MODE_CU_MASKED,
         "wg_capped": MODE_WG_CAPPED}

CONFIG_FIELDS = (
    "dtype", "n_views", "img_h", "img_w", "patch",
    "vit_dim", "vit_heads", "vit_mlp", "vit_layers",
    "lm_dim", "lm_heads", "lm_kv_heads", "head_dim", "lm_mlp", "lm_layers",
    "vocab", "n_text", "state_dim",
    "ex_dim", "ex_mlp", "ex_layers", "chunk_len", "action_dim", "n_steps",
    "head", "shuffle", "ex_heads", "sampler",
)
HEAD_PI0, HEAD_DIT, HEAD_COG = 0, 1, 2
SAMPLER_EULER, SAMPLER_DDIM = 0, 1


class vla_config(ctypes.Structure):
    _fields_ = [(f, ctypes.c_int32) for f in CONFIG_FIELDS]


class vla_frame(ctypes.Structure):
    _fields_ = [("pixels", ctypes.c_void_p), ("text_ids", ctypes.c_void_p), ("state", ctypes.c_void_p)]


class vla_sched(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int32), ("vlm_cus", ctypes.c_int32), ("act_cus", ctypes.c_int32),
                ("vlm_wg_cap", ctypes.c_int32), ("act_streams", ctypes.c_int32), ("graphs", ctypes.c_int32),
                ("vlm_streams", ctypes.c_int32), ("act_batch", ctypes.c_int32),
                ("vlm_batch", ctypes.c_int32), ("act_chunks", ctypes.c_int32)]


class vla_timing(ctypes.Structure):
    _fields_ = [("wall_ms", ctypes.c_double), ("frames_per_s", ctypes.c_double),
                ("actions_per_s", ctypes.c_double), ("vlm_ms", ctypes.c_double),
                ("act_ms", ctypes.c_double)]


class vla_debug_epi(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("skinny", ctypes.c_int32), ("bias", ctypes.c_void_p),
                ("out", ctypes.c_void_p), ("nq", ctypes.c_int32), ("nkv", ctypes.c_int32),
                ("hd", ctypes.c_int32), ("pos0", ctypes.c_int32), ("q_out", ctypes.c_void_p),
                ("k_out", ctypes.c_void_p), ("v_out", ctypes.c_void_p), ("x", ctypes.c_void_p),
                ("xs", ctypes.c_float), ("dt", ctypes.c_float), ("resid", ctypes.c_void_p),
                ("gain", ctypes.c_void_p), ("plan_out", ctypes.c_void_p)]


DEBUG_EPI = {"bias": 0, "t": 1, "gelu": 2, "swish": 3, "geglu": 4, "qkv_rope": 5, "qkv_plain": 6, "step": 7,
             "resid_norm": 8}


class VlaError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"vla status {code}: {msg}")
        self.code = code


def _share_hip_runtime_with_torch():
    # PyTorch ships its own copy of the HIP runtime under the same soname as
    # the ROCm one the library links. One copy serves both only when torch
    # loads first (libvla's dependency then resolves to it by soname);
    # loading libvla first would bring in a second runtime and leave torch
    # without a device. So torch, when present, is imported first.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass


def _load():
    _share_hip_runtime_with_torch()
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python paper_2609_22335_amd/build.py`")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, U64, D = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_double
    sig = {
        "vla_preset": [ctypes.c_char_p, ctypes.POINTER(vla_config)],
        "vla_validate": [ctypes.POINTER(vla_config)],
        "vla_model_config": [P, ctypes.POINTER(vla_config)],
        "vla_create": [ctypes.POINTER(vla_config), U64, ctypes.POINTER(P)],
        "vla_destroy": [P],
        "vla_ctx_create": [P, ctypes.POINTER(P)],
        "vla_ctx_destroy": [P],
        "vla_vlm_prefill": [P, ctypes.POINTER(vla_frame), P, P],
        "vla_action_denoise": [P, P, P, P, P],
        "vla_pipeline_run": [P, ctypes.POINTER(vla_frame), P, I32, ctypes.POINTER(vla_sched), P,
                             ctypes.POINTER(vla_timing)],
        "vla_param_count": [P, ctypes.POINTER(I32)],
        "vla_param_info": [P, I32, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(I64)],
        "vla_export_param": [P, ctypes.c_char_p, P, I64],
        "vla_ctx_export_kv": [P, P, I32, P, P],
        "vla_ctx_export_cross": [P, P, I32, P, P],
        "vla_ctx_export_cog": [P, P, P],
        "vla_wavelog_enable": [P, I64],
        "vla_wavelog_read": [P, P, I64, ctypes.POINTER(I64)],
        "vla_debug_gemm": [I32, I32, I32, I32, P, I32, P, I32, P, P, P],
        "vla_gemm_noalloc": [I32, I32, I32, I32, P, I32, P, I32, P, P, P],
        "vla_debug_gemm_epi": [I32, I32, I32, I32, P, P, ctypes.POINTER(vla_debug_epi), P],
        "vla_debug_attention": [I32, I32, I32, I32, I32, P, P, P, I32, P, P, I32, P, P],
        "vla_debug_generate": [U64, ctypes.c_char_p, I64, D, D, P],
        "vla_debug_gemm_plan": [I32, I32, I32, I32, I32, I32, I32, I32, P, ctypes.POINTER(I64)],
        "vla_debug_attention_cache": [I32, I32, I32, I32, I32, P, P, P, I32, P, P, I32, P, P],
        "vla_debug_norm": [I32, I32, I32, P, I32, P, I32, P, P, P, I32, P, I32, P, I32, P],
        "vla_kernel_timer": [P, ctypes.c_char_p],
        "vla_kernel_timer_read": [P, ctypes.POINTER(D), ctypes.POINTER(I64)],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    lib.vla_last_error.argtypes = []
    lib.vla_last_error.restype = ctypes.c_char_p
    return lib


_lib = _load()


def vla_last_error() -> str:
    return _lib.vla_last_error().decode()


def _check(rc: int) -> None:
    if rc != 0:
        raise VlaError(rc, vla_last_error())


def _cfg(cfg: Dict[str, int]) -> vla_config:
    return vla_config(*[int(cfg[f]) for f in CONFIG_FIELDS])


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    return int(x)


def vla_preset(name: str) -> Dict[str, int]:
    c = vla_config()
    _check(_lib.vla_preset(name.encode(), ctypes.byref(c)))
    return {f: int(getattr(c, f)) for f in CONFIG_FIELDS}


def vla_validate(cfg: Dict[str, int]) -> None:
    _check(_lib.vla_validate(ctypes.byref(_cfg(cfg))))


def vla_create(cfg: Dict[str, int], seed: int) -> int:
    out = ctypes.c_void_p()
    _check(_lib.vla_create(ctypes.byref(_cfg(cfg)), ctypes.c_uint64(seed), ctypes.byref(out)))
    return out.value


def vla_destroy(model: Optional[int]) -> None:
    _check(_lib.vla_destroy(model))


def vla_ctx_create(model: int) -> int:
    out = ctypes.c_void_p()
    _check(_lib.vla_ctx_create(model, ctypes.byref(out)))
    return out.value


def vla_ctx_destroy(ctx: Optional[int]) -> None:
    _check(_lib.vla_ctx_destroy(ctx))


def vla_model_config(model: int) -> Dict[str, int]:
    c = vla_config()
    _check(_lib.vla_model_config(model, ctypes.byref(c)))
    return {f: int(getattr(c, f)) for f in CONFIG_FIELDS}


def _einval(msg: str) -> VlaError:
    return VlaError(-1, msg)


def _check_buffer(x, what: str, numel: int, dtype: str) -> None:
    """A tensor handed to the library as a device buffer: on the GPU,
    contiguous, of the element type the entry point reads, and at least
    `numel` elements long. Raises before anything is launched. Integer
    pointers cannot be checked and are passed as given."""
    if x is None:
        raise _einval(f"{what} is None")
    if not hasattr(x, "data_ptr"):
        return
    if not getattr(x, "is_cuda", False):
        raise _einval(f"{what} must be a device (cuda) tensor")
    if str(x.dtype) != f"torch.{dtype}":
        raise _einval(f"{what} must be {dtype}, got {x.dtype}")
    if not x.is_contiguous():
        raise _einval(f"{what} must be contiguous")
    if x.numel() < numel:
        raise _einval(f"{what} holds {x.numel()} elements, needs at least {numel}")


def _check_frame(cfg: Dict[str, int], fr: vla_frame, i: int) -> None:
    src = getattr(fr, "_src", None)
    if src is None:
        return
    pixels, ids, state = src
    _check_buffer(pixels, f"frame {i} pixels", cfg["n_views"] * cfg["img_h"] * cfg["img_w"] * 3, "float32")
    if cfg["n_text"] > 0:
        _check_buffer(ids, f"frame {i} text_ids", cfg["n_text"], "int32")
    if cfg["state_dim"] > 0:
        _check_buffer(state, f"frame {i} state", cfg["state_dim"], "float32")


def make_frame(pixels, text_ids, state=None) -> vla_frame:
    """A vla_frame from device buffers (tensors or integer pointers); the
    tensors are kept with it so the calls below can check them."""
    f = vla_frame(_ptr(pixels), _ptr(text_ids), _ptr(state))
    f._src = (pixels, text_ids, state)
    return f


def vla_vlm_prefill(model: int, frame: vla_frame, ctx: int, stream: int = 0) -> None:
    if model:
        _check_frame(vla_model_config(model), frame, 0)
    _check(_lib.vla_vlm_prefill(model, ctypes.byref(frame), ctx, stream or None))


def vla_action_denoise(model: int, ctx: int, noise, actions, stream: int = 0) -> None:
    if model:
        cfg = vla_model_config(model)
        n = cfg["chunk_len"] * cfg["action_dim"]
        _check_buffer(noise, "noise", n, "float32")
        _check_buffer(actions, "actions", n, "float32")
    _check(_lib.vla_action_denoise(model, ctx, _ptr(noise), _ptr(actions), stream or None))


def vla_pipeline_run(model: int, frames: Sequence[vla_frame], noise, R: int, mode="serial",
                     vlm_cus: int = 0, act_cus: int = 0, vlm_wg_cap: int = 0, actions=None,
                     act_streams: int = 1, graphs: bool = False, vlm_streams: int = 1,
                     act_batch: int = 1, vlm_batch: int = 1, act_chunks: int = 1) -> Dict[str, float]:
    if model and int(R) >= 1:
        # the library reads frames[0 .. R-1] and R * k chunks of noise and
        # actions (k = act_chunks): check them all before anything runs
        if len(frames) < int(R):
            raise _einval(f"{len(frames)} frames given for R = {R}")
        cfg = vla_model_config(model)
        n = int(R) * max(1, int(act_chunks)) * cfg["chunk_len"] * cfg["action_dim"]
        _check_buffer(noise, "noise", n, "float32")
        _check_buffer(actions, "actions", n, "float32")
        for i in range(int(R)):
            _check_frame(cfg, frames[i], i)
    arr = (vla_frame * len(frames))(*frames)
    s = vla_sched(MODES[mode] if isinstance(mode, str) else int(mode), vlm_cus, act_cus, vlm_wg_cap,
                  act_streams, 1 if graphs else 0, vlm_streams, act_batch, vlm_batch, act_chunks)
    t = vla_timing()
    _check(_lib.vla_pipeline_run(model, arr, _ptr(noise), int(R), ctypes.byref(s), _ptr(actions),
                                 ctypes.byref(t)))
    return {k: getattr(t, k) for k, _ in vla_timing._fields_}


def vla_param_count(model: int) -> int:
    n = ctypes.c_int32()
    _check(_lib.vla_param_count(model, ctypes.byref(n)))
    return n.value


def vla_param_info(model: int, i: int) -> Tuple[str, int]:
    name = ctypes.c_char_p()
    numel = ctypes.c_int64()
    _check(_lib.vla_param_info(model, i, ctypes.byref(name), ctypes.byref(numel)))
    return name.value.decode(), numel.value


def vla_export_param(model: int, name: str, numel: int) -> np.ndarray:
    out = np.empty(numel, dtype=np.float32)
    _check(_lib.vla_export_param(model, name.encode(), out.ctypes.data, numel))
    return out


def vla_ctx_export_kv(model: int, ctx: int, layer: int, n: int) -> Tuple[np.ndarray, np.ndarray]:
    k = np.empty(n, dtype=np.float32)
    v = np.empty(n, dtype=np.float32)
    _check(_lib.vla_ctx_export_kv(model, ctx, layer, k.ctypes.data, v.ctypes.data))
    return k, v


def vla_ctx_export_cross(model: int, ctx: int, layer: int, n: int) -> Tuple[np.ndarray, np.ndarray]:
    k = np.empty(n, dtype=np.float32)
    v = np.empty(n, dtype=np.float32)
    _check(_lib.vla_ctx_export_cross(model, ctx, layer, k.ctypes.data, v.ctypes.data))
    return k, v


def vla_ctx_export_cog(model: int, ctx: int, n: int) -> np.ndarray:
    c = np.empty(n, dtype=np.float32)
    _check(_lib.vla_ctx_export_cog(model, ctx, c.ctypes.data))
    return c


WAVE_REC = np.dtype([("t", "<u8"), ("hwid", "<u4"), ("xcc", "<u4"), ("kind", "<u4"), ("end", "<u4")])


def vla_wavelog_enable(model: int, capacity: int) -> None:
    _check(_lib.vla_wavelog_enable(model, int(capacity)))


def vla_wavelog_read(model: int, max_records: int) -> Tuple[np.ndarray, int]:
    buf = np.empty(int(max_records), dtype=WAVE_REC)
    n = ctypes.c_int64()
    _check(_lib.vla_wavelog_read(model, buf.ctypes.data if max_records else None, int(max_records),
                                 ctypes.byref(n)))
    return buf[:min(n.value, max_records)], n.value


def vla_debug_gemm(dtype: int, M: int, N: int, K: int, A, lda: int, W, ldw: int, bias, C,
                   stream: int = 0) -> None:
    _check(_lib.vla_debug_gemm(dtype, M, N, K, _ptr(A), lda, _ptr(W), ldw, _ptr(bias), _ptr(C),
                               stream or None))


def vla_debug_gemm_epi(dtype: int, M: int, N: int, K: int, A, W, kind: str, skinny: bool = False, bias=None,
                       out=None, nq: int = 0, nkv: int = 0, hd: int = 0, pos0: int = 0, q_out=None, k_out=None,
                       v_out=None, x=None, xs: float = 1.0, dt: float = 0.0, resid=None, gain=None,
                       stream: int = 0) -> Tuple[int, int]:
    """Returns (tile rows, tile columns, split-K factor) of the launch; the
    skinny kernel reports 0 rows."""
    plan = (ctypes.c_int32 * 3)()
    e = vla_debug_epi(DEBUG_EPI[kind], 1 if skinny else 0, _ptr(bias), _ptr(out), nq, nkv, hd, pos0, _ptr(q_out),
                      _ptr(k_out), _ptr(v_out), _ptr(x), xs, dt, _ptr(resid), _ptr(gain),
                      ctypes.cast(plan, ctypes.c_void_p))
    _check(_lib.vla_debug_gemm_epi(dtype, M, N, K, _ptr(A), _ptr(W), ctypes.byref(e), stream or None))
    return int(plan[0]), int(plan[1]), int(plan[2])


def vla_gemm_noalloc(dtype: int, M: int, N: int, K: int, A, lda: int, W, ldw: int, bias, C,
                     stream: int = 0) -> None:
    _check(_lib.vla_gemm_noalloc(dtype, M, N, K, _ptr(A), lda, _ptr(W), ldw, _ptr(bias), _ptr(C),
                                 stream or None))


def vla_debug_attention(dtype: int, Sq: int, nq: int, nkv: int, hd: int, q, k0, v0, S0: int,
                        k1, v1, S1: int, out, stream: int = 0) -> None:
    _check(_lib.vla_debug_attention(dtype, Sq, nq, nkv, hd, _ptr(q), _ptr(k0), _ptr(v0), S0,
                                    _ptr(k1), _ptr(v1), S1, _ptr(out), stream or None))


def vla_debug_attention_cache(dtype: int, Sq: int, nq: int, nkv: int, hd: int, q, k0, v0, S0: int,
                              k1, v1, S1: int, out, stream: int = 0) -> None:
    _check(_lib.vla_debug_attention_cache(dtype, Sq, nq, nkv, hd, _ptr(q), _ptr(k0), _ptr(v0), S0,
                                          _ptr(k1), _ptr(v1), S1, _ptr(out), stream or None))


def vla_debug_norm(dtype: int, rows: int, d: int, x, ldx: int, part, splits: int, bias, colscale, gain,
                   gain_plus_one: int, shift, rms: int, out, ldo: int, stream: int = 0) -> None:
    _check(_lib.vla_debug_norm(dtype, rows, d, _ptr(x), ldx, _ptr(part), splits, _ptr(bias), _ptr(colscale),
                               _ptr(gain), gain_plus_one, _ptr(shift), rms, _ptr(out), ldo, stream or None))


def vla_kernel_timer(model: int, tag: Optional[str]) -> None:
    _check(_lib.vla_kernel_timer(model, tag.encode() if tag else None))


def vla_kernel_timer_read(model: int) -> Tuple[float, int]:
    ms = ctypes.c_double()
    n = ctypes.c_int64()
    _check(_lib.vla_kernel_timer_read(model, ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


def vla_debug_generate(seed: int, name: str, n: int, mean: float, std: float) -> np.ndarray:
    out = np.empty(n, dtype=np.float32)
    _check(_lib.vla_debug_generate(ctypes.c_uint64(seed), name.encode(), n, mean, std, out.ctypes.data))
    return out


def vla_debug_gemm_plan(dtype: int, M: int, N: int, K: int, kind: int, skinny: bool = False, plan_m: int = 0,
                        plan_batch: int = 1) -> dict:
    """The launch plan of an M x N x K GEMM (host only): tile rows and
    columns, split-K factor, workgroups and fp32 scratch floats."""
    out = np.zeros(4, dtype=np.int32)
    scratch = ctypes.c_int64(0)
    _check(_lib.vla_debug_gemm_plan(dtype, M, N, K, kind, int(skinny), plan_m, plan_batch, out.ctypes.data,
                                    ctypes.byref(scratch)))
    return {"tile": (int(out[0]), int(out[1])), "splits": int(out[2]), "workgroups": int(out[3]),
            "scratch_floats": int(scratch.value)}


def exported_symbols() -> Iterable[str]:
    """Names of the C entry points this binding wraps."""
    return ["vla_preset", "vla_validate", "vla_model_config", "vla_create", "vla_destroy", "vla_ctx_create",
            "vla_ctx_destroy", "vla_vlm_prefill", "vla_action_denoise", "vla_pipeline_run",
            "vla_param_count", "vla_param_info", "vla_export_param", "vla_ctx_export_kv", "vla_ctx_export_cross", "vla_ctx_export_cog", "vla_wavelog_enable", "vla_wavelog_read",
            "vla_debug_gemm", "vla_debug_gemm_epi", "vla_gemm_noalloc", "vla_debug_attention", "vla_debug_attention_cache", "vla_debug_norm", "vla_debug_generate",
            "vla_debug_gemm_plan",
            "vla_kernel_timer",
            "vla_kernel_timer_read", "vla_last_error"]
