"""ctypes binding of libmoddit.so with the C names (argument marshalling only).

Tensors are passed as device pointers (``tensor.data_ptr()``); every step of
the path runs in the HIP kernels of the library.  The stream defaults to
torch's current stream on the current device.  A non-zero status raises
ModError with the library's message.  Importing fails loudly when the
library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_double, c_float, c_int, c_int32, c_size_t, c_void_p

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmoddit.so")

MOD_OK = 0
MOD_ERR_INVALID_ARG = 1
MOD_ERR_UNSUPPORTED = 2
MOD_ERR_BAD_STATE = 3
MOD_ERR_HIP = 4
MOD_ERR_NOMEM = 5
MOD_BUDGET_TOPK = 0
MOD_BUDGET_MASS = 1
MOD_BUDGET_PATTERN = 2


class ModError(RuntimeError):
    def __init__(self, status: int, func: str, msg: str):
        super().__init__(f"{func}: {_status_name(status)}: {msg}")
        self.status = status


class mod_shape(ctypes.Structure):
    _fields_ = [("B", c_int), ("H", c_int), ("L", c_int), ("d", c_int), ("block", c_int),
                ("frame_tokens", c_int), ("text_tokens", c_int)]


class mod_params(ctypes.Structure):
    _fields_ = [("warmup_m", c_int), ("delta_t", c_int), ("tau_e", c_float),
                ("anchor_rule", c_int), ("statistic", c_int), ("eta", c_float)]


class mod_budget(ctypes.Structure):
    _fields_ = [("mode", c_int), ("density", c_float), ("mass", c_float), ("patterns", c_int)]


# torch bundles its own HIP runtime (SONAME libamdhip64.so.7).  Loading torch
# first makes the dynamic loader bind this library to that same runtime
# instead of mapping a second one from /opt/rocm into the process.
try:
    import torch  # noqa: F401
except ImportError:  # pragma: no cover - torch is optional for the ABI itself
    torch = None

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                      "(or python paper_2601_11641_amd/build_lib.py)")
_lib = ctypes.CDLL(LIB_PATH)

_SIGS = {
    "mod_num_blocks": (c_int, [POINTER(mod_shape)]),
    "mod_num_coeffs": (c_int, [POINTER(mod_shape)]),
    "mod_stats_create": (c_int, [POINTER(mod_shape), POINTER(mod_params), POINTER(c_void_p)]),
    "mod_stats_destroy": (c_int, [c_void_p]),
    "mod_collect_stats": (c_int, [c_void_p, c_void_p, c_void_p, c_int, c_void_p]),
    "mod_update_stats": (c_int, [c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_int,
                                 c_void_p]),
    "mod_predict_block_mask": (c_int, [c_void_p, c_void_p, c_void_p, c_int, POINTER(mod_budget),
                                       c_void_p, c_void_p, c_void_p]),
    "mod_attn_workspace_bytes": (c_size_t, [POINTER(mod_shape)]),
    "mod_attn_plan_bytes": (c_size_t, [POINTER(mod_shape)]),
    "mod_block_sparse_attn_fwd": (c_int, [POINTER(mod_shape), c_void_p, c_void_p, c_void_p,
                                          c_void_p, c_void_p, c_float, c_void_p, c_void_p,
                                          c_void_p, c_size_t, c_void_p]),
    "mod_block_sparse_attn_fwd_noalloc": (c_int, [POINTER(mod_shape), c_void_p, c_void_p, c_void_p,
                                                  c_void_p, c_void_p, c_float, c_void_p, c_void_p,
                                                  c_void_p]),
    "mod_stats_get_anchor": (c_int, [c_void_p, c_int, POINTER(c_double), POINTER(c_int)]),
    "mod_stats_get_pooled": (c_int, [c_void_p, POINTER(c_double), POINTER(c_double)]),
    "mod_stats_get_block_mass": (c_int, [c_void_p, POINTER(c_double)]),
    "mod_stats_get_prediction": (c_int, [c_void_p, POINTER(c_double)]),
    "mod_stats_get_gate": (c_int, [c_void_p, POINTER(c_int32)]),
    "mod_status_string": (ctypes.c_char_p, [c_int]),
    "mod_last_error": (ctypes.c_char_p, []),
}
for _name, (_res, _args) in _SIGS.items():
    _f = getattr(_lib, _name)
    _f.restype = _res
    _f.argtypes = _args

EXPORTED = tuple(_SIGS)


def _status_name(st: int) -> str:
    return _lib.mod_status_string(st).decode()


def _check(st: int, func: str):
    if st != MOD_OK:
        raise ModError(st, func, _lib.mod_last_error().decode())


def _ptr(x, what: str, dtype=None):
    """Device pointer of a tensor (checked contiguous / dtype), an int, or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        if not x.is_contiguous():
            raise ValueError(f"{what} must be contiguous")
        if dtype is not None and str(x.dtype) != dtype:
            raise ValueError(f"{what} must be {dtype}, got {x.dtype}")
        if not x.is_cuda:
            raise ValueError(f"{what} must be a device tensor")
        return x.data_ptr()
    raise TypeError(f"{what}: unsupported argument type {type(x)}")


def _stream(stream):
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def make_shape(B, H, L, d, block, frame_tokens=0, text_tokens=0) -> mod_shape:
    return mod_shape(B, H, L, d, block, frame_tokens, text_tokens)


def num_video_blocks(shape: mod_shape) -> int:
    """nv: the blocks of the video tokens, over which the MOD model and the
    introspection arrays are sized."""
    return -(-(shape.L - shape.text_tokens) // shape.block)


def make_params(warmup_m=1, delta_t=0, tau_e=0.0, anchor_rule=0, statistic=0, eta=1e-4) -> mod_params:
    s = {"pooled": 0, "attention": 1}.get(statistic, statistic)
    return mod_params(warmup_m, delta_t, tau_e, anchor_rule, int(s), eta)


def make_budget(mode="topk", density=1.0, mass=1.0, patterns=1) -> mod_budget:
    m = {"topk": MOD_BUDGET_TOPK, "mass": MOD_BUDGET_MASS, "pattern": MOD_BUDGET_PATTERN}.get(mode, mode)
    return mod_budget(int(m), density, mass, int(patterns))


# ---------------------------------------------------------------- entry points

def _ref(x):
    return None if x is None else ctypes.byref(x)


def mod_num_blocks(shape: mod_shape) -> int:
    return _lib.mod_num_blocks(_ref(shape))


def mod_num_coeffs(shape: mod_shape) -> int:
    return _lib.mod_num_coeffs(_ref(shape))


def mod_stats_create(shape: mod_shape, params: mod_params) -> int:
    h = c_void_p()
    _check(_lib.mod_stats_create(ctypes.byref(shape), ctypes.byref(params), ctypes.byref(h)),
           "mod_stats_create")
    return h.value


def mod_stats_destroy(stats) -> None:
    _check(_lib.mod_stats_destroy(stats), "mod_stats_destroy")


def mod_collect_stats(stats, q, k, step: int, stream=None) -> None:
    _check(_lib.mod_collect_stats(stats, _ptr(q, "q", "torch.bfloat16"),
                                  _ptr(k, "k", "torch.bfloat16"), step, _stream(stream)),
           "mod_collect_stats")


def mod_update_stats(stats, q, k, lse, kv_idx, kv_cnt, step: int, stream=None) -> None:
    _check(_lib.mod_update_stats(stats, _ptr(q, "q", "torch.bfloat16"), _ptr(k, "k", "torch.bfloat16"),
                                 _ptr(lse, "lse", "torch.float32"), _ptr(kv_idx, "kv_idx", "torch.int32"),
                                 _ptr(kv_cnt, "kv_cnt", "torch.int32"), step, _stream(stream)),
           "mod_update_stats")


def mod_predict_block_mask(stats, q, k, step: int, budget: mod_budget, kv_idx, kv_cnt,
                           stream=None) -> None:
    _check(_lib.mod_predict_block_mask(stats, _ptr(q, "q", "torch.bfloat16"),
                                       _ptr(k, "k", "torch.bfloat16"), step,
                                       ctypes.byref(budget), _ptr(kv_idx, "kv_idx", "torch.int32"),
                                       _ptr(kv_cnt, "kv_cnt", "torch.int32"), _stream(stream)),
           "mod_predict_block_mask")


def mod_attn_workspace_bytes(shape: mod_shape) -> int:
    return int(_lib.mod_attn_workspace_bytes(_ref(shape)))


def mod_attn_plan_bytes(shape: mod_shape) -> int:
    return int(_lib.mod_attn_plan_bytes(_ref(shape)))


def mod_block_sparse_attn_fwd(shape: mod_shape, q, k, v, kv_idx, kv_cnt, scale: float, o,
                              lse=None, workspace=None, ws_bytes: int = 0, stream=None) -> None:
    """workspace=None: a device buffer of mod_attn_workspace_bytes(shape)
    bytes is allocated for the call (pass one to keep allocations out of a
    loop)."""
    if workspace is None and hasattr(q, "device"):
        ws_bytes = mod_attn_workspace_bytes(shape)
        workspace = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=q.device)
    _check(_lib.mod_block_sparse_attn_fwd(
        ctypes.byref(shape), _ptr(q, "q", "torch.bfloat16"), _ptr(k, "k", "torch.bfloat16"),
        _ptr(v, "v", "torch.bfloat16"), _ptr(kv_idx, "kv_idx", "torch.int32"),
        _ptr(kv_cnt, "kv_cnt", "torch.int32"), float(scale), _ptr(o, "o", "torch.bfloat16"),
        _ptr(lse, "lse", "torch.float32"), _ptr(workspace, "workspace"), ws_bytes,
        _stream(stream)), "mod_block_sparse_attn_fwd")


MOD_ATTN_NOALLOC_MAX_BYTES = 2 << 20


def mod_block_sparse_attn_fwd_noalloc(shape: mod_shape, q, k, v, kv_idx, kv_cnt, scale: float, o,
                                      lse=None, stream=None) -> None:
    """The attention forward with its work plan in the library's own device
    array (no workspace, no allocation in the library or here)."""
    _check(_lib.mod_block_sparse_attn_fwd_noalloc(
        ctypes.byref(shape), _ptr(q, "q", "torch.bfloat16"), _ptr(k, "k", "torch.bfloat16"),
        _ptr(v, "v", "torch.bfloat16"), _ptr(kv_idx, "kv_idx", "torch.int32"),
        _ptr(kv_cnt, "kv_cnt", "torch.int32"), float(scale), _ptr(o, "o", "torch.bfloat16"),
        _ptr(lse, "lse", "torch.float32"), _stream(stream)), "mod_block_sparse_attn_fwd_noalloc")


def _dbl(n):
    a = np.empty(n, dtype=np.float64)
    return a, a.ctypes.data_as(POINTER(c_double))


def mod_stats_get_anchor(stats, slot: int, B: int, H: int, p: int):
    a, ptr = _dbl(B * H * p)
    step = c_int()
    _check(_lib.mod_stats_get_anchor(stats, slot, ptr, ctypes.byref(step)), "mod_stats_get_anchor")
    return a.reshape(B, H, p), step.value


def mod_stats_get_pooled(stats, B: int, H: int, n: int, d: int):
    qa, qp = _dbl(B * H * n * d)
    ka, kp = _dbl(B * H * n * d)
    _check(_lib.mod_stats_get_pooled(stats, qp, kp), "mod_stats_get_pooled")
    return qa.reshape(B, H, n, d), ka.reshape(B, H, n, d)


def mod_stats_get_block_mass(stats, B: int, H: int, n: int):
    a, ptr = _dbl(B * H * n * n)
    _check(_lib.mod_stats_get_block_mass(stats, ptr), "mod_stats_get_block_mass")
    return a.reshape(B, H, n, n)


def mod_stats_get_prediction(stats, B: int, H: int, n: int):
    a, ptr = _dbl(B * H * (3 * n - 1))
    _check(_lib.mod_stats_get_prediction(stats, ptr), "mod_stats_get_prediction")
    return a.reshape(B, H, 3 * n - 1)


def mod_stats_get_gate(stats, B: int, H: int):
    a = np.empty(B * H, dtype=np.int32)
    _check(_lib.mod_stats_get_gate(stats, a.ctypes.data_as(POINTER(c_int32))),
           "mod_stats_get_gate")
    return a.reshape(B, H)


def mod_status_string(status: int) -> str:
    return _status_name(status)


def mod_last_error() -> str:
    return _lib.mod_last_error().decode()


def raw_lib():
    """The loaded ctypes library (for status-code tests)."""
    return _lib


class Stats:
    """Owner of a mod_stats handle (destroyed on close / garbage collection)."""

    def __init__(self, shape: mod_shape, params: mod_params):
        self.shape, self.params = shape, params
        self.handle = mod_stats_create(shape, params)
        self.n = mod_num_blocks(shape)
        self.n_video = num_video_blocks(shape)
        self.p = mod_num_coeffs(shape)

    def close(self):
        if self.handle:
            mod_stats_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()
