"""Thin ctypes binding of libmoepd (the C ABI declared in include/moepd.h).

Argument marshalling only: every step of the layer runs in the HIP library.
Device buffers may be passed as integers (device addresses) or as objects
with a ``data_ptr()`` method (torch tensors); streams as integers
(``hipStream_t`` handles) or objects with a ``cuda_stream`` attribute
(``torch.cuda.Stream``).  Every wrapper returns the library's status code,
except ``moe_ctx_create`` which returns ``(status, ctx)``.  ``check`` turns a
status into an exception.

The library must have been built (``python -m paper_2609_00993_amd.build``);
importing this module fails loudly otherwise.
"""

from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, byref, c_char_p, c_double, c_int, c_int32, c_void_p

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmoepd.so")

MOE_PHASE_P, MOE_PHASE_D, MOE_NUM_PHASES = 0, 1, 2
MOE_DTYPE_F32, MOE_DTYPE_BF16 = 0, 1

MOE_OK = 0
MOE_ERR_INVALID_ARG = -1
MOE_ERR_INVALID_PHASE = -2
MOE_ERR_CAPACITY = -3
MOE_ERR_STATE = -4
MOE_ERR_BUSY = -5
MOE_ERR_OOM = -6
MOE_ERR_HIP = -7

MOE_STATE_IDLE, MOE_STATE_ROUTED, MOE_STATE_DISPATCHED, MOE_STATE_COMPUTED = 0, 1, 2, 3

MOE_KERNEL_ROUTE = 0
MOE_KERNEL_COUNT = 1
MOE_KERNEL_PLACE = 2
MOE_KERNEL_PERMUTE = 3
MOE_KERNEL_GEMM1 = 4
MOE_KERNEL_GEMM2 = 5
MOE_KERNEL_COMBINE = 6
MOE_NUM_KERNELS = 7


class moe_config_t(ctypes.Structure):
    _fields_ = [
        ("num_experts", c_int32),
        ("expert_begin", c_int32),
        ("num_local_experts", c_int32),
        ("top_k", c_int32),
        ("hidden", c_int32),
        ("inter", c_int32),
        ("dtype", c_int32),
        ("max_tokens", c_int32 * 2),
        ("flags", c_int32),
        ("d_priority_us", c_int32),
    ]


class moe_weights_t(ctypes.Structure):
    _fields_ = [("w_gate_up", c_void_p), ("w_down", c_void_p)]


class moe_phase_view_t(ctypes.Structure):
    _fields_ = [
        ("state", c_int32),
        ("tokens", c_int32),
        ("rows_capacity", c_int32),
        ("reserved", c_int32),
        ("topk_idx", c_void_p),
        ("topk_w", c_void_p),
        ("counts", c_void_p),
        ("offsets", c_void_p),
        ("row_of_slot", c_void_p),
        ("token_of_row", c_void_p),
        ("x_perm", c_void_p),
        ("h", c_void_p),
        ("y", c_void_p),
    ]


# Every symbol the header declares, with its ctypes signature.
_SIGNATURES = {
    "moe_ctx_create": (c_int, [POINTER(moe_config_t), POINTER(moe_weights_t), POINTER(c_void_p)]),
    "moe_route": (c_int, [c_void_p, c_int, c_void_p, c_int32, c_void_p]),
    "moe_dispatch": (c_int, [c_void_p, c_int, c_void_p, c_void_p]),
    "moe_expert_ffn": (c_int, [c_void_p, c_int, c_void_p]),
    "moe_combine": (c_int, [c_void_p, c_int, c_void_p, c_void_p]),
    "moe_phase_view": (c_int, [c_void_p, c_int, POINTER(moe_phase_view_t)]),
    "moe_phase_reset": (c_int, [c_void_p, c_int]),
    "moe_ctx_destroy": (c_int, [c_void_p]),
    "moe_status_string": (c_char_p, [c_int]),
    "moe_timing_enable": (c_int, [c_void_p, c_int32]),
    "moe_timing_read": (c_int, [c_void_p, c_int, c_int, POINTER(c_double), POINTER(c_int32)]),
    "moe_kernel_name": (c_char_p, [c_int]),
}
SYMBOLS = tuple(_SIGNATURES)


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"libmoepd.so is not built ({LIB_PATH} missing); run `python -m paper_2609_00993_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    for name, (res, args) in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_lib = _load()


class MoeError(RuntimeError):
    def __init__(self, status: int, what: str = ""):
        self.status = status
        super().__init__(f"{what}: {moe_status_string(status)} ({status})" if what else moe_status_string(status))


def check(status: int, what: str = "") -> None:
    if status != MOE_OK:
        raise MoeError(status, what)


def _ptr(p) -> int:
    if p is None:
        return 0
    if isinstance(p, int):
        return p
    return int(p.data_ptr())


def _stream(s) -> int:
    if s is None:
        return 0
    if isinstance(s, int):
        return s
    return int(s.cuda_stream)


def make_config(num_experts, expert_begin, num_local_experts, top_k, hidden, inter, dtype, max_tokens_p,
                max_tokens_d, flags=0, d_priority_us=0) -> moe_config_t:
    c = moe_config_t()
    c.num_experts = num_experts
    c.expert_begin = expert_begin
    c.num_local_experts = num_local_experts
    c.top_k = top_k
    c.hidden = hidden
    c.inter = inter
    c.dtype = dtype
    c.max_tokens[0] = max_tokens_p
    c.max_tokens[1] = max_tokens_d
    c.flags = flags
    c.d_priority_us = d_priority_us
    return c


def moe_ctx_create(cfg: moe_config_t, w_gate_up, w_down):
    w = moe_weights_t(_ptr(w_gate_up), _ptr(w_down))
    out = c_void_p()
    st = _lib.moe_ctx_create(byref(cfg) if cfg is not None else None, byref(w), byref(out))
    return st, out.value


def moe_route(ctx, phase: int, logits, T: int, stream) -> int:
    return _lib.moe_route(ctx, phase, _ptr(logits), T, _stream(stream))


def moe_dispatch(ctx, phase: int, x, stream) -> int:
    return _lib.moe_dispatch(ctx, phase, _ptr(x), _stream(stream))


def moe_expert_ffn(ctx, phase: int, stream) -> int:
    return _lib.moe_expert_ffn(ctx, phase, _stream(stream))


def moe_combine(ctx, phase: int, out, stream) -> int:
    return _lib.moe_combine(ctx, phase, _ptr(out), _stream(stream))


def moe_phase_view(ctx, phase: int):
    v = moe_phase_view_t()
    st = _lib.moe_phase_view(ctx, phase, byref(v))
    return st, v


def moe_phase_reset(ctx, phase: int) -> int:
    return _lib.moe_phase_reset(ctx, phase)


def moe_ctx_destroy(ctx) -> int:
    return _lib.moe_ctx_destroy(ctx)


def moe_status_string(status: int) -> str:
    return _lib.moe_status_string(status).decode()


def moe_timing_enable(ctx, max_launches: int) -> int:
    return _lib.moe_timing_enable(ctx, max_launches)


def moe_timing_read(ctx, phase: int, kernel: int):
    ms = c_double()
    n = c_int32()
    st = _lib.moe_timing_read(ctx, phase, kernel, byref(ms), byref(n))
    return st, ms.value, n.value


def moe_kernel_name(kernel: int) -> str:
    return _lib.moe_kernel_name(kernel).decode()


def layer(ctx, phase: int, logits, T: int, x, out, stream) -> None:
    """The four calls of one phase batch, in order, raising on any error."""
    check(moe_route(ctx, phase, logits, T, stream), "moe_route")
    check(moe_dispatch(ctx, phase, x, stream), "moe_dispatch")
    check(moe_expert_ffn(ctx, phase, stream), "moe_expert_ffn")
    check(moe_combine(ctx, phase, out, stream), "moe_combine")
