"""Thin ctypes binding of libmoepd (the C ABI declared in include/moepd.h and
include/moepd_turnstile.h).

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
from ctypes import POINTER, byref, c_char_p, c_double, c_int, c_int32, c_int64, c_void_p

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmoepd.so")

MOE_PHASE_P, MOE_PHASE_D, MOE_NUM_PHASES = 0, 1, 2
MOE_DTYPE_F32, MOE_DTYPE_BF16, MOE_DTYPE_FP8 = 0, 1, 2

MOE_OK = 0
MOE_ERR_INVALID_ARG = -1
MOE_ERR_INVALID_PHASE = -2
MOE_ERR_CAPACITY = -3
MOE_ERR_STATE = -4
MOE_ERR_BUSY = -5
MOE_ERR_OOM = -6
MOE_ERR_HIP = -7
MOE_ERR_REJECTED = -8
MOE_ERR_TIMEOUT = -9

MOE_TS_IDLE, MOE_TS_ACTIVE, MOE_TS_DONE = 0, 1, 2
MOE_TS_EV_BEGIN, MOE_TS_EV_PUBLISH, MOE_TS_EV_RESUME, MOE_TS_EV_ENTER, MOE_TS_EV_RELEASE, MOE_TS_EV_DONE = range(6)

MOE_STATE_IDLE, MOE_STATE_ROUTED, MOE_STATE_DISPATCHED, MOE_STATE_COMPUTED, MOE_STATE_LAID_OUT = 0, 1, 2, 3, 4

MOE_KERNEL_ROUTE = 0
MOE_KERNEL_COUNT = 1
MOE_KERNEL_PLACE = 2
MOE_KERNEL_PERMUTE = 3
MOE_KERNEL_GEMM1 = 4
MOE_KERNEL_GEMM2 = 5
MOE_KERNEL_COMBINE = 6
MOE_KERNEL_ROUTER = 7
MOE_NUM_KERNELS = 8


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
    _fields_ = [("w_gate_up", c_void_p), ("w_down", c_void_p), ("w_gate_up_scales", c_void_p),
                ("w_down_scales", c_void_p)]


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
        ("logits", c_void_p),
        ("x_perm_scales", c_void_p),
        ("h_scales", c_void_p),
    ]


class moe_turnstile_state_t(ctypes.Structure):
    _fields_ = [
        ("epoch", c_int64),
        ("reached", c_int64),
        ("permit", c_int64),
        ("span", c_int32),
        ("task", c_int32),
        ("rounds", c_int64),
        ("rejected", c_int64),
        ("p_wait_us", c_double),
        ("d_wait_us", c_double),
        ("d_entries", c_int64),
        ("log_dropped", c_int64),
    ]


class moe_turnstile_event_t(ctypes.Structure):
    _fields_ = [("kind", c_int32), ("reserved", c_int32), ("epoch", c_int64), ("value", c_int64),
                ("t_ns", c_int64)]


class moe_p_epoch_stats_t(ctypes.Structure):
    _fields_ = [
        ("status", c_int32),
        ("layers_done", c_int32),
        ("enqueue_us", c_double),
        ("wait_us", c_double),
        ("t_begin_ns", c_int64),
        ("t_end_ns", c_int64),
    ]


# Every symbol the headers declare, with its ctypes signature.
_SIGNATURES = {
    "moe_ctx_create": (c_int, [POINTER(moe_config_t), POINTER(moe_weights_t), POINTER(c_void_p)]),
    "moe_route": (c_int, [c_void_p, c_int, c_void_p, c_int32, c_void_p]),
    "moe_route_from_hidden": (c_int, [c_void_p, c_int, c_void_p, c_void_p, c_void_p, c_int32, c_void_p]),
    "moe_dispatch": (c_int, [c_void_p, c_int, c_void_p, c_void_p]),
    "moe_dispatch_layout": (c_int, [c_void_p, c_int, c_void_p]),
    "moe_dispatch_permute": (c_int, [c_void_p, c_int, c_void_p, c_void_p]),
    "moe_dispatch_layout_noalloc": (c_int, [c_void_p, c_int32, c_int32, c_int32, c_int32, c_void_p, c_void_p,
                                            c_void_p, c_void_p, c_void_p]),
    "moe_expert_ffn": (c_int, [c_void_p, c_int, c_void_p]),
    "moe_combine": (c_int, [c_void_p, c_int, c_void_p, c_void_p]),
    "moe_phase_view": (c_int, [c_void_p, c_int, POINTER(moe_phase_view_t)]),
    "moe_phase_reset": (c_int, [c_void_p, c_int]),
    "moe_ctx_destroy": (c_int, [c_void_p]),
    "moe_status_string": (c_char_p, [c_int]),
    "moe_timing_enable": (c_int, [c_void_p, c_int32]),
    "moe_timing_read": (c_int, [c_void_p, c_int, c_int, POINTER(c_double), POINTER(c_int32)]),
    "moe_kernel_name": (c_char_p, [c_int]),
    "moe_clock_probe": (c_int, [c_void_p, c_int32, c_void_p]),
    "moe_turnstile_create": (c_int, [c_int32, c_int32, POINTER(c_void_p)]),
    "moe_turnstile_destroy": (c_int, [c_void_p]),
    "moe_turnstile_set_span": (c_int, [c_void_p, c_int32]),
    "moe_turnstile_begin": (c_int, [c_void_p, c_int64, c_int32]),
    "moe_turnstile_publish": (c_int, [c_void_p, c_int64, c_int64]),
    "moe_turnstile_wait_permit": (c_int, [c_void_p, c_int64, c_int64, c_int64]),
    "moe_turnstile_done": (c_int, [c_void_p, c_int64]),
    "moe_turnstile_wait_boundary": (c_int, [c_void_p, c_int64]),
    "moe_turnstile_release": (c_int, [c_void_p]),
    "moe_turnstile_query": (c_int, [c_void_p, POINTER(moe_turnstile_state_t)]),
    "moe_turnstile_log": (c_int, [c_void_p, POINTER(moe_turnstile_event_t), c_int32, POINTER(c_int32)]),
    "moe_p_epoch_start": (c_int, [c_void_p, c_void_p, c_int64, c_int32, c_int32, c_int32, POINTER(c_void_p),
                                  POINTER(c_void_p), POINTER(c_void_p), c_void_p, c_int64, POINTER(c_void_p)]),
    "moe_p_epoch_join": (c_int, [c_void_p, POINTER(moe_p_epoch_stats_t)]),
}
SYMBOLS = tuple(_SIGNATURES)


def _load():
    # The library links the HIP runtime by its soname.  PyTorch's ROCm wheel
    # carries its own copy of that runtime; when torch is loaded first, the
    # dynamic linker binds the library to the copy already in the process,
    # so torch's allocations and streams and the library's calls share one
    # runtime.  Loaded the other way round, the process would hold two.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
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


def moe_ctx_create(cfg: moe_config_t, w_gate_up, w_down, w_gate_up_scales=None, w_down_scales=None):
    w = moe_weights_t(_ptr(w_gate_up), _ptr(w_down), _ptr(w_gate_up_scales), _ptr(w_down_scales))
    out = c_void_p()
    st = _lib.moe_ctx_create(byref(cfg) if cfg is not None else None, byref(w), byref(out))
    return st, out.value


def moe_route(ctx, phase: int, logits, T: int, stream) -> int:
    return _lib.moe_route(ctx, phase, _ptr(logits), T, _stream(stream))


def moe_route_from_hidden(ctx, phase: int, x, w_router, bias, T: int, stream) -> int:
    return _lib.moe_route_from_hidden(ctx, phase, _ptr(x), _ptr(w_router), _ptr(bias), T, _stream(stream))


def moe_dispatch(ctx, phase: int, x, stream) -> int:
    return _lib.moe_dispatch(ctx, phase, _ptr(x), _stream(stream))


def moe_dispatch_layout(ctx, phase: int, stream) -> int:
    return _lib.moe_dispatch_layout(ctx, phase, _stream(stream))


def moe_dispatch_layout_noalloc(topk_idx, T: int, top_k: int, expert_begin: int, num_local_experts: int, counts,
                                offsets, row_of_slot, token_of_row, stream) -> int:
    return _lib.moe_dispatch_layout_noalloc(_ptr(topk_idx), T, top_k, expert_begin, num_local_experts, _ptr(counts),
                                            _ptr(offsets), _ptr(row_of_slot), _ptr(token_of_row), _stream(stream))


def moe_dispatch_permute(ctx, phase: int, x, stream) -> int:
    return _lib.moe_dispatch_permute(ctx, phase, _ptr(x), _stream(stream))


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


def moe_clock_probe(stream, spin_us: int, out_dev) -> int:
    """out_dev: device buffer of two uint64 (shader-clock ticks, 100 MHz ticks)."""
    return _lib.moe_clock_probe(_stream(stream), spin_us, _ptr(out_dev))


# ---- turnstile (include/moepd_turnstile.h) ----

def moe_turnstile_create(span: int, log_capacity: int = 0):
    out = c_void_p()
    st = _lib.moe_turnstile_create(span, log_capacity, byref(out))
    return st, out.value


def moe_turnstile_destroy(ts) -> int:
    return _lib.moe_turnstile_destroy(ts)


def moe_turnstile_set_span(ts, span: int) -> int:
    return _lib.moe_turnstile_set_span(ts, span)


def moe_turnstile_begin(ts, epoch: int, d_enqueued: bool) -> int:
    return _lib.moe_turnstile_begin(ts, epoch, int(bool(d_enqueued)))


def moe_turnstile_publish(ts, epoch: int, boundary: int) -> int:
    return _lib.moe_turnstile_publish(ts, epoch, boundary)


def moe_turnstile_wait_permit(ts, epoch: int, boundary: int, timeout_us: int) -> int:
    return _lib.moe_turnstile_wait_permit(ts, epoch, boundary, timeout_us)


def moe_turnstile_done(ts, epoch: int) -> int:
    return _lib.moe_turnstile_done(ts, epoch)


def moe_turnstile_wait_boundary(ts, timeout_us: int) -> int:
    return _lib.moe_turnstile_wait_boundary(ts, timeout_us)


def moe_turnstile_release(ts) -> int:
    return _lib.moe_turnstile_release(ts)


def moe_turnstile_query(ts):
    q = moe_turnstile_state_t()
    st = _lib.moe_turnstile_query(ts, byref(q))
    return st, q


def moe_turnstile_log(ts, capacity: int = 4096):
    """(status, [(kind, epoch, value, t_ns), ...]) of the events moved out of the log."""
    buf = (moe_turnstile_event_t * max(capacity, 1))()
    n = c_int32()
    st = _lib.moe_turnstile_log(ts, buf, capacity, byref(n))
    return st, [(buf[i].kind, buf[i].epoch, buf[i].value, buf[i].t_ns) for i in range(n.value)]


def moe_p_epoch_start(ctx, ts, epoch: int, d_enqueued: bool, T: int, logits, x, out, stream, timeout_us: int):
    """Start a P-epoch runner over len(logits) layers; logits, x and out are
    sequences of device buffers (one per layer).  Returns (status, runner)."""
    L = len(logits)
    if len(x) != L or len(out) != L:
        return MOE_ERR_INVALID_ARG, None
    arr = lambda seq: (c_void_p * L)(*[_ptr(b) for b in seq])
    r = c_void_p()
    st = _lib.moe_p_epoch_start(ctx, ts, epoch, int(bool(d_enqueued)), L, T, arr(logits), arr(x), arr(out),
                                _stream(stream), timeout_us, byref(r))
    return st, r.value


def moe_p_epoch_join(runner):
    s = moe_p_epoch_stats_t()
    st = _lib.moe_p_epoch_join(runner, byref(s))
    return st, s


def layer(ctx, phase: int, logits, T: int, x, out, stream) -> None:
    """The four calls of one phase batch, in order, raising on any error."""
    check(moe_route(ctx, phase, logits, T, stream), "moe_route")
    check(moe_dispatch(ctx, phase, x, stream), "moe_dispatch")
    check(moe_expert_ffn(ctx, phase, stream), "moe_expert_ffn")
    check(moe_combine(ctx, phase, out, stream), "moe_combine")
