"""Python binding of ``libcomera.so`` (the C ABI declared in include/comera.h).

Argument marshalling only: every function here has the name of the C entry
point it calls and passes device pointers, sizes and the stream straight
through.  Tensors (anything with ``data_ptr()``) are passed by pointer; plain
ints are taken as raw addresses.  The library must have been built (see
``build.py``); loading fails loudly otherwise -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libcomera.so")

MAX_CORES = 8
F32, BF16 = 0, 1
OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP, ERR_INTERNAL = 0, -1, -2, -3, -4, -5
ORDER_DENSE, ORDER_SWEEP_RL, ORDER_SWEEP_LR, ORDER_ZERO, ORDER_FUSED_RL = 0, 1, 2, 3, 4

# every function declared in include/comera.h
EXPORTS = (
    "comera_ttm_plan", "comera_ttm_plan_num_orders", "comera_ttm_plan_chosen",
    "comera_ttm_plan_order_info", "comera_ttm_workspace_bytes", "comera_ttm_forward",
    "comera_ttm_backward", "comera_ttm_plan_destroy", "comera_tt_embed_workspace_bytes",
    "comera_tt_embed_forward", "comera_tt_embed_backward", "comera_status_string", "comera_last_hip_error",
    "comera_ttm_plan_set_timing", "comera_ttm_plan_kernel_time", "comera_ttm_plan_set_reuse_forward",
    "comera_ttm_backward_masks", "comera_tt_embed_backward_ex", "comera_ttm_plan_set_fp8", "comera_fp8_quantize",
    "comera_ttm_regularizer_grads", "comera_debug_launch_check", "comera_debug_launch_count",
    "comera_debug_launch_info", "comera_ttm_forward_noalloc",
)
FP8_QUANTIZE_WS_BYTES = 2048
KERNEL_FWD, KERNEL_DX, KERNEL_DW = 0, 1, 2


class ComeraError(RuntimeError):
    def __init__(self, status: int, where: str):
        extra = f": {comera_last_hip_error()}" if status == ERR_HIP else ""
        super().__init__(f"{where}: status {status} ({comera_status_string(status)}){extra}")
        self.status = status


class comera_ttm_shape(ctypes.Structure):
    _fields_ = [("d", ctypes.c_int32), ("act", ctypes.c_int32),
                ("n", ctypes.c_int64 * MAX_CORES), ("m", ctypes.c_int64 * MAX_CORES),
                ("r", ctypes.c_int64 * (MAX_CORES + 1))]


class comera_tt_embed_shape(ctypes.Structure):
    _fields_ = [("d", ctypes.c_int32), ("pad_", ctypes.c_int32),
                ("v", ctypes.c_int64 * MAX_CORES), ("e", ctypes.c_int64 * MAX_CORES),
                ("r", ctypes.c_int64 * (MAX_CORES + 1))]


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the library once; raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with paper_2405_14377_amd/build.py "
                          "(the HIP library is required; there is no CPU fallback)")
    # One HIP runtime per process: torch ships its own libamdhip64 under a
    # different file name, so if this library were opened first the process
    # would end up with two runtimes and the second one finds no device.
    # Loading torch first makes this library bind to torch's runtime.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(path)
    vp, i32, i64, sz, dbl = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_double
    P = ctypes.POINTER
    lib.comera_ttm_plan.argtypes = [P(comera_ttm_shape), i64, vp, i32, P(vp)]
    lib.comera_ttm_plan.restype = i32
    lib.comera_ttm_plan_num_orders.argtypes = [vp]
    lib.comera_ttm_plan_num_orders.restype = i32
    lib.comera_ttm_plan_chosen.argtypes = [vp]
    lib.comera_ttm_plan_chosen.restype = i32
    lib.comera_ttm_plan_order_info.argtypes = [vp, i32, ctypes.c_char_p, sz, P(i32), P(dbl), P(dbl), P(dbl), P(i32)]
    lib.comera_ttm_plan_order_info.restype = i32
    lib.comera_ttm_workspace_bytes.argtypes = [vp]
    lib.comera_ttm_workspace_bytes.restype = sz
    lib.comera_ttm_forward.argtypes = [vp, i64, vp, vp, vp, vp, vp, sz, vp]
    lib.comera_ttm_forward.restype = i32
    lib.comera_ttm_forward_noalloc.argtypes = [vp, i64, vp, vp, vp, vp, vp]
    lib.comera_ttm_forward_noalloc.restype = i32
    lib.comera_ttm_backward.argtypes = [vp, i64, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.comera_ttm_backward.restype = i32
    lib.comera_ttm_backward_masks.argtypes = [vp, i64, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.comera_ttm_backward_masks.restype = i32
    lib.comera_ttm_regularizer_grads.argtypes = [P(comera_ttm_shape), ctypes.c_float, ctypes.c_float, vp, vp, vp, vp,
                                                 vp]
    lib.comera_ttm_regularizer_grads.restype = i32
    lib.comera_ttm_plan_destroy.argtypes = [vp]
    lib.comera_ttm_plan_destroy.restype = None
    lib.comera_tt_embed_workspace_bytes.argtypes = [P(comera_tt_embed_shape), i64]
    lib.comera_tt_embed_workspace_bytes.restype = sz
    lib.comera_tt_embed_forward.argtypes = [P(comera_tt_embed_shape), vp, i64, vp, vp, vp, vp, sz, vp, vp]
    lib.comera_tt_embed_forward.restype = i32
    lib.comera_tt_embed_backward.argtypes = [P(comera_tt_embed_shape), vp, i64, vp, vp, vp, vp, i32, vp, sz, vp, vp]
    lib.comera_tt_embed_backward.restype = i32
    lib.comera_tt_embed_backward_ex.argtypes = [P(comera_tt_embed_shape), vp, i64, vp, vp, vp, vp, i32, vp, sz, vp,
                                                vp]
    lib.comera_tt_embed_backward_ex.restype = i32
    lib.comera_ttm_plan_set_timing.argtypes = [vp, i32]
    lib.comera_ttm_plan_set_reuse_forward.argtypes = [vp, i32]
    lib.comera_ttm_plan_set_reuse_forward.restype = i32
    lib.comera_ttm_plan_set_fp8.argtypes = [vp, i32]
    lib.comera_ttm_plan_set_fp8.restype = i32
    lib.comera_fp8_quantize.argtypes = [vp, i32, i64, i64, vp, i64, vp, i64, vp, vp, sz, vp]
    lib.comera_fp8_quantize.restype = i32
    lib.comera_ttm_plan_set_timing.restype = i32
    lib.comera_ttm_plan_kernel_time.argtypes = [vp, i32, P(dbl), P(i32)]
    lib.comera_ttm_plan_kernel_time.restype = i32
    lib.comera_status_string.argtypes = [i32]
    lib.comera_status_string.restype = ctypes.c_char_p
    lib.comera_last_hip_error.argtypes = []
    lib.comera_last_hip_error.restype = ctypes.c_char_p
    lib.comera_debug_launch_check.argtypes = [i32]
    lib.comera_debug_launch_check.restype = i32
    lib.comera_debug_launch_count.argtypes = []
    lib.comera_debug_launch_count.restype = i32
    u32, u64 = ctypes.c_uint32, ctypes.c_uint64
    lib.comera_debug_launch_info.argtypes = [i32, ctypes.c_char_p, sz, P(u32), P(u32), P(u64), P(i32)]
    lib.comera_debug_launch_info.restype = i32
    _lib = lib
    return lib


# ------------------------------------------------------------------ marshalling helpers
def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return int(x.data_ptr())


def _ptr_array(xs: Optional[Sequence]):
    """Host array of device pointers (NULL entries allowed), or NULL."""
    if xs is None:
        return None
    arr = (ctypes.c_void_p * max(1, len(xs)))()
    for i, x in enumerate(xs):
        arr[i] = _ptr(x)
    return arr


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return int(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return stream
    return int(stream.cuda_stream)


def _nbytes(ws) -> int:
    if ws is None:
        return 0
    return int(ws.numel() * ws.element_size())


def _check(status: int, where: str) -> None:
    if status != OK:
        raise ComeraError(status, where)


def ttm_shape(n: Sequence[int], m: Sequence[int], r: Sequence[int], act: int = F32) -> comera_ttm_shape:
    s = comera_ttm_shape()
    s.d = len(n)
    s.act = act
    for k in range(len(n)):
        s.n[k] = int(n[k])
        s.m[k] = int(m[k])
    for k in range(len(r)):
        s.r[k] = int(r[k])
    return s


def tt_embed_shape(v: Sequence[int], e: Sequence[int], r: Sequence[int]) -> comera_tt_embed_shape:
    s = comera_tt_embed_shape()
    s.d = len(v)
    for k in range(len(v)):
        s.v[k] = int(v[k])
        s.e[k] = int(e[k])
    for k in range(len(r)):
        s.r[k] = int(r[k])
    return s


# ------------------------------------------------------------------ entry points
def comera_status_string(status: int) -> str:
    return load().comera_status_string(int(status)).decode()


def comera_last_hip_error() -> str:
    return load().comera_last_hip_error().decode()


def comera_ttm_plan(shape: comera_ttm_shape, batch: int, mask_active=None, force_order: int = -1,
                    raise_on_error: bool = True):
    """Returns a plan handle (int) or, with raise_on_error=False, (status, handle)."""
    lib = load()
    h = ctypes.c_void_p()
    buf = None
    if mask_active is not None:
        data = bytes(int(bool(x)) for x in mask_active)
        buf = ctypes.create_string_buffer(data, max(1, len(data)))
    st = lib.comera_ttm_plan(ctypes.byref(shape), int(batch), buf, int(force_order), ctypes.byref(h))
    if not raise_on_error:
        return st, h.value
    _check(st, "comera_ttm_plan")
    return h.value


def comera_ttm_plan_num_orders(plan) -> int:
    return int(load().comera_ttm_plan_num_orders(plan))


def comera_ttm_plan_chosen(plan) -> int:
    return int(load().comera_ttm_plan_chosen(plan))


def comera_ttm_plan_order_info(plan, i: int) -> dict:
    buf = ctypes.create_string_buffer(160)
    kind = ctypes.c_int32()
    ff, fb, by = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    ex = ctypes.c_int32()
    st = load().comera_ttm_plan_order_info(plan, int(i), buf, 160, ctypes.byref(kind), ctypes.byref(ff),
                                           ctypes.byref(fb), ctypes.byref(by), ctypes.byref(ex))
    _check(st, "comera_ttm_plan_order_info")
    return {"desc": buf.value.decode(), "kind": kind.value, "flops_fwd": ff.value, "flops_bwd": fb.value,
            "bytes": by.value, "executable": bool(ex.value)}


def comera_ttm_workspace_bytes(plan) -> int:
    return int(load().comera_ttm_workspace_bytes(plan))


def comera_ttm_forward(plan, b: int, X, G, D, Y, ws, stream=None) -> int:
    st = load().comera_ttm_forward(plan, int(b), _ptr(X), _ptr_array(G), _ptr_array(D), _ptr(Y), _ptr(ws),
                                   _nbytes(ws), _stream(stream))
    _check(st, "comera_ttm_forward")
    return st


def comera_ttm_forward_noalloc(plan, b: int, X, G, D, Y, stream=None, raise_on_error: bool = True) -> int:
    st = load().comera_ttm_forward_noalloc(plan, int(b), _ptr(X), _ptr_array(G), _ptr_array(D), _ptr(Y),
                                           _stream(stream))
    if raise_on_error:
        _check(st, "comera_ttm_forward_noalloc")
    return st


def comera_ttm_backward(plan, b: int, X, dY, G, D, dX, dG, ws, stream=None) -> int:
    st = load().comera_ttm_backward(plan, int(b), _ptr(X), _ptr(dY), _ptr_array(G), _ptr_array(D), _ptr(dX),
                                    _ptr_array(dG), _ptr(ws), _nbytes(ws), _stream(stream))
    _check(st, "comera_ttm_backward")
    return st


def comera_ttm_regularizer_grads(shape, gamma: float, beta: float, G, D, dG, dD, stream=None) -> int:
    """Add the early-stage regulariser gradients in place (eq. pretrain-rank):
    dG_k += 2 beta G_k, dD_k += gamma dS^/dD_k.  `shape` is a comera_ttm_shape;
    G, dG, D, dD are lists of device tensors (or None)."""
    st = load().comera_ttm_regularizer_grads(ctypes.byref(shape), float(gamma), float(beta), _ptr_array(G),
                                             _ptr_array(D), _ptr_array(dG), _ptr_array(dD), _stream(stream))
    _check(st, "comera_ttm_regularizer_grads")
    return st


def comera_ttm_backward_masks(plan, b: int, X, dY, G, D, dX, dG, dD, ws, stream=None) -> int:
    st = load().comera_ttm_backward_masks(plan, int(b), _ptr(X), _ptr(dY), _ptr_array(G), _ptr_array(D), _ptr(dX),
                                          _ptr_array(dG), _ptr_array(dD), _ptr(ws), _nbytes(ws), _stream(stream))
    _check(st, "comera_ttm_backward_masks")
    return st


def comera_ttm_plan_destroy(plan) -> None:
    if plan:
        load().comera_ttm_plan_destroy(plan)


def comera_ttm_plan_set_timing(plan, enable: bool) -> None:
    _check(load().comera_ttm_plan_set_timing(plan, int(bool(enable))), "comera_ttm_plan_set_timing")


def comera_ttm_plan_set_reuse_forward(plan, enable: bool) -> None:
    _check(load().comera_ttm_plan_set_reuse_forward(plan, int(bool(enable))), "comera_ttm_plan_set_reuse_forward")


def comera_ttm_plan_set_fp8(plan, enable: bool) -> None:
    _check(load().comera_ttm_plan_set_fp8(plan, int(bool(enable))), "comera_ttm_plan_set_fp8")


def comera_fp8_quantize(x, dtype: int, rows: int, cols: int, q, ldq: int, qt, ldt: int, scale, ws,
                        stream=None) -> int:
    st = load().comera_fp8_quantize(_ptr(x), int(dtype), int(rows), int(cols), _ptr(q), int(ldq), _ptr(qt), int(ldt),
                                    _ptr(scale), _ptr(ws), _nbytes(ws), _stream(stream))
    _check(st, "comera_fp8_quantize")
    return st


def comera_ttm_plan_kernel_time(plan, kernel: int):
    """(mean ms, launches) of one kernel since the last query; clears the record."""
    ms, cnt = ctypes.c_double(), ctypes.c_int32()
    _check(load().comera_ttm_plan_kernel_time(plan, int(kernel), ctypes.byref(ms), ctypes.byref(cnt)),
           "comera_ttm_plan_kernel_time")
    return ms.value, cnt.value


def comera_tt_embed_workspace_bytes(shape: comera_tt_embed_shape, n_tokens: int) -> int:
    return int(load().comera_tt_embed_workspace_bytes(ctypes.byref(shape), int(n_tokens)))


def comera_tt_embed_forward(shape, ids, n_tokens: int, G, D, Y, ws, err_flag=None, stream=None) -> int:
    st = load().comera_tt_embed_forward(ctypes.byref(shape), _ptr(ids), int(n_tokens), _ptr_array(G), _ptr_array(D),
                                        _ptr(Y), _ptr(ws), _nbytes(ws), _ptr(err_flag), _stream(stream))
    _check(st, "comera_tt_embed_forward")
    return st


def comera_tt_embed_backward(shape, ids, n_tokens: int, dY, G, D, dG, deterministic: int, ws, err_flag=None,
                             stream=None) -> int:
    st = load().comera_tt_embed_backward(ctypes.byref(shape), _ptr(ids), int(n_tokens), _ptr(dY), _ptr_array(G),
                                         _ptr_array(D), _ptr_array(dG), int(deterministic), _ptr(ws), _nbytes(ws),
                                         _ptr(err_flag), _stream(stream))
    _check(st, "comera_tt_embed_backward")
    return st


EMBED_REUSE_FORWARD = 1


def comera_debug_launch_check(enable: bool) -> None:
    _check(load().comera_debug_launch_check(int(bool(enable))), "comera_debug_launch_check")


def comera_debug_launch_log() -> list:
    """Every launch recorded since launch check mode was switched on:
    dicts with the kernel expression, grid, block, LDS bytes and whether the
    configuration is within the limits."""
    lib = load()
    out = []
    name = ctypes.create_string_buffer(256)
    g3, b3 = (ctypes.c_uint32 * 3)(), (ctypes.c_uint32 * 3)()
    lds, ok = ctypes.c_uint64(), ctypes.c_int32()
    for i in range(int(lib.comera_debug_launch_count())):
        _check(lib.comera_debug_launch_info(i, name, 256, g3, b3, ctypes.byref(lds), ctypes.byref(ok)),
               "comera_debug_launch_info")
        out.append({"kernel": name.value.decode(), "grid": tuple(g3), "block": tuple(b3), "lds": lds.value,
                    "ok": bool(ok.value)})
    return out


def comera_tt_embed_backward_ex(shape, ids, n_tokens: int, dY, G, D, dG, flags: int, ws, err_flag=None,
                                stream=None) -> int:
    st = load().comera_tt_embed_backward_ex(ctypes.byref(shape), _ptr(ids), int(n_tokens), _ptr(dY), _ptr_array(G),
                                            _ptr_array(D), _ptr_array(dG), int(flags), _ptr(ws), _nbytes(ws),
                                            _ptr(err_flag), _stream(stream))
    _check(st, "comera_tt_embed_backward_ex")
    return st


class TTMPlan:
    """Owns a plan handle (destroyed with the object)."""

    def __init__(self, n, m, r, act: int = F32, batch: int = 0, mask_active=None, force_order: int = -1):
        self.shape = ttm_shape(n, m, r, act)
        self.n, self.m, self.r, self.act, self.batch = tuple(n), tuple(m), tuple(r), act, batch
        self.handle = comera_ttm_plan(self.shape, batch, mask_active, force_order)

    @property
    def workspace_bytes(self) -> int:
        return comera_ttm_workspace_bytes(self.handle)

    @property
    def num_orders(self) -> int:
        return comera_ttm_plan_num_orders(self.handle)

    @property
    def chosen(self) -> int:
        return comera_ttm_plan_chosen(self.handle)

    def order_info(self, i: int) -> dict:
        return comera_ttm_plan_order_info(self.handle, i)

    def set_reuse_forward(self, enable: bool = True) -> None:
        comera_ttm_plan_set_reuse_forward(self.handle, enable)

    def set_fp8(self, enable: bool = True) -> None:
        comera_ttm_plan_set_fp8(self.handle, enable)

    def __del__(self):
        try:
            comera_ttm_plan_destroy(self.handle)
        except Exception:
            pass
        self.handle = None
