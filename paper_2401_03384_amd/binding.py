"""ctypes binding of libconvein.so: the C ABI of include/convein.h, one Python
function per C entry point, same names, argument marshalling only.

Raises ImportError when the library has not been built: there is no fallback
of any kind.
"""
from __future__ import annotations

import ctypes as C
import functools
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libconvein.so")

CE_OK = 0
CE_ERR_PARSE = -1
CE_ERR_SHAPE = -2
CE_ERR_UNSUPPORTED = -3
CE_ERR_ARG = -4
CE_ERR_WORKSPACE = -5
CE_ERR_OVERFLOW = -6
CE_ERR_HIP = -7

CE_F32 = 0
CE_BF16 = 1
CE_COST_FWD = 0
CE_COST_TRAIN_PAPER = 1
CE_FLAG_GENERIC_ONLY = 0x1
CE_FLAG_NO_FUSION = 0x2
CE_FLAG_SAVE_INTERMEDIATES = 0x4
CE_FLAG_WIDE_OFFSETS = 0x8
CE_NOALLOC_WORKSPACE_BYTES = 64 << 20
CE_PAD_SAME_ZERO = 0
CE_PAD_CIRCULAR = 1

_STATUS_NAMES = {0: "CE_OK", -1: "CE_ERR_PARSE", -2: "CE_ERR_SHAPE", -3: "CE_ERR_UNSUPPORTED",
                 -4: "CE_ERR_ARG", -5: "CE_ERR_WORKSPACE", -6: "CE_ERR_OVERFLOW", -7: "CE_ERR_HIP"}

# Every symbol the header declares (checked by the test-suite).
EXPORTS = [
    "ce_expr_parse", "ce_expr_set_feature", "ce_expr_set_conv", "ce_expr_set_stride",
    "ce_expr_output_shape",
    "ce_expr_destroy",
    "ce_plan_create", "ce_plan_create_limited", "ce_plan_create_ex", "ce_plan_checkpoint",
    "ce_plan_create_with_path", "ce_plan_num_steps",
    "ce_plan_step",
    "ce_plan_cost", "ce_plan_left_to_right_cost", "ce_plan_workspace_size", "ce_plan_describe",
    "ce_plan_destroy", "ce_forward", "ce_backward", "ce_backward_noalloc", "ce_timing_begin", "ce_timing_begin_kernel",
    "ce_timing_end", "ce_timing_record", "ce_last_error", "ce_version",
]


class PlanOptions(C.Structure):
    """ce_plan_options of include/convein.h."""
    _fields_ = [("mode", C.c_int), ("dtype", C.c_int), ("flags", C.c_uint),
                ("max_step_cost", C.c_uint64), ("max_elements", C.c_uint64),
                ("save_budget", C.c_uint64)]


class CeError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{_STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


_lib = None


def lib():
    """Load libconvein.so (once)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run paper_2401_03384_amd.build.build()")
        L = C.CDLL(LIB_PATH)
        vp, i64p = C.c_void_p, C.POINTER(C.c_int64)
        L.ce_expr_parse.argtypes = [C.c_char_p, C.c_int, C.POINTER(C.c_int), C.POINTER(i64p),
                                    C.POINTER(vp)]
        L.ce_expr_set_feature.argtypes = [vp, C.c_int]
        L.ce_expr_set_conv.argtypes = [vp, C.c_char_p, C.c_int]
        L.ce_expr_set_stride.argtypes = [vp, C.c_char_p, C.c_int]
        L.ce_expr_output_shape.argtypes = [vp, C.POINTER(C.c_int), i64p]
        L.ce_expr_destroy.argtypes = [vp]
        L.ce_expr_destroy.restype = None
        L.ce_plan_create.argtypes = [vp, C.c_int, C.c_int, C.c_uint, C.POINTER(vp)]
        L.ce_plan_create_limited.argtypes = [vp, C.c_int, C.c_int, C.c_uint, C.c_uint64, C.POINTER(vp)]
        L.ce_plan_create_ex.argtypes = [vp, C.POINTER(PlanOptions), C.POINTER(vp)]
        L.ce_plan_checkpoint.argtypes = [vp, C.POINTER(C.c_uint64), C.POINTER(C.c_uint64),
                                         C.POINTER(C.c_uint64)]
        L.ce_plan_create_with_path.argtypes = [vp, C.POINTER(C.c_int), C.c_int, C.c_int, C.c_uint,
                                               C.POINTER(vp)]
        L.ce_plan_num_steps.argtypes = [vp, C.POINTER(C.c_int)]
        L.ce_plan_step.argtypes = [vp, C.c_int, C.POINTER(C.c_uint64), C.POINTER(C.c_uint64),
                                   C.POINTER(C.c_uint64)]
        L.ce_plan_cost.argtypes = [vp, C.POINTER(C.c_uint64), C.POINTER(C.c_uint64)]
        L.ce_plan_left_to_right_cost.argtypes = [vp, C.POINTER(C.c_uint64)]
        L.ce_plan_workspace_size.argtypes = [vp, C.c_int, C.POINTER(C.c_size_t)]
        L.ce_plan_describe.argtypes = [vp]
        L.ce_plan_describe.restype = C.c_char_p
        L.ce_plan_destroy.argtypes = [vp]
        L.ce_plan_destroy.restype = None
        L.ce_forward.argtypes = [vp, C.POINTER(vp), vp, vp, C.c_size_t, vp]
        L.ce_backward.argtypes = [vp, C.POINTER(vp), vp, C.POINTER(vp), vp, C.c_size_t, vp]
        L.ce_backward_noalloc.argtypes = [vp, C.POINTER(vp), vp, C.POINTER(vp), vp]
        L.ce_timing_begin.argtypes = []
        L.ce_timing_begin_kernel.argtypes = [C.c_char_p]
        L.ce_timing_end.argtypes = [C.POINTER(C.c_int)]
        L.ce_timing_record.argtypes = [C.c_int, C.POINTER(C.c_char_p), C.POINTER(C.c_char_p),
                                       C.POINTER(C.c_float), C.POINTER(C.c_double),
                                       C.POINTER(C.c_double)]
        L.ce_last_error.restype = C.c_char_p
        L.ce_version.restype = C.c_char_p
        for name in ("ce_expr_parse", "ce_expr_set_feature", "ce_expr_set_conv", "ce_expr_set_stride",
    "ce_expr_output_shape",
                     "ce_plan_create", "ce_plan_create_limited", "ce_plan_create_ex", "ce_plan_checkpoint",
    "ce_plan_create_with_path",
                     "ce_plan_num_steps",
                     "ce_plan_step", "ce_plan_cost", "ce_plan_left_to_right_cost",
                     "ce_plan_workspace_size", "ce_forward", "ce_backward", "ce_timing_begin",
                     "ce_timing_begin_kernel", "ce_timing_end", "ce_timing_record"):
            getattr(L, name).restype = C.c_int
        _lib = L
    return _lib


def _check(status):
    if status != CE_OK:
        raise CeError(status, lib().ce_last_error().decode())


def ce_last_error() -> str:
    return lib().ce_last_error().decode()


def ce_version() -> str:
    return lib().ce_version().decode()


@functools.lru_cache(maxsize=256)
def _shape_args(shapes: tuple):
    """ctypes arrays for a tuple of shapes (kept alive by the cache)."""
    n = len(shapes)
    ranks = (C.c_int * n)(*[len(s) for s in shapes])
    bufs = [(C.c_int64 * max(1, len(s)))(*s) for s in shapes]
    dims = (C.POINTER(C.c_int64) * n)(*[C.cast(b, C.POINTER(C.c_int64)) for b in bufs])
    return n, ranks, bufs, dims


@functools.lru_cache(maxsize=256)
def _ptr_array(ptrs: tuple):
    """A void* array of the given addresses (None for a null pointer)."""
    return (C.c_void_p * len(ptrs))(*ptrs)


def ce_expr_parse(spec: str, shapes) -> int:
    n, ranks, _, dims = _shape_args(tuple(tuple(int(d) for d in s) for s in shapes))
    out = C.c_void_p()
    _check(lib().ce_expr_parse(spec.encode(), n, ranks, dims, C.byref(out)))
    return out.value


def ce_expr_set_feature(e: int, operand: int) -> None:
    _check(lib().ce_expr_set_feature(e, operand))


def ce_expr_set_conv(e: int, label: str, pad: int = CE_PAD_SAME_ZERO) -> None:
    _check(lib().ce_expr_set_conv(e, label.encode(), pad))


def ce_expr_set_stride(e: int, label: str, stride: int) -> None:
    _check(lib().ce_expr_set_stride(e, label.encode(), int(stride)))


def ce_expr_output_shape(e: int) -> tuple:
    rank = C.c_int()
    _check(lib().ce_expr_output_shape(e, C.byref(rank), None))
    dims = (C.c_int64 * max(1, rank.value))()
    _check(lib().ce_expr_output_shape(e, C.byref(rank), dims))
    return tuple(dims[i] for i in range(rank.value))


def ce_expr_destroy(e: int) -> None:
    lib().ce_expr_destroy(e)


def ce_plan_create(e: int, mode: int = CE_COST_FWD, dtype: int = CE_F32, flags: int = 0) -> int:
    out = C.c_void_p()
    _check(lib().ce_plan_create(e, mode, dtype, flags, C.byref(out)))
    return out.value


def ce_plan_create_limited(e: int, mode: int, dtype: int, flags: int, max_elements: int) -> int:
    out = C.c_void_p()
    _check(lib().ce_plan_create_limited(e, mode, dtype, flags, max_elements, C.byref(out)))
    return out.value


def ce_plan_create_ex(e: int, mode: int, dtype: int, flags: int, max_step_cost: int = 0,
                      max_elements: int = 0, save_budget: int = 0) -> int:
    opt = PlanOptions(mode, dtype, flags, max_step_cost, max_elements, save_budget)
    out = C.c_void_p()
    _check(lib().ce_plan_create_ex(e, C.byref(opt), C.byref(out)))
    return out.value


def ce_plan_checkpoint(p: int):
    """(saved step bitmask, saved bytes, recompute multiplications)."""
    a, b, c = C.c_uint64(), C.c_uint64(), C.c_uint64()
    _check(lib().ce_plan_checkpoint(p, C.byref(a), C.byref(b), C.byref(c)))
    return a.value, b.value, c.value


def ce_plan_create_with_path(e: int, pairs, dtype: int = CE_F32, flags: int = 0) -> int:
    flat = [int(x) for pr in pairs for x in pr]
    arr = (C.c_int * max(1, len(flat)))(*flat)
    out = C.c_void_p()
    _check(lib().ce_plan_create_with_path(e, arr, len(pairs), dtype, flags, C.byref(out)))
    return out.value


def ce_plan_num_steps(p: int) -> int:
    n = C.c_int()
    _check(lib().ce_plan_num_steps(p, C.byref(n)))
    return n.value


def ce_plan_step(p: int, i: int):
    a, b, m = C.c_uint64(), C.c_uint64(), C.c_uint64()
    _check(lib().ce_plan_step(p, i, C.byref(a), C.byref(b), C.byref(m)))
    return a.value, b.value, m.value


def ce_plan_cost(p: int):
    t, f = C.c_uint64(), C.c_uint64()
    _check(lib().ce_plan_cost(p, C.byref(t), C.byref(f)))
    return t.value, f.value


def ce_plan_left_to_right_cost(p: int) -> int:
    c = C.c_uint64()
    _check(lib().ce_plan_left_to_right_cost(p, C.byref(c)))
    return c.value


def ce_plan_workspace_size(p: int, for_backward: int) -> int:
    n = C.c_size_t()
    _check(lib().ce_plan_workspace_size(p, int(for_backward), C.byref(n)))
    return n.value


def ce_plan_describe(p: int) -> str:
    return lib().ce_plan_describe(p).decode()


def ce_plan_destroy(p: int) -> None:
    lib().ce_plan_destroy(p)


def ce_forward(p: int, in_ptrs, out_ptr: int, ws_ptr: int, ws_bytes: int, stream: int) -> None:
    arr = _ptr_array(tuple(in_ptrs))
    _check(lib().ce_forward(p, arr, out_ptr, ws_ptr or None, ws_bytes, stream or None))


def ce_backward(p: int, in_ptrs, dout_ptr: int, din_ptrs, ws_ptr: int, ws_bytes: int,
                stream: int) -> None:
    arr = _ptr_array(tuple(in_ptrs))
    darr = _ptr_array(tuple(d or None for d in din_ptrs))
    _check(lib().ce_backward(p, arr, dout_ptr, darr, ws_ptr or None, ws_bytes, stream or None))


def ce_backward_noalloc(p: int, in_ptrs, dout_ptr: int, din_ptrs, stream: int) -> None:
    arr = _ptr_array(tuple(in_ptrs))
    darr = _ptr_array(tuple(d or None for d in din_ptrs))
    _check(lib().ce_backward_noalloc(p, arr, dout_ptr, darr, stream or None))


def ce_timing_begin() -> None:
    _check(lib().ce_timing_begin())


def ce_timing_begin_kernel(kernel) -> None:
    _check(lib().ce_timing_begin_kernel(kernel.encode() if kernel else None))


def ce_timing_end() -> int:
    n = C.c_int()
    _check(lib().ce_timing_end(C.byref(n)))
    return n.value


def ce_timing_record(i: int):
    """(kernel, step, ms, algorithmic bytes, algorithmic flops) of record i."""
    k, s = C.c_char_p(), C.c_char_p()
    ms, by, fl = C.c_float(), C.c_double(), C.c_double()
    _check(lib().ce_timing_record(i, C.byref(k), C.byref(s), C.byref(ms), C.byref(by), C.byref(fl)))
    return k.value.decode(), s.value.decode(), ms.value, by.value, fl.value
