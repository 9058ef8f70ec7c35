"""MI355X (gfx950) TPP library: thin Python binding of the C ABI in include/tpp_brgemm.h,
include/tpp_transform.h, include/tpp_embedding.h and include/tpp_equation.h.

Argument marshalling only: every step of the computation runs in the HIP kernels of
``libtpp_mi355x.so``.  The functions keep the C names; pointers are plain integers (device
addresses) or objects with ``data_ptr()`` (torch tensors), streams are integers (a hipStream_t)
or None for the default stream.  A non-OK status raises :class:`TppError`.

The library must have been built (``__graft_entry__.build()`` or
``python paper_2104_05755_amd/build.py``); importing this package without it raises ImportError.
"""
from __future__ import annotations

import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libtpp_mi355x.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build the HIP library first "
                      "(python paper_2104_05755_amd/build.py)")

_lib = ctypes.CDLL(LIB_PATH)

# ---- constants (mirroring include/tpp_brgemm.h) ---------------------------------------------
TPP_OK, TPP_ERR_INVALID_ARG, TPP_ERR_UNSUPPORTED, TPP_ERR_HIP, TPP_ERR_NO_MEMORY = 0, -1, -2, -4, -5
TPP_DT_F32, TPP_DT_BF16 = 0, 1
TPP_BR_STRIDE, TPP_BR_OFFSET, TPP_BR_ADDRESS = 0, 1, 2
TPP_EPI_BIAS, TPP_EPI_RELU, TPP_EPI_GELU_TANH = 1, 2, 4
TPP_EPI_RELU_INV, TPP_EPI_GELU_TANH_INV, TPP_EPI_SAVE_PREACT = 8, 16, 32
TPP_LAYOUT_A_TRANS, TPP_LAYOUT_B_TRANS = 256, 512
TPP_RED_SUM, TPP_RED_MUL, TPP_RED_MIN, TPP_RED_MAX = 0, 1, 2, 3
TPP_RED_BY_COLS, TPP_RED_BY_ROWS, TPP_RED_X, TPP_RED_X2 = 1, 2, 4, 8
TPP_TR_TRANSPOSE, TPP_TR_VNNI, TPP_TR_VNNI_TO_VNNI_T = 0, 1, 2

_c_void_p, _i64, _i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32


class tpp_brgemm_desc(ctypes.Structure):
    _fields_ = [("m", _i32), ("n", _i32), ("k", _i32),
                ("lda", _i64), ("ldb", _i64), ("ldc", _i64),
                ("a_type", _i32), ("b_type", _i32), ("c_type", _i32), ("comp_type", _i32),
                ("beta", ctypes.c_float), ("kind", _i32),
                ("stride_a", _i64), ("stride_b", _i64), ("flags", ctypes.c_uint32)]


class tpp_grid_strided(ctypes.Structure):
    _fields_ = [(f, _i64) for f in ("gm", "gn", "a_step_m", "b_step_n", "c_step_m", "c_step_n",
                                    "bias_step_m")]


class TppError(RuntimeError):
    def __init__(self, status: int, where: str):
        msg = _lib.tpp_last_error_message().decode()
        super().__init__(f"{where}: {_lib.tpp_status_string(status).decode()} ({msg})")
        self.status = status


def _sig(name, restype, *argtypes):
    f = getattr(_lib, name)
    f.restype = restype
    f.argtypes = list(argtypes)
    return f


_sig("tpp_status_string", ctypes.c_char_p, _i32)
_sig("tpp_last_error_message", ctypes.c_char_p)
_sig("tpp_brgemm_dispatch", _i32, ctypes.POINTER(tpp_brgemm_desc), ctypes.POINTER(_c_void_p))
_sig("tpp_brgemm_execute_stride", _i32, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p,
     _i64, _c_void_p)
_sig("tpp_brgemm_execute_offset", _i32, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p,
     _c_void_p, _c_void_p, _i64, _c_void_p)
_sig("tpp_brgemm_execute_address", _i32, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p,
     _i64, _c_void_p)
_sig("tpp_brgemm_execute_batched", _i32, _c_void_p, ctypes.POINTER(tpp_grid_strided), _i64,
     _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p,
     _i64, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p)
_sig("tpp_brgemm_execute_batched_aux", _i32, _c_void_p, ctypes.POINTER(tpp_grid_strided), _i64,
     _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p,
     _c_void_p, _i64, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p)
_sig("tpp_brgemm_execute_batched_noalloc", _i32, _c_void_p, ctypes.POINTER(tpp_grid_strided), _i64,
     _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p,
     _i64, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p)
_sig("tpp_brgemm_release", None, _c_void_p)
_sig("tpp_brgemm_describe", _i32, _c_void_p, ctypes.c_char_p, ctypes.c_size_t)
_sig("tpp_brgemm_describe_launch", _i32, _c_void_p, ctypes.POINTER(tpp_grid_strided), _i64,
     _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p,
     _i64, _c_void_p, _c_void_p, _c_void_p, _c_void_p, _c_void_p, ctypes.c_char_p,
     ctypes.c_size_t)
_sig("tpp_reduce", _i32, _i32, _i32, _i64, _i32, _c_void_p, _i32, ctypes.c_uint32, _c_void_p,
     _c_void_p, _c_void_p)
_sig("tpp_transform", _i32, _i32, _i32, _i32, _i64, _i64, _i32, _i32, _c_void_p, _c_void_p,
     _c_void_p)
class tpp_eq_node(ctypes.Structure):
    _fields_ = [("arity", _i32), ("op", _i32), ("child", _i32 * 3), ("leaf", _i32)]


class tpp_eq_plan_node(ctypes.Structure):
    _fields_ = [("score", _i32), ("timestamp", _i32), ("tmp", _i32)]


class tpp_eq_arg(ctypes.Structure):
    _fields_ = [("ptr", _c_void_p), ("ld", _i64), ("dtype", _i32), ("bcast", _i32)]


TPP_EQ_OPS = {"identity": 0, "neg": 1, "exp": 2, "tanh": 3, "relu": 4, "gelu_tanh": 5, "sqrt": 6,
              "rcp": 7, "square": 8, "sigmoid": 9, "add": 16, "sub": 17, "mul": 18, "div": 19,
              "max": 20, "min": 21, "muladd": 32}
TPP_BC = {"none": 0, "col": 1, "row": 2, "scalar": 3}

_sig("tpp_equation_plan", _i32, ctypes.POINTER(tpp_eq_node), _i32, _i32,
     ctypes.POINTER(tpp_eq_plan_node), ctypes.POINTER(_i32))
_sig("tpp_equation_execute", _i32, ctypes.POINTER(tpp_eq_node), _i32, _i32, _i32, _i32,
     ctypes.POINTER(tpp_eq_arg), _i32, _c_void_p, _i64, _i32, _c_void_p)
_sig("tpp_embedding_bag", _i32, _i64, _i32, _i32, _c_void_p, _i64, _i64, _c_void_p, _c_void_p,
     _i32, _c_void_p, _i64, _c_void_p)
_sig("tpp_reduce_batched", _i32, _i32, _i32, _i64, _i32, _c_void_p, _i64, _i64, _i32,
     ctypes.c_uint32, _c_void_p, _c_void_p, _i64, _c_void_p)
_sig("tpp_transform_batched", _i32, _i32, _i32, _i32, _i64, _i64, _i32, _i32, _c_void_p, _i64,
     _c_void_p, _i64, _i64, _c_void_p)


def _p(x):
    """Device address of x: None, an int, or an object with data_ptr()."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _check(status: int, where: str):
    if status != TPP_OK:
        raise TppError(status, where)


def current_stream() -> int:
    """hipStream_t of torch's current stream on the current device (torch is the memory and
    stream provider; the library itself does not depend on it)."""
    import torch
    return torch.cuda.current_stream().cuda_stream


def tpp_brgemm_dispatch(desc: tpp_brgemm_desc) -> int:
    h = _c_void_p()
    _check(_lib.tpp_brgemm_dispatch(ctypes.byref(desc), ctypes.byref(h)), "tpp_brgemm_dispatch")
    return h.value


def tpp_brgemm_execute_stride(h, a, b, c, bias, count, stream=None):
    _check(_lib.tpp_brgemm_execute_stride(h, _p(a), _p(b), _p(c), _p(bias), count, stream),
           "tpp_brgemm_execute_stride")


def tpp_brgemm_execute_offset(h, a, b, offs_a, offs_b, c, bias, count, stream=None):
    _check(_lib.tpp_brgemm_execute_offset(h, _p(a), _p(b), _p(offs_a), _p(offs_b), _p(c),
                                          _p(bias), count, stream), "tpp_brgemm_execute_offset")


def tpp_brgemm_execute_address(h, ptrs_a, ptrs_b, c, bias, count, stream=None):
    _check(_lib.tpp_brgemm_execute_address(h, _p(ptrs_a), _p(ptrs_b), _p(c), _p(bias), count,
                                           stream), "tpp_brgemm_execute_address")


def _grid(grid):
    if grid is None or isinstance(grid, tpp_grid_strided):
        return grid
    return tpp_grid_strided(*(int(grid[f]) for f in ("gm", "gn", "a_step_m", "b_step_n",
                                                     "c_step_m", "c_step_n", "bias_step_m")))


def tpp_brgemm_execute_batched(h, grid, G, a_off, b_off, c_off, bias_off, a, b, c, bias, count,
                               offs_a, offs_b, begin, ptrs_a, ptrs_b, stream=None):
    """grid: tpp_grid_strided, a dict with its fields, or None (explicit offset arrays)."""
    g = _grid(grid)
    _check(_lib.tpp_brgemm_execute_batched(
        h, ctypes.byref(g) if g is not None else None, G, _p(a_off), _p(b_off), _p(c_off),
        _p(bias_off), _p(a), _p(b), _p(c), _p(bias), count, _p(offs_a), _p(offs_b), _p(begin),
        _p(ptrs_a), _p(ptrs_b), stream), "tpp_brgemm_execute_batched")


def tpp_brgemm_execute_batched_aux(h, grid, G, a_off, b_off, c_off, bias_off, a, b, c, aux, bias,
                                   count, offs_a, offs_b, begin, ptrs_a, ptrs_b, stream=None):
    """tpp_brgemm_execute_batched with the aux tensor (shaped and laid out as c)."""
    g = _grid(grid)
    _check(_lib.tpp_brgemm_execute_batched_aux(
        h, ctypes.byref(g) if g is not None else None, G, _p(a_off), _p(b_off), _p(c_off),
        _p(bias_off), _p(a), _p(b), _p(c), _p(aux), _p(bias), count, _p(offs_a), _p(offs_b),
        _p(begin), _p(ptrs_a), _p(ptrs_b), stream), "tpp_brgemm_execute_batched_aux")


def tpp_brgemm_execute_batched_noalloc(h, grid, G, a_off, b_off, c_off, bias_off, a, b, c, bias,
                                       count, offs_a, offs_b, begin, ptrs_a, ptrs_b, stream=None):
    """tpp_brgemm_execute_batched without any device allocation (the library's per-GPU scratch
    array holds a split reduction's partial tiles)."""
    g = _grid(grid)
    _check(_lib.tpp_brgemm_execute_batched_noalloc(
        h, ctypes.byref(g) if g is not None else None, G, _p(a_off), _p(b_off), _p(c_off),
        _p(bias_off), _p(a), _p(b), _p(c), _p(bias), count, _p(offs_a), _p(offs_b), _p(begin),
        _p(ptrs_a), _p(ptrs_b), stream), "tpp_brgemm_execute_batched_noalloc")


def tpp_brgemm_describe_launch(h, grid, G, a_off, b_off, c_off, bias_off, a, b, c, bias, count,
                               offs_a, offs_b, begin, ptrs_a, ptrs_b) -> str:
    """Names of the kernels tpp_brgemm_execute_batched would launch with these arguments (as the
    profiler names them).  Only the pointers' values are looked at: plain ints will do."""
    g = _grid(grid)
    buf = ctypes.create_string_buffer(512)
    _check(_lib.tpp_brgemm_describe_launch(
        h, ctypes.byref(g) if g is not None else None, G, _p(a_off), _p(b_off), _p(c_off),
        _p(bias_off), _p(a), _p(b), _p(c), _p(bias), count, _p(offs_a), _p(offs_b), _p(begin),
        _p(ptrs_a), _p(ptrs_b), buf, 512), "tpp_brgemm_describe_launch")
    return buf.value.decode()


def tpp_brgemm_release(h):
    _lib.tpp_brgemm_release(h)


def tpp_brgemm_describe(h) -> str:
    buf = ctypes.create_string_buffer(256)
    _check(_lib.tpp_brgemm_describe(h, buf, 256), "tpp_brgemm_describe")
    return buf.value.decode()


def tpp_reduce(m, n, ld, in_type, x, op, flags, out_x, out_x2, stream=None):
    _check(_lib.tpp_reduce(m, n, ld, in_type, _p(x), op, flags, _p(out_x), _p(out_x2), stream),
           "tpp_reduce")


def tpp_transform(kind, m, n, ld_in, ld_out, dtype, alpha, x, out, stream=None):
    _check(_lib.tpp_transform(kind, m, n, ld_in, ld_out, dtype, alpha, _p(x), _p(out), stream),
           "tpp_transform")


def tpp_reduce_batched(m, n, ld, in_type, x, G, in_stride, op, flags, out_x, out_x2, out_stride,
                       stream=None):
    _check(_lib.tpp_reduce_batched(m, n, ld, in_type, _p(x), G, in_stride, op, flags, _p(out_x),
                                   _p(out_x2), out_stride, stream), "tpp_reduce_batched")


def tpp_transform_batched(kind, m, n, ld_in, ld_out, dtype, alpha, x, in_stride, out, out_stride,
                          G, stream=None):
    _check(_lib.tpp_transform_batched(kind, m, n, ld_in, ld_out, dtype, alpha, _p(x), in_stride,
                                      _p(out), out_stride, G, stream), "tpp_transform_batched")


def tpp_embedding_bag(M, E, w_type, W, ldw, n_bags, begin, idx, out_type, out, ldo, stream=None):
    _check(_lib.tpp_embedding_bag(M, E, w_type, _p(W), ldw, n_bags, _p(begin), _p(idx), out_type,
                                  _p(out), ldo, stream), "tpp_embedding_bag")


def eq_nodes(nodes):
    """An equation tree from ("leaf", argument index) and (op name, child, ...) tuples."""
    arr = (tpp_eq_node * len(nodes))()
    for i, nd in enumerate(nodes):
        if nd[0] == "leaf":
            arr[i].arity, arr[i].op, arr[i].leaf = 0, 0, nd[1]
            arr[i].child[:] = [-1, -1, -1]
        else:
            kids = list(nd[1:])
            arr[i].arity, arr[i].op, arr[i].leaf = len(kids), TPP_EQ_OPS[nd[0]], -1
            arr[i].child[:] = kids + [-1] * (3 - len(kids))
    return arr


def tpp_equation_plan(nodes, root):
    """(scores, timestamps, tmp ids, number of tmps) of an equation tree (host only)."""
    arr = eq_nodes(nodes)
    plan = (tpp_eq_plan_node * len(nodes))()
    nt = _i32()
    _check(_lib.tpp_equation_plan(arr, len(nodes), root, plan, ctypes.byref(nt)),
           "tpp_equation_plan")
    return ([p.score for p in plan], [p.timestamp for p in plan], [p.tmp for p in plan], nt.value)


def tpp_equation_execute(nodes, root, m, n, args, out, ldo, out_type, stream=None):
    """args: list of (tensor or address, ld, dtype code, broadcast name)."""
    arr = eq_nodes(nodes)
    ga = (tpp_eq_arg * max(1, len(args)))()
    for i, (x, ld, dt, bc) in enumerate(args):
        ga[i].ptr, ga[i].ld, ga[i].dtype, ga[i].bcast = _p(x), ld, dt, TPP_BC[bc]
    _check(_lib.tpp_equation_execute(arr, len(nodes), root, m, n, ga, len(args), _p(out), ldo,
                                     out_type, stream), "tpp_equation_execute")


def tpp_status_string(s: int) -> str:
    return _lib.tpp_status_string(s).decode()


def tpp_last_error_message() -> str:
    return _lib.tpp_last_error_message().decode()


def make_desc(m, n, k, lda, ldb, ldc, ab_type="bf16", c_type="f32", beta=0.0, kind="stride",
              stride_a=0, stride_b=0, flags=()) -> tpp_brgemm_desc:
    """Convenience: a descriptor from readable names (dtype "f32"/"bf16", kind
    "stride"/"offset"/"address", flags from {"bias", "relu", "gelu_tanh", "relu_inv",
    "gelu_tanh_inv", "save_preact"} and the layout flags "a_trans", "b_trans")."""
    dt = {"f32": TPP_DT_F32, "bf16": TPP_DT_BF16}
    kd = {"stride": TPP_BR_STRIDE, "offset": TPP_BR_OFFSET, "address": TPP_BR_ADDRESS}
    fl = {"bias": TPP_EPI_BIAS, "relu": TPP_EPI_RELU, "gelu_tanh": TPP_EPI_GELU_TANH,
          "relu_inv": TPP_EPI_RELU_INV, "gelu_tanh_inv": TPP_EPI_GELU_TANH_INV,
          "save_preact": TPP_EPI_SAVE_PREACT, "a_trans": TPP_LAYOUT_A_TRANS,
          "b_trans": TPP_LAYOUT_B_TRANS}
    bits = 0
    for f in flags:
        bits |= fl[f]
    return tpp_brgemm_desc(m, n, k, lda, ldb, ldc, dt[ab_type], dt[ab_type], dt[c_type],
                           TPP_DT_F32, float(beta), kd[kind], stride_a, stride_b, bits)
