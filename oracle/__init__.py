"""Plain CPU oracle for the batch-reduce GEMM TPP, its fused epilogue (forward, and the inverse
activations of back-propagation), the Reduce TPP and the Transform TPP.

TEST INFRASTRUCTURE ONLY.  The product path (the HIP library and its Python binding) never
imports, links or calls anything in this package; only ``tests/``, the smoke check and the
benchmark's CPU-baseline leg do.  The arithmetic lives in ``oracle.c`` (plain C, fp64 loops);
this module only marshals numpy arrays into it.

Operand conventions (shared with nothing, stated here again): every 2D block is column-major
with a leading dimension; bf16 tensors are numpy ``uint16`` arrays holding the bit patterns,
fp32 tensors are ``float32`` arrays; strides and offsets count elements of the operand type.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_SRC = os.path.join(_HERE, "oracle.c")

F32, BF16 = 0, 1
STRIDE, OFFSET, ADDRESS = 0, 1, 2
EPI_BIAS, EPI_RELU, EPI_GELU_TANH = 1, 2, 4
EPI_RELU_INV, EPI_GELU_TANH_INV, EPI_SAVE_PREACT = 8, 16, 32
_EPI_BITS = {"bias": EPI_BIAS, "relu": EPI_RELU, "gelu_tanh": EPI_GELU_TANH,
             "relu_inv": EPI_RELU_INV, "gelu_tanh_inv": EPI_GELU_TANH_INV,
             "save_preact": EPI_SAVE_PREACT, "a_trans": 256, "b_trans": 512}
RED_SUM, RED_MUL, RED_MIN, RED_MAX = 0, 1, 2, 3
RED_BY_COLS, RED_BY_ROWS, RED_X, RED_X2 = 1, 2, 4, 8
TR_TRANSPOSE, TR_VNNI, TR_VNNI_TO_VNNI_T = 0, 1, 2

_DTYPES = {"f32": F32, "bf16": BF16}
_KINDS = {"stride": STRIDE, "offset": OFFSET, "address": ADDRESS}


def build(force: bool = False) -> str:
    """Compile oracle.c with gcc into liboracle.so next to it."""
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + f".tmp{os.getpid()}"
        subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall",
                        "-o", tmp, _SRC, "-lm"], check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


class _Desc(ctypes.Structure):
    _fields_ = [("m", ctypes.c_int32), ("n", ctypes.c_int32), ("k", ctypes.c_int32),
                ("lda", ctypes.c_int64), ("ldb", ctypes.c_int64), ("ldc", ctypes.c_int64),
                ("ab_type", ctypes.c_int32), ("c_type", ctypes.c_int32), ("beta", ctypes.c_double),
                ("kind", ctypes.c_int32), ("stride_a", ctypes.c_int64), ("stride_b", ctypes.c_int64),
                ("flags", ctypes.c_uint32)]


class _Grid(ctypes.Structure):
    _fields_ = [(f, ctypes.c_int64) for f in
                ("gm", "gn", "a_step_m", "b_step_n", "c_step_m", "c_step_n", "bias_step_m")]


_lib = None


def lib():
    """Load the oracle library (built on first use).  ORACLE_LIB_OVERRIDE names another build
    of it; the mutation tests use that to load copies with planted mistakes."""
    global _lib
    if _lib is None:
        override = os.environ.get("ORACLE_LIB_OVERRIDE")
        _lib = ctypes.CDLL(override if override else build())
        vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
        _lib.oracle_brgemm.restype = ctypes.c_int
        _lib.oracle_brgemm.argtypes = [ctypes.POINTER(_Desc), vp, vp, vp, vp, i64, vp, vp, vp, vp, vp]
        _lib.oracle_brgemm_batched.restype = ctypes.c_int
        _lib.oracle_brgemm_batched.argtypes = [ctypes.POINTER(_Desc), ctypes.POINTER(_Grid), i64,
                                               vp, vp, vp, vp, vp, vp, vp, vp, i64, vp, vp, vp, vp,
                                               vp, i64, vp, vp, ctypes.c_int]
        _lib.oracle_brgemm_batched_aux.restype = ctypes.c_int
        _lib.oracle_brgemm_batched_aux.argtypes = [ctypes.POINTER(_Desc), ctypes.POINTER(_Grid),
                                                   i64, vp, vp, vp, vp, vp, vp, vp, vp, vp, i64,
                                                   vp, vp, vp, vp, vp, i64, vp, vp, ctypes.c_int]
        _lib.oracle_reduce_batched.restype = ctypes.c_int
        _lib.oracle_reduce_batched.argtypes = [i32, i32, i64, i32, vp, i64, i64, i32,
                                               ctypes.c_uint32, vp, vp, i64]
        _lib.oracle_transform_batched.restype = ctypes.c_int
        _lib.oracle_transform_batched.argtypes = [i32, i32, i32, i64, i64, i32, i32, vp, i64, vp,
                                                  i64, i64]
        _lib.oracle_embedding_bag.restype = ctypes.c_int
        _lib.oracle_embedding_bag.argtypes = [i64, i32, i32, vp, i64, i64, vp, vp, i32, vp, i64,
                                              vp]
        _lib.oracle_eq_scores.restype = ctypes.c_int
        _lib.oracle_eq_scores.argtypes = [vp, i32, i32, vp]
        _lib.oracle_eq_plan.restype = ctypes.c_int
        _lib.oracle_eq_plan.argtypes = [vp, i32, i32, vp, vp, vp, vp]
        _lib.oracle_eq_eval.restype = ctypes.c_int
        _lib.oracle_eq_eval.argtypes = [vp, i32, i32, i32, i32, vp, i32, vp, i64, i32, vp]
        _lib.oracle_gelu_tanh_grad.restype = ctypes.c_double
        _lib.oracle_gelu_tanh_grad.argtypes = [ctypes.c_double]
        _lib.oracle_reduce.restype = ctypes.c_int
        _lib.oracle_reduce.argtypes = [i32, i32, i64, i32, vp, i32, ctypes.c_uint32, vp, vp]
        _lib.oracle_transform.restype = ctypes.c_int
        _lib.oracle_transform.argtypes = [i32, i32, i32, i64, i64, i32, i32, vp, vp]
        _lib.oracle_f32_to_bf16.restype = ctypes.c_uint16
        _lib.oracle_f32_to_bf16.argtypes = [ctypes.c_float]
        _lib.oracle_f32_to_bf16_array.restype = None
        _lib.oracle_f32_to_bf16_array.argtypes = [vp, vp, i64]
        _lib.oracle_bf16_to_f32.restype = ctypes.c_float
        _lib.oracle_bf16_to_f32.argtypes = [ctypes.c_uint16]
        _lib.oracle_gelu_tanh.restype = ctypes.c_double
        _lib.oracle_gelu_tanh.argtypes = [ctypes.c_double]
        _lib.oracle_max_threads.restype = ctypes.c_int
    return _lib


@dataclass
class Desc:
    """BRGEMM problem description (the dispatch-time fields of the TPP)."""
    m: int
    n: int
    k: int
    lda: int
    ldb: int
    ldc: int
    ab_type: str = "bf16"
    c_type: str = "f32"
    beta: float = 0.0
    kind: str = "stride"
    stride_a: int = 0
    stride_b: int = 0
    # subset of {"bias", "relu", "gelu_tanh", "relu_inv", "gelu_tanh_inv", "save_preact"}
    flags: set = field(default_factory=set)

    def _c(self) -> _Desc:
        fl = 0
        for f in self.flags:
            fl |= _EPI_BITS[f]
        return _Desc(self.m, self.n, self.k, self.lda, self.ldb, self.ldc, _DTYPES[self.ab_type],
                     _DTYPES[self.c_type], float(self.beta), _KINDS[self.kind], self.stride_a,
                     self.stride_b, fl)


def _ptr(x):
    return None if x is None else x.ctypes.data


def _check_dtype(arr, dt, name):
    want = np.float32 if dt == "f32" else np.uint16
    if arr is not None and arr.dtype != want:
        raise TypeError(f"{name}: expected {np.dtype(want).name}, got {arr.dtype}")


def _as_i64(x):
    return None if x is None else np.ascontiguousarray(x, dtype=np.int64)


def _pointer_list(base: np.ndarray, elem_offsets, es: int):
    """Host addresses base + off*es for each element offset: the address variant's lists."""
    offs = np.asarray(elem_offsets, dtype=np.int64)
    if offs.size and (offs.min() < 0 or offs.max() >= base.size):
        raise ValueError("pointer list leaves the pool")
    return (np.uint64(base.ctypes.data) + offs.astype(np.uint64) * np.uint64(es)).astype(np.uint64)


def brgemm_batched(desc: Desc, a, b, c, bias=None, *, grid=None, G=1, a_off=None, b_off=None,
                   c_off=None, bias_off=None, count=0, offs_a=None, offs_b=None, begin=None,
                   idx_a=None, idx_b=None, sel=None, want_ref64=False, nthreads=0, aux=None):
    """Run G BRGEMM instances in place on ``c``.

    grid: dict with gm, gn, a_step_m, b_step_n, c_step_m, c_step_n, bias_step_m (strided form),
    or None for the explicit per-instance offset arrays.  Address variant: ``idx_a``/``idx_b`` are
    element offsets into the pools ``a``/``b``; they become host addresses here, and ``begin``
    (G+1 entries) splits them into per-instance lists.  Returns the unrounded fp64 results of the
    selected instances when ``want_ref64``.  ``aux``: the tensor of C's type and layout that
    "save_preact" writes and "relu_inv" / "gelu_tanh_inv" read (in place).
    """
    _check_dtype(a, desc.ab_type, "a")
    _check_dtype(b, desc.ab_type, "b")
    _check_dtype(c, desc.c_type, "c")
    _check_dtype(aux, desc.c_type, "aux")
    if aux is not None and (aux.shape != c.shape or not aux.flags.c_contiguous):
        raise ValueError("aux must be a contiguous array shaped as c")
    if bias is not None and bias.dtype != np.float32:
        raise TypeError("bias must be float32")
    for arr in (a, b, c, bias):
        if arr is not None and not arr.flags.c_contiguous:
            raise ValueError("arrays must be contiguous")
    d = desc._c()
    g = None
    if grid is not None:
        g = _Grid(*(int(grid[f]) for f in ("gm", "gn", "a_step_m", "b_step_n", "c_step_m",
                                           "c_step_n", "bias_step_m")))
    a_off, b_off, c_off, bias_off = map(_as_i64, (a_off, b_off, c_off, bias_off))
    offs_a, offs_b, begin = map(_as_i64, (offs_a, offs_b, begin))
    ptrs_a = ptrs_b = None
    es = 4 if desc.ab_type == "f32" else 2
    if desc.kind == "address":
        ptrs_a = _pointer_list(a, idx_a, es)
        ptrs_b = _pointer_list(b, idx_b, es)
        if begin is None:
            raise ValueError("address variant needs begin[]")
    sel_arr = None if sel is None else _as_i64(sel)
    n_sel = G if sel_arr is None else len(sel_arr)
    ref = np.empty((n_sel, desc.n, desc.m), dtype=np.float64) if want_ref64 else None
    rc = lib().oracle_brgemm_batched_aux(
        ctypes.byref(d), ctypes.byref(g) if g is not None else None, G,
        _ptr(a_off), _ptr(b_off), _ptr(c_off), _ptr(bias_off),
        _ptr(a) if desc.kind != "address" else None, _ptr(b) if desc.kind != "address" else None,
        _ptr(c), _ptr(aux), _ptr(bias), count, _ptr(offs_a), _ptr(offs_b), _ptr(begin), _ptr(ptrs_a),
        _ptr(ptrs_b), n_sel, _ptr(sel_arr), _ptr(ref), nthreads)
    if rc != 0:
        raise ValueError("oracle_brgemm_batched rejected its arguments")
    return ref


def brgemm(desc: Desc, a, b, c, bias=None, *, count=0, offs_a=None, offs_b=None, idx_a=None,
           idx_b=None, want_ref64=False):
    """One BRGEMM call (the paper's call API) on host arrays, in place on ``c``."""
    _check_dtype(a, desc.ab_type, "a")
    _check_dtype(b, desc.ab_type, "b")
    _check_dtype(c, desc.c_type, "c")
    d = desc._c()
    offs_a, offs_b = map(_as_i64, (offs_a, offs_b))
    ptrs_a = ptrs_b = None
    es = 4 if desc.ab_type == "f32" else 2
    if desc.kind == "address":
        ptrs_a = _pointer_list(a, idx_a, es)
        ptrs_b = _pointer_list(b, idx_b, es)
    ref = np.empty((desc.n, desc.m), dtype=np.float64) if want_ref64 else None
    rc = lib().oracle_brgemm(ctypes.byref(d), _ptr(a) if desc.kind != "address" else None,
                             _ptr(b) if desc.kind != "address" else None, _ptr(c), _ptr(bias),
                             count, _ptr(offs_a), _ptr(offs_b), _ptr(ptrs_a), _ptr(ptrs_b), _ptr(ref))
    if rc != 0:
        raise ValueError("oracle_brgemm rejected its arguments")
    return ref


def reduce(x, m: int, n: int, ld: int, in_type: str, op: str, by: str, want=("x",)):
    """Reduce TPP: op in sum/mul/min/max, by in cols/rows, want subset of {"x", "x2"}."""
    _check_dtype(x, in_type, "x")
    ops = {"sum": RED_SUM, "mul": RED_MUL, "min": RED_MIN, "max": RED_MAX}
    flags = (RED_BY_COLS if by == "cols" else RED_BY_ROWS)
    flags |= (RED_X if "x" in want else 0) | (RED_X2 if "x2" in want else 0)
    outn = m if by == "cols" else n
    ox = np.empty(outn, dtype=np.float64) if "x" in want else None
    ox2 = np.empty(outn, dtype=np.float64) if "x2" in want else None
    rc = lib().oracle_reduce(m, n, ld, _DTYPES[in_type], _ptr(x), ops[op], flags, _ptr(ox), _ptr(ox2))
    if rc != 0:
        raise ValueError("oracle_reduce rejected its arguments")
    return ox, ox2


def reduce_batched(x, m: int, n: int, ld: int, in_type: str, G: int, in_stride: int, op: str,
                   by: str, want=("x",), out_stride=None):
    """G Reduce TPP calls on blocks ``in_stride`` elements apart; returns (G x outputs) arrays
    (the outputs of call g start g*out_stride apart; default: packed)."""
    _check_dtype(x, in_type, "x")
    ops = {"sum": RED_SUM, "mul": RED_MUL, "min": RED_MIN, "max": RED_MAX}
    flags = (RED_BY_COLS if by == "cols" else RED_BY_ROWS)
    flags |= (RED_X if "x" in want else 0) | (RED_X2 if "x2" in want else 0)
    outn = m if by == "cols" else n
    ostride = outn if out_stride is None else out_stride
    size = (G - 1) * ostride + outn if G > 0 else 0
    ox = np.zeros(size, dtype=np.float64) if "x" in want else None
    ox2 = np.zeros(size, dtype=np.float64) if "x2" in want else None
    rc = lib().oracle_reduce_batched(m, n, ld, _DTYPES[in_type], _ptr(x), G, in_stride, ops[op],
                                     flags, _ptr(ox), _ptr(ox2), ostride)
    if rc != 0:
        raise ValueError("oracle_reduce_batched rejected its arguments")
    return ox, ox2


_TR_KINDS = {"transpose": TR_TRANSPOSE, "vnni": TR_VNNI, "vnni_t": TR_VNNI_TO_VNNI_T}


def transform_out_len(kind: str, m: int, n: int, ld_out: int, alpha: int) -> int:
    """Elements of an output buffer that holds every position the transformation defines."""
    if m == 0 or n == 0:
        return 0
    groups = {"transpose": m, "vnni": -(-n // alpha), "vnni_t": -(-m // alpha)}[kind]
    return ld_out * groups


def transform(kind: str, m: int, n: int, ld_in: int, ld_out: int, dtype: str, alpha: int,
              x: np.ndarray, out: np.ndarray) -> np.ndarray:
    """Transform TPP (kind "transpose", "vnni" or "vnni_t") from host array x into host array
    out, in place; positions the transformation does not define keep their values."""
    _check_dtype(x, dtype, "x")
    _check_dtype(out, dtype, "out")
    es = 4 if dtype == "f32" else 2
    rc = lib().oracle_transform(_TR_KINDS[kind], m, n, ld_in, ld_out, es, alpha, _ptr(x), _ptr(out))
    if rc != 0:
        raise ValueError("oracle_transform rejected its arguments")
    return out


def transform_batched(kind: str, m: int, n: int, ld_in: int, ld_out: int, dtype: str,
                      alpha: int, x: np.ndarray, in_stride: int, out: np.ndarray,
                      out_stride: int, G: int) -> np.ndarray:
    """G Transform TPP calls: block g of x (``in_stride`` elements apart) into block g of out
    (``out_stride`` apart), in place on out."""
    _check_dtype(x, dtype, "x")
    _check_dtype(out, dtype, "out")
    es = 4 if dtype == "f32" else 2
    rc = lib().oracle_transform_batched(_TR_KINDS[kind], m, n, ld_in, ld_out, es, alpha, _ptr(x),
                                        in_stride, _ptr(out), out_stride, G)
    if rc != 0:
        raise ValueError("oracle_transform_batched rejected its arguments")
    return out


def f32_to_bf16(x: float) -> int:
    return int(lib().oracle_f32_to_bf16(float(x)))


def f32_to_bf16_array(x: np.ndarray) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, dtype=np.uint16)
    lib().oracle_f32_to_bf16_array(_ptr(x), _ptr(out), x.size)
    return out


def bf16_to_f32(h: int) -> float:
    return float(lib().oracle_bf16_to_f32(int(h)))


def gelu_tanh(x: float) -> float:
    return float(lib().oracle_gelu_tanh(float(x)))


def embedding_bag(w: np.ndarray, M: int, E: int, ldw: int, w_type: str, begin, idx,
                  out: np.ndarray, ldo: int, out_type: str, want_ref64=False):
    """Sparse embedding gather-reduce (Alg. 5) into ``out`` (in place); returns the unrounded
    sums (n_bags x E) when ``want_ref64``."""
    _check_dtype(w, w_type, "w")
    _check_dtype(out, out_type, "out")
    begin, idx = _as_i64(begin), _as_i64(idx)
    n_bags = len(begin) - 1
    ref = np.empty((n_bags, E), dtype=np.float64) if want_ref64 else None
    rc = lib().oracle_embedding_bag(M, E, _DTYPES[w_type], _ptr(w), ldw, n_bags, _ptr(begin),
                                    _ptr(idx), _DTYPES[out_type], _ptr(out), ldo, _ptr(ref))
    if rc != 0:
        raise ValueError("oracle_embedding_bag rejected its arguments")
    return ref


# ---- TPP matrix equations (Sec. 4) ----------------------------------------------------------
EQ_OPS = {"identity": 0, "neg": 1, "exp": 2, "tanh": 3, "relu": 4, "gelu_tanh": 5, "sqrt": 6,
          "rcp": 7, "square": 8, "sigmoid": 9, "add": 16, "sub": 17, "mul": 18, "div": 19,
          "max": 20, "min": 21, "muladd": 32}
EQ_BCAST = {"none": 0, "col": 1, "row": 2, "scalar": 3}


class _EqNode(ctypes.Structure):
    _fields_ = [("arity", ctypes.c_int32), ("op", ctypes.c_int32),
                ("child", ctypes.c_int32 * 3), ("leaf", ctypes.c_int32)]


class _EqLeaf(ctypes.Structure):
    _fields_ = [("ptr", ctypes.c_void_p), ("ld", ctypes.c_int64), ("dtype", ctypes.c_int32),
                ("bcast", ctypes.c_int32)]


def _eq_nodes(nodes):
    """nodes: list of ("leaf", leaf_index) or (op_name, child, ...) tuples."""
    arr = (_EqNode * len(nodes))()
    for i, nd in enumerate(nodes):
        if nd[0] == "leaf":
            arr[i].arity, arr[i].op, arr[i].leaf = 0, 0, nd[1]
            arr[i].child[:] = [-1, -1, -1]
        else:
            kids = list(nd[1:])
            arr[i].arity, arr[i].op, arr[i].leaf = len(kids), EQ_OPS[nd[0]], -1
            arr[i].child[:] = kids + [-1] * (3 - len(kids))
    return arr


def eq_scores(nodes, root):
    """Alg. 3: register score of every node."""
    arr = _eq_nodes(nodes)
    sc = (ctypes.c_int32 * len(nodes))()
    if lib().oracle_eq_scores(arr, len(nodes), root, sc) != 0:
        raise ValueError("malformed equation tree")
    return list(sc)


def eq_plan(nodes, root):
    """Alg. 4: (timestamps, tmp ids, number of tmps) of every node (leaves -1)."""
    arr = _eq_nodes(nodes)
    n = len(nodes)
    sc = (ctypes.c_int32 * n)()
    if lib().oracle_eq_scores(arr, n, root, sc) != 0:
        raise ValueError("malformed equation tree")
    ts, tm, nt = (ctypes.c_int32 * n)(), (ctypes.c_int32 * n)(), ctypes.c_int32()
    if lib().oracle_eq_plan(arr, n, root, sc, ts, tm, ctypes.byref(nt)) != 0:
        raise ValueError("malformed equation tree")
    return list(ts), list(tm), nt.value


def eq_eval(nodes, root, m, n, leaves, out, ldo, out_type, want_ref64=False):
    """The equation's value on an m x n output (in place on ``out``).  leaves: list of
    (array, ld, dtype, bcast) with bcast in "none"/"col"/"row"/"scalar"."""
    arr = _eq_nodes(nodes)
    lv = (_EqLeaf * max(1, len(leaves)))()
    for i, (a, ld, dt, bc) in enumerate(leaves):
        _check_dtype(a, dt, f"leaf {i}")
        lv[i].ptr, lv[i].ld, lv[i].dtype, lv[i].bcast = a.ctypes.data, ld, _DTYPES[dt], EQ_BCAST[bc]
    _check_dtype(out, out_type, "out")
    ref = np.empty((n, m), dtype=np.float64) if want_ref64 else None
    rc = lib().oracle_eq_eval(arr, len(nodes), root, m, n, lv, len(leaves), _ptr(out), ldo,
                              _DTYPES[out_type], _ptr(ref))
    if rc != 0:
        raise ValueError("oracle_eq_eval rejected its arguments")
    return ref


def gelu_tanh_grad(x: float) -> float:
    return float(lib().oracle_gelu_tanh_grad(float(x)))


def max_threads() -> int:
    return int(lib().oracle_max_threads())
