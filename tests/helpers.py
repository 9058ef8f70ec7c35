"""Shared test helpers: run a workload call through the oracle, compare results."""
from __future__ import annotations

import numpy as np

import oracle
from workloads import (Call, EmbeddingStep, EquationStep, ReduceStep, TransformStep, Workload,
                       bf16_values)


def oracle_desc(call: Call) -> oracle.Desc:
    return oracle.Desc(call.m, call.n, call.k, call.lda, call.ldb, call.ldc, call.ab_type,
                       call.c_type, call.beta, call.kind, call.stride_a, call.stride_b,
                       set(call.flags))


def run_call_oracle(call: Call, arrs: dict, sel=None, want_ref64=False, nthreads=0):
    """One BRGEMM call through the oracle, in place on arrs[call.c] (and arrs[call.aux])."""
    return oracle.brgemm_batched(
        oracle_desc(call), arrs[call.a], arrs[call.b], arrs[call.c],
        arrs[call.bias] if call.bias else None, grid=call.grid, G=call.G,
        a_off=call.a_off, b_off=call.b_off, c_off=call.c_off, bias_off=call.bias_off,
        count=call.count, offs_a=call.offs_a, offs_b=call.offs_b, begin=call.begin,
        idx_a=call.idx_a, idx_b=call.idx_b, sel=sel, want_ref64=want_ref64, nthreads=nthreads,
        aux=arrs[call.aux] if call.aux else None)


def run_step_oracle(step, arrs: dict, nthreads=0):
    """One step of a chained workload through the oracle, in place on ``arrs`` (host arrays).
    Reduce outputs are stored as fp32 (the type the library writes) for the steps after."""
    if isinstance(step, Call):
        run_call_oracle(step, arrs, nthreads=nthreads)
    elif isinstance(step, TransformStep):
        oracle.transform_batched(step.kind, step.m, step.n, step.ld_in, step.ld_out, step.dtype,
                                 step.alpha, arrs[step.src], step.in_stride, arrs[step.dst],
                                 step.out_stride, step.G)
    elif isinstance(step, ReduceStep):
        want = tuple(w for w, d in (("x", step.dst_x), ("x2", step.dst_x2)) if d)
        ox, ox2 = oracle.reduce_batched(arrs[step.src], step.m, step.n, step.ld, step.in_type,
                                        step.G, step.in_stride, step.op, step.by, want,
                                        out_stride=step.out_stride or None)
        for d, o in ((step.dst_x, ox), (step.dst_x2, ox2)):
            if d:
                arrs[d].reshape(-1)[: o.size] = o.astype(np.float32)
    elif isinstance(step, EquationStep):
        leaves = [(arrs[name], ld, dt, bc) for name, ld, dt, bc in step.leaves]
        oracle.eq_eval(step.nodes, step.root, step.m, step.n, leaves, arrs[step.out], step.ldo,
                       step.out_type)
    elif isinstance(step, EmbeddingStep):
        oracle.embedding_bag(arrs[step.w], step.M, step.E, step.ldw, step.w_type,
                             arrs[step.begin], arrs[step.idx], arrs[step.out], step.ldo,
                             step.out_type)
    else:
        raise TypeError(f"unknown step {step!r}")


def run_steps_oracle(wl: Workload, nthreads=0) -> dict:
    """Every step of a chained workload through the oracle, on copies of its arrays."""
    arrs = {k: np.array(v, copy=True) for k, v in wl.arrays.items()}
    for st in wl.steps:
        run_step_oracle(st, arrs, nthreads=nthreads)
    return arrs


def run_oracle(wl: Workload, ci: int = 0, c_init=None, sel=None, want_ref64=False, nthreads=0):
    """Run call ``ci`` of ``wl`` through the oracle on a copy of its C array.

    Returns (c_out, ref64).  ``c_init`` overrides the C array (e.g. the output of an earlier
    call for chained workloads)."""
    call = wl.calls[ci]
    arrs = wl.arrays
    c = np.array(arrs[call.c] if c_init is None else c_init, copy=True)
    bias = arrs[call.bias] if call.bias else None
    ref = oracle.brgemm_batched(
        oracle_desc(call), arrs[call.a], arrs[call.b], c, bias, grid=call.grid, G=call.G,
        a_off=call.a_off, b_off=call.b_off, c_off=call.c_off, bias_off=call.bias_off,
        count=call.count, offs_a=call.offs_a, offs_b=call.offs_b, begin=call.begin,
        idx_a=call.idx_a, idx_b=call.idx_b, sel=sel, want_ref64=want_ref64, nthreads=nthreads)
    return c, ref


def values(arr: np.ndarray, dtype: str) -> np.ndarray:
    """Numeric values of an operand array (bf16 bit patterns or fp32) as float64."""
    if dtype == "bf16":
        return bf16_values(arr).astype(np.float64)
    return arr.astype(np.float64)


def rel_fro(got: np.ndarray, ref: np.ndarray) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref)
    num = np.linalg.norm(got - ref)
    return float(num / den) if den > 0 else float(num)
