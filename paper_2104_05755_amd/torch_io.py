"""torch glue for the binding: device copies of host operands and one batched call per workload.

torch supplies device memory and the stream; every computation happens in the HIP library.
A workload call (see ``workloads.Call``) names its operand arrays, its instance grid and its pair
list; :func:`prepare` uploads what the call needs once, and :func:`launch` issues the batched
BRGEMM on the current stream.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional

import numpy as np
import torch

import paper_2104_05755_amd as tpp


def to_device(arr: np.ndarray, device="cuda") -> torch.Tensor:
    """Copy a host array to the device; bf16 bit patterns (uint16) travel as int16."""
    if arr.dtype == np.uint16:
        return torch.from_numpy(arr.view(np.int16)).to(device)
    return torch.from_numpy(np.ascontiguousarray(arr)).to(device)


def to_host(t: torch.Tensor, like: np.ndarray) -> np.ndarray:
    out = t.cpu().numpy()
    return out.view(np.uint16) if like.dtype == np.uint16 else out


@dataclass
class DeviceCall:
    handle: int
    call: object
    a: Optional[torch.Tensor]
    b: Optional[torch.Tensor]
    c: torch.Tensor
    bias: Optional[torch.Tensor]
    aux: Optional[torch.Tensor] = None
    a_off: Optional[torch.Tensor] = None
    b_off: Optional[torch.Tensor] = None
    c_off: Optional[torch.Tensor] = None
    bias_off: Optional[torch.Tensor] = None
    offs_a: Optional[torch.Tensor] = None
    offs_b: Optional[torch.Tensor] = None
    begin: Optional[torch.Tensor] = None
    ptrs_a: Optional[torch.Tensor] = None
    ptrs_b: Optional[torch.Tensor] = None


def descriptor(call) -> tpp.tpp_brgemm_desc:
    return tpp.make_desc(call.m, call.n, call.k, call.lda, call.ldb, call.ldc, call.ab_type,
                         call.c_type, call.beta, call.kind, call.stride_a, call.stride_b,
                         sorted(call.flags))


def _i64(x, device):
    """int64 device array; an empty list still gets one (unused) element so that its address is
    not NULL."""
    if x is None:
        return None
    arr = np.ascontiguousarray(x, dtype=np.int64)
    if arr.size == 0:
        arr = np.zeros(1, dtype=np.int64)
    return torch.from_numpy(arr).to(device)


def prepare(call, dev: dict, device="cuda") -> DeviceCall:
    """Dispatch the call's descriptor and upload its offset / pointer / CSR arrays.  ``dev`` maps
    array names to device tensors (the operands, already resident)."""
    h = tpp.tpp_brgemm_dispatch(descriptor(call))
    a = dev[call.a] if call.a else None
    b = dev[call.b] if call.b else None
    dc = DeviceCall(h, call, a, b, dev[call.c], dev[call.bias] if call.bias else None,
                    dev[call.aux] if getattr(call, "aux", None) else None)
    if call.grid is None:
        dc.a_off, dc.b_off = _i64(call.a_off, device), _i64(call.b_off, device)
        dc.c_off, dc.bias_off = _i64(call.c_off, device), _i64(call.bias_off, device)
    dc.offs_a, dc.offs_b = _i64(call.offs_a, device), _i64(call.offs_b, device)
    if call.kind == "address":
        es = 4 if call.ab_type == "f32" else 2
        dc.begin = _i64(call.begin, device)
        dc.ptrs_a = _i64(a.data_ptr() + np.asarray(call.idx_a, dtype=np.int64) * es, device)
        dc.ptrs_b = _i64(b.data_ptr() + np.asarray(call.idx_b, dtype=np.int64) * es, device)
    return dc


def describe(dc: DeviceCall) -> str:
    """The kernels launch(dc) runs, as the profiler names them."""
    call = dc.call
    a = dc.a if call.kind != "address" else None
    b = dc.b if call.kind != "address" else None
    return tpp.tpp_brgemm_describe_launch(
        dc.handle, call.grid, call.G, dc.a_off, dc.b_off, dc.c_off, dc.bias_off, a, b, dc.c,
        dc.bias, call.count, dc.offs_a, dc.offs_b, dc.begin, dc.ptrs_a, dc.ptrs_b)


def launch(dc: DeviceCall, stream: Optional[int] = None, noalloc: bool = False):
    """One batched BRGEMM launch for the whole call (all G instances); noalloc takes the
    allocation-free entry point."""
    call = dc.call
    if stream is None:
        stream = tpp.current_stream()
    a = dc.a if call.kind != "address" else None
    b = dc.b if call.kind != "address" else None
    if noalloc:
        tpp.tpp_brgemm_execute_batched_noalloc(
            dc.handle, call.grid, call.G, dc.a_off, dc.b_off, dc.c_off, dc.bias_off, a, b, dc.c,
            dc.bias, call.count, dc.offs_a, dc.offs_b, dc.begin, dc.ptrs_a, dc.ptrs_b, stream)
        return
    if dc.aux is not None:
        tpp.tpp_brgemm_execute_batched_aux(
            dc.handle, call.grid, call.G, dc.a_off, dc.b_off, dc.c_off, dc.bias_off, a, b, dc.c,
            dc.aux, dc.bias, call.count, dc.offs_a, dc.offs_b, dc.begin, dc.ptrs_a, dc.ptrs_b,
            stream)
        return
    tpp.tpp_brgemm_execute_batched(
        dc.handle, call.grid, call.G, dc.a_off, dc.b_off, dc.c_off, dc.bias_off, a, b,
        dc.c, dc.bias, call.count, dc.offs_a, dc.offs_b, dc.begin, dc.ptrs_a, dc.ptrs_b, stream)


_DT = {"f32": tpp.TPP_DT_F32, "bf16": tpp.TPP_DT_BF16}
_TR = {"transpose": tpp.TPP_TR_TRANSPOSE, "vnni": tpp.TPP_TR_VNNI,
       "vnni_t": tpp.TPP_TR_VNNI_TO_VNNI_T}
_RED = {"sum": tpp.TPP_RED_SUM, "mul": tpp.TPP_RED_MUL, "min": tpp.TPP_RED_MIN,
        "max": tpp.TPP_RED_MAX}


def prepare_step(step, dev: dict, device="cuda"):
    """A chained workload's step ready to launch: a DeviceCall for a BRGEMM call, the step itself
    for a Transform or Reduce step (their arguments are all sizes and array names)."""
    if hasattr(step, "kind") and hasattr(step, "grid"):
        return prepare(step, dev, device)
    return step


def launch_step(st, dev: dict, stream: Optional[int] = None):
    """One step of a chained workload (see ``workloads.TransformStep``, ``ReduceStep``,
    ``EmbeddingStep`` and ``EquationStep``)."""
    if stream is None:
        stream = tpp.current_stream()
    if isinstance(st, DeviceCall):
        launch(st, stream)
    elif hasattr(st, "nodes"):      # matrix equation
        args = [(dev[name], ld, _DT[dt], bc) for name, ld, dt, bc in st.leaves]
        tpp.tpp_equation_execute(st.nodes, st.root, st.m, st.n, args, dev[st.out], st.ldo,
                                 _DT[st.out_type], stream)
    elif hasattr(st, "ldw"):        # embedding gather-reduce
        begin = dev[st.begin]
        tpp.tpp_embedding_bag(st.M, st.E, _DT[st.w_type], dev[st.w], st.ldw, begin.numel() - 1,
                              begin, dev[st.idx], _DT[st.out_type], dev[st.out], st.ldo, stream)
    elif hasattr(st, "ld_in"):      # transform
        tpp.tpp_transform_batched(_TR[st.kind], st.m, st.n, st.ld_in, st.ld_out, _DT[st.dtype],
                                  st.alpha, dev[st.src], st.in_stride, dev[st.dst], st.out_stride,
                                  st.G, stream)
    else:                           # reduce
        flags = tpp.TPP_RED_BY_COLS if st.by == "cols" else tpp.TPP_RED_BY_ROWS
        flags |= (tpp.TPP_RED_X if st.dst_x else 0) | (tpp.TPP_RED_X2 if st.dst_x2 else 0)
        tpp.tpp_reduce_batched(st.m, st.n, st.ld, _DT[st.in_type], dev[st.src], st.G,
                               st.in_stride, _RED[st.op], flags,
                               dev[st.dst_x] if st.dst_x else None,
                               dev[st.dst_x2] if st.dst_x2 else None, st.out_stride, stream)


def upload(wl, device="cuda") -> dict:
    return {name: to_device(arr, device) for name, arr in wl.arrays.items()}
