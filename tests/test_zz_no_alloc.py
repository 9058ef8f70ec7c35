"""GPU test of tpp_brgemm_execute_batched_noalloc: it computes what tpp_brgemm_execute_batched
computes, with the same kernels, keeping a split reduction's partial tiles in the library's
per-GPU scratch array instead of an allocated work buffer.

Two calls in a row through the allocation-free entry point (the second on a smaller input, so it
reuses the scratch the first one left behind), then the same two calls through the allocating
entry point: the outputs must be identical bit for bit (same kernels, same split, same order of
the chunk sums), and within the bf16 bar of the oracle where the oracle is cheap enough.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import workloads as wk
from helpers import rel_fro, run_oracle, values

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    import paper_2104_05755_amd  # noqa: F401  (fails loudly if the HIP library is missing)
    return torch.device("cuda:0")


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _run_pair(wls, noalloc):
    """Each workload's single call on fresh device copies, all launched back to back on the
    current stream, then one synchronisation; host copies of the outputs."""
    from paper_2104_05755_amd import torch_io
    devs, outs = [], []
    for wl in wls:
        dev = torch_io.upload(wl)
        dc = torch_io.prepare(wl.calls[0], dev)
        devs.append((dev, dc))
    torch.cuda.synchronize()
    for dev, dc in devs:
        torch_io.launch(dc, noalloc=noalloc)
    torch.cuda.synchronize()
    for wl, (dev, dc) in zip(wls, devs):
        outs.append(torch_io.to_host(dev[wl.calls[0].c], wl.arrays[wl.calls[0].c]))
    return outs


def _blocks(flat, call, sel):
    """The output blocks of the instances in sel (all when None) of a strided-grid call."""
    if sel is None:
        return flat
    out = []
    for g in sel:
        gi_m, gi_n = g % call.grid["gm"], g // call.grid["gm"]
        off = gi_m * call.grid["c_step_m"] + gi_n * call.grid["c_step_n"]
        idx = off + np.arange(call.n)[:, None] * call.ldc + np.arange(call.m)[None, :]
        out.append(flat.reshape(-1)[idx])
    return np.stack(out)


CASES = {
    # 144 tiles of 128 x 128, 256 stages: split 3 ways, 432 partial tiles (27 MiB of scratch);
    # then half the stages, the same split
    "split_128": (lambda: wk.mlp_fc(seed=41, minibatch=1536, c_in=16384, k_out=1536),
                  lambda: wk.mlp_fc(seed=42, minibatch=1536, c_in=8192, k_out=1536)),
    # 16 tiles of 64 x 64, 64 stages: split 8 ways; then 6 tiles, 32 stages: split 4 ways
    "split_64": (lambda: wk.mlp_fc(seed=43, minibatch=256, c_in=4096, k_out=256),
                 lambda: wk.mlp_fc(seed=44, minibatch=128, c_in=2048, k_out=192)),
    # the fp32 kernel's pair-list split (16 pairs on one tile), then a call of 8 pairs
    "split_fp32": (lambda: wk.fp32_single(seed=45),
                   lambda: wk.fp32_single(seed=46, count=8)),
    # no split at all: the scratch is never looked up
    "no_split": (lambda: wk.mlp_fc(seed=47, minibatch=2048, c_in=1024, k_out=1024),
                 lambda: wk.mlp_fc(seed=48, minibatch=512, c_in=512, k_out=512)),
}


@pytest.mark.parametrize("case", sorted(CASES))
def test_noalloc_matches_allocating_entry_point(case):
    from paper_2104_05755_amd import torch_io
    first, second = (f() for f in CASES[case])
    wls = [first, second]
    for wl in wls:
        dev = torch_io.upload(wl)
        name = torch_io.describe(torch_io.prepare(wl.calls[0], dev))
        say(f"noalloc {case}: {wl.name} G={wl.calls[0].G} count={wl.calls[0].count} -> {name}")
        if case != "no_split":
            assert " + " in name, f"{case} does not split its reduction: {name}"
        del dev
    torch.cuda.synchronize()
    got = _run_pair(wls, noalloc=True)
    want = _run_pair(wls, noalloc=False)
    for i, (g, w) in enumerate(zip(got, want)):
        assert g.dtype == w.dtype and g.shape == w.shape
        view = np.uint16 if g.dtype == np.uint16 else np.uint32
        assert np.array_equal(g.view(view), w.view(view)), f"{case} call {i}: outputs differ"
    # the second call against the oracle as well: whole output, or 24 sampled instances
    call = second.calls[0]
    sel = None if call.G * call.count <= 16384 else sorted(
        np.random.default_rng(7).choice(call.G, size=24, replace=False).tolist())
    ref, _ = run_oracle(second, sel=sel)
    g_blk, r_blk = _blocks(got[1], call, sel), _blocks(ref, call, sel)
    err = rel_fro(values(g_blk, call.c_type), values(r_blk, call.c_type))
    bar = 1e-5 if call.ab_type == "f32" and call.c_type == "f32" else 5e-3
    assert err <= bar, f"{case}: rel Frobenius error {err:.3e} > {bar}"
