"""GPU parity of the sparse embedding gather-reduce (Alg. 5), through the C ABI, against the CPU
oracle: bit-exact on small-integer tables (every fp32 partial sum exact), relative Frobenius
error <= 1e-5 for fp32 tables and outputs and <= 5e-3 once bf16 is involved, on both load paths
(16-byte chunks with 1, 2, 4 or more rows per wavefront load, and entry per lane), empty and
ragged bags, padded strides, skipped out-of-range indices, and the full-size lookup workload on
sampled bags."""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import oracle
import workloads as wk
from helpers import rel_fro, values

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    import paper_2104_05755_amd  # noqa: F401  (fails loudly if the HIP library is missing)
    return torch.device("cuda:0")


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def run_gpu(wl):
    from paper_2104_05755_amd import torch_io
    dev = torch_io.upload(wl)
    st = wl.steps[0]
    torch_io.launch_step(torch_io.prepare_step(st, dev), dev)
    torch.cuda.synchronize()
    return torch_io.to_host(dev[st.out], wl.arrays[st.out])


def run_ref(wl):
    st = wl.steps[0]
    out = np.array(wl.arrays[st.out], copy=True)
    oracle.embedding_bag(wl.arrays[st.w], st.M, st.E, st.ldw, st.w_type, wl.arrays[st.begin],
                         wl.arrays[st.idx], out, st.ldo, st.out_type)
    return out


def small(seed, rows, dim, bags, pool, w_type, out_type, pad=0, integer=False):
    wl = wk.embedding_bag(seed=seed, rows=rows, dim=dim, bags=bags, min_pool=pool[0],
                          max_pool=pool[1], w_type=w_type, out_type=out_type, pad=pad)
    if integer:
        rng = np.random.default_rng(seed + 1)
        wv = rng.integers(-8, 9, size=wl.arrays["w"].size).astype(np.float32)
        wl.arrays["w"] = wv if w_type == "f32" else wk.bf16_bits(wv)
    return wl


CASES = [  # rows, dim, bags, pooling, w_type, out_type, pad
    (500, 128, 37, (0, 40), "f32", "f32", 0),     # 32 chunks: two row slots
    (500, 64, 21, (1, 9), "f32", "f32", 0),       # 16 chunks: four slots
    (300, 96, 19, (0, 70), "f32", "f32", 0),      # 24 chunks: two slots, 16 lanes idle
    (300, 512, 9, (1, 20), "bf16", "f32", 0),     # 64 chunks: one slot
    (200, 1024, 5, (1, 12), "f32", "bf16", 0),    # 256 chunks: four column groups
    (400, 128, 33, (0, 30), "bf16", "bf16", 8),   # padded strides, still 16-byte aligned
    (400, 13, 17, (0, 25), "f32", "f32", 0),      # entry-per-lane path
    (400, 64, 17, (0, 25), "bf16", "bf16", 3),    # misaligned stride: entry-per-lane path
    (1, 8, 6, (0, 5), "f32", "f32", 0),           # a one-row table
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"M{c[0]}-E{c[1]}-B{c[2]}-{c[4]}-{c[5]}-pad{c[6]}")
@pytest.mark.parametrize("integer", [True, False])
def test_embedding_matches_oracle(case, integer):
    rows, dim, bags, pool, wt, ot, pad = case
    wl = small(rows * 7 + dim + bags, rows, dim, bags, pool, wt, ot, pad, integer)
    say(f"embedding {case} integer={integer}")
    got = run_gpu(wl)
    ref = run_ref(wl)
    st = wl.steps[0]
    g = values(got, ot).reshape(bags, st.ldo)
    r = values(ref, ot).reshape(bags, st.ldo)
    assert not np.isnan(g[:, :dim]).any()
    if integer:
        assert np.array_equal(got.reshape(bags, st.ldo)[:, :dim], ref.reshape(bags, st.ldo)[:, :dim])
    else:
        bar = 1e-5 if (wt == "f32" and ot == "f32") else 5e-3
        assert rel_fro(g[:, :dim], r[:, :dim]) <= bar
    if pad:   # the output rows' gaps are untouched
        assert np.array_equal(got.reshape(bags, st.ldo)[:, dim:].view(np.uint8),
                              wl.arrays["out"].reshape(bags, st.ldo)[:, dim:].view(np.uint8))


def test_out_of_range_indices_are_skipped():
    wl = small(61, 300, 128, 25, (1, 30), "f32", "f32", integer=True)
    idx = wl.arrays["idx"]
    bad = np.arange(0, idx.size, 7)
    idx_bad = idx.copy()
    idx_bad[bad[::2]] = 300                       # one past the last row
    idx_bad[bad[1::2]] = -5
    wl_bad = wk.Workload(wl.name, dict(wl.arrays, idx=idx_bad), [], steps=wl.steps)
    say("embedding with out-of-range indices")
    got = run_gpu(wl_bad)
    # the reference: the same bags with those entries removed from the lists
    keep = np.ones(idx.size, bool)
    keep[bad] = False
    begin = wl.arrays["begin"]
    new_begin = np.concatenate([[0], np.cumsum([keep[begin[b]:begin[b + 1]].sum()
                                                for b in range(len(begin) - 1)])]).astype(np.int64)
    ref = run_ref(wk.Workload(wl.name, dict(wl.arrays, idx=idx[keep], begin=new_begin), [],
                              steps=wl.steps))
    assert np.array_equal(got, ref)


def test_embedding_is_deterministic():
    wl = small(62, 2000, 128, 64, (20, 60), "f32", "f32")
    a, b = run_gpu(wl), run_gpu(wl)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_embedding_full_size_sampled():
    wl = wk.embedding_bag()
    st = wl.steps[0]
    begin = wl.arrays["begin"]
    n_bags = len(begin) - 1
    say(f"embedding full size: {st.M} rows x {st.E}, {n_bags} bags, {begin[-1]} lookups")
    got = run_gpu(wl).reshape(n_bags, st.ldo)
    rng = np.random.default_rng(63)
    sel = np.unique(np.concatenate([[0, n_bags - 1], rng.choice(n_bags, 200, replace=False)]))
    lens = begin[sel + 1] - begin[sel]
    sub_begin = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    sub_idx = np.concatenate([wl.arrays["idx"][begin[b]:begin[b + 1]] for b in sel])
    out = np.full(len(sel) * st.ldo, np.nan, np.float32)
    oracle.embedding_bag(wl.arrays["w"], st.M, st.E, st.ldw, st.w_type, sub_begin, sub_idx, out,
                         st.ldo, st.out_type)
    assert rel_fro(got[sel], out.reshape(len(sel), st.ldo)) <= 1e-5


def test_embedding_table_past_2_pow_32_bytes():
    """A 20,000,000 x 128 fp32 table (10.2 GB: row offsets past 2^31 elements and 2^32 bytes) with
    W[r][e] = ((128 r + e) mod 251) - 125 built on the device; 2048 bags of 1..64 seeded lookups
    (the last row among them).  Sums of at most 64 integers of magnitude <= 125 are exact in fp32,
    so every output element is checked against the closed form."""
    import paper_2104_05755_amd as tpp
    M, E = 20_000_000, 128
    assert M * E * 4 > 2 ** 32
    say(f"embedding table past 2^32 bytes: {M} x {E}")
    dev = torch.device("cuda:0")
    total = M * E
    chunk = 1 << 28
    W = torch.empty(total, dtype=torch.float32, device=dev)
    for s in range(0, total, chunk):
        e = torch.arange(s, min(s + chunk, total), dtype=torch.int64, device=dev)
        W[s:s + e.numel()] = ((e % 251) - 125).to(torch.float32)
    rng = np.random.default_rng(93)
    n_bags = 2048
    lens = rng.integers(1, 65, n_bags)
    begin = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    idx = rng.integers(0, M, int(begin[-1])).astype(np.int64)
    idx[-1] = M - 1
    out = torch.full((n_bags * E,), float("nan"), device=dev)
    tpp.tpp_embedding_bag(M, E, tpp.TPP_DT_F32, W, E, n_bags, torch.from_numpy(begin).to(dev),
                          torch.from_numpy(idx).to(dev), tpp.TPP_DT_F32, out, E,
                          tpp.current_stream())
    torch.cuda.synchronize()
    rows = ((idx[:, None] * E + np.arange(E)[None, :]) % 251) - 125          # lookups x E
    want = np.add.reduceat(rows, begin[:-1], axis=0).astype(np.float32)      # bags x E
    assert np.array_equal(out.cpu().numpy().reshape(n_bags, E), want)
