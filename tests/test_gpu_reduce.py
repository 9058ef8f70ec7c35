"""GPU parity of the Reduce TPP (through the C ABI) against the CPU oracle.

SUM and MUL are fp32 folds in an unspecified order: |gpu - ref| <= 1e-5 * (sum of |terms|)
(SUM) or (4 sqrt(count) 2^-24 + 1e-6) * |ref| (MUL, factors near 1).  MIN and MAX decide nothing but comparisons, and
fp32 rounding is monotone, so they are bit-exact against the oracle's value rounded to fp32 (also
for x*x: min of rounded squares = rounded min of squares)."""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import oracle
import workloads as wk
from helpers import values

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"


def gpu_reduce(x_host, m, n, ld, in_type, op, by, want):
    import paper_2104_05755_amd as tpp
    from paper_2104_05755_amd import torch_io
    x = torch_io.to_device(x_host)
    nout = m if by == "cols" else n
    ox = torch.full((nout,), float("nan"), device="cuda") if "x" in want else None
    ox2 = torch.full((nout,), float("nan"), device="cuda") if "x2" in want else None
    ops = dict(sum=tpp.TPP_RED_SUM, mul=tpp.TPP_RED_MUL, min=tpp.TPP_RED_MIN, max=tpp.TPP_RED_MAX)
    flags = (tpp.TPP_RED_BY_COLS if by == "cols" else tpp.TPP_RED_BY_ROWS)
    flags |= (tpp.TPP_RED_X if "x" in want else 0) | (tpp.TPP_RED_X2 if "x2" in want else 0)
    dt = tpp.TPP_DT_BF16 if in_type == "bf16" else tpp.TPP_DT_F32
    tpp.tpp_reduce(m, n, ld, dt, x, ops[op], flags, ox, ox2, tpp.current_stream())
    torch.cuda.synchronize()
    return (None if ox is None else ox.cpu().numpy(), None if ox2 is None else ox2.cpu().numpy())


def check(got, ref, absdata, op, by, what):
    count = absdata.shape[1] if by == "cols" else absdata.shape[0]
    assert got is not None and not np.isnan(got).any(), what
    if op in ("min", "max"):
        assert np.array_equal(got, ref.astype(np.float32)), what
    elif op == "sum":
        scale = absdata.sum(axis=1 if by == "cols" else 0)
        assert np.all(np.abs(got - ref) <= 1e-5 * scale + 1e-30), what
    else:
        # each of the count-1 products rounds once: a random walk of fp32 rounding errors
        rtol = 4.0 * np.sqrt(count) * 2.0 ** -24 + 1e-6
        assert np.all(np.abs(got - ref) <= rtol * np.abs(ref) + 1e-30), what


# (1024, 4096) by columns and (8192, 1024) by rows fold over 100+ and 4 partial results per
# output in the many-outputs combine pass.  By rows, 8192 columns or more take whole columns,
# several per wavefront: (8, 200000) and (77, 16387) four (the latter with a last group of three
# and a row tail), (512, 8193) two, (300, 9000, ld 301) two with element loads.
SHAPES = [(1, 1, 1), (3, 5, 3), (64, 100, 64), (64, 100, 67), (37, 513, 40), (1000, 7, 1000),
          (100000, 3, 100003), (8, 200000, 8), (257, 1031, 264), (4096, 64, 4096),
          (1024, 4096, 1024), (8192, 1024, 8192), (77, 16387, 80), (512, 8193, 512),
          (300, 9000, 301)]


@pytest.mark.parametrize("m,n,ld", SHAPES)
@pytest.mark.parametrize("in_type", ["f32", "bf16"])
@pytest.mark.parametrize("by", ["cols", "rows"])
def test_reduce_matches_oracle(m, n, ld, in_type, by):
    rng = np.random.default_rng(m * 7 + n * 13 + ld)
    for op in ("sum", "max", "min", "mul"):
        lo, hi = (0.97, 1.03) if op == "mul" else (-2.0, 2.0)
        raw = rng.uniform(lo, hi, size=n * ld).astype(np.float32)
        x = raw if in_type == "f32" else wk.bf16_bits(raw)
        print(f"reduce {op} by {by} m={m} n={n} ld={ld} {in_type}", flush=True)
        sys.stdout.flush()
        want = ("x",) if op == "mul" else ("x", "x2")
        rx, rx2 = oracle.reduce(x, m, n, ld, in_type, op, by, want)
        gx, gx2 = gpu_reduce(x, m, n, ld, in_type, op, by, want)
        X = np.abs(values(x, in_type).reshape(n, ld)[:, :m].T)          # m x n
        check(gx, rx, X, op, by, f"{op} x")
        if "x2" in want:
            check(gx2, rx2, X * X, op, by, f"{op} x2")


def test_reduce_batchnorm_statistics_shape():
    """The per-channel statistics of a conv output: NHWc bf16 with c = 64, reduced by columns."""
    rng = np.random.default_rng(17)
    t = wk.bf16_bits(rng.standard_normal((28, 56, 56, 64)).astype(np.float32) * 0.5)
    m, n = 64, 28 * 56 * 56
    rx, rx2 = oracle.reduce(t.reshape(-1), m, n, m, "bf16", "sum", "cols", ("x", "x2"))
    gx, gx2 = gpu_reduce(t.reshape(-1), m, n, m, "bf16", "sum", "cols", ("x", "x2"))
    X = np.abs(values(t.reshape(-1), "bf16").reshape(n, m).T)
    check(gx, rx, X, "sum", "cols", "bn sum")
    check(gx2, rx2, X * X, "sum", "cols", "bn sumsq")


def test_reduce_past_2_pow_32_elements():
    """65536 x 65537 bf16 (8.6 GB, past 2^32 elements): 64-bit column offsets in the by-rows
    (several columns per wavefront) and by-columns (whole columns per workgroup) kernels.  X is the
    closed-form pattern x(e) = (e mod 251) - 125 built on the device, so every result has a closed
    form: each period of 251 sums to zero, every partial sum stays below 2^24 (exact in fp32 in
    any order), and every column holds all 251 residues (its maximum is 125)."""
    import paper_2104_05755_amd as tpp
    m, n = 65536, 65537
    total = m * n
    assert total > 2 ** 32
    print(f"reduce past 2^32: {m} x {n}", flush=True)
    dev = torch.device("cuda:0")
    chunk = 1 << 28
    x = torch.empty(total, dtype=torch.bfloat16, device=dev)
    for s in range(0, total, chunk):
        e = torch.arange(s, min(s + chunk, total), dtype=torch.int64, device=dev)
        x[s:s + e.numel()] = ((e % 251) - 125).to(torch.bfloat16)
    stream = tpp.current_stream()
    by_rows = torch.full((n,), float("nan"), device=dev)
    mx = torch.full((n,), float("nan"), device=dev)
    by_cols = torch.full((m,), float("nan"), device=dev)
    tpp.tpp_reduce(m, n, m, tpp.TPP_DT_BF16, x, tpp.TPP_RED_SUM, tpp.TPP_RED_BY_ROWS | tpp.TPP_RED_X,
                   by_rows, None, stream)
    tpp.tpp_reduce(m, n, m, tpp.TPP_DT_BF16, x, tpp.TPP_RED_MAX, tpp.TPP_RED_BY_ROWS | tpp.TPP_RED_X,
                   mx, None, stream)
    tpp.tpp_reduce(m, n, m, tpp.TPP_DT_BF16, x, tpp.TPP_RED_SUM, tpp.TPP_RED_BY_COLS | tpp.TPP_RED_X,
                   by_cols, None, stream)
    torch.cuda.synchronize()

    def prefix(N):   # sum of x(e) for e < N
        r = N % 251
        return r * (r - 1) // 2 - 125 * r

    c = np.arange(n, dtype=np.int64)
    want_rows = prefix((c + 1) * m) - prefix(c * m)
    tail = np.arange((n // 251) * 251, n, dtype=np.int64)          # the columns past whole periods
    r = np.arange(m, dtype=np.int64)
    want_cols = (((r[:, None] + tail[None, :] * m) % 251) - 125).sum(axis=1)
    assert np.array_equal(by_rows.cpu().numpy(), want_rows.astype(np.float32))
    assert np.array_equal(mx.cpu().numpy(), np.full(n, 125.0, np.float32))
    assert np.array_equal(by_cols.cpu().numpy(), want_cols.astype(np.float32))


def test_concurrent_calls_on_two_streams():
    """Two host threads, each on its own stream, make Reduce calls that need a work buffer
    (several partials per output), with growing sizes so that the buffers are regrown while the
    other thread's work is queued; every result matches the oracle."""
    import threading
    import paper_2104_05755_amd as tpp
    dev = torch.device("cuda:0")
    rng = np.random.default_rng(95)
    cases = []
    for i in range(6):
        m, n = 64 * (i + 1), 20000 + 7000 * i          # by columns: many partials per output
        x = wk.bf16_bits(rng.uniform(-2, 2, m * n).astype(np.float32))
        rx, _ = oracle.reduce(x, m, n, m, "bf16", "sum", "cols", ("x",))
        cases.append((m, n, x, rx))
    errors = []

    def worker(order):
        try:
            s = torch.cuda.Stream(device=dev)
            with torch.cuda.stream(s):
                for _ in range(3):
                    for i in order:
                        m, n, x, rx = cases[i]
                        xd = torch.from_numpy(x.view(np.int16)).to(dev).view(torch.bfloat16)
                        out = torch.full((m,), float("nan"), device=dev)
                        tpp.tpp_reduce(m, n, m, tpp.TPP_DT_BF16, xd, tpp.TPP_RED_SUM,
                                       tpp.TPP_RED_BY_COLS | tpp.TPP_RED_X, out, None,
                                       s.cuda_stream)
                        s.synchronize()
                        X = np.abs(values(x, "bf16").reshape(n, m).T)
                        if not np.all(np.abs(out.cpu().numpy() - rx) <= 1e-5 * X.sum(axis=1)):
                            errors.append((order, i))
        except Exception as e:   # reported below, on the test's thread
            errors.append(repr(e))

    threads = [threading.Thread(target=worker, args=(o,)) for o in (range(6), range(5, -1, -1))]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
