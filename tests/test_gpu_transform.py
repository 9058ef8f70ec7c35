"""GPU parity of the Transform TPP (through the C ABI) against the CPU oracle.

A transform only moves entries, so the bar is bit-exact: the whole output buffer, including the
positions outside the transformation's extent (gaps when ld_out exceeds it), which start as a
sentinel pattern on both sides and must keep it.  Inputs are arbitrary bit patterns (NaN
payloads, denormals and negative zero included).  Shapes cover whole 64 x 64 tiles (the 16-byte
path), ragged edges, padded leading dimensions, misaligned bases (the entry path), partial last
VNNI groups, empty shapes and the full-size tensors the benchmark moves."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu

SENT = {"bf16": 0xBEEF, "f32": 0xDEADBEEF}
KINDS = {"transpose": 0, "vnni": 1, "vnni_t": 2}


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"


def _np(dtype):
    return np.uint32 if dtype == "f32" else np.uint16


def _bits(rng, size, dtype):
    if dtype == "f32":
        return rng.integers(0, 2**32, size=size, dtype=np.uint64).astype(np.uint32)
    return rng.integers(0, 2**16, size=size, dtype=np.uint32).astype(np.uint16)


def _in_len(kind, m, n, ld_in, alpha):
    if m == 0 or n == 0:
        return 1
    return ld_in * (n if kind != "vnni_t" else -(-n // alpha))


def ref(kind, m, n, ld_in, ld_out, dtype, alpha, x, out_len):
    out = np.full(out_len, SENT[dtype], dtype=_np(dtype))
    view = (lambda a: a.view(np.float32)) if dtype == "f32" else (lambda a: a)
    oracle.transform(kind, m, n, ld_in, ld_out, dtype, alpha, view(x), view(out))
    return out


def gpu(kind, m, n, ld_in, ld_out, dtype, alpha, x, out_len, in_shift=0, out_shift=0):
    """Run the GPU transform with the input / output bases moved by in_shift / out_shift
    entries from a fresh allocation (misaligned when not a multiple of 16 bytes)."""
    import paper_2104_05755_amd as tpp
    sdt = torch.int32 if dtype == "f32" else torch.int16
    sint = np.int32 if dtype == "f32" else np.int16
    xd = torch.zeros(x.size + in_shift, dtype=sdt, device="cuda")
    xd[in_shift:] = torch.from_numpy(x.view(sint)).cuda()
    od = torch.from_numpy(np.full(out_len + out_shift, SENT[dtype], dtype=_np(dtype)).view(sint)).cuda()
    dt = tpp.TPP_DT_F32 if dtype == "f32" else tpp.TPP_DT_BF16
    tpp.tpp_transform(KINDS[kind], m, n, ld_in, ld_out, dt, alpha, xd[in_shift:], od[out_shift:],
                      tpp.current_stream())
    torch.cuda.synchronize()
    return od[out_shift:].cpu().numpy().view(_np(dtype))


def check(kind, m, n, pad_in, pad_out, dtype, alpha, seed, in_shift=0, out_shift=0):
    rng = np.random.default_rng(seed)
    ld_in = (m if kind != "vnni_t" else m * alpha) + pad_in
    ld_out = {"transpose": n, "vnni": m * alpha, "vnni_t": n * alpha}[kind] + pad_out
    x = _bits(rng, _in_len(kind, m, n, ld_in, alpha), dtype)
    out_len = max(oracle.transform_out_len(kind, m, n, ld_out, alpha), 1)
    want = ref(kind, m, n, ld_in, ld_out, dtype, alpha, x, out_len)
    got = gpu(kind, m, n, ld_in, ld_out, dtype, alpha, x, out_len, in_shift, out_shift)
    if not np.array_equal(got, want):
        bad = np.flatnonzero(got != want)
        raise AssertionError(f"{kind} {dtype} alpha={alpha} m={m} n={n} ld_in={ld_in} "
                             f"ld_out={ld_out}: {bad.size} positions differ, first {bad[:8]}")


SHAPES = [(1, 1, 0, 0), (64, 64, 0, 0), (128, 192, 0, 0), (65, 63, 0, 0), (333, 517, 3, 5),
          (256, 256, 8, 8), (1000, 70, 0, 0), (7, 1000, 1, 0), (130, 9, 0, 16)]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_transpose_matches_oracle(dtype, shape):
    m, n, pi, po = shape
    check("transpose", m, n, pi, po, dtype, 1, seed=m * 7 + n)


@pytest.mark.parametrize("kind", ["vnni", "vnni_t"])
@pytest.mark.parametrize("alpha", [1, 2, 4])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_vnni_kinds_match_oracle(kind, alpha, dtype, shape):
    m, n, pi, po = shape
    check(kind, m, n, pi, po, dtype, alpha, seed=m * 11 + n + alpha)


@pytest.mark.parametrize("kind,alpha", [("transpose", 1), ("vnni", 2), ("vnni", 4), ("vnni_t", 2)])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("shift", [(1, 0), (0, 1), (3, 5)])
def test_misaligned_bases_take_the_entry_path(kind, alpha, dtype, shift):
    check(kind, 192, 128, 0, 0, dtype, alpha, seed=5, in_shift=shift[0], out_shift=shift[1])


@pytest.mark.parametrize("kind", ["transpose", "vnni", "vnni_t"])
def test_empty_shapes_leave_the_output_alone(kind):
    for m, n in ((0, 9), (9, 0)):
        check(kind, m, n, 16, 16, "bf16", 2, seed=1)


@pytest.mark.parametrize("kind,m,n,alpha", [
    ("transpose", 8192, 4096, 1),    # the hidden activations of the MLP block (64 MB), as timed
    ("transpose", 4096, 1024, 1),    # its first weight matrix
    ("vnni", 1024, 4096, 2),         # that weight as [K/2][M][2]
    ("vnni_t", 1024, 4096, 2),
])
def test_full_size_tensors(kind, m, n, alpha):
    check(kind, m, n, 0, 0, "bf16", alpha, seed=9)


@pytest.mark.parametrize("m,n", [(65537, 65537), (65536, 65544)], ids=["entry", "vector"])
def test_transpose_past_2_pow_32_entries(m, n):
    """Transposes of m x n bf16 past 2^32 entries (8.6 GB each way): odd leading dimensions
    (entry loads) and whole 16-byte units (16-byte chunks).  The input is x(e) = (e mod 251) - 125
    built on the device; output entry (i, j) must be input entry (j, i), checked everywhere."""
    import paper_2104_05755_amd as tpp
    total = m * n
    assert total > 2 ** 32
    print(f"transpose past 2^32: {m} x {n}", flush=True)
    dev = torch.device("cuda:0")
    chunk = 1 << 28
    x = torch.empty(total, dtype=torch.bfloat16, device=dev)
    for s in range(0, total, chunk):
        e = torch.arange(s, min(s + chunk, total), dtype=torch.int64, device=dev)
        x[s:s + e.numel()] = ((e % 251) - 125).to(torch.bfloat16)
    out = torch.full((total,), float("nan"), dtype=torch.bfloat16, device=dev)
    tpp.tpp_transform(tpp.TPP_TR_TRANSPOSE, m, n, m, n, tpp.TPP_DT_BF16, 1, x, out,
                      tpp.current_stream())
    torch.cuda.synchronize()
    del x
    bad = 0
    for s in range(0, total, chunk):
        f = torch.arange(s, min(s + chunk, total), dtype=torch.int64, device=dev)
        src = f // n + (f % n) * m          # output (i = f % n, j = f // n) <- input (j, i)
        want = ((src % 251) - 125).to(torch.float32)
        bad += int((out[s:s + f.numel()].to(torch.float32) != want).sum().item())
    assert bad == 0, f"{bad} wrong entries"
