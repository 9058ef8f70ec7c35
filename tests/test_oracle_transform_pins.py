"""Pins of the oracle's Transform TPP (Table 1; Sec. 3.1) against what the definitions fix.

Transpose is pinned to numpy's transpose; VNNI formatting ([D1][D0] -> [D1/a][D0][a], the
[K/a][M][a] reformatting of Sec. 3.2.2) to numpy reshape / axis swaps of the logical tensor;
VNNI to VNNI-transpose to the composition un-VNNI -> transpose -> VNNI done in numpy.  Tiny
examples are worked out by hand from the definitions, and the permutations must move every bit
pattern unchanged, leave positions outside their extent alone and complete a last partial
group with zeros.  No GPU needed."""
from __future__ import annotations

import numpy as np
import pytest

import oracle

SENT16, SENT32 = 0xBEEF, 0xDEADBEEF


def _np_dtype(dtype):
    return np.uint32 if dtype == "f32" else np.uint16


def _sentinel(dtype):
    return SENT32 if dtype == "f32" else SENT16


def _random_bits(rng, size, dtype):
    """Arbitrary bit patterns (NaN payloads, denormals, negative zero included)."""
    if dtype == "f32":
        return rng.integers(0, 2**32, size=size, dtype=np.uint64).astype(np.uint32)
    return rng.integers(0, 2**16, size=size, dtype=np.uint32).astype(np.uint16)


def _oracle(kind, m, n, ld_in, ld_out, dtype, alpha, x):
    """The oracle on bit patterns (fp32 moved as uint32 views, bf16 as uint16)."""
    size = oracle.transform_out_len(kind, m, n, ld_out, alpha)
    out = np.full(size, _sentinel(dtype), dtype=_np_dtype(dtype))
    xin = x.view(np.float32) if dtype == "f32" else x
    oin = out.view(np.float32) if dtype == "f32" else out
    oracle.transform(kind, m, n, ld_in, ld_out, dtype, alpha, xin, oin)
    return out


def _logical(x, m, n, ld):
    """The m x n column-major tensor stored in x with leading dimension ld, as an (m, n) array."""
    return x[: ld * n].reshape(n, ld)[:, :m].T


def _store_colmajor(O, ld, dtype):
    """O (rows x cols) stored column-major with leading dimension ld, sentinel in the gaps."""
    rows, cols = O.shape
    out = np.full(ld * cols, _sentinel(dtype), dtype=_np_dtype(dtype))
    out.reshape(cols, ld)[:, :rows] = O.T
    return out


def _vnni_numpy(X, alpha):
    """[D1][D0] -> [D1/a][D0][a] for X of shape (D0, D1) = (m, n), via numpy: pad D1 with zero
    columns to a multiple of alpha, split D1 into (groups, alpha), move alpha innermost."""
    m, n = X.shape
    groups = -(-n // alpha)
    Xp = np.zeros((m, groups * alpha), dtype=X.dtype)
    Xp[:, :n] = X
    return Xp.T.reshape(groups, alpha, m).transpose(0, 2, 1)   # (groups, m, alpha)


def _store_groups(blocks, ld_out, dtype):
    """(groups, rows, alpha) blocks at group stride ld_out, sentinel in the gaps."""
    g, rows, alpha = blocks.shape
    out = np.full(g * ld_out, _sentinel(dtype), dtype=_np_dtype(dtype))
    for i in range(g):
        out[i * ld_out: i * ld_out + rows * alpha] = blocks[i].reshape(-1)
    return out


# ----------------------------------------------------------------------------------------------
# Tiny examples worked out by hand from the definitions
# ----------------------------------------------------------------------------------------------
def test_hand_examples_3x4():
    # X is 3 x 4, column-major, entry (r, c) = 3c + r: columns [0 1 2] [3 4 5] [6 7 8] [9 10 11]
    x = np.arange(12, dtype=np.uint16)
    # transpose: the 4 x 3 result, column r of it is row r of X
    assert _oracle("transpose", 3, 4, 3, 4, "bf16", 1, x).tolist() == \
        [0, 3, 6, 9, 1, 4, 7, 10, 2, 5, 8, 11]
    # VNNI, alpha 2: group g interleaves columns 2g and 2g+1 row by row
    v = _oracle("vnni", 3, 4, 3, 6, "bf16", 2, x)
    assert v.tolist() == [0, 3, 1, 4, 2, 5, 6, 9, 7, 10, 8, 11]
    # VNNI -> VNNI-transpose, alpha 2: the 4 x 3 transpose in VNNI form; its columns are X's rows
    # 0..2, grouped (0, 1) and (2, pad)
    assert _oracle("vnni_t", 3, 4, 6, 8, "bf16", 2, v).tolist() == \
        [0, 1, 3, 4, 6, 7, 9, 10, 2, 0, 5, 0, 8, 0, 11, 0]
    # VNNI, alpha 4, n = 4: one group, four columns interleaved
    assert _oracle("vnni", 3, 4, 3, 12, "bf16", 4, x).tolist() == \
        [0, 3, 6, 9, 1, 4, 7, 10, 2, 5, 8, 11]


# ----------------------------------------------------------------------------------------------
# Library routines
# ----------------------------------------------------------------------------------------------
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("m,n,pad_in,pad_out", [(1, 1, 0, 0), (7, 5, 3, 2), (64, 64, 0, 0),
                                                 (65, 130, 1, 7), (200, 33, 8, 0)])
def test_transpose_is_numpy_transpose(dtype, m, n, pad_in, pad_out):
    rng = np.random.default_rng(m * 1000 + n)
    ld_in, ld_out = m + pad_in, n + pad_out
    x = _random_bits(rng, ld_in * n, dtype)
    got = _oracle("transpose", m, n, ld_in, ld_out, dtype, 1, x)
    want = _store_colmajor(np.transpose(_logical(x, m, n, ld_in)), ld_out, dtype)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("alpha", [1, 2, 4])
@pytest.mark.parametrize("m,n,pad_in,pad_out", [(1, 4, 0, 0), (5, 8, 2, 3), (64, 64, 0, 0),
                                                 (33, 20, 1, 0), (9, 7, 0, 5), (16, 1, 0, 0)])
def test_vnni_is_numpy_reshape(dtype, alpha, m, n, pad_in, pad_out):
    rng = np.random.default_rng(7 * m + n + alpha)
    ld_in, ld_out = m + pad_in, m * alpha + pad_out
    x = _random_bits(rng, ld_in * n, dtype)
    got = _oracle("vnni", m, n, ld_in, ld_out, dtype, alpha, x)
    want = _store_groups(_vnni_numpy(_logical(x, m, n, ld_in), alpha), ld_out, dtype)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("alpha", [1, 2, 4])
@pytest.mark.parametrize("m,n,pad_in,pad_out", [(4, 4, 0, 0), (6, 10, 2, 1), (64, 32, 0, 0),
                                                 (13, 9, 0, 3), (2, 17, 5, 0)])
def test_vnni_to_vnni_t_is_unvnni_transpose_vnni(dtype, alpha, m, n, pad_in, pad_out):
    rng = np.random.default_rng(11 * m + n + alpha)
    groups_in = -(-n // alpha)
    ld_in, ld_out = m * alpha + pad_in, n * alpha + pad_out
    x = _random_bits(rng, ld_in * groups_in, dtype)
    # un-VNNI in numpy: entry (r, c) of the logical tensor is x[(c // a) * ld_in + r * a + c % a]
    blocks = np.stack([x[g * ld_in: g * ld_in + m * alpha].reshape(m, alpha)
                       for g in range(groups_in)])                  # (groups, m, alpha)
    X = blocks.transpose(1, 0, 2).reshape(m, groups_in * alpha)[:, :n]
    want = _store_groups(_vnni_numpy(X.T.copy(), alpha), ld_out, dtype)
    got = _oracle("vnni_t", m, n, ld_in, ld_out, dtype, alpha, x)
    assert np.array_equal(got, want)


# ----------------------------------------------------------------------------------------------
# Invariants and special cases
# ----------------------------------------------------------------------------------------------
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_transpose_twice_is_identity(dtype):
    rng = np.random.default_rng(3)
    m, n = 37, 53
    x = _random_bits(rng, m * n, dtype)
    t = _oracle("transpose", m, n, m, n, dtype, 1, x)
    assert np.array_equal(_oracle("transpose", n, m, n, m, dtype, 1, t), x)


@pytest.mark.parametrize("alpha", [1, 2, 4])
def test_vnni_to_vnni_t_twice_is_identity(alpha):
    rng = np.random.default_rng(alpha)
    m, n = 8 * alpha, 4 * alpha
    x = _random_bits(rng, m * alpha * (n // alpha), "bf16")
    t = _oracle("vnni_t", m, n, m * alpha, n * alpha, "bf16", alpha, x)
    assert np.array_equal(_oracle("vnni_t", n, m, n * alpha, m * alpha, "bf16", alpha, t), x)


def test_vnni_alpha_one_is_a_column_copy_and_vnni_t_alpha_one_is_transpose():
    rng = np.random.default_rng(5)
    m, n = 11, 6
    x = _random_bits(rng, m * n, "f32")
    assert np.array_equal(_oracle("vnni", m, n, m, m, "f32", 1, x), x)
    assert np.array_equal(_oracle("vnni_t", m, n, m, n, "f32", 1, x),
                          _oracle("transpose", m, n, m, n, "f32", 1, x))


def test_partial_last_group_is_zero_filled():
    x = np.arange(1, 3 * 5 + 1, dtype=np.uint16)     # 3 x 5, no zero entries
    v = _oracle("vnni", 3, 5, 3, 12, "bf16", 4, x)   # groups: columns 0-3, then 4 + 3 zeros
    second = v[12:24].reshape(3, 4)
    assert second[:, 0].tolist() == [13, 14, 15] and not second[:, 1:].any()


def test_empty_shapes_write_nothing_and_bad_arguments_are_rejected():
    out = np.full(8, SENT16, dtype=np.uint16)
    x = np.zeros(8, dtype=np.uint16)
    for kind in ("transpose", "vnni", "vnni_t"):
        oracle.transform(kind, 0, 4, 16, 16, "bf16", 2, x, out)
        oracle.transform(kind, 4, 0, 16, 16, "bf16", 2, x, out)
    assert (out == SENT16).all()
    for args in [("transpose", 4, 4, 3, 4, 1), ("transpose", 4, 4, 4, 3, 1),
                 ("vnni", 4, 4, 4, 7, 2), ("vnni", 4, 4, 4, 8, 3),
                 ("vnni_t", 4, 4, 7, 8, 2), ("vnni_t", 4, 4, 8, 7, 2)]:
        kind, m, n, ld_in, ld_out, alpha = args
        with pytest.raises(ValueError):
            oracle.transform(kind, m, n, ld_in, ld_out, "bf16", alpha, np.zeros(64, np.uint16),
                             np.zeros(64, np.uint16))
