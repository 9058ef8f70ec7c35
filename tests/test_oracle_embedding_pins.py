"""Pins of the oracle's sparse embedding gather-reduce (Alg. 5), CPU only.

The definition the paper gives is o^T = a^T x W with a the multi-hot vector of a bag's indices;
numpy's dense product of that vector (or, with repeated indices, of the count vector) with the
table is the independent check, exact on small-integer tables.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import workloads as wk
from helpers import values


def _case(rng, M, E, lens, pad=0, integer=True, distinct=False, w_type="f32"):
    ldw = E + pad
    wv = (rng.integers(-8, 9, size=M * ldw) if integer else rng.uniform(-1, 1, M * ldw)) \
        .astype(np.float32)
    w = wv if w_type == "f32" else wk.bf16_bits(wv)
    begin = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    if distinct:
        idx = np.concatenate([rng.permutation(M)[:n] for n in lens]).astype(np.int64)
    else:
        idx = rng.integers(0, M, size=int(begin[-1])).astype(np.int64)
    return w, ldw, begin, idx


def _dense(w, M, E, ldw, w_type):
    return values(w, w_type).reshape(M, ldw)[:, :E]


def _multi_hot(begin, idx, M):
    """Row b: how often each table row appears in bag b (a^T for distinct indices)."""
    A = np.zeros((len(begin) - 1, M))
    for b in range(len(begin) - 1):
        np.add.at(A[b], idx[begin[b]:begin[b + 1]], 1.0)
    return A


@pytest.mark.parametrize("distinct", [True, False])
def test_embedding_is_multi_hot_times_table(distinct):
    rng = np.random.default_rng(51)
    M, E = 60, 24
    lens = rng.integers(0, 9, size=13)
    w, ldw, begin, idx = _case(rng, M, E, lens, pad=5, distinct=distinct)
    out = np.full(13 * (E + 3), -7.0, np.float32)
    oracle.embedding_bag(w, M, E, ldw, "f32", begin, idx, out, E + 3, "f32")
    A = _multi_hot(begin, idx, M)
    if distinct:
        assert A.max() <= 1.0           # a true multi-hot vector per bag
    want = A @ _dense(w, M, E, ldw, "f32")                # integers: exact
    got = out.reshape(13, E + 3)
    assert np.array_equal(got[:, :E], want)
    assert np.all(got[:, E:] == -7.0)                     # output row gaps untouched


def test_empty_bags_are_zero_and_no_bags_is_a_no_op():
    rng = np.random.default_rng(52)
    w, ldw, begin, idx = _case(rng, 10, 8, [0, 3, 0, 0, 2])
    out = np.full(5 * 8, np.nan, np.float32)
    oracle.embedding_bag(w, 10, 8, ldw, "f32", begin, idx, out, 8, "f32")
    o = out.reshape(5, 8)
    assert not o[0].any() and not o[2].any() and not o[3].any()
    empty = np.full(4, 5.0, np.float32)
    oracle.embedding_bag(w, 10, 8, ldw, "f32", np.zeros(1, np.int64), idx, empty, 8, "f32")
    assert np.all(empty == 5.0)


@pytest.mark.parametrize("w_type,out_type", [("bf16", "bf16"), ("f32", "bf16"), ("bf16", "f32")])
def test_embedding_rounding_and_types(w_type, out_type):
    rng = np.random.default_rng(53)
    M, E = 40, 16
    lens = rng.integers(1, 30, size=9)
    w, ldw, begin, idx = _case(rng, M, E, lens, integer=False, w_type=w_type)
    out = np.zeros(9 * E, np.float32 if out_type == "f32" else np.uint16)
    ref = oracle.embedding_bag(w, M, E, ldw, w_type, begin, idx, out, E, out_type,
                               want_ref64=True)
    want = _multi_hot(begin, idx, M) @ _dense(w, M, E, ldw, w_type)
    np.testing.assert_allclose(ref, want, rtol=1e-13, atol=1e-13)
    # the output is the fp64 sum rounded to fp32, then (bf16 outputs) by torch's fp32 -> bf16
    r32 = ref.astype(np.float32).reshape(-1)
    expect = r32 if out_type == "f32" else wk.bf16_bits(r32)
    assert np.array_equal(out, expect)


@pytest.mark.parametrize("bad", ["index_high", "index_negative", "begin_decreasing"])
def test_embedding_rejects_bad_lists(bad):
    rng = np.random.default_rng(54)
    w, ldw, begin, idx = _case(rng, 10, 8, [2, 2])
    if bad == "index_high":
        idx[1] = 10
    elif bad == "index_negative":
        idx[2] = -1
    else:
        begin[1] = 5
    with pytest.raises(ValueError):
        oracle.embedding_bag(w, 10, 8, ldw, "f32", begin, idx, np.zeros(16, np.float32), 8, "f32")
