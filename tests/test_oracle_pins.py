"""Pins of the CPU oracle against what the paper and the mathematics fix (no GPU needed).

Each test ties the oracle to something other than itself: a library routine (numpy matmul,
torch conv2d / gelu / bf16 conversion), an exact rational brute force, a closed form, or an
invariant stated by the paper (Table 3: GEMM is the batch-count-1 BRGEMM; Sec. 2.3: the three
addressing variants name the same blocks)."""
from __future__ import annotations

import itertools
import math
import zlib
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
import workloads as wk
from helpers import oracle_desc, rel_fro, run_oracle, values


# ----------------------------------------------------------------------------------------------
# Numeric conversions
# ----------------------------------------------------------------------------------------------
def _torch_bf16(x_f32: np.ndarray) -> np.ndarray:
    return torch.from_numpy(x_f32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def test_bf16_rne_matches_torch_on_ties_and_random_patterns():
    rng = np.random.default_rng(11)
    hi = np.arange(0, 1 << 16, dtype=np.uint32)
    patterns = [hi << 16 | 0x8000, hi << 16 | 0x7FFF, hi << 16 | 0x8001, hi << 16,
                rng.integers(0, 1 << 32, size=1 << 20, dtype=np.uint64).astype(np.uint32)]
    bits = np.concatenate(patterns)
    x = bits.view(np.float32)
    got = oracle.f32_to_bf16_array(x)
    ref = _torch_bf16(x)
    nan = np.isnan(x)
    assert np.array_equal(got[~nan], ref[~nan])
    # NaN stays NaN (payload not compared)
    got_f = wk.bf16_values(got[nan])
    assert np.all(np.isnan(got_f))


def test_bf16_rne_special_values():
    cases = [(1.0, 0x3F80), (-2.0, 0xC000), (float("inf"), 0x7F80), (float("-inf"), 0xFF80),
             (0.0, 0x0000), (-0.0, 0x8000)]
    for v, want in cases:
        assert oracle.f32_to_bf16(v) == want
    # largest finite fp32 rounds past the largest finite bf16 (0x7F7F) to +inf
    big = np.array([3.4028235e38], dtype=np.float32)
    assert oracle.f32_to_bf16(float(big[0])) == 0x7F80
    # exact halfway between 1.0 (0x3F80) and next (0x3F81): ties to even -> 0x3F80
    assert oracle.f32_to_bf16(1.00390625) == 0x3F80
    # halfway between 0x3F81 and 0x3F82 goes up to the even 0x3F82
    assert oracle.f32_to_bf16(float(np.array([0x3F818000], np.uint32).view(np.float32)[0])) == 0x3F82


def test_bf16_widening_is_exact_for_all_patterns():
    h = np.arange(0, 1 << 16, dtype=np.uint16)
    ref = torch.from_numpy(h.view(np.int16)).view(torch.bfloat16).to(torch.float32).numpy()
    got = np.array([oracle.bf16_to_f32(int(v)) for v in h[::97]], dtype=np.float32)
    r = ref[::97]
    ok = np.isnan(r) & np.isnan(got) | (got.view(np.uint32) == r.view(np.uint32))
    assert ok.all()


def test_gelu_tanh_matches_library_and_is_odd_plus_identity():
    xs = np.linspace(-12, 12, 4001)
    got = np.array([oracle.gelu_tanh(float(v)) for v in xs])
    ref = torch.nn.functional.gelu(torch.from_numpy(xs), approximate="tanh").numpy()
    assert np.max(np.abs(got - ref)) < 1e-14
    # g(x) - g(-x) = x because tanh is odd
    back = np.array([oracle.gelu_tanh(float(-v)) for v in xs])
    assert np.max(np.abs(got - back - xs)) < 1e-13
    assert oracle.gelu_tanh(0.0) == 0.0
    assert abs(oracle.gelu_tanh(30.0) - 30.0) < 1e-12
    assert abs(oracle.gelu_tanh(-30.0)) < 1e-12


# ----------------------------------------------------------------------------------------------
# Brute force: an exact rational evaluation of the definition, written independently
# ----------------------------------------------------------------------------------------------
def _blocks(call: wk.Call, arrs: dict):
    """Dense (m x k, k x n) float64 views of each pair, built from numpy strides."""
    a_all = values(arrs[call.a], call.ab_type)
    b_all = values(arrs[call.b], call.ab_type)
    if call.kind == "stride":
        starts = [(i * call.stride_a, i * call.stride_b) for i in range(call.count)]
    elif call.kind == "offset":
        starts = list(zip(call.offs_a.tolist(), call.offs_b.tolist()))
    else:
        starts = list(zip(call.idx_a.tolist(), call.idx_b.tolist()))
    out = []
    for sa, sb in starts:
        A = np.lib.stride_tricks.as_strided(a_all[sa:], shape=(call.m, call.k),
                                            strides=(8, 8 * call.lda))
        B = np.lib.stride_tricks.as_strided(b_all[sb:], shape=(call.k, call.n),
                                            strides=(8, 8 * call.ldb))
        out.append((A.copy(), B.copy()))
    return out


def _exact_sum(pairs, r, c):
    total = Fraction(0)
    for A, B in pairs:
        for p in range(A.shape[1]):
            total += Fraction(float(A[r, p])) * Fraction(float(B[p, c]))
    return total


@pytest.mark.parametrize("kind", ["stride", "offset", "address"])
@pytest.mark.parametrize("ab_type,c_type", [("f32", "f32"), ("bf16", "f32"), ("bf16", "bf16")])
def test_brute_force_exact_rational(kind, ab_type, c_type):
    rng = np.random.default_rng(zlib.crc32(repr((kind, ab_type, c_type)).encode()))
    for (m, n, k, count) in [(1, 1, 1, 1), (2, 3, 5, 2), (5, 2, 3, 3), (3, 4, 2, 0)]:
        for beta in (0.0, 1.0, -0.5):
            wl = wk.small_case(rng, m, n, k, count, kind, ab_type, c_type, beta, {"bias"}, pad=1)
            call = wl.calls[0]
            c_in = values(wl.arrays["c"], c_type).reshape(n, call.ldc)
            _, ref = run_oracle(wl, want_ref64=True)
            pairs = _blocks(call, wl.arrays)
            bias = wl.arrays["bias"]
            for r in range(m):
                for c in range(n):
                    s = _exact_sum(pairs, r, c)
                    if beta != 0.0:
                        s += Fraction(beta) * Fraction(float(c_in[c, r]))
                    s += Fraction(float(bias[r]))
                    scale = sum(abs(float(A[r, p] * B[p, c])) for A, B in pairs
                                for p in range(k)) + 1.0
                    assert abs(float(s) - ref[0, c, r]) <= 1e-12 * scale


@pytest.mark.parametrize("kind", ["stride", "offset", "address"])
def test_integer_inputs_give_exact_rounded_outputs(kind):
    """Small integers: every partial sum is exact, so the rounded outputs are exactly the
    integer results (bf16 keeps integers up to 256 exactly; larger ones round to even)."""
    rng = np.random.default_rng(5)
    wl = wk.small_case(rng, 7, 5, 9, 4, kind, "bf16", "bf16", 0.0, {"bias", "relu"}, integer=True)
    call = wl.calls[0]
    c_out, _ = run_oracle(wl)
    pairs = _blocks(call, wl.arrays)
    dense = sum(A @ B for A, B in pairs) + wl.arrays["bias"].astype(np.float64)[:, None]
    dense = np.maximum(dense, 0.0)
    want = _torch_bf16(dense.astype(np.float32).T.copy())
    got = c_out.reshape(call.n, call.ldc)[:, :call.m]
    assert np.array_equal(got, want)


# ----------------------------------------------------------------------------------------------
# Invariants the paper states
# ----------------------------------------------------------------------------------------------
def test_batch_count_one_is_plain_gemm():
    """Table 3: GEMM C = beta C + A x B is the BRGEMM with one pair."""
    rng = np.random.default_rng(21)
    for (m, n, k) in [(17, 33, 65), (64, 64, 64), (1, 40, 3)]:
        wl = wk.small_case(rng, m, n, k, 1, "stride", "f32", "f32", 0.75, set(), pad=3)
        call = wl.calls[0]
        c0 = values(wl.arrays["c"], "f32").reshape(n, call.ldc)[:, :m].T
        _, ref = run_oracle(wl, want_ref64=True)
        (A, B), = _blocks(call, wl.arrays)
        want = 0.75 * c0 + np.matmul(A, B)
        assert np.allclose(ref[0].T, want, rtol=1e-12, atol=1e-12)


def test_batch_reduce_equals_gemm_over_concatenated_k():
    """sum_i A_i B_i = [A_0 | ... | A_{n-1}] x [B_0; ...; B_{n-1}]."""
    rng = np.random.default_rng(22)
    for kind in ("stride", "offset", "address"):
        wl = wk.small_case(rng, 19, 11, 13, 7, kind, "bf16", "f32", 0.0, set(), pad=2)
        call = wl.calls[0]
        _, ref = run_oracle(wl, want_ref64=True)
        pairs = _blocks(call, wl.arrays)
        A_cat = np.concatenate([A for A, _ in pairs], axis=1)
        B_cat = np.concatenate([B for _, B in pairs], axis=0)
        assert np.allclose(ref[0].T, A_cat @ B_cat, rtol=1e-12, atol=1e-12)


def test_three_variants_name_the_same_blocks():
    """Sec. 2.3: stride s == offsets i*s == addresses A + i*s give identical results."""
    rng = np.random.default_rng(23)
    base = wk.small_case(rng, 9, 6, 10, 5, "stride", "bf16", "bf16", 0.0, {"relu"})
    call = base.calls[0]
    out_s, _ = run_oracle(base)
    off = wk.Workload("o", base.arrays, [wk.Call(**{**call.__dict__, "kind": "offset",
                                                    "grid": None,
                                                    "offs_a": np.arange(5) * call.stride_a,
                                                    "offs_b": np.arange(5) * call.stride_b})])
    out_o, _ = run_oracle(off)
    adr = wk.Workload("p", base.arrays, [wk.Call(**{**call.__dict__, "kind": "address",
                                                    "grid": None,
                                                    "begin": np.array([0, 5]),
                                                    "idx_a": np.arange(5) * call.stride_a,
                                                    "idx_b": np.arange(5) * call.stride_b})])
    out_p, _ = run_oracle(adr)
    assert np.array_equal(out_s, out_o) and np.array_equal(out_s, out_p)


def test_a_and_b_may_alias():
    """Sec. 2.3: A and B may alias.  A_i = B_i = the same square block X gives X @ X."""
    rng = np.random.default_rng(24)
    x = rng.uniform(-1, 1, size=(8 * 8,)).astype(np.float32)
    d = oracle.Desc(8, 8, 8, 8, 8, 8, "f32", "f32", 0.0, "stride", 0, 0, set())
    c = np.zeros(64, dtype=np.float32)
    ref = oracle.brgemm(d, x, x, c, count=3, want_ref64=True)
    X = x.reshape(8, 8).T.astype(np.float64)
    assert np.allclose(ref.T, 3 * X @ X, rtol=1e-12, atol=1e-12)


def test_beta_linearity_and_zero_count():
    rng = np.random.default_rng(25)
    wl = wk.small_case(rng, 12, 10, 8, 3, "offset", "bf16", "f32", 1.0, {"bias"})
    call = wl.calls[0]
    c0 = values(wl.arrays["c"], "f32").reshape(call.n, call.ldc)[:, :call.m]
    refs = {}
    for beta in (0.0, 0.5, -2.0):
        call.beta = beta
        _, refs[beta] = run_oracle(wl, want_ref64=True)
    for beta in (0.5, -2.0):
        assert np.allclose(refs[beta][0] - beta * c0, refs[0.0][0], rtol=0, atol=1e-12)
    # count = 0 gives epi(beta * C)
    call.beta, call.count = 0.5, 0
    call.flags = {"bias", "relu"}
    _, ref = run_oracle(wl, want_ref64=True)
    want = np.maximum(0.5 * c0 + wl.arrays["bias"][None, :].astype(np.float64), 0.0)
    assert np.allclose(ref[0], want, rtol=0, atol=1e-15)


def test_beta_zero_never_reads_c():
    rng = np.random.default_rng(26)
    wl = wk.small_case(rng, 5, 5, 5, 2, "stride", "f32", "f32", 0.0, set())
    assert np.isnan(wl.arrays["c"]).all()
    c_out, _ = run_oracle(wl)
    assert not np.isnan(c_out).any()


def test_epilogue_bias_is_a_column_broadcast_and_relu_gelu_act_on_it():
    rng = np.random.default_rng(27)
    wl = wk.small_case(rng, 6, 9, 4, 2, "stride", "f32", "f32", 0.0, {"bias"})
    call = wl.calls[0]
    _, with_bias = run_oracle(wl, want_ref64=True)
    call.flags = set()
    _, plain = run_oracle(wl, want_ref64=True)
    diff = with_bias[0] - plain[0]                    # [n][m]
    assert np.allclose(diff, np.broadcast_to(wl.arrays["bias"], diff.shape), atol=1e-15)
    call.flags = {"bias", "relu"}
    _, relu = run_oracle(wl, want_ref64=True)
    assert np.array_equal(relu[0], np.maximum(with_bias[0], 0.0))
    call.flags = {"bias", "gelu_tanh"}
    _, gelu = run_oracle(wl, want_ref64=True)
    lib = torch.nn.functional.gelu(torch.from_numpy(with_bias[0]), approximate="tanh").numpy()
    assert np.max(np.abs(gelu[0] - lib)) < 1e-14


def test_output_rounding_is_fp32_then_bf16():
    rng = np.random.default_rng(28)
    wl = wk.small_case(rng, 16, 16, 32, 4, "stride", "bf16", "bf16", 0.0, set())
    c_out, ref = run_oracle(wl, want_ref64=True)
    want = _torch_bf16(ref[0].astype(np.float32))
    assert np.array_equal(c_out.reshape(16, 16), want)


# ----------------------------------------------------------------------------------------------
# The workloads against independent formulations
# ----------------------------------------------------------------------------------------------
def test_conv3x3_offsets_equal_direct_convolution():
    """Sec. 5.1.4 offset-based BRGEMM per output row == torch conv2d (pad 1) on the unpadded
    input; pins the offset lists, the padding and the blocked index maps."""
    wl = wk.conv3x3(seed=3, images=2, h=5, w=7, c=16, k=8)
    out, ref = run_oracle(wl, want_ref64=True)
    x = values(wl.arrays["x"], "bf16").reshape(2, 5, 7, 16)            # NHWc
    wt = values(wl.arrays["wt"], "bf16").reshape(3, 3, 16, 8)          # r s c k
    xt = torch.from_numpy(x).permute(0, 3, 1, 2)                        # N c H W
    wt_t = torch.from_numpy(wt).permute(3, 2, 0, 1)                     # k c r s
    y = torch.relu(torch.nn.functional.conv2d(xt, wt_t, padding=1))    # N k H W
    y = y.permute(0, 2, 3, 1).numpy()                                   # N H W k
    got = ref.reshape(2, 5, 7, 8)                                       # (img, oj) x [ow][k]
    assert np.allclose(got, y, rtol=1e-12, atol=1e-12)
    assert np.array_equal(out, _torch_bf16(y.astype(np.float32)))


def test_mlp_fc_equals_dense_linear_layer():
    """Alg. 6 on the blocked layout == relu(X W^T + b) on unblocked matrices."""
    wl = wk.mlp_fc(seed=2, minibatch=192, c_in=128, k_out=256)
    _, ref = run_oracle(wl, want_ref64=True)
    nb, cb, kb = 3, 2, 4
    x = values(wl.arrays["x"], "bf16").reshape(nb, cb, 64, 64)          # [nb][cb][n][c]
    w = values(wl.arrays["w"], "bf16").reshape(kb, cb, 64, 64)          # [kb][cb][c][k]
    X = x.transpose(0, 2, 1, 3).reshape(nb * 64, cb * 64)               # N x C
    W = w.transpose(1, 2, 0, 3).reshape(cb * 64, kb * 64)               # C x K
    Y = np.maximum(X @ W + wl.arrays["bias"].astype(np.float64), 0.0)   # N x K
    # instance g = kb_i + kb * nb_i holds the (kb_i, nb_i) block as [n][k]
    got = ref.reshape(nb, kb, 64, 64).transpose(0, 2, 1, 3).reshape(nb * 64, kb * 64)
    assert np.allclose(got, Y, rtol=1e-12, atol=1e-12)


def test_mlp_block_gemm1_equals_dense_with_gelu():
    wl = wk.mlp_block(seed=4, tokens=128, hidden=128, inter=192)
    _, ref = run_oracle(wl, 0, want_ref64=True)
    nb, hb, ib = 2, 2, 3
    x = values(wl.arrays["x"], "bf16").reshape(nb, hb, 64, 64)
    w1 = values(wl.arrays["w1"], "bf16").reshape(ib, hb, 64, 64)
    X = x.transpose(0, 2, 1, 3).reshape(nb * 64, hb * 64)
    W1 = w1.transpose(1, 2, 0, 3).reshape(hb * 64, ib * 64)
    pre = torch.from_numpy(X @ W1 + wl.arrays["b1"].astype(np.float64))
    H = torch.nn.functional.gelu(pre, approximate="tanh").numpy()
    got = ref.reshape(nb, ib, 64, 64).transpose(0, 2, 1, 3).reshape(nb * 64, ib * 64)
    assert np.max(np.abs(got - H)) < 1e-12


def test_gathered_equals_sum_of_listed_products():
    wl = wk.gathered(seed=5, n_out=6, pool=10, m=16, n=8, k=4, min_len=0, max_len=5)
    call = wl.calls[0]
    _, ref = run_oracle(wl, want_ref64=True)
    ap = values(wl.arrays["apool"], "bf16").reshape(10, 4, 16)          # [blk][k][m]
    bp = values(wl.arrays["bpool"], "bf16").reshape(10, 8, 4)           # [blk][n][k]
    c0 = wl.arrays["c"].astype(np.float64).reshape(6, 8, 16)            # [g][n][m]
    for g in range(6):
        acc = c0[g].T.copy()
        for j in range(call.begin[g], call.begin[g + 1]):
            A = ap[call.idx_a[j] // 64].T                               # m x k
            B = bp[call.idx_b[j] // 32].T                               # k x n
            acc += A @ B
        assert np.allclose(ref[g].T, acc, rtol=1e-12, atol=1e-12)


def test_selected_instances_match_full_run():
    wl = wk.mlp_fc(seed=2, minibatch=128, c_in=128, k_out=128)
    full, _ = run_oracle(wl)
    sel = np.array([3, 0, 2])
    part, _ = run_oracle(wl, sel=sel)
    blocks_full = full.reshape(2, 2, 64, 64)
    blocks_part = part.reshape(2, 2, 64, 64)
    for g in sel:
        assert np.array_equal(blocks_part[g // 2, g % 2], blocks_full[g // 2, g % 2])
    assert np.all(blocks_part[0, 1] == 0x7FC0)                          # not selected: untouched


# ----------------------------------------------------------------------------------------------
# Reduce TPP
# ----------------------------------------------------------------------------------------------
@pytest.mark.parametrize("in_type", ["f32", "bf16"])
def test_reduce_against_numpy(in_type):
    rng = np.random.default_rng(31)
    m, n, ld = 37, 23, 41
    raw = rng.uniform(0.5, 1.5, size=(n, ld)).astype(np.float32)
    x = raw if in_type == "f32" else wk.bf16_bits(raw)
    X = values(x, in_type).reshape(n, ld)[:, :m].T                      # m x n
    ones = np.ones(n)
    sx, sx2 = oracle.reduce(x, m, n, ld, in_type, "sum", "cols", ("x", "x2"))
    assert np.allclose(sx, X @ ones, rtol=1e-13)
    assert np.allclose(sx2, np.diag(X @ X.T), rtol=1e-13)
    sy, _ = oracle.reduce(x, m, n, ld, in_type, "sum", "rows")
    assert np.allclose(sy, np.ones(m) @ X, rtol=1e-13)
    mx, _ = oracle.reduce(x, m, n, ld, in_type, "max", "cols")
    mn, mn2 = oracle.reduce(x, m, n, ld, in_type, "min", "rows", ("x", "x2"))
    assert np.array_equal(mx, X.max(axis=1)) and np.array_equal(mn, X.min(axis=0))
    assert np.array_equal(mn2, (X * X).min(axis=0))
    pr, _ = oracle.reduce(x, m, n, ld, in_type, "mul", "cols")
    assert np.allclose(pr, np.prod(X, axis=1), rtol=1e-13)


def test_reduce_batchnorm_statistics_of_a_conv_output():
    """Sec. 5.1.2: per-channel sum and sum of squares over N, H, W of an NHWc tensor."""
    rng = np.random.default_rng(32)
    t = wk.bf16_bits(rng.standard_normal((3, 4, 5, 16)).astype(np.float32))
    sx, sx2 = oracle.reduce(t.reshape(-1), 16, 60, 16, "bf16", "sum", "cols", ("x", "x2"))
    v = values(t, "bf16")
    assert np.allclose(sx, v.sum(axis=(0, 1, 2)), rtol=1e-12)
    assert np.allclose(sx2, (v * v).sum(axis=(0, 1, 2)), rtol=1e-12)


# ----------------------------------------------------------------------------------------------
# Argument checking
# ----------------------------------------------------------------------------------------------
def test_oracle_rejects_bad_descriptors():
    x = np.zeros(16, dtype=np.float32)
    for bad in (dict(m=0), dict(lda=1), dict(flags={"relu", "gelu_tanh"})):
        kw = dict(m=4, n=4, k=4, lda=4, ldb=4, ldc=4, ab_type="f32", c_type="f32",
                  kind="stride", stride_a=0, stride_b=0, flags=set())
        kw.update(bad)
        with pytest.raises(ValueError):
            oracle.brgemm(oracle.Desc(**kw), x, x, x.copy(), count=1)


@pytest.mark.parametrize("kind", ["stride", "offset", "address"])
def test_a_trans_layout_is_the_transposed_block(kind):
    """The transposed-A layout (element (r, p) of A_i at r * lda + p) gives the bit-identical
    result of the column-major layout holding the numpy transpose of each block, for every batch
    variant, with a padded lda; a lda below k is rejected."""
    rng = np.random.default_rng(61)
    m, n, k, count = 24, 20, 32, 5
    lda_t = k + 3
    blocks = rng.uniform(-1, 1, (count, k, m)).astype(np.float32)        # block i: A_i[r, p] = blocks[i, p, r]
    plain = wk.bf16_bits(blocks.reshape(-1))                              # column-major, lda = m
    tr = np.zeros((count, m, lda_t), np.float32)
    tr[:, :, :k] = np.swapaxes(blocks, 1, 2)                              # row r holds A_i[r, :]
    trans = wk.bf16_bits(tr.reshape(-1))
    b = wk.bf16_bits(rng.uniform(-1, 1, count * k * n).astype(np.float32))
    outs = []
    for a, lda, flags, step in ((plain, m, set(), m * k), (trans, lda_t, {"a_trans"}, m * lda_t)):
        c = np.full(m * n, np.nan, np.float32)
        d = oracle.Desc(m, n, k, lda, k, m, "bf16", "f32", 0.0, kind,
                        step if kind == "stride" else 0, k * n if kind == "stride" else 0, flags)
        if kind == "stride":
            oracle.brgemm(d, a, b, c, count=count)
        elif kind == "offset":
            oracle.brgemm(d, a, b, c, count=count, offs_a=np.arange(count) * step,
                          offs_b=np.arange(count) * k * n)
        else:
            oracle.brgemm(d, a, b, c, idx_a=np.arange(count) * step, idx_b=np.arange(count) * k * n)
        outs.append(c)
    assert np.array_equal(outs[0], outs[1]) and not np.isnan(outs[0]).any()
    with pytest.raises(ValueError):
        oracle.brgemm(oracle.Desc(m, n, k, k - 1, k, m, "bf16", "f32", 0.0, "stride", m * k, k * n,
                                  {"a_trans"}), trans, b, np.zeros(m * n, np.float32), count=1)


@pytest.mark.parametrize("kind", ["stride", "offset", "address"])
def test_b_trans_layout_is_the_transposed_block(kind):
    """The transposed-B layout (element (p, c) of B_i at p * ldb + c) gives the bit-identical
    result of the column-major layout holding numpy's transpose of each block; ldb below n is
    rejected."""
    rng = np.random.default_rng(62)
    m, n, k, count = 24, 16, 32, 5
    ldb_t = n + 5
    blocks = rng.uniform(-1, 1, (count, n, k)).astype(np.float32)        # block i: B_i[p, c] = blocks[i, c, p]
    plain = wk.bf16_bits(blocks.reshape(-1))                              # column-major, ldb = k
    tr = np.zeros((count, k, ldb_t), np.float32)
    tr[:, :, :n] = np.swapaxes(blocks, 1, 2)                              # k-row p holds B_i[p, :]
    trans = wk.bf16_bits(tr.reshape(-1))
    a = wk.bf16_bits(rng.uniform(-1, 1, count * m * k).astype(np.float32))
    outs = []
    for b, ldb, flags, step in ((plain, k, set(), k * n), (trans, ldb_t, {"b_trans"}, k * ldb_t)):
        c = np.full(m * n, np.nan, np.float32)
        d = oracle.Desc(m, n, k, m, ldb, m, "bf16", "f32", 0.0, kind,
                        m * k if kind == "stride" else 0, step if kind == "stride" else 0, flags)
        if kind == "stride":
            oracle.brgemm(d, a, b, c, count=count)
        elif kind == "offset":
            oracle.brgemm(d, a, b, c, count=count, offs_a=np.arange(count) * m * k,
                          offs_b=np.arange(count) * step)
        else:
            oracle.brgemm(d, a, b, c, idx_a=np.arange(count) * m * k, idx_b=np.arange(count) * step)
        outs.append(c)
    assert np.array_equal(outs[0], outs[1]) and not np.isnan(outs[0]).any()
    with pytest.raises(ValueError):
        oracle.brgemm(oracle.Desc(m, n, k, m, n - 1, m, "bf16", "f32", 0.0, "stride", m * k, k * n,
                                  {"b_trans"}), a, trans, np.zeros(m * n, np.float32), count=1)
