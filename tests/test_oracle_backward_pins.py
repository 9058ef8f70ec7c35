"""Pins of the oracle's back-propagation pieces (CPU only).

The inverse activations of Table 1 (RELU_inv, GELU_inv) fused after the BRGEMM, the
pre-activation kept by a forward call, the loops of Alg. 6 around the Reduce and Transform TPPs,
and the whole backward pass of the transformer MLP (Sec. 5.1.6 builds the back-propagation of the
fully-connected layer from the same TPPs) are checked against what does not come from the
oracle: torch autograd in float64, numpy, central differences, and exact integer arithmetic.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import workloads as wk
from helpers import oracle_desc, rel_fro, run_call_oracle, run_steps_oracle, values

BLK = wk.BLK


def _torch_gelu_grad(x: np.ndarray) -> np.ndarray:
    t = torch.tensor(x, dtype=torch.float64, requires_grad=True)
    torch.nn.functional.gelu(t, approximate="tanh").sum().backward()
    return t.grad.numpy()


def test_gelu_grad_matches_torch_autograd():
    xs = np.concatenate([np.linspace(-12.0, 12.0, 2401), [0.0, -0.0, 1e-8, -1e-8, 30.0, -30.0]])
    ours = np.array([oracle.gelu_tanh_grad(x) for x in xs])
    ref = _torch_gelu_grad(xs)
    # absolute slack for the far tails, where 0.5 (1 + tanh u) cancels in both formulas
    np.testing.assert_allclose(ours, ref, rtol=1e-13, atol=1e-14)


def test_gelu_grad_is_derivative_of_gelu():
    # central differences of the oracle's own GELU: the derivative pins the forward and the
    # inverse to each other (a dropped term in either shows)
    h = 1e-5
    for x in np.linspace(-6.0, 6.0, 241):
        fd = (oracle.gelu_tanh(x + h) - oracle.gelu_tanh(x - h)) / (2 * h)
        assert abs(fd - oracle.gelu_tanh_grad(x)) < 1e-8, x
    assert oracle.gelu_tanh_grad(0.0) == 0.5
    assert abs(oracle.gelu_tanh_grad(40.0) - 1.0) < 1e-15 and abs(oracle.gelu_tanh_grad(-40.0)) < 1e-15


def _one_block(rng, m, n, k, count, flags, c_type="bf16", integer=True):
    wl = wk.small_case(rng, m, n, k, count, "stride", "bf16", c_type, 0.0, flags, integer=integer)
    call = wl.calls[0]
    return wl, call


def _dense_sum(wl, call):
    """sum_i A_i B_i in float64 by numpy from the operand arrays (column-major blocks)."""
    a, b = values(wl.arrays["a"], "bf16"), values(wl.arrays["b"], "bf16")
    s = np.zeros((call.m, call.n))
    for i in range(call.count):
        ai = a[i * call.stride_a:][: call.lda * call.k].reshape(call.k, call.lda).T[: call.m]
        bi = b[i * call.stride_b:][: call.ldb * call.n].reshape(call.n, call.ldb).T[: call.k]
        s += ai @ bi
    return s


@pytest.mark.parametrize("c_type", ["bf16", "f32"])
def test_relu_inv_masks_exactly(c_type):
    rng = np.random.default_rng(31)
    wl, call = _one_block(rng, 48, 40, 32, 3, {"relu_inv"}, c_type)
    zv = rng.integers(-3, 4, size=wl.arrays["c"].shape).astype(np.float32)
    zv[:5] = 0.0                                   # the derivative at 0 is taken as 0
    z = zv if c_type == "f32" else wk.bf16_bits(zv)
    arrs = dict(wl.arrays, z=z)
    call.aux = "z"
    run_call_oracle(call, arrs)
    s = _dense_sum(wl, call)                       # integers: exact in every format
    want = np.where(zv.reshape(call.n, call.ldc).T[: call.m] > 0, s, 0.0)
    if c_type == "bf16":   # sums past 256 round in bf16: torch's rounding of the exact value
        want = values(wk.bf16_bits(want.astype(np.float32)), "bf16")
    got = values(arrs["c"], c_type).reshape(call.n, call.ldc).T[: call.m]
    assert np.array_equal(got, want)
    assert np.array_equal(arrs["z"], z)            # aux is read only


def test_gelu_inv_unrounded_matches_autograd():
    rng = np.random.default_rng(32)
    wl, call = _one_block(rng, 64, 24, 48, 4, {"gelu_tanh_inv"}, "bf16", integer=False)
    zv = (rng.standard_normal(wl.arrays["c"].shape) * 2.0).astype(np.float32)
    arrs = dict(wl.arrays, z=wk.bf16_bits(zv))
    call.aux = "z"
    ref = run_call_oracle(call, arrs, want_ref64=True)[0].T      # m x n, unrounded
    zb = values(arrs["z"], "bf16").reshape(call.n, call.ldc).T[: call.m]
    want = _dense_sum(wl, call) * _torch_gelu_grad(zb)
    np.testing.assert_allclose(ref, want, rtol=1e-12, atol=1e-12)


def test_save_preact_equals_bias_only_forward():
    rng = np.random.default_rng(33)
    for act in ("gelu_tanh", "relu"):
        wl, call = _one_block(rng, 64, 64, 64, 5, {"bias", act, "save_preact"}, integer=False)
        arrs = dict(wl.arrays, z=np.full_like(wl.arrays["c"], 0x7FC0))
        call.aux = "z"
        run_call_oracle(call, arrs)
        plain = dict(wl.arrays, c=np.array(wl.arrays["c"], copy=True))
        fwd = wk.Call(**{**call.__dict__, "flags": {"bias"}, "aux": None})
        run_call_oracle(fwd, plain)
        assert np.array_equal(arrs["z"], plain["c"])           # the saved Z
        act_only = dict(wl.arrays, c=np.array(wl.arrays["c"], copy=True))
        run_call_oracle(wk.Call(**{**call.__dict__, "flags": {"bias", act}, "aux": None}), act_only)
        assert np.array_equal(arrs["c"], act_only["c"])        # the output is unchanged


@pytest.mark.parametrize("flags", [{"relu_inv", "gelu_tanh_inv"}, {"relu_inv", "relu"},
                                   {"gelu_tanh_inv", "gelu_tanh"}, {"save_preact"},
                                   {"save_preact", "bias"}, {"gelu_tanh_inv", "save_preact"}])
def test_bad_inverse_flag_combinations_rejected(flags):
    rng = np.random.default_rng(34)
    wl, call = _one_block(rng, 8, 8, 8, 1, flags)
    arrs = dict(wl.arrays, z=np.zeros_like(wl.arrays["c"]))
    call.aux = "z"
    with pytest.raises(ValueError):
        run_call_oracle(call, arrs)


def test_aux_flags_need_the_aux_tensor():
    rng = np.random.default_rng(35)
    wl, call = _one_block(rng, 8, 8, 8, 1, {"relu_inv"})
    with pytest.raises(ValueError):
        run_call_oracle(call, dict(wl.arrays))


def test_transform_batched_is_blockwise_transpose():
    rng = np.random.default_rng(36)
    x = rng.integers(0, 65535, size=(6, 5, 24, 40)).astype(np.uint16)   # 30 blocks, 40 x 24
    out = np.full((6, 5, 40, 24), 7, dtype=np.uint16)
    oracle.transform_batched("transpose", 40, 24, 40, 24, "bf16", 1, x, 40 * 24, out, 40 * 24, 30)
    assert np.array_equal(out, np.swapaxes(x, 2, 3))


def test_reduce_batched_is_blockwise_reduce():
    rng = np.random.default_rng(37)
    x = rng.standard_normal((7, 16, 24)).astype(np.float32)   # 7 blocks of 24 x 16 (ld 24)
    ox, ox2 = oracle.reduce_batched(x, 24, 16, 24, "f32", 7, 16 * 24, "sum", "cols", ("x", "x2"),
                                    out_stride=30)
    for g in range(7):
        blk = x[g].astype(np.float64).T                        # 24 x 16
        np.testing.assert_allclose(ox[g * 30: g * 30 + 24], blk.sum(1), rtol=1e-13)
        np.testing.assert_allclose(ox2[g * 30: g * 30 + 24], (blk * blk).sum(1), rtol=1e-13)
        assert not ox[g * 30 + 24: g * 30 + 30].any()          # gaps untouched


# ---- the whole backward pass against torch autograd on the dense layer ----------------------

def _dense_act(arr, nb, fb):   # activations [Nb][Fb][64n][64f] -> (F x N)
    return values(arr, "bf16" if arr.dtype == np.uint16 else "f32").reshape(nb, fb, BLK, BLK) \
        .transpose(1, 3, 0, 2).reshape(fb * BLK, nb * BLK)


def _dense_w(arr, ob, ib):     # weights [Ob][Ib][64i][64o] -> (O x I)
    return values(arr, "bf16" if arr.dtype == np.uint16 else "f32").reshape(ob, ib, BLK, BLK) \
        .transpose(0, 3, 1, 2).reshape(ob * BLK, ib * BLK)


def test_backward_chain_matches_autograd():
    tokens, hidden, inter = 256, 128, 256
    nb, hb, ib = tokens // BLK, hidden // BLK, inter // BLK
    wl = wk.mlp_backward(seed=38, tokens=tokens, hidden=hidden, inter=inter)
    out = run_steps_oracle(wl)
    a = wl.arrays
    X = torch.tensor(_dense_act(a["x"], nb, hb), requires_grad=True)
    W1 = torch.tensor(_dense_w(a["w1"], ib, hb), requires_grad=True)
    b1 = torch.tensor(a["b1"].astype(np.float64), requires_grad=True)
    W2 = torch.tensor(_dense_w(a["w2"], hb, ib), requires_grad=True)
    dY = torch.tensor(_dense_act(a["dy"], nb, hb))
    Z = W1 @ X + b1[:, None]
    Y = W2 @ torch.nn.functional.gelu(Z, approximate="tanh")
    Y.backward(dY)
    # the oracle keeps Z, H and dZ in bf16 as the library does, hence the few-1e-3 agreement;
    # a transposed or misplaced block would be off by O(1)
    checks = [("dx", _dense_act(out["dx"], nb, hb), X.grad), ("dw1", _dense_w(out["dw1"], ib, hb), W1.grad),
              ("db1", out["db1"].astype(np.float64), b1.grad),
              ("dw2", _dense_w(out["dw2"], hb, ib), W2.grad),
              ("db2", out["db2"].astype(np.float64), dY.sum(1))]
    for name, got, ref in checks:
        e = rel_fro(got, ref.detach().numpy())
        assert e < 1.5e-2, (name, e)
    # tight: each gradient from the oracle's own bf16 intermediates, by numpy matmuls
    Hb = _dense_act(out["h"], nb, ib)
    dZb = _dense_act(out["dz"], nb, ib)
    dYd = dY.numpy()
    tight = [("dw2", _dense_w(out["dw2"], hb, ib), dYd @ Hb.T),
             ("db2", out["db2"], dYd.sum(1)),
             ("dw1", _dense_w(out["dw1"], ib, hb), dZb @ X.detach().numpy().T),
             ("db1", out["db1"], dZb.sum(1)),
             ("dx", _dense_act(out["dx"], nb, hb), W1.detach().numpy().T @ dZb)]
    for name, got, ref in tight:
        e = rel_fro(got, ref)
        assert e < (4e-3 if name == "dx" else 1e-6), (name, e)   # dx is bf16, the rest fp32
    # dZ itself: the bf16 rounding of (W2^T dY) * gelu'(Z) at the saved Z
    Zs = _dense_act(out["z"], nb, ib)
    dz_ref = (W2.detach().numpy().T @ dYd) * _torch_gelu_grad(Zs)
    assert rel_fro(dZb, dz_ref) < 4e-3
