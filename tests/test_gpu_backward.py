"""GPU parity of the back-propagation pieces, through the C ABI, against the CPU oracle.

- The aux epilogue bits (SAVE_PREACT in the forward call, RELU_INV and GELU_TANH_INV after the
  data-gradient BRGEMM; Table 1's inverse activations) on every kernel instance.
- The batched Transform and Reduce TPPs (the loops of Alg. 6 around a TPP).
- The transformer MLP's backward pass (Sec. 5.1.6 builds the backward pass of the fully-connected
  layer from the same TPPs): step by step on the oracle's own inputs, end to end, and at full size
  on sampled output blocks.
Bars as for the forward path: bit-exact on small-integer data and for data movement, relative
Frobenius error <= 5e-3 with bf16 involved (<= 1e-5 for fp32 in and out).
"""
from __future__ import annotations

import sys
import zlib

import numpy as np
import pytest
import torch

import oracle
import workloads as wk
from helpers import rel_fro, run_call_oracle, run_step_oracle, run_steps_oracle, values

pytestmark = pytest.mark.gpu
BLK = wk.BLK


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    import paper_2104_05755_amd  # noqa: F401  (fails loudly if the HIP library is missing)
    return torch.device("cuda:0")


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def gpu_steps(steps, arrays, names=None):
    """Run steps on the GPU from host arrays; host copies of the named (default: all) arrays."""
    from paper_2104_05755_amd import torch_io
    dev = torch_io.upload(wk.Workload("x", arrays, []))
    for st in steps:
        torch_io.launch_step(torch_io.prepare_step(st, dev), dev)
    torch.cuda.synchronize()
    return {k: torch_io.to_host(dev[k], arrays[k]) for k in (names or arrays)}


def tol(ab, ct):
    return 1e-5 if (ab == "f32" and ct == "f32") else 5e-3


# ---- aux epilogue bits on every kernel instance -------------------------------------------
KERNELS = [0, 1, 2, 3, 5, 6, 7, 8, 9, 10, 11]
AUX_FLAGS = [("relu_inv",), ("gelu_tanh_inv",), ("bias", "relu_inv"),
             ("bias", "relu", "save_preact"), ("bias", "gelu_tanh", "save_preact")]


@pytest.mark.parametrize("flags", AUX_FLAGS)
@pytest.mark.parametrize("kid", KERNELS)
def test_aux_epilogue_every_kernel(kid, flags, monkeypatch):
    monkeypatch.setenv("TPP_FORCE_KERNEL", str(kid))
    gelu = any("gelu" in f for f in flags)
    rng = np.random.default_rng(kid * 100 + len(flags) * 7 + gelu)
    # a strided grid of 3 x 2 instances of 72 x 64 blocks (ragged for every tile shape), k = 64
    m, n, k, count = 72, 64, 64, 3
    integer = not gelu
    draw = (lambda s: rng.integers(-3, 4, size=s).astype(np.float32)) if integer else \
        (lambda s: rng.standard_normal(s).astype(np.float32))
    gm, gn = 3, 2
    a = wk.bf16_bits(draw((gm * count * k * m,)))
    b = wk.bf16_bits(draw((gn * count * n * k,)))
    zv = draw((gm * gn * m * n,)) * (1.0 if integer else 1.5)
    arrays = dict(a=a, b=b, c=np.full(gm * gn * m * n, 0x7FC0, np.uint16),
                  bias=draw((gm * m,)),
                  z=wk.bf16_bits(zv) if "save_preact" not in flags else
                  np.full(gm * gn * m * n, 0x7FC0, np.uint16))
    call = wk.Call(m, n, k, m, k, m, "bf16", "bf16", 0.0, "stride", k * m, n * k, set(flags),
                   G=gm * gn, grid=dict(gm=gm, gn=gn, a_step_m=count * k * m,
                                        b_step_n=count * n * k, c_step_m=m * n,
                                        c_step_n=gm * m * n, bias_step_m=m),
                   count=count, a="a", b="b", c="c", bias="bias" if "bias" in flags else None,
                   aux="z")
    say(f"aux epilogue kernel {kid} flags {flags}")
    ref = {k2: np.array(v, copy=True) for k2, v in arrays.items()}
    run_call_oracle(call, ref)
    got = gpu_steps([call], arrays, ["c", "z"])
    if integer:
        assert np.array_equal(got["c"], ref["c"])
        assert np.array_equal(got["z"], ref["z"])
    else:
        assert rel_fro(values(got["c"], "bf16"), values(ref["c"], "bf16")) <= 5e-3
        assert rel_fro(values(got["z"], "bf16"), values(ref["z"], "bf16")) <= 5e-3


@pytest.mark.parametrize("ab,ct", [("f32", "f32"), ("bf16", "f32"), ("f32", "bf16")])
@pytest.mark.parametrize("flags", [("gelu_tanh_inv",), ("bias", "relu_inv"),
                                   ("bias", "gelu_tanh", "save_preact")])
def test_aux_epilogue_other_types(ab, ct, flags):
    rng = np.random.default_rng(zlib.crc32(repr((ab, ct, flags)).encode()))
    wl = wk.small_case(rng, 40, 24, 16, 3, "stride", ab, ct, 0.5, set(flags), pad=3)
    zv = (rng.standard_normal(wl.arrays["c"].shape) * 1.5).astype(np.float32)
    arrays = dict(wl.arrays, z=zv if ct == "f32" else wk.bf16_bits(zv))
    call = wl.calls[0]
    call.aux = "z"
    say(f"aux epilogue {ab}->{ct} {flags}")
    ref = {k: np.array(v, copy=True) for k, v in arrays.items()}
    run_call_oracle(call, ref)
    got = gpu_steps([call], arrays, ["c", "z"])
    live = lambda x: values(x, ct).reshape(call.n, call.ldc)[:, : call.m]
    assert rel_fro(live(got["c"]), live(ref["c"])) <= tol(ab, ct)
    assert rel_fro(live(got["z"]), live(ref["z"])) <= tol(ab, ct)


def test_aux_call_needs_aux_and_plain_calls_refuse_aux_handles():
    import paper_2104_05755_amd as tpp
    h = tpp.tpp_brgemm_dispatch(tpp.make_desc(64, 64, 64, 64, 64, 64, "bf16", "bf16",
                                              flags=("relu_inv",)))
    x = torch.zeros(64 * 64, dtype=torch.int16, device="cuda")
    with pytest.raises(tpp.TppError):
        tpp.tpp_brgemm_execute_batched(h, dict(gm=1, gn=1, a_step_m=0, b_step_n=0, c_step_m=0,
                                               c_step_n=0, bias_step_m=0), 1, None, None, None,
                                       None, x, x, x, None, 1, None, None, None, None, None)
    with pytest.raises(tpp.TppError):
        tpp.tpp_brgemm_execute_batched_aux(h, dict(gm=1, gn=1, a_step_m=0, b_step_n=0,
                                                   c_step_m=0, c_step_n=0, bias_step_m=0), 1,
                                           None, None, None, None, x, x, x, None, None, 1, None,
                                           None, None, None, None)
    with pytest.raises(tpp.TppError):
        tpp.tpp_brgemm_execute_stride(h, x, x, x, None, 1)


# ---- batched Transform and Reduce ---------------------------------------------------------
TR_CASES = [("transpose", 64, 64, 64, 64, "bf16", 1, 37, 4096, 4096),
            ("transpose", 40, 24, 40, 24, "bf16", 1, 5, 1000, 977),     # ragged, unaligned
            ("transpose", 64, 64, 64, 64, "f32", 1, 9, 4096, 4100),
            ("transpose", 130, 70, 136, 72, "bf16", 1, 3, 136 * 70, 72 * 130 + 8),
            ("vnni", 64, 64, 64, 128, "bf16", 2, 6, 4096, 4096),
            ("vnni_t", 32, 64, 64, 128, "bf16", 2, 4, 2048, 4096)]


@pytest.mark.parametrize("case", TR_CASES, ids=lambda c: f"{c[0]}-{c[1]}x{c[2]}-{c[5]}-G{c[7]}")
def test_transform_batched_bit_exact(case):
    kind, m, n, ld_in, ld_out, dt, alpha, G, s_in, s_out = case
    rng = np.random.default_rng(G * 31 + m)
    npdt = np.uint16 if dt == "bf16" else np.uint32
    src = rng.integers(0, np.iinfo(npdt).max, size=G * s_in + 64, dtype=np.uint64).astype(npdt)
    n_out = oracle.transform_out_len(kind, m, n, ld_out, alpha)
    dst = np.full(G * s_out + n_out + 64, 0xA5A5 if dt == "bf16" else 0xA5A5A5A5, dtype=npdt)
    view = (lambda x: x) if dt == "bf16" else (lambda x: x.view(np.float32))
    ref = view(np.array(dst, copy=True))
    oracle.transform_batched(kind, m, n, ld_in, ld_out, dt, alpha, view(src), s_in, ref, s_out, G)
    st = wk.TransformStep(kind, m, n, ld_in, ld_out, dt, "src", "dst", G=G, in_stride=s_in,
                          out_stride=s_out, alpha=alpha)
    say(f"transform batched {case}")
    got = gpu_steps([st], dict(src=view(src), dst=view(np.array(dst, copy=True))), ["dst"])["dst"]
    assert np.array_equal(got.view(npdt), ref.view(npdt))


RED_CASES = [(64, 64, 64, "f32", 16, 4096, 64, "cols", "sum"),
             (64, 64, 64, "bf16", 16, 4096, 80, "cols", "max"),
             (1024, 128, 1024, "bf16", 3, 1024 * 128, 1100, "cols", "sum"),
             (512, 40, 520, "f32", 5, 520 * 40 + 7, 50, "rows", "sum"),
             (3000, 6, 3000, "bf16", 4, 3000 * 6, 6, "rows", "min")]


@pytest.mark.parametrize("case", RED_CASES, ids=lambda c: f"{c[0]}x{c[1]}-{c[3]}-G{c[4]}-{c[7]}-{c[8]}")
def test_reduce_batched_matches_oracle(case):
    m, n, ld, dt, G, s_in, s_out, by, op = case
    rng = np.random.default_rng(m + G)
    xv = rng.standard_normal(G * s_in + ld * n).astype(np.float32)
    x = xv if dt == "f32" else wk.bf16_bits(xv)
    nout = m if by == "cols" else n
    ox, ox2 = oracle.reduce_batched(x, m, n, ld, dt, G, s_in, op, by, ("x", "x2"), out_stride=s_out)
    size = (G - 1) * s_out + nout
    st = wk.ReduceStep("x", m, n, ld, dt, op, by, dst_x="ox", dst_x2="ox2", G=G, in_stride=s_in,
                       out_stride=s_out)
    say(f"reduce batched {case}")
    fill = np.full(size, -7.0, dtype=np.float32)
    got = gpu_steps([st], dict(x=x, ox=fill, ox2=fill.copy()), ["ox", "ox2"])
    for g in range(G):
        sl = slice(g * s_out, g * s_out + nout)
        if op == "sum":
            blk = values(x, dt)[g * s_in:][: ld * n].reshape(n, ld)[:, :m]
            scale = np.abs(blk).sum(axis=0) if by == "cols" else np.abs(blk).sum(axis=1)
            assert np.all(np.abs(got["ox"][sl] - ox[sl]) <= 1e-5 * scale + 1e-30)
            np.testing.assert_allclose(got["ox2"][sl], ox2[sl], rtol=1e-5)
        else:
            assert np.array_equal(got["ox"][sl], ox[sl].astype(np.float32))
        gap = slice(g * s_out + nout, (g + 1) * s_out) if g + 1 < G else slice(0, 0)
        assert np.all(got["ox"][gap] == -7.0)   # between the calls' outputs nothing is written


# ---- the MLP backward pass ----------------------------------------------------------------
def _outputs(st):
    if isinstance(st, wk.Call):
        return [st.c] + ([st.aux] if "save_preact" in st.flags else [])
    if isinstance(st, wk.TransformStep):
        return [st.dst]
    return [d for d in (st.dst_x, st.dst_x2) if d]


def _compare(name, got, ref, st):
    if isinstance(st, wk.TransformStep):
        assert np.array_equal(got, ref), name
        return
    dt = "bf16" if got.dtype == np.uint16 else "f32"
    g, r = values(got, dt), values(ref, dt)
    assert not np.isnan(g).any(), f"{name}: NaN"
    bar = 5e-3 if (dt == "bf16" or (isinstance(st, wk.Call) and st.ab_type == "bf16")) else 1e-5
    e = rel_fro(g, r)
    assert e <= bar, f"{name}: rel Frobenius error {e:.3e} > {bar}"


def test_mlp_backward_step_by_step():
    """Each step on the oracle's inputs for it, against the oracle's output of that step."""
    wl = wk.mlp_backward(seed=41, tokens=320, hidden=192, inter=256)
    state = {k: np.array(v, copy=True) for k, v in wl.arrays.items()}
    for i, st in enumerate(wl.steps):
        say(f"backward step {i}: {type(st).__name__} -> {_outputs(st)}")
        got = gpu_steps([st], state, _outputs(st))
        run_step_oracle(st, state)
        for name in _outputs(st):
            _compare(f"step {i} {name}", got[name], state[name], st)


def test_mlp_backward_end_to_end():
    wl = wk.mlp_backward(seed=42, tokens=256, hidden=128, inter=256)
    say("backward end to end")
    ref = run_steps_oracle(wl)
    got = gpu_steps(wl.steps, wl.arrays, ["dx", "dw1", "db1", "dw2", "db2", "dz", "z", "h"])
    for name, st in (("z", wl.steps[0]), ("dz", wl.calls[1]), ("dw2", wl.calls[2]),
                     ("dx", wl.calls[3]), ("dw1", wl.calls[4])):
        _compare(name, got[name], ref[name], st)
    for name in ("db1", "db2"):
        assert rel_fro(got[name], ref[name]) <= 5e-3, name


def _blocks(flat, call, insts):
    gm = call.grid["gm"]
    out = []
    for g in insts:
        off = (g % gm) * call.grid["c_step_m"] + (g // gm) * call.grid["c_step_n"]
        idx = off + np.arange(call.n)[:, None] * call.ldc + np.arange(call.m)[None, :]
        out.append(flat.reshape(-1)[idx])
    return np.stack(out)


def test_mlp_backward_full_size_sampled():
    """Full size (8192 tokens, 1024 -> 4096 -> 1024) on the GPU; the oracle computes the sampled
    output blocks and the blocks of the intermediates they depend on, no more."""
    wl = wk.mlp_backward()
    fwd, b1, b2, b3, b4 = wl.calls
    nb, hb, ib = fwd.grid["gn"], b3.grid["gm"], fwd.grid["gm"]
    say(f"backward full size: tokens {nb * BLK}, hidden {hb * BLK}, inter {ib * BLK}")
    got = gpu_steps(wl.steps, wl.arrays, ["z", "dz", "dx", "dw1", "dw2", "db1", "db2"])
    ibs, nbs, hbs = [0, 37, ib - 1], [0, 77, nb - 1], [0, 9, hb - 1]
    arrs = {k: np.array(v, copy=True) for k, v in wl.arrays.items()}
    # instances (i, n) of the forward and of dZ that the sampled dX, dW1 and dW2 blocks read
    sel_in = sorted({i + ib * n for i in range(ib) for n in range(nb) if i in ibs or n in nbs})
    run_call_oracle(fwd, arrs, sel=sel_in)
    for st in wl.steps:                            # the block transposes, whole
        if isinstance(st, wk.TransformStep):
            run_step_oracle(st, arrs)
    run_call_oracle(b1, arrs, sel=sel_in)
    checks = [(fwd, "z", [i + ib * n for i in ibs for n in nbs]), (b1, "dz", sel_in[::7]),
              (b2, "dw2", [h + hb * i for h in hbs for i in ibs]),
              (b3, "dx", [h + hb * n for h in hbs for n in nbs]),
              (b4, "dw1", [i + ib * h for i in ibs for h in hbs])]
    for call, name, sel in checks:
        if call in (b2, b3, b4):
            run_call_oracle(call, arrs, sel=sel)
        dt = call.c_type if name != "z" else "bf16"
        g = values(_blocks(got[name], call, sel), dt)
        r = values(_blocks(arrs[name], call, sel), dt)
        e = rel_fro(g, r)
        say(f"  {name}: {len(sel)} blocks, rel err {e:.2e}")
        assert not np.isnan(g).any() and e <= 5e-3, (name, e)
    # bias gradients: db2 whole (dY is an input); db1 on the sampled feature blocks, from the
    # oracle's dZ blocks of every token block
    # dY as a column-major (hb * 4096) x nb matrix: row h + 64 n + 4096 hb, column = token block
    ox, _ = oracle.reduce(wl.arrays["dy"].reshape(-1), hb * BLK * BLK, nb, hb * BLK * BLK,
                          "bf16", "sum", "cols")
    db2 = ox.reshape(hb, BLK, BLK).sum(axis=1)
    assert rel_fro(got["db2"], db2.reshape(-1)) <= 5e-3
    dz = arrs["dz"].reshape(nb, ib, BLK, BLK)
    for i in ibs:
        blk = np.ascontiguousarray(dz[:, i]).reshape(-1)   # 64 x (nb * 64), column-major
        o, _ = oracle.reduce(blk, BLK, nb * BLK, BLK, "bf16", "sum", "cols")
        assert rel_fro(got["db1"][i * BLK:(i + 1) * BLK], o) <= 5e-3


# ---- split stage lists (long batch reductions on grids of few tiles) -----------------------
DL_KERNELS = [5, 6, 7, 8, 9, 10, 11]


@pytest.mark.parametrize("split", [2, 3, 5])
@pytest.mark.parametrize("kid", DL_KERNELS)
def test_split_stage_list_integer_bit_exact(kid, split, monkeypatch):
    """Every direct-LDS instance with its stage list split into chunks (partial tiles summed in
    chunk order by the finishing kernel): bit-exact on small-integer data, with the bias, the
    ReLU_inv aux step and a ragged strided grid, for bf16 and fp32 outputs."""
    monkeypatch.setenv("TPP_FORCE_KERNEL", str(kid))
    monkeypatch.setenv("TPP_SPLIT", str(split))
    rng = np.random.default_rng(kid * 10 + split)
    m, n, k, count, gm, gn = 72, 64, 64, 7, 3, 2
    draw = lambda s: rng.integers(-3, 4, size=s).astype(np.float32)
    for ct in ("bf16", "f32"):
        a = wk.bf16_bits(draw((gm * count * k * m,)))
        b = wk.bf16_bits(draw((gn * count * n * k,)))
        zv = draw((gm * gn * m * n,))
        fill = np.full(gm * gn * m * n, 0x7FC0, np.uint16) if ct == "bf16" else \
            np.full(gm * gn * m * n, np.nan, np.float32)
        arrays = dict(a=a, b=b, c=fill, bias=draw((gm * m,)),
                      z=wk.bf16_bits(zv) if ct == "bf16" else zv)
        call = wk.Call(m, n, k, m, k, m, "bf16", ct, 0.0, "stride", k * m, n * k,
                       {"bias", "relu_inv"}, G=gm * gn,
                       grid=dict(gm=gm, gn=gn, a_step_m=count * k * m, b_step_n=count * n * k,
                                 c_step_m=m * n, c_step_n=gm * m * n, bias_step_m=m),
                       count=count, a="a", b="b", c="c", bias="bias", aux="z")
        say(f"split {split} kernel {kid} {ct}")
        ref = {k2: np.array(v, copy=True) for k2, v in arrays.items()}
        run_call_oracle(call, ref)
        got = gpu_steps([call], arrays, ["c"])["c"]
        assert np.array_equal(got, ref["c"])


@pytest.mark.parametrize("case", ["bias_relu", "beta1", "m68"])
@pytest.mark.parametrize("split", [2, 3])
@pytest.mark.parametrize("kid", [6, 9, 10, 11])
def test_split_finish_epilogue_bit_exact(kid, split, case, monkeypatch):
    """The finishing kernel's epilogue on small-integer data without an aux step: bias + ReLU,
    beta = 1 reading C, and m = 68 (four-row groups that are not eight-row aligned), over a
    ragged strided grid."""
    monkeypatch.setenv("TPP_FORCE_KERNEL", str(kid))
    monkeypatch.setenv("TPP_SPLIT", str(split))
    rng = np.random.default_rng(kid * 100 + split * 10 + len(case))
    m = 68 if case == "m68" else 72
    n, k, count, gm, gn = 64, 64, 7, 3, 2
    draw = lambda s: rng.integers(-3, 4, size=s).astype(np.float32)
    beta = 1.0 if case == "beta1" else 0.0
    flags = {"bias", "relu"} if case != "beta1" else {"bias"}
    a = wk.bf16_bits(draw((gm * count * k * m,)))
    b = wk.bf16_bits(draw((gn * count * n * k,)))
    c0 = wk.bf16_bits(draw((gm * gn * m * n,))) if beta else \
        np.full(gm * gn * m * n, 0x7FC0, np.uint16)
    arrays = dict(a=a, b=b, c=c0, bias=draw((gm * m,)))
    call = wk.Call(m, n, k, m, k, m, "bf16", "bf16", beta, "stride", k * m, n * k, flags,
                   G=gm * gn, grid=dict(gm=gm, gn=gn, a_step_m=count * k * m,
                                        b_step_n=count * n * k, c_step_m=m * n,
                                        c_step_n=gm * m * n, bias_step_m=m),
                   count=count, a="a", b="b", c="c", bias="bias")
    say(f"split finish {case} split {split} kernel {kid}")
    ref = {k2: np.array(v, copy=True) for k2, v in arrays.items()}
    run_call_oracle(call, ref)
    got = gpu_steps([call], arrays, ["c"])["c"]
    assert np.array_equal(got, ref["c"])


@pytest.mark.parametrize("split", [2, 4])
@pytest.mark.parametrize("kid", [9, 10])
def test_split_mlp_block_matches_oracle(kid, split, monkeypatch):
    """The MLP block's two calls (bias + GELU, bias) with split stage lists, random data."""
    monkeypatch.setenv("TPP_FORCE_KERNEL", str(kid))
    monkeypatch.setenv("TPP_SPLIT", str(split))
    wl = wk.mlp_block(seed=43, tokens=512, hidden=512, inter=512)
    say(f"split {split} kernel {kid} mlp_block")
    ref = run_steps_oracle(wk.Workload(wl.name, wl.arrays, wl.calls, steps=wl.calls))
    got = gpu_steps(wl.calls, wl.arrays, ["h", "y"])
    _compare("h", got["h"], ref["h"], wl.calls[0])
    _compare("y", got["y"], ref["y"], wl.calls[1])
    again = gpu_steps(wl.calls, wl.arrays, ["y"])   # chunk-order sums: the same bits every run
    assert np.array_equal(again["y"], got["y"])


@pytest.mark.parametrize("ldc", [(1 << 29) + 64, (1 << 30) + 64], ids=["1GB", "2GB"])
def test_inverse_epilogue_aux_columns_far_apart(ldc):
    """RELU_inv through the bf16 register epilogue on an output whose two columns lie ldc
    elements apart (small-integer data, exact).  A wave copies its aux tile into LDS with 32-bit
    buffer offsets from its first element: at 1 GB apart the second column still fits them, at
    2 GB it does not and the wave loads the tile through registers instead.  Both against the
    oracle on compact copies."""
    import paper_2104_05755_amd as tpp
    dev = torch.device("cuda:0")
    stream = tpp.current_stream()
    rng = np.random.default_rng(ldc % 1000003)
    m, n, k, count = 64, 2, 64, 2
    say(f"relu_inv with C columns {ldc} elements apart")
    a = wk.bf16_bits(rng.integers(-4, 5, count * m * k).astype(np.float32))
    b = wk.bf16_bits(rng.integers(-4, 5, count * k * n).astype(np.float32))
    z = wk.bf16_bits(rng.integers(-3, 4, (n, m)).astype(np.float32))
    A = torch.from_numpy(a.view(np.int16)).to(dev)
    B = torch.from_numpy(b.view(np.int16)).to(dev)
    C = torch.empty(ldc * (n - 1) + m, dtype=torch.int16, device=dev)
    Z = torch.zeros(ldc * (n - 1) + m, dtype=torch.int16, device=dev)
    for c in range(n):
        Z[c * ldc:c * ldc + m] = torch.from_numpy(z[c].view(np.int16)).to(dev)
    h = tpp.tpp_brgemm_dispatch(tpp.make_desc(m, n, k, m, k, ldc, "bf16", "bf16", 0.0, "stride",
                                              m * k, k * n, flags=("relu_inv",)))
    grid = dict(gm=1, gn=1, a_step_m=0, b_step_n=0, c_step_m=0, c_step_n=0, bias_step_m=0)
    tpp.tpp_brgemm_execute_batched_aux(h, grid, 1, None, None, None, None, A, B, C, Z, None,
                                       count, None, None, None, None, None, stream)
    torch.cuda.synchronize()
    got = np.stack([C[c * ldc:c * ldc + m].cpu().numpy().view(np.uint16) for c in range(n)])
    del C, Z
    ref = np.full((n, m), 0x7FC0, dtype=np.uint16)
    oracle.brgemm_batched(oracle.Desc(m, n, k, m, k, m, "bf16", "bf16", 0.0, "stride", m * k,
                                      k * n, flags={"relu_inv"}),
                          a, b, ref, aux=np.ascontiguousarray(z), count=count)
    assert np.array_equal(got, ref)
