"""GPU parity: the HIP BRGEMM path (through the C ABI) against the CPU oracle.

Bars: relative Frobenius error <= 1e-5 for fp32 inputs and <= 5e-3 for bf16 inputs with fp32
accumulation, against the oracle's output rounded to the GPU's output type; bit-exact equality
where the arithmetic is exact (small-integer data: every product and partial sum is an integer
below 2^24, so any summation order gives the same fp32 value, and the fp32 -> bf16 narrowing is
then the same decision on both sides).  No oracle input comes from the GPU."""
from __future__ import annotations

import sys
import zlib

import numpy as np
import pytest
import torch

import oracle
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


def run_gpu(wl, calls=None, dev=None):
    """Run the workload's calls in order on the GPU; returns host copies of every array."""
    from paper_2104_05755_amd import torch_io
    dev = dev if dev is not None else torch_io.upload(wl)
    for ci in (calls if calls is not None else range(len(wl.calls))):
        dc = torch_io.prepare(wl.calls[ci], dev)
        torch_io.launch(dc)
    torch.cuda.synchronize()
    return {k: torch_io.to_host(v, wl.arrays[k]) for k, v in dev.items()}


def tol(call):
    """1e-5 when inputs and output are fp32; 5e-3 as soon as bf16 is involved (bf16 inputs, or
    a bf16 output whose rounding-boundary flips alone move single elements by 2^-8)."""
    return 1e-5 if (call.ab_type == "f32" and call.c_type == "f32") else 5e-3


def blocks(flat, call, insts):
    """The m x n output blocks of the given instances (as [n][m] arrays) from a flat C."""
    out = []
    for g in insts:
        if call.grid is not None:
            gi_m, gi_n = g % call.grid["gm"], g // call.grid["gm"]
            off = gi_m * call.grid["c_step_m"] + gi_n * call.grid["c_step_n"]
        else:
            off = int(call.c_off[g]) if call.c_off is not None else 0
        idx = off + np.arange(call.n)[:, None] * call.ldc + np.arange(call.m)[None, :]
        out.append(flat.reshape(-1)[idx])
    return np.stack(out)


def check_close(got, ref, call, what):
    g = values(got, call.c_type)
    r = values(ref, call.c_type)
    assert not np.isnan(g).any(), f"{what}: NaN in GPU output"
    err = rel_fro(g, r)
    assert err <= tol(call), f"{what}: rel Frobenius error {err:.3e} > {tol(call)}"
    return err


# ----------------------------------------------------------------------------------------------
# Small shapes: every kind, dtype combination, epilogue, beta, ragged sizes, padding
# ----------------------------------------------------------------------------------------------
SHAPES = [(1, 1, 1, 1), (5, 3, 7, 2), (16, 16, 16, 3), (17, 33, 65, 2), (64, 64, 64, 4),
          (64, 56, 64, 9), (72, 40, 24, 5), (128, 128, 64, 3), (200, 136, 80, 2), (64, 64, 64, 0),
          (8, 8, 8, 1), (96, 160, 128, 2), (40, 72, 8, 6)]
TYPES = [("f32", "f32"), ("bf16", "f32"), ("bf16", "bf16"), ("f32", "bf16")]
EPIS = [set(), {"bias"}, {"relu"}, {"bias", "relu"}, {"bias", "gelu_tanh"}]


def _cases():
    rng = np.random.default_rng(7)
    cases = []
    for si, (m, n, k, cnt) in enumerate(SHAPES):
        for ti, (ab, ct) in enumerate(TYPES):
            kind = ("stride", "offset", "address")[(si + ti) % 3]
            beta = (0.0, 1.0, 0.5)[(si * 3 + ti) % 3]
            epi = EPIS[(si + 2 * ti) % len(EPIS)]
            pad = (0, 8, 3)[(si + ti) % 3]
            cases.append((m, n, k, cnt, kind, ab, ct, beta, tuple(sorted(epi)), pad))
    return cases


@pytest.mark.parametrize("m,n,k,count,kind,ab,ct,beta,epi,pad", _cases())
def test_small_shapes_match_oracle(m, n, k, count, kind, ab, ct, beta, epi, pad):
    rng = np.random.default_rng(zlib.crc32(repr((m, n, k, count, kind, ab, ct, beta, epi, pad)).encode()))
    wl = wk.small_case(rng, m, n, k, count, kind, ab, ct, beta, set(epi), pad=pad)
    say(f"case m={m} n={n} k={k} count={count} {kind} {ab}->{ct} beta={beta} {epi} pad={pad}")
    ref, _ = run_oracle(wl)
    got = run_gpu(wl)["c"]
    call = wl.calls[0]
    live = blocks(got, call, [0]), blocks(ref, call, [0])
    check_close(live[0], live[1], call, "small")
    if beta == 0.0:   # C was NaN-filled: the padding of C (ldc > m) must be untouched
        pad_g = got.reshape(n, call.ldc)[:, m:]
        assert np.array_equal(pad_g.view(np.uint8), wl.arrays["c"].reshape(n, call.ldc)[:, m:].view(np.uint8))


@pytest.mark.parametrize("kind", ["stride", "offset", "address"])
@pytest.mark.parametrize("ab,ct", [("bf16", "bf16"), ("bf16", "f32"), ("f32", "f32")])
@pytest.mark.parametrize("m,n,k,count", [(64, 64, 64, 16), (128, 128, 64, 8), (24, 17, 40, 3),
                                         (64, 56, 64, 9)])
def test_integer_data_bit_exact(kind, ab, ct, m, n, k, count):
    rng = np.random.default_rng(m * 1000 + n * 10 + count)
    wl = wk.small_case(rng, m, n, k, count, kind, ab, ct, 1.0, {"bias", "relu"}, integer=True)
    say(f"integer case {m}x{n}x{k} count={count} {kind} {ab}->{ct}")
    ref, _ = run_oracle(wl)
    got = run_gpu(wl)["c"]
    assert np.array_equal(got, ref)


def test_three_variants_bit_identical_on_gpu():
    rng = np.random.default_rng(99)
    base = wk.small_case(rng, 128, 96, 64, 7, "stride", "bf16", "bf16", 0.0, {"bias", "gelu_tanh"})
    call = base.calls[0]
    outs = [run_gpu(base)["c"]]
    for kind in ("offset", "address"):
        kw = dict(call.__dict__, kind=kind, grid=None)
        if kind == "offset":
            kw.update(offs_a=np.arange(7) * call.stride_a, offs_b=np.arange(7) * call.stride_b)
        else:
            kw.update(begin=np.array([0, 7]), idx_a=np.arange(7) * call.stride_a,
                      idx_b=np.arange(7) * call.stride_b)
        outs.append(run_gpu(wk.Workload(kind, base.arrays, [wk.Call(**kw)]))["c"])
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])


def test_fp32_split_pair_list_is_deterministic():
    """A one-tile fp32 call splits its pair list over workgroups and adds the chunk sums in a fixed
    order: repeated calls give identical bits, within the fp32 bar of the oracle."""
    wl = wk.fp32_single()
    first = run_gpu(wl)["c"]
    again = run_gpu(wl)["c"]
    assert np.array_equal(first.view(np.uint32), again.view(np.uint32))
    ref, _ = run_oracle(wl)
    check_close(first, ref, wl.calls[0], "fp32 split")


def test_single_call_entry_points_match_batched():
    """The paper-shaped single calls (stride / offset / address) equal one-instance batches."""
    import paper_2104_05755_amd as tpp
    from paper_2104_05755_amd import torch_io
    rng = np.random.default_rng(5)
    wl = wk.small_case(rng, 64, 48, 64, 5, "stride", "bf16", "f32", 0.5, {"bias"})
    call = wl.calls[0]
    ref, _ = run_oracle(wl)
    dev = torch_io.upload(wl)
    h = tpp.tpp_brgemm_dispatch(torch_io.descriptor(call))
    tpp.tpp_brgemm_execute_stride(h, dev["a"], dev["b"], dev["c"], dev["bias"], 5,
                                  tpp.current_stream())
    got_s = torch_io.to_host(dev["c"], wl.arrays["c"])
    dev = torch_io.upload(wl)
    ho = tpp.tpp_brgemm_dispatch(torch_io.descriptor(wk.Call(**dict(call.__dict__, kind="offset"))))
    offs_a = torch.arange(5, device="cuda", dtype=torch.int64) * call.stride_a
    offs_b = torch.arange(5, device="cuda", dtype=torch.int64) * call.stride_b
    tpp.tpp_brgemm_execute_offset(ho, dev["a"], dev["b"], offs_a, offs_b, dev["c"], dev["bias"], 5,
                                  tpp.current_stream())
    got_o = torch_io.to_host(dev["c"], wl.arrays["c"])
    dev = torch_io.upload(wl)
    ha = tpp.tpp_brgemm_dispatch(torch_io.descriptor(wk.Call(**dict(call.__dict__, kind="address"))))
    pa = dev["a"].data_ptr() + offs_a * 2
    pb = dev["b"].data_ptr() + offs_b * 2
    tpp.tpp_brgemm_execute_address(ha, pa, pb, dev["c"], dev["bias"], 5, tpp.current_stream())
    got_a = torch_io.to_host(dev["c"], wl.arrays["c"])
    torch.cuda.synchronize()
    assert np.array_equal(got_s, got_o) and np.array_equal(got_s, got_a)
    check_close(got_s, ref, call, "single stride")


# ----------------------------------------------------------------------------------------------
# The five workloads: reduced sizes (whole output vs oracle), then full sizes (sampled)
# ----------------------------------------------------------------------------------------------
REDUCED = {
    1: lambda: wk.fp32_single(),
    2: lambda: wk.mlp_fc(minibatch=320, c_in=256, k_out=448),
    3: lambda: wk.conv3x3(images=2, h=9, w=56, c=64, k=64),
    4: lambda: wk.mlp_block(tokens=576, hidden=320, inter=512),
    5: lambda: wk.gathered(n_out=24, pool=64, min_len=0, max_len=12),
}


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_workload_reduced_size_whole_output(cfg):
    wl = REDUCED[cfg]()
    say(f"workload {wl.name} reduced")
    got = run_gpu(wl)
    if wl.name == "mlp_block":
        h_ref, _ = run_oracle(wl, 0)
        check_close(got["h"], h_ref, wl.calls[0], "mlp_block h")
        wl2 = wk.Workload(wl.name, dict(wl.arrays, h=h_ref), wl.calls)
        y_ref, _ = run_oracle(wl2, 1)
        check_close(got["y"], y_ref, wl.calls[1], "mlp_block y")
    else:
        call = wl.calls[0]
        ref, _ = run_oracle(wl)
        check_close(got[call.c], ref, call, wl.name)


def _sample(G, k, seed):
    rng = np.random.default_rng(seed)
    s = set(rng.choice(G, size=min(k, G), replace=False).tolist()) | {0, G - 1}
    return sorted(s)


@pytest.mark.parametrize("cfg", [1, 2, 3, 5])
def test_workload_full_size_sampled(cfg):
    wl = wk.CONFIGS[cfg]()
    call = wl.calls[0]
    say(f"workload {wl.name} full size, G={call.G}")
    got = run_gpu(wl)[call.c]
    sel = _sample(call.G, 48, cfg)
    ref, _ = run_oracle(wl, sel=sel)
    check_close(blocks(got, call, sel), blocks(ref, call, sel), call, wl.name)


def test_mlp_block_full_size_sampled():
    wl = wk.mlp_block()
    g1, g2 = wl.calls
    say("workload mlp_block full size")
    got = run_gpu(wl)
    nbs = [0, 77, 127]
    # GEMM2 instances of token blocks nbs need every GEMM1 instance of those token blocks.
    sel1 = [ib + g1.grid["gm"] * nb for nb in nbs for ib in range(g1.grid["gm"])]
    h_ref, _ = run_oracle(wl, 0, sel=sel1)
    check_close(blocks(got["h"], g1, sel1), blocks(h_ref, g1, sel1), g1, "mlp_block h")
    sel2 = [hb + g2.grid["gm"] * nb for nb in nbs for hb in range(g2.grid["gm"])]
    wl2 = wk.Workload(wl.name, dict(wl.arrays, h=h_ref), wl.calls)
    y_ref, _ = run_oracle(wl2, 1, sel=sel2)
    check_close(blocks(got["y"], g2, sel2), blocks(y_ref, g2, sel2), g2, "mlp_block y")


# ----------------------------------------------------------------------------------------------
# The device downconvert: fp32 -> bf16 round to nearest even, against the oracle's bit-level one
# ----------------------------------------------------------------------------------------------
def test_device_bf16_narrowing_is_rne():
    rng = np.random.default_rng(3)
    hi = np.arange(0, 1 << 16, dtype=np.uint32)
    bits = np.concatenate([hi << 16 | 0x8000, hi << 16 | 0x7FFF, hi << 16 | 0x8001,
                           rng.integers(0, 1 << 32, size=1 << 21, dtype=np.uint64).astype(np.uint32)])
    x = bits.view(np.float32)
    keep = np.isfinite(x) & (np.abs(x) >= np.float32(1.1754944e-38))   # no zeros, denormals
    x = np.ascontiguousarray(x[keep])
    m = x.size
    call = wk.Call(m, 1, 1, m, 1, m, "f32", "bf16", 0.0, "stride", 0, 0, set(), G=1,
                   grid=dict(gm=1, gn=1, a_step_m=0, b_step_n=0, c_step_m=0, c_step_n=0,
                             bias_step_m=0), count=1, a="a", b="b", c="c")
    wl = wk.Workload("cvt", dict(a=x, b=np.ones(1, np.float32),
                                 c=np.full(m, 0x7FC0, np.uint16)), [call])
    got = run_gpu(wl)["c"]
    want = oracle.f32_to_bf16_array(x)
    assert np.array_equal(got, want)


# ----------------------------------------------------------------------------------------------
# Every tile instance of the 16-byte-load family, forced one at a time (complete and ragged tiles)
# ----------------------------------------------------------------------------------------------
VEC_KERNEL_IDS = [0, 1, 2, 5, 6, 7, 8, 9, 10, 11]


@pytest.mark.parametrize("kid", VEC_KERNEL_IDS)
@pytest.mark.parametrize("shape", ["full", "ragged"])
def test_every_tile_kernel_matches_oracle(kid, shape, monkeypatch):
    monkeypatch.setenv("TPP_FORCE_KERNEL", str(kid))
    if shape == "full":
        wl = wk.mlp_block(seed=11, tokens=512, hidden=512, inter=512)
    else:   # 5 x 7 instances of 64 x 64: no tile shape divides the virtual C
        wl = wk.mlp_fc(seed=12, minibatch=7 * 64, c_in=192, k_out=5 * 64)
    say(f"kernel {kid} {shape} {wl.name}")
    got = run_gpu(wl)
    if wl.name == "mlp_block":
        h_ref, _ = run_oracle(wl, 0)
        check_close(got["h"], h_ref, wl.calls[0], f"k{kid} h")
        y_ref, _ = run_oracle(wk.Workload(wl.name, dict(wl.arrays, h=h_ref), wl.calls), 1)
        check_close(got["y"], y_ref, wl.calls[1], f"k{kid} y")
    else:
        ref, _ = run_oracle(wl)
        check_close(got["out"], ref, wl.calls[0], f"k{kid} ragged")


# A_i stored transposed (TPP_LAYOUT_A_TRANS): the 64-k direct-to-LDS instances, every batch
# variant.  Each workload's A blocks are read as transposed blocks with lda = k (the block extent
# m * k never exceeds the column-major one), by the GPU and by the oracle alike.
AT_KERNEL_IDS = [9, 10, 11]
AT_CASES = {
    "full": lambda: wk.mlp_block(seed=13, tokens=512, hidden=512, inter=512),
    "ragged": lambda: wk.mlp_fc(seed=14, minibatch=7 * 64, c_in=192, k_out=5 * 64),
    "offset": lambda: wk.conv3x3(seed=15, images=2, h=9, w=56, c=64, k=64),
    "address": lambda: wk.gathered(seed=16, n_out=24, pool=64, min_len=0, max_len=12),
}


@pytest.mark.parametrize("layout", ["a_trans", "b_trans", "both"])
@pytest.mark.parametrize("kid", AT_KERNEL_IDS)
@pytest.mark.parametrize("case", sorted(AT_CASES))
def test_a_trans_matches_oracle(kid, case, layout, monkeypatch):
    # B blocks are read as transposed blocks with ldb = n in the same way (extent k * n)
    monkeypatch.setenv("TPP_FORCE_KERNEL", str(kid))
    wl = AT_CASES[case]()
    for c in wl.calls:
        if layout in ("a_trans", "both"):
            c.flags = set(c.flags) | {"a_trans"}
            c.lda = c.k
        if layout in ("b_trans", "both"):
            c.flags = set(c.flags) | {"b_trans"}
            c.ldb = c.n
    say(f"{layout} kernel {kid} {case} {wl.name}")
    got = run_gpu(wl)
    if wl.name == "mlp_block":
        h_ref, _ = run_oracle(wl, 0)
        check_close(got["h"], h_ref, wl.calls[0], f"k{kid} at h")
        y_ref, _ = run_oracle(wk.Workload(wl.name, dict(wl.arrays, h=h_ref), wl.calls), 1)
        check_close(got["y"], y_ref, wl.calls[1], f"k{kid} at y")
    else:
        ref, _ = run_oracle(wl)
        out = wl.calls[0].c
        check_close(got[out], ref, wl.calls[0], f"k{kid} at {case}")


def test_a_trans_unsupported_shapes_are_refused():
    # k not a multiple of 64: no instance takes a transposed A
    import paper_2104_05755_amd as tpp
    dev = torch.device("cuda:0")
    a = torch.zeros(64 * 40, dtype=torch.bfloat16, device=dev)
    b = torch.zeros(40 * 64, dtype=torch.bfloat16, device=dev)
    c = torch.zeros(64 * 64, device=dev)
    h = tpp.tpp_brgemm_dispatch(tpp.make_desc(64, 64, 40, 40, 40, 64, "bf16", "f32", 0.0, "stride",
                                              64 * 40, 40 * 64, flags=("a_trans",)))
    with pytest.raises(RuntimeError):
        tpp.tpp_brgemm_execute_stride(h, a, b, c, None, 1, tpp.current_stream())


def _bf16_dev(v, dev):
    return torch.tensor(np.asarray(v, np.float32), dtype=torch.bfloat16, device=dev)


def test_operands_spread_past_2_pow_32_bytes():
    """Addresses past 2^32 bytes, small-integer data (exact):
    - stride variant, 16 pairs of 64x64x64 blocks 2^28 elements (512 MB) apart, so each operand
      spans 8 GB: 64-bit pair bases in the direct-to-LDS kernel;
    - a B block of 2 columns 2^30 + 64 elements (2 GB) apart: its span exceeds the 32-bit offsets
      of the direct-to-LDS kernels, so the host takes the register-staged kernel.
    Each is checked against the oracle on compact copies of the same blocks."""
    import paper_2104_05755_amd as tpp
    dev = torch.device("cuda:0")
    stream = tpp.current_stream()
    rng = np.random.default_rng(94)
    m = n = k = 64
    count, step = 16, 1 << 28
    say("brgemm: 16 pairs 512 MB apart")
    ablk = rng.integers(-4, 5, (count, m * k)).astype(np.float32)
    bblk = rng.integers(-4, 5, (count, k * n)).astype(np.float32)
    A = torch.empty(count * step, dtype=torch.bfloat16, device=dev)
    B = torch.empty(count * step, dtype=torch.bfloat16, device=dev)
    for i in range(count):
        A[i * step:i * step + m * k] = _bf16_dev(ablk[i], dev)
        B[i * step:i * step + k * n] = _bf16_dev(bblk[i], dev)
    C = torch.full((m * n,), float("nan"), device=dev)
    h = tpp.tpp_brgemm_dispatch(tpp.make_desc(m, n, k, m, k, m, "bf16", "f32", 0.0, "stride",
                                              step, step))
    tpp.tpp_brgemm_execute_stride(h, A, B, C, None, count, stream)
    torch.cuda.synchronize()
    del A, B
    ref = np.full(m * n, np.nan, np.float32)
    oracle.brgemm_batched(oracle.Desc(m, n, k, m, k, m, "bf16", "f32", 0.0, "stride", m * k, k * n),
                          wk.bf16_bits(ablk.ravel()), wk.bf16_bits(bblk.ravel()), ref, count=count)
    assert np.array_equal(C.cpu().numpy(), ref)

    say("brgemm: B columns 2 GB apart")
    n2, ldb = 2, (1 << 30) + 64
    a1 = rng.integers(-4, 5, m * k).astype(np.float32)
    b1 = rng.integers(-4, 5, (n2, k)).astype(np.float32)
    B2 = torch.empty(ldb * (n2 - 1) + k, dtype=torch.bfloat16, device=dev)
    for c in range(n2):
        B2[c * ldb:c * ldb + k] = _bf16_dev(b1[c], dev)
    C2 = torch.full((m * n2,), float("nan"), device=dev)
    h2 = tpp.tpp_brgemm_dispatch(tpp.make_desc(m, n2, k, m, ldb, m, "bf16", "f32", 0.0, "stride"))
    tpp.tpp_brgemm_execute_stride(h2, _bf16_dev(a1, dev), B2, C2, None, 1, stream)
    torch.cuda.synchronize()
    del B2
    ref2 = np.full(m * n2, np.nan, np.float32)
    oracle.brgemm_batched(oracle.Desc(m, n2, k, m, k, m, "bf16", "f32", 0.0, "stride"),
                          wk.bf16_bits(a1), wk.bf16_bits(b1.ravel()), ref2, count=1)
    assert np.array_equal(C2.cpu().numpy(), ref2)
