"""GPU parity, bit-exact: the benchmarked launches and the transposed operand layouts on
small-integer data.

With every input a small integer (exact in bf16), every product and every partial sum of the
batch reduction is an integer below 2^24, so it is exact in fp32 whatever the summation order;
bias and ReLU keep it an integer, and the fp32 -> bf16 narrowing is then one round-to-nearest-even
decision on the same fp32 value on both sides.  The GPU output must therefore equal the oracle's
bit for bit: any wrong block address (Sec. 2.3's stride, offset and address formulas), tile
position (Alg. 6's ib_m / ib_n grid), swizzle, or epilogue store shows up as a mismatch.

The bounds are stated per case: the largest partial sum any order can form is at most
sum |a||b| over the reduction plus |bias|, checked against 2^24 below before the GPU runs.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import workloads as wk
from helpers import run_oracle

pytestmark = pytest.mark.gpu

EXACT_LIMIT = 1 << 24


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    import paper_2104_05755_amd  # noqa: F401  (fails loudly if the HIP library is missing)
    return torch.device("cuda:0")


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def integerize(wl, seed, ranges=None):
    """The workload with every array some call reads before any call writes it redrawn as
    integers in [-r, r] (r = ranges.get(name, 4)), stored in the array's own type (bf16 bits or
    fp32); GELU epilogues become ReLU (GELU of an integer is not exact)."""
    rng = np.random.default_rng(seed)
    ranges = ranges or {}
    arrs = dict(wl.arrays)
    written, inputs = set(), []
    for c in wl.calls:
        reads = [c.a, c.b, c.bias] + ([c.c] if c.beta != 0.0 else [])
        for name in reads:
            if name and name not in written and name not in inputs:
                inputs.append(name)
        written.add(c.c)
    for name in inputs:
        r = ranges.get(name, 4)
        v = rng.integers(-r, r + 1, size=arrs[name].shape).astype(np.float32)
        arrs[name] = wk.bf16_bits(v) if arrs[name].dtype == np.uint16 else v
    calls = []
    for c in wl.calls:
        kw = dict(c.__dict__)
        if "gelu_tanh" in kw["flags"]:
            kw["flags"] = (set(kw["flags"]) - {"gelu_tanh"}) | {"relu"}
        calls.append(wk.Call(**kw))
    return wk.Workload(wl.name, arrs, calls)


def max_partial(call, arrs, in_max):
    """Bound on |partial sum| of one instance: pairs x k x max|a| x max|b| (+ |beta| max|c|,
    + max|bias|).  The address kind's longest list is used for its pair count."""
    pairs = call.count if call.kind != "address" else int(np.max(np.diff(call.begin)))
    bound = pairs * call.k * in_max[call.a] * in_max[call.b]
    if call.beta != 0.0:
        bound += abs(call.beta) * in_max[call.c]
    if call.bias:
        bound += in_max[call.bias]
    return bound


def run_gpu(wl):
    from paper_2104_05755_amd import torch_io
    dev = torch_io.upload(wl)
    names = []
    for c in wl.calls:
        dc = torch_io.prepare(c, dev)
        names.append(torch_io.describe(dc))
        torch_io.launch(dc)
    torch.cuda.synchronize()
    return {k: torch_io.to_host(v, wl.arrays[k]) for k, v in dev.items()}, names


def assert_bits_equal(got, ref, what):
    g = got.view(np.uint16 if got.dtype == np.uint16 else np.uint32)
    r = ref.view(np.uint16 if ref.dtype == np.uint16 else np.uint32)
    bad = np.flatnonzero(g.reshape(-1) != r.reshape(-1))
    assert bad.size == 0, f"{what}: {bad.size} of {g.size} elements differ (first at {bad[:5]})"


# ----------------------------------------------------------------------------------------------
# The benchmarked launches: the 256 x 256 (16 waves) and 128 x 128 (4 waves) 64-k instances on
# complete tiles of a fused strided grid (the FULL instances), beta = 0, bf16 out through the
# register epilogue, bias only and bias + ReLU; and the fp32-out epilogue on the same tiles.
# Transformer-MLP shape: 1024 tokens, 256 -> 2560 -> 256, so GEMM1's virtual C is 2560 x 1024 (40
# tiles of 256 or 160 of 128: more than one XCD run and more than one band of 8 tile rows) and
# GEMM2 reduces 40 pairs.  W2 in [-1, 1] bounds GEMM2's sums (2560 * 4100 < 2^24).
# ----------------------------------------------------------------------------------------------
def _bench_shape(seed, epi, out_type="bf16"):
    base = wk.mlp_block(seed=seed, tokens=1024, hidden=256, inter=2560)
    g1, g2 = base.calls
    g1 = wk.Call(**dict(g1.__dict__, flags=set(epi)))
    arrs = dict(base.arrays)
    if out_type == "f32":
        g1 = wk.Call(**dict(g1.__dict__, c_type="f32"))
        arrs["h"] = np.full(arrs["h"].shape, np.nan, np.float32)
        return integerize(wk.Workload("mlp_block", arrs, [g1]), seed)
    return integerize(wk.Workload("mlp_block", arrs, [g1, g2]), seed, ranges={"w2": 1})


@pytest.mark.parametrize("kid,tile", [(9, "256, 256, 4, 4"), (10, "128, 128, 2, 2")])
@pytest.mark.parametrize("epi", [("bias",), ("bias", "relu")])
def test_benchmarked_launch_bit_exact(kid, tile, epi, monkeypatch):
    monkeypatch.setenv("TPP_FORCE_KERNEL", str(kid))
    monkeypatch.setenv("TPP_SPLIT", "1")   # the benchmarked launches reduce whole stage lists
    wl = _bench_shape(21 + kid, epi)
    g1, g2 = wl.calls
    in_max = {k: float(np.max(np.abs(wk.bf16_values(v) if v.dtype == np.uint16 else v)))
              for k, v in wl.arrays.items() if k not in ("h", "y")}
    b1 = max_partial(g1, wl.arrays, in_max)
    assert b1 < EXACT_LIMIT
    in_max["h"] = b1   # |H| <= GEMM1's bound (bf16 rounding of an integer never grows past it)
    assert max_partial(g2, wl.arrays, in_max) < EXACT_LIMIT
    say(f"benchmarked launch kernel {kid} {epi}")
    got, names = run_gpu(wl)
    # the launches ran the FULL, aligned, stride instance the bench times (no split)
    for nm in names:
        assert nm == f"brgemm_bf16_dl_kernel<{tile}, true, 0, true, 0, 64, 0, false, false>", nm
    h_ref, _ = run_oracle(wl, 0)
    assert_bits_equal(got["h"], h_ref, f"k{kid} {epi} H")
    y_ref, _ = run_oracle(wk.Workload(wl.name, dict(wl.arrays, h=h_ref), wl.calls), 1)
    assert_bits_equal(got["y"], y_ref, f"k{kid} {epi} Y")


@pytest.mark.parametrize("kid", [9, 10])
def test_benchmarked_tiles_fp32_out_bit_exact(kid, monkeypatch):
    monkeypatch.setenv("TPP_FORCE_KERNEL", str(kid))
    wl = _bench_shape(31 + kid, ("bias", "relu"), out_type="f32")
    say(f"benchmarked tiles, fp32 out, kernel {kid}")
    got, names = run_gpu(wl)
    assert ", true, 0, true, 0, 64, 0, false, false>" in names[0], names[0]
    h_ref, _ = run_oracle(wl, 0)
    assert_bits_equal(got["h"], h_ref, f"k{kid} fp32 H")


@pytest.mark.parametrize("kid", [9, 10, 11])
def test_benchmarked_tiles_save_preact_bit_exact(kid, monkeypatch):
    """The forward call that keeps the pre-activation (bias + ReLU + SAVE_PREACT) on complete
    tiles: the register epilogue parks the pre-activation, stores it to aux, then parks and
    stores the activation.  Both outputs bit for bit against the oracle."""
    from helpers import run_call_oracle
    monkeypatch.setenv("TPP_FORCE_KERNEL", str(kid))
    monkeypatch.setenv("TPP_SPLIT", "1")
    base = _bench_shape(41 + kid, ("bias", "relu", "save_preact"))
    g1 = wk.Call(**dict(base.calls[0].__dict__, aux="z"))
    arrs = dict(base.arrays, z=np.full(base.arrays["h"].shape, 0x7FC0, np.uint16))
    wl = wk.Workload("mlp_block", arrs, [g1])
    in_max = {k: float(np.max(np.abs(wk.bf16_values(v) if v.dtype == np.uint16 else v)))
              for k, v in arrs.items() if k not in ("h", "y", "z")}
    assert max_partial(g1, arrs, in_max) < EXACT_LIMIT
    say(f"benchmarked tiles, SAVE_PREACT, kernel {kid}")
    got, names = run_gpu(wl)
    assert ", true, 0, true, 0, 64, 0, false, false>" in names[0], names[0]
    ref = {k: np.array(v, copy=True) for k, v in arrs.items()}
    run_call_oracle(g1, ref)
    assert_bits_equal(got["z"], ref["z"], f"k{kid} Z")
    assert_bits_equal(got["h"], ref["h"], f"k{kid} H")


# ----------------------------------------------------------------------------------------------
# Operands stored transposed (A_TRANS, B_TRANS, both) on every 64-k instance and every batch
# variant: a virtual C that is a multiple of 256 on both sides (FULL tiles, bf16 register
# epilogue), a ragged one, the offset-based convolution and the address-based gathered lists.
# ----------------------------------------------------------------------------------------------
EXACT_AT_CASES = {
    # GEMM1 K = 512: |H| <= 8196; GEMM2 K = 512 with W2 in [-1, 1]: 4.2e6
    "full": lambda: integerize(wk.mlp_block(seed=13, tokens=512, hidden=512, inter=512), 13,
                               ranges={"w2": 1}),
    "ragged": lambda: integerize(wk.mlp_fc(seed=14, minibatch=7 * 64, c_in=192, k_out=5 * 64), 14),
    "offset": lambda: integerize(wk.conv3x3(seed=15, images=2, h=9, w=56, c=64, k=64), 15),
    "address": lambda: integerize(wk.gathered(seed=16, n_out=24, pool=64, min_len=0,
                                              max_len=12), 16),
}


@pytest.mark.parametrize("pairs", [1, 2, 3])
def test_a_trans_full_tiles_short_stage_lists(pairs, monkeypatch):
    """The 16-wave instance with A stored transposed on complete tiles defers each stage's last
    k-step past the next barrier; stage lists of one, two and three stages (the first and last
    stages of that schedule) bit for bit against the oracle, with bias + ReLU."""
    monkeypatch.setenv("TPP_FORCE_KERNEL", "9")
    monkeypatch.setenv("TPP_SPLIT", "1")
    base = wk.mlp_block(seed=60 + pairs, tokens=512, hidden=64 * pairs, inter=512)
    g1 = wk.Call(**dict(base.calls[0].__dict__, flags={"bias", "relu", "a_trans"},
                        lda=base.calls[0].k))
    wl = integerize(wk.Workload("mlp_block", dict(base.arrays), [g1]), 60 + pairs)
    say(f"a_trans full tiles, {pairs} pairs")
    got, names = run_gpu(wl)
    assert names[0].endswith("true, false>") and "<256, 256, 4, 4, true, 0, true," in names[0], \
        names[0]
    h_ref, _ = run_oracle(wl, 0)
    assert_bits_equal(got["h"], h_ref, f"a_trans {pairs} pairs H")


@pytest.mark.parametrize("layout", ["a_trans", "b_trans", "both"])
@pytest.mark.parametrize("kid", [9, 10, 11])
@pytest.mark.parametrize("case", sorted(EXACT_AT_CASES))
def test_transposed_layouts_bit_exact(kid, case, layout, monkeypatch):
    monkeypatch.setenv("TPP_FORCE_KERNEL", str(kid))
    wl = EXACT_AT_CASES[case]()
    for c in wl.calls:
        if layout in ("a_trans", "both"):
            c.flags = set(c.flags) | {"a_trans"}
            c.lda = c.k
        if layout in ("b_trans", "both"):
            c.flags = set(c.flags) | {"b_trans"}
            c.ldb = c.n
    say(f"{layout} kernel {kid} {case} (integer data)")
    got, names = run_gpu(wl)
    want_at, want_bt = layout in ("a_trans", "both"), layout in ("b_trans", "both")
    tail = f"{'true' if want_at else 'false'}, {'true' if want_bt else 'false'}>"
    for nm in names:
        assert nm.split(" + ")[0].endswith(tail), nm
    if wl.name == "mlp_block":
        h_ref, _ = run_oracle(wl, 0)
        assert_bits_equal(got["h"], h_ref, f"k{kid} {layout} H")
        y_ref, _ = run_oracle(wk.Workload(wl.name, dict(wl.arrays, h=h_ref), wl.calls), 1)
        assert_bits_equal(got["y"], y_ref, f"k{kid} {layout} Y")
    else:
        ref, _ = run_oracle(wl)
        out = wl.calls[0].c
        assert_bits_equal(got[out], ref, f"k{kid} {layout} {case}")


# ----------------------------------------------------------------------------------------------
# Offset and pointer lists (Sec. 2.3's offset and address variants) with one 64-k stage per pair
# on every 64-k instance: every listed block 16-byte aligned (on the four-wave instances each lane
# then holds one pair's byte addresses), one block or every block off that alignment (the copies
# go element by element through registers), lists longer than the 64 lanes, and stage lists
# split over workgroups (a chunk starts mid-list).  192 x 136 leaves ragged tiles on every
# instance.
# ----------------------------------------------------------------------------------------------
def _list_case(seed, kind, count, shift):
    rng = np.random.default_rng(seed)
    wl = wk.small_case(rng, 192, 136, 64, count, kind, "bf16", "bf16", 0.0, {"bias", "relu"},
                       integer=True)
    call = wl.calls[0]
    arrs = dict(wl.arrays)
    tail = wk.bf16_bits(np.zeros(8, np.float32))       # room for blocks moved up to 7 elements
    arrs["a"] = np.concatenate([arrs["a"], tail])
    arrs["b"] = np.concatenate([arrs["b"], tail])
    la, lb = ("offs_a", "offs_b") if kind == "offset" else ("idx_a", "idx_b")
    ea = np.array(getattr(call, la), dtype=np.int64)
    eb = np.array(getattr(call, lb), dtype=np.int64)
    if shift == "one":
        ea[count // 2] += 3
    elif shift == "all":
        ea += 1
        eb += 5
    kw = dict(call.__dict__)
    kw[la], kw[lb] = ea, eb
    return wk.Workload(wl.name, arrs, [wk.Call(**kw)])


@pytest.mark.parametrize("split", ["1", "3"])
@pytest.mark.parametrize("count", [9, 70])
@pytest.mark.parametrize("shift", ["none", "one", "all"])
@pytest.mark.parametrize("kind", ["offset", "address"])
@pytest.mark.parametrize("kid,tile", [(9, "<256, 256, 4, 4,"), (10, "<128, 128, 2, 2,"),
                                      (11, "<64, 64, 2, 2,")])
def test_pair_lists_one_stage_per_pair(kid, tile, kind, shift, count, split, monkeypatch):
    monkeypatch.setenv("TPP_FORCE_KERNEL", str(kid))
    monkeypatch.setenv("TPP_SPLIT", split)
    wl = _list_case(1000 + 7 * kid + count, kind, count, shift)
    call = wl.calls[0]
    in_max = {k: float(np.max(np.abs(wk.bf16_values(v) if v.dtype == np.uint16 else v)))
              for k, v in wl.arrays.items() if k != "c"}
    assert max_partial(call, wl.arrays, in_max) < EXACT_LIMIT
    say(f"pair lists: kernel {kid} {kind} shift={shift} count={count} split={split}")
    got, names = run_gpu(wl)
    assert tile in names[0], names[0]
    ref, _ = run_oracle(wl)
    assert_bits_equal(got["c"], ref, f"k{kid} {kind} {shift} {count} pairs split {split}")


# ----------------------------------------------------------------------------------------------
# Empty pair lists (count 0, Table 3: C = epilogue(beta C)) on every 16-byte-load instance, forced
# one at a time, on complete tiles with beta = 0 and bf16 out: the output is the activated bias,
# bit for bit (the register epilogue's accumulators start at the bias and no stage runs).  The
# 64-k instances also with SAVE_PREACT (the pre-activation is the bias itself).
# ----------------------------------------------------------------------------------------------
@pytest.mark.parametrize("kid,save", [(k, False) for k in (0, 1, 2, 5, 6, 7, 8)] +
                         [(k, s) for k in (9, 10, 11) for s in (False, True)])
def test_empty_pair_lists_give_the_activated_bias(kid, save, monkeypatch):
    from helpers import run_call_oracle
    monkeypatch.setenv("TPP_FORCE_KERNEL", str(kid))
    base = wk.mlp_block(seed=70 + kid, tokens=512, hidden=512, inter=512)
    flags = {"bias", "relu"} | ({"save_preact"} if save else set())
    g1 = wk.Call(**dict(base.calls[0].__dict__, count=0, flags=flags,
                        aux="z" if save else None))
    arrs = dict(base.arrays)
    if save:
        arrs["z"] = np.full(arrs["h"].shape, 0x7FC0, np.uint16)
    wl = integerize(wk.Workload("mlp_block", arrs, [g1]), 70 + kid)
    say(f"empty pair lists, kernel {kid}, save_preact={save}")
    got, names = run_gpu(wl)
    tile = {0: 256, 1: 128, 2: 64, 5: 256, 6: 128, 7: 64, 8: 256, 9: 256, 10: 128, 11: 64}[kid]
    assert f"<{tile}, {tile}," in names[0], names[0]
    ref = {k: np.array(v, copy=True) for k, v in wl.arrays.items()}
    run_call_oracle(g1, ref)
    assert_bits_equal(got["h"], ref["h"], f"k{kid} H")
    if save:
        assert_bits_equal(got["z"], ref["z"], f"k{kid} Z")


# ----------------------------------------------------------------------------------------------
# beta != 0 (Alg. 2: C loaded into the accumulators; the fp32-slab epilogue reads C) on every
# 16-byte-load instance, forced one at a time and unsplit, on complete tiles of a fused strided
# grid, bf16 and fp32 C, bias + ReLU: bit for bit (beta * C is a multiple of 0.5 below 2^24).
# ----------------------------------------------------------------------------------------------
@pytest.mark.parametrize("beta", [1.0, -0.5])
@pytest.mark.parametrize("ct", ["bf16", "f32"])
@pytest.mark.parametrize("kid", [0, 1, 2, 5, 6, 7, 8, 9, 10, 11])
def test_beta_reads_c_on_every_instance(kid, ct, beta, monkeypatch):
    monkeypatch.setenv("TPP_FORCE_KERNEL", str(kid))
    monkeypatch.setenv("TPP_SPLIT", "1")
    base = wk.mlp_block(seed=80 + kid, tokens=512, hidden=512, inter=512)
    g1 = wk.Call(**dict(base.calls[0].__dict__, beta=beta, c_type=ct, flags={"bias", "relu"}))
    arrs = dict(base.arrays)
    if ct == "f32":
        arrs["h"] = np.zeros(arrs["h"].shape, np.float32)
    wl = integerize(wk.Workload("mlp_block", arrs, [g1]), 80 + kid)
    in_max = {k: float(np.max(np.abs(wk.bf16_values(v) if v.dtype == np.uint16 else v)))
              for k, v in wl.arrays.items()}
    assert max_partial(g1, wl.arrays, in_max) < EXACT_LIMIT
    say(f"beta {beta} {ct} C, kernel {kid}")
    got, names = run_gpu(wl)
    tile = {0: 256, 1: 128, 2: 64, 5: 256, 6: 128, 7: 64, 8: 256, 9: 256, 10: 128, 11: 64}[kid]
    assert f"<{tile}, {tile}," in names[0], names[0]
    h_ref, _ = run_oracle(wl, 0)
    assert_bits_equal(got["h"], h_ref, f"k{kid} beta {beta} {ct} H")
