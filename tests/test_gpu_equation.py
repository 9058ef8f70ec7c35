"""GPU parity of the TPP matrix equations (Sec. 4), through the C ABI, against the CPU oracle's
recursive fp64 evaluation of the tree: relative Frobenius error <= 1e-5 with fp32 leaves and
output (the fp32 transcendentals are within a few ulp), <= 5e-3 with bf16 involved; exact where
the arithmetic is (integer data, max / min / relu / neg, broadcast copies).  Covers every
operation, every broadcast form, ragged shapes, padded leading dimensions, a leaf as the root,
the paper's example at full size, and a layer norm built from a Reduce TPP and equations."""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import oracle
import workloads as wk
from helpers import rel_fro, run_steps_oracle, values

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    import paper_2104_05755_amd  # noqa: F401  (fails loudly if the HIP library is missing)
    return torch.device("cuda:0")


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def gpu_steps(steps, arrays, names):
    from paper_2104_05755_amd import torch_io
    dev = torch_io.upload(wk.Workload("x", arrays, []))
    for st in steps:
        torch_io.launch_step(torch_io.prepare_step(st, dev), dev)
    torch.cuda.synchronize()
    return {k: torch_io.to_host(dev[k], arrays[k]) for k in names}


def one(nodes, root, m, n, leaf_specs, out_type="f32", ldo=None, seed=0, integer=False):
    """Random leaves per spec (lo, hi, dtype, bcast, pad) and the GPU / oracle outputs."""
    rng = np.random.default_rng(seed)
    ldo = ldo or m
    arrays, leaves = {}, []
    for i, (lo, hi, dt, bc, pad) in enumerate(leaf_specs):
        ld = m + pad
        size = {"none": ld * n, "col": m, "row": n, "scalar": 1}[bc]
        v = (rng.integers(lo, hi + 1, size) if integer else rng.uniform(lo, hi, size)).astype(np.float32)
        arrays[f"l{i}"] = v if dt == "f32" else wk.bf16_bits(v)
        leaves.append((f"l{i}", ld if bc == "none" else 1, dt, bc))
    arrays["out"] = (np.full(ldo * n, np.nan, np.float32) if out_type == "f32"
                     else np.full(ldo * n, 0x7FC0, np.uint16))
    st = wk.EquationStep(nodes, root, m, n, leaves, "out", ldo, out_type)
    got = gpu_steps([st], arrays, ["out"])["out"]
    ref = np.array(arrays["out"], copy=True)
    oracle.eq_eval(nodes, root, m, n, [(arrays[a], ld, dt, bc) for a, ld, dt, bc in leaves], ref,
                   ldo, out_type)
    live = lambda x: values(x, out_type).reshape(n, ldo)[:, :m]
    return live(got), live(ref), got, arrays["out"]


UNARY = [("identity", -2, 2), ("neg", -2, 2), ("exp", -4, 4), ("tanh", -4, 4), ("relu", -2, 2),
         ("gelu_tanh", -5, 5), ("sqrt", 0.1, 9), ("rcp", 0.5, 3), ("square", -3, 3),
         ("sigmoid", -6, 6)]
BINARY = ["add", "sub", "mul", "div", "max", "min"]


@pytest.mark.parametrize("op,lo,hi", UNARY, ids=[u[0] for u in UNARY])
def test_every_unary_op(op, lo, hi):
    say(f"equation unary {op}")
    g, r, _, _ = one([("leaf", 0), (op, 0)], 1, 200, 33, [(lo, hi, "f32", "none", 0)], seed=1)
    assert rel_fro(g, r) <= 1e-5
    if op in ("identity", "neg", "relu", "square"):
        assert np.array_equal(g, r)


@pytest.mark.parametrize("op", BINARY)
def test_every_binary_op(op):
    say(f"equation binary {op}")
    g, r, _, _ = one([("leaf", 0), ("leaf", 1), (op, 0, 1)], 1 + 1, 130, 17,
                     [(-3, 3, "f32", "none", 5), (0.5, 2, "f32", "none", 0)], seed=2)
    assert rel_fro(g, r) <= 1e-5
    if op in ("add", "sub", "mul", "max", "min"):
        assert np.array_equal(g, r)   # one fp32 rounding of the exact result on both sides


def test_muladd_is_fused():
    g, r, _, _ = one([("leaf", 0), ("leaf", 1), ("leaf", 2), ("muladd", 0, 1, 2)], 3, 64, 40,
                     [(-2, 2, "f32", "none", 0)] * 3, seed=3)
    # fma rounds once; the oracle rounds the fp64 value (exact product, rounded sum) to fp32
    assert rel_fro(g, r) <= 1e-7


@pytest.mark.parametrize("bc", ["col", "row", "scalar"])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_broadcast_forms(bc, dt):
    say(f"equation broadcast {bc} {dt}")
    g, r, _, _ = one([("leaf", 0), ("leaf", 1), ("sub", 0, 1)], 2, 300, 29,
                     [(-8, 8, dt, "none", 3), (-8, 8, dt, bc, 0)], seed=4, integer=True)
    assert np.array_equal(g, r)


MIXED = [("leaf", 0), ("leaf", 1), ("sub", 0, 1), ("leaf", 2), ("leaf", 3), ("leaf", 4),
         ("add", 4, 5), ("muladd", 2, 3, 6)]


@pytest.mark.parametrize("out_type", ["f32", "bf16"])
@pytest.mark.parametrize("pad", [8, 1])
def test_all_leaf_kinds_in_one_tree(out_type, pad):
    # m a multiple of 8: with pad 8 every column starts 16-byte aligned (16-byte loads and
    # stores of 8 rows per thread); with pad 1 the same tree runs element by element
    say(f"equation mixed leaves pad {pad} {out_type}")
    g, r, got, init = one(MIXED, 7, 248, 23,
                          [(-8, 8, "bf16", "none", pad), (-8, 8, "f32", "col", 0),
                           (-4, 4, "bf16", "row", 0), (-4, 4, "f32", "scalar", 0),
                           (-4, 4, "bf16", "col", 0)],
                          out_type=out_type, ldo=248 + pad, seed=10, integer=True)
    assert np.array_equal(g, r)   # integers below 256 in magnitude: exact in bf16 and fp32
    # the gaps hold NaN: compare their bits
    gaps = lambda x: x.view(np.uint32 if x.dtype == np.float32 else np.uint16) \
        .reshape(23, 248 + pad)[:, 248:]
    assert np.array_equal(gaps(got), gaps(init))


def test_paper_example_small_bf16_out_padded():
    g, r, got, init = one(wk.EXAMPLE_EQUATION, 9, 257, 31,
                          [(-2, 2, "bf16", "none", 1), (-1, 1, "f32", "none", 0),
                           (-1, 1, "f32", "none", 7), (1, 2, "f32", "none", 0),
                           (-2, -1, "bf16", "none", 0)], out_type="bf16", ldo=260, seed=5)
    assert rel_fro(g, r) <= 5e-3
    gaps = lambda x: x.reshape(31, 260)[:, 257:]
    assert np.array_equal(gaps(got), gaps(init))          # the output's gaps are untouched


def test_leaf_root_is_a_copy():
    g, r, _, _ = one([("leaf", 0)], 0, 100, 7, [(-9, 9, "bf16", "none", 2)], seed=6,
                     integer=True)
    assert np.array_equal(g, r)


def test_paper_example_full_size():
    wl = wk.equation_example()
    st = wl.steps[0]
    say(f"equation example full size {st.m} x {st.n}")
    got = gpu_steps(wl.steps, wl.arrays, ["out"])["out"]
    ref = np.array(wl.arrays["out"], copy=True)
    oracle.eq_eval(st.nodes, st.root, st.m, st.n,
                   [(wl.arrays[a], ld, dt, bc) for a, ld, dt, bc in st.leaves], ref, st.ldo,
                   st.out_type)
    assert not np.isnan(got).any()
    assert rel_fro(got, ref) <= 1e-5


def test_layernorm_chain_matches_oracle():
    wl = wk.layernorm(seed=91, features=1024, tokens=512)
    say("layernorm chain")
    got = gpu_steps(wl.steps, wl.arrays, ["s", "rs", "y"])
    ref = run_steps_oracle(wl)
    assert rel_fro(got["s"], ref["s"]) <= 1e-5
    assert rel_fro(got["rs"], ref["rs"]) <= 1e-5
    assert rel_fro(values(got["y"], "bf16"), values(ref["y"], "bf16")) <= 5e-3


@pytest.mark.parametrize("keys,columns", [(512, 300), (77, 50)])
def test_softmax_chain_matches_oracle(keys, columns):
    # 512 keys: both equations on the vector path; 77: element path
    wl = wk.softmax(seed=92, keys=keys, columns=columns)
    say(f"softmax chain {keys} x {columns}")
    got = gpu_steps(wl.steps, wl.arrays, ["mx", "xe", "s", "y"])
    ref = run_steps_oracle(wl)
    assert np.array_equal(got["mx"], ref["mx"])          # max is exact
    assert rel_fro(got["xe"], ref["xe"]) <= 1e-5
    assert rel_fro(got["s"], ref["s"]) <= 1e-5
    assert rel_fro(values(got["y"], "bf16"), values(ref["y"], "bf16")) <= 5e-3
    cols = values(got["y"], "bf16").astype(np.float64).reshape(columns, keys).sum(axis=1)
    assert np.max(np.abs(cols - 1.0)) <= keys * 2.0 ** -8  # each column a distribution


def _balanced(depth):
    """A balanced tree of 2^depth leaf nodes (over at most 16 arguments, reused in turn) under
    add / sub / max / min nodes: Alg. 3 scores it depth, the temporaries its plan needs."""
    nodes = [("leaf", i % 16) for i in range(2 ** depth)]
    level = list(range(2 ** depth))
    ops = ["add", "sub", "max", "min"]
    while len(level) > 1:
        nxt = []
        for j in range(0, len(level), 2):
            nodes.append((ops[len(nodes) % 4], level[j], level[j + 1]))
            nxt.append(len(nodes) - 1)
        level = nxt
    return nodes, level[0]


@pytest.mark.parametrize("depth", [3, 5])
@pytest.mark.parametrize("m", [256, 100])
def test_deep_trees_use_more_temporaries(depth, m):
    # 3 and 5 temporaries: the vector kernel's 4- and 8-temporary variants (m = 256) and the
    # element path (m = 100); small integers keep every result exact
    nodes, root = _balanced(depth)
    from paper_2104_05755_amd import tpp_equation_plan
    assert tpp_equation_plan(nodes, root)[3] == depth
    say(f"equation balanced depth {depth} m {m}")
    g, r, _, _ = one(nodes, root, m, 19, [(-3, 3, "f32", "none", 0)] * min(2 ** depth, 16),
                     seed=11, integer=True)
    assert np.array_equal(g, r)


@pytest.mark.parametrize("m,n", [(65537, 65537), (65544, 65536)], ids=["element", "vector"])
def test_equation_past_2_pow_32_elements(m, n):
    """m * n just past 2^32 (8.6 GB per bf16 tensor): 64-bit element indices on the element path
    (odd m) and on the vector path.  X is the closed-form pattern x(e) = (e mod 251) - 125 built
    on the device in chunks, and Y = muladd(X, 2, row[c]) with row[c] = (c mod 7) - 3 is checked
    against the same closed form at every element (small integers: exact in bf16)."""
    from paper_2104_05755_amd import TPP_DT_BF16, TPP_DT_F32, current_stream, tpp_equation_execute
    total = m * n
    assert total > 2 ** 32
    say(f"equation past 2^32: {m} x {n}")
    dev = torch.device("cuda:0")
    chunk = 1 << 28
    x = torch.empty(total, dtype=torch.bfloat16, device=dev)
    for s in range(0, total, chunk):
        e = torch.arange(s, min(s + chunk, total), dtype=torch.int64, device=dev)
        x[s:s + e.numel()] = ((e % 251) - 125).to(torch.bfloat16)
    row = ((torch.arange(n, dtype=torch.int64, device=dev) % 7) - 3).to(torch.float32)
    two = torch.full((1,), 2.0, dtype=torch.float32, device=dev)
    y = torch.full((total,), float("nan"), dtype=torch.bfloat16, device=dev)
    nodes = [("leaf", 0), ("leaf", 1), ("leaf", 2), ("muladd", 0, 1, 2)]
    tpp_equation_execute(nodes, 3, m, n, [(x, m, TPP_DT_BF16, "none"), (two, 1, TPP_DT_F32, "scalar"),
                                          (row, 1, TPP_DT_F32, "row")],
                         y, m, TPP_DT_BF16, current_stream())
    torch.cuda.synchronize()
    del x
    bad = 0
    for s in range(0, total, chunk):
        e = torch.arange(s, min(s + chunk, total), dtype=torch.int64, device=dev)
        want = (2 * ((e % 251) - 125) + ((e // m) % 7) - 3).to(torch.float32)
        bad += int((y[s:s + e.numel()].to(torch.float32) != want).sum().item())
    assert bad == 0, f"{bad} wrong elements"


@pytest.mark.parametrize("n,pad", [(4096, 0), (1001, 0), (4096, 2)], ids=["n4096", "n1001", "ld3"])
def test_single_row_equations(n, pad):
    # single-row equations (the shape of a norm's statistics), every leaf kind, contiguous and
    # padded leading dimensions
    say(f"equation 1 x {n} pad {pad}")
    g, r, _, _ = one(MIXED, 7, 1, n,
                     [(-8, 8, "bf16", "none", pad), (-8, 8, "f32", "col", 0),
                      (-4, 4, "bf16", "row", 0), (-4, 4, "f32", "scalar", 0),
                      (-4, 4, "bf16", "col", 0)], seed=12, integer=True)
    assert np.array_equal(g, r)


# Outputs of at most 2^16 elements that the vector path does not take run one element per
# thread with every leaf loaded up front; the cases above (a few thousand elements) exercise that
# kernel.  Larger outputs off the vector path run the element kernel: the same trees past the
# small-output limit (m odd, so never the vector path).
@pytest.mark.parametrize("out_type", ["f32", "bf16"])
def test_element_path_past_small_outputs(out_type):
    say(f"equation element path, mixed leaves, {out_type}")
    m, n = 251, 300   # 75,300 elements
    g, r, got, init = one(MIXED, 7, m, n,
                          [(-8, 8, "bf16", "none", 1), (-8, 8, "f32", "col", 0),
                           (-4, 4, "bf16", "row", 0), (-4, 4, "f32", "scalar", 0),
                           (-4, 4, "bf16", "col", 0)],
                          out_type=out_type, ldo=m + 3, seed=11, integer=True)
    assert np.array_equal(g, r)
    gaps = lambda x: x.view(np.uint32 if x.dtype == np.float32 else np.uint16) \
        .reshape(n, m + 3)[:, m:]
    assert np.array_equal(gaps(got), gaps(init))


@pytest.mark.parametrize("op,lo,hi", UNARY, ids=[u[0] for u in UNARY])
def test_every_unary_op_element_path(op, lo, hi):
    g, r, _, _ = one([("leaf", 0), (op, 0)], 1, 201, 400, [(lo, hi, "f32", "none", 0)], seed=12)
    assert rel_fro(g, r) <= 1e-5
    if op in ("identity", "neg", "relu", "square"):
        assert np.array_equal(g, r)
