"""Pins of the oracle's TPP matrix equations (Sec. 4), CPU only.

- Alg. 3 on the paper's example equation Out = Tanh(T0) + (T1 x T2) / (T3 - T4): the paper prints
  the root's register score, 2.
- Alg. 4 on the same tree, worked out by hand from the algorithm's text.
- For trees of unary and binary TPPs, the root score is the fewest temporaries any evaluation
  order needs (brute force over every order), and the plan runs in exactly that many without
  overwriting a live temporary (simulated).
- The equation's value against torch's float64 operations, broadcast forms against full tensors
  built by numpy, and identities.
"""
from __future__ import annotations

import itertools

import numpy as np
import pytest
import torch

import oracle
import workloads as wk

EXAMPLE = [("leaf", 0), ("leaf", 1), ("leaf", 2), ("leaf", 3), ("leaf", 4),
           ("tanh", 0), ("mul", 1, 2), ("sub", 3, 4), ("div", 6, 7), ("add", 5, 8)]


def test_paper_example_root_score_is_two():
    sc = oracle.eq_scores(EXAMPLE, 9)
    assert sc[9] == 2
    assert sc[5:] == [1, 1, 1, 2, 2]


def test_paper_example_execution_plan():
    ts, tmp, n = oracle.eq_plan(EXAMPLE, 9)
    # Add visits Div (score 2) before Tanh (1); Div visits Mul, then Sub (equal scores: left
    # first).  Mul and Sub reserve tmps 0 and 1; Div keeps Mul's and recycles Sub's; Tanh
    # reserves the lowest free (1); Add keeps its left child's (Tanh's) and recycles Div's.
    assert ts[5:] == [3, 0, 1, 2, 4]
    assert tmp[5:] == [1, 0, 1, 0, 1]
    assert n == 2 and ts[:5] == [-1] * 5 and tmp[:5] == [-1] * 5


def _random_tree(rng, n_internal, ternary=False):
    """A random tree of unary / binary (and, if asked, ternary) nodes over fresh leaves."""
    nodes = []

    def leaf():
        nodes.append(("leaf", len([x for x in nodes if x[0] == "leaf"])))
        return len(nodes) - 1

    def build(k):
        if k == 0:
            return leaf()
        kinds = ["u", "b"] + (["t"] if ternary and k >= 1 else [])
        kind = kinds[rng.integers(len(kinds))]
        if kind == "u":
            c = build(k - 1)
            nodes.append(("exp", c))
        elif kind == "b":
            kl = int(rng.integers(0, k))
            a, b = build(kl), build(k - 1 - kl)
            nodes.append(("add", a, b))
        else:
            ks = rng.multinomial(k - 1, [1 / 3] * 3)
            a, b, c = (build(int(x)) for x in ks)
            nodes.append(("muladd", a, b, c))
        return len(nodes) - 1

    root = build(n_internal)
    return nodes, root


def _min_tmps(nodes, root):
    """Fewest temporaries over every evaluation order (a topological order of the internal nodes):
    a node's result needs one temporary, which may be one its non-leaf children free; leaves are
    read where they are."""
    internal = [i for i, x in enumerate(nodes) if x[0] != "leaf"]
    kids = {i: [c for c in nodes[i][1:] if nodes[c][0] != "leaf"] for i in internal}
    parent = {c: i for i in internal for c in kids[i]}
    best = [len(internal)]

    def go(done, live, peak):
        if peak >= best[0]:
            return
        if len(done) == len(internal):
            best[0] = peak
            return
        for i in internal:
            if i in done or any(c not in done for c in kids[i]):
                continue
            freed = len(kids[i])               # the children's results die here
            now = live - freed + 1
            go(done | {i}, now, max(peak, now if freed == 0 else max(live, now)))
    go(frozenset(), 0, 0)
    return best[0]


def _simulate(nodes, root, ts, tmp):
    """Run the plan: nodes in timestamp order, each writing its tmp; a tmp must not be written
    while it holds a value some later node still reads (other than the writer itself)."""
    order = sorted((t, i) for i, t in enumerate(ts) if t >= 0)
    holder = {}                                 # tmp -> node whose value it holds
    consumed = set()
    for _, i in order:
        kids = [c for c in nodes[i][1:] if nodes[c][0] != "leaf"]
        for c in kids:
            assert holder.get(tmp[c]) == c, "a child's value was overwritten before its use"
            consumed.add(c)
        prev = holder.get(tmp[i])
        assert prev is None or prev in consumed, "a live temporary was overwritten"
        holder[tmp[i]] = i
    assert holder[tmp[root]] == root


@pytest.mark.parametrize("seed", range(40))
def test_scores_are_minimal_and_plan_is_valid(seed):
    rng = np.random.default_rng(seed)
    nodes, root = _random_tree(rng, int(rng.integers(1, 8)))
    sc = oracle.eq_scores(nodes, root)
    ts, tmp, n = oracle.eq_plan(nodes, root)
    assert sc[root] == _min_tmps(nodes, root)
    assert n == sc[root]
    _simulate(nodes, root, ts, tmp)
    assert sorted(t for t in ts if t >= 0) == list(range(sum(x[0] != "leaf" for x in nodes)))


@pytest.mark.parametrize("seed", range(20))
def test_ternary_plans_are_valid_within_the_score(seed):
    # Alg. 3 gives a ternary node with a non-leaf child at least 3 (as printed): an upper bound
    rng = np.random.default_rng(100 + seed)
    nodes, root = _random_tree(rng, int(rng.integers(1, 8)), ternary=True)
    sc = oracle.eq_scores(nodes, root)
    ts, tmp, n = oracle.eq_plan(nodes, root)
    _simulate(nodes, root, ts, tmp)
    assert n <= max(sc[root], 1)


def test_malformed_trees_rejected():
    with pytest.raises(ValueError):
        oracle.eq_scores([("add", 0, 1), ("leaf", 0)], 0)       # a node is its own child
    with pytest.raises(ValueError):
        oracle.eq_scores([("leaf", 0), ("exp", 5)], 1)           # child out of range


def _leaves(rng, m, n, specs):
    out = []
    for lo, hi, dt, bc in specs:
        size = {"none": m * n, "col": m, "row": n, "scalar": 1}[bc]
        v = rng.uniform(lo, hi, size).astype(np.float32)
        out.append((v if dt == "f32" else wk.bf16_bits(v), m, dt, bc))
    return out


def test_example_value_against_torch():
    rng = np.random.default_rng(71)
    m, n = 37, 23
    lv = _leaves(rng, m, n, [(-2, 2, "f32", "none"), (-1, 1, "f32", "none"), (-1, 1, "bf16", "none"),
                             (1, 2, "f32", "none"), (-2, -1, "f32", "none")])
    out = np.zeros(m * n, np.float32)
    ref = oracle.eq_eval(EXAMPLE, 9, m, n, lv, out, m, "f32", want_ref64=True)
    T = [torch.tensor(wk.bf16_values(a) if dt == "bf16" else a, dtype=torch.float64)
         .reshape(n, m) for a, _, dt, _ in lv]
    want = torch.tanh(T[0]) + (T[1] * T[2]) / (T[3] - T[4])
    np.testing.assert_allclose(ref, want.numpy(), rtol=1e-15, atol=1e-15)
    assert np.array_equal(out, ref.astype(np.float32).reshape(-1))


@pytest.mark.parametrize("bc", ["col", "row", "scalar"])
def test_broadcast_equals_full_tensor(bc):
    rng = np.random.default_rng(72)
    m, n = 19, 11
    x = rng.uniform(-1, 1, m * n).astype(np.float32)
    size = {"col": m, "row": n, "scalar": 1}[bc]
    b = rng.uniform(-1, 1, size).astype(np.float32)
    full = {"col": np.tile(b, n), "row": np.repeat(b, m), "scalar": np.full(m * n, b[0])}[bc]
    nodes = [("leaf", 0), ("leaf", 1), ("mul", 0, 1)]
    o1, o2 = np.zeros(m * n, np.float32), np.zeros(m * n, np.float32)
    oracle.eq_eval(nodes, 2, m, n, [(x, m, "f32", "none"), (b, 1, "f32", bc)], o1, m, "f32")
    oracle.eq_eval(nodes, 2, m, n, [(x, m, "f32", "none"), (full.astype(np.float32), m, "f32",
                                                             "none")], o2, m, "f32")
    assert np.array_equal(o1, o2)
    assert np.array_equal(o1, (x.astype(np.float64) * full).astype(np.float32))


def test_unary_identities():
    rng = np.random.default_rng(73)
    m, n = 16, 8
    y = rng.uniform(-0.9, 0.9, m * n)
    x = np.arctanh(y).astype(np.float32)
    # tanh(atanh(y)) = y; sigmoid(2x) = (1 + tanh(x)) / 2; relu(x) - relu(-x) = x;
    # sqrt(square(x)) = |x|; rcp(rcp(x)) = x
    lv = [(x, m, "f32", "none")]
    ev = lambda nodes, root: oracle.eq_eval(nodes, root, m, n, lv, np.zeros(m * n, np.float32),
                                            m, "f32", want_ref64=True).reshape(-1)
    xd = x.astype(np.float64)
    np.testing.assert_allclose(ev([("leaf", 0), ("tanh", 0)], 1), np.tanh(xd), rtol=1e-15)
    np.testing.assert_allclose(ev([("leaf", 0), ("leaf", 0), ("add", 0, 1), ("sigmoid", 2)], 3),
                               (1 + np.tanh(xd)) / 2, rtol=1e-14)
    np.testing.assert_array_equal(ev([("leaf", 0), ("relu", 0), ("neg", 0), ("relu", 2),
                                      ("sub", 1, 3)], 4), xd)
    np.testing.assert_allclose(ev([("leaf", 0), ("square", 0), ("sqrt", 1)], 2), np.abs(xd),
                               rtol=1e-15)
    np.testing.assert_allclose(ev([("leaf", 0), ("rcp", 0), ("rcp", 1)], 2), xd, rtol=1e-15)
    np.testing.assert_allclose(ev([("leaf", 0), ("leaf", 0), ("leaf", 0), ("muladd", 0, 1, 2)], 3),
                               xd * xd + xd, rtol=1e-15)


def test_layernorm_chain_against_torch():
    """Reduce + equations give torch's layer_norm over the features of each token."""
    from helpers import run_steps_oracle
    F, T = 96, 40
    wl = wk.layernorm(seed=74, features=F, tokens=T)
    out = run_steps_oracle(wl)
    x = torch.tensor(wk.bf16_values(wl.arrays["x"]).astype(np.float64)).reshape(T, F)
    ref = torch.nn.functional.layer_norm(x, (F,), torch.tensor(wl.arrays["gamma"], dtype=torch.float64),
                                         torch.tensor(wl.arrays["beta"], dtype=torch.float64), eps=1e-5)
    got = wk.bf16_values(out["y"]).astype(np.float64).reshape(T, F)
    # bf16 output, fp32 statistics: agreement to bf16 rounding
    assert np.max(np.abs(got - ref.numpy())) <= 2.0 ** -7 * (np.abs(ref.numpy()).max() + 1)


def _softmax_oracle(x_bits, keys, columns):
    from helpers import run_steps_oracle
    wl = wk.softmax(seed=0, keys=keys, columns=columns)
    wl.arrays["x"] = x_bits
    return run_steps_oracle(wl)


def test_softmax_chain_against_torch():
    """Reduce MAX + exp equation + Reduce SUM + scaling equation give torch's softmax over the
    keys of each column (float64), to the bf16 rounding of the output."""
    from helpers import run_steps_oracle
    K, C = 96, 40
    wl = wk.softmax(seed=75, keys=K, columns=C)
    out = run_steps_oracle(wl)
    x = wk.bf16_values(wl.arrays["x"]).astype(np.float64).reshape(C, K)
    ref = torch.softmax(torch.tensor(x), dim=1).numpy()
    got = wk.bf16_values(out["y"]).astype(np.float64).reshape(C, K)
    assert np.max(np.abs(got - ref) / ref) <= 2.0 ** -8
    np.testing.assert_array_equal(out["mx"], x.max(axis=1).astype(np.float32))
    xe = out["xe"].astype(np.float64).reshape(C, K)
    np.testing.assert_allclose(xe, np.exp(x - x.max(axis=1, keepdims=True)), rtol=6e-8)
    np.testing.assert_allclose(out["s"], xe.sum(axis=1), rtol=1e-6)


def test_softmax_subtracts_the_column_maximum():
    # scores near 100: exp(x) alone overflows fp32, exp(x - max) does not; each column's largest
    # X' entry is exactly exp(0) = 1
    rng = np.random.default_rng(76)
    K, C = 64, 16
    x = 100.0 + rng.integers(-8, 1, size=K * C).astype(np.float32)
    out = _softmax_oracle(wk.bf16_bits(x), K, C)
    xe = out["xe"].reshape(C, K)
    assert np.all(np.isfinite(xe)) and np.array_equal(xe.max(axis=1), np.ones(C, np.float32))
    y = wk.bf16_values(out["y"]).astype(np.float64).reshape(C, K)
    ref = torch.softmax(torch.tensor(x.astype(np.float64).reshape(C, K) - 100.0), dim=1).numpy()
    assert np.max(np.abs(y - ref) / ref) <= 2.0 ** -8


def test_softmax_shift_invariance_is_exact():
    # integer scores shifted by an integer: X - max is the same exact value, so every output bit
    # agrees
    rng = np.random.default_rng(77)
    K, C = 48, 24
    x = rng.integers(-6, 7, size=K * C).astype(np.float32)
    a = _softmax_oracle(wk.bf16_bits(x), K, C)
    b = _softmax_oracle(wk.bf16_bits(x + 8.0), K, C)
    assert np.array_equal(a["y"], b["y"]) and np.array_equal(a["xe"], b["xe"])
