"""The C-ABI library on the host: it loads, exports every declared symbol, and its host-only
paths (dispatch validation, the handle cache, argument checks that precede any launch) behave
as include/tpp_brgemm.h and include/tpp_transform.h state.  No device work happens here."""
from __future__ import annotations

import ctypes
import glob
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = sorted(glob.glob(os.path.join(ROOT, "include", "*.h")))


@pytest.fixture(scope="module")
def tpp():
    import paper_2104_05755_amd as tpp
    return tpp


def declared_functions():
    names = set()
    for h in HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(tpp_[a-z_]+)\s*\(", text))
    return sorted(names)


def test_library_exports_every_declared_function(tpp):
    names = declared_functions()
    assert {"tpp_brgemm_dispatch", "tpp_reduce", "tpp_transform"} <= set(names)
    lib = ctypes.CDLL(tpp.LIB_PATH)
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, f"not exported: {missing}"


def test_library_is_built_for_gfx950_only(tpp):
    """The offload bundle of our own build names its target; gfx950 must be the only one."""
    blob = open(tpp.LIB_PATH, "rb").read()
    targets = set(re.findall(rb"amdgcn-amd-amdhsa-+(gfx[0-9a-f]+)", blob))
    assert targets == {b"gfx950"}, targets


def test_struct_layout_matches_header(tpp):
    # int32 m,n,k | pad | int64 lda,ldb,ldc | int32 x4 | float | int32 | int64 x2 | uint32
    assert ctypes.sizeof(tpp.tpp_brgemm_desc) == 88
    assert tpp.tpp_brgemm_desc.lda.offset == 16
    assert tpp.tpp_brgemm_desc.beta.offset == 56
    assert tpp.tpp_brgemm_desc.stride_a.offset == 64
    assert tpp.tpp_brgemm_desc.flags.offset == 80
    assert ctypes.sizeof(tpp.tpp_grid_strided) == 56


def test_dispatch_caches_equal_descriptors(tpp):
    d1 = tpp.make_desc(64, 64, 64, 64, 64, 64, "bf16", "bf16", 0.0, "stride", 4096, 4096, ["bias", "relu"])
    d2 = tpp.make_desc(64, 64, 64, 64, 64, 64, "bf16", "bf16", 0.0, "stride", 4096, 4096, ["bias", "relu"])
    d3 = tpp.make_desc(64, 64, 64, 64, 64, 64, "bf16", "bf16", 0.0, "stride", 4096, 4096, ["bias"])
    h1, h2, h3 = (tpp.tpp_brgemm_dispatch(d) for d in (d1, d2, d3))
    assert h1 == h2 and h1 != h3
    assert "bf16" in tpp.tpp_brgemm_describe(h1) and "vec" in tpp.tpp_brgemm_describe(h1)
    odd = tpp.make_desc(17, 5, 3, 17, 3, 17, "bf16", "f32")
    assert "generic" in tpp.tpp_brgemm_describe(tpp.tpp_brgemm_dispatch(odd))
    tpp.tpp_brgemm_release(h1)
    tpp.tpp_brgemm_release(None)


@pytest.mark.parametrize("field,value,status", [
    ("m", 0, -1), ("n", -3, -1), ("k", 0, -1),
    ("lda", 10, -1), ("ldb", 5, -1), ("ldc", 1, -1),
    ("a_type", 7, -1), ("comp_type", 1, -2), ("kind", 3, -1), ("flags", 64, -1),
    ("flags", 2 | 4, -1), ("beta", float("nan"), -1),
    # back-propagation bits: the inverses exclude each other and every forward activation,
    # SAVE_PREACT needs an activation
    ("flags", 8 | 16, -1), ("flags", 8 | 2, -1), ("flags", 16 | 4, -1), ("flags", 16 | 32 | 4, -1),
    ("flags", 32, -1), ("flags", 32 | 1, -1),
])
def test_dispatch_rejects(tpp, field, value, status):
    d = tpp.make_desc(16, 16, 16, 16, 16, 16, "bf16", "f32")
    setattr(d, field, value)
    with pytest.raises(tpp.TppError) as e:
        tpp.tpp_brgemm_dispatch(d)
    assert e.value.status == status
    assert tpp.tpp_last_error_message()


def test_dispatch_rejects_mixed_input_types(tpp):
    d = tpp.make_desc(16, 16, 16, 16, 16, 16, "bf16", "f32")
    d.b_type = tpp.TPP_DT_F32
    with pytest.raises(tpp.TppError) as e:
        tpp.tpp_brgemm_dispatch(d)
    assert e.value.status == tpp.TPP_ERR_UNSUPPORTED


def test_execute_argument_checks_precede_any_launch(tpp):
    hs = tpp.tpp_brgemm_dispatch(tpp.make_desc(16, 16, 16, 16, 16, 16, "bf16", "f32", kind="stride"))
    ho = tpp.tpp_brgemm_dispatch(tpp.make_desc(16, 16, 16, 16, 16, 16, "bf16", "f32", kind="offset"))
    hb = tpp.tpp_brgemm_dispatch(tpp.make_desc(16, 16, 16, 16, 16, 16, "bf16", "f32", flags=["bias"]))
    ha = tpp.tpp_brgemm_dispatch(tpp.make_desc(16, 16, 16, 16, 16, 16, "bf16", "f32", kind="address"))
    fake = 1 << 40   # never dereferenced: every call below fails its checks first
    bad = [
        lambda: tpp.tpp_brgemm_execute_stride(None, fake, fake, fake, None, 1),
        lambda: tpp.tpp_brgemm_execute_stride(hs, fake, fake, fake, None, -1),
        lambda: tpp.tpp_brgemm_execute_stride(hs, None, fake, fake, None, 2),
        lambda: tpp.tpp_brgemm_execute_stride(hs, fake, fake, None, None, 0),
        lambda: tpp.tpp_brgemm_execute_stride(ho, fake, fake, fake, None, 1),      # wrong kind
        lambda: tpp.tpp_brgemm_execute_offset(ho, fake, fake, None, fake, fake, None, 1),
        lambda: tpp.tpp_brgemm_execute_stride(hb, fake, fake, fake, None, 1),      # bias missing
        lambda: tpp.tpp_brgemm_execute_address(ha, None, fake, fake, None, 1),
        lambda: tpp.tpp_brgemm_execute_batched(hs, dict(gm=2, gn=2, a_step_m=0, b_step_n=0,
                                                        c_step_m=0, c_step_n=0, bias_step_m=0),
                                               3, None, None, None, None, fake, fake, fake, None,
                                               1, None, None, None, None, None),    # gm*gn != G
        lambda: tpp.tpp_brgemm_execute_batched(hs, dict(gm=1, gn=1, a_step_m=0, b_step_n=0,
                                                        c_step_m=0, c_step_n=0, bias_step_m=0),
                                               1, fake, None, None, None, fake, fake, fake, None,
                                               1, None, None, None, None, None),    # grid + arrays
        lambda: tpp.tpp_brgemm_execute_batched(ha, None, 4, None, None, fake, None, None, None,
                                               fake, None, 0, None, None, None, fake, fake),
        lambda: tpp.tpp_brgemm_execute_batched(hs, None, -1, None, None, None, None, fake, fake,
                                               fake, None, 1, None, None, None, None, None),
    ]
    for i, f in enumerate(bad):
        with pytest.raises(tpp.TppError) as e:
            f()
        assert e.value.status == tpp.TPP_ERR_INVALID_ARG, i


def test_aux_handles_need_the_aux_call(tpp):
    fake = 1 << 40   # never dereferenced
    grid = dict(gm=1, gn=1, a_step_m=0, b_step_n=0, c_step_m=0, c_step_n=0, bias_step_m=0)
    for flags in (["relu_inv"], ["gelu_tanh_inv"], ["bias", "gelu_tanh", "save_preact"]):
        h = tpp.tpp_brgemm_dispatch(tpp.make_desc(16, 16, 16, 16, 16, 16, "bf16", "bf16",
                                                  flags=flags))
        bias = fake if "bias" in flags else None
        bad = [
            lambda: tpp.tpp_brgemm_execute_stride(h, fake, fake, fake, bias, 1),
            lambda: tpp.tpp_brgemm_execute_batched(h, grid, 1, None, None, None, None, fake, fake,
                                                   fake, bias, 1, None, None, None, None, None),
            lambda: tpp.tpp_brgemm_execute_batched_aux(h, grid, 1, None, None, None, None, fake,
                                                       fake, fake, None, bias, 1, None, None,
                                                       None, None, None),   # aux missing
        ]
        for i, f in enumerate(bad):
            with pytest.raises(tpp.TppError) as e:
                f()
            assert e.value.status == tpp.TPP_ERR_INVALID_ARG, (flags, i)


def test_batched_reduce_and_transform_argument_checks(tpp):
    fake = 1 << 40
    for G, si, so in ((-1, 0, 0), (2, -1, 4), (2, 16, -4)):
        with pytest.raises(tpp.TppError) as e:
            tpp.tpp_reduce_batched(4, 4, 4, 0, fake, G, si, 0, 1 | 4, fake, None, so)
        assert e.value.status == tpp.TPP_ERR_INVALID_ARG
        with pytest.raises(tpp.TppError) as e:
            tpp.tpp_transform_batched(0, 4, 4, 4, 4, 0, 1, fake, si, fake, so, G)
        assert e.value.status == tpp.TPP_ERR_INVALID_ARG
    # G == 0 does nothing (the pointers are never touched)
    tpp.tpp_reduce_batched(4, 4, 4, 0, fake, 0, 16, 0, 1 | 4, fake, None, 4)
    tpp.tpp_transform_batched(0, 4, 4, 4, 4, 0, 1, fake, 16, fake, 16, 0)


def test_zero_instances_is_a_no_op(tpp):
    hs = tpp.tpp_brgemm_dispatch(tpp.make_desc(16, 16, 16, 16, 16, 16, "bf16", "f32"))
    tpp.tpp_brgemm_execute_batched(hs, None, 0, None, None, None, None, None, None, None, None,
                                   0, None, None, None, None, None)


@pytest.mark.parametrize("args", [
    (0, 4, 4, 0, 1, 0, 1 | 4),           # m = 0
    (4, 4, 3, 0, 1, 0, 1 | 4),           # ld < m
    (4, 4, 4, 9, 1, 0, 1 | 4),           # bad dtype
    (4, 4, 4, 0, 1, 7, 1 | 4),           # bad op
    (4, 4, 4, 0, 1, 0, 1 | 2 | 4),       # both directions
    (4, 4, 4, 0, 1, 0, 1),               # no output selected
    (4, 4, 4, 0, 1, 0, 1 | 8),           # X2 without out_x2
    (4, 4, 4, 0, None, 0, 1 | 4),        # NULL input
])
def test_reduce_argument_checks(tpp, args):
    m, n, ld, dt, x, op, flags = args
    fake = 1 << 40
    with pytest.raises(tpp.TppError) as e:
        tpp.tpp_reduce(m, n, ld, dt, fake if x else None, op, flags, fake, None)
    assert e.value.status == tpp.TPP_ERR_INVALID_ARG


@pytest.mark.parametrize("args,status", [
    ((3, 4, 4, 4, 4, 0, 1), "INVALID_ARG"),            # unknown kind
    ((0, -1, 4, 4, 4, 1, 1), "INVALID_ARG"),           # m < 0
    ((0, 4, 4, 3, 4, 1, 1), "INVALID_ARG"),            # ld_in < m
    ((0, 4, 4, 4, 3, 1, 1), "INVALID_ARG"),            # ld_out < n
    ((1, 4, 4, 4, 7, 1, 2), "INVALID_ARG"),            # VNNI ld_out < m * alpha
    ((1, 4, 4, 4, 8, 1, 3), "INVALID_ARG"),            # alpha 3
    ((2, 4, 4, 7, 8, 1, 2), "INVALID_ARG"),            # VNNI_T ld_in < m * alpha
    ((2, 4, 4, 8, 7, 1, 2), "INVALID_ARG"),            # VNNI_T ld_out < n * alpha
    ((0, 4, 4, 4, 4, 7, 1), "INVALID_ARG"),            # unknown dtype
])
def test_transform_argument_checks(tpp, args, status):
    kind, m, n, ld_in, ld_out, dtype, alpha = args
    with pytest.raises(tpp.TppError) as e:
        tpp.tpp_transform(kind, m, n, ld_in, ld_out, dtype, alpha, 16, 16)
    assert e.value.status == getattr(tpp, f"TPP_ERR_{status}")


def test_transform_null_pointers_and_empty_shapes(tpp):
    with pytest.raises(tpp.TppError) as e:
        tpp.tpp_transform(tpp.TPP_TR_TRANSPOSE, 4, 4, 4, 4, tpp.TPP_DT_BF16, 1, None, 16)
    assert e.value.status == tpp.TPP_ERR_INVALID_ARG
    # nothing to move: no pointer is looked at, nothing is launched
    for kind in (tpp.TPP_TR_TRANSPOSE, tpp.TPP_TR_VNNI, tpp.TPP_TR_VNNI_TO_VNNI_T):
        tpp.tpp_transform(kind, 0, 5, 8, 8 * 2, tpp.TPP_DT_BF16, 2, None, None)
        tpp.tpp_transform(kind, 5, 0, 16, 16, tpp.TPP_DT_BF16, 2, None, None)


def test_embedding_argument_checks(tpp):
    fake = 1 << 40   # never dereferenced: every call below fails its checks first
    bad = [(-1, 8, 0, 8, 1, 8), (10, 0, 0, 8, 1, 8), (10, 8, 0, 7, 1, 8), (10, 8, 0, 8, 1, 7),
           (10, 8, 5, 8, 1, 8), (10, 8, 0, 8, -1, 8)]
    for M, E, wt, ldw, nb, ldo in bad:
        with pytest.raises(tpp.TppError) as e:
            tpp.tpp_embedding_bag(M, E, wt, fake, ldw, nb, fake, fake, 0, fake, ldo)
        assert e.value.status == tpp.TPP_ERR_INVALID_ARG
    with pytest.raises(tpp.TppError) as e:
        tpp.tpp_embedding_bag(10, 8, 0, fake, 8, 1, None, fake, 0, fake, 8)
    assert e.value.status == tpp.TPP_ERR_INVALID_ARG
    tpp.tpp_embedding_bag(10, 8, 0, fake, 8, 0, fake, fake, 0, fake, 8)   # no bags: a no-op


# ---- the equation planner (Alg. 3 / Alg. 4) is host code: checked here against the oracle ---
EXAMPLE_EQ = [("leaf", 0), ("leaf", 1), ("leaf", 2), ("leaf", 3), ("leaf", 4),
              ("tanh", 0), ("mul", 1, 2), ("sub", 3, 4), ("div", 6, 7), ("add", 5, 8)]


def _rand_tree(rng, k, ternary):
    nodes = []

    def build(k):
        if k == 0:
            nodes.append(("leaf", sum(x[0] == "leaf" for x in nodes)))
            return len(nodes) - 1
        kinds = ["exp", "add"] + (["muladd"] if ternary else [])
        kind = kinds[rng.integers(len(kinds))]
        if kind == "exp":
            c = build(k - 1)
            nodes.append(("exp", c))
        elif kind == "add":
            kl = int(rng.integers(0, k))
            a, b = build(kl), build(k - 1 - kl)
            nodes.append(("add", a, b))
        else:
            ks = rng.multinomial(k - 1, [1 / 3] * 3)
            a, b, c = (build(int(x)) for x in ks)
            nodes.append(("muladd", a, b, c))
        return len(nodes) - 1

    return nodes, build(k)


def test_equation_planner_matches_oracle(tpp):
    import numpy as np
    import oracle
    sc, ts, tm, n = tpp.tpp_equation_plan(EXAMPLE_EQ, 9)
    assert sc[9] == 2 and n == 2
    assert (ts, tm, n) == oracle.eq_plan(EXAMPLE_EQ, 9) and sc == oracle.eq_scores(EXAMPLE_EQ, 9)
    rng = np.random.default_rng(81)
    for trial in range(300):
        nodes, root = _rand_tree(rng, int(rng.integers(1, 12)), ternary=trial % 2 == 1)
        sc, ts, tm, n = tpp.tpp_equation_plan(nodes, root)
        assert sc == oracle.eq_scores(nodes, root), nodes
        assert (ts, tm, n) == oracle.eq_plan(nodes, root), nodes


def test_equation_planner_rejects_malformed_trees(tpp):
    bad = [([("add", 0, 1), ("leaf", 0)], 0),                     # cycle through the root
           ([("leaf", 0), ("exp", 7)], 1),                         # child out of range
           ([("leaf", 0), ("add", 0, 0)], 1),                      # a node reached twice
           ([("leaf", 0)], 3)]                                     # root out of range
    for nodes, root in bad:
        with pytest.raises(tpp.TppError) as e:
            tpp.tpp_equation_plan(nodes, root)
        assert e.value.status == tpp.TPP_ERR_INVALID_ARG
    arr = tpp.eq_nodes([("leaf", 0), ("exp", 0)])
    arr[1].op = tpp.TPP_EQ_OPS["add"]                              # a binary op on one child
    plan = (tpp.tpp_eq_plan_node * 2)()
    import ctypes
    st = tpp._lib.tpp_equation_plan(arr, 2, 1, plan, ctypes.byref(ctypes.c_int32()))
    assert st == tpp.TPP_ERR_INVALID_ARG


def test_equation_execute_host_checks(tpp):
    fake = 1 << 40   # never dereferenced
    nodes = [("leaf", 0), ("leaf", 1), ("add", 0, 1)]
    with pytest.raises(tpp.TppError) as e:           # leaf 1 has no argument
        tpp.tpp_equation_execute(nodes, 2, 4, 4, [(fake, 4, 0, "none")], fake, 4, 0)
    assert e.value.status == tpp.TPP_ERR_INVALID_ARG
    with pytest.raises(tpp.TppError) as e:           # ld < m
        tpp.tpp_equation_execute(nodes, 2, 4, 4, [(fake, 3, 0, "none"), (fake, 4, 0, "none")],
                                 fake, 4, 0)
    assert e.value.status == tpp.TPP_ERR_INVALID_ARG
    # a balanced binary tree of 63 nodes needs 5 temporaries (within the executor's 8; a tree of
    # at most 64 nodes never needs more than that)
    def grow(level):
        if level == 0:
            deep.append(("leaf", 0))
            return len(deep) - 1
        a, b = grow(level - 1), grow(level - 1)
        deep.append(("add", a, b))
        return len(deep) - 1
    deep = []
    root = grow(5)                                    # 63 nodes, score 5: fits
    assert tpp.tpp_equation_plan(deep, root)[3] == 5
    tpp.tpp_equation_execute(deep, root, 0, 4, [(fake, 4, 0, "none")], fake, 4, 0)   # m = 0


def test_a_trans_dispatch_checks(tpp):
    # with A_TRANS the rows of A_i hold k entries: lda >= k is required and suffices (lda < m)
    ok = tpp.make_desc(128, 64, 64, 64, 64, 128, "bf16", "f32", 0.0, "stride", 128 * 64, 64 * 64,
                       flags=("a_trans",))
    assert tpp.tpp_brgemm_dispatch(ok)
    assert "_atrans" in tpp.tpp_brgemm_describe(tpp.tpp_brgemm_dispatch(ok))
    for bad in (tpp.make_desc(128, 64, 64, 32, 64, 128, "bf16", "f32", 0.0, "stride", 128 * 64,
                              64 * 64, flags=("a_trans",)),
                tpp.make_desc(128, 64, 64, 64, 64, 128, "bf16", "f32", 0.0, "stride", 128 * 64,
                              64 * 64)):
        with pytest.raises(tpp.TppError):
            tpp.tpp_brgemm_dispatch(bad)


def test_b_trans_dispatch_checks(tpp):
    # with B_TRANS the k-rows of B_i hold n entries: ldb >= n is required and suffices (ldb < k)
    ok = tpp.make_desc(64, 64, 128, 64, 64, 64, "bf16", "f32", 0.0, "stride", 64 * 128, 128 * 64,
                       flags=("b_trans",))
    assert "_btrans" in tpp.tpp_brgemm_describe(tpp.tpp_brgemm_dispatch(ok))
    with pytest.raises(tpp.TppError):
        tpp.tpp_brgemm_dispatch(tpp.make_desc(64, 64, 128, 64, 32, 64, "bf16", "f32", 0.0,
                                              "stride", 64 * 128, 128 * 64, flags=("b_trans",)))


# ----------------------------------------------------------------------------------------------
# tpp_brgemm_describe_launch: the launch path's own kernel choice, named as the profiler names
# the kernels, without launching (fake device addresses are never dereferenced)
# ----------------------------------------------------------------------------------------------
def _describe(tpp, call, a=1 << 40, b=1 << 41, c=1 << 42, bias=1 << 43):
    h = tpp.tpp_brgemm_dispatch(
        tpp.make_desc(call.m, call.n, call.k, call.lda, call.ldb, call.ldc, call.ab_type,
                      call.c_type, call.beta, call.kind, call.stride_a, call.stride_b,
                      sorted(call.flags)))
    fake = 1 << 44
    offs = fake if call.kind == "offset" else None
    lists = fake if call.kind == "address" else None
    explicit = fake if call.grid is None and call.kind != "address" else None
    return tpp.tpp_brgemm_describe_launch(
        h, call.grid, call.G, explicit, explicit, fake if call.grid is None else None, None,
        a if call.kind != "address" else None, b if call.kind != "address" else None, c,
        bias if call.bias else None, call.count, offs, offs, lists, lists, lists)


def test_describe_launch_names_the_headline_instances(tpp):
    import workloads as wk
    g1, g2 = wk.mlp_block().calls
    assert _describe(tpp, g1) == ("brgemm_bf16_dl_kernel<256, 256, 4, 4, true, 0, true, 0, 64, 0, "
                                  "false, false>")
    assert _describe(tpp, g2) == ("brgemm_bf16_dl_kernel<128, 128, 2, 2, true, 0, true, 0, 64, 0, "
                                  "false, false>")
    # a base off 16-byte alignment takes the unaligned instance of the same tile
    assert _describe(tpp, g1, a=(1 << 40) + 2) == ("brgemm_bf16_dl_kernel<256, 256, 4, 4, true, 0, "
                                                   "false, 0, 64, 0, false, false>")


def test_describe_launch_other_workloads(tpp):
    import workloads as wk
    assert _describe(tpp, wk.fp32_single().calls[0]) == ("brgemm_f32_kernel<true> + "
                                                         "brgemm_f32_split_finish")
    conv = _describe(tpp, wk.conv3x3().calls[0])
    assert conv.startswith("brgemm_bf16_dl_kernel<64, 64, 2, 2, false, 1, false, 0, 64"), conv
    gath = _describe(tpp, wk.gathered().calls[0])
    assert gath.startswith("brgemm_bf16_dl_kernel<128, 128, 2, 2, true, 2, false, 0, 64"), gath
    # the weight gradient of the MLP backward pass splits its stage list
    bw = wk.mlp_backward()
    dw = [c for c in bw.calls if c.c == "dw1"][0]
    assert _describe(tpp, dw).endswith(" + brgemm_dl_split_finish")


def test_describe_launch_empty_grid_and_errors(tpp):
    import workloads as wk
    call = wk.mlp_fc().calls[0]
    h = tpp.tpp_brgemm_dispatch(
        tpp.make_desc(call.m, call.n, call.k, call.lda, call.ldb, call.ldc, call.ab_type,
                      call.c_type, call.beta, call.kind, call.stride_a, call.stride_b,
                      sorted(call.flags)))
    fake = 1 << 40
    g0 = dict(call.grid, gm=0, gn=0)
    assert tpp.tpp_brgemm_describe_launch(h, None, 0, None, None, None, None, fake, fake, fake,
                                          fake, call.count, None, None, None, None, None) == ""
    with pytest.raises(tpp.TppError):   # gm * gn != G
        tpp.tpp_brgemm_describe_launch(h, call.grid, call.G + 1, None, None, None, None, fake,
                                       fake, fake, fake, call.count, None, None, None, None, None)
    with pytest.raises(tpp.TppError):   # bias missing
        tpp.tpp_brgemm_describe_launch(h, call.grid, call.G, None, None, None, None, fake, fake,
                                       fake, None, call.count, None, None, None, None, None)
    del g0


# ----------------------------------------------------------------------------------------------
# tpp_brgemm_execute_batched_noalloc: host-side refusals happen before any device work
# ----------------------------------------------------------------------------------------------
def test_noalloc_refuses_before_device_work(tpp, monkeypatch):
    import workloads as wk
    fake = 1 << 40
    # a handle with an aux bit is refused
    ha = tpp.tpp_brgemm_dispatch(tpp.make_desc(64, 64, 64, 64, 64, 64, "bf16", "bf16",
                                               flags=["relu_inv"]))
    with pytest.raises(tpp.TppError) as e:
        tpp.tpp_brgemm_execute_batched_noalloc(ha, None, 1, None, None, None, None, fake, fake,
                                               fake, None, 1, None, None, None, None, None, 0)
    assert e.value.status == tpp.TPP_ERR_INVALID_ARG
    # a split larger than the scratch array (forced with TPP_SPLIT) is refused with the sizes
    bw = wk.mlp_backward()
    dw = [c for c in bw.calls if c.c == "dw1"][0]
    h = tpp.tpp_brgemm_dispatch(
        tpp.make_desc(dw.m, dw.n, dw.k, dw.lda, dw.ldb, dw.ldc, dw.ab_type, dw.c_type, dw.beta,
                      dw.kind, dw.stride_a, dw.stride_b, sorted(dw.flags)))
    monkeypatch.setenv("TPP_SPLIT", "64")
    with pytest.raises(tpp.TppError) as e:
        tpp.tpp_brgemm_execute_batched_noalloc(h, dw.grid, dw.G, None, None, None, None, fake,
                                               fake, fake, fake if dw.bias else None, dw.count,
                                               None, None, None, None, None, 0)
    assert e.value.status == tpp.TPP_ERR_UNSUPPORTED
    assert "scratch" in tpp.tpp_last_error_message()
