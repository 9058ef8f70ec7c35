"""Seeded synthetic inputs for the batch-reduce GEMM TPP workloads.

This module is the one piece shared by the oracle side (tests, CPU baseline) and the HIP side
(tests, benchmark): it draws random numbers and lays them out, and holds none of the method's
arithmetic.  bf16 inputs are fp32 samples rounded by torch's CPU conversion (a library routine),
stored as ``uint16`` bit patterns; fp32 inputs are ``float32``.

Workloads (all blocks column-major with a leading dimension, i.e. element (r, c) of a block at
base + r + c*ld, the way Alg. 6 lays out its blocked tensors with the b_m / b_k index innermost):

  fp32_single   one stride-based fp32 BRGEMM, m = n = k = 64, 16 pairs, beta = 0
  mlp_fc        fully-connected forward on the blocked layout of Alg. 6, bias + ReLU, bf16 out
  conv3x3       3x3 convolution (stride 1, pad 1) on NCHWc with c = 64 as an offset-based BRGEMM
                per output row (Sec. 5.1.4), ReLU, bf16 out
  mlp_block     transformer MLP: 1024 -> 4096 (bias + GELU-tanh) -> 1024 (bias), bf16 blocked
  gathered      address-based BRGEMM over seeded random block lists (8..64 pairs per output
                block) drawn from pools of blocks, beta = 1, fp32 out
  reduce_bn     the Reduce TPP on a conv output: per-channel sum and sum of squares (the
                statistics step of batchnorm, Sec. 5.1.2)
  embedding_bag sparse embedding lookups (Alg. 5): per bag, the sum of the table rows it lists
  equation_example / layernorm  TPP matrix equations (Sec. 4): the paper's example tree, and a
                layer norm from a Reduce TPP and equations
  mlp_backward  the transformer MLP trained: GEMM1 keeping its pre-activation, then the backward
                pass through both layers (weight transposes, GELU_inv fused into the data
                gradient, weight gradients batch-reduced over token blocks, bias gradients by the
                Reduce TPP)

The default sizes are the full sizes; every generator takes smaller sizes for oracle-speed tests.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np
import torch

BLK = 64


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 samples -> bf16 bit patterns (uint16), rounded by torch's CPU conversion."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16).copy()


def bf16_values(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> the fp32 values they denote (a reinterpretation, no rounding)."""
    return (bits.astype(np.uint32) << 16).view(np.float32)


@dataclass
class Call:
    """One batched BRGEMM call: descriptor fields + instance grid + operand arrays (host)."""
    m: int
    n: int
    k: int
    lda: int
    ldb: int
    ldc: int
    ab_type: str
    c_type: str
    beta: float
    kind: str
    stride_a: int = 0
    stride_b: int = 0
    flags: set = field(default_factory=set)
    G: int = 1
    grid: Optional[dict] = None            # strided form
    a_off: Optional[np.ndarray] = None     # explicit form (element offsets per instance)
    b_off: Optional[np.ndarray] = None
    c_off: Optional[np.ndarray] = None
    bias_off: Optional[np.ndarray] = None
    count: int = 0
    offs_a: Optional[np.ndarray] = None    # offset variant
    offs_b: Optional[np.ndarray] = None
    begin: Optional[np.ndarray] = None     # address variant: CSR over pairs
    idx_a: Optional[np.ndarray] = None     # address variant: element offsets into the pools
    idx_b: Optional[np.ndarray] = None
    a: Optional[str] = None                # names of the arrays in Workload.arrays
    b: Optional[str] = None
    c: Optional[str] = None
    bias: Optional[str] = None
    aux: Optional[str] = None              # tensor shaped as C: saved / read pre-activation

    @property
    def pairs(self) -> int:
        if self.kind == "address":
            return int(self.begin[-1] - self.begin[0])
        return self.G * self.count

    @property
    def flops(self) -> int:
        """Algorithmic FLOPs: 2*m*n*k per multiplied pair of blocks."""
        return 2 * self.m * self.n * self.k * self.pairs


@dataclass
class TransformStep:
    """G Transform TPP calls over blocks ``in_stride`` / ``out_stride`` elements apart."""
    kind: str
    m: int
    n: int
    ld_in: int
    ld_out: int
    dtype: str
    src: str
    dst: str
    G: int = 1
    in_stride: int = 0
    out_stride: int = 0
    alpha: int = 1


@dataclass
class ReduceStep:
    """G Reduce TPP calls; outputs of call g start ``out_stride`` floats after call g - 1's."""
    src: str
    m: int
    n: int
    ld: int
    in_type: str
    op: str
    by: str
    dst_x: Optional[str] = None
    dst_x2: Optional[str] = None
    G: int = 1
    in_stride: int = 0
    out_stride: int = 0


@dataclass
class EmbeddingStep:
    """Sparse embedding gather-reduce (Alg. 5): out row b = sum of the table rows idx[j] for j in
    [begin[b], begin[b+1]); table rows ldw apart, output rows ldo apart."""
    M: int
    E: int
    ldw: int
    ldo: int
    w_type: str
    out_type: str
    w: str = "w"
    begin: str = "begin"
    idx: str = "idx"
    out: str = "out"

    @property
    def n_bags(self) -> int:
        return -1   # from the begin array's length - 1


@dataclass
class EquationStep:
    """A TPP matrix equation (Sec. 4) over an m x n output: ``nodes`` as ("leaf", i) or
    (op, child, ...) tuples, ``leaves`` as (array name, ld, dtype, broadcast) with broadcast in
    "none" / "col" / "row" / "scalar"."""
    nodes: list
    root: int
    m: int
    n: int
    leaves: list
    out: str
    ldo: int
    out_type: str


@dataclass
class Workload:
    name: str
    arrays: dict
    calls: list
    reduce: Optional[dict] = None
    notes: str = ""
    steps: Optional[list] = None   # ordered Call / TransformStep / ReduceStep (chained workloads)

    @property
    def flops(self) -> int:
        return sum(c.flops for c in self.calls)


def _uniform(rng, shape):
    return rng.uniform(-1.0, 1.0, size=shape).astype(np.float32)


def _normal(rng, shape, std):
    return (rng.standard_normal(size=shape) * std).astype(np.float32)


def fp32_single(seed: int = 1, m: int = 64, n: int = 64, k: int = 64, count: int = 16) -> Workload:
    rng = np.random.default_rng(seed)
    a = _uniform(rng, (count, k, m))          # block i: m x k, column-major, lda = m
    b = _uniform(rng, (count, n, k))          # block i: k x n, column-major, ldb = k
    c = np.full((n, m), np.nan, dtype=np.float32)
    call = Call(m, n, k, m, k, m, "f32", "f32", 0.0, "stride", m * k, k * n, set(), G=1,
                grid=dict(gm=1, gn=1, a_step_m=0, b_step_n=0, c_step_m=0, c_step_n=0, bias_step_m=0),
                count=count, a="a", b="b", c="c")
    return Workload("fp32_single", dict(a=a, b=b, c=c), [call])


def mlp_fc(seed: int = 2, minibatch: int = 2048, c_in: int = 1024, k_out: int = 1024) -> Workload:
    """Alg. 6: A = W[Kb][Cb][b_c][b_k] (A role, m = output feature), B = X[Nb][Cb][b_n][b_c]."""
    rng = np.random.default_rng(seed)
    nb, cb, kb = minibatch // BLK, c_in // BLK, k_out // BLK
    x = bf16_bits(_uniform(rng, (nb, cb, BLK, BLK)))
    w = bf16_bits(_uniform(rng, (kb, cb, BLK, BLK)))
    bias = _uniform(rng, (k_out,))
    out = np.full((nb, kb, BLK, BLK), 0x7FC0, dtype=np.uint16)   # NaN-filled, beta = 0
    blk = BLK * BLK
    call = Call(BLK, BLK, BLK, BLK, BLK, BLK, "bf16", "bf16", 0.0, "stride", blk, blk,
                {"bias", "relu"}, G=kb * nb,
                grid=dict(gm=kb, gn=nb, a_step_m=cb * blk, b_step_n=cb * blk, c_step_m=blk,
                          c_step_n=kb * blk, bias_step_m=BLK),
                count=cb, a="w", b="x", c="out", bias="bias")
    return Workload("mlp_fc", dict(x=x, w=w, bias=bias, out=out), [call])


def conv3x3(seed: int = 3, images: int = 28, h: int = 56, w: int = 56, c: int = 64,
            k: int = 64) -> Workload:
    """3x3 convolution, stride 1, pad 1, as an offset-based BRGEMM per output row.

    Input I[img][H][W][c] (NCHWc with one channel block), zero-padded by a setup copy to
    [img][H+2][W+2][c].  Weights Wt[r][s][c][k] (k innermost): the A block for tap (r, s) is the
    k x c matrix at Wt[r][s], column-major with lda = k.  Instance (img, oj) computes output row
    oj: C = out[img][oj] (k x W, ldc = k), pairs (r, s) with B block = the c x W slab of the padded
    input starting at [img][oj + r][s], ldb = c.
    """
    rng = np.random.default_rng(seed)
    x = bf16_bits(_normal(rng, (images, h, w, c), 0.1))
    wt = bf16_bits(_normal(rng, (3, 3, c, k), 0.1))
    xp = np.zeros((images, h + 2, w + 2, c), dtype=np.uint16)
    xp[:, 1:h + 1, 1:w + 1, :] = x
    out = np.full((images, h, w, k), 0x7FC0, dtype=np.uint16)
    taps = [(r, s) for r in range(3) for s in range(3)]
    offs_a = np.array([(r * 3 + s) * c * k for r, s in taps], dtype=np.int64)
    offs_b = np.array([(r * (w + 2) + s) * c for r, s in taps], dtype=np.int64)
    img, oj = np.meshgrid(np.arange(images), np.arange(h), indexing="ij")
    b_off = ((img * (h + 2) * (w + 2) + oj * (w + 2)) * c).reshape(-1).astype(np.int64)
    c_off = ((img * h * w + oj * w) * k).reshape(-1).astype(np.int64)
    call = Call(k, w, c, k, c, k, "bf16", "bf16", 0.0, "offset", 0, 0, {"relu"}, G=images * h,
                a_off=np.zeros(images * h, dtype=np.int64), b_off=b_off, c_off=c_off,
                count=9, offs_a=offs_a, offs_b=offs_b, a="wt", b="xp", c="out")
    return Workload("conv3x3", dict(x=x, wt=wt, xp=xp, out=out), [call],
                    reduce=dict(src="out", m=k, n=images * h * w, ld=k, in_type="bf16", op="sum",
                                by="cols", want=("x", "x2")))


def mlp_block(seed: int = 4, tokens: int = 8192, hidden: int = 1024, inter: int = 4096) -> Workload:
    """Transformer MLP as two blocked stride-based BRGEMM calls (Alg. 6 twice)."""
    rng = np.random.default_rng(seed)
    nb, hb, ib = tokens // BLK, hidden // BLK, inter // BLK
    blk = BLK * BLK
    x = bf16_bits(_normal(rng, (nb, hb, BLK, BLK), 1.0))
    w1 = bf16_bits(_normal(rng, (ib, hb, BLK, BLK), 0.02))
    b1 = _normal(rng, (inter,), 0.02)
    w2 = bf16_bits(_normal(rng, (hb, ib, BLK, BLK), 0.02))
    b2 = _normal(rng, (hidden,), 0.02)
    hmid = np.full((nb, ib, BLK, BLK), 0x7FC0, dtype=np.uint16)
    y = np.full((nb, hb, BLK, BLK), 0x7FC0, dtype=np.uint16)
    g1 = Call(BLK, BLK, BLK, BLK, BLK, BLK, "bf16", "bf16", 0.0, "stride", blk, blk,
              {"bias", "gelu_tanh"}, G=ib * nb,
              grid=dict(gm=ib, gn=nb, a_step_m=hb * blk, b_step_n=hb * blk, c_step_m=blk,
                        c_step_n=ib * blk, bias_step_m=BLK),
              count=hb, a="w1", b="x", c="h", bias="b1")
    g2 = Call(BLK, BLK, BLK, BLK, BLK, BLK, "bf16", "bf16", 0.0, "stride", blk, blk,
              {"bias"}, G=hb * nb,
              grid=dict(gm=hb, gn=nb, a_step_m=ib * blk, b_step_n=ib * blk, c_step_m=blk,
                        c_step_n=hb * blk, bias_step_m=BLK),
              count=ib, a="w2", b="h", c="y", bias="b2")
    return Workload("mlp_block", dict(x=x, w1=w1, b1=b1, w2=w2, b2=b2, h=hmid, y=y), [g1, g2])


def gathered(seed: int = 5, n_out: int = 4096, pool: int = 8192, m: int = 128, n: int = 128,
             k: int = 64, min_len: int = 8, max_len: int = 64) -> Workload:
    """Address-based BRGEMM: each output block reduces a random list of (A, B) pool blocks.

    List lengths are uniform on {min_len..max_len}; A and B indices are independent, uniform on
    the pool, with replacement.  A pool block is m x k (lda = m), a B pool block k x n (ldb = k).
    """
    rng = np.random.default_rng(seed)
    apool = bf16_bits(_uniform(rng, (pool, k, m)))
    bpool = bf16_bits(_uniform(rng, (pool, n, k)))
    c = _uniform(rng, (n_out, n, m))
    lens = rng.integers(min_len, max_len + 1, size=n_out)
    begin = np.zeros(n_out + 1, dtype=np.int64)
    begin[1:] = np.cumsum(lens)
    ia = rng.integers(0, pool, size=int(begin[-1]))
    ib = rng.integers(0, pool, size=int(begin[-1]))
    call = Call(m, n, k, m, k, m, "bf16", "f32", 1.0, "address", 0, 0, set(), G=n_out,
                c_off=(np.arange(n_out, dtype=np.int64) * m * n), begin=begin,
                idx_a=(ia * m * k).astype(np.int64), idx_b=(ib * k * n).astype(np.int64),
                a="apool", b="bpool", c="c")
    return Workload("gathered", dict(apool=apool, bpool=bpool, c=c), [call])


def mlp_backward(seed: int = 6, tokens: int = 8192, hidden: int = 1024,
                 inter: int = 4096) -> Workload:
    """One training step's worth of the transformer MLP's first layer forward and both layers'
    backward, on the blocked layouts of :func:`mlp_block` (column-major 64 x 64 blocks).

    Forward (kept for back-propagation): Z = W1 X + b1 saved in ``z`` (bf16, H's layout), H =
    gelu(Z) in ``h``.  The incoming gradient dY (N(0,1), Y's layout [Nb][Hb][64n][64h]) then gives
      dZ  = (W2^T dY) * gelu'(Z)      B1: A = W2 blocks read transposed (A_TRANS), GELU_inv, bf16
      dW2 = sum over tokens dY H^T    B2: A = dY, B = H blocks read transposed (B_TRANS), fp32
      db2 = sum over tokens dY        two Reduce TPP calls (over token blocks, then within one)
      dX  = W1^T dZ                   B3: A = W1 blocks read transposed (A_TRANS), bf16
      dW1 = sum over tokens dZ X^T    B4: A = dZ, B = X blocks read transposed (B_TRANS), fp32
      db1 = sum over tokens dZ        two Reduce TPP calls
    A block read with A_TRANS or B_TRANS is its own transpose as stored (k contiguous per row of
    W^T, n contiguous per k-row of H^T and X^T), so no transposed copy is made.  The weight
    gradients keep W's blocked layout, dX keeps X's.
    """
    rng = np.random.default_rng(seed)
    nb, hb, ib = tokens // BLK, hidden // BLK, inter // BLK
    blk = BLK * BLK
    x = bf16_bits(_normal(rng, (nb, hb, BLK, BLK), 1.0))
    w1 = bf16_bits(_normal(rng, (ib, hb, BLK, BLK), 0.02))
    b1 = _normal(rng, (inter,), 0.02)
    w2 = bf16_bits(_normal(rng, (hb, ib, BLK, BLK), 0.02))
    dy = bf16_bits(_normal(rng, (nb, hb, BLK, BLK), 1.0))
    nan16 = lambda shape: np.full(shape, 0x7FC0, dtype=np.uint16)
    nan32 = lambda shape: np.full(shape, np.nan, dtype=np.float32)
    arrays = dict(x=x, w1=w1, b1=b1, w2=w2, dy=dy,
                  z=nan16((nb, ib, BLK, BLK)), h=nan16((nb, ib, BLK, BLK)),
                  dz=nan16((nb, ib, BLK, BLK)), dx=nan16((nb, hb, BLK, BLK)),
                  dw1=nan32((ib, hb, BLK, BLK)), dw2=nan32((hb, ib, BLK, BLK)),
                  p1=nan32((ib * blk,)), p2=nan32((hb * blk,)),
                  db1=nan32((inter,)), db2=nan32((hidden,)))
    sq = lambda **kw: dict(dict(gm=1, gn=1, a_step_m=0, b_step_n=0, c_step_m=0, c_step_n=0,
                                bias_step_m=0), **kw)
    fwd = Call(BLK, BLK, BLK, BLK, BLK, BLK, "bf16", "bf16", 0.0, "stride", blk, blk,
               {"bias", "gelu_tanh", "save_preact"}, G=ib * nb,
               grid=sq(gm=ib, gn=nb, a_step_m=hb * blk, b_step_n=hb * blk, c_step_m=blk,
                       c_step_n=ib * blk, bias_step_m=BLK),
               count=hb, a="w1", b="x", c="h", bias="b1", aux="z")
    # dZ[nb][ib] (i x n) = gelu'(Z) * sum_hb W2[hb][ib]^T (i x h) dY[nb][hb] (h x n)
    b1c = Call(BLK, BLK, BLK, BLK, BLK, BLK, "bf16", "bf16", 0.0, "stride", ib * blk, blk,
               {"gelu_tanh_inv", "a_trans"}, G=ib * nb,
               grid=sq(gm=ib, gn=nb, a_step_m=blk, b_step_n=hb * blk, c_step_m=blk,
                       c_step_n=ib * blk),
               count=hb, a="w2", b="dy", c="dz", aux="z")
    # dW2[hb][ib] (h x i) = sum_nb dY[nb][hb] (h x n) H[nb][ib]^T (n x i)
    b2c = Call(BLK, BLK, BLK, BLK, BLK, BLK, "bf16", "f32", 0.0, "stride", hb * blk, ib * blk,
               {"b_trans"}, G=hb * ib,
               grid=sq(gm=hb, gn=ib, a_step_m=blk, b_step_n=blk, c_step_m=ib * blk,
                       c_step_n=blk),
               count=nb, a="dy", b="h", c="dw2")
    # dX[nb][hb] (h x n) = sum_ib W1[ib][hb]^T (h x i) dZ[nb][ib] (i x n)
    b3c = Call(BLK, BLK, BLK, BLK, BLK, BLK, "bf16", "bf16", 0.0, "stride", hb * blk, blk,
               {"a_trans"}, G=hb * nb,
               grid=sq(gm=hb, gn=nb, a_step_m=blk, b_step_n=ib * blk, c_step_m=blk,
                       c_step_n=hb * blk),
               count=ib, a="w1", b="dz", c="dx")
    # dW1[ib][hb] (i x h) = sum_nb dZ[nb][ib] (i x n) X[nb][hb]^T (n x h)
    b4c = Call(BLK, BLK, BLK, BLK, BLK, BLK, "bf16", "f32", 0.0, "stride", ib * blk, hb * blk,
               {"b_trans"}, G=ib * hb,
               grid=sq(gm=ib, gn=hb, a_step_m=blk, b_step_n=blk, c_step_m=hb * blk,
                       c_step_n=blk),
               count=nb, a="dz", b="x", c="dw1")
    # bias gradients: rows (feature within block, token within block, feature block) of the
    # gradient summed over the token blocks, then each 64 x 64 block's columns summed
    red = lambda src, fb, p, db: [
        ReduceStep(src, fb * blk, nb, fb * blk, "bf16", "sum", "cols", dst_x=p),
        ReduceStep(p, BLK, BLK, BLK, "f32", "sum", "cols", dst_x=db, G=fb, in_stride=blk,
                   out_stride=BLK)]
    steps = [fwd, b1c, b2c, *red("dy", hb, "p2", "db2"), b3c, b4c,
             *red("dz", ib, "p1", "db1")]
    return Workload("mlp_backward", arrays, [fwd, b1c, b2c, b3c, b4c], steps=steps)


def embedding_bag(seed: int = 7, rows: int = 1_000_000, dim: int = 128, bags: int = 16384,
                  min_pool: int = 1, max_pool: int = 64, w_type: str = "f32",
                  out_type: str = "f32", pad: int = 0) -> Workload:
    """DLRM-style sparse embedding lookups (Alg. 5): a table of ``rows`` x ``dim`` entries, U[-1,1];
    ``bags`` multi-hot lookups of a pooling factor uniform on {min_pool..max_pool}, indices
    uniform on the table with replacement (CSR: begin[bags + 1], idx).  ``pad`` widens the table's
    and the output's row strides.  The paper defers DLRM's table sizes to earlier work; these
    sizes stand in for one large table of its MLPerf-style configuration."""
    rng = np.random.default_rng(seed)
    ldw, ldo = dim + pad, dim + pad
    wv = _uniform(rng, (rows * ldw,))
    w = wv if w_type == "f32" else bf16_bits(wv)
    lens = rng.integers(min_pool, max_pool + 1, size=bags)
    begin = np.zeros(bags + 1, dtype=np.int64)
    begin[1:] = np.cumsum(lens)
    idx = rng.integers(0, rows, size=int(begin[-1])).astype(np.int64)
    out = np.full(bags * ldo, np.nan, np.float32) if out_type == "f32" else \
        np.full(bags * ldo, 0x7FC0, np.uint16)
    st = EmbeddingStep(rows, dim, ldw, ldo, w_type, out_type)
    return Workload("embedding_bag", dict(w=w, begin=begin, idx=idx, out=out), [], steps=[st])


# The paper's example equation Out = Tanh(T0) + (T1 x T2) / (T3 - T4), elementwise.
EXAMPLE_EQUATION = [("leaf", 0), ("leaf", 1), ("leaf", 2), ("leaf", 3), ("leaf", 4),
                    ("tanh", 0), ("mul", 1, 2), ("sub", 3, 4), ("div", 6, 7), ("add", 5, 8)]


def equation_example(seed: int = 8, m: int = 4096, n: int = 4096) -> Workload:
    """The example equation of Sec. 4 on m x n fp32 tensors: T0 U[-2,2], T1 and T2 U[-1,1],
    T3 U[1,2] and T4 U[-2,-1] (the divisor stays at least 2 away from zero); fp32 output."""
    rng = np.random.default_rng(seed)
    t = [rng.uniform(lo, hi, m * n).astype(np.float32)
         for lo, hi in ((-2, 2), (-1, 1), (-1, 1), (1, 2), (-2, -1))]
    arrays = {f"t{i}": t[i] for i in range(5)}
    arrays["out"] = np.full(m * n, np.nan, np.float32)
    st = EquationStep(EXAMPLE_EQUATION, 9, m, n, [(f"t{i}", m, "f32", "none") for i in range(5)],
                      "out", m, "f32")
    return Workload("equation_example", arrays, [], steps=[st])


def layernorm(seed: int = 9, features: int = 1024, tokens: int = 8192, eps: float = 1e-5) -> Workload:
    """Layer normalization over the features of each token, from TPPs (Sec. 5.1.2 builds its
    norms from reduce and equation TPPs): X (features x tokens, bf16, column per token) ->
      1. Reduce by rows: per token, sum of x and of x^2 (fp32)
      2. equation on 1 x tokens: rs = 1 / sqrt(s2 / F - mu^2 + eps), mu = s / F a subtree
      3. equation on features x tokens: Y = (X - mu) * rs * gamma + beta, mu = s / F again a
         subtree; s and rs broadcast over the rows, gamma and beta over the columns; bf16
         output.
    (mu as its own 1 x tokens launch, or rs as a subtree of step 3 evaluated per element, both
    measured slower.)  X ~ N(0.5, 1), gamma ~ N(1, 0.1), beta ~ N(0, 0.1)."""
    rng = np.random.default_rng(seed)
    x = bf16_bits((rng.standard_normal(features * tokens) + 0.5).astype(np.float32))
    gamma = (1.0 + 0.1 * rng.standard_normal(features)).astype(np.float32)
    beta = (0.1 * rng.standard_normal(features)).astype(np.float32)
    inv_f = np.array([1.0 / features], np.float32)
    eps_a = np.array([eps], np.float32)
    nan = lambda k: np.full(k, np.nan, np.float32)
    arrays = dict(x=x, gamma=gamma, beta=beta, inv_f=inv_f, eps=eps_a, s=nan(tokens),
                  s2=nan(tokens), rs=nan(tokens), y=np.full(features * tokens, 0x7FC0, np.uint16))
    red = ReduceStep("x", features, tokens, features, "bf16", "sum", "rows", dst_x="s",
                     dst_x2="s2")
    # rs = rcp(sqrt(add(sub(mul(s2, 1/F), square(mul(s, 1/F))), eps)))
    rs = EquationStep([("leaf", 0), ("leaf", 1), ("mul", 0, 1), ("leaf", 2), ("leaf", 1),
                       ("mul", 3, 4), ("square", 5), ("sub", 2, 6), ("leaf", 3), ("add", 7, 8),
                       ("sqrt", 9), ("rcp", 10)], 11, 1, tokens,
                      [("s2", 1, "f32", "none"), ("inv_f", 1, "f32", "scalar"),
                       ("s", 1, "f32", "none"), ("eps", 1, "f32", "scalar")], "rs", 1, "f32")
    # Y = muladd(mul(sub(x, mul(s, 1/F)), rs), gamma, beta)
    y = EquationStep([("leaf", 0), ("leaf", 1), ("leaf", 2), ("mul", 1, 2), ("sub", 0, 3),
                      ("leaf", 3), ("mul", 4, 5), ("leaf", 4), ("leaf", 5),
                      ("muladd", 6, 7, 8)], 9, features, tokens,
                     [("x", features, "bf16", "none"), ("s", 1, "f32", "row"),
                      ("inv_f", 1, "f32", "scalar"), ("rs", 1, "f32", "row"),
                      ("gamma", 1, "f32", "col"), ("beta", 1, "f32", "col")], "y", features, "bf16")
    return Workload("layernorm", arrays, [], steps=[red, rs, y])


def softmax(seed: int = 10, keys: int = 512, columns: int = 32768) -> Workload:
    """Softmax over the keys of each column of attention scores, from TPPs (Sec. 5.1.1 expresses
    it as two equation trees around reduce TPPs): X (keys x columns, bf16, a column per query and
    head) ->
      1. Reduce by rows with MAX: per column, the largest score (fp32)
      2. equation X' = exp(X - max), the maximum broadcast over the rows; fp32 output
      3. Reduce by rows with SUM of X' (fp32)
      4. equation Y = X' * rcp(sum), the sum broadcast over the rows; bf16 output.
    The stand-in for BERT-Large attention: 512 keys, 32768 columns (16 heads x 512 queries x 4
    sequences), scores 2 * N(0, 1)."""
    rng = np.random.default_rng(seed)
    x = bf16_bits((2.0 * rng.standard_normal(keys * columns)).astype(np.float32))
    nan = lambda k: np.full(k, np.nan, np.float32)
    arrays = dict(x=x, mx=nan(columns), xe=nan(keys * columns), s=nan(columns),
                  y=np.full(keys * columns, 0x7FC0, np.uint16))
    red_max = ReduceStep("x", keys, columns, keys, "bf16", "max", "rows", dst_x="mx")
    # X' = exp(sub(x, max))
    e = EquationStep([("leaf", 0), ("leaf", 1), ("sub", 0, 1), ("exp", 2)], 3, keys, columns,
                     [("x", keys, "bf16", "none"), ("mx", 1, "f32", "row")], "xe", keys, "f32")
    red_sum = ReduceStep("xe", keys, columns, keys, "f32", "sum", "rows", dst_x="s")
    # Y = mul(x', rcp(sum))
    y = EquationStep([("leaf", 0), ("leaf", 1), ("rcp", 1), ("mul", 0, 2)], 3, keys, columns,
                     [("xe", keys, "f32", "none"), ("s", 1, "f32", "row")], "y", keys, "bf16")
    return Workload("softmax", arrays, [], steps=[red_max, e, red_sum, y])


CONFIGS = {
    1: fp32_single,
    2: mlp_fc,
    3: conv3x3,
    4: mlp_block,
    5: gathered,
}


def small_case(rng: np.random.Generator, m: int, n: int, k: int, count: int, kind: str,
               ab_type: str, c_type: str, beta: float, flags: set, pad: int = 0,
               integer: bool = False) -> Workload:
    """One random BRGEMM call of arbitrary shape for sweeps.

    Operands live in one pool per side; the pairs are laid out per ``kind`` (stride: blocks
    ``stride`` apart; offset: a shuffled list of block offsets; address: a shuffled list of
    block addresses, with repeats).  ``pad`` widens every leading dimension.  ``integer`` draws
    small integers (exact in bf16 and in fp32 sums) for bit-exact checks.
    """
    lda, ldb, ldc = m + pad, k + pad, m + pad
    a_blk, b_blk = lda * k, ldb * n
    nblk = max(count, 1) + 2
    draw = (lambda shape: rng.integers(-4, 5, size=shape).astype(np.float32)) if integer \
        else (lambda shape: _uniform(rng, shape))
    conv = (lambda v: v) if ab_type == "f32" else bf16_bits
    a = conv(draw((nblk * a_blk,)))
    b = conv(draw((nblk * b_blk,)))
    cval = draw((n * ldc,))
    c = cval if c_type == "f32" else bf16_bits(cval)
    if beta == 0.0:
        c = np.full_like(c, np.nan) if c_type == "f32" else np.full_like(c, 0x7FC0)
    bias = draw((m,)) if "bias" in flags else None
    call = Call(m, n, k, lda, ldb, ldc, ab_type, c_type, beta, kind, flags=set(flags), G=1,
                a="a", b="b", c="c", bias="bias" if bias is not None else None)
    if kind == "stride":
        call.stride_a, call.stride_b = a_blk, b_blk
        call.count = count
        call.grid = dict(gm=1, gn=1, a_step_m=0, b_step_n=0, c_step_m=0, c_step_n=0,
                         bias_step_m=0)
    elif kind == "offset":
        call.count = count
        call.offs_a = (rng.permutation(nblk)[:count] * a_blk).astype(np.int64)
        call.offs_b = (rng.permutation(nblk)[:count] * b_blk).astype(np.int64)
    else:
        call.begin = np.array([0, count], dtype=np.int64)
        call.idx_a = (rng.integers(0, nblk, size=count) * a_blk).astype(np.int64)
        call.idx_b = (rng.integers(0, nblk, size=count) * b_blk).astype(np.int64)
    arrays = dict(a=a, b=b, c=c)
    if bias is not None:
        arrays["bias"] = bias
    return Workload("small", arrays, [call])
