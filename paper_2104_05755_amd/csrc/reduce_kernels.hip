// reduce_kernels.hip -- the Reduce TPP (Table 1) for gfx950.
//
// Folds an m x n column-major tensor (leading dimension ld, fp32 or bf16) along its rows or its
// columns with SUM / MUL / MIN / MAX, of x and/or of x*x, into fp32 outputs.  Reduction by
// columns turns m x n into m x 1 (Sec. 3.1); reduction by rows gives 1 x n.
//
//   BY_ROWS (out[c] = fold over r): each column is contiguous, so one wavefront folds one
//     column (or one row segment of it) with 16-byte loads per lane, then across its 64 lanes
//     with cross-lane shuffles.
//   BY_COLS (out[r] = fold over c): a thread owns 16 bytes of consecutive rows and walks the
//     columns of its workgroup's column range; the column lanes of a workgroup then meet in
//     LDS.  Column ranges of different workgroups meet in a second, tiny pass.
// A batch of G calls (the loop of Alg. 6 around the TPP) runs as one launch: each pass has its
// per-call workgroups G times over, and workgroup b serves call b / per.
// Arithmetic is fp32.  When a shape needs several partial results per output (row segments or
// column ranges), they go to a device work buffer and a second kernel folds them in a fixed
// order (which depends only on the shape), so results do not depend on scheduling.
#include <hip/hip_runtime.h>

#include <math.h>

#include "internal.h"

namespace tpp {
namespace {

constexpr int RT = 256;   // threads per workgroup

template <int OP>
__device__ __forceinline__ float fold(float acc, float v) {
  if (OP == TPP_RED_SUM) return acc + v;
  if (OP == TPP_RED_MUL) return acc * v;
  if (OP == TPP_RED_MIN) return v < acc ? v : acc;
  return v > acc ? v : acc;
}

template <int OP>
__device__ __forceinline__ float fold_identity() {
  if (OP == TPP_RED_SUM) return 0.0f;
  if (OP == TPP_RED_MUL) return 1.0f;
  if (OP == TPP_RED_MIN) return INFINITY;
  return -INFINITY;
}

template <int OP>
__device__ __forceinline__ float wave_fold(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fold<OP>(v, __shfl_xor(v, off, 64));
  return v;
}

template <bool BF16>
__device__ __forceinline__ float load1(const void* base, int64_t idx) {
  if (BF16) return __uint_as_float((uint32_t) static_cast<const uint16_t*>(base)[idx] << 16);
  return static_cast<const float*>(base)[idx];
}

// V consecutive elements starting at idx (16 bytes, aligned): V = 8 for bf16, 4 for fp32.
template <bool BF16, int V>
__device__ __forceinline__ void loadv(const void* base, int64_t idx, float out[V]) {
  if (BF16) {
    const uint4 w = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(base) + idx);
    const uint32_t d[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      out[2 * e] = __uint_as_float(d[e] << 16);
      out[2 * e + 1] = __uint_as_float(d[e] & 0xffff0000u);
    }
  } else {
    const float4 w = *reinterpret_cast<const float4*>(static_cast<const float*>(base) + idx);
    out[0] = w.x; out[1] = w.y; out[2] = w.z; out[3] = w.w;
  }
}

// Batched calls: workgroup b of a launch works on call g = b / per (per workgroups per call).
// Moves p's input and outputs and the work buffer to call g's and returns the workgroup's index
// within its call.  Each call's partials take wsize floats of the work buffer.
template <bool BF16>
__device__ __forceinline__ int64_t batch_of(ReduceParams& p, int64_t per, float*& work,
                                            int64_t wsize) {
  const int64_t bid = blockIdx.x;
  const int64_t g = bid / per;
  if (g > 0) {
    p.in = static_cast<const char*>(p.in) + g * p.in_stride * (BF16 ? 2 : 4);
    if (p.out_x) p.out_x += g * p.out_stride;
    if (p.out_x2) p.out_x2 += g * p.out_stride;
    if (work) work += g * wsize;
  }
  return bid - g * per;
}

// BY_ROWS: wavefront wid folds rows [s*seg_rows, min(m, (s+1)*seg_rows)) of column c, where
// c = wid % n, s = wid / n.  V == 1 means element loads.
template <int OP, bool BF16, int V>
__global__ __launch_bounds__(RT) void reduce_rows_kernel(ReduceParams p, int32_t seg_rows,
                                                         int32_t nseg, float* work, int64_t per) {
  const int lane = threadIdx.x & 63;
  const int64_t lb = batch_of<BF16>(p, per, work, 2LL * nseg * p.n);
  const int64_t wid = lb * (RT / 64) + (threadIdx.x >> 6);
  if (wid >= (int64_t)p.n * nseg) return;
  const int32_t c = (int32_t)(wid % p.n), s = (int32_t)(wid / p.n);
  const int32_t r_lo = s * seg_rows;
  const int32_t r_hi = min(p.m, r_lo + seg_rows);
  const int64_t col = (int64_t)c * p.ld;
  const bool want_x = (p.flags & TPP_RED_X) != 0, want_x2 = (p.flags & TPP_RED_X2) != 0;
  float ax = fold_identity<OP>(), ax2 = fold_identity<OP>();
  const int32_t nv = (r_hi - r_lo) / V;   // full V-chunks
  for (int32_t j = lane; j < nv; j += 64) {
    float x[V];
    if (V == 1) {
      x[0] = load1<BF16>(p.in, col + r_lo + j);
    } else {
      loadv<BF16, V>(p.in, col + r_lo + (int64_t)j * V, x);
    }
#pragma unroll
    for (int e = 0; e < V; ++e) {
      ax = fold<OP>(ax, x[e]);
      ax2 = fold<OP>(ax2, x[e] * x[e]);
    }
  }
  for (int32_t r = r_lo + nv * V + lane; r < r_hi; r += 64) {
    const float x = load1<BF16>(p.in, col + r);
    ax = fold<OP>(ax, x);
    ax2 = fold<OP>(ax2, x * x);
  }
  ax = wave_fold<OP>(ax);
  ax2 = wave_fold<OP>(ax2);
  if (lane == 0) {
    if (nseg == 1) {
      if (want_x) p.out_x[c] = ax;
      if (want_x2) p.out_x2[c] = ax2;
    } else {
      work[(int64_t)s * p.n + c] = ax;
      work[(int64_t)nseg * p.n + (int64_t)s * p.n + c] = ax2;
    }
  }
}

// BY_ROWS with one segment per column and many columns: wavefront wid folds the CG columns
// [wid*CG, min(n, wid*CG + CG)) whole, with every column's chunk of a pass loaded before any is
// folded (CG loads in flight per lane in place of one).
template <int OP, bool BF16, int V, int CG>
__global__ __launch_bounds__(RT) void reduce_rows_group_kernel(ReduceParams p, int64_t per) {
  const int lane = threadIdx.x & 63;
  float* no_work = nullptr;
  const int64_t lb = batch_of<BF16>(p, per, no_work, 0);
  const int64_t wid = lb * (RT / 64) + (threadIdx.x >> 6);
  const int64_t c0 = wid * CG;
  if (c0 >= p.n) return;
  const bool want_x = (p.flags & TPP_RED_X) != 0, want_x2 = (p.flags & TPP_RED_X2) != 0;
  // columns past n repeat the last column's address: loaded, folded, never stored
  int64_t col[CG];
#pragma unroll
  for (int q = 0; q < CG; ++q) col[q] = (c0 + q < p.n ? c0 + q : p.n - 1) * p.ld;
  float ax[CG], ax2[CG];
#pragma unroll
  for (int q = 0; q < CG; ++q) ax[q] = ax2[q] = fold_identity<OP>();
  const int32_t nv = p.m / V;   // full V-chunks
  for (int32_t j = lane; j < nv; j += 64) {
    float x[CG][V];
#pragma unroll
    for (int q = 0; q < CG; ++q) {
      if (V == 1) x[q][0] = load1<BF16>(p.in, col[q] + j);
      else loadv<BF16, V>(p.in, col[q] + (int64_t)j * V, x[q]);
    }
#pragma unroll
    for (int q = 0; q < CG; ++q)
#pragma unroll
      for (int e = 0; e < V; ++e) {
        ax[q] = fold<OP>(ax[q], x[q][e]);
        ax2[q] = fold<OP>(ax2[q], x[q][e] * x[q][e]);
      }
  }
  for (int32_t r = nv * V + lane; r < p.m; r += 64) {
#pragma unroll
    for (int q = 0; q < CG; ++q) {
      const float x = load1<BF16>(p.in, col[q] + r);
      ax[q] = fold<OP>(ax[q], x);
      ax2[q] = fold<OP>(ax2[q], x * x);
    }
  }
#pragma unroll
  for (int q = 0; q < CG; ++q) {
    const float fx = wave_fold<OP>(ax[q]);
    const float fx2 = wave_fold<OP>(ax2[q]);
    if (lane == 0 && c0 + q < p.n) {
      if (want_x) p.out_x[c0 + q] = fx;
      if (want_x2) p.out_x2[c0 + q] = fx2;
    }
  }
}

// BY_COLS: workgroup (rb, s) folds columns [s*col_seg, min(n, (s+1)*col_seg)) for rows
// [rb*TR*V, (rb+1)*TR*V).  Thread t: row vector tr = t % TR, column lane tc = t / TR.
template <int OP, bool BF16, int V>
__global__ __launch_bounds__(RT) void reduce_cols_kernel(ReduceParams p, int32_t TR,
                                                         int32_t col_seg, int32_t nseg,
                                                         int32_t nrb, float* work, int64_t per) {
  __shared__ float sx[RT * V];
  __shared__ float sx2[RT * V];
  const int t = threadIdx.x;
  const int TC = RT / TR;
  const int tr = t % TR, tc = t / TR;
  const int64_t lb = batch_of<BF16>(p, per, work, 2LL * nseg * p.m);
  const int32_t rb = (int32_t)(lb % nrb), s = (int32_t)(lb / nrb);
  const int32_t r0 = rb * TR * V + tr * V;
  const int32_t c_lo = s * col_seg, c_hi = min(p.n, c_lo + col_seg);
  float ax[V], ax2[V];
#pragma unroll
  for (int e = 0; e < V; ++e) ax[e] = ax2[e] = fold_identity<OP>();
  const bool full = r0 + V <= p.m;
  auto load_vec = [&](int32_t c, float (&x)[V]) {
    const int64_t base = (int64_t)c * p.ld + r0;
    if (V > 1 && full) {
      loadv<BF16, V>(p.in, base, x);
    } else {
#pragma unroll
      for (int e = 0; e < V; ++e) x[e] = (r0 + e < p.m) ? load1<BF16>(p.in, base + e) : 0.0f;
    }
  };
  // Four columns per trip, all loads issued before any is folded, into four accumulator sets
  // (combined in a fixed order below): four loads in flight per thread instead of one.
  float bx[4][V], bx2[4][V];
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int e = 0; e < V; ++e) bx[u][e] = bx2[u][e] = fold_identity<OP>();
  int32_t c = c_lo + tc;
  for (; c + 3 * TC < c_hi; c += 4 * TC) {
    float x[4][V];
#pragma unroll
    for (int u = 0; u < 4; ++u) load_vec(c + u * TC, x[u]);
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int e = 0; e < V; ++e) {
        bx[u][e] = fold<OP>(bx[u][e], x[u][e]);
        bx2[u][e] = fold<OP>(bx2[u][e], x[u][e] * x[u][e]);
      }
  }
  for (; c < c_hi; c += TC) {
    float x[V];
    load_vec(c, x);
#pragma unroll
    for (int e = 0; e < V; ++e) {
      bx[0][e] = fold<OP>(bx[0][e], x[e]);
      bx2[0][e] = fold<OP>(bx2[0][e], x[e] * x[e]);
    }
  }
#pragma unroll
  for (int e = 0; e < V; ++e) {
    ax[e] = fold<OP>(fold<OP>(bx[0][e], bx[1][e]), fold<OP>(bx[2][e], bx[3][e]));
    ax2[e] = fold<OP>(fold<OP>(bx2[0][e], bx2[1][e]), fold<OP>(bx2[2][e], bx2[3][e]));
  }
#pragma unroll
  for (int e = 0; e < V; ++e) {
    sx[tc * TR * V + tr * V + e] = ax[e];
    sx2[tc * TR * V + tr * V + e] = ax2[e];
  }
  __syncthreads();
  // Fold the TC column lanes; thread t handles row slot t (and t + RT, ... when TR*V > RT).
  const bool want_x = (p.flags & TPP_RED_X) != 0, want_x2 = (p.flags & TPP_RED_X2) != 0;
  for (int slot = t; slot < TR * V; slot += RT) {
    float fx = sx[slot], fx2 = sx2[slot];
    for (int l = 1; l < TC; ++l) {
      fx = fold<OP>(fx, sx[l * TR * V + slot]);
      fx2 = fold<OP>(fx2, sx2[l * TR * V + slot]);
    }
    const int32_t r = rb * TR * V + slot;
    if (r >= p.m) continue;
    if (nseg == 1) {
      if (want_x) p.out_x[r] = fx;
      if (want_x2) p.out_x2[r] = fx2;
    } else {
      work[(int64_t)s * p.m + r] = fx;
      work[(int64_t)nseg * p.m + (int64_t)s * p.m + r] = fx2;
    }
  }
}

// Second pass: out[o] = fold over s < nseg of work[s * n_out + o] (x part, then x2 part).
// One wavefront per output: lanes take every 64th partial, then fold across the wavefront.
// Moves the combine pass's pointers to call g = blockIdx.x / per of a batch and returns the
// workgroup's index within its call.
__device__ __forceinline__ int64_t combine_batch(int64_t per, int32_t n_out, int32_t nseg,
                                                 int64_t out_stride, const float*& work,
                                                 float*& out_x, float*& out_x2) {
  const int64_t bid = blockIdx.x;
  const int64_t g = bid / per;
  if (g > 0) {
    work += g * 2LL * nseg * n_out;
    if (out_x) out_x += g * out_stride;
    if (out_x2) out_x2 += g * out_stride;
  }
  return bid - g * per;
}

template <int OP>
__global__ __launch_bounds__(RT) void reduce_combine_kernel(const float* work, int32_t n_out,
                                                            int32_t nseg, uint32_t flags,
                                                            float* out_x, float* out_x2,
                                                            int64_t per, int64_t out_stride) {
  const int lane = threadIdx.x & 63;
  const int64_t lb = combine_batch(per, n_out, nseg, out_stride, work, out_x, out_x2);
  const int64_t o = lb * (RT / 64) + (threadIdx.x >> 6);
  if (o >= n_out) return;
  float fx = fold_identity<OP>(), fx2 = fold_identity<OP>();
  for (int32_t s = lane; s < nseg; s += 64) {
    fx = fold<OP>(fx, work[(int64_t)s * n_out + o]);
    fx2 = fold<OP>(fx2, work[(int64_t)nseg * n_out + (int64_t)s * n_out + o]);
  }
  fx = wave_fold<OP>(fx);
  fx2 = wave_fold<OP>(fx2);
  if (lane == 0) {
    if (flags & TPP_RED_X) out_x[o] = fx;
    if (flags & TPP_RED_X2) out_x2[o] = fx2;
  }
}

// Second pass for many outputs: workgroup b folds outputs [64 b, 64 b + 64), lane = output, so
// every partial load is a coalesced 256-byte row; wave w folds partials s = w, w + 4, ... in
// increasing s, and the four wave results are folded in wave order.
template <int OP>
__global__ __launch_bounds__(RT) void reduce_combine_wide_kernel(const float* work, int32_t n_out,
                                                                 int32_t nseg, uint32_t flags,
                                                                 float* out_x, float* out_x2,
                                                                 int64_t per, int64_t out_stride) {
  __shared__ float sx[4][64], sx2[4][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t lb = combine_batch(per, n_out, nseg, out_stride, work, out_x, out_x2);
  const int64_t o = lb * 64 + lane;
  float fx = fold_identity<OP>(), fx2 = fold_identity<OP>();
  if (o < n_out) {
    const float* px = work + o;
    const float* px2 = work + (int64_t)nseg * n_out + o;
    int32_t s = w;
    for (; s + 12 < nseg; s += 16) {   // four partials of each half in flight
      float a[4], b[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        a[u] = px[(int64_t)(s + 4 * u) * n_out];
        b[u] = px2[(int64_t)(s + 4 * u) * n_out];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        fx = fold<OP>(fx, a[u]);
        fx2 = fold<OP>(fx2, b[u]);
      }
    }
    for (; s < nseg; s += 4) {
      fx = fold<OP>(fx, px[(int64_t)s * n_out]);
      fx2 = fold<OP>(fx2, px2[(int64_t)s * n_out]);
    }
  }
  sx[w][lane] = fx;
  sx2[w][lane] = fx2;
  __syncthreads();
  if (w == 0 && o < n_out) {
    fx = fold<OP>(fold<OP>(sx[0][lane], sx[1][lane]), fold<OP>(sx[2][lane], sx[3][lane]));
    fx2 = fold<OP>(fold<OP>(sx2[0][lane], sx2[1][lane]), fold<OP>(sx2[2][lane], sx2[3][lane]));
    if (flags & TPP_RED_X) out_x[o] = fx;
    if (flags & TPP_RED_X2) out_x2[o] = fx2;
  }
}

struct Plan {
  bool by_cols;
  int v;          // elements per load (1, 4 or 8)
  int32_t nseg;   // partial results per output
  int32_t seg;    // rows per segment (BY_ROWS) or columns per range (BY_COLS)
  int32_t tr;     // BY_COLS: row vectors per workgroup
  int32_t nrb;    // BY_COLS: row blocks
  int64_t blocks; // first-pass workgroups
  int32_t cg;     // BY_ROWS with one segment: columns per wavefront (1: the segment kernel)
};

Plan make_plan(const ReduceParams& p) {
  Plan pl{};
  pl.by_cols = (p.flags & TPP_RED_BY_COLS) != 0;
  const int es = p.in_bf16 ? 2 : 4;
  const bool aligned = (reinterpret_cast<uintptr_t>(p.in) & 15) == 0 && ((p.ld * es) % 16) == 0;
  pl.v = aligned ? 16 / es : 1;
  if (!pl.by_cols) {
    const int64_t rows_per_pass = 64LL * pl.v;
    const int64_t max_seg = (p.m + rows_per_pass - 1) / rows_per_pass;
    int64_t nseg = (4096 + p.n - 1) / p.n;   // aim for >= 4096 wavefronts
    nseg = nseg < 1 ? 1 : (nseg > max_seg ? max_seg : nseg);
    if (nseg > 256) nseg = 256;
    const int64_t per = (p.m + nseg - 1) / nseg;
    pl.seg = (int32_t)(((per + rows_per_pass - 1) / rows_per_pass) * rows_per_pass);
    pl.nseg = (int32_t)((p.m + pl.seg - 1) / pl.seg);
    pl.blocks = ((int64_t)p.n * pl.nseg + (RT / 64) - 1) / (RT / 64);
    // whole columns and plenty of them: 2 or 4 columns per wavefront, still >= 4096 wavefronts
    pl.cg = 1;
    if (pl.nseg == 1) {
      pl.cg = p.n >= 4 * 4096 ? 4 : (p.n >= 2 * 4096 ? 2 : 1);
      const int64_t waves = (p.n + pl.cg - 1) / pl.cg;
      pl.blocks = (waves + (RT / 64) - 1) / (RT / 64);
    }
  } else {
    // Up to 64 row vectors per workgroup (at least four column lanes): a tall input gets more
    // row blocks rather than more column ranges, which keeps the partials per output few.
    const int64_t vecs = (p.m + pl.v - 1) / pl.v;
    int32_t tr = 1;
    while (tr < vecs && tr < RT / 4) tr <<= 1;
    // A tall input with enough rows for 512 row blocks of at least 8 row vectors takes fewer
    // row vectors per workgroup (down to 8, up to 2048 row blocks) instead of column ranges:
    // every workgroup then folds whole columns, no combine pass runs, and the many short
    // workgroups keep more loads in flight per CU.
    if (vecs >= 512LL * 8)
      while (tr > 8 && (vecs + tr - 1) / tr < 2048) tr >>= 1;
    pl.tr = tr;
    pl.nrb = (int32_t)((p.m + (int64_t)tr * pl.v - 1) / ((int64_t)tr * pl.v));
    const int32_t tc = RT / tr;
    // otherwise aim for ~1024 workgroups (four per CU), each walking at least 8 columns per
    // column lane, and at most 512 partial results per output for the combine pass
    int64_t nseg = pl.nrb >= 512 ? 1 : (1024 + pl.nrb - 1) / pl.nrb;
    const int64_t max_seg = (p.n + 8LL * tc - 1) / (8LL * tc);
    nseg = nseg < 1 ? 1 : (nseg > max_seg ? max_seg : nseg);
    if (nseg > 512) nseg = 512;
    pl.seg = (int32_t)((p.n + nseg - 1) / nseg);
    pl.nseg = (int32_t)((p.n + pl.seg - 1) / pl.seg);
    pl.blocks = (int64_t)pl.nrb * pl.nseg;
  }
  return pl;
}

template <int OP, bool BF16, int V>
void launch_first(const ReduceParams& p, const Plan& pl, float* work, hipStream_t stream) {
  // with one partial per output the first pass writes the outputs itself (no work buffer)
  float* w = pl.nseg > 1 ? work : nullptr;
  const dim3 grid((unsigned)(pl.blocks * p.G));
  if (!pl.by_cols && pl.cg == 4)
    hipLaunchKernelGGL((reduce_rows_group_kernel<OP, BF16, V, 4>), grid, dim3(RT), 0, stream, p,
                       pl.blocks);
  else if (!pl.by_cols && pl.cg == 2)
    hipLaunchKernelGGL((reduce_rows_group_kernel<OP, BF16, V, 2>), grid, dim3(RT), 0, stream, p,
                       pl.blocks);
  else if (!pl.by_cols)
    hipLaunchKernelGGL((reduce_rows_kernel<OP, BF16, V>), grid, dim3(RT), 0, stream, p, pl.seg,
                       pl.nseg, w, pl.blocks);
  else
    hipLaunchKernelGGL((reduce_cols_kernel<OP, BF16, V>), grid, dim3(RT), 0, stream, p, pl.tr,
                       pl.seg, pl.nseg, pl.nrb, w, pl.blocks);
}

template <int OP>
void launch_op(const ReduceParams& p, const Plan& pl, float* work, hipStream_t stream) {
  if (p.in_bf16) {
    if (pl.v == 8) launch_first<OP, true, 8>(p, pl, work, stream);
    else launch_first<OP, true, 1>(p, pl, work, stream);
  } else {
    if (pl.v == 4) launch_first<OP, false, 4>(p, pl, work, stream);
    else launch_first<OP, false, 1>(p, pl, work, stream);
  }
  if (pl.nseg > 1) {
    const int32_t n_out = pl.by_cols ? p.m : p.n;
    if (n_out >= 512) {   // many outputs: coalesced over outputs
      const int64_t per = (n_out + 63) / 64;
      hipLaunchKernelGGL(reduce_combine_wide_kernel<OP>, dim3((unsigned)(per * p.G)), dim3(RT), 0,
                         stream, work, n_out, pl.nseg, p.flags, p.out_x, p.out_x2, per,
                         p.out_stride);
    } else {              // few outputs: one wavefront per output, lanes over the partials
      const int64_t per = (n_out + 3) / 4;
      hipLaunchKernelGGL(reduce_combine_kernel<OP>, dim3((unsigned)(per * p.G)), dim3(RT), 0,
                         stream, work, n_out, pl.nseg, p.flags, p.out_x, p.out_x2, per,
                         p.out_stride);
    }
  }
}

}  // namespace

int64_t reduce_work_floats(const ReduceParams& p) {
  const Plan pl = make_plan(p);
  const int32_t n_out = pl.by_cols ? p.m : p.n;
  // every pass of the launch (first pass, combine) must fit 2^31 - 1 workgroups
  const int64_t per = pl.blocks > (n_out + 3) / 4 ? pl.blocks : (n_out + 3) / 4;
  if (per > 0x7fffffff / (p.G > 0 ? p.G : 1)) return -1;
  if (pl.nseg <= 1) return 0;
  return 2LL * pl.nseg * n_out * p.G;
}

hipError_t launch_reduce(const ReduceParams& p, float* work, hipStream_t stream) {
  const Plan pl = make_plan(p);
  switch (p.op) {
    case TPP_RED_SUM: launch_op<TPP_RED_SUM>(p, pl, work, stream); break;
    case TPP_RED_MUL: launch_op<TPP_RED_MUL>(p, pl, work, stream); break;
    case TPP_RED_MIN: launch_op<TPP_RED_MIN>(p, pl, work, stream); break;
    default: launch_op<TPP_RED_MAX>(p, pl, work, stream); break;
  }
  return hipGetLastError();
}

}  // namespace tpp
