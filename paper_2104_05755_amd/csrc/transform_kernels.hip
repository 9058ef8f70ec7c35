// transform_kernels.hip -- the Transform TPP (Table 1; Sec. 3.1): Transpose, VNNI formatting
// ([D1][D0] -> [D1/alpha][D0][alpha], the layout of Sec. 3.2.2) and VNNI to VNNI-transpose.
//
// All three only move entries, so they are bound by HBM traffic: each entry is read once and
// written once.  The paper builds its transposes from register shuffle networks (Sec. 3.3.1);
// here a workgroup stages a 64 x 64 tile in LDS, reading it along the input's contiguous
// direction and writing it along the output's, so both sides are coalesced.
//   - Transpose: 16-byte loads and stores when the operands allow (aligned bases, leading
//     dimensions of whole 16-byte units) and the tile is whole; the LDS tile keeps 16-byte
//     chunks XOR-swizzled by column, so the column-wise gathers of the write phase hit distinct
//     banks.  Ragged tiles and other operands move entry by entry.
//   - VNNI: no LDS: each thread writes one 16-byte chunk of an output group, gathering its
//     alpha columns with one (16 / alpha)-byte load each.
//   - VNNI to VNNI-transpose: the tiled kernel with both sides addressed in the VNNI layout,
//     16-byte chunks on whole aligned tiles, entry by entry otherwise.
#include <hip/hip_runtime.h>

#include "brgemm_device.h"
#include "internal.h"

namespace tpp {
namespace {

using dev::gld;
using dev::gst;
using dev::u32x4;

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int TT = 64;     // tile edge, entries
constexpr int TPB = 256;   // threads per workgroup

template <int ES>
struct Entry;
template <>
struct Entry<2> {
  using T = uint16_t;
};
template <>
struct Entry<4> {
  using T = uint32_t;
};

// 16 bytes from V entries, and entry e of a loaded chunk of `words` 32-bit words.
template <int ES>
__device__ __forceinline__ u32x4 pack16(const typename Entry<ES>::T* v) {
  if constexpr (ES == 4) {
    return (u32x4){v[0], v[1], v[2], v[3]};
  } else {
    return (u32x4){v[0] | ((uint32_t)v[1] << 16), v[2] | ((uint32_t)v[3] << 16),
                   v[4] | ((uint32_t)v[5] << 16), v[6] | ((uint32_t)v[7] << 16)};
  }
}
template <int ES>
__device__ __forceinline__ typename Entry<ES>::T entry_of(const uint32_t* words, int e) {
  if constexpr (ES == 4)
    return words[e];
  else
    return (uint16_t)(words[e >> 1] >> (16 * (e & 1)));
}

// Position of entry (c, r) of a staged tile ([c][r], 64 entries per c) with the 16-byte chunks
// of each c XOR-swizzled by c / V: a chunk keeps its 16 bytes together, and V consecutive c of
// one r fall in different chunks.
template <int ES>
__device__ __forceinline__ int tile_pos(int c, int r) {
  constexpr int V = 16 / ES, CH = TT / V;
  return c * TT + (((r / V) ^ ((c / V) % CH)) * V) + r % V;
}

// Workgroup b of a batched launch works on call g = b / per (per workgroups per call), whose
// blocks start g * in_stride and g * out_stride entries on; returns the workgroup's index within
// its call.
template <typename T>
__device__ __forceinline__ int64_t batch_of(const TransformParams& p, int64_t per, const T*& in,
                                            T*& out) {
  const int64_t bid = blockIdx.x;
  const int64_t g = bid / per;
  in = static_cast<const T*>(p.in) + g * p.in_stride;
  out = static_cast<T*>(p.out) + g * p.out_stride;
  return bid - g * per;
}

// Transpose: the n x m output's entry (c, r) = in(r, c).  Tile (r0, c0) of a flattened grid
// (tiles_m tiles along m, per tiles per call).
template <int ES>
__global__ __launch_bounds__(TPB) void transpose_kernel(TransformParams p, int64_t per) {
  using T = typename Entry<ES>::T;
  constexpr int V = 16 / ES, CH = TT / V;
  __shared__ __attribute__((aligned(16))) T lds[TT * TT];
  const int t = threadIdx.x;
  const T* in;
  T* out;
  const int64_t bid = batch_of<T>(p, per, in, out);
  const int32_t r0 = (int32_t)(bid % p.tiles_m) * TT, c0 = (int32_t)(bid / p.tiles_m) * TT;
  const bool whole = r0 + TT <= p.m && c0 + TT <= p.n;
  if (whole && p.vec) {
    // chunk q: input column c0 + q / CH, rows r0 + (q % CH) * V .. + V - 1
    for (int q = t; q < TT * CH; q += TPB) {
      const int cc = q / CH, rv = (q % CH) * V;
      const u32x4 v = gld<u32x4>(in + (int64_t)(c0 + cc) * p.ld_in + r0 + rv);
      *reinterpret_cast<u32x4*>(lds + tile_pos<ES>(cc, rv)) = v;
    }
    __syncthreads();
    // chunk q: output column r0 + q / CH (an input row), entries c0 + (q % CH) * V .. + V - 1
    for (int q = t; q < TT * CH; q += TPB) {
      const int rr = q / CH, cv = (q % CH) * V;
      T v[V];
#pragma unroll
      for (int j = 0; j < V; ++j) v[j] = lds[tile_pos<ES>(cv + j, rr)];
      gst<u32x4>(out + (int64_t)(r0 + rr) * p.ld_out + c0 + cv, pack16<ES>(v));
    }
  } else {
    for (int q = t; q < TT * TT; q += TPB) {
      const int cc = q / TT, rr = q % TT;
      if (r0 + rr < p.m && c0 + cc < p.n)
        lds[tile_pos<ES>(cc, rr)] = gld<T>(in + (int64_t)(c0 + cc) * p.ld_in + r0 + rr);
    }
    __syncthreads();
    for (int q = t; q < TT * TT; q += TPB) {
      const int rr = q / TT, cc = q % TT;
      if (r0 + rr < p.m && c0 + cc < p.n)
        gst<T>(out + (int64_t)(r0 + rr) * p.ld_out + c0 + cc, lds[tile_pos<ES>(cc, rr)]);
    }
  }
}

// VNNI to VNNI-transpose: logical tile rows [r0, r0 + 64), columns [c0, c0 + 64) (both multiples
// of alpha, so groups never straddle tiles), staged as lds[c][r].  Reads walk the input's
// contiguous order (c % alpha fastest, then r), writes the output's (r % alpha fastest, then c).
// Whole tiles with aligned operands move 16-byte chunks on both sides: an input chunk is
// V / alpha rows of one group's alpha columns, an output chunk V / alpha columns of one output
// group's alpha rows.  Output rows from m up to the next multiple of alpha are the zero
// completion of the last group (never in a whole tile).
template <int ES, int ALPHA>
__global__ __launch_bounds__(TPB) void vnni_t_kernel(TransformParams p, int64_t per) {
  using T = typename Entry<ES>::T;
  constexpr int V = 16 / ES, CPG = TT * ALPHA / V;   // 16-byte chunks per group of a tile
  __shared__ T lds[TT][TT + 1];
  const int t = threadIdx.x;
  const T* in;
  T* out;
  const int64_t bid = batch_of<T>(p, per, in, out);
  const int32_t r0 = (int32_t)(bid % p.tiles_m) * TT, c0 = (int32_t)(bid / p.tiles_m) * TT;
  if (r0 + TT <= p.m && c0 + TT <= p.n && p.vec) {
    for (int q = t; q < TT * TT / V; q += TPB) {
      const int gi = q / CPG, j0 = (q % CPG) * V, rr0 = j0 / ALPHA;
      const u32x4 w4 = gld<u32x4>(in + (int64_t)(c0 / ALPHA + gi) * p.ld_in +
                                  (int64_t)(r0 + rr0) * ALPHA);
      const uint32_t w[4] = {w4[0], w4[1], w4[2], w4[3]};
#pragma unroll
      for (int e = 0; e < V; ++e) lds[gi * ALPHA + e % ALPHA][rr0 + e / ALPHA] = entry_of<ES>(w, e);
    }
    __syncthreads();
    for (int q = t; q < TT * TT / V; q += TPB) {
      const int gi = q / CPG, j0 = (q % CPG) * V, cc0 = j0 / ALPHA;
      T v[V];
#pragma unroll
      for (int e = 0; e < V; ++e) v[e] = lds[cc0 + e / ALPHA][gi * ALPHA + e % ALPHA];
      gst<u32x4>(out + (int64_t)(r0 / ALPHA + gi) * p.ld_out + (int64_t)(c0 + cc0) * ALPHA,
                 pack16<ES>(v));
    }
    return;
  }
  const int32_t m_pad = (p.m + ALPHA - 1) / ALPHA * ALPHA;
  for (int q = t; q < TT * TT; q += TPB) {
    const int a = q % ALPHA, rr = (q / ALPHA) % TT, cc = (q / (ALPHA * TT)) * ALPHA + a;
    const int32_t r = r0 + rr, c = c0 + cc;
    if (r < p.m && c < p.n)
      lds[cc][rr] = gld<T>(in + (int64_t)(c / ALPHA) * p.ld_in + (int64_t)r * ALPHA + a);
  }
  __syncthreads();
  for (int q = t; q < TT * TT; q += TPB) {
    const int a = q % ALPHA, cc = (q / ALPHA) % TT, rr = (q / (ALPHA * TT)) * ALPHA + a;
    const int32_t r = r0 + rr, c = c0 + cc;
    if (c < p.n && r < m_pad)
      gst<T>(out + (int64_t)(r / ALPHA) * p.ld_out + (int64_t)c * ALPHA + a,
             r < p.m ? lds[cc][rr] : (T)0);
  }
}

// A (16 / ALPHA)-byte load of the vector path, as 32-bit words.
template <int BYTES>
__device__ __forceinline__ void load_words(const void* src, uint32_t* w) {
  if constexpr (BYTES == 16) {
    const u32x4 x = gld<u32x4>(src);
    w[0] = x[0], w[1] = x[1], w[2] = x[2], w[3] = x[3];
  } else if constexpr (BYTES == 8) {
    const u32x2 x = gld<u32x2>(src);
    w[0] = x[0], w[1] = x[1];
  } else {
    w[0] = gld<uint32_t>(src);
  }
}

// VNNI formatting: thread q writes 16-byte chunk q % cpg of output group g = q / cpg (cpg chunks
// cover the group's m * ALPHA entries): entries j0 .. j0 + V - 1, i.e. rows j0 / ALPHA ..
// (j0 + V) / ALPHA - 1 of the group's ALPHA columns.  Columns past n are the zero completion.
template <int ES, int ALPHA>
__global__ __launch_bounds__(TPB) void vnni_kernel(TransformParams p, int64_t cpg, int64_t total,
                                                   int64_t per) {
  using T = typename Entry<ES>::T;
  constexpr int V = 16 / ES, ROWS = V / ALPHA;
  const T* in;
  T* out;
  const int64_t q = batch_of<T>(p, per, in, out) * TPB + threadIdx.x;
  if (q >= total) return;
  const int64_t g = q / cpg;
  const int64_t j0 = (q - g * cpg) * V;
  const int64_t extent = (int64_t)p.m * ALPHA;
  T* o = out + g * p.ld_out + j0;
  if (p.vec && j0 + V <= extent) {
    const int64_t r0 = j0 / ALPHA;
    T v[V];
#pragma unroll
    for (int a = 0; a < ALPHA; ++a) {
      const int64_t c = g * ALPHA + a;
      uint32_t w[(ROWS * ES + 3) / 4] = {};
      if (c < p.n) load_words<ROWS * ES>(in + c * p.ld_in + r0, w);
#pragma unroll
      for (int e = 0; e < ROWS; ++e) v[e * ALPHA + a] = entry_of<ES>(w, e);
    }
    gst<u32x4>(o, pack16<ES>(v));
  } else {
    for (int e = 0; e < V && j0 + e < extent; ++e) {
      const int64_t j = j0 + e, r = j / ALPHA, c = g * ALPHA + j % ALPHA;
      gst<T>(o + e, c < p.n ? gld<T>(in + c * p.ld_in + r) : (T)0);
    }
  }
}

// A launch of per workgroups for each of the G calls: at most 2^31 - 1 workgroups in all.
inline bool grid_fits(int64_t per, int64_t G) { return per <= 0x7fffffff / (G > 0 ? G : 1); }

template <int ES>
hipError_t launch_es(TransformParams& p, hipStream_t stream) {
  const int64_t tiles_n = (p.n + TT - 1) / TT;
  const int64_t G = p.G;
  if (p.kind == 0) {
    p.tiles_m = (p.m + TT - 1) / TT;
    const int64_t tiles = p.tiles_m * tiles_n;
    if (!grid_fits(tiles, G)) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(transpose_kernel<ES>, dim3((uint32_t)(tiles * G)), dim3(TPB), 0, stream, p,
                       tiles);
  } else if (p.kind == 1) {
    constexpr int V = 16 / ES;
    const int64_t cpg = ((int64_t)p.m * p.alpha + V - 1) / V;
    const int64_t total = cpg * ((p.n + p.alpha - 1) / p.alpha);
    const int64_t blocks = (total + TPB - 1) / TPB;
    if (!grid_fits(blocks, G)) return hipErrorInvalidConfiguration;
    const dim3 grid((uint32_t)(blocks * G));
    switch (p.alpha) {
      case 1: hipLaunchKernelGGL((vnni_kernel<ES, 1>), grid, dim3(TPB), 0, stream, p, cpg, total, blocks); break;
      case 2: hipLaunchKernelGGL((vnni_kernel<ES, 2>), grid, dim3(TPB), 0, stream, p, cpg, total, blocks); break;
      default: hipLaunchKernelGGL((vnni_kernel<ES, 4>), grid, dim3(TPB), 0, stream, p, cpg, total, blocks); break;
    }
  } else {
    const int64_t m_pad = ((int64_t)p.m + p.alpha - 1) / p.alpha * p.alpha;
    p.tiles_m = (m_pad + TT - 1) / TT;
    const int64_t tiles = p.tiles_m * tiles_n;
    if (!grid_fits(tiles, G)) return hipErrorInvalidConfiguration;
    const dim3 grid((uint32_t)(tiles * G));
    switch (p.alpha) {
      case 1: hipLaunchKernelGGL((vnni_t_kernel<ES, 1>), grid, dim3(TPB), 0, stream, p, tiles); break;
      case 2: hipLaunchKernelGGL((vnni_t_kernel<ES, 2>), grid, dim3(TPB), 0, stream, p, tiles); break;
      default: hipLaunchKernelGGL((vnni_t_kernel<ES, 4>), grid, dim3(TPB), 0, stream, p, tiles); break;
    }
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_transform(TransformParams& p, hipStream_t stream) {
  return p.es == 2 ? launch_es<2>(p, stream) : launch_es<4>(p, stream);
}

}  // namespace tpp
