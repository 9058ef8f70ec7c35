// embedding_kernels.hip -- the sparse embedding gather-reduce of Alg. 5 for gfx950.
//
// One wavefront per bag.  A table row is split into 16-byte chunks (4 fp32 or 8 bf16 entries);
// lpr lanes cover one row's chunks (all of them when the row has at most 64 chunks) and the
// wavefront's 64 / lpr row slots take every slot-th listed index, so one load instruction reads
// that many rows.  Each slot keeps U rows in flight (their index loads, then their row loads,
// then the additions), which plays the part of Alg. 5's unrolled accumulators and next-row
// prefetch.  The slots meet through cross-lane shuffles in slot order, and the accumulation
// order depends only on the bag's list, so results do not vary between runs.  The sum is fp32
// in registers and each output row is stored once.  Rows whose chunks are not 16-byte aligned
// take an entry-per-lane kernel.  Indices outside [0, M) add nothing (the table is never read
// outside its rows).
#include <hip/hip_runtime.h>

#include "brgemm_device.h"
#include "internal.h"

namespace tpp {
namespace {

using namespace dev;

constexpr int ET = 256;   // threads per workgroup: 4 wavefronts, one bag each
constexpr int U = 4;      // rows in flight per row slot

// V entries of a 16-byte chunk, widened to fp32 (bf16: the top half of an fp32, exact).
template <bool W_BF16, int V>
__device__ __forceinline__ void widen16(u32x4 w, float (&x)[V]) {
  if constexpr (W_BF16) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[2 * e] = __uint_as_float(w[e] << 16);
      x[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) x[e] = __uint_as_float(w[e]);
  }
}

// N consecutive output entries at o (rounded to bf16 or stored as fp32), 16-byte stores when
// aligned.
template <bool OUT_BF16, int N>
__device__ __forceinline__ void store_row_part(void* o, const float (&v)[N]) {
  if constexpr (OUT_BF16) {
    uint16_t* q = static_cast<uint16_t*>(o);
    if constexpr (N == 8) {
      if ((reinterpret_cast<uintptr_t>(q) & 15) == 0) {
        gst<u32x4>(q, (u32x4){pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                              pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7])});
        return;
      }
    }
    if constexpr (N == 4) {
      if ((reinterpret_cast<uintptr_t>(q) & 7) == 0) {
        gst<u32x2>(q, (u32x2){pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])});
        return;
      }
    }
#pragma unroll
    for (int e = 0; e < N; ++e) gst<uint16_t>(q + e, f32_to_bf16_bits(v[e]));
  } else {
    float* q = static_cast<float*>(o);
    if constexpr (N % 4 == 0) {
      if ((reinterpret_cast<uintptr_t>(q) & 15) == 0) {
#pragma unroll
        for (int g = 0; g < N / 4; ++g)
          gst<f32x4>(q + 4 * g, (f32x4){v[4 * g], v[4 * g + 1], v[4 * g + 2], v[4 * g + 3]});
        return;
      }
    }
#pragma unroll
    for (int e = 0; e < N; ++e) gst<float>(q + e, v[e]);
  }
}

// 16-byte chunk path: E a multiple of V, the table and its row stride 16-byte aligned.
// lpr lanes per row (chunks c0 + lane % lpr of a column group), rpw = 64 / lpr row slots.
template <bool W_BF16, bool OUT_BF16>
__global__ __launch_bounds__(ET) void embedding_vec_kernel(EmbeddingParams p, int32_t lpr,
                                                           int32_t rpw) {
  constexpr int V = W_BF16 ? 8 : 4;
  constexpr int ES = W_BF16 ? 2 : 4;
  const int lane = threadIdx.x & 63;
  const int64_t b = (int64_t)blockIdx.x * (ET / 64) + (threadIdx.x >> 6);
  if (b >= p.n_bags) return;   // b is the same for the whole wavefront
  const int64_t j0 = p.begin[b], j1 = p.begin[b + 1];
  const int32_t cpr = p.E / V;
  const int r = lane / lpr, cl = lane - (lane / lpr) * lpr;
  const bool slot_ok = r < rpw;
  const char* wb = static_cast<const char*>(p.W);
  for (int32_t c0 = 0; c0 < cpr; c0 += lpr) {
    const int32_t c = c0 + cl;
    const bool ok = slot_ok && c < cpr;
    float acc[V];
#pragma unroll
    for (int e = 0; e < V; ++e) acc[e] = 0.0f;
    for (int64_t j = j0 + r; j < j1; j += (int64_t)rpw * U) {
      int64_t row[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t jj = j + (int64_t)u * rpw;
        row[u] = jj < j1 ? gld<int64_t>(p.idx + jj) : -1;
      }
      u32x4 x[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const bool take = ok && row[u] >= 0 && row[u] < p.M;
        x[u] = take ? gld<u32x4>(wb + (row[u] * p.ldw + (int64_t)c * V) * ES)
                    : (u32x4){0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        float v[V];
        widen16<W_BF16, V>(x[u], v);
#pragma unroll
        for (int e = 0; e < V; ++e) acc[e] += v[e];
      }
    }
    // slot 0 adds slots 1, 2, ... in order
    for (int s = 1; s < rpw; ++s) {
#pragma unroll
      for (int e = 0; e < V; ++e) {
        const float t = __shfl(acc[e], cl + s * lpr, 64);
        if (r == 0) acc[e] += t;
      }
    }
    if (r == 0 && c < cpr) {
      char* ob = static_cast<char*>(p.out) + (b * p.ldo + (int64_t)c * V) * (OUT_BF16 ? 2 : 4);
      store_row_part<OUT_BF16, V>(ob, acc);
    }
  }
}

// Entry-per-lane path for any E, stride and alignment.
template <bool W_BF16, bool OUT_BF16>
__global__ __launch_bounds__(ET) void embedding_elem_kernel(EmbeddingParams p) {
  const int lane = threadIdx.x & 63;
  const int64_t b = (int64_t)blockIdx.x * (ET / 64) + (threadIdx.x >> 6);
  if (b >= p.n_bags) return;
  const int64_t j0 = p.begin[b], j1 = p.begin[b + 1];
  for (int32_t e = lane; e < p.E; e += 64) {
    float acc = 0.0f;
    for (int64_t j = j0; j < j1; ++j) {
      const int64_t row = gld<int64_t>(p.idx + j);
      if (row < 0 || row >= p.M) continue;
      const int64_t at = row * p.ldw + e;
      acc += W_BF16 ? bf16_bits_to_f32(gld<uint16_t>(static_cast<const uint16_t*>(p.W) + at))
                    : gld<float>(static_cast<const float*>(p.W) + at);
    }
    const float v[1] = {acc};
    char* ob = static_cast<char*>(p.out) + (b * p.ldo + e) * (OUT_BF16 ? 2 : 4);
    store_row_part<OUT_BF16, 1>(ob, v);
  }
}

template <bool W_BF16, bool OUT_BF16>
void launch_typed(const EmbeddingParams& p, dim3 grid, hipStream_t stream) {
  constexpr int V = W_BF16 ? 8 : 4;
  const int es = W_BF16 ? 2 : 4;
  const bool vec = p.E % V == 0 && (reinterpret_cast<uintptr_t>(p.W) & 15) == 0 &&
                   (p.ldw * es) % 16 == 0;
  if (vec) {
    const int32_t cpr = p.E / V;
    const int32_t lpr = cpr < 64 ? cpr : 64;
    hipLaunchKernelGGL((embedding_vec_kernel<W_BF16, OUT_BF16>), grid, dim3(ET), 0, stream, p,
                       lpr, 64 / lpr);
  } else {
    hipLaunchKernelGGL((embedding_elem_kernel<W_BF16, OUT_BF16>), grid, dim3(ET), 0, stream, p);
  }
}

}  // namespace

hipError_t launch_embedding(const EmbeddingParams& p, hipStream_t stream) {
  const int64_t blocks = (p.n_bags + ET / 64 - 1) / (ET / 64);
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  const dim3 grid((uint32_t)blocks);
  if (p.w_bf16)
    p.out_bf16 ? launch_typed<true, true>(p, grid, stream) : launch_typed<true, false>(p, grid, stream);
  else
    p.out_bf16 ? launch_typed<false, true>(p, grid, stream) : launch_typed<false, false>(p, grid, stream);
  return hipGetLastError();
}

}  // namespace tpp
