// brgemm_kernels.hip -- the batch-reduce GEMM TPP kernel family for gfx950 (CDNA4).
//
// Computes, for every instance g of a launch and every (r, c) of its m x n output block,
//     C(r, c) = cvt( act( beta * C(r, c) + sum_i sum_p A_i(r, p) B_i(p, c) + bias[r] ) )
// (Table 3 BRGEMM; Sec. 2.3 variants; the epilogue TPPs of Table 1 / Table 2 fused before the
// single store as Sec. 2.1 principle 5 allows).
//
// Structure, following Alg. 2 re-tiled for the GPU:
//   - a workgroup owns one BM x BN tile of the "virtual C" of its tile group.  For a strided
//     instance grid the virtual C is the (gm*m) x (gn*n) matrix formed by the instances' output
//     blocks side by side, so a tile may fuse several neighbouring instances (they share their
//     A_i rows and B_i columns, as the ib_m / ib_n loops of Alg. 6 do); for an explicit grid the
//     virtual C is one instance's m x n block;
//   - Alg. 2's loops over the pairs i and over k become one flat loop, in steps of BK=64, over
//     stages; each stage copies an A_i panel (BM x 64) and a B_i panel (64 x BN) from HBM into
//     one of two LDS buffers with 16-byte loads, while the MFMAs consume the other buffer;
//   - A is M-contiguous in memory but the MFMA wants 8 consecutive k per lane, so every thread
//     loads an 8x8 bf16 sub-block (8 columns of 8 rows) and transposes it in registers before
//     its LDS store; B is already K-contiguous and is copied as is;
//   - fp32 accumulators stay in registers for the whole reduction (v_mfma_f32_32x32x16_bf16);
//   - the epilogue (beta*C, bias, ReLU / GELU-tanh, fp32 -> bf16) runs on the accumulators and
//     each output element is stored once.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <string>

#include "brgemm_device.h"
#include "internal.h"

namespace tpp {
namespace {

using namespace dev;

// ---------------------------------------------------------------------------------------------
// Epilogue shared by all kernels.  The accumulator layout of a 32x32 MFMA tile: lane l holds
// column l%32, and in register v the row 8*(v/4) + 4*(l/32) + v%4.
// ---------------------------------------------------------------------------------------------
template <bool GENERIC>
__device__ __forceinline__ void store_group(const BrgemmParams& p, const Instance& in, int32_t R0,
                                            int32_t C, const float v_in[4]) {
  // Column C of the virtual C -> element offset in C (relative to the instance base).
  int64_t col_off;
  if (p.fused) {
    if (C >= p.vcols) return;
    const int32_t gi = C / p.n, c = C - gi * p.n;
    col_off = (int64_t)gi * p.c_step_n + (int64_t)c * p.ldc;
  } else {
    if (C >= p.n) return;
    col_off = (int64_t)C * p.ldc;
  }
  const float* bias = p.bias;
  const bool has_bias = (p.flags & TPP_EPI_BIAS) != 0;
  if (!GENERIC) {
    // m % 8 == 0: the four rows R0..R0+3 are valid together and belong to one instance.
    int64_t row_off, bias_idx;
    if (p.fused) {
      if (R0 >= p.vrows) return;
      const int32_t gi = R0 / p.m, r = R0 - gi * p.m;
      row_off = (int64_t)gi * p.c_step_m + r;
      bias_idx = (int64_t)gi * p.bias_step_m + r;
    } else {
      if (R0 >= p.m) return;
      row_off = R0;
      bias_idx = in.bias + R0;
    }
    const int64_t e0 = in.c + row_off + col_off;
    float v[4] = {v_in[0], v_in[1], v_in[2], v_in[3]};
    if (p.c_bf16) {
      uint16_t* cp = static_cast<uint16_t*>(p.c) + e0;
      const bool vec = (reinterpret_cast<uintptr_t>(cp) & 7) == 0;
      if (p.beta != 0.0f) {
        uint32_t h[4];
        if (vec) {
          const uint2 w = *reinterpret_cast<const uint2*>(cp);
          h[0] = w.x & 0xffff; h[1] = w.x >> 16; h[2] = w.y & 0xffff; h[3] = w.y >> 16;
        } else {
          for (int e = 0; e < 4; ++e) h[e] = cp[e];
        }
        for (int e = 0; e < 4; ++e) v[e] = p.beta * bf16_bits_to_f32(h[e]) + v[e];
      }
      if (has_bias)
        for (int e = 0; e < 4; ++e) v[e] += bias[bias_idx + e];
      if (p.flags & EPI_AUX_MASK) epi_aux<4>(p, e0, v);
      uint32_t o[4];
      for (int e = 0; e < 4; ++e) o[e] = f32_to_bf16_bits(activate(v[e], p.flags));
      if (vec) {
        *reinterpret_cast<uint2*>(cp) = make_uint2(o[0] | (o[1] << 16), o[2] | (o[3] << 16));
      } else {
        for (int e = 0; e < 4; ++e) cp[e] = (uint16_t)o[e];
      }
    } else {
      float* cp = static_cast<float*>(p.c) + e0;
      const bool vec = (reinterpret_cast<uintptr_t>(cp) & 15) == 0;
      if (p.beta != 0.0f) {
        if (vec) {
          const float4 w = *reinterpret_cast<const float4*>(cp);
          v[0] = p.beta * w.x + v[0]; v[1] = p.beta * w.y + v[1];
          v[2] = p.beta * w.z + v[2]; v[3] = p.beta * w.w + v[3];
        } else {
          for (int e = 0; e < 4; ++e) v[e] = p.beta * cp[e] + v[e];
        }
      }
      if (has_bias)
        for (int e = 0; e < 4; ++e) v[e] += bias[bias_idx + e];
      if (p.flags & EPI_AUX_MASK) epi_aux<4>(p, e0, v);
      for (int e = 0; e < 4; ++e) v[e] = activate(v[e], p.flags);
      if (vec) {
        *reinterpret_cast<float4*>(cp) = make_float4(v[0], v[1], v[2], v[3]);
      } else {
        for (int e = 0; e < 4; ++e) cp[e] = v[e];
      }
    }
  } else {
    for (int e = 0; e < 4; ++e) {
      const int32_t R = R0 + e;
      int64_t row_off, bias_idx;
      if (p.fused) {
        if (R >= p.vrows) continue;
        const int32_t gi = R / p.m, r = R - gi * p.m;
        row_off = (int64_t)gi * p.c_step_m + r;
        bias_idx = (int64_t)gi * p.bias_step_m + r;
      } else {
        if (R >= p.m) continue;
        row_off = R;
        bias_idx = in.bias + R;
      }
      const int64_t ei = in.c + row_off + col_off;
      float v1[1] = {v_in[e]};
      if (p.c_bf16) {
        uint16_t* cp = static_cast<uint16_t*>(p.c) + ei;
        if (p.beta != 0.0f) v1[0] = p.beta * bf16_bits_to_f32(*cp) + v1[0];
        if (has_bias) v1[0] += bias[bias_idx];
        if (p.flags & EPI_AUX_MASK) epi_aux<1>(p, ei, v1);
        *cp = f32_to_bf16_bits(activate(v1[0], p.flags));
      } else {
        float* cp = static_cast<float*>(p.c) + ei;
        if (p.beta != 0.0f) v1[0] = p.beta * *cp + v1[0];
        if (has_bias) v1[0] += bias[bias_idx];
        if (p.flags & EPI_AUX_MASK) epi_aux<1>(p, ei, v1);
        *cp = activate(v1[0], p.flags);
      }
    }
  }
}

// ---------------------------------------------------------------------------------------------
// bf16 kernel family
// ---------------------------------------------------------------------------------------------
// 16 bytes = 8 bf16 of one column, zero when `ok` is false; element loads if the address is not
// 16-byte aligned.
__device__ __forceinline__ uint4 load8(const uint16_t* ptr, bool ok, bool aligned) {
  uint4 v = make_uint4(0u, 0u, 0u, 0u);
  if (ok) {
    if (aligned) {
      v = *reinterpret_cast<const uint4*>(ptr);
    } else {
      v.x = (uint32_t)ptr[0] | ((uint32_t)ptr[1] << 16);
      v.y = (uint32_t)ptr[2] | ((uint32_t)ptr[3] << 16);
      v.z = (uint32_t)ptr[4] | ((uint32_t)ptr[5] << 16);
      v.w = (uint32_t)ptr[6] | ((uint32_t)ptr[7] << 16);
    }
  }
  return v;
}

__device__ __forceinline__ uint32_t word(const uint4& v, int d) {
  return d == 0 ? v.x : d == 1 ? v.y : d == 2 ? v.z : v.w;
}

// Transpose an 8x8 bf16 sub-block held as 8 k-columns of 8 rows into 8 rows of 8 k, and store
// the rows (16 B each) into the K-contiguous LDS panel.
__device__ __forceinline__ void store_a_transposed(uint16_t* dst_row0, const uint4 col[8]) {
#pragma unroll
  for (int mi = 0; mi < 8; ++mi) {
    const int d = mi >> 1;
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t lo = word(col[2 * e], d), hi = word(col[2 * e + 1], d);
      w[e] = (mi & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
    }
    *reinterpret_cast<uint4*>(dst_row0 + mi * LDS_ROW) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

template <int BM, int BN, int WAVES_M, int WAVES_N, bool GENERIC>
__global__ __launch_bounds__(NT) void brgemm_bf16_kernel(BrgemmParams p) {
  constexpr int WTM = BM / WAVES_M, WTN = BN / WAVES_N;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int KCH = BK / 8;                        // 8-element k chunks per stage
  constexpr int A_SUB = (BM / 8) * KCH;              // 8x8 sub-blocks of the A panel
  constexpr int A_REP = (A_SUB + NT - 1) / NT;
  constexpr int B_CH = BN * KCH;                     // 16-byte chunks of the B panel
  constexpr int B_REP = (B_CH + NT - 1) / NT;
  constexpr int STAGE = (BM + BN) * LDS_ROW;
  static_assert(WAVES_M * WAVES_N * 64 == NT, "4 waves");
  static_assert(TM >= 1 && TN >= 1, "wave tile at least 32x32");

  __shared__ __attribute__((aligned(16))) uint16_t lds[2 * STAGE];

  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int wm = wave % WAVES_M, wn = wave / WAVES_M;
  const TileCoord tc = decode_tile(p, BM, BN);
  const Instance in = instance_of(p, tc.g);
  const int32_t ksteps = (p.k + BK - 1) / BK;
  const int64_t stages = in.npairs * ksteps;

  // Staging assignments, fixed for the whole reduction.
  int64_t a_off[A_REP][GENERIC ? 8 : 1];
  bool a_ok[A_REP][GENERIC ? 8 : 1];
  int a_kc[A_REP], a_row[A_REP];
#pragma unroll
  for (int rep = 0; rep < A_REP; ++rep) {
    const int q = t + NT * rep;
    a_kc[rep] = q % KCH;
    a_row[rep] = (q / KCH) * 8;
#pragma unroll
    for (int e = 0; e < (GENERIC ? 8 : 1); ++e) {
      a_off[rep][e] = 0;
      a_ok[rep][e] = (q < A_SUB) && row_in_a(p, tc.row0 + a_row[rep] + e, a_off[rep][e]);
    }
  }
  int64_t b_off[B_REP];
  bool b_ok[B_REP];
  int b_kc[B_REP], b_col[B_REP];
#pragma unroll
  for (int rep = 0; rep < B_REP; ++rep) {
    const int q = t + NT * rep;
    b_kc[rep] = q % KCH;
    b_col[rep] = q / KCH;
    b_off[rep] = 0;
    b_ok[rep] = (q < B_CH) && col_in_b(p, tc.col0 + b_col[rep], b_off[rep]);
  }

  uint4 a_reg[A_REP][8];
  uint4 b_reg[B_REP];

  auto load_stage = [&](int64_t s) {
    const int64_t i = s / ksteps;
    const int32_t kk = (int32_t)(s - i * ksteps) * BK;
    const uint16_t* pa;
    const uint16_t* pb;
    pair_bases<uint16_t>(p, in, i, pa, pb);
    const bool aligned =
        !GENERIC && ((reinterpret_cast<uintptr_t>(pa) | reinterpret_cast<uintptr_t>(pb)) & 15) == 0;
#pragma unroll
    for (int rep = 0; rep < A_REP; ++rep) {
      const int32_t k0 = kk + a_kc[rep] * 8;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if (!GENERIC) {
          const bool ok = a_ok[rep][0] && k0 < p.k;
          a_reg[rep][j] = load8(pa + a_off[rep][0] + (int64_t)(k0 + j) * p.lda, ok, aligned);
        } else {
          // element loads: each of the 8 rows and the k index checked on its own
          uint32_t h[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const bool ok = a_ok[rep][e] && (k0 + j) < p.k;
            h[e] = ok ? pa[a_off[rep][e] + (int64_t)(k0 + j) * p.lda] : 0u;
          }
          a_reg[rep][j] = make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16),
                                     h[4] | (h[5] << 16), h[6] | (h[7] << 16));
        }
      }
    }
#pragma unroll
    for (int rep = 0; rep < B_REP; ++rep) {
      const int32_t k0 = kk + b_kc[rep] * 8;
      if (!GENERIC) {
        b_reg[rep] = load8(pb + b_off[rep] + k0, b_ok[rep] && k0 < p.k, aligned);
      } else {
        uint32_t h[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const bool ok = b_ok[rep] && (k0 + e) < p.k;
          h[e] = ok ? pb[b_off[rep] + k0 + e] : 0u;
        }
        b_reg[rep] = make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16),
                                h[6] | (h[7] << 16));
      }
    }
  };

  auto store_stage = [&](int buf) {
    uint16_t* As = lds + buf * STAGE;
    uint16_t* Bs = As + BM * LDS_ROW;
#pragma unroll
    for (int rep = 0; rep < A_REP; ++rep) {
      if (t + NT * rep < A_SUB)
        store_a_transposed(As + a_row[rep] * LDS_ROW + a_kc[rep] * 8, a_reg[rep]);
    }
#pragma unroll
    for (int rep = 0; rep < B_REP; ++rep) {
      if (t + NT * rep < B_CH)
        *reinterpret_cast<uint4*>(Bs + b_col[rep] * LDS_ROW + b_kc[rep] * 8) = b_reg[rep];
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[tm][tn][v] = 0.0f;

  const int frag_row = lane & 31;
  const int frag_k = (lane >> 5) * 8;

  if (stages > 0) {
    load_stage(0);
    store_stage(0);
    __syncthreads();
    for (int64_t s = 0; s < stages; ++s) {
      const int buf = (int)(s & 1);
      if (s + 1 < stages) load_stage(s + 1);   // global loads in flight during the MFMAs
      const uint16_t* As = lds + buf * STAGE;
      const uint16_t* Bs = As + BM * LDS_ROW;
#pragma unroll
      for (int kq = 0; kq < BK / 16; ++kq) {
        bf16x8 af[TM], bfr[TN];
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
          af[tm] = *reinterpret_cast<const bf16x8*>(
              As + (wm * WTM + tm * 32 + frag_row) * LDS_ROW + kq * 16 + frag_k);
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
          bfr[tn] = *reinterpret_cast<const bf16x8*>(
              Bs + (wn * WTN + tn * 32 + frag_row) * LDS_ROW + kq * 16 + frag_k);
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
#pragma unroll
          for (int tn = 0; tn < TN; ++tn)
            acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[tm], bfr[tn], acc[tm][tn],
                                                                  0, 0, 0);
      }
      if (s + 1 < stages) store_stage(buf ^ 1);
      __syncthreads();
    }
  }

  // Epilogue on the accumulators, one store per output element.
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const int32_t C = tc.col0 + wn * WTN + tn * 32 + (lane & 31);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int32_t R0 = tc.row0 + wm * WTM + tm * 32 + q * 8 + (lane >> 5) * 4;
        const float v[4] = {acc[tm][tn][q * 4 + 0], acc[tm][tn][q * 4 + 1],
                            acc[tm][tn][q * 4 + 2], acc[tm][tn][q * 4 + 3]};
        store_group<GENERIC>(p, in, R0, C, v);
      }
    }
}

// ---------------------------------------------------------------------------------------------
// bf16 16-byte-load kernel.  Preconditions (checked on the host): m, k, lda, ldb and every
// element step of the grid are multiples of 8, so each 8-element chunk a thread moves is
// contiguous and, when the pair's block bases are 16-byte aligned (checked per stage, uniform
// over the workgroup), aligned.  FULL: every tile is complete (no row, column or k tail), so
// the loads carry no bounds logic at all; otherwise out-of-range chunks read a clamped,
// in-range address and are replaced by zeros without branching.
// ---------------------------------------------------------------------------------------------
// Transpose an 8 x SK bf16 sub-block held as SK k-columns of 8 rows into 8 rows of SK k, and
// store the rows (2*SK bytes each) into the K-contiguous LDS panel.
template <int SK>
__device__ __forceinline__ void store_a_transposed_v(uint16_t* dst_row0, const u32x4 col[SK]) {
#pragma unroll
  for (int mi = 0; mi < 8; ++mi) {
    const int d = mi >> 1;
    uint32_t w[SK / 2];
#pragma unroll
    for (int e = 0; e < SK / 2; ++e) {
      const uint32_t lo = col[2 * e][d], hi = col[2 * e + 1][d];
      w[e] = (mi & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
    }
    if constexpr (SK == 8)
      *reinterpret_cast<u32x4*>(dst_row0 + mi * LDS_ROW) = (u32x4){w[0], w[1], w[2], w[3]};
    else
      *reinterpret_cast<uint2*>(dst_row0 + mi * LDS_ROW) = make_uint2(w[0], w[1]);
  }
}

template <int BM, int BN, int WAVES_M, int WAVES_N, bool FULL, int KIND, bool ALIGNED>
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N) void brgemm_bf16_vec_kernel(BrgemmParams p) {
  // Register prefetch depth: two stages ahead with one wave per SIMD, one stage ahead with two
  // waves per SIMD (the second wave hides the latency, and the registers are needed for it).
  constexpr int DEPTH = (WAVES_M * WAVES_N > 4) ? 1 : 2;
  constexpr int NTH = 64 * WAVES_M * WAVES_N;        // threads per workgroup
  constexpr int WTM = BM / WAVES_M, WTN = BN / WAVES_N;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int KCH = BK / 8;                        // 8-element k chunks per stage
  // A moves in 8-row x SK-k sub-blocks; SK = 4 when 8x8 sub-blocks would leave threads idle.
  constexpr int SK = ((BM / 8) * (BK / 8) >= NTH) ? 8 : 4;
  constexpr int KCA = BK / SK;
  constexpr int A_SUB = (BM / 8) * KCA;
  constexpr int A_REP = (A_SUB + NTH - 1) / NTH;
  constexpr int B_CH = BN * KCH;                     // 16-byte chunks of the B panel
  constexpr int B_REP = (B_CH + NTH - 1) / NTH;
  constexpr int STAGE = (BM + BN) * LDS_ROW;
  constexpr int EP_ROW = WTM + 4;                    // epilogue slab: 32 columns x WTM rows fp32
  static_assert(TM >= 1 && TN >= 1, "wave tile at least 32x32");
  static_assert(WAVES_M * WAVES_N * 32 * EP_ROW * 4 <= 2 * STAGE * 2,
                "epilogue slabs fit in the stage buffers");

  __shared__ __attribute__((aligned(16))) uint16_t lds[2 * STAGE];

  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int wm = wave % WAVES_M, wn = wave / WAVES_M;
  const TileCoord tc = decode_tile(p, BM, BN);
  const Instance in = instance_of(p, tc.g);
  const int32_t ksteps = (p.k + BK - 1) / BK;
  const int32_t stages = (int32_t)(in.npairs * ksteps);

  // Staging assignments, fixed for the whole reduction.  Out-of-range rows / columns keep
  // offset 0 (an in-range address) and a false flag.
  int64_t a_off[A_REP];
  bool a_ok[A_REP];
  int a_kc[A_REP], a_row[A_REP];
#pragma unroll
  for (int rep = 0; rep < A_REP; ++rep) {
    const int q = t + NTH * rep;
    a_kc[rep] = q % KCA;
    a_row[rep] = (q / KCA) * 8;
    a_off[rep] = 0;
    a_ok[rep] = (q < A_SUB) && row_in_a(p, tc.row0 + a_row[rep], a_off[rep]);
    if (!a_ok[rep]) a_off[rep] = 0;
  }
  int64_t b_off[B_REP];
  bool b_ok[B_REP];
  int b_kc[B_REP], b_col[B_REP];
#pragma unroll
  for (int rep = 0; rep < B_REP; ++rep) {
    const int q = t + NTH * rep;
    b_kc[rep] = q % KCH;
    b_col[rep] = q / KCH;
    b_off[rep] = 0;
    b_ok[rep] = (q < B_CH) && col_in_b(p, tc.col0 + b_col[rep], b_off[rep]);
    if (!b_ok[rep]) b_off[rep] = 0;
  }

  // Two register sets for staged operands: while the MFMAs consume LDS buffer s&1, set s&1
  // receives the global loads of stage s+2 and set (s+1)&1 (loaded one stage earlier) is written
  // to LDS buffer (s+1)&1 in between the MFMAs.
  struct Staged {
    u32x4 a[A_REP][SK];
    u32x4 b[B_REP];
  };
  Staged st0;
  Staged st1;

  auto load_stage = [&](int32_t s, Staged& r) {
    const int32_t i = s / ksteps;
    const int32_t kk = (s - i * ksteps) * BK;
    const uint16_t* pa;
    const uint16_t* pb;
    pair_bases_k<KIND, uint16_t>(p, in, i, pa, pb);
    const bool aligned =
        ALIGNED || ((reinterpret_cast<uintptr_t>(pa) | reinterpret_cast<uintptr_t>(pb)) & 15) == 0;
    if (ALIGNED || aligned) {
#pragma unroll
      for (int rep = 0; rep < A_REP; ++rep) {
        const int32_t k0 = kk + a_kc[rep] * SK;
        const bool ok = FULL || (a_ok[rep] && k0 < p.k);
        const int32_t kc = (FULL || k0 < p.k) ? k0 : 0;
        const uint16_t* base = pa + a_off[rep] + (int64_t)kc * p.lda;
#pragma unroll
        for (int j = 0; j < SK; ++j) {
          const u32x4 v = ld16(base + (int64_t)j * p.lda);
          r.a[rep][j] = FULL ? v : keep_if(v, ok);
        }
      }
#pragma unroll
      for (int rep = 0; rep < B_REP; ++rep) {
        const int32_t k0 = kk + b_kc[rep] * 8;
        const bool ok = FULL || (b_ok[rep] && k0 < p.k);
        const int32_t kc = (FULL || k0 < p.k) ? k0 : 0;
        const u32x4 v = ld16(pb + b_off[rep] + kc);
        r.b[rep] = FULL ? v : keep_if(v, ok);
      }
    } else {
#pragma unroll
      for (int rep = 0; rep < A_REP; ++rep) {
        const int32_t k0 = kk + a_kc[rep] * SK;
        const bool ok = FULL || (a_ok[rep] && k0 < p.k);
        const int32_t kc = (FULL || k0 < p.k) ? k0 : 0;
        const uint16_t* base = pa + a_off[rep] + (int64_t)kc * p.lda;
#pragma unroll
        for (int j = 0; j < SK; ++j)
          r.a[rep][j] = keep_if(ld16_unaligned(base + (int64_t)j * p.lda), ok);
      }
#pragma unroll
      for (int rep = 0; rep < B_REP; ++rep) {
        const int32_t k0 = kk + b_kc[rep] * 8;
        const bool ok = FULL || (b_ok[rep] && k0 < p.k);
        const int32_t kc = (FULL || k0 < p.k) ? k0 : 0;
        r.b[rep] = keep_if(ld16_unaligned(pb + b_off[rep] + kc), ok);
      }
    }
  };

  auto store_a = [&](int buf, const Staged& r) {
    uint16_t* As = lds + buf * STAGE;
#pragma unroll
    for (int rep = 0; rep < A_REP; ++rep) {
      if (A_SUB % NTH == 0 || t + NTH * rep < A_SUB)
        store_a_transposed_v<SK>(As + a_row[rep] * LDS_ROW + a_kc[rep] * SK, r.a[rep]);
    }
  };
  auto store_b = [&](int buf, const Staged& r) {
    uint16_t* Bs = lds + buf * STAGE + BM * LDS_ROW;
#pragma unroll
    for (int rep = 0; rep < B_REP; ++rep) {
      if (B_CH % NTH == 0 || t + NTH * rep < B_CH)
        *reinterpret_cast<u32x4*>(Bs + b_col[rep] * LDS_ROW + b_kc[rep] * 8) = r.b[rep];
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[tm][tn][v] = 0.0f;

  const int frag_row = lane & 31;
  const int frag_k = (lane >> 5) * 8;

  // MFMAs of one LDS buffer: the fragments of k-step kq+1 are read while the MFMAs of kq run;
  // hook(kq) runs after the MFMAs of k-step kq are issued.
  auto compute = [&](int buf, auto&& hook) {
    const uint16_t* As = lds + buf * STAGE;
    const uint16_t* Bs = As + BM * LDS_ROW;
    bf16x8 fa[2][TM], fb[2][TN];
    auto frags = [&](int kq, bf16x8* a, bf16x8* b) {
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
        a[tm] = *reinterpret_cast<const bf16x8*>(
            As + (wm * WTM + tm * 32 + frag_row) * LDS_ROW + kq * 16 + frag_k);
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
        b[tn] = *reinterpret_cast<const bf16x8*>(
            Bs + (wn * WTN + tn * 32 + frag_row) * LDS_ROW + kq * 16 + frag_k);
    };
    frags(0, fa[0], fb[0]);
#pragma unroll
    for (int kq = 0; kq < BK / 16; ++kq) {
      if (kq + 1 < BK / 16) frags(kq + 1, fa[(kq + 1) & 1], fb[(kq + 1) & 1]);
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
          acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[kq & 1][tm], fb[kq & 1][tn],
                                                                acc[tm][tn], 0, 0, 0);
      hook(kq);
    }
  };

  if (stages > 0) {
    load_stage(0, st0);
    if (DEPTH == 2 && stages > 1) load_stage(1, st1);
    store_a(0, st0);
    store_b(0, st0);
    __syncthreads();
    int32_t s = 0;
    // One stage; PAR = s & 1 is a compile-time constant so the register sets are never indexed
    // at run time.
    auto step = [&](auto par) {
      constexpr int PAR = decltype(par)::value;
      const bool more = s + 1 < stages;
      if constexpr (DEPTH == 2) {
        Staged& cur = PAR ? st1 : st0;   // stage s (already in LDS buffer PAR): free for s+2
        Staged& nxt = PAR ? st0 : st1;   // stage s+1, loaded one stage ago
        if (s + 2 < stages) load_stage(s + 2, cur);
        compute(PAR, [&](int kq) {
          if (more && kq == 1) store_a(PAR ^ 1, nxt);
          if (more && kq == 2) store_b(PAR ^ 1, nxt);
        });
      } else {
        // one register set: stage s+1 is loaded now and written to LDS after the MFMAs
        if (more) load_stage(s + 1, st0);
        compute(PAR, [&](int) {});
        if (more) {
          store_a(PAR ^ 1, st0);
          store_b(PAR ^ 1, st0);
        }
      }
      __syncthreads();
      ++s;
    };
    while (s + 1 < stages) {
      step(IntC<0>());
      step(IntC<1>());
    }
    if (s < stages) step(IntC<0>());
  }

  epilogue_via_lds<WTM, WTN, TM, TN, FULL>(p, in, tc, wm, wn, lane, wave,
                                          reinterpret_cast<float*>(lds), acc);
}

// ---------------------------------------------------------------------------------------------
// fp32 kernel: 64x64 tile, 4 waves of 32x32, v_mfma_f32_32x32x2f32, element loads with full
// bounds checks (any shape, leading dimension or alignment).
// ---------------------------------------------------------------------------------------------
constexpr int F_BM = 64, F_BN = 64, F_BK = 32;
constexpr int F_AROW = F_BM + 4;   // A panel stored k-major: As[k][m]
constexpr int F_BROW = F_BK + 1;   // B panel stored n-major: Bs[n][k], odd stride

__global__ __launch_bounds__(NT) void brgemm_f32_kernel(BrgemmParams p) {
  __shared__ float As[F_BK * F_AROW];
  __shared__ float Bs[F_BN * F_BROW];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  // With a split, workgroup bid takes chunk bid % split of tile bid / split's pair list.
  const int32_t split = p.split > 1 ? p.split : 1;
  const int64_t tile_bid = (int64_t)blockIdx.x / split;
  const int32_t chunk = (int32_t)((int64_t)blockIdx.x - tile_bid * split);
  const TileCoord tc = decode_tile_at(p, F_BM, F_BN, tile_bid);
  const Instance in = instance_of(p, tc.g);
  const int64_t pair_lo = in.npairs * chunk / split;
  const int64_t pair_hi = in.npairs * (chunk + 1) / split;
  const int32_t ksteps = (p.k + F_BK - 1) / F_BK;
  const int64_t stages = (pair_hi - pair_lo) * ksteps;

  // A element e = t + 256*j: row t%64 (fixed), k = t/64 + 4*j.
  const int a_r = t & 63, a_k0 = t >> 6;
  int64_t a_off = 0;
  const bool a_ok = row_in_a(p, tc.row0 + a_r, a_off);
  // B element e = t + 256*j: k = t%32 (fixed), column t/32 + 8*j.
  const int b_k = t & 31, b_c0 = t >> 5;
  int64_t b_off[8];
  bool b_ok[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    b_off[j] = 0;
    b_ok[j] = col_in_b(p, tc.col0 + b_c0 + 8 * j, b_off[j]);
  }

  f32x16 acc;
#pragma unroll
  for (int v = 0; v < 16; ++v) acc[v] = 0.0f;
  float ar[8], br[8];
  auto load = [&](int64_t s) {
    const int64_t i = s / ksteps;
    const int32_t kk = (int32_t)(s - i * ksteps) * F_BK;
    const float* pa;
    const float* pb;
    pair_bases<float>(p, in, pair_lo + i, pa, pb);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int32_t ka = kk + a_k0 + 4 * j;
      ar[j] = (a_ok && ka < p.k) ? pa[a_off + (int64_t)ka * p.lda] : 0.0f;
      const int32_t kb = kk + b_k;
      br[j] = (b_ok[j] && kb < p.k) ? pb[b_off[j] + kb] : 0.0f;
    }
  };
  if (stages > 0) load(0);
  for (int64_t s = 0; s < stages; ++s) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      As[(a_k0 + 4 * j) * F_AROW + a_r] = ar[j];
      Bs[(b_c0 + 8 * j) * F_BROW + b_k] = br[j];
    }
    __syncthreads();
    if (s + 1 < stages) load(s + 1);
#pragma unroll
    for (int kq = 0; kq < F_BK / 2; ++kq) {
      const float a = As[(kq * 2 + (lane >> 5)) * F_AROW + wm * 32 + (lane & 31)];
      const float b = Bs[(wn * 32 + (lane & 31)) * F_BROW + kq * 2 + (lane >> 5)];
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc, 0, 0, 0);
    }
    __syncthreads();
  }
  if (split > 1) {
    // raw partial sums: tile-local column-major 64 x 64 block of this (tile, chunk)
    float* w = p.ws + ((size_t)tile_bid * split + chunk) * (F_BM * F_BN);
    const int c_local = wn * 32 + (lane & 31);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r_local = wm * 32 + q * 8 + (lane >> 5) * 4;
      gst<f32x4>(w + c_local * F_BM + r_local,
                 (f32x4){acc[q * 4 + 0], acc[q * 4 + 1], acc[q * 4 + 2], acc[q * 4 + 3]});
    }
    return;
  }
  const int32_t C = tc.col0 + wn * 32 + (lane & 31);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int32_t R0 = tc.row0 + wm * 32 + q * 8 + (lane >> 5) * 4;
    const float v[4] = {acc[q * 4 + 0], acc[q * 4 + 1], acc[q * 4 + 2], acc[q * 4 + 3]};
    store_group<true>(p, in, R0, C, v);
  }
}

// Finishing step of a split fp32 launch: four workgroups per tile, each thread four consecutive
// rows of one column (16 rows x 64 columns per workgroup).  It sums the split partial tiles in
// chunk order (so the result does not depend on timing), eight chunk loads in flight at a time,
// and applies beta * C, bias, activation and the store exactly as the unsplit kernel's epilogue.
__global__ __launch_bounds__(NT) void brgemm_f32_split_finish(BrgemmParams p) {
  const int t = threadIdx.x;
  const int64_t tile_bid = blockIdx.x / 4;
  const int quarter = (int)(blockIdx.x - tile_bid * 4);
  const TileCoord tc = decode_tile_at(p, F_BM, F_BN, tile_bid);
  const Instance in = instance_of(p, tc.g);
  const int c_local = t & 63, r0 = quarter * 16 + (t >> 6) * 4;
  const float* w = p.ws + (size_t)tile_bid * p.split * (F_BM * F_BN) + c_local * F_BM + r0;
  const size_t step = F_BM * F_BN;
  f32x4 sum = {0.0f, 0.0f, 0.0f, 0.0f};
  int32_t ch = 0;
  for (; ch + 8 <= p.split; ch += 8) {
    f32x4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = gld<f32x4>(w + (size_t)(ch + u) * step);
#pragma unroll
    for (int u = 0; u < 8; ++u) sum += v[u];
  }
  for (; ch < p.split; ++ch) sum += gld<f32x4>(w + (size_t)ch * step);
  const float v4[4] = {sum[0], sum[1], sum[2], sum[3]};
  store_group<true>(p, in, tc.row0 + r0, tc.col0 + c_local, v4);
}

// Finishing step of a split direct-LDS launch.  A partial tile holds, for each wave (waves_m x
// waves_n of them, a WTM x WTN tile each) and 32x32 block (tm, tn), every lane's 16 accumulators
// (f32x16, lane-contiguous).  Thread item i = ((wave * TM + tm) * TN + tn) * 256 + lane * 4 + q
// takes the four consecutive rows of MFMA register group q (rows 32 tm + 8 q + 4 (lane / 32) ..
// + 3 and column 32 tn + lane % 32 of the wave tile), so consecutive threads read consecutive 16
// bytes.  It sums them over the chunks in chunk order (the result does not depend on timing) and
// applies beta * C, bias, activation, the aux steps and the store as an unsplit epilogue does.
__global__ __launch_bounds__(NT) void brgemm_dl_split_finish(BrgemmParams p, int32_t bm,
                                                             int32_t bn, int32_t waves_m,
                                                             int32_t waves_n, int32_t per_tile) {
  const int64_t tile_bid = blockIdx.x / per_tile;
  const int32_t item = (int32_t)(blockIdx.x - tile_bid * per_tile) * NT + threadIdx.x;
  const TileCoord tc = decode_tile_at(p, bm, bn, tile_bid);
  const Instance in = instance_of(p, tc.g);
  const int32_t wtm = bm / waves_m, wtn = bn / waves_n;
  const int32_t tms = wtm / 32, tns = wtn / 32;
  const int32_t lane = (item & 255) >> 2, q = item & 3;
  const int32_t rest = item >> 8;
  const int32_t tn = rest % tns, tm = (rest / tns) % tms, wave = rest / (tns * tms);
  const int32_t wm = wave % waves_m, wn = wave / waves_m;
  const float* w = p.ws + (size_t)tile_bid * (bm * bn) + (size_t)item * 4;
  const size_t step = (size_t)p.total_tiles * bm * bn;
  f32x4 sum = {0.0f, 0.0f, 0.0f, 0.0f};
  int32_t ch = 0;
  for (; ch + 4 <= p.split; ch += 4) {
    f32x4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = gld<f32x4>(w + (size_t)(ch + u) * step);
#pragma unroll
    for (int u = 0; u < 4; ++u) sum += v[u];
  }
  for (; ch < p.split; ++ch) sum += gld<f32x4>(w + (size_t)ch * step);
  const float v4[4] = {sum[0], sum[1], sum[2], sum[3]};
  store_group<false>(p, in, tc.row0 + wm * wtm + tm * 32 + 8 * q + 4 * (lane >> 5),
                     tc.col0 + wn * wtn + tn * 32 + (lane & 31), v4);
}

struct KernelInfo {
  const char* name;
  int bm, bn;
  int kstep;   // k must be a multiple of this (direct buffer->LDS stages); 1 = any k
};

constexpr KernelInfo kInfo[K_COUNT] = {
    {"bf16_256x256_w8_vec", 256, 256, 1},
    {"bf16_128x128_w4_vec", 128, 128, 1},
    {"bf16_64x64_w4_vec", 64, 64, 1},
    {"bf16_64x64_generic", 64, 64, 1},
    {"f32_64x64_generic", 64, 64, 1},
    {"bf16_256x256_w8_direct_lds", 256, 256, 32},
    {"bf16_128x128_w4_direct_lds", 128, 128, 32},
    {"bf16_64x64_w4_direct_lds", 64, 64, 32},
    {"bf16_256x256_w8_direct_lds_pingpong", 256, 256, 32},
    {"bf16_256x256_w8_direct_lds_bk64", 256, 256, 64},
    {"bf16_128x128_w4_direct_lds_bk64", 128, 128, 64},
    {"bf16_64x64_w4_direct_lds_bk64", 64, 64, 64},
};

}  // namespace

const char* kernel_name(int32_t id) { return (id >= 0 && id < K_COUNT) ? kInfo[id].name : "?"; }
int kernel_tile_m(int32_t id) { return (id >= 0 && id < K_COUNT) ? kInfo[id].bm : 64; }
int kernel_tile_n(int32_t id) { return (id >= 0 && id < K_COUNT) ? kInfo[id].bn : 64; }
int kernel_k_step(int32_t id) { return (id >= 0 && id < K_COUNT) ? kInfo[id].kstep : 1; }

bool kernel_full(int32_t id, const BrgemmParams& p) {
  const int bm = kernel_tile_m(id), bn = kernel_tile_n(id);
  return (p.k % BK == 0) && (p.vrows % bm == 0) && (p.vcols % bn == 0);
}

namespace {

const char* tf(bool v) { return v ? "true" : "false"; }

template <int BM, int BN, int WM, int WN, bool FULL, int KIND, bool ALIGNED>
void launch_vec_kk(const BrgemmParams& p, dim3 grid, hipStream_t stream, std::string* name_out) {
  if (name_out) {
    char buf[128];
    std::snprintf(buf, sizeof buf, "brgemm_bf16_vec_kernel<%d, %d, %d, %d, %s, %d, %s>", BM, BN,
                  WM, WN, tf(FULL), KIND, tf(ALIGNED));
    *name_out = buf;
    return;
  }
  hipLaunchKernelGGL((brgemm_bf16_vec_kernel<BM, BN, WM, WN, FULL, KIND, ALIGNED>), grid,
                     dim3(64 * WM * WN), 0, stream, p);
}

template <int BM, int BN, int WM, int WN, bool FULL, int KIND>
void launch_vec_k(const BrgemmParams& p, dim3 grid, hipStream_t stream, std::string* name_out) {
  if constexpr (KIND == TPP_BR_STRIDE) {
    if (p.aligned) {
      launch_vec_kk<BM, BN, WM, WN, FULL, KIND, true>(p, grid, stream, name_out);
      return;
    }
  }
  launch_vec_kk<BM, BN, WM, WN, FULL, KIND, false>(p, grid, stream, name_out);
}

template <int BM, int BN, int WM, int WN>
void launch_vec(const BrgemmParams& p, bool full, dim3 grid, hipStream_t stream,
                std::string* name_out) {
  switch (p.kind) {
    case TPP_BR_STRIDE:
      full ? launch_vec_k<BM, BN, WM, WN, true, TPP_BR_STRIDE>(p, grid, stream, name_out)
           : launch_vec_k<BM, BN, WM, WN, false, TPP_BR_STRIDE>(p, grid, stream, name_out);
      break;
    case TPP_BR_OFFSET:
      full ? launch_vec_k<BM, BN, WM, WN, true, TPP_BR_OFFSET>(p, grid, stream, name_out)
           : launch_vec_k<BM, BN, WM, WN, false, TPP_BR_OFFSET>(p, grid, stream, name_out);
      break;
    default:
      full ? launch_vec_k<BM, BN, WM, WN, true, TPP_BR_ADDRESS>(p, grid, stream, name_out)
           : launch_vec_k<BM, BN, WM, WN, false, TPP_BR_ADDRESS>(p, grid, stream, name_out);
      break;
  }
}

}  // namespace

hipError_t launch_brgemm(BrgemmParams& p, int32_t id, hipStream_t stream, std::string* name_out) {
  if (id < 0 || id >= K_COUNT) return hipErrorInvalidValue;
  // transposed operands only on the 64-k direct-to-LDS instances
  if ((p.a_trans || p.b_trans) && id != K_BF16_DL64K_256x256 && id != K_BF16_DL64K_128x128 &&
      id != K_BF16_DL64K_64x64)
    return hipErrorInvalidValue;
  const int bm = kInfo[id].bm, bn = kInfo[id].bn;
  p.tiles_m = (p.vrows + bm - 1) / bm;
  p.tiles_n = (p.vcols + bn - 1) / bn;
  p.total_tiles = p.groups * p.tiles_m * p.tiles_n;
  if (p.total_tiles <= 0) {
    if (name_out) *name_out = "";
    return hipSuccess;
  }
  const dim3 grid((unsigned)p.total_tiles), block(NT);
  const bool full = kernel_full(id, p);
  switch (id) {
    case K_BF16_256x256: launch_vec<256, 256, 2, 4>(p, full, grid, stream, name_out); break;
    case K_BF16_128x128: launch_vec<128, 128, 2, 2>(p, full, grid, stream, name_out); break;
    case K_BF16_64x64: launch_vec<64, 64, 2, 2>(p, full, grid, stream, name_out); break;
    case K_BF16_DL_256x256:
    case K_BF16_DL_128x128:
    case K_BF16_DL_64x64:
    case K_BF16_PP_256x256:
    case K_BF16_DL64K_256x256:
    case K_BF16_DL64K_128x128:
    case K_BF16_DL64K_64x64: {
      if (p.split <= 1) return launch_brgemm_dl(p, id, full, grid, stream, name_out);
      // split over the stage list: chunk partials, then the finishing sum and epilogue
      const hipError_t e = launch_brgemm_dl(p, id, full, dim3((unsigned)(p.total_tiles * p.split)),
                                            stream, name_out);
      if (e != hipSuccess) return e;
      int wm = 0, wn = 0;
      if (!dl_wave_grid(id, wm, wn)) return hipErrorInvalidValue;
      if (name_out) {
        *name_out += " + brgemm_dl_split_finish";
        return hipSuccess;
      }
      const int32_t per_tile = bm * bn / 4 / NT;
      hipLaunchKernelGGL(brgemm_dl_split_finish, dim3((unsigned)(p.total_tiles * per_tile)),
                         block, 0, stream, p, bm, bn, wm, wn, per_tile);
      break;
    }
    case K_BF16_GENERIC:
      if (name_out) {
        *name_out = "brgemm_bf16_kernel<64, 64, 2, 2, true>";
        return hipSuccess;
      }
      hipLaunchKernelGGL((brgemm_bf16_kernel<64, 64, 2, 2, true>), grid, block, 0, stream, p);
      break;
    default:
      if (name_out) {
        *name_out = p.split > 1 ? "brgemm_f32_kernel + brgemm_f32_split_finish"
                                : "brgemm_f32_kernel";
        return hipSuccess;
      }
      if (p.split > 1) {
        hipLaunchKernelGGL(brgemm_f32_kernel, dim3((unsigned)(p.total_tiles * p.split)), block, 0,
                           stream, p);
        hipLaunchKernelGGL(brgemm_f32_split_finish, dim3((unsigned)(p.total_tiles * 4)), block, 0,
                           stream, p);
      } else {
        hipLaunchKernelGGL(brgemm_f32_kernel, grid, block, 0, stream, p);
      }
      break;
  }
  return name_out ? hipSuccess : hipGetLastError();
}

int64_t f32_split_ws_floats(int32_t split, int64_t total_tiles) {
  return (int64_t)split * total_tiles * F_BM * F_BN;
}

}  // namespace tpp
