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
    // m % 4 == 0 and R0 % 4 == 0: the four rows R0..R0+3 are valid together and belong to one
    // instance.
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
// fp32 kernel: 64x64 tile, 4 waves of 32x32, v_mfma_f32_32x32x2f32, stages of 32 k.
//   - VEC (stride kind; m, k, lda, ldb and the grid steps multiples of 4, every pair base 16-byte
//     aligned and every block within 2 GB of its base, all checked on the host per launch): each
//     thread moves two 16-byte vectors of A (4 rows of one k-column) and two of B (4 k of one
//     column) per stage with buffer loads; otherwise element loads.  Out-of-range rows, columns
//     and k read as zero (any shape).
//   - Two LDS buffers (both panels k-major, rows padded against bank conflicts) fed from a ring
//     of four register sets: the global loads of the next four stages are in flight while the
//     MFMAs run on the current buffer; one barrier per stage.
//   - Split launches (few tiles, long pair lists): workgroup b reduces chunk b % split of tile
//     b / split's pair list into a partial tile of the work space, and brgemm_f32_split_finish
//     adds the chunks and applies the epilogue.  (Finishing in the same launch, by the last
//     workgroup of a tile to arrive at a per-tile counter, measured 3.4 us slower per call on
//     the single 64 x 64 instance: the returning device-scope atomic and one workgroup loading
//     every chunk cost more than a second launch queued behind the first.)
// ---------------------------------------------------------------------------------------------
constexpr int F_BM = 64, F_BN = 64, F_BK = 32;
constexpr int F_ROW = F_BM + 4;   // padded k-row of a panel (floats)
constexpr int F_RING = 4;         // stages of global loads in flight (register sets)
// Buffer descriptors of the vector path: F_RANGE bytes addressable from a pair base (the host
// checks that every block fits), offsets at F_OUT_OF_RANGE and beyond read as zero.
constexpr int32_t F_RANGE = 0x7fff0000;
constexpr int32_t F_OUT_OF_RANGE = F_RANGE;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t f32_rsrc(const float* base) {
  // pair bases are uniform over the workgroup: keep the descriptor in scalar registers
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  const uint64_t u = (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)b) |
                     ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(b >> 32)) << 32);
  return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(u), 0, F_RANGE, 0x00020000);
}

template <bool VEC>
__global__ __launch_bounds__(NT) void brgemm_f32_kernel(BrgemmParams p) {
  __shared__ __attribute__((aligned(16))) float As[2][F_BK * F_ROW];
  __shared__ __attribute__((aligned(16))) float Bs[2][F_BK * F_ROW];
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

  // Thread t moves A vectors q = t + 256 j (j < 2): k-column kq = q / 16, rows 4 (q % 16) .. +3;
  // and B vectors q = t + 256 j: column q / 8, k 4 (q % 8) .. +3.
  int64_t a_off[2][4], b_off[2];
  bool a_ok[2][4], b_ok[2];
  int a_k[2], a_r[2], b_c[2], b_k[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int q = t + NT * j;
    a_k[j] = q >> 4;
    a_r[j] = (q & 15) * 4;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      a_off[j][e] = 0;
      a_ok[j][e] = row_in_a(p, tc.row0 + a_r[j] + e, a_off[j][e]);
    }
    b_c[j] = q >> 3;
    b_k[j] = (q & 7) * 4;
    b_off[j] = 0;
    b_ok[j] = col_in_b(p, tc.col0 + b_c[j], b_off[j]);
  }

  f32x16 acc;
#pragma unroll
  for (int v = 0; v < 16; ++v) acc[v] = 0.0f;
  // Ring of F_RING register sets: stage s is loaded into set s % F_RING about F_RING stages
  // before it is written to LDS, so that many stages' global loads are in flight behind the MFMAs
  // (a stage's MFMAs take far less time than a load's round trip to memory).
  f32x4 ra[F_RING][2], rb[F_RING][2];
  // Stages are loaded strictly in order, so a cursor walks them: pair ld_i (pair bases ld_pa /
  // ld_pb), k offset ld_kk; no division per stage.
  int64_t ld_s = 0, ld_i = pair_lo;
  int32_t ld_kk = 0;
  const float* ld_pa = nullptr;
  const float* ld_pb = nullptr;
  if (stages > 0) pair_bases<float>(p, in, ld_i, ld_pa, ld_pb);
  auto advance = [&]() {
    ++ld_s;
    ld_kk += F_BK;
    if (ld_kk >= p.k) {
      ld_kk = 0;
      ++ld_i;
      if constexpr (VEC) {   // stride kind
        ld_pa += p.stride_a;
        ld_pb += p.stride_b;
      } else if (ld_s < stages) {
        pair_bases<float>(p, in, ld_i, ld_pa, ld_pb);
      }
    }
  };
  auto load = [&](auto slot) {
    constexpr int R = decltype(slot)::value;
    if constexpr (VEC) {
      // Exactly four 16-byte buffer loads per call, no branches, so the compiler can count the
      // loads in flight: a vector outside the block (rows past the tile group, k past the end;
      // whole vectors, since m and k are multiples of 4) or of a stage past the chunk's last gets
      // an offset past the descriptor's range and reads as zero.
      const bool live = ld_s < stages;
      const __amdgpu_buffer_rsrc_t sa = f32_rsrc(ld_pa), sb = f32_rsrc(ld_pb);
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int32_t ka = ld_kk + a_k[j];
        const int32_t oa = live && a_ok[j][0] && ka < p.k
                               ? (int32_t)((a_off[j][0] + (int64_t)ka * p.lda) * 4)
                               : F_OUT_OF_RANGE;
        ra[R][j] = __builtin_amdgcn_raw_buffer_load_b128(sa, oa, 0, 0);
        const int32_t kb = ld_kk + b_k[j];
        const int32_t ob =
            live && b_ok[j] && kb < p.k ? (int32_t)((b_off[j] + kb) * 4) : F_OUT_OF_RANGE;
        rb[R][j] = __builtin_amdgcn_raw_buffer_load_b128(sb, ob, 0, 0);
      }
    } else {
      const float* const pa = ld_pa;
      const float* const pb = ld_pb;
      const int32_t kk = ld_kk;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int32_t ka = kk + a_k[j];
        const int32_t kb = kk + b_k[j];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          ra[R][j][e] = (a_ok[j][e] && ka < p.k)
                            ? gld<float>(pa + a_off[j][e] + (int64_t)ka * p.lda)
                            : 0.0f;
          rb[R][j][e] = (b_ok[j] && kb + e < p.k) ? gld<float>(pb + b_off[j] + kb + e) : 0.0f;
        }
      }
    }
    advance();
  };
  auto store = [&](int buf, auto slot) {
    constexpr int R = decltype(slot)::value;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      *reinterpret_cast<f32x4*>(&As[buf][a_k[j] * F_ROW + a_r[j]]) = ra[R][j];
#pragma unroll
      for (int e = 0; e < 4; ++e) Bs[buf][(b_k[j] + e) * F_ROW + b_c[j]] = rb[R][j][e];
    }
  };
  // Prologue: stages 0 .. F_RING - 1 in flight, stage 0 in LDS buffer 0, stage F_RING loading.
  // (The vector path always issues its loads; past the last stage they read zeros.)
  if (stages > 0) {
    load(IntC<0>());
    if (VEC || 1 < stages) load(IntC<1>());
    if (VEC || 2 < stages) load(IntC<2>());
    if (VEC || 3 < stages) load(IntC<3>());
    store(0, IntC<0>());
    if (VEC || F_RING < stages) load(IntC<0>());
    lds_barrier();
  }
  // Iteration s: MFMAs on LDS buffer s & 1 (stage s); stage s + 1 from its register set into the
  // other buffer (free: every wave passed the barrier after stage s - 1's MFMAs); that set then
  // takes stage s + 1 + F_RING.  One barrier per stage.  The slot index (s + 1) % F_RING and the
  // buffer parity are compile-time constants of the unrolled steps.
  int64_t s = 0;
  auto step = [&](auto nslot) {
    constexpr int NS = decltype(nslot)::value;   // (s + 1) % F_RING
    const int buf = (int)(s & 1);
#pragma unroll
    for (int kq = 0; kq < F_BK / 2; ++kq) {
      const int kr = kq * 2 + (lane >> 5);
      const float a = As[buf][kr * F_ROW + wm * 32 + (lane & 31)];
      const float b = Bs[buf][kr * F_ROW + wn * 32 + (lane & 31)];
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc, 0, 0, 0);
    }
    if (s + 1 < stages) store(buf ^ 1, IntC<NS>());
    if (VEC || s + 1 + F_RING < stages) load(IntC<NS>());
    lds_barrier();   // LDS traffic only: the ring's global loads stay in flight
    ++s;
  };
  while (s < stages) {
    step(IntC<1>());
    if (s >= stages) break;
    step(IntC<2>());
    if (s >= stages) break;
    step(IntC<3>());
    if (s >= stages) break;
    step(IntC<0>());
  }

  if (split > 1) {
    // This chunk's partial tile, the accumulators in register order: thread t's group q at float
    // ((wave * 4 + q) * 64 + lane) * 4 of the chunk's 64 x 64 block, so each wave-wide 16-byte
    // store covers 1 KB of consecutive bytes.
    float* const w = p.ws + ((size_t)tile_bid * split + chunk) * (F_BM * F_BN) +
                     ((wave * 4) * 64 + lane) * 4;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      gst<f32x4>(w + q * 256,
                 (f32x4){acc[q * 4 + 0], acc[q * 4 + 1], acc[q * 4 + 2], acc[q * 4 + 3]});
    return;
  }
  // Four consecutive rows per group: with m a multiple of 4 (the vector instance) they are valid
  // together and lie in one instance, and the group is one 16-byte store when aligned.
  const int32_t C = tc.col0 + wn * 32 + (lane & 31);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int32_t R0 = tc.row0 + wm * 32 + q * 8 + (lane >> 5) * 4;
    const float v[4] = {acc[q * 4 + 0], acc[q * 4 + 1], acc[q * 4 + 2], acc[q * 4 + 3]};
    store_group<!VEC>(p, in, R0, C, v);
  }
}

// Finishing step of a split fp32 launch: four workgroups per tile, thread f of a tile's 1024
// taking the partial tiles' 16-byte group f (wave f / 256, register group (f / 64) % 4, lane
// f % 64 of the main kernel: four consecutive rows of one column).  It sums the chunks in chunk
// order (the result does not depend on timing), eight loads in flight at a time, and applies
// beta * C, bias, activation and the store exactly as the unsplit kernel's epilogue.
__global__ __launch_bounds__(NT) void brgemm_f32_split_finish(BrgemmParams p) {
  const int64_t tile_bid = blockIdx.x / 4;
  const int f = (int)(blockIdx.x - tile_bid * 4) * NT + threadIdx.x;
  const int wave = f >> 8, q = (f >> 6) & 3, lane = f & 63;
  const int wm = wave & 1, wn = wave >> 1;
  const TileCoord tc = decode_tile_at(p, F_BM, F_BN, tile_bid);
  const Instance in = instance_of(p, tc.g);
  const float* w = p.ws + (size_t)tile_bid * p.split * (F_BM * F_BN) + f * 4;
  f32x4 sum = {0.0f, 0.0f, 0.0f, 0.0f};
  int32_t ch = 0;
  for (; ch + 8 <= p.split; ch += 8) {
    f32x4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = gld<f32x4>(w + (size_t)(ch + u) * (F_BM * F_BN));
#pragma unroll
    for (int u = 0; u < 8; ++u) sum += v[u];
  }
  for (; ch < p.split; ++ch) sum += gld<f32x4>(w + (size_t)ch * (F_BM * F_BN));
  const int32_t C = tc.col0 + wn * 32 + (lane & 31);
  const int32_t R0 = tc.row0 + wm * 32 + q * 8 + (lane >> 5) * 4;
  const float v[4] = {sum[0], sum[1], sum[2], sum[3]};
  if (p.m % 4 == 0)
    store_group<false>(p, in, R0, C, v);
  else
    store_group<true>(p, in, R0, C, v);
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
    default: {
      // 16-byte buffer loads when every k-column of A and every k-run of B splits into whole
      // aligned vectors (stride kind: all pair bases follow from the bases and the steps) and every
      // block lies within the descriptor's range of its pair base
      const auto fits = [](int64_t last) { return last >= 0 && (last + 4) * 4 <= F_RANGE; };
      const int64_t a_last = (p.fused ? (p.gm - 1) * p.a_step_m : 0) + p.m - 4 +
                             (int64_t)(p.k - 1) * p.lda;
      const int64_t b_last = (p.fused ? (p.gn - 1) * p.b_step_n : 0) +
                             (int64_t)(p.n - 1) * p.ldb + p.k - 4;
      const bool vec = p.kind == TPP_BR_STRIDE && p.aligned && p.m % 4 == 0 && p.k % 4 == 0 &&
                       p.lda % 4 == 0 && p.ldb % 4 == 0 &&
                       (!p.fused || (p.a_step_m % 4 == 0 && p.b_step_n % 4 == 0 &&
                                     p.a_step_m >= 0 && p.b_step_n >= 0)) &&
                       fits(a_last) && fits(b_last);
      if (name_out) {
        *name_out = vec ? "brgemm_f32_kernel<true>" : "brgemm_f32_kernel<false>";
        if (p.split > 1) *name_out += " + brgemm_f32_split_finish";
        return hipSuccess;
      }
      const dim3 g = p.split > 1 ? dim3((unsigned)(p.total_tiles * p.split)) : grid;
      if (vec)
        hipLaunchKernelGGL(brgemm_f32_kernel<true>, g, block, 0, stream, p);
      else
        hipLaunchKernelGGL(brgemm_f32_kernel<false>, g, block, 0, stream, p);
      if (p.split > 1)
        hipLaunchKernelGGL(brgemm_f32_split_finish, dim3((unsigned)(p.total_tiles * 4)), block, 0,
                           stream, p);
      break;
    }
  }
  return name_out ? hipSuccess : hipGetLastError();
}

int64_t f32_split_ws_floats(int32_t split, int64_t total_tiles) {
  return (int64_t)split * total_tiles * F_BM * F_BN;
}

}  // namespace tpp
