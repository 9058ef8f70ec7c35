// brgemm_device.h -- device-side pieces shared by the BRGEMM kernel files: vector types, global
// accesses, the epilogue arithmetic, tile / instance decoding, the Sec. 2.3 pair addresses and the
// LDS-staged epilogue.
#pragma once

#include <hip/hip_runtime.h>

#include "internal.h"

namespace tpp {
namespace dev {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Global-memory accesses through address-space-1 pointers, so that they compile to global_*
// instructions.  (Through generic pointers they become flat_* instructions, which also count
// against the LDS wait counter: every wait for an LDS operand would then wait for the global
// prefetch as well.)
#define GLOBAL_AS __attribute__((address_space(1)))
template <typename T>
__device__ __forceinline__ T gld(const void* p) {
  return *(const GLOBAL_AS T*)p;
}
template <typename T>
__device__ __forceinline__ void gst(void* p, T v) {
  *(GLOBAL_AS T*)p = v;
}

template <int V>
struct IntC {
  static constexpr int value = V;
};

constexpr int NT = 256;            // threads per workgroup: 4 wavefronts of 64
constexpr int BK = 64;             // k extent of one stage (bf16)
constexpr int LDS_ROW = BK + 8;    // bf16 per LDS row: 128 B of data + 16 B against bank conflicts

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  // Lowers to v_cvt_pk_bf16_f32 on gfx950: round to nearest even, NaN stays NaN.
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
// Two floats narrowed together (one v_cvt_pk_bf16_f32, round to nearest even): lo in bits 15:0.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t));
}

// GELU in its tanh form, 0.5 x (1 + tanh(u)) with u = sqrt(2/pi) (x + 0.044715 x^3).
// Since 0.5 (1 + tanh(u)) = 1 / (1 + e^(-2u)), this is x / (1 + 2^(-2u log2(e))): one hardware
// exp2 (v_exp_f32) and one hardware reciprocal (v_rcp_f32), a few ulp of fp32 in all, and no
// cancellation anywhere (for u -> -inf the denominator goes to +inf and the result to -0).
// The exponent -2u log2(e) = x (k1 + k2 x^2) has its constants folded: 5 VALU operations and two
// transcendental ones per element.
__device__ __forceinline__ float gelu_tanh(float x) {
  const float k1 = -2.3022082f;    // -2 log2(e) sqrt(2/pi)
  const float k2 = -0.10294324f;   // k1 * 0.044715
  const float e = __builtin_amdgcn_exp2f(x * __builtin_fmaf(k2, x * x, k1));
  return x * __builtin_amdgcn_rcpf(1.0f + e);
}

__device__ __forceinline__ float activate(float v, uint32_t flags) {
  if (flags & TPP_EPI_RELU) return v > 0.0f ? v : 0.0f;
  if (flags & TPP_EPI_GELU_TANH) return gelu_tanh(v);
  return v;
}

// Derivative of gelu_tanh, for GELU_inv (Table 1).  With s = 0.5 (1 + tanh u) = 1 / (1 + e^(-2u))
// the GELU is x s, so its derivative is s + 2 x s (1 - s) u', where 1 - s = e^(-2u) s (no
// cancellation) and u' = sqrt(2/pi) (1 + 3 * 0.044715 x^2).  The argument is clamped to [-9, 9]:
// beyond it the derivative is 0 or 1 to within 3e-27, and the clamp keeps e^(-2u) finite and s a
// normal number, so no inf * 0 arises.
__device__ __forceinline__ float gelu_tanh_grad(float z) {
  const float x = fminf(fmaxf(z, -9.0f), 9.0f);
  const float k1 = -2.3022082f;    // -2 log2(e) sqrt(2/pi), as in gelu_tanh
  const float k2 = -0.10294324f;   // k1 * 0.044715
  const float e = __builtin_amdgcn_exp2f(x * __builtin_fmaf(k2, x * x, k1));   // e^(-2u)
  const float s = __builtin_amdgcn_rcpf(1.0f + e);
  const float c2 = 1.5957691f;     // 2 sqrt(2/pi)
  return s * __builtin_fmaf(c2 * x * (e * s), __builtin_fmaf(0.134145f, x * x, 1.0f), 1.0f);
}

// The aux tensor of the back-propagation epilogue bits has C's type and layout: N consecutive
// rows of one column start at element e0, exactly where C's do.
template <int N>
__device__ __forceinline__ void aux_load(const BrgemmParams& p, int64_t e0, float (&z)[N]) {
  if (p.c_bf16) {
    const uint16_t* ap = static_cast<const uint16_t*>(p.aux) + e0;
    if constexpr (N == 4) {
      if ((reinterpret_cast<uintptr_t>(ap) & 7) == 0) {
        const u32x2 w = gld<u32x2>(ap);
        z[0] = bf16_bits_to_f32(w[0] & 0xffffu);
        z[1] = bf16_bits_to_f32(w[0] >> 16);
        z[2] = bf16_bits_to_f32(w[1] & 0xffffu);
        z[3] = bf16_bits_to_f32(w[1] >> 16);
        return;
      }
    }
    if constexpr (N == 8) {
      if ((reinterpret_cast<uintptr_t>(ap) & 15) == 0) {
        const u32x4 w = gld<u32x4>(ap);
        const uint32_t d[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          z[2 * e] = bf16_bits_to_f32(d[e] & 0xffffu);
          z[2 * e + 1] = bf16_bits_to_f32(d[e] >> 16);
        }
        return;
      }
    }
#pragma unroll
    for (int e = 0; e < N; ++e) z[e] = bf16_bits_to_f32(gld<uint16_t>(ap + e));
  } else {
    const float* ap = static_cast<const float*>(p.aux) + e0;
    if constexpr (N % 4 == 0) {
      if ((reinterpret_cast<uintptr_t>(ap) & 15) == 0) {
#pragma unroll
        for (int q = 0; q < N / 4; ++q) {
          const f32x4 w = gld<f32x4>(ap + 4 * q);
#pragma unroll
          for (int e = 0; e < 4; ++e) z[4 * q + e] = w[e];
        }
        return;
      }
    }
#pragma unroll
    for (int e = 0; e < N; ++e) z[e] = gld<float>(ap + e);
  }
}

template <int N>
__device__ __forceinline__ void aux_store(const BrgemmParams& p, int64_t e0, const float (&v)[N]) {
  if (p.c_bf16) {
    uint16_t* ap = static_cast<uint16_t*>(p.aux) + e0;
    if constexpr (N == 4) {
      if ((reinterpret_cast<uintptr_t>(ap) & 7) == 0) {
        gst<u32x2>(ap, (u32x2){pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])});
        return;
      }
    }
    if constexpr (N == 8) {
      if ((reinterpret_cast<uintptr_t>(ap) & 15) == 0) {
        gst<u32x4>(ap, (u32x4){pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                               pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7])});
        return;
      }
    }
#pragma unroll
    for (int e = 0; e < N; ++e) gst<uint16_t>(ap + e, f32_to_bf16_bits(v[e]));
  } else {
    float* ap = static_cast<float*>(p.aux) + e0;
    if constexpr (N % 4 == 0) {
      if ((reinterpret_cast<uintptr_t>(ap) & 15) == 0) {
#pragma unroll
        for (int q = 0; q < N / 4; ++q)
          gst<f32x4>(ap + 4 * q, (f32x4){v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]});
        return;
      }
    }
#pragma unroll
    for (int e = 0; e < N; ++e) gst<float>(ap + e, v[e]);
  }
}

// The aux steps of the epilogue on N consecutive rows of one column (element e0 of C's layout),
// after beta*C and the bias: SAVE_PREACT keeps v (rounded to C's type) before the activation;
// RELU_INV / GELU_TANH_INV, which never come with an activation, multiply v by the activation's
// derivative at the saved pre-activation z.  activate() then runs on the result as usual.
template <int N>
__device__ __forceinline__ void epi_aux(const BrgemmParams& p, int64_t e0, float (&v)[N]) {
  if (p.flags & TPP_EPI_SAVE_PREACT) aux_store<N>(p, e0, v);
  if (p.flags & (TPP_EPI_RELU_INV | TPP_EPI_GELU_TANH_INV)) {
    float z[N];
    aux_load<N>(p, e0, z);
    if (p.flags & TPP_EPI_RELU_INV) {
#pragma unroll
      for (int e = 0; e < N; ++e) v[e] = z[e] > 0.0f ? v[e] : 0.0f;
    } else {
#pragma unroll
      for (int e = 0; e < N; ++e) v[e] = v[e] * gelu_tanh_grad(z[e]);
    }
  }
}

// XCD-aware tile order: workgroups are handed to the 8 XCDs round-robin, so consecutive block
// ids land on different L2s.  Remapping gives each XCD a contiguous run of tiles (neighbouring
// tiles share A rows or B columns and so share that XCD's L2).
__device__ __forceinline__ int64_t xcd_tile(int64_t bid, int64_t total) {
  if ((total & 7) != 0) return bid;
  return (bid & 7) * (total >> 3) + (bid >> 3);
}

struct TileCoord {
  int64_t g;        // instance (explicit form) or 0 (strided form)
  int32_t row0;     // first virtual row of the tile
  int32_t col0;     // first virtual column of the tile
};

__device__ __forceinline__ TileCoord decode_tile_at(const BrgemmParams& p, int bm, int bn,
                                                   int64_t bid) {
  const int64_t t = xcd_tile(bid, p.total_tiles);
  const int64_t per_group = (int64_t)p.tiles_m * p.tiles_n;
  TileCoord tc;
  tc.g = t / per_group;
  const int64_t tin = t - tc.g * per_group;
  // Bands of up to 8 tile rows: consecutive tiles walk down a band, then move one tile column
  // right, so the 32 tiles an XCD runs at once cover about 8 rows x 4 columns and share both
  // their A rows and their B columns in that XCD's L2.
  const int32_t band = p.tiles_m < 8 ? p.tiles_m : 8;
  const int64_t per_band = (int64_t)band * p.tiles_n;
  const int32_t b0 = (int32_t)(tin / per_band) * band;
  const int32_t bh = (p.tiles_m - b0) < band ? (p.tiles_m - b0) : band;
  const int64_t tb = tin - (int64_t)b0 * p.tiles_n;
  tc.row0 = (b0 + (int32_t)(tb % bh)) * bm;
  tc.col0 = (int32_t)(tb / bh) * bn;
  return tc;
}

__device__ __forceinline__ TileCoord decode_tile(const BrgemmParams& p, int bm, int bn) {
  return decode_tile_at(p, bm, bn, blockIdx.x);
}

// Virtual row R -> element offset of that row inside A (relative to the instance's A base) and
// whether it exists.  Fused strided grid: R = gi_m * m + r.  One instance per group: R = r.
__device__ __forceinline__ bool row_in_a(const BrgemmParams& p, int32_t R, int64_t& off) {
  if (p.fused) {
    if (R >= p.vrows) return false;
    const int32_t gi = R / p.m, r = R - gi * p.m;
    off = (int64_t)gi * p.a_step_m + r;
    return true;
  }
  off = R;
  return R < p.m;
}

// The same for a transposed A (row r's k-run starts at r * lda).
__device__ __forceinline__ bool row_in_at(const BrgemmParams& p, int32_t R, int64_t& off) {
  if (p.fused) {
    if (R >= p.vrows) return false;
    const int32_t gi = R / p.m, r = R - gi * p.m;
    off = (int64_t)gi * p.a_step_m + (int64_t)r * p.lda;
    return true;
  }
  off = (int64_t)R * p.lda;
  return R < p.m;
}

// The same for a transposed B: element offset of column C in k-row 0 (columns are contiguous).
__device__ __forceinline__ bool col_in_bt(const BrgemmParams& p, int32_t C, int64_t& off) {
  if (p.fused) {
    if (C >= p.vcols) return false;
    const int32_t gi = C / p.n, c = C - gi * p.n;
    off = (int64_t)gi * p.b_step_n + c;
    return true;
  }
  off = C;
  return C < p.n;
}

// Virtual column C -> element offset of that column inside B (relative to the instance base).
__device__ __forceinline__ bool col_in_b(const BrgemmParams& p, int32_t C, int64_t& off) {
  if (p.fused) {
    if (C >= p.vcols) return false;
    const int32_t gi = C / p.n, c = C - gi * p.n;
    off = (int64_t)gi * p.b_step_n + (int64_t)c * p.ldb;
    return true;
  }
  off = (int64_t)C * p.ldb;
  return C < p.n;
}

// Per-launch instance data for tile group g: bases added to every A_i / B_i / C / bias address,
// and the pair list.
struct Instance {
  int64_t a, b, c, bias;   // element offsets
  int64_t pair0, npairs;
};

__device__ __forceinline__ Instance instance_of(const BrgemmParams& p, int64_t g) {
  Instance in;
  in.a = in.b = in.c = in.bias = 0;
  if (!p.fused && p.grid_form) {
    const int64_t gi_m = g % p.gm, gi_n = g / p.gm;
    in.a = gi_m * p.a_step_m;
    in.b = gi_n * p.b_step_n;
    in.c = gi_m * p.c_step_m + gi_n * p.c_step_n;
    in.bias = gi_m * p.bias_step_m;
  } else if (!p.fused) {
    in.a = p.a_off ? p.a_off[g] : 0;
    in.b = p.b_off ? p.b_off[g] : 0;
    in.c = p.c_off ? p.c_off[g] : 0;
    in.bias = p.bias_off ? p.bias_off[g] : 0;
  }
  in.pair0 = 0;
  in.npairs = p.count;
  if (p.kind == TPP_BR_ADDRESS && p.begin) {   // a single address call has no begin[]
    in.pair0 = p.begin[g];
    in.npairs = p.begin[g + 1] - in.pair0;
  }
  return in;
}

// Addresses of pair i (Sec. 2.3): stride A + i*stride, offset A + offs[i], address ptrs[i].
template <typename T>
__device__ __forceinline__ void pair_bases(const BrgemmParams& p, const Instance& in, int64_t i,
                                           const T*& pa, const T*& pb) {
  if (p.kind == TPP_BR_STRIDE) {
    pa = static_cast<const T*>(p.a) + in.a + i * p.stride_a;
    pb = static_cast<const T*>(p.b) + in.b + i * p.stride_b;
  } else if (p.kind == TPP_BR_OFFSET) {
    pa = static_cast<const T*>(p.a) + in.a + p.offs_a[i];
    pb = static_cast<const T*>(p.b) + in.b + p.offs_b[i];
  } else {
    pa = static_cast<const T*>(p.ptrs_a[in.pair0 + i]);
    pb = static_cast<const T*>(p.ptrs_b[in.pair0 + i]);
  }
}

// The same, with the variant fixed at compile time (no per-stage branch on the kind).
template <int KIND, typename T>
__device__ __forceinline__ void pair_bases_k(const BrgemmParams& p, const Instance& in, int64_t i,
                                             const T*& pa, const T*& pb) {
  if constexpr (KIND == TPP_BR_STRIDE) {
    pa = static_cast<const T*>(p.a) + in.a + i * p.stride_a;
    pb = static_cast<const T*>(p.b) + in.b + i * p.stride_b;
  } else if constexpr (KIND == TPP_BR_OFFSET) {
    pa = static_cast<const T*>(p.a) + in.a + p.offs_a[i];
    pb = static_cast<const T*>(p.b) + in.b + p.offs_b[i];
  } else {
    pa = static_cast<const T*>(p.ptrs_a[in.pair0 + i]);
    pb = static_cast<const T*>(p.ptrs_b[in.pair0 + i]);
  }
}

// Workgroup barrier that first waits for this wave's own LDS operations only.  __syncthreads()
// also waits for every outstanding global load (vmcnt 0), which would drain direct-to-LDS loads of
// later pipeline stages at each barrier; kernels that keep such loads in flight wait for the ones
// they need with an explicit s_waitcnt vmcnt before calling this.  The memory clobber keeps the
// compiler from moving LDS accesses across the barrier.
// The scheduling barriers keep register-only work (MFMAs) on its side of it as well.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// Direct global -> LDS copies (used by the direct-to-LDS main loops and by the epilogue's aux
// loads).
#define LDS_AS __attribute__((address_space(3)))

// s_waitcnt immediate waiting until at most n vector-memory operations are outstanding (gfx9
// encoding: vmcnt in bits 3:0 and 15:14, expcnt 6:4 and lgkmcnt 11:8 left at their maxima).
constexpr int vmcnt_imm(int n) {
  return (n & 0xF) | (((n >> 4) & 3) << 14) | (0x7 << 4) | (0xF << 8);
}

// Buffer descriptor of a raw (unswizzled, stride 0) buffer at `base`: 2^31 bytes addressable,
// out-of-range offsets read as zero.  Built from wave-uniform values, so it lives in SGPRs.
typedef int i32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ i32x4 raw_buffer(const void* base) {
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  return (i32x4){__builtin_amdgcn_readfirstlane((int)(uint32_t)b),
                 __builtin_amdgcn_readfirstlane((int)((uint32_t)(b >> 32) & 0xffffu)), 0x7fffffff,
                 0x00020000};
}

// 16-byte buffer -> LDS copy of a whole wave (buffer_load_dwordx4 ... offen lds): lane j's 16
// bytes from rsrc base + voff land at l + 16 j.  The buffer form takes one 32-bit offset per lane
// where the global form takes a 64-bit address, and unlike the global form it runs alongside the
// MFMAs of the same compute unit instead of stalling them (measured on gfx950: a stream of 32x32x16
// MFMAs beside 8 KB of loads per iteration took the MFMA time with buffer loads, the sum of both
// times with global loads).  It is issued through inline asm so that the compiler does not see a
// pending LDS write: the compiler would otherwise wait for every outstanding load (vmcnt 0)
// before the next LDS read and so drain the stages kept in flight.  Callers order these loads
// themselves with s_waitcnt vmcnt and lds_barrier().  M0 is saved and restored around it.
__device__ __forceinline__ void buffer_load_lds16(i32x4 rsrc, uint32_t voff, char* l) {
  const uint32_t lds_addr =
      __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(LDS_AS char*)l);
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %3\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %1, %2, 0 offen lds\n\t"
      "s_nop 0\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(voff), "s"(rsrc), "s"(lds_addr)
      : "memory");
}

// N consecutive 16-byte buffer -> LDS wave-loads: load r reads rsrc base + voff[r] and lands at
// lds_addr + 1024 r.  One asm block sets M0 once and steps it by 1 KB between the loads, so a
// wave-load costs two scalar instructions instead of the nine of a separate buffer_load_lds16
// (M0 save, set, wait state, restore, and the null check of the LDS pointer's address-space
// conversion).  The scalar unit is shared by the compute unit's waves, and every wave copies its
// share of a stage right after the same barrier: measured per wave and stage, issuing the copies
// of the 256 x 256 tile took ~980 cycles one by one and ~845 in blocks, of the 128 x 128 tile 758
// and 587.  (The rest is the copies themselves: each direct-to-LDS load takes ~100 cycles to
// issue while all waves copy.)  One wait state after each M0 write, as the ISA requires before an
// LDS-DMA load.
#define TPP_LDS16_FIRST "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %[lds]\n\ts_nop 0\n\t"
#define TPP_LDS16_LOAD(i) "buffer_load_dwordx4 %[v" #i "], %[rsrc], 0 offen lds\n\t"
#define TPP_LDS16_STEP "s_add_u32 m0, m0, 0x400\n\ts_nop 0\n\t"
#define TPP_LDS16_LAST "s_nop 0\n\ts_mov_b32 m0, %0"
template <int N>
__device__ __forceinline__ void buffer_load_lds16_block(i32x4 rsrc, const uint32_t* voff,
                                                        uint32_t lds_addr) {
  uint32_t saved;
  if constexpr (N == 1) {
    asm volatile(TPP_LDS16_FIRST TPP_LDS16_LOAD(0) TPP_LDS16_LAST
                 : "=&s"(saved)
                 : [v0] "v"(voff[0]), [rsrc] "s"(rsrc), [lds] "s"(lds_addr)
                 : "memory", "scc");
  } else if constexpr (N == 2) {
    asm volatile(TPP_LDS16_FIRST TPP_LDS16_LOAD(0) TPP_LDS16_STEP TPP_LDS16_LOAD(1) TPP_LDS16_LAST
                 : "=&s"(saved)
                 : [v0] "v"(voff[0]), [v1] "v"(voff[1]), [rsrc] "s"(rsrc), [lds] "s"(lds_addr)
                 : "memory", "scc");
  } else if constexpr (N == 4) {
    asm volatile(TPP_LDS16_FIRST TPP_LDS16_LOAD(0) TPP_LDS16_STEP TPP_LDS16_LOAD(1)
                     TPP_LDS16_STEP TPP_LDS16_LOAD(2) TPP_LDS16_STEP TPP_LDS16_LOAD(3)
                         TPP_LDS16_LAST
                 : "=&s"(saved)
                 : [v0] "v"(voff[0]), [v1] "v"(voff[1]), [v2] "v"(voff[2]), [v3] "v"(voff[3]),
                   [rsrc] "s"(rsrc), [lds] "s"(lds_addr)
                 : "memory", "scc");
  } else if constexpr (N == 8) {
    asm volatile(TPP_LDS16_FIRST TPP_LDS16_LOAD(0) TPP_LDS16_STEP TPP_LDS16_LOAD(1)
                     TPP_LDS16_STEP TPP_LDS16_LOAD(2) TPP_LDS16_STEP TPP_LDS16_LOAD(3)
                         TPP_LDS16_STEP TPP_LDS16_LOAD(4) TPP_LDS16_STEP TPP_LDS16_LOAD(5)
                             TPP_LDS16_STEP TPP_LDS16_LOAD(6) TPP_LDS16_STEP TPP_LDS16_LOAD(7)
                                 TPP_LDS16_LAST
                 : "=&s"(saved)
                 : [v0] "v"(voff[0]), [v1] "v"(voff[1]), [v2] "v"(voff[2]), [v3] "v"(voff[3]),
                   [v4] "v"(voff[4]), [v5] "v"(voff[5]), [v6] "v"(voff[6]), [v7] "v"(voff[7]),
                   [rsrc] "s"(rsrc), [lds] "s"(lds_addr)
                 : "memory", "scc");
  } else {
    static_assert(N == 1 || N == 2 || N == 4 || N == 8, "block sizes 1, 2, 4, 8");
  }
}
#undef TPP_LDS16_FIRST
#undef TPP_LDS16_LOAD
#undef TPP_LDS16_STEP
#undef TPP_LDS16_LAST

// 16 bytes of bf16 from global memory, aligned or not; zeroing without branches.
__device__ __forceinline__ u32x4 ld16(const uint16_t* ptr) { return gld<u32x4>(ptr); }

__device__ __forceinline__ u32x4 ld16_unaligned(const uint16_t* ptr) {
  uint32_t h[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) h[e] = gld<uint16_t>(ptr + e);
  return (u32x4){h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16),
                 h[6] | (h[7] << 16)};
}

__device__ __forceinline__ u32x4 keep_if(u32x4 v, bool ok) {
  return (u32x4){ok ? v.x : 0u, ok ? v.y : 0u, ok ? v.z : 0u, ok ? v.w : 0u};
}

// ---------------------------------------------------------------------------------------------
// Epilogue of the 16-byte-load kernels, through LDS.  Each wave parks one 32-column slab of its
// accumulators (WTM rows x 32 columns, fp32) in its own LDS region, then every lane takes 8
// consecutive rows of one column: beta*C, bias, activation and narrowing on 8 values, one 16-byte
// store.  The caller has passed a barrier after the last LDS read of the main loop.
// The accumulator layout of a 32x32 MFMA tile: lane l holds column l%32, and in register v the
// row 8*(v/4) + 4*(l/32) + v%4.
// ---------------------------------------------------------------------------------------------
template <int WTM, int WTN, int TM, int TN, bool FULL>
__device__ __forceinline__ void epilogue_via_lds(const BrgemmParams& p, const Instance& in,
                                                 const TileCoord& tc, int wm, int wn, int lane,
                                                 int wave, float* lds_f, f32x16 (&acc)[TM][TN]) {
  constexpr int EP_ROW = WTM + 4;                    // slab: 32 columns x WTM rows fp32
  constexpr int CPC = WTM / 8;                       // 8-row chunks per slab column
  constexpr int EP_ITERS = 32 * CPC / 64;
  static_assert(64 % CPC == 0, "row chunks per column divide the wavefront");
  float* slab = lds_f + wave * 32 * EP_ROW;
  const int my_chunk = lane % CPC;
  const int32_t R = tc.row0 + wm * WTM + my_chunk * 8;
  bool row_ok = true;
  int64_t row_off, bias_idx;
  if (p.fused) {
    const int32_t gi = R / p.m, r = R - gi * p.m;
    row_ok = FULL || R < p.vrows;
    row_off = (int64_t)gi * p.c_step_m + r;
    bias_idx = (int64_t)gi * p.bias_step_m + r;
  } else {
    row_ok = FULL || R < p.m;
    row_off = R;
    bias_idx = in.bias + R;
  }
  float bias8[8];
  const bool has_bias = (p.flags & TPP_EPI_BIAS) != 0;
#pragma unroll
  for (int e = 0; e < 8; ++e)
    bias8[e] = (has_bias && row_ok) ? gld<float>(p.bias + bias_idx + e) : 0.0f;

#pragma unroll
  for (int tn = 0; tn < TN; ++tn) {
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float4 w = make_float4(acc[tm][tn][q * 4 + 0], acc[tm][tn][q * 4 + 1],
                               acc[tm][tn][q * 4 + 2], acc[tm][tn][q * 4 + 3]);
        *reinterpret_cast<float4*>(slab + (lane & 31) * EP_ROW + tm * 32 + q * 8 +
                                   (lane >> 5) * 4) = w;
      }
    __syncthreads();
    // kept rolled: the accumulators are not indexed here, and unrolling the activation code
    // would only grow the kernel
#pragma unroll 1
    for (int it = 0; it < EP_ITERS; ++it) {
      const int col_local = it * (64 / CPC) + lane / CPC;
      const float4 lo = *reinterpret_cast<const float4*>(slab + col_local * EP_ROW + my_chunk * 8);
      const float4 hi =
          *reinterpret_cast<const float4*>(slab + col_local * EP_ROW + my_chunk * 8 + 4);
      const int32_t C = tc.col0 + wn * WTN + tn * 32 + col_local;
      int64_t col_off;
      bool col_ok;
      if (p.fused) {
        const int32_t gi = C / p.n, c = C - gi * p.n;
        col_ok = FULL || C < p.vcols;
        col_off = (int64_t)gi * p.c_step_n + (int64_t)c * p.ldc;
      } else {
        col_ok = FULL || C < p.n;
        col_off = (int64_t)C * p.ldc;
      }
      if (row_ok && col_ok) {
        float v[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
        const int64_t e0 = in.c + row_off + col_off;
        if (p.c_bf16) {
          uint16_t* cp = static_cast<uint16_t*>(p.c) + e0;
          const bool vec = (reinterpret_cast<uintptr_t>(cp) & 15) == 0;
          if (p.beta != 0.0f) {
            const u32x4 w = vec ? ld16(cp) : ld16_unaligned(cp);
            const uint32_t d[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              v[2 * e] = p.beta * bf16_bits_to_f32(d[e] & 0xffffu) + v[2 * e];
              v[2 * e + 1] = p.beta * bf16_bits_to_f32(d[e] >> 16) + v[2 * e + 1];
            }
          }
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] += bias8[e];
          if (p.flags & EPI_AUX_MASK) epi_aux<8>(p, e0, v);
          uint32_t o[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) o[e] = f32_to_bf16_bits(activate(v[e], p.flags));
          if (vec) {
            gst<u32x4>(cp, (u32x4){o[0] | (o[1] << 16), o[2] | (o[3] << 16),
                                   o[4] | (o[5] << 16), o[6] | (o[7] << 16)});
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) gst<uint16_t>(cp + e, (uint16_t)o[e]);
          }
        } else {
          float* cp = static_cast<float*>(p.c) + e0;
          const bool vec = (reinterpret_cast<uintptr_t>(cp) & 15) == 0;
          if (p.beta != 0.0f) {
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = p.beta * gld<float>(cp + e) + v[e];
          }
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] += bias8[e];
          if (p.flags & EPI_AUX_MASK) epi_aux<8>(p, e0, v);
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] = activate(v[e], p.flags);
          if (vec) {
            gst<f32x4>(cp, (f32x4){v[0], v[1], v[2], v[3]});
            gst<f32x4>(cp + 4, (f32x4){v[4], v[5], v[6], v[7]});
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) gst<float>(cp + e, v[e]);
          }
        }
      }
    }
    __syncthreads();
  }
}

// Bias of a lane's rows in the 32x32 MFMA accumulator layout, all issued before any is used: for
// group tm and q, the four rows row_base + 32 tm + 8 q + 4 (lane / 32) + e (an 8-row chunk never
// straddles an instance: m % 8 == 0).  The chunks are 8 rows apart, so the instance row and bias
// index advance by additions.  Rows outside C, and every row without TPP_EPI_BIAS, get zeros.
template <int TM, bool FULL>
__device__ __forceinline__ void load_bias4(const BrgemmParams& p, const Instance& in,
                                           int32_t row_base, int lane, f32x4 (&bias4)[TM][4]) {
  const bool has_bias = (p.flags & TPP_EPI_BIAS) != 0;
  const int half = lane >> 5;
  const int32_t R0 = row_base + 4 * half;
  int32_t gi = 0, r = R0;
  if (p.fused) {
    gi = R0 / p.m;
    r = R0 - gi * p.m;
  }
  int64_t idx = p.fused ? (int64_t)gi * p.bias_step_m + r : in.bias + R0;
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int32_t R = R0 + tm * 32 + 8 * q;
      const bool ok = FULL || R < (p.fused ? p.vrows : p.m);
      f32x4 b = {0.0f, 0.0f, 0.0f, 0.0f};
      if (has_bias && ok) {
        const float* bp = p.bias + idx;
        if ((reinterpret_cast<uintptr_t>(bp) & 15) == 0) {
          b = gld<f32x4>(bp);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) b[e] = gld<float>(bp + e);
        }
      }
      bias4[tm][q] = b;
      // next chunk, 8 rows on
      idx += 8;
      if (p.fused) {
        r += 8;
        while (r >= p.m) {
          r -= p.m;
          idx += p.bias_step_m - p.m;
        }
      }
    }
}

// ---------------------------------------------------------------------------------------------
// Epilogue for a bf16 C that is not read (beta = 0).  The kernel starts the accumulators at the
// bias (load_bias4), so they hold sum + bias here; the activation is applied to them where they
// are, each lane narrows its four consecutive rows of a column to bf16
// and parks them in its own wave's LDS slab (column-major, WTM rows per column, 16-byte row
// chunks XOR-swizzled by the column), and the wave then stores the slab as 16-byte runs of 8
// rows, so every global store instruction writes whole 128-byte lines.  A wave touches only its
// own slab, so no workgroup barrier is involved; the caller has passed one after the last LDS
// read of the main loop.  ACT: 0 none, 1 ReLU, 2 GELU-tanh, 3 ReLU_inv, 4 GELU-tanh_inv.
// For the inverse activations the aux tensor (C's layout) is first loaded into the slab with the
// store's 16-byte runs, and each lane reads its saved pre-activations from the very 8 bytes
// where it then parks its result.  LDS operations of one wave complete in order, so every read
// sees the wave's earlier writes and every write lands after the wave's earlier reads.
// Keeping the pre-activation (SAVE_PREACT; ACT 5 = RELU, 6 = GELU_TANH): one pass parks each
// value (bias included) as the pre-activation and narrows its activation into registers (half the
// accumulators' count); the slab goes to aux, then the activated values are parked and stored
// to C.
// ---------------------------------------------------------------------------------------------
template <int WTM, int WTN, int TM, int TN, bool FULL, int ACT>
__device__ __forceinline__ void epilogue_bf16_act(const BrgemmParams& p, const Instance& in,
                                                  const TileCoord& tc, int wm, int wn, int lane,
                                                  int wave, char* lds, f32x16 (&acc)[TM][TN]) {
  constexpr int CPC = WTM / 8;                 // 16-byte row chunks per slab column
  constexpr int COL_BYTES = WTM * 2;
  static_assert((CPC & (CPC - 1)) == 0 && CPC <= 64, "power-of-two chunks per column");
  char* slab = lds + wave * WTN * COL_BYTES;
  const int32_t row_base = tc.row0 + wm * WTM;
  const int half = lane >> 5;                  // rows 4*half.. of each 8-row group
  // The slab <-> global walk: 64 lanes = 64 / CPC columns x CPC chunks per instruction, columns
  // advancing by COLS_PER_IT (instance column and offset tracked by additions, one division per
  // lane).  fn(slab chunk, global element offset relative to the instance's C base, valid).
  constexpr int COLS_PER_IT = 64 / CPC;
  const int chunk = lane % CPC, csub = lane / CPC;
  auto walk = [&](auto&& fn) {
    const int32_t R = row_base + chunk * 8;
    bool row_ok;
    int64_t row_off;
    if (p.fused) {
      const int32_t gi = R / p.m, r = R - gi * p.m;
      row_ok = FULL || R < p.vrows;
      row_off = (int64_t)gi * p.c_step_m + r;
    } else {
      row_ok = FULL || R < p.m;
      row_off = R;
    }
    int32_t C = tc.col0 + wn * WTN + csub;
    int32_t cin = C;
    int64_t col_off;
    if (p.fused) {
      const int32_t gi = C / p.n;
      cin = C - gi * p.n;
      col_off = (int64_t)gi * p.c_step_n + (int64_t)cin * p.ldc;
    } else {
      col_off = (int64_t)C * p.ldc;
    }
    const int32_t c_lim = p.fused ? p.vcols : p.n;
    const int64_t wrap = p.c_step_n - (int64_t)p.n * p.ldc;   // next instance, column 0
#pragma unroll 4
    for (int it = 0; it < WTN / COLS_PER_IT; ++it) {
      const int col_local = it * COLS_PER_IT + csub;
      char* sp = slab + col_local * COL_BYTES + ((chunk ^ (col_local & (CPC - 1))) << 4);
      fn(sp, in.c + row_off + col_off, row_ok && (FULL || C < c_lim));
      C += COLS_PER_IT;
      col_off += (int64_t)COLS_PER_IT * p.ldc;
      if (p.fused) {
        cin += COLS_PER_IT;
        while (cin >= p.n) {
          cin -= p.n;
          col_off += wrap;
        }
      }
    }
  };
  // slab -> tensor at base (C or aux): 16-byte runs of 8 rows
  auto store_slab = [&](void* base) {
    uint16_t* const b16 = static_cast<uint16_t*>(base);
    walk([&](const char* sp, int64_t off, bool ok) {
      const u32x4 w = *reinterpret_cast<const u32x4*>(sp);
      if (!ok) return;
      uint16_t* cp = b16 + off;
      if ((reinterpret_cast<uintptr_t>(cp) & 15) == 0) {
        gst<u32x4>(cp, w);
      } else {
        const uint32_t d[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          gst<uint16_t>(cp + 2 * e, (uint16_t)(d[e] & 0xffffu));
          gst<uint16_t>(cp + 2 * e + 1, (uint16_t)(d[e] >> 16));
        }
      }
    });
  };
  // Each lane's four rows of one column in the slab: the 8 bytes of its 8-row group's chunk.
  auto slab_at = [&](int tm, int tn, int q) -> char* {
    const int col = tn * 32 + (lane & 31);
    const int ch = tm * 4 + q;                 // 16-byte chunk of this lane's 8-row group
    return slab + col * COL_BYTES + ((ch ^ (col & (CPC - 1))) << 4) + half * 8;
  };
  // The lane's four values of (tm, tn, q) (the accumulators, which already hold the bias) through
  // activation A, narrowed.  A 3 / 4 read the saved pre-activations at sp, the slab bytes the
  // result then goes to.
  auto narrow = [&](auto act_now, int tm, int tn, int q, const char* sp) {
    constexpr int A = decltype(act_now)::value;
    float v[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = acc[tm][tn][4 * q + e];
    if constexpr (A == 3 || A == 4) {
      const uint2 zb = *reinterpret_cast<const uint2*>(sp);   // saved pre-activations
      const float z[4] = {bf16_bits_to_f32(zb.x & 0xffffu), bf16_bits_to_f32(zb.x >> 16),
                          bf16_bits_to_f32(zb.y & 0xffffu), bf16_bits_to_f32(zb.y >> 16)};
#pragma unroll
      for (int e = 0; e < 4; ++e)
        v[e] = A == 3 ? (z[e] > 0.0f ? v[e] : 0.0f) : v[e] * gelu_tanh_grad(z[e]);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if constexpr (A == 1) v[e] = v[e] > 0.0f ? v[e] : 0.0f;
      if constexpr (A == 2) v[e] = gelu_tanh(v[e]);
    }
    return make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
  };
  // All of the lane's values, through activation A, narrowed into the slab.
  auto park = [&](auto act_now) {
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          char* sp = slab_at(tm, tn, q);
          *reinterpret_cast<uint2*>(sp) = narrow(act_now, tm, tn, q, sp);
        }
  };
  if constexpr (ACT == 3 || ACT == 4) {
    // aux -> slab.  Direct global -> LDS copies: copy r fills slab bytes [1 KB r, 1 KB (r + 1)),
    // lane j's 16 bytes at 16 j, which is slot j % CPC of column r COLS_PER_IT + j / CPC; the
    // lane reads the 8-row chunk that the slab's swizzle puts there, (j % CPC) ^ (column %
    // CPC), the same chunk for every r since COLS_PER_IT is a multiple of CPC.  All of the
    // wave's copies are in flight before the one wait (16 KB per wave of a 256 x 256 tile), where
    // register loads would hold 64 more registers.  Rows and columns outside C read as zero (an
    // offset past the descriptor's range) and are never read back into a stored value.  When
    // some element lies outside the 2^31 bytes a buffer offset reaches from the wave's first
    // one, the wave takes the walk's 16-byte register loads instead.
    constexpr int NR = WTN / COLS_PER_IT;
    constexpr int BLK = NR >= 8 ? 8 : NR;   // copies per asm block
    constexpr bool DIRECT = COLS_PER_IT % CPC == 0 && NR % BLK == 0;
    const int32_t C0 = tc.col0 + wn * WTN;
    auto row_offset = [&](int32_t R, bool& ok) -> int64_t {
      if (p.fused) {
        const int32_t gi = R / p.m, r = R - gi * p.m;
        ok = FULL || R < p.vrows;
        return (int64_t)gi * p.c_step_m + r;
      }
      ok = FULL || R < p.m;
      return R;
    };
    auto col_offset = [&](int32_t C) -> int64_t {
      if (p.fused) {
        const int32_t gi = C / p.n;
        return (int64_t)gi * p.c_step_n + (int64_t)(C - gi * p.n) * p.ldc;
      }
      return (int64_t)C * p.ldc;
    };
    bool base_ok;
    const int64_t base = in.c + row_offset(row_base, base_ok) + col_offset(C0);   // wave-uniform
    const int csub = lane / CPC;
    const int ch = (lane % CPC) ^ (csub & (CPC - 1));
    bool row_ok;
    const int64_t row_off = row_offset(row_base + ch * 8, row_ok);
    const int32_t c_lim = p.fused ? p.vcols : p.n;
    uint32_t voff[NR];
    bool bad = false;
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      const int32_t C = C0 + r * COLS_PER_IT + csub;
      const bool ok = row_ok && (FULL || C < c_lim);
      const int64_t rel = in.c + row_off + col_offset(C) - base;   // elements
      const bool fits = rel >= 0 && rel < (int64_t)0x3fff0000;
      bad |= ok && !fits;
      voff[r] = ok && fits ? (uint32_t)(rel * 2) : 0x80000000u;
    }
    if (DIRECT && !__any(bad)) {
      const i32x4 rsrc = raw_buffer(static_cast<const uint16_t*>(p.aux) + base);
      const uint32_t l0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(LDS_AS char*)slab);
#pragma unroll
      for (int r = 0; r < NR; r += BLK)
        buffer_load_lds16_block<BLK>(rsrc, voff + r, l0 + r * 1024);
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    } else {
      const uint16_t* const a16 = static_cast<const uint16_t*>(p.aux);
      walk([&](char* sp, int64_t off, bool ok) {
        if (!ok) return;
        const uint16_t* ap = a16 + off;
        *reinterpret_cast<u32x4*>(sp) =
            (reinterpret_cast<uintptr_t>(ap) & 15) == 0 ? ld16(ap) : ld16_unaligned(ap);
      });
    }
  }
  if constexpr (ACT == 5 || ACT == 6) {
    // One pass over the accumulators: each value goes to the slab as the pre-activation
    // and, through the activation, into registers (half the accumulators' count), so that the
    // accumulators die as the pass goes and are dead during the aux store.
    uint2 h[TM][TN][4];
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = acc[tm][tn][4 * q + e];
          *reinterpret_cast<uint2*>(slab_at(tm, tn, q)) =
              make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = ACT == 5 ? (v[e] > 0.0f ? v[e] : 0.0f) : gelu_tanh(v[e]);
          h[tm][tn][q] = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
          // pinned here: the compiler would otherwise sink the activation to its use after the
          // aux store and hold the accumulators (in scratch) across it
          asm volatile("" : "+v"(h[tm][tn][q].x), "+v"(h[tm][tn][q].y));
        }
    __builtin_amdgcn_sched_barrier(0);
    store_slab(p.aux);   // the slab's reads complete before the writes below (in order)
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
#pragma unroll
        for (int q = 0; q < 4; ++q) *reinterpret_cast<uint2*>(slab_at(tm, tn, q)) = h[tm][tn][q];
  } else {
    park(IntC<ACT>());
  }
  store_slab(p.c);
}

template <int WTM, int WTN, int TM, int TN, bool FULL>
__device__ __forceinline__ void epilogue_bf16(const BrgemmParams& p, const Instance& in,
                                              const TileCoord& tc, int wm, int wn, int lane,
                                              int wave, char* lds, f32x16 (&acc)[TM][TN]) {
  const uint32_t f = p.flags;
#define TPP_EPI_BF16(A) \
  epilogue_bf16_act<WTM, WTN, TM, TN, FULL, A>(p, in, tc, wm, wn, lane, wave, lds, acc)
  if (f & TPP_EPI_GELU_TANH_INV) {
    TPP_EPI_BF16(4);
  } else if (f & TPP_EPI_RELU_INV) {
    TPP_EPI_BF16(3);
  } else if (f & TPP_EPI_GELU_TANH) {
    if (f & TPP_EPI_SAVE_PREACT) TPP_EPI_BF16(6); else TPP_EPI_BF16(2);
  } else if (f & TPP_EPI_RELU) {
    if (f & TPP_EPI_SAVE_PREACT) TPP_EPI_BF16(5); else TPP_EPI_BF16(1);
  } else {
    TPP_EPI_BF16(0);
  }
#undef TPP_EPI_BF16
}

}  // namespace dev
}  // namespace tpp
