// brgemm_dl_kernels.hip -- bf16 batch-reduce GEMM with direct global -> LDS staging (gfx950).
//
// Same computation and tiling as the 16-byte-load kernels (see brgemm_kernels.hip), with the
// operand staging rebuilt around two gfx950 instructions:
//   - global_load_lds_dwordx4 writes each lane's 16 bytes straight into LDS (lane j at M0 + 16 j),
//     so staging needs no registers and no LDS-write instructions: a ring of DL_SLOTS LDS slots
//     keeps DL_SLOTS - 1 stages of 32 k in flight while the MFMAs consume the oldest;
//   - ds_read_b64_tr_b16 reads an M-contiguous A panel transposed, so A is staged in its own
//     layout and the MFMA still gets 8 consecutive k per lane (two transposing reads per
//     fragment).
// Both panels are XOR-swizzled at 16-byte granularity so that the fragment reads of a wavefront
// spread over all LDS banks.
// Requirements on top of the 16-byte-load path: k a multiple of 32 (the k tail is never zeroed:
// out-of-range rows and columns load clamped, in-range data that only reaches discarded outputs).
#include <hip/hip_runtime.h>

#include "brgemm_device.h"
#include "internal.h"

namespace tpp {
namespace {

using namespace dev;

typedef short v4i16 __attribute__((ext_vector_type(4)));
#define LDS_AS __attribute__((address_space(3)))

constexpr int DL_BK = 32;     // k per stage
constexpr int DL_SLOTS = 4;   // LDS ring slots: three stages in flight

// s_waitcnt immediate waiting until at most n vector-memory operations are outstanding (gfx9
// encoding: vmcnt in bits 3:0 and 15:14, expcnt 6:4 and lgkmcnt 11:8 left at their maxima).
constexpr int vmcnt_imm(int n) {
  return (n & 0xF) | (((n >> 4) & 3) << 14) | (0x7 << 4) | (0xF << 8);
}

// 16-byte global -> LDS copy of a whole wave (global_load_lds_dwordx4): lane j's 16 bytes land at
// l + 16 j, where l is wave-uniform.  It is issued through inline asm so that the compiler does
// not see a pending LDS write: the compiler would otherwise wait for every outstanding load
// (vmcnt 0) before the next LDS read and so drain the stages kept in flight.  Callers order these
// loads themselves with s_waitcnt vmcnt and lds_barrier().  M0 is saved and restored around it.
__device__ __forceinline__ void load_lds16(const void* g, char* l) {
  const uint32_t lds_addr =
      __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(LDS_AS char*)l);
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off\n\t"
      "s_nop 0\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(g), "s"(lds_addr)
      : "memory");
}

// XOR swizzle of the 16-byte chunks of an A-panel k-row (row pitch ROW bytes): the four k-rows a
// transposing read touches land in four different 64-byte bank groups.
template <int ROW>
__device__ __forceinline__ int swz_a(int k) {
  if constexpr (ROW >= 256)
    return (k & 3) << 2;
  else
    return ((k >> 1) & 1) << 2;
}

template <int BM, int BN, int WAVES_M, int WAVES_N, bool FULL, int KIND, bool ALIGNED, bool PP>
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N) void brgemm_bf16_dl_kernel(BrgemmParams p) {
  constexpr int NW = WAVES_M * WAVES_N;
  constexpr int WTM = BM / WAVES_M, WTN = BN / WAVES_N;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int A_ROW = BM * 2;                 // bytes per k-row of the A panel
  constexpr int A_BYTES = DL_BK * A_ROW;        // A panel of one slot
  constexpr int B_BYTES = BN * DL_BK * 2;       // B panel of one slot (64 B per column)
  constexpr int SLOT = A_BYTES + B_BYTES;
  constexpr int A_PER_W = A_BYTES / 1024 / NW;  // 1 KB wave-loads per wave and stage
  constexpr int B_PER_W = B_BYTES / 1024 / NW;
  constexpr int LPS = A_PER_W + B_PER_W;        // vector-memory operations per wave and stage
  constexpr int EP_BYTES = NW * 32 * (WTM + 4) * 4;
  constexpr int LDS_BYTES = (DL_SLOTS * SLOT > EP_BYTES) ? DL_SLOTS * SLOT : EP_BYTES;
  static_assert(A_BYTES % (1024 * NW) == 0 && B_BYTES % (1024 * NW) == 0, "whole wave-loads");
  static_assert(A_PER_W >= 1 && B_PER_W >= 1, "every wave loads both panels");
  static_assert(TM >= 1 && TN >= 1, "wave tile at least 32x32");
  static_assert(BM * BN * 2 <= LDS_BYTES, "bf16 epilogue slabs fit in the ring");

  __shared__ __attribute__((aligned(1024))) char lds[LDS_BYTES];

  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);   // wave-uniform: kept in SGPRs
  const int wm = wave % WAVES_M, wn = wave / WAVES_M;
  const TileCoord tc = decode_tile(p, BM, BN);
  const Instance in = instance_of(p, tc.g);
  const int32_t ksteps = p.k / DL_BK;
  const int32_t stages = (int32_t)(in.npairs * ksteps);

  // Per-lane load assignments.  A wave-load r covers bytes [q*1024, q*1024 + 1024) of the A
  // panel (q = wave * A_PER_W + r); lane j fills the 16-byte chunk at q*1024 + 16 j, i.e. k-row
  // kr and swizzled chunk position sc, which holds the 8 rows m = 8 * (sc ^ swz(kr)).
  int64_t a_off[A_PER_W];
  int a_kr[A_PER_W];
#pragma unroll
  for (int r = 0; r < A_PER_W; ++r) {
    const int byte = (wave * A_PER_W + r) * 1024 + lane * 16;
    const int kr = byte / A_ROW, sc = (byte % A_ROW) / 16;
    const int m_local = (sc ^ swz_a<A_ROW>(kr)) * 8;
    a_kr[r] = kr;
    int64_t off = 0;
    const bool ok = row_in_a(p, tc.row0 + m_local, off);
    a_off[r] = ok ? off : 0;   // out-of-range rows read row 0: only discarded outputs see it
  }
  // B wave-load r: 16 columns of 64 bytes; lane j fills column 4*q + j/4 (q-th group of 16
  // columns), chunk position j%4, which holds k-chunk (j%4) ^ ((column >> 2) & 3).
  int64_t b_off[B_PER_W];
#pragma unroll
  for (int r = 0; r < B_PER_W; ++r) {
    const int byte = (wave * B_PER_W + r) * 1024 + lane * 16;
    const int col = byte / 64, sc = (byte % 64) / 16;
    const int kc = sc ^ ((col >> 2) & 3);
    int64_t off = 0;
    const bool ok = col_in_b(p, tc.col0 + col, off);
    b_off[r] = (ok ? off : 0) + kc * 8;
  }

  // Byte offset of each wave-load's 16 bytes inside a pair's A / B block at k = 0: constant over
  // the stages, so a stage's address is one wave-uniform base plus this per-lane offset.
  int64_t la[A_PER_W], lb[B_PER_W];
#pragma unroll
  for (int r = 0; r < A_PER_W; ++r) la[r] = (a_off[r] + (int64_t)a_kr[r] * p.lda) * 2;
#pragma unroll
  for (int r = 0; r < B_PER_W; ++r) lb[r] = b_off[r] * 2;

  // Stages are issued in order; (iss_i, iss_kk) is the pair and k offset of the next one, so no
  // stage index is ever divided.
  int32_t iss_i = 0, iss_kk = 0, iss_s = 0;
  auto issue = [&]() {
    const uint16_t* pa;
    const uint16_t* pb;
    pair_bases_k<KIND, uint16_t>(p, in, iss_i, pa, pb);
    const char* ua = reinterpret_cast<const char*>(pa) + (int64_t)iss_kk * p.lda * 2;
    const char* ub = reinterpret_cast<const char*>(pb) + (int64_t)iss_kk * 2;
    char* slot = lds + (iss_s % DL_SLOTS) * SLOT;
    const bool aligned =
        ALIGNED || ((reinterpret_cast<uintptr_t>(pa) | reinterpret_cast<uintptr_t>(pb)) & 15) == 0;
    if (ALIGNED || aligned) {
#pragma unroll
      for (int r = 0; r < A_PER_W; ++r) load_lds16(ua + la[r], slot + (wave * A_PER_W + r) * 1024);
#pragma unroll
      for (int r = 0; r < B_PER_W; ++r)
        load_lds16(ub + lb[r], slot + A_BYTES + (wave * B_PER_W + r) * 1024);
    } else {
      // A pair block off 16-byte alignment (offset or pointer lists): the same chunks through
      // registers, element by element.
#pragma unroll
      for (int r = 0; r < A_PER_W; ++r)
        *reinterpret_cast<u32x4*>(slot + (wave * A_PER_W + r) * 1024 + lane * 16) =
            ld16_unaligned(reinterpret_cast<const uint16_t*>(ua + la[r]));
#pragma unroll
      for (int r = 0; r < B_PER_W; ++r)
        *reinterpret_cast<u32x4*>(slot + A_BYTES + (wave * B_PER_W + r) * 1024 + lane * 16) =
            ld16_unaligned(reinterpret_cast<const uint16_t*>(ub + lb[r]));
    }
    ++iss_s;
    iss_kk += DL_BK;
    if (iss_kk == p.k) {
      iss_kk = 0;
      ++iss_i;
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[tm][tn][v] = 0.0f;

  // Fragment addressing, fixed per lane.  A (transposing reads): lane j of 16-lane group g reads
  // k-row kq*16 + 8*(g/2) + 4*h + j/4, rows m = base + 16*(g%2) + 4*(j%4) .. +3; the wavefront
  // then holds A[m = lane%32][k = 8*(lane/32) + 4*h + e].  B (plain reads): column lane%32 of the
  // tile, k-chunk 2*kq + lane/32.
  const int g = lane >> 4, j = lane & 15;
  const int a_lo = 2 * (g & 1) + ((j >> 1) & 1);      // chunk within the 32-row group
  const int a_sub = 8 * (j & 1);                      // byte within the chunk
  const int b_swz = (lane >> 2) & 3;

  constexpr int KQ = DL_BK / 16;   // MFMA k-steps per stage
  // Fragments of k-step kq of the stage held in slot slot_idx.
  auto read_frags = [&](int slot_idx, int kq, bf16x8 (&af)[TM], bf16x8 (&bfr)[TN]) {
    const char* As = lds + slot_idx * SLOT;
    const char* Bs = As + A_BYTES;
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
      const int hi = (wm * WTM + tm * 32) >> 3;     // first chunk of the 32-row group
      v4i16 half[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int k = kq * 16 + 8 * (g >> 1) + 4 * h + (j >> 2);
        const int byte = k * A_ROW + (((hi ^ swz_a<A_ROW>(k)) + a_lo) << 4) + a_sub;
        half[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS v4i16*)(As + byte));
      }
      const u32x4 w = {(uint32_t)(uint16_t)half[0][0] | ((uint32_t)(uint16_t)half[0][1] << 16),
                       (uint32_t)(uint16_t)half[0][2] | ((uint32_t)(uint16_t)half[0][3] << 16),
                       (uint32_t)(uint16_t)half[1][0] | ((uint32_t)(uint16_t)half[1][1] << 16),
                       (uint32_t)(uint16_t)half[1][2] | ((uint32_t)(uint16_t)half[1][3] << 16)};
      af[tm] = __builtin_bit_cast(bf16x8, w);
    }
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const int col = wn * WTN + tn * 32 + (lane & 31);
      const int kc = 2 * kq + (lane >> 5);
      bfr[tn] = *reinterpret_cast<const bf16x8*>(Bs + col * 64 + ((kc ^ b_swz) << 4));
    }
  };
  auto mfmas = [&](const bf16x8 (&af)[TM], const bf16x8 (&bfr)[TN]) {
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
        acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[tm], bfr[tn], acc[tm][tn], 0, 0, 0);
  };
  auto compute = [&](int slot_idx) {
#pragma unroll
    for (int kq = 0; kq < KQ; ++kq) {
      bf16x8 af[TM], bfr[TN];
      read_frags(slot_idx, kq, af, bfr);
      mfmas(af, bfr);
    }
  };
  // Wait until this wave's loads of the stage `ahead` stages before its newest issued one landed.
  auto wait_loads = [&](int32_t ahead) {
    if (ahead >= 2)
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * LPS));
    else if (ahead == 1)
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(LPS));
    else
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
  };

  const int32_t pre = stages < DL_SLOTS - 1 ? stages : DL_SLOTS - 1;
  for (int32_t s = 0; s < pre; ++s) issue();
  if constexpr (!PP) {
    for (int32_t s = 0; s < stages; ++s) {
      // This wave's loads of stage s are done once at most the later stages' loads are pending;
      // the barrier then publishes every wave's stage s and retires everyone's reads of s - 1.
      wait_loads(stages - 1 - s < 2 ? stages - 1 - s : 2);
      lds_barrier();
      if (s + DL_SLOTS - 1 < stages) issue();   // stage s + 3 refills the slot of stage s - 1
      compute(s % DL_SLOTS);
    }
  } else {
    // Ping-pong: waves 0-3 (one per SIMD) lead, waves 4-7 lag by one half-period.  Each stage is
    // a memory half (fragment reads of the stage, global->LDS issue of stage s + 3) and a compute
    // half (the stage's MFMAs on registers); while one wave of a SIMD computes, the other reads,
    // so every barrier finds the next MFMA phase's operands already in registers.
    //   barrier j:  leading waves end M(j/2) (j even) or C(j/2) (j odd);
    //               lagging waves end C(j/2 - 1) (j even, the first one is the offset barrier) or
    //               M(j/2) (j odd).
    // Stage s + 1 must have landed before barrier 2s + 1, the last barrier before anyone reads it:
    // the leading waves wait at the end of C(s), the lagging ones at the end of M(s).
    static_assert(NW == 8, "two groups of four waves");
    const bool lead = wave < 4;
    wait_loads(stages - 1 < 2 ? stages - 1 : 2);   // stage 0, before anyone reads it
    lds_barrier();
    if (!lead) lds_barrier();
    bf16x8 af[KQ][TM], bfr[KQ][TN];
    for (int32_t s = 0; s < stages; ++s) {
      const int32_t later = stages - 2 - s < 2 ? stages - 2 - s : 2;
#pragma unroll
      for (int kq = 0; kq < KQ; ++kq) read_frags(s % DL_SLOTS, kq, af[kq], bfr[kq]);
      if (s + DL_SLOTS - 1 < stages) issue();   // stage s + 3
      if (!lead && s + 1 < stages) wait_loads(later);
      lds_barrier();
#pragma unroll
      for (int kq = 0; kq < KQ; ++kq) mfmas(af[kq], bfr[kq]);
      if (lead && s + 1 < stages) wait_loads(later);
      lds_barrier();
    }
    if (lead) lds_barrier();
  }
  __syncthreads();
  if (p.c_bf16 && p.beta == 0.0f)
    epilogue_bf16<WTM, WTN, TM, TN, FULL>(p, in, tc, wm, wn, lane, wave, lds, acc);
  else
    epilogue_via_lds<WTM, WTN, TM, TN, FULL>(p, in, tc, wm, wn, lane, wave,
                                            reinterpret_cast<float*>(lds), acc);
}

template <int BM, int BN, int WM, int WN, bool FULL, int KIND, bool PP>
void launch_dl_k(const BrgemmParams& p, dim3 grid, hipStream_t stream) {
  const dim3 block(64 * WM * WN);
  if constexpr (KIND == TPP_BR_STRIDE) {
    if (p.aligned) {
      hipLaunchKernelGGL((brgemm_bf16_dl_kernel<BM, BN, WM, WN, FULL, KIND, true, PP>), grid, block,
                         0, stream, p);
      return;
    }
  }
  hipLaunchKernelGGL((brgemm_bf16_dl_kernel<BM, BN, WM, WN, FULL, KIND, false, PP>), grid, block, 0,
                     stream, p);
}

template <int BM, int BN, int WM, int WN, bool PP = false>
void launch_dl(const BrgemmParams& p, bool full, dim3 grid, hipStream_t stream) {
  switch (p.kind) {
    case TPP_BR_STRIDE:
      full ? launch_dl_k<BM, BN, WM, WN, true, TPP_BR_STRIDE, PP>(p, grid, stream)
           : launch_dl_k<BM, BN, WM, WN, false, TPP_BR_STRIDE, PP>(p, grid, stream);
      break;
    case TPP_BR_OFFSET:
      full ? launch_dl_k<BM, BN, WM, WN, true, TPP_BR_OFFSET, PP>(p, grid, stream)
           : launch_dl_k<BM, BN, WM, WN, false, TPP_BR_OFFSET, PP>(p, grid, stream);
      break;
    default:
      full ? launch_dl_k<BM, BN, WM, WN, true, TPP_BR_ADDRESS, PP>(p, grid, stream)
           : launch_dl_k<BM, BN, WM, WN, false, TPP_BR_ADDRESS, PP>(p, grid, stream);
      break;
  }
}

}  // namespace

hipError_t launch_brgemm_dl(const BrgemmParams& p, int32_t id, bool full, dim3 grid,
                            hipStream_t stream) {
  switch (id) {
    case K_BF16_DL_256x256: launch_dl<256, 256, 2, 4>(p, full, grid, stream); break;
    case K_BF16_DL_128x128: launch_dl<128, 128, 2, 2>(p, full, grid, stream); break;
    case K_BF16_DL_64x64: launch_dl<64, 64, 2, 2>(p, full, grid, stream); break;
    case K_BF16_PP_256x256: launch_dl<256, 256, 2, 4, true>(p, full, grid, stream); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace tpp
