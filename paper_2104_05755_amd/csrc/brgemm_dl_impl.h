// brgemm_dl_impl.h -- bf16 batch-reduce GEMM with direct global -> LDS staging (gfx950).
//
// Same computation and tiling as the 16-byte-load kernels (see brgemm_kernels.hip), with the
// operand staging rebuilt around two gfx950 instructions:
//   - buffer_load_dwordx4 ... lds writes each lane's 16 bytes straight into LDS (lane j at M0 + 16 j),
//     so staging needs no registers and no LDS-write instructions: a ring of SLOTS = 4 LDS slots
//     keeps SLOTS - 1 stages of 32 k in flight while the MFMAs consume the oldest;
//   - ds_read_b64_tr_b16 reads an M-contiguous A panel transposed, so A is staged in its own
//     layout and the MFMA still gets 8 consecutive k per lane (two transposing reads per
//     fragment).
// Both panels are XOR-swizzled at 16-byte granularity so that the fragment reads of a wavefront
// spread over all LDS banks.
// Requirements on top of the 16-byte-load path: k a multiple of 32 (the k tail is never zeroed:
// out-of-range rows and columns load clamped, in-range data that only reaches discarded outputs).
#pragma once
#include <hip/hip_runtime.h>

#include <cstdio>
#include <string>

#include "brgemm_device.h"
#include "internal.h"

namespace tpp {
namespace {

using namespace dev;

typedef short v4i16 __attribute__((ext_vector_type(4)));
constexpr int LDS_MAX = 160 * 1024;   // bytes of LDS per workgroup on gfx950

// XOR swizzle of the 16-byte k-chunks of a B-panel column (COLB = 2 BK bytes): the 16 columns a
// ds_read_b128 serves per cycle land in 16 distinct 16-byte bank groups of a 256-byte row.
template <int BK>
__device__ __forceinline__ int swz_b(int col) {
  if constexpr (BK == 64)
    return (col >> 1) & 7;
  else
    return (col >> 2) & 3;
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

// SCHED: 0 = every wave loads, reads and multiplies in turn; 1 = ping-pong (memory half = fragment
// reads + load issue, compute half = MFMAs, two wave groups offset by a half-period).
// BKT: k per stage, 32 or 64.  At 64 every stage reads whole 128-byte lines of the K-contiguous B
// blocks (a column of a 64-k block is 128 bytes); at 32 each B column load covers half a line.
template <int BM, int BN, int WAVES_M, int WAVES_N, bool FULL, int KIND, bool ALIGNED, int SCHED,
          int BKT, int SLOTS_T, bool AT, bool BT>
// Four-wave instances run two workgroups per CU, i.e. two waves per SIMD: at most 256 registers.
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N, (WAVES_M * WAVES_N == 4) ? 2 : 1)
void brgemm_bf16_dl_kernel(BrgemmParams p) {
  constexpr int DL_BK = BKT;
  static_assert(BKT == 32 || BKT == 64, "stage depth");
  constexpr int NW = WAVES_M * WAVES_N;
  constexpr int WTM = BM / WAVES_M, WTN = BN / WAVES_N;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int A_ROW = BM * 2;                 // bytes per k-row of the A panel
  constexpr int A_BYTES = DL_BK * A_ROW;        // A panel of one slot
  constexpr int COLB = DL_BK * 2;               // bytes of one B column in a slot
  constexpr int B_ROW = BN * 2;                 // bytes per k-row of a transposed B panel (BT)
  constexpr int B_BYTES = BN * COLB;            // B panel of one slot
  constexpr int SLOT = A_BYTES + B_BYTES;
  constexpr int A_PER_W = A_BYTES / 1024 / NW;  // 1 KB wave-loads per wave and stage
  constexpr int B_PER_W = B_BYTES / 1024 / NW;
  constexpr int LPS = A_PER_W + B_PER_W;        // vector-memory operations per wave and stage
  constexpr int EP_BYTES = NW * 32 * (WTM + 4) * 4;
  // LDS ring slots: three 32-k stages in flight (a fifth slot, which fits, measured slower), or
  // one 64-k stage (two 64 KB slots for the 256x256 tile).
  constexpr int SLOTS = SLOTS_T > 0 ? SLOTS_T : (BKT == 64 ? 2 : 4);
  static_assert(BKT == 32 || SCHED == 0, "the ping-pong schedule keeps three stages in flight");
  static_assert(SLOTS * SLOT <= LDS_MAX, "ring fits in LDS");
  constexpr int LDS_BYTES = (SLOTS * SLOT > EP_BYTES) ? SLOTS * SLOT : EP_BYTES;
  static_assert(A_BYTES % (1024 * NW) == 0 && B_BYTES % (1024 * NW) == 0, "whole wave-loads");
  static_assert(A_PER_W >= 1 && B_PER_W >= 1, "every wave loads both panels");
  static_assert(TM >= 1 && TN >= 1, "wave tile at least 32x32");
  static_assert(BM * BN * 2 <= LDS_BYTES, "bf16 epilogue slabs fit in the ring");

  __shared__ __attribute__((aligned(1024))) char lds[LDS_BYTES];

  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);   // wave-uniform: kept in SGPRs
  const int wm = wave % WAVES_M, wn = wave / WAVES_M;
  // Split launches (p.split > 1): workgroup b reduces chunk b / total_tiles of the stage list of
  // tile b % total_tiles (consecutive block ids still alternate over the XCDs, as the tile order
  // assumes) into a partial tile of the work buffer; a finishing kernel adds the chunks.
  const int64_t bid = blockIdx.x;
  const int32_t chunk = p.split > 1 ? (int32_t)(bid / p.total_tiles) : 0;
  const int64_t tile_bid = bid - (int64_t)chunk * p.total_tiles;
  const TileCoord tc = decode_tile_at(p, BM, BN, tile_bid);
  const Instance in = instance_of(p, tc.g);
  const int32_t ksteps = p.k / DL_BK;
  const int32_t all_stages = (int32_t)(in.npairs * ksteps);
  const int32_t s_first = p.split > 1 ? (int32_t)((int64_t)all_stages * chunk / p.split) : 0;
  const int32_t stages =
      p.split > 1 ? (int32_t)((int64_t)all_stages * (chunk + 1) / p.split) - s_first : all_stages;

  // Element offsets of the first instance block the tile touches in A and in B: every row / column
  // offset of the tile is at least this (the host takes this kernel only for non-negative steps
  // and a tile span below 2^31 bytes), so loads address the operands as base + 32-bit offset.
  const int64_t base_a = p.fused ? (int64_t)(tc.row0 / p.m) * p.a_step_m : 0;
  const int64_t base_b = p.fused ? (int64_t)(tc.col0 / p.n) * p.b_step_n : 0;

  // Per-lane load assignments.  A wave-load r covers bytes [q*1024, q*1024 + 1024) of the A
  // panel (q = wave * A_PER_W + r); lane j fills the 16-byte chunk at q*1024 + 16 j, i.e. k-row
  // kr and swizzled chunk position sc, which holds the 8 rows m = 8 * (sc ^ swz(kr)).
  // AT (A_i stored transposed): the A panel is laid out and loaded like the B panel, BM rows of
  // COLB bytes (row m's k-run of the stage), swizzled by row as B is by column.
  int64_t a_off[A_PER_W];
  int a_kr[A_PER_W];
#pragma unroll
  for (int r = 0; r < A_PER_W; ++r) {
    if constexpr (AT) {
      const int byte = (wave * A_PER_W + r) * 1024 + lane * 16;
      const int row = byte / COLB, sc = (byte % COLB) / 16;
      const int kc = sc ^ swz_b<BKT>(row);
      int64_t off = 0;
      const bool ok = row_in_at(p, tc.row0 + row, off);
      a_kr[r] = 0;
      a_off[r] = (ok ? off : base_a) + kc * 8;
      continue;
    }
    const int byte = (wave * A_PER_W + r) * 1024 + lane * 16;
    const int kr = byte / A_ROW, sc = (byte % A_ROW) / 16;
    const int m_local = (sc ^ swz_a<A_ROW>(kr)) * 8;
    a_kr[r] = kr;
    int64_t off = 0;
    const bool ok = row_in_a(p, tc.row0 + m_local, off);
    a_off[r] = ok ? off : base_a;   // out-of-range rows read a valid row: only discarded outputs see it
  }
  // B wave-load r: 16 columns of 64 bytes; lane j fills column 4*q + j/4 (q-th group of 16
  // columns), chunk position j%4, which holds k-chunk (j%4) ^ ((column >> 2) & 3).
  // BT (B_i stored transposed): the B panel is laid out and loaded like the A panel, DL_BK
  // k-rows of B_ROW bytes holding 8 consecutive columns per 16-byte chunk, swizzled by k-row.
  int64_t b_off[B_PER_W];
  int b_kr[B_PER_W];
#pragma unroll
  for (int r = 0; r < B_PER_W; ++r) {
    if constexpr (BT) {
      const int byte = (wave * B_PER_W + r) * 1024 + lane * 16;
      const int kr = byte / B_ROW, sc = (byte % B_ROW) / 16;
      const int n_local = (sc ^ swz_a<B_ROW>(kr)) * 8;
      b_kr[r] = kr;
      int64_t off = 0;
      const bool ok = col_in_bt(p, tc.col0 + n_local, off);
      b_off[r] = ok ? off : base_b;   // out-of-range columns read a valid one (discarded)
      continue;
    }
    b_kr[r] = 0;
    const int byte = (wave * B_PER_W + r) * 1024 + lane * 16;
    const int col = byte / COLB, sc = (byte % COLB) / 16;
    const int kc = sc ^ swz_b<BKT>(col);
    int64_t off = 0;
    const bool ok = col_in_b(p, tc.col0 + col, off);
    b_off[r] = (ok ? off : base_b) + kc * 8;
  }

  // Byte offset of each wave-load's 16 bytes from the tile's base inside a pair's A / B block at
  // k = 0: constant over the stages, so a stage's address is one wave-uniform base (a buffer
  // descriptor) plus this per-lane offset.
  uint32_t la[A_PER_W], lb[B_PER_W];
#pragma unroll
  for (int r = 0; r < A_PER_W; ++r)
    la[r] = (uint32_t)((a_off[r] - base_a + (AT ? 0 : (int64_t)a_kr[r] * p.lda)) * 2);
#pragma unroll
  for (int r = 0; r < B_PER_W; ++r)
    lb[r] = (uint32_t)((b_off[r] - base_b + (BT ? (int64_t)b_kr[r] * p.ldb : 0)) * 2);

  // Stages are issued in order; (iss_i, iss_kk) is the pair and k offset of the next one, so no
  // stage index is ever divided.  A stage's wave-loads can be spread over other work:
  // stage_begin(), issue_load(r) for r < LPS (A loads first, then B), stage_end().
  int32_t iss_i = s_first / ksteps, iss_kk = (s_first - iss_i * ksteps) * DL_BK, iss_s = 0;
  const char* ua = nullptr;
  const char* ub = nullptr;
  i32x4 ra, rb;
  char* slot = lds;
  bool aligned = true;
  // Offset and pointer lists: lane j holds pair j's two entries (the first 64 pairs), loaded
  // once; a stage picks its pair's with readlane instead of a memory load per stage.
  uint64_t pair_a = 0, pair_b = 0;
  if constexpr (KIND == TPP_BR_OFFSET) {
    if (lane < in.npairs) {
      pair_a = (uint64_t)p.offs_a[lane];
      pair_b = (uint64_t)p.offs_b[lane];
    }
  } else if constexpr (KIND == TPP_BR_ADDRESS) {
    if (lane < in.npairs) {
      pair_a = reinterpret_cast<uint64_t>(p.ptrs_a[in.pair0 + lane]);
      pair_b = reinterpret_cast<uint64_t>(p.ptrs_b[in.pair0 + lane]);
    }
  }
  auto lane_u64 = [](uint64_t v, int32_t src) {
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)v, src);
    const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(v >> 32), src);
    return ((uint64_t)hi << 32) | lo;
  };
  auto stage_begin = [&]() {
    const uint16_t* pa;
    const uint16_t* pb;
    if (KIND != TPP_BR_STRIDE && iss_i < 64) {
      const uint64_t ea = lane_u64(pair_a, iss_i), eb = lane_u64(pair_b, iss_i);
      if constexpr (KIND == TPP_BR_OFFSET) {
        pa = static_cast<const uint16_t*>(p.a) + in.a + (int64_t)ea;
        pb = static_cast<const uint16_t*>(p.b) + in.b + (int64_t)eb;
      } else {
        pa = reinterpret_cast<const uint16_t*>(ea);
        pb = reinterpret_cast<const uint16_t*>(eb);
      }
    } else {
      pair_bases_k<KIND, uint16_t>(p, in, iss_i, pa, pb);
    }
    ua = reinterpret_cast<const char*>(pa + base_a) + (int64_t)iss_kk * (AT ? 1 : p.lda) * 2;
    ub = reinterpret_cast<const char*>(pb + base_b) + (int64_t)iss_kk * (BT ? p.ldb : 1) * 2;
    ra = raw_buffer(ua);
    rb = raw_buffer(ub);
    slot = lds + (iss_s % SLOTS) * SLOT;
    aligned =
        ALIGNED || ((reinterpret_cast<uintptr_t>(pa) | reinterpret_cast<uintptr_t>(pb)) & 15) == 0;
  };
  auto issue_load = [&](int r) {
    const bool is_a = r < A_PER_W;
    char* dst = is_a ? slot + (wave * A_PER_W + r) * 1024
                     : slot + A_BYTES + (wave * B_PER_W + (r - A_PER_W)) * 1024;
    if (ALIGNED || aligned) {
      buffer_load_lds16(is_a ? ra : rb, is_a ? la[r] : lb[r - A_PER_W], dst);
    } else {
      // a pair block off 16-byte alignment (offset or pointer lists): the same chunk through
      // registers, element by element
      const char* src = is_a ? ua + la[r] : ub + lb[r - A_PER_W];
      *reinterpret_cast<u32x4*>(dst + lane * 16) =
          ld16_unaligned(reinterpret_cast<const uint16_t*>(src));
    }
  };
  auto stage_end = [&]() {
    ++iss_s;
    iss_kk += DL_BK;
    if (iss_kk == p.k) {
      iss_kk = 0;
      ++iss_i;
    }
  };
  auto issue = [&]() {
    stage_begin();
#pragma unroll
    for (int r = 0; r < LPS; ++r) issue_load(r);
    stage_end();
  };
  // The same issue with each operand's wave-loads in one block (buffer_load_lds16_block), and for
  // the stride kind the stage's byte addresses advanced by additions: a pair's A / B base moves
  // by the stride, a stage within the pair by the k-step (no 64-bit multiplies per stage).
  const uint32_t lds_u32 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(LDS_AS char*)lds);
  auto uni64 = [](uint64_t v) {
    return ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(v >> 32)) << 32) |
           (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)v);
  };
  const uint64_t a_kstep = (uint64_t)DL_BK * (AT ? 1 : p.lda) * 2;
  const uint64_t b_kstep = (uint64_t)DL_BK * (BT ? p.ldb : 1) * 2;
  uint64_t sa_pair = 0, sb_pair = 0, sa = 0, sb = 0;
  if constexpr (KIND == TPP_BR_STRIDE) {
    sa_pair = uni64(reinterpret_cast<uint64_t>(static_cast<const uint16_t*>(p.a) + in.a + base_a +
                                               (int64_t)iss_i * p.stride_a));
    sb_pair = uni64(reinterpret_cast<uint64_t>(static_cast<const uint16_t*>(p.b) + in.b + base_b +
                                               (int64_t)iss_i * p.stride_b));
    sa = sa_pair + (uint64_t)(iss_kk / DL_BK) * a_kstep;
    sb = sb_pair + (uint64_t)(iss_kk / DL_BK) * b_kstep;
  }
  // Offset and pointer lists with one stage per pair (k equal to the stage depth), at most 64
  // pairs and every listed block 16-byte aligned (four-wave instances): lane j holds pair j's
  // byte addresses, so a stage's copies take two readlanes per operand instead of the pair's
  // address arithmetic and alignment test on the scalar unit, which the compute unit's waves
  // share (the 3x3 convolution runs six workgroups per CU).
  uint64_t fa = 0, fb = 0;
  bool fast_list = false;
  if constexpr (KIND != TPP_BR_STRIDE && NW == 4) {
    if (p.k == DL_BK && in.npairs <= 64) {
      bool ok = true;
      if (lane < in.npairs) {
        const uint16_t* pa;
        const uint16_t* pb;
        if constexpr (KIND == TPP_BR_OFFSET) {
          pa = static_cast<const uint16_t*>(p.a) + in.a + (int64_t)pair_a;
          pb = static_cast<const uint16_t*>(p.b) + in.b + (int64_t)pair_b;
        } else {
          pa = reinterpret_cast<const uint16_t*>(pair_a);
          pb = reinterpret_cast<const uint16_t*>(pair_b);
        }
        ok = ((reinterpret_cast<uintptr_t>(pa) | reinterpret_cast<uintptr_t>(pb)) & 15) == 0;
        fa = reinterpret_cast<uint64_t>(pa + base_a);
        fb = reinterpret_cast<uint64_t>(pb + base_b);
      }
      fast_list = __all(ok);
    }
  }
  auto issue_block = [&]() {
    if (KIND != TPP_BR_STRIDE && NW == 4 && fast_list) {
      const uint32_t slot_u32 = lds_u32 + (uint32_t)(iss_s % SLOTS) * SLOT;
      buffer_load_lds16_block<A_PER_W>(raw_buffer(reinterpret_cast<const void*>(lane_u64(fa, iss_i))),
                                       la, slot_u32 + wave * A_PER_W * 1024);
      buffer_load_lds16_block<B_PER_W>(raw_buffer(reinterpret_cast<const void*>(lane_u64(fb, iss_i))),
                                       lb, slot_u32 + A_BYTES + wave * B_PER_W * 1024);
      ++iss_s;
      ++iss_i;
      return;
    }
    if constexpr (KIND == TPP_BR_STRIDE && ALIGNED) {
      const uint32_t slot_u32 = lds_u32 + (uint32_t)(iss_s % SLOTS) * SLOT;
      buffer_load_lds16_block<A_PER_W>(raw_buffer(reinterpret_cast<const void*>(sa)), la,
                                       slot_u32 + wave * A_PER_W * 1024);
      buffer_load_lds16_block<B_PER_W>(raw_buffer(reinterpret_cast<const void*>(sb)), lb,
                                       slot_u32 + A_BYTES + wave * B_PER_W * 1024);
      ++iss_s;
      iss_kk += DL_BK;
      if (iss_kk == p.k) {
        iss_kk = 0;
        ++iss_i;
        sa_pair += (uint64_t)p.stride_a * 2;
        sb_pair += (uint64_t)p.stride_b * 2;
        sa = sa_pair;
        sb = sb_pair;
      } else {
        sa += a_kstep;
        sb += b_kstep;
      }
    } else {
      stage_begin();
      if (ALIGNED || aligned) {
        const uint32_t slot_u32 = lds_u32 + (uint32_t)(iss_s % SLOTS) * SLOT;
        buffer_load_lds16_block<A_PER_W>(ra, la, slot_u32 + wave * A_PER_W * 1024);
        buffer_load_lds16_block<B_PER_W>(rb, lb, slot_u32 + A_BYTES + wave * B_PER_W * 1024);
      } else {
#pragma unroll
        for (int r = 0; r < LPS; ++r) issue_load(r);
      }
      stage_end();
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
  const int b_swz = swz_b<BKT>(lane & 31);   // the column's swizzle (wave tiles start at 32k)

  constexpr int KQ = DL_BK / 16;   // MFMA k-steps per stage
  // Fragments of k-step kq of the stage held in slot slot_idx: A fragment tm (two transposing
  // reads), B fragment tn (one 16-byte read).
  auto read_a = [&](int slot_idx, int kq, int tm) {
    const char* As = lds + slot_idx * SLOT;
    if constexpr (AT) {   // one plain 16-byte read, as for B: row lane%32, k-chunk 2 kq + lane/32
      const int row = wm * WTM + tm * 32 + (lane & 31);
      const int kc = 2 * kq + (lane >> 5);
      return *reinterpret_cast<const bf16x8*>(As + row * COLB + ((kc ^ b_swz) << 4));
    }
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
    return __builtin_bit_cast(bf16x8, w);
  };
  auto read_b = [&](int slot_idx, int kq, int tn) {
    const char* Bs = lds + slot_idx * SLOT + A_BYTES;
    if constexpr (BT) {   // two transposing reads, as for a column-major A: column lane%32
      const int hi = (wn * WTN + tn * 32) >> 3;
      v4i16 half[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int k = kq * 16 + 8 * (g >> 1) + 4 * h + (j >> 2);
        const int byte = k * B_ROW + (((hi ^ swz_a<B_ROW>(k)) + a_lo) << 4) + a_sub;
        half[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS v4i16*)(Bs + byte));
      }
      const u32x4 w = {(uint32_t)(uint16_t)half[0][0] | ((uint32_t)(uint16_t)half[0][1] << 16),
                       (uint32_t)(uint16_t)half[0][2] | ((uint32_t)(uint16_t)half[0][3] << 16),
                       (uint32_t)(uint16_t)half[1][0] | ((uint32_t)(uint16_t)half[1][1] << 16),
                       (uint32_t)(uint16_t)half[1][2] | ((uint32_t)(uint16_t)half[1][3] << 16)};
      return __builtin_bit_cast(bf16x8, w);
    }
    const int col = wn * WTN + tn * 32 + (lane & 31);
    const int kc = 2 * kq + (lane >> 5);
    return *reinterpret_cast<const bf16x8*>(Bs + col * COLB + ((kc ^ b_swz) << 4));
  };
  auto read_frags = [&](int slot_idx, int kq, bf16x8 (&af)[TM], bf16x8 (&bfr)[TN]) {
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) af[tm] = read_a(slot_idx, kq, tm);
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) bfr[tn] = read_b(slot_idx, kq, tn);
  };
  auto mfmas = [&](const bf16x8 (&af)[TM], const bf16x8 (&bfr)[TN]) {
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
        acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[tm], bfr[tn], acc[tm][tn], 0, 0, 0);
  };
  // One stage's MFMAs with the fragments double-buffered: k-step kq + 1's reads are issued
  // before k-step kq's MFMAs (a scheduling barrier keeps the compiler from sinking them to their
  // use), so the MFMAs do not wait on LDS latency at each k-step.
  auto compute = [&](int slot_idx) {
    bf16x8 af[2][TM], bfr[2][TN];
    read_frags(slot_idx, 0, af[0], bfr[0]);
#pragma unroll
    for (int kq = 0; kq < KQ; ++kq) {
      if (kq + 1 < KQ) read_frags(slot_idx, kq + 1, af[(kq + 1) & 1], bfr[(kq + 1) & 1]);
      __builtin_amdgcn_sched_barrier(0);   // keep the reads ahead of the MFMAs
      mfmas(af[kq & 1], bfr[kq & 1]);
    }
  };
  // Wait until this wave's loads of the stage `ahead` stages before its newest issued one landed.
  // (ahead is at most SLOTS - 2.)
  auto wait_loads = [&](int32_t ahead) {
    if (ahead >= 3)
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(3 * LPS));
    else if (ahead == 2)
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * LPS));
    else if (ahead == 1)
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(LPS));
    else
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
  };
  static_assert(SLOTS - 2 <= 3 && 3 * LPS <= 63, "vmcnt immediates cover the ring");
  auto lmin = [](int32_t a, int32_t b) { return a < b ? a : b; };

  const int32_t pre = stages < SLOTS - 1 ? stages : SLOTS - 1;
  for (int32_t s = 0; s < pre; ++s) {
    if constexpr (SCHED == 0) issue_block(); else issue();
  }
  // The register epilogue (bf16 C, beta = 0, whole stage lists) takes accumulators that start at
  // the bias: the products accumulate onto it, the epilogue spends no addition per element on it,
  // and the bias loads overlap the first stage's copies instead of opening the epilogue.
  if (p.c_bf16 && p.beta == 0.0f && p.split <= 1 && (p.flags & TPP_EPI_BIAS)) {
    f32x4 b4[TM][4];
    load_bias4<TM, FULL>(p, in, tc.row0 + wm * WTM, lane, b4);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[tm][tn][v] = b4[tm][v >> 2][v & 3];
  }
  // The 16-wave instance with A stored transposed (one 16-byte fragment read per A fragment), on
  // complete tiles of an aligned strided grid, defers each stage's last k-step past the next
  // barrier: its fragments are read into registers
  // before the barrier, and its MFMAs are issued right after it, ahead of the wave's copies of the
  // stage it refills and of the next stage's fragment reads, so every SIMD has MFMAs to run while
  // the compute unit accepts the copies.  The k-steps still accumulate in order (stage s - 1's
  // last k-step before stage s's first).  With A in its own layout (two transposing reads per
  // fragment), on other batch kinds and on partial tiles, the held fragments push the kernel
  // past its 128 registers into scratch; the 128x128 tile measured slower with it.
  constexpr bool SKEW =
      SCHED == 0 && NW == 16 && AT && !BT && FULL && KIND == TPP_BR_STRIDE && ALIGNED;
  if constexpr (SKEW) {
    bf16x8 af[2][TM], bfr[2][TN];
    for (int32_t s = 0; s < stages; ++s) {
      wait_loads(lmin(stages - 1 - s, SLOTS - 2));
      lds_barrier();
      if (s > 0) mfmas(af[(KQ - 1) & 1], bfr[(KQ - 1) & 1]);   // stage s - 1, last k-step
      __builtin_amdgcn_sched_barrier(0);
      if (s + SLOTS - 1 < stages) issue_block();   // stage s + SLOTS - 1 refills the slot of s - 1
      const int slot = s % SLOTS;
      read_frags(slot, 0, af[0], bfr[0]);
#pragma unroll
      for (int kq = 0; kq + 1 < KQ; ++kq) {
        read_frags(slot, kq + 1, af[(kq + 1) & 1], bfr[(kq + 1) & 1]);
        __builtin_amdgcn_sched_barrier(0);   // keep the reads ahead of the MFMAs
        mfmas(af[kq & 1], bfr[kq & 1]);
      }
    }
    if (stages > 0) mfmas(af[(KQ - 1) & 1], bfr[(KQ - 1) & 1]);
  } else if constexpr (SCHED == 0) {
    for (int32_t s = 0; s < stages; ++s) {
      // This wave's loads of stage s are done once at most the later stages' loads are pending;
      // the barrier then publishes every wave's stage s and retires everyone's reads of s - 1.
      wait_loads(lmin(stages - 1 - s, SLOTS - 2));
      lds_barrier();
      if (s + SLOTS - 1 < stages) issue_block();   // stage s + SLOTS - 1 refills the slot of s - 1
      compute(s % SLOTS);
    }
  } else if constexpr (SCHED == 1) {
    // Ping-pong: waves 0-3 (one per SIMD) lead, waves 4-7 lag by one half-period.  Each stage is
    // a memory half (fragment reads of the stage, global->LDS issue of stage s + SLOTS - 1) and a compute
    // half (the stage's MFMAs on registers); while one wave of a SIMD computes, the other reads,
    // so every barrier finds the next MFMA phase's operands already in registers.
    //   barrier j:  leading waves end M(j/2) (j even) or C(j/2) (j odd);
    //               lagging waves end C(j/2 - 1) (j even, the first one is the offset barrier) or
    //               M(j/2) (j odd).
    // Stage s + 1 must have landed before barrier 2s + 1, the last barrier before anyone reads it:
    // the leading waves wait at the end of C(s), the lagging ones at the end of M(s).
    static_assert(NW == 8, "two groups of four waves");
    const bool lead = wave < 4;
    wait_loads(lmin(stages - 1, SLOTS - 2));   // stage 0, before anyone reads it
    lds_barrier();
    if (!lead) lds_barrier();
    bf16x8 af[KQ][TM], bfr[KQ][TN];
    for (int32_t s = 0; s < stages; ++s) {
      const int32_t later = lmin(stages - 2 - s, SLOTS - 2);
      // Memory half: the fragment reads of stage s with stage s + SLOTS - 1's wave-loads spread among
      // them, so that the LDS and the load unit work at the same time.
      // (Load indices are compile-time constants: a runtime index would put the per-lane offset
      // arrays in scratch memory.)
      constexpr int SPOTS = KQ * TM / 2;   // after every second A fragment
      const bool more = s + SLOTS - 1 < stages;
      if (more) stage_begin();
#pragma unroll
      for (int kq = 0; kq < KQ; ++kq) {
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) {
          af[kq][tm] = read_a(s % SLOTS, kq, tm);
          const int spot = kq * (TM / 2) + (tm >> 1);
          if ((tm & 1) && spot < LPS && more) issue_load(spot);
        }
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) bfr[kq][tn] = read_b(s % SLOTS, kq, tn);
      }
      if (more) {
#pragma unroll
        for (int r = SPOTS; r < LPS; ++r) issue_load(r);
        stage_end();
      }
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
  if (p.split > 1) {
    // the chunk's partial tile: f32x16 (tm, tn) accumulators of each lane, lane-contiguous
    float* w = p.ws + (size_t)(chunk * p.total_tiles + tile_bid) * (BM * BN) +
               (size_t)wave * (TM * TN * 1024) + lane * 16;
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          gst<f32x4>(w + (tm * TN + tn) * 1024 + 4 * q,
                     (f32x4){acc[tm][tn][4 * q], acc[tm][tn][4 * q + 1], acc[tm][tn][4 * q + 2],
                             acc[tm][tn][4 * q + 3]});
    return;
  }
  if (p.c_bf16 && p.beta == 0.0f)
    epilogue_bf16<WTM, WTN, TM, TN, FULL>(p, in, tc, wm, wn, lane, wave, lds, acc);
  else
    epilogue_via_lds<WTM, WTN, TM, TN, FULL>(p, in, tc, wm, wn, lane, wave,
                                            reinterpret_cast<float*>(lds), acc);
}

// The kernel's name as the profiler prints it (template arguments in declaration order).
template <int BM, int BN, int WM, int WN, bool FULL, int KIND, bool ALIGNED, int PP, int BKT,
          int SL, bool AT, bool BT>
std::string dl_kernel_name() {
  const auto tf = [](bool v) { return v ? "true" : "false"; };
  char buf[160];
  std::snprintf(buf, sizeof buf,
                "brgemm_bf16_dl_kernel<%d, %d, %d, %d, %s, %d, %s, %d, %d, %d, %s, %s>", BM, BN, WM,
                WN, tf(FULL), KIND, tf(ALIGNED), PP, BKT, SL, tf(AT), tf(BT));
  return buf;
}

template <int BM, int BN, int WM, int WN, bool FULL, int KIND, bool ALIGNED, int PP, int BKT,
          int SL, bool AT, bool BT>
void launch_dl_kk(const BrgemmParams& p, dim3 grid, hipStream_t stream, std::string* name_out) {
  if (name_out) {
    *name_out = dl_kernel_name<BM, BN, WM, WN, FULL, KIND, ALIGNED, PP, BKT, SL, AT, BT>();
    return;
  }
  hipLaunchKernelGGL(
      (brgemm_bf16_dl_kernel<BM, BN, WM, WN, FULL, KIND, ALIGNED, PP, BKT, SL, AT, BT>), grid,
      dim3(64 * WM * WN), 0, stream, p);
}

template <int BM, int BN, int WM, int WN, bool FULL, int KIND, int PP, int BKT, int SL, bool AT,
          bool BT>
void launch_dl_k(const BrgemmParams& p, dim3 grid, hipStream_t stream, std::string* name_out) {
  if constexpr (KIND == TPP_BR_STRIDE) {
    if (p.aligned) {
      launch_dl_kk<BM, BN, WM, WN, FULL, KIND, true, PP, BKT, SL, AT, BT>(p, grid, stream,
                                                                         name_out);
      return;
    }
  }
  launch_dl_kk<BM, BN, WM, WN, FULL, KIND, false, PP, BKT, SL, AT, BT>(p, grid, stream, name_out);
}

template <int BM, int BN, int WM, int WN, int PP = 0, int BKT = 32, int SL = 0, bool AT = false,
          bool BT = false>
void launch_dl(const BrgemmParams& p, bool full, dim3 grid, hipStream_t stream,
               std::string* name_out) {
  switch (p.kind) {
    case TPP_BR_STRIDE:
      full ? launch_dl_k<BM, BN, WM, WN, true, TPP_BR_STRIDE, PP, BKT, SL, AT, BT>(p, grid, stream, name_out)
           : launch_dl_k<BM, BN, WM, WN, false, TPP_BR_STRIDE, PP, BKT, SL, AT, BT>(p, grid, stream, name_out);
      break;
    case TPP_BR_OFFSET:
      full ? launch_dl_k<BM, BN, WM, WN, true, TPP_BR_OFFSET, PP, BKT, SL, AT, BT>(p, grid, stream, name_out)
           : launch_dl_k<BM, BN, WM, WN, false, TPP_BR_OFFSET, PP, BKT, SL, AT, BT>(p, grid, stream, name_out);
      break;
    default:
      full ? launch_dl_k<BM, BN, WM, WN, true, TPP_BR_ADDRESS, PP, BKT, SL, AT, BT>(p, grid, stream, name_out)
           : launch_dl_k<BM, BN, WM, WN, false, TPP_BR_ADDRESS, PP, BKT, SL, AT, BT>(p, grid, stream, name_out);
      break;
  }
}

}  // namespace
}  // namespace tpp
