// internal.h -- structures shared by the C-ABI front end and the HIP kernels (not installed).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

#include "tpp_brgemm.h"
#include "tpp_embedding.h"
#include "tpp_equation.h"
#include "tpp_transform.h"

namespace tpp {

// Everything one batched BRGEMM launch needs, resolved on the host and passed by value.
struct BrgemmParams {
  const void* a;
  const void* b;
  void* c;
  const float* bias;
  int32_t m, n, k;
  int64_t lda, ldb, ldc;
  float beta;
  uint32_t flags;
  int32_t c_bf16;  // 1: C is bf16, 0: C is fp32
  int32_t aligned; // host-verified: every A_i / B_i base is 16-byte aligned (stride kind)
  int32_t a_trans; // 1: A_i stored transposed (k contiguous per row, lda >= k)
  int32_t b_trans; // 1: B_i stored transposed (n contiguous per k-row, ldb >= n)
  int32_t kind;    // tpp_br_kind
  int64_t count;
  int64_t stride_a, stride_b;
  const int64_t* offs_a;
  const int64_t* offs_b;
  const int64_t* begin;
  const void* const* ptrs_a;
  const void* const* ptrs_b;
  // Instance grid.  fused = 1: the gm x gn instances of a strided grid are laid side by side
  // into one virtual (gm*m) x (gn*n) C, tiled as one group (tiles may span instances).
  // fused = 0: G separate instances, each its own m x n virtual C and tile group; their bases
  // come from the strided formula (grid_form = 1) or from the offset arrays (grid_form = 0).
  int32_t fused;
  int32_t grid_form;
  int64_t gm, gn;
  int64_t a_step_m, b_step_n, c_step_m, c_step_n, bias_step_m;
  const int64_t* a_off;
  const int64_t* b_off;
  const int64_t* c_off;
  const int64_t* bias_off;
  // Tiling, filled by the launcher.
  int32_t vrows, vcols;      // virtual C extent of one tile group
  int32_t tiles_m, tiles_n;  // tiles per group
  int64_t groups;            // 1 (strided) or G (explicit)
  int64_t total_tiles;
  // Split over the pair list (grids too small to fill the GPU): split > 1 chunks of each
  // instance's pairs (fp32 kernel) or stages (direct-to-LDS kernels) are reduced by separate
  // workgroups into ws (split x total_tiles fp32 tiles), then summed in chunk order by a
  // finishing kernel that applies the epilogue.
  int32_t split;             // 1: no split
  float* ws;
  // Tensor of C's type and layout read or written by the back-propagation epilogue bits.
  void* aux;
};

// Epilogue bits that use the aux tensor.
constexpr uint32_t EPI_AUX_MASK = TPP_EPI_RELU_INV | TPP_EPI_GELU_TANH_INV | TPP_EPI_SAVE_PREACT;

// Kernel instances of the bf16 family (tile shape + load path) and the fp32 kernel.
enum KernelId : int32_t {
  K_BF16_256x256 = 0,   // 8 waves, 128x64 per wave, 16-byte loads
  K_BF16_128x128 = 1,   // 4 waves, 64x64 per wave, 16-byte loads (two workgroups per CU)
  K_BF16_64x64 = 2,     // 4 waves, 32x32 per wave, 16-byte loads
  K_BF16_GENERIC = 3,   // 64x64, element loads with full bounds checks (any shape / alignment)
  K_F32_GENERIC = 4,    // 64x64 fp32 MFMA, element loads with full bounds checks
  K_BF16_DL_256x256 = 5,  // direct global->LDS staging, 8 waves (k a multiple of 32)
  K_BF16_DL_128x128 = 6,  // direct global->LDS staging, 4 waves
  K_BF16_DL_64x64 = 7,    // direct global->LDS staging, 4 waves
  K_BF16_PP_256x256 = 8,  // direct global->LDS staging, 8 waves in two alternating groups
  K_BF16_DL64K_256x256 = 9,  // direct global->LDS staging, 16 waves, 64-k stages (k % 64 == 0)
  K_BF16_DL64K_128x128 = 10, // as 9, 128x128 tiles, 4 waves (two workgroups per CU)
  K_BF16_DL64K_64x64 = 11,   // as 9, 64x64 tiles, 4 waves
  K_COUNT = 12
};

const char* kernel_name(int32_t id);
int kernel_tile_m(int32_t id);   // tile rows of kernel instance id
// fp32 workspace floats a split launch of the fp32 kernel needs (split x tiles x 64 x 64).
int64_t f32_split_ws_floats(int32_t split, int64_t total_tiles);
int kernel_tile_n(int32_t id);   // tile columns
int kernel_k_step(int32_t id);   // k granularity the instance needs (1 = any k)

// Whether kernel `id` runs every tile of p complete (no row, column or k tail: the FULL
// instances); p.vrows / p.vcols / p.k filled.
bool kernel_full(int32_t id, const BrgemmParams& p);
// Fill the tiling fields of p for kernel `id` and launch on `stream`.  With name_out set nothing
// is launched: the same dispatch writes the names of the kernels it would launch, as the
// profiler names them ("brgemm_bf16_dl_kernel<256, 256, 4, 4, true, 0, true, ...>", and
// " + <finishing kernel>" for a split).
hipError_t launch_brgemm(BrgemmParams& p, int32_t id, hipStream_t stream,
                         std::string* name_out = nullptr);
// The direct-to-LDS instances (brgemm_dl_kernels.hip); p's tiling fields already filled.
// With p.split > 1, grid covers total_tiles * split workgroups writing partial tiles to p.ws.
hipError_t launch_brgemm_dl(const BrgemmParams& p, int32_t id, bool full, dim3 grid,
                            hipStream_t stream, std::string* name_out = nullptr);
// Wave layout (waves along m, along n) of a direct-to-LDS instance; false for other ids.
bool dl_wave_grid(int32_t id, int& waves_m, int& waves_n);

// Reduce TPP launcher; `work` is a device buffer of `work_floats` floats for partial results.
struct ReduceParams {
  const void* in;
  int32_t m, n;
  int64_t ld;
  int32_t in_bf16;
  int32_t op;
  uint32_t flags;
  float* out_x;
  float* out_x2;
  // Batch of G calls: call g reads in + g * in_stride (elements), writes outputs g * out_stride
  // floats on.
  int64_t G;
  int64_t in_stride;
  int64_t out_stride;
};
// Number of floats of work space a reduce of this shape (and batch) needs: 0 if none, -1 if one
// of its launches would need more than 2^31 - 1 workgroups.
int64_t reduce_work_floats(const ReduceParams& p);
hipError_t launch_reduce(const ReduceParams& p, float* work, hipStream_t stream);

// Transform TPP launcher (transform_kernels.hip).  kind: 0 transpose, 1 VNNI, 2 VNNI to
// VNNI-transpose; es: entry bytes (2 or 4); vec: both operands 16-byte aligned with leading
// dimensions of whole 16-byte units (the vector paths).  tiles_m is filled by the launcher.
// hipErrorInvalidConfiguration when one launch would need more than 2^31 - 1 workgroups.
struct TransformParams {
  const void* in;
  void* out;
  int32_t kind, m, n;
  int64_t ld_in, ld_out;
  int32_t es, alpha;
  int32_t vec;
  int64_t tiles_m;
  // Batch of G calls: call g reads in + g * in_stride and writes out + g * out_stride (elements).
  int64_t G;
  int64_t in_stride;
  int64_t out_stride;
};
hipError_t launch_transform(TransformParams& p, hipStream_t stream);

// Embedding gather-reduce launcher (embedding_kernels.hip).  hipErrorInvalidConfiguration when
// one launch would need more than 2^31 - 1 workgroups.
struct EmbeddingParams {
  int64_t M;
  int32_t E;
  int32_t w_bf16, out_bf16;
  const void* W;
  int64_t ldw;
  int64_t n_bags;
  const int64_t* begin;
  const int64_t* idx;
  void* out;
  int64_t ldo;
};
hipError_t launch_embedding(const EmbeddingParams& p, hipStream_t stream);

// TPP matrix equations (equation.hip).  The planner of Alg. 3 / Alg. 4 runs on the host; a
// compiled program lists the internal nodes in timestamp order, each with its operation, the
// temporary it writes and its operands (a temporary id below EQ_LEAF_BASE, or EQ_LEAF_BASE + the
// leaf's argument index), and travels to the executor kernel by value.
constexpr int EQ_MAX_NODES = 64;
constexpr int EQ_MAX_TMPS = 8;
constexpr int EQ_MAX_ARGS = 16;
constexpr int EQ_LEAF_BASE = 16;
// The kernel reads these arrays at indices known only at run time, with scalar loads from the
// kernel-argument block; every element is a whole number of dwords, so every such address stays
// dword aligned (scalar loads drop the low address bits).
struct EqInstr {
  int32_t op, arity, dst;
  int32_t src[3];
};
struct EqArg {
  const void* ptr;
  int64_t ld;
  int32_t bf16, bcast;
};
struct EqProgram {
  int32_t n_instr;
  int32_t result;                       // temporary holding the root's value
  int32_t m, n;
  int64_t ldo;
  void* out;
  int32_t out_bf16, n_args;
  EqInstr instr[EQ_MAX_NODES];
  EqArg arg[EQ_MAX_ARGS];
};
// Layout guards for the scalar-load reads above: every record, and every field the kernel reads
// from a record, sits at a whole-dword offset, and the arrays start on dword boundaries.
static_assert(sizeof(EqInstr) == 24 && sizeof(EqInstr) % 4 == 0, "EqInstr is 6 dwords");
static_assert(offsetof(EqInstr, op) == 0 && offsetof(EqInstr, arity) == 4 &&
                  offsetof(EqInstr, dst) == 8 && offsetof(EqInstr, src) == 12,
              "EqInstr fields on dword boundaries");
static_assert(sizeof(EqArg) == 24 && sizeof(EqArg) % 8 == 0, "EqArg is 3 qwords");
static_assert(offsetof(EqArg, ptr) == 0 && offsetof(EqArg, ld) == 8 &&
                  offsetof(EqArg, bf16) == 16 && offsetof(EqArg, bcast) == 20,
              "EqArg fields on dword boundaries");
static_assert(offsetof(EqProgram, instr) % 8 == 0 && offsetof(EqProgram, arg) % 8 == 0 &&
                  offsetof(EqProgram, ldo) % 8 == 0 && offsetof(EqProgram, out) % 8 == 0,
              "EqProgram arrays and 64-bit fields 8-byte aligned");
static_assert(sizeof(EqProgram) % 8 == 0, "EqProgram a whole number of qwords");
// nullptr on success, else what is wrong with the tree.
const char* equation_plan(const tpp_eq_node* nodes, int32_t n_nodes, int32_t root,
                          tpp_eq_plan_node* plan, int32_t* n_tmps);
// The program of a planned tree (a root that is a leaf becomes one IDENTITY instruction);
// nullptr on success, else what is wrong.  *too_many_tmps is set when the plan needs more than
// EQ_MAX_TMPS temporaries.
const char* equation_compile(const tpp_eq_node* nodes, int32_t n_nodes, int32_t root,
                             EqProgram& prog, bool* too_many_tmps);
hipError_t launch_equation(const EqProgram& prog, hipStream_t stream);

}  // namespace tpp
