// brgemm_dl_kernels.hip -- dispatch over the direct-to-LDS bf16 BRGEMM instances.
//
// The kernel template is in brgemm_dl_impl.h; its instances are compiled in parts from
// brgemm_dl_inst.hip (one object per tile and operand layout, and one for the 32-k stages).
#include <hip/hip_runtime.h>

#include "internal.h"

namespace tpp {

// The parts (brgemm_dl_inst.hip).
hipError_t launch_dl_part_bk32(const BrgemmParams& p, int32_t id, bool full, dim3 grid,
                               hipStream_t stream, std::string* name_out);
#define DL_PART_DECL(t, a, b)                                                                 \
  hipError_t launch_dl64_t##t##_a##a##_b##b(const BrgemmParams& p, bool full, dim3 grid,      \
                                            hipStream_t stream, std::string* name_out);
#define DL_PART_DECL_ALL(t) DL_PART_DECL(t, 0, 0) DL_PART_DECL(t, 1, 0) DL_PART_DECL(t, 0, 1) \
  DL_PART_DECL(t, 1, 1)
DL_PART_DECL_ALL(256)
DL_PART_DECL_ALL(128)
DL_PART_DECL_ALL(64)
#undef DL_PART_DECL_ALL
#undef DL_PART_DECL

// The 64-k stage instance of one tile with each combination of transposed operands.
#define DL_PART_PICK(t)                                                                        \
  (p.a_trans ? (p.b_trans ? launch_dl64_t##t##_a1_b1 : launch_dl64_t##t##_a1_b0)             \
             : (p.b_trans ? launch_dl64_t##t##_a0_b1 : launch_dl64_t##t##_a0_b0))

bool dl_wave_grid(int32_t id, int& waves_m, int& waves_n) {
  switch (id) {
    case K_BF16_DL_256x256: waves_m = 2; waves_n = 4; return true;
    case K_BF16_PP_256x256: waves_m = 4; waves_n = 2; return true;
    case K_BF16_DL64K_256x256: waves_m = 4; waves_n = 4; return true;
    case K_BF16_DL_128x128:
    case K_BF16_DL_64x64:
    case K_BF16_DL64K_128x128:
    case K_BF16_DL64K_64x64: waves_m = 2; waves_n = 2; return true;
    default: return false;
  }
}

hipError_t launch_brgemm_dl(const BrgemmParams& p, int32_t id, bool full, dim3 grid,
                            hipStream_t stream, std::string* name_out) {
  // transposed operands only on the 64-k instances (the host never picks another for them)
  if ((p.a_trans || p.b_trans) && id != K_BF16_DL64K_256x256 && id != K_BF16_DL64K_128x128 &&
      id != K_BF16_DL64K_64x64)
    return hipErrorInvalidValue;
  switch (id) {
    case K_BF16_DL_256x256:
    case K_BF16_DL_128x128:
    case K_BF16_DL_64x64:
    case K_BF16_PP_256x256: return launch_dl_part_bk32(p, id, full, grid, stream, name_out);
    case K_BF16_DL64K_256x256: return DL_PART_PICK(256)(p, full, grid, stream, name_out);
    case K_BF16_DL64K_128x128: return DL_PART_PICK(128)(p, full, grid, stream, name_out);
    case K_BF16_DL64K_64x64: return DL_PART_PICK(64)(p, full, grid, stream, name_out);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace tpp
