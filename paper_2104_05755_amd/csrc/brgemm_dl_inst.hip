// brgemm_dl_inst.hip -- one part of the direct-to-LDS kernel instances (brgemm_dl_impl.h).
//
// The build compiles this file several times, each with one choice of the macros below, so that
// the instances compile in parallel:
//   DL_BK32                      the 32-k stage instances (ids 5-8), every batch kind;
//   DL_TILE = 256 | 128 | 64,
//   DL_AT, DL_BT = 0 | 1         the 64-k stage instance of that tile with A / B stored transposed.
#include "brgemm_dl_impl.h"

namespace tpp {

#if defined(DL_BK32)
hipError_t launch_dl_part_bk32(const BrgemmParams& p, int32_t id, bool full, dim3 grid,
                               hipStream_t stream, std::string* name_out) {
  switch (id) {
    case K_BF16_DL_256x256: launch_dl<256, 256, 2, 4>(p, full, grid, stream, name_out); break;
    case K_BF16_DL_128x128: launch_dl<128, 128, 2, 2>(p, full, grid, stream, name_out); break;
    case K_BF16_DL_64x64: launch_dl<64, 64, 2, 2>(p, full, grid, stream, name_out); break;
    case K_BF16_PP_256x256: launch_dl<256, 256, 4, 2, 1>(p, full, grid, stream, name_out); break;
    default: return hipErrorInvalidValue;
  }
  return name_out ? hipSuccess : hipGetLastError();
}
#elif defined(DL_TILE) && defined(DL_AT) && defined(DL_BT)
#define DL_CAT2(a, b, c, d) launch_dl64_t##a##_a##b##_b##c##d
#define DL_CAT(a, b, c) DL_CAT2(a, b, c, )
hipError_t DL_CAT(DL_TILE, DL_AT, DL_BT)(const BrgemmParams& p, bool full, dim3 grid,
                                         hipStream_t stream, std::string* name_out) {
#if DL_TILE == 256
  launch_dl<256, 256, 4, 4, 0, 64, 0, DL_AT != 0, DL_BT != 0>(p, full, grid, stream, name_out);
#elif DL_TILE == 128
  launch_dl<128, 128, 2, 2, 0, 64, 0, DL_AT != 0, DL_BT != 0>(p, full, grid, stream, name_out);
#elif DL_TILE == 64
  launch_dl<64, 64, 2, 2, 0, 64, 0, DL_AT != 0, DL_BT != 0>(p, full, grid, stream, name_out);
#else
#error "DL_TILE must be 256, 128 or 64"
#endif
  return name_out ? hipSuccess : hipGetLastError();
}
#else
#error "compile with DL_BK32, or with DL_TILE, DL_AT and DL_BT"
#endif

}  // namespace tpp
