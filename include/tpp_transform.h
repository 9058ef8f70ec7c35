/*
 * tpp_transform.h -- C ABI of the Transform TPP of the MI355X (gfx950) TPP library.
 *
 * Tensor Processing Primitives (arXiv 2104.05755), Table 1 and Sec. 3.1: a unary TPP that
 * rearranges the entries of a 2D input as a flag selects -- the matrix Transpose, VNNI
 * formatting, and VNNI to VNNI-transpose.  VNNI is the layout of Sec. 3.2.2: a logical tensor
 * [D1][D0] (D0 innermost) stored as [D1/alpha][D0][alpha], i.e. alpha consecutive D1 entries
 * next to each other; for a column-major m x n block D0 is the row index (m) and D1 the column
 * index (n), which is the [K/alpha][M][alpha] reformatting of an M x K operand.  On MI355X it is
 * the operand pre-format step upstream of the batch-reduce GEMM (the MFMA reads 8 consecutive k
 * per lane) and the transpose a backward pass needs (W^T).
 *
 * Conventions are those of tpp_brgemm.h: column-major blocks with leading dimensions counted in
 * elements, caller-owned DEVICE memory, asynchronous on `stream` (a hipStream_t as void*, NULL =
 * the default stream), a tpp_status result and tpp_last_error_message() for the detail.
 */
#ifndef TPP_TRANSFORM_H
#define TPP_TRANSFORM_H

#include "tpp_brgemm.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TPP_TR_TRANSPOSE = 0,        /* matrix transpose                                             */
  TPP_TR_VNNI = 1,             /* [D1][D0] -> [D1/alpha][D0][alpha]                             */
  TPP_TR_VNNI_TO_VNNI_T = 2    /* [D1/alpha][D0][alpha] -> [D0/alpha][D1][alpha]                */
} tpp_transform_kind;

/* Transform TPP (Table 1; Sec. 3.1).  The input is a logical m x n tensor of `dtype`
 * (TPP_DT_F32 or TPP_DT_BF16); entries are moved bit for bit, nothing is computed.
 *   TPP_TR_TRANSPOSE       in: entry (r, c) at in + r + c*ld_in (ld_in >= m).
 *                          out: the n x m transpose, entry (c, r) at out + c + r*ld_out
 *                          (ld_out >= n).  alpha is ignored.
 *   TPP_TR_VNNI            in: as for TRANSPOSE.  out: column c = alpha*g + a of the input
 *                          goes to group g, entry (r, c) at out + g*ld_out + r*alpha + a
 *                          (ld_out >= m*alpha: the group stride).  ceil(n/alpha) groups; a
 *                          last group with fewer than alpha columns is completed with zeros.
 *   TPP_TR_VNNI_TO_VNNI_T  in: an m x n tensor in that layout, entry (r, c) at
 *                          in + (c/alpha)*ld_in + r*alpha + c%alpha (ld_in >= m*alpha).
 *                          out: its n x m transpose in the same layout with the same alpha,
 *                          entry (c, r) at out + (r/alpha)*ld_out + c*alpha + r%alpha
 *                          (ld_out >= n*alpha); ceil(m/alpha) groups, the last completed with
 *                          zeros when m % alpha != 0.
 * alpha: 1, 2 or 4 for the VNNI kinds (2 is the 16-bit VNNI of Sec. 3.2.2).  Output positions
 * outside the extents above (gaps when ld_out exceeds them) are not written.  m == 0 or n == 0
 * is a no-op.  in and out must not overlap.
 * Errors: INVALID_ARG for an unknown kind or dtype, m or n < 0, alpha not in {1, 2, 4} for a
 * VNNI kind, a leading dimension below its bound, or a NULL pointer when there is work;
 * UNSUPPORTED when the tile count of one launch would exceed 2^31 - 1; HIP if the launch fails. */
tpp_status tpp_transform(int32_t kind, int32_t m, int32_t n, int64_t ld_in, int64_t ld_out,
                         int32_t dtype, int32_t alpha, const void* in, void* out, void* stream);

/* G Transform TPP calls in one launch (the loop Alg. 6 writes around a TPP; e.g. the transpose
 * of every 64 x 64 block of a blocked weight tensor that the backward pass multiplies by):
 * call g transforms the block at in + g * in_stride into out + g * out_stride (elements), each
 * as tpp_transform does with the arguments above.  G == 0 is a no-op.  No output block may
 * overlap an input block or another output block.
 * Errors: those of tpp_transform, plus INVALID_ARG for G, in_stride or out_stride < 0. */
tpp_status tpp_transform_batched(int32_t kind, int32_t m, int32_t n, int64_t ld_in,
                                 int64_t ld_out, int32_t dtype, int32_t alpha, const void* in,
                                 int64_t in_stride, void* out, int64_t out_stride, int64_t G,
                                 void* stream);

#ifdef __cplusplus
}
#endif
#endif /* TPP_TRANSFORM_H */
