/*
 * tpp_embedding.h -- C ABI of the sparse embedding gather-reduce of the MI355X (gfx950) TPP
 * library.
 *
 * Tensor Processing Primitives (arXiv 2104.05755), Alg. 5 (sparse embedding kernel, Sec. 5.1):
 * the lookups of a multi-hot vector a into an embedding table W (M rows of E entries) give the
 * output row o^T = a^T x W, i.e. the sum of the table rows the bag lists.  The paper builds it
 * from a gather TPP and a reduce TPP fused in registers; here one kernel gathers each listed row
 * and accumulates it in fp32 registers before a single store.
 *
 * Conventions are those of tpp_brgemm.h: caller-owned DEVICE memory, element counts for strides,
 * asynchronous on `stream` (a hipStream_t as void*, NULL = the default stream), a tpp_status
 * result and tpp_last_error_message() for the detail.
 */
#ifndef TPP_EMBEDDING_H
#define TPP_EMBEDDING_H

#include "tpp_brgemm.h"

#ifdef __cplusplus
extern "C" {
#endif

/* out[b * ldo + e] = sum over j in [begin[b], begin[b+1]) of W[idx[j] * ldw + e],
 * for b < n_bags and e < E.
 *   W:      the table, M rows of E entries of w_type (TPP_DT_F32 or TPP_DT_BF16), row r at
 *           W + r * ldw (ldw >= E).
 *   d_begin: device int64[n_bags + 1], the bags as a CSR list over d_idx (non-decreasing; a
 *           decreasing pair is an empty bag).  d_idx: device int64 row indices, begin[n_bags] of
 *           them.  A row listed twice counts twice (the loop of Alg. 5 over the listed indices).
 *   out:    n_bags rows of E entries of out_type (TPP_DT_F32 or TPP_DT_BF16, rounded to nearest
 *           even once, from the fp32 sums), row b at out + b * ldo (ldo >= E).  An empty bag
 *           gives a row of zeros.
 * Accumulation is fp32 in an order that depends only on the bag's list (results do not vary
 * between runs).  Indices outside [0, M) are skipped: they add nothing and the table is never
 * read outside its M rows.  n_bags == 0 is a no-op.
 * Errors: INVALID_ARG for M < 0, E <= 0, n_bags < 0, ldw < E, ldo < E, an unknown datatype, or a
 * NULL pointer when there is work; UNSUPPORTED when one launch would need more than 2^31 - 1
 * workgroups; HIP if the launch fails. */
tpp_status tpp_embedding_bag(int64_t M, int32_t E, int32_t w_type, const void* W, int64_t ldw,
                             int64_t n_bags, const int64_t* d_begin, const int64_t* d_idx,
                             int32_t out_type, void* out, int64_t ldo, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* TPP_EMBEDDING_H */
