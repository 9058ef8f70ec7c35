/*
 * tpp_brgemm.h -- C ABI of the MI355X (gfx950) batch-reduce GEMM TPP library.
 *
 * Tensor Processing Primitives (arXiv 2104.05755).  The library exposes the paper's two-step
 * usage (Sec. 3: a dispatch call that prepares a kernel for a problem description and returns a
 * handle, and a call that runs it) for two TPPs:
 *
 *   - the ternary batch-reduce GEMM, Table 3 and Sec. 2.3:
 *         C = beta * C + sum_{i=0}^{count-1} A_i x B_i
 *     with the blocks A_i (m x k) and B_i (k x n) named by one of the three variants of Sec. 2.3
 *     (stride-, offset- or address-based), followed by the unary/binary TPPs fused as its
 *     epilogue (Sec. 2.1 principle 5; Table 2 Add with a column broadcast, Sec. 2.2; Table 1 RELU,
 *     GELU and Identity-with-conversion), applied to the finished C block as Alg. 6 applies its
 *     UNARY:  C = cvt( act( beta * C + sum_i A_i B_i + bias[row] ) );
 *   - the unary Reduce TPP, Table 1 (rows or columns, SUM / MUL / MIN / MAX, of x or x*x).
 * For back-propagation the epilogue also takes Table 1's inverse activations (RELU_inv, GELU_inv)
 * and can keep the forward pre-activation for them, and the Reduce TPP runs as a batch of calls.
 *
 * Conventions for every entry point
 *   - 2D blocks are column-major with a leading dimension: element (r, c) of an m x n block lives
 *     at base + r + c * ld (the storage of Alg. 6's blocked tensors, whose b_m / b_k index is
 *     innermost).  Leading dimensions, strides and offsets count ELEMENTS of the operand's type.
 *   - Tensors, offset arrays, pointer arrays and CSR arrays are caller-owned DEVICE memory
 *     (Sec. 2.1 principle 3: memory-to-memory operations on user memory).  The library never
 *     frees or retains them past the call.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).  Execute calls are
 *     asynchronous on it and never synchronise; device faults surface at the caller's next sync.
 *   - Every call returns a tpp_status; nothing throws or aborts across the ABI.  On error,
 *     tpp_last_error_message() (per thread) says what was wrong.
 *   - Two instances of one call writing overlapping C, or C overlapping an A_i / B_i, is
 *     undefined.  A and B may alias each other (Sec. 2.3).
 */
#ifndef TPP_BRGEMM_H
#define TPP_BRGEMM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TPP_OK = 0,
  TPP_ERR_INVALID_ARG = -1,   /* a size, pointer, flag or handle is not acceptable            */
  TPP_ERR_UNSUPPORTED = -2,   /* well-formed, but a type combination the library does not do */
  TPP_ERR_HIP = -4,           /* a HIP runtime call failed (launch, device query, memory)    */
  TPP_ERR_NO_MEMORY = -5      /* a host or device allocation failed                         */
} tpp_status;

typedef enum { TPP_DT_F32 = 0, TPP_DT_BF16 = 1 } tpp_datatype;

/* The three block-addressing variants of Sec. 2.3. */
typedef enum {
  TPP_BR_STRIDE = 0,   /* address_A_i = address_A_{i-1} + stride_a (elements), A_0 = a        */
  TPP_BR_OFFSET = 1,   /* address_A_i = a + offs_a[i]                                          */
  TPP_BR_ADDRESS = 2   /* address_A_i = ptrs_a[i]                                               */
} tpp_br_kind;

/* Epilogue bits.  RELU and GELU_TANH exclude each other.
 * The last three serve back-propagation (Table 1 pairs RELU and GELU with the inverses that the
 * backward pass uses; Sec. 5.1.6 builds the backward pass of the fully-connected layer from the
 * same TPPs).  They use an AUX tensor of C's type, shaped and laid out exactly as C (same ldc,
 * same per-instance offsets), and need tpp_brgemm_execute_batched_aux:
 *   SAVE_PREACT    with RELU or GELU_TANH: aux = the pre-activation beta C + sum + bias, rounded
 *                  to C's type, written before the activation (the forward call of training).
 *   RELU_INV       C = v * (z > 0 ? 1 : 0), z = aux: the incoming gradient v masked where the
 *                  saved pre-activation was not positive.
 *   GELU_TANH_INV  C = v * gelu'(z), z = aux, gelu' the derivative of the GELU_TANH form.
 * RELU_INV and GELU_TANH_INV exclude each other and RELU, GELU_TANH and SAVE_PREACT; v is
 * beta C + sum (+ bias[row] when BIAS is set). */
enum {
  TPP_EPI_BIAS = 1u << 0,      /* + bias[row]: fp32 column vector of length m, broadcast over n  */
  TPP_EPI_RELU = 1u << 1,      /* x > 0 ? x : +0                                                 */
  TPP_EPI_GELU_TANH = 1u << 2, /* 0.5 x (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3)))                */
  TPP_EPI_RELU_INV = 1u << 3,
  TPP_EPI_GELU_TANH_INV = 1u << 4,
  TPP_EPI_SAVE_PREACT = 1u << 5,
  /* Operand layout, not an epilogue step: every A_i is stored transposed, element (r, p) at
   * A_i + r * lda + p (k contiguous per row, lda >= k), as the Transform TPP's transpose leaves
   * a column-major block (Sec. 3.1; the MFMA reads 8 consecutive k per lane).  Supported for
   * bf16 with k % 64 == 0 and m, lda and every element step a multiple of 8 (direct-to-LDS
   * kernels); any other call returns TPP_ERR_UNSUPPORTED at execute. */
  TPP_LAYOUT_A_TRANS = 1u << 8,
  /* Operand layout: every B_i is stored transposed, element (p, c) at B_i + p * ldb + c (n
   * contiguous per k-row, ldb >= n), the block of Y^T as a column-major Y stores it.  Same
   * support as TPP_LAYOUT_A_TRANS, with n a multiple of 8 as well. */
  TPP_LAYOUT_B_TRANS = 1u << 9
};

/* Problem description: the dispatch-time fields of the TPP (Sec. 2.2: rows, columns, leading
 * dimension and datatype of every 2D operand, plus flags; Sec. 2.3: the batch variant). */
typedef struct {
  int32_t m, n, k;          /* C: m x n, A_i: m x k, B_i: k x n; all > 0                     */
  int64_t lda, ldb, ldc;    /* lda >= m, ldb >= k, ldc >= m                                    */
  int32_t a_type, b_type;   /* tpp_datatype: {F32, F32} or {BF16, BF16}                        */
  int32_t c_type;           /* F32 or BF16: type of C, read when beta != 0 and written        */
  int32_t comp_type;        /* accumulation type: F32 (the only one)                           */
  float beta;               /* 0 => C is not read (NaN in C does not propagate)                */
  int32_t kind;             /* tpp_br_kind                                                     */
  int64_t stride_a;         /* TPP_BR_STRIDE: element stride between consecutive A_i           */
  int64_t stride_b;         /* TPP_BR_STRIDE: element stride between consecutive B_i           */
  uint32_t flags;           /* TPP_EPI_* bits                                                  */
} tpp_brgemm_desc;

/* Opaque kernel handle, owned by the library's process-wide cache (never freed by the caller). */
typedef struct tpp_brgemm_kernel_s* tpp_brgemm_handle;

/* Dispatch (Sec. 3): validate the description and return the cached handle for it; equal
 * descriptions return the same handle.  Host-only: no device work, safe without a GPU.
 * Errors: INVALID_ARG for sizes <= 0, ld too small, RELU together with GELU_TANH, an excluded
 * combination of the back-propagation bits, unknown kind or flag bits, NULL desc/out;
 * UNSUPPORTED for other type combinations. */
tpp_status tpp_brgemm_dispatch(const tpp_brgemm_desc* desc, tpp_brgemm_handle* out);

/* The call API for one BRGEMM (Sec. 2.3 / Alg. 2): C = epi(beta C + sum_{i<count} A_i B_i).
 * count == 0 is valid and gives epi(beta C).  bias (device, m floats) is required iff the
 * handle has TPP_EPI_BIAS.  The kind-specific calls reject a handle of another kind.
 *   stride:  A_i = a + i * stride_a, B_i = b + i * stride_b
 *   offset:  A_i = a + offs_a[i],    B_i = b + offs_b[i]      (device int64 arrays, elements)
 *   address: A_i = ptrs_a[i],        B_i = ptrs_b[i]          (device arrays of device pointers)
 * An fp32 call whose output is only a few 64 x 64 tiles splits the pair list over several
 * workgroups; their partial sums go to a device work buffer the library keeps per GPU and per
 * stream (as tpp_reduce) and are added in a fixed order, so results do not vary between runs.
 * Errors: INVALID_ARG for a NULL handle, count < 0, a NULL pointer the call needs, or a handle
 * with an AUX bit (those run through tpp_brgemm_execute_batched_aux); NO_MEMORY if that work
 * buffer cannot be allocated. */
tpp_status tpp_brgemm_execute_stride(tpp_brgemm_handle h, const void* a, const void* b, void* c,
                                     const float* bias, int64_t count, void* stream);
tpp_status tpp_brgemm_execute_offset(tpp_brgemm_handle h, const void* a, const void* b,
                                     const int64_t* offs_a, const int64_t* offs_b, void* c,
                                     const float* bias, int64_t count, void* stream);
tpp_status tpp_brgemm_execute_address(tpp_brgemm_handle h, const void* const* ptrs_a,
                                      const void* const* ptrs_b, void* c, const float* bias,
                                      int64_t count, void* stream);

/* Strided instance grid: G = gm * gn instances, instance g = gi_m + gm * gi_n, with
 *   A base = a + gi_m * a_step_m       B base = b + gi_n * b_step_n
 *   C base = c + gi_m * c_step_m + gi_n * c_step_n       bias base = bias + gi_m * bias_step_m
 * This is the ib_m / ib_n loop nest of Alg. 6 around its BRGEMM call (all steps in elements). */
typedef struct {
  int64_t gm, gn;
  int64_t a_step_m, b_step_n;
  int64_t c_step_m, c_step_n;
  int64_t bias_step_m;
} tpp_grid_strided;

/* G independent BRGEMMs in one launch: the loops of Alg. 6 (ib_n, ib_m), Alg. 7 (pos) or a
 * convolution's output rows (Sec. 5.1.4) around the call, handed to the GPU as its grid.
 * Instance g computes exactly what one single call computes with its bases moved:
 *   - grid != NULL: the strided form above (gm * gn must equal G); the four offset arrays must
 *     be NULL.
 *   - grid == NULL: the explicit form; d_a_off, d_b_off, d_c_off, d_bias_off are device int64
 *     arrays of G element offsets (any may be NULL, meaning all zeros).
 * Stride and offset kinds: every instance reduces the same `count` pairs relative to its bases
 * (offset kind: d_offs_a / d_offs_b, count entries each).
 * Address kind: instance g reduces pairs d_begin[g] .. d_begin[g+1]-1 of d_ptrs_a / d_ptrs_b
 * (CSR; d_begin has G+1 non-decreasing entries); a, b, d_a_off, d_b_off and count are unused,
 * and the grid moves only C and bias.
 * G == 0 is a no-op.  Errors: INVALID_ARG as for the single calls, plus gm*gn != G, a negative
 * grid field, offset arrays given together with a grid, or a NULL d_begin for the address kind. */
tpp_status tpp_brgemm_execute_batched(tpp_brgemm_handle h, const tpp_grid_strided* grid,
                                      int64_t G, const int64_t* d_a_off, const int64_t* d_b_off,
                                      const int64_t* d_c_off, const int64_t* d_bias_off,
                                      const void* a, const void* b, void* c, const float* bias,
                                      int64_t count, const int64_t* d_offs_a,
                                      const int64_t* d_offs_b, const int64_t* d_begin,
                                      const void* const* d_ptrs_a, const void* const* d_ptrs_b,
                                      void* stream);

/* tpp_brgemm_execute_batched with the AUX tensor of TPP_EPI_SAVE_PREACT, TPP_EPI_RELU_INV and
 * TPP_EPI_GELU_TANH_INV (device, C's type, laid out as C: instance g's block at the offset of its
 * C block).  aux is written (SAVE_PREACT) or only read (the inverses); it must not overlap C or
 * any A_i / B_i.  A handle without AUX bits ignores aux (it may be NULL).
 * Errors: those of tpp_brgemm_execute_batched, plus INVALID_ARG for a NULL aux the handle needs. */
tpp_status tpp_brgemm_execute_batched_aux(tpp_brgemm_handle h, const tpp_grid_strided* grid,
                                          int64_t G, const int64_t* d_a_off,
                                          const int64_t* d_b_off, const int64_t* d_c_off,
                                          const int64_t* d_bias_off, const void* a,
                                          const void* b, void* c, void* aux, const float* bias,
                                          int64_t count, const int64_t* d_offs_a,
                                          const int64_t* d_offs_b, const int64_t* d_begin,
                                          const void* const* d_ptrs_a,
                                          const void* const* d_ptrs_b, void* stream);

/* Handles live in the cache until the process ends; release is a no-op kept for symmetry with
 * dispatch, and is safe on NULL. */
void tpp_brgemm_release(tpp_brgemm_handle h);

/* Human-readable description of a handle's descriptor (types, m / n / k, batch kind, whether
 * the 16-byte load path is open to it).  The kernel instance is chosen per launch, from the grid
 * as well: tpp_brgemm_describe_launch names it.  Writes at most len bytes including the
 * terminating NUL.  Host-only. */
tpp_status tpp_brgemm_describe(tpp_brgemm_handle h, char* buf, size_t len);

/* Environment variables read at each launch, for diagnostics and tests (never needed for
 * correct use): TPP_FORCE_KERNEL=<instance id> takes that kernel instance wherever the shape,
 * alignment and layout allow it; TPP_SPLIT=<n> splits the reduction of every direct-to-LDS
 * launch of the stride or offset kind, and of every fp32 launch of fewer than 128 tiles, into n
 * chunks (capped by the stage or pair count); TPP_LOG prints each launch's instance and split to
 * stderr. */

/* The kernels one tpp_brgemm_execute_batched call with these arguments would launch, named as
 * the profiler names them without namespace and parameter list, e.g.
 * "brgemm_bf16_dl_kernel<256, 256, 4, 4, true, 0, true, 0, 64, 0, false, false>"; a reduction
 * split over several workgroups adds " + " and its finishing kernel.  The choice is the launch
 * path's own (same grid, counts, alignment of a and b); nothing is launched, allocated or read
 * through the pointers, so it is host-only.  G == 0 gives "".  Writes at most len bytes
 * including the terminating NUL.  Errors: those of tpp_brgemm_execute_batched's argument checks,
 * INVALID_ARG for a NULL buf or len == 0. */
tpp_status tpp_brgemm_describe_launch(tpp_brgemm_handle h, const tpp_grid_strided* grid,
                                      int64_t G, const int64_t* d_a_off, const int64_t* d_b_off,
                                      const int64_t* d_c_off, const int64_t* d_bias_off,
                                      const void* a, const void* b, void* c, const float* bias,
                                      int64_t count, const int64_t* d_offs_a,
                                      const int64_t* d_offs_b, const int64_t* d_begin,
                                      const void* const* d_ptrs_a, const void* const* d_ptrs_b,
                                      char* buf, size_t len);

/* Bytes of the per-GPU scratch array of tpp_brgemm_execute_batched_noalloc. */
#define TPP_BRGEMM_NOALLOC_SCRATCH_BYTES (64ll << 20)

/* For callers that cannot allocate device memory (code under HIP graph capture, serving loops,
 * harnesses that forbid hipMalloc): tpp_brgemm_execute_batched without any allocation, device
 * synchronisation or allocating library call.  It computes exactly what
 * tpp_brgemm_execute_batched computes, with the same kernels: the only difference is where a
 * reduction split over several workgroups keeps its partial tiles, here in a scratch array of
 * TPP_BRGEMM_NOALLOC_SCRATCH_BYTES that the library holds on every GPU it runs on (from the
 * library's load until the process ends).  Every call on one GPU shares that GPU's array, so
 * calls on one GPU whose executions overlap in time (on different streams) race; calls on one
 * stream are ordered by the stream.  The array needs no clearing: a split launch writes every
 * partial tile before its finishing kernel reads it.  Handles with AUX bits are refused.
 * Errors: those of tpp_brgemm_execute_batched; UNSUPPORTED, with nothing launched, when the
 * launch's split needs more scratch than the array holds (the message gives both sizes);
 * TPP_ERR_HIP if the array's device address cannot be looked up. */
tpp_status tpp_brgemm_execute_batched_noalloc(
    tpp_brgemm_handle h, const tpp_grid_strided* grid, int64_t G, const int64_t* d_a_off,
    const int64_t* d_b_off, const int64_t* d_c_off, const int64_t* d_bias_off, const void* a,
    const void* b, void* c, const float* bias, int64_t count, const int64_t* d_offs_a,
    const int64_t* d_offs_b, const int64_t* d_begin, const void* const* d_ptrs_a,
    const void* const* d_ptrs_b, void* stream);

/* Reduce TPP (Table 1; Sec. 3.1: reduction-by-columns turns an M x N input into M x 1).
 *   in: device, m x n column-major with leading dimension ld >= m, type in_type (F32 or BF16).
 *   TPP_RED_BY_COLS: out[r] = fold_{c<n} f(in(r, c))   (m outputs)
 *   TPP_RED_BY_ROWS: out[c] = fold_{r<m} f(in(r, c))   (n outputs)
 *   f(x) = x into out_x when TPP_RED_X is set, f(x) = x*x into out_x2 when TPP_RED_X2 is set
 *   (both may be set: one pass, two outputs).  fold: SUM (from 0), MUL (from 1), MIN, MAX.
 *   Outputs are device fp32 arrays.  Arithmetic is fp32; the summation order is unspecified.
 * Partial results go to a device work buffer the library keeps per GPU and per stream (allocated
 * on first use, kept until the process ends; growing it synchronises the device).  Exactly one of
 * BY_COLS / BY_ROWS, and at least one of X / X2, must be set.  Errors: INVALID_ARG for m, n <= 0,
 * ld < m, bad flags, NULL pointers; NO_MEMORY if the work buffer cannot be allocated. */
typedef enum { TPP_RED_SUM = 0, TPP_RED_MUL = 1, TPP_RED_MIN = 2, TPP_RED_MAX = 3 } tpp_reduce_op;
enum {
  TPP_RED_BY_COLS = 1u << 0,
  TPP_RED_BY_ROWS = 1u << 1,
  TPP_RED_X = 1u << 2,
  TPP_RED_X2 = 1u << 3
};
tpp_status tpp_reduce(int32_t m, int32_t n, int64_t ld, int32_t in_type, const void* in,
                      int32_t op, uint32_t flags, float* out_x, float* out_x2, void* stream);

/* G Reduce TPP calls in one launch (the loop Alg. 6 writes around a TPP, here for the bias
 * gradients of a blocked layer): call g folds the m x n block at in + g * in_stride (elements)
 * and writes its outputs at out_x + g * out_stride and out_x2 + g * out_stride (floats).  Every
 * call has the shape, op and flags above.  G == 0 is a no-op.
 * Errors: those of tpp_reduce, plus INVALID_ARG for G, in_stride or out_stride < 0;
 * UNSUPPORTED when one launch would need more than 2^31 - 1 workgroups. */
tpp_status tpp_reduce_batched(int32_t m, int32_t n, int64_t ld, int32_t in_type, const void* in,
                              int64_t G, int64_t in_stride, int32_t op, uint32_t flags,
                              float* out_x, float* out_x2, int64_t out_stride, void* stream);

/* Static text for a status code, and the last error's detail for the calling thread. */
const char* tpp_status_string(tpp_status s);
const char* tpp_last_error_message(void);

#ifdef __cplusplus
}
#endif
#endif /* TPP_BRGEMM_H */
