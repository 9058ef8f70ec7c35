/*
 * oracle.h -- plain CPU reference for the batch-reduce GEMM TPP and the Reduce TPP.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may include, link or call this code;
 * only the test suite, the smoke check and the benchmark's CPU-baseline leg use it.  It shares
 * no header, helper, table or constant with the HIP library: every definition below is its own.
 *
 * What it computes (Tensor Processing Primitives, arXiv 2104.05755):
 *   - Ternary BRGEMM TPP, Table 3 and Sec. 2.3: C = beta*C + sum_{i<n} A_i x B_i, with the three
 *     block-addressing variants of Sec. 2.3 (address-, offset- and stride-based).
 *   - The unary/binary TPPs fused after it (Sec. 2.1 principle 5; Table 1 Identity-with-conversion,
 *     RELU, GELU; Table 2 Add with column broadcast, Sec. 2.2), applied as Alg. 6 applies its UNARY
 *     to the finished C block.
 *   - Unary Reduce TPP, Table 1 and Sec. 3.1 (reduction-by-columns turns M x N into M x 1).
 *   - Unary Transform TPP, Table 1 and Sec. 3.1: Transpose, VNNI formatting and VNNI to
 *     VNNI-transpose (entry permutations; no arithmetic).
 *   - For back-propagation through the fused layers (Sec. 5.1.6 implements the backward pass of
 *     the fully-connected layer with TPPs as well): the RELU_inv / GELU_inv TPPs of Table 1 fused
 *     after the BRGEMM, the pre-activation kept by the forward call, and the loops of Alg. 6 around
 *     the Reduce and Transform TPPs.
 *   - The sparse embedding gather-reduce of Alg. 5 (a multi-hot vector times a table).
 *   - TPP matrix equations (Sec. 4): the register scores of Alg. 3, the execution plan of
 *     Alg. 4, and the value of an elementwise equation tree.
 *
 * Storage reading: every 2D block is column-major with a leading dimension (element (r, c) of an
 * m x n block sits at base + r + c*ld), which is how Alg. 6 lays out its blocked tensors (the
 * b_m / b_k index innermost).  Strides and offsets count elements of the operand's own type.
 * Arithmetic is fp64; bf16 values widen exactly (bf16 is the top half of an fp32, Sec. 3.2.2).
 */
#ifndef TPP_ORACLE_H
#define TPP_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { ORACLE_F32 = 0, ORACLE_BF16 = 1 };
enum { ORACLE_STRIDE = 0, ORACLE_OFFSET = 1, ORACLE_ADDRESS = 2 };
enum { ORACLE_EPI_BIAS = 1u, ORACLE_EPI_RELU = 2u, ORACLE_EPI_GELU_TANH = 4u,
       ORACLE_EPI_RELU_INV = 8u, ORACLE_EPI_GELU_TANH_INV = 16u, ORACLE_EPI_SAVE_PREACT = 32u,
       /* layout: A_i stored transposed, element (row, p) at row * lda + p (lda >= k) */
       ORACLE_A_TRANS = 256u,
       /* layout: B_i stored transposed, element (p, col) at p * ldb + col (ldb >= n) */
       ORACLE_B_TRANS = 512u };
enum { ORACLE_RED_SUM = 0, ORACLE_RED_MUL = 1, ORACLE_RED_MIN = 2, ORACLE_RED_MAX = 3 };
enum { ORACLE_RED_BY_COLS = 1u, ORACLE_RED_BY_ROWS = 2u, ORACLE_RED_X = 4u, ORACLE_RED_X2 = 8u };
enum { ORACLE_TR_TRANSPOSE = 0, ORACLE_TR_VNNI = 1, ORACLE_TR_VNNI_TO_VNNI_T = 2 };

typedef struct {
  int32_t m, n, k;           /* C is m x n, A_i is m x k, B_i is k x n                        */
  int64_t lda, ldb, ldc;     /* leading dimensions, elements                                    */
  int32_t ab_type;           /* ORACLE_F32 or ORACLE_BF16 (A and B share it)                   */
  int32_t c_type;            /* ORACLE_F32 or ORACLE_BF16                                       */
  double  beta;              /* 0 => C is not read                                              */
  int32_t kind;              /* ORACLE_STRIDE / ORACLE_OFFSET / ORACLE_ADDRESS                  */
  int64_t stride_a, stride_b;/* elements, stride variant                                        */
  uint32_t flags;            /* ORACLE_EPI_* bits                                               */
} oracle_desc;

typedef struct { int64_t gm, gn, a_step_m, b_step_n, c_step_m, c_step_n, bias_step_m; } oracle_grid;

/* One BRGEMM call (the paper's call API).  a/b: base addresses (stride, offset variants);
 * offs_a/offs_b: count element offsets (offset variant); ptrs_a/ptrs_b: count block addresses
 * (address variant).  bias: m floats (ORACLE_EPI_BIAS).  ref64 (optional): m*n doubles,
 * column-major with ld m, receiving the unrounded result.  Returns 0, or -1 on bad arguments. */
int oracle_brgemm(const oracle_desc* d, const void* a, const void* b, void* c, const float* bias,
                  int64_t count, const int64_t* offs_a, const int64_t* offs_b,
                  const void* const* ptrs_a, const void* const* ptrs_b, double* ref64);

/* G independent calls (the outer loops of Alg. 6 / Alg. 7 around the BRGEMM).  Instance g's
 * bases: strided form when grid != NULL (gi_m = g % gm, gi_n = g / gm), else the explicit
 * per-instance offset arrays (any may be NULL = zeros).  Address variant: instance g reduces the
 * pairs [begin[g], begin[g+1]) of ptrs_a/ptrs_b.  sel (optional, n_sel entries) restricts the
 * work to those instances; ref64 then holds n_sel blocks of m*n doubles.  nthreads <= 0 uses
 * the OpenMP default. */
int oracle_brgemm_batched(const oracle_desc* d, const oracle_grid* grid, int64_t G,
                          const int64_t* a_off, const int64_t* b_off, const int64_t* c_off,
                          const int64_t* bias_off,
                          const void* a, const void* b, void* c, const float* bias,
                          int64_t count, const int64_t* offs_a, const int64_t* offs_b,
                          const int64_t* begin, const void* const* ptrs_a, const void* const* ptrs_b,
                          int64_t n_sel, const int64_t* sel, double* ref64, int nthreads);

/* As oracle_brgemm_batched, with an aux tensor of C's type, shaped and laid out as C (same
 * leading dimension and per-instance offsets).  SAVE_PREACT (with RELU or GELU_TANH) writes the
 * pre-activation beta*C + sum + bias, rounded to C's type, into aux before the activation;
 * RELU_INV / GELU_TANH_INV (Table 1's inverse activations for back-propagation) multiply the
 * block by the activation's derivative at z = aux.  Calls without these flags may pass NULL. */
int oracle_brgemm_batched_aux(const oracle_desc* d, const oracle_grid* grid, int64_t G,
                              const int64_t* a_off, const int64_t* b_off, const int64_t* c_off,
                              const int64_t* bias_off,
                              const void* a, const void* b, void* c, void* aux, const float* bias,
                              int64_t count, const int64_t* offs_a, const int64_t* offs_b,
                              const int64_t* begin, const void* const* ptrs_a,
                              const void* const* ptrs_b, int64_t n_sel, const int64_t* sel,
                              double* ref64, int nthreads);

/* Reduce TPP on an m x n column-major tensor.  BY_COLS folds across the n columns (m outputs),
 * BY_ROWS folds across the m rows (n outputs).  X / X2 select the input x or its square x*x;
 * both may be set.  Outputs are unrounded doubles. */
int oracle_reduce(int32_t m, int32_t n, int64_t ld, int32_t in_type, const void* in,
                  int32_t op, uint32_t flags, double* out_x, double* out_x2);

/* Transform TPP (Table 1; Sec. 3.1): a permutation of the entries of an m x n input whose entry
 * (r, c) sits at in + r + c*ld_in (elements of es bytes: 4 for fp32, 2 for bf16).
 *   TRANSPOSE       the matrix transpose: the n x m output has entry (c, r) = in(r, c) at
 *                   out + c + r*ld_out (ld_in >= m, ld_out >= n; alpha unused).
 *   VNNI            the logical tensor [D1][D0] = [n][m] (columns of m contiguous rows) laid out
 *                   as [D1/alpha][D0][alpha]: column c = alpha*g + a goes to
 *                   out + g*ld_out + r*alpha + a (ld_in >= m, ld_out >= m*alpha).  A last group
 *                   with fewer than alpha columns is completed with zero entries.
 *   VNNI_TO_VNNI_T  the input is an m x n tensor in that layout (group stride ld_in >= m*alpha);
 *                   the output is its transpose (n x m) in the same layout with the same alpha
 *                   (group stride ld_out >= n*alpha), i.e. [D1/a][D0][a] -> [D0/a][D1][a];
 *                   zero entries complete the output's last group when m % alpha != 0.
 * alpha is 1, 2 or 4.  Positions of out outside these (gaps when ld_out exceeds the extent) are
 * left as they were.  m == 0 or n == 0 writes nothing.  Returns 0, or -1 for a bad argument. */
int oracle_transform(int32_t kind, int32_t m, int32_t n, int64_t ld_in, int64_t ld_out,
                     int32_t es, int32_t alpha, const void* in, void* out);

/* G calls of the Reduce / Transform TPP on blocks in_stride elements apart (the loops Alg. 6
 * writes around a TPP); outputs of call g start out_stride elements (doubles for the reduce)
 * after those of call g - 1. */
int oracle_reduce_batched(int32_t m, int32_t n, int64_t ld, int32_t in_type, const void* in,
                          int64_t G, int64_t in_stride, int32_t op, uint32_t flags,
                          double* out_x, double* out_x2, int64_t out_stride);
int oracle_transform_batched(int32_t kind, int32_t m, int32_t n, int64_t ld_in, int64_t ld_out,
                             int32_t es, int32_t alpha, const void* in, int64_t in_stride,
                             void* out, int64_t out_stride, int64_t G);

/* Sparse embedding gather-reduce (Alg. 5): out[b][e] = sum over j in [begin[b], begin[b+1]) of
 * W[idx[j]][e] (row r at W + r*ldw, output row b at out + b*ldo), fp64 sums rounded once to
 * out_type; repeated indices count as often as listed; an empty bag gives zeros.  ref64
 * (optional): n_bags x E unrounded sums.  Returns -1 for an index outside [0, M), a decreasing
 * begin, or a bad size. */
int oracle_embedding_bag(int64_t M, int32_t E, int32_t w_type, const void* W, int64_t ldw,
                         int64_t n_bags, const int64_t* begin, const int64_t* idx,
                         int32_t out_type, void* out, int64_t ldo, double* ref64);

/* TPP matrix equations (Sec. 4): a tree whose internal nodes are unary / binary / ternary TPPs
 * and whose leaves are the 2D input tensors.  Node i: arity (0 = leaf), op, children (node
 * indices; first, second, third = Left, Middle / Right as the paper names them), leaf = the
 * input index of a leaf. */
enum { ORACLE_EQ_LEAF = 0, ORACLE_EQ_UNARY = 1, ORACLE_EQ_BINARY = 2, ORACLE_EQ_TERNARY = 3 };
enum { ORACLE_EQ_IDENTITY = 0, ORACLE_EQ_NEG = 1, ORACLE_EQ_EXP = 2, ORACLE_EQ_TANH = 3,
       ORACLE_EQ_RELU = 4, ORACLE_EQ_GELU_TANH = 5, ORACLE_EQ_SQRT = 6, ORACLE_EQ_RCP = 7,
       ORACLE_EQ_SQUARE = 8, ORACLE_EQ_SIGMOID = 9,
       ORACLE_EQ_ADD = 16, ORACLE_EQ_SUB = 17, ORACLE_EQ_MUL = 18, ORACLE_EQ_DIV = 19,
       ORACLE_EQ_MAX = 20, ORACLE_EQ_MIN = 21,
       ORACLE_EQ_MULADD = 32 };
/* Leaf broadcast (Sec. 2.2): 0 a full m x n tensor, 1 a column of m entries repeated over the n
 * columns, 2 a row of n entries repeated over the m rows, 3 one scalar. */
enum { ORACLE_BC_NONE = 0, ORACLE_BC_COL = 1, ORACLE_BC_ROW = 2, ORACLE_BC_SCALAR = 3 };
typedef struct { int32_t arity, op, child[3], leaf; } oracle_eq_node;
typedef struct { const void* ptr; int64_t ld; int32_t dtype, bcast; } oracle_eq_leaf;

/* Alg. 3: register score of every node (leaves 0).  Returns -1 for a malformed tree. */
int oracle_eq_scores(const oracle_eq_node* nodes, int32_t n_nodes, int32_t root, int32_t* score);
/* Alg. 4 on the scores of Alg. 3: evaluation timestamp and temporary tensor id of every internal
 * node (leaves: -1), and the number of temporaries the plan uses. */
int oracle_eq_plan(const oracle_eq_node* nodes, int32_t n_nodes, int32_t root,
                   const int32_t* score, int32_t* timestamp, int32_t* tmp, int32_t* n_tmps);
/* The equation's value at every (r, c) of an m x n output: the tree evaluated recursively in
 * fp64 (libm transcendentals), rounded once to out_type; ref64 (optional, m x n column-major)
 * gets the unrounded values. */
int oracle_eq_eval(const oracle_eq_node* nodes, int32_t n_nodes, int32_t root, int32_t m,
                   int32_t n, const oracle_eq_leaf* leaves, int32_t n_leaves, void* out,
                   int64_t ldo, int32_t out_type, double* ref64);

/* Helpers the tests pin on their own: exact widening and the round-to-nearest-even narrowing
 * used for every output element. */
double   oracle_widen(const void* base, int64_t idx, int32_t dtype);
uint16_t oracle_f32_to_bf16(float f);
void     oracle_f32_to_bf16_array(const float* in, uint16_t* out, int64_t n);
float    oracle_bf16_to_f32(uint16_t h);
double   oracle_gelu_tanh(double x);
double   oracle_gelu_tanh_grad(double x);
int      oracle_max_threads(void);

#ifdef __cplusplus
}
#endif
#endif
