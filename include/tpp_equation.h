/*
 * tpp_equation.h -- C ABI of the TPP matrix equations of the MI355X (gfx950) TPP library.
 *
 * Tensor Processing Primitives (arXiv 2104.05755), Sec. 4: a composite elementwise operator is
 * given as an equation tree whose internal nodes are unary, binary or ternary TPPs and whose
 * leaves are the 2D input tensors (with the broadcast forms of Sec. 2.2).  The planner assigns
 * every node the register score of Alg. 3 and derives the execution plan of Alg. 4 (evaluation
 * timestamps and temporary-tensor ids that reuse temporaries as far as the tree allows).  The
 * executor evaluates the plan per output element with the temporaries in registers (the paper's
 * Strategy 2: temporaries as register blocks), reading each leaf where it is and storing the
 * root once.
 *
 * Conventions are those of tpp_brgemm.h: column-major 2D tensors with leading dimensions counted
 * in elements, caller-owned DEVICE tensors, asynchronous on `stream`, a tpp_status result and
 * tpp_last_error_message() for the detail.  The tree itself (nodes, arguments) is host memory,
 * read during the call only.
 */
#ifndef TPP_EQUATION_H
#define TPP_EQUATION_H

#include "tpp_brgemm.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { TPP_EQ_LEAF = 0, TPP_EQ_UNARY = 1, TPP_EQ_BINARY = 2, TPP_EQ_TERNARY = 3 } tpp_eq_arity;

/* Operations (Table 1 unary, Table 2 binary, Table 3 ternary TPPs that act elementwise).
 * Unary: IDENTITY x, NEG -x, EXP e^x, TANH, RELU (x > 0 ? x : +0), GELU_TANH (the tanh form of
 * TPP_EPI_GELU_TANH), SQRT, RCP 1/x, SQUARE x*x, SIGMOID 1 / (1 + e^-x).
 * Binary: ADD a + b, SUB a - b, MUL a * b, DIV a / b, MAX, MIN.  Ternary: MULADD a * b + c. */
typedef enum {
  TPP_EQ_IDENTITY = 0, TPP_EQ_NEG = 1, TPP_EQ_EXP = 2, TPP_EQ_TANH = 3, TPP_EQ_RELU = 4,
  TPP_EQ_GELU_TANH = 5, TPP_EQ_SQRT = 6, TPP_EQ_RCP = 7, TPP_EQ_SQUARE = 8, TPP_EQ_SIGMOID = 9,
  TPP_EQ_ADD = 16, TPP_EQ_SUB = 17, TPP_EQ_MUL = 18, TPP_EQ_DIV = 19, TPP_EQ_MAX = 20,
  TPP_EQ_MIN = 21,
  TPP_EQ_MULADD = 32
} tpp_eq_op;

/* Leaf broadcast (Sec. 2.2): NONE a full m x n tensor (entry (r, c) at ptr + r + c*ld); COL a
 * column of m entries repeated over the n columns (entry r); ROW a row of n entries repeated over
 * the m rows (entry c); SCALAR one entry. */
typedef enum { TPP_BC_NONE = 0, TPP_BC_COL = 1, TPP_BC_ROW = 2, TPP_BC_SCALAR = 3 } tpp_eq_bcast;

/* One tree node.  arity: tpp_eq_arity; op: tpp_eq_op of that arity (ignored for a leaf);
 * child[0..arity-1]: node indices (Left, then Middle / Right as the paper names them);
 * leaf: for a leaf, the index of its argument. */
typedef struct {
  int32_t arity, op;
  int32_t child[3];
  int32_t leaf;
} tpp_eq_node;

/* Per node: the register score of Alg. 3, and the timestamp and temporary-tensor id of Alg. 4
 * (-1 for leaves). */
typedef struct {
  int32_t score, timestamp, tmp;
} tpp_eq_plan_node;

/* The planner (host only, no device work).  Fills plan[0 .. n_nodes-1] and *n_tmps (the number
 * of temporaries the plan uses).  Children are visited in order of decreasing register score
 * (the earlier child first among equals); a node whose children are all leaves reserves the
 * lowest free temporary; otherwise it takes the temporary of its Left child if that is not a
 * leaf, else of its Right child (ternary), else of its remaining non-leaf child, and the other
 * children's temporaries return to the pool.
 * Errors: INVALID_ARG for NULL pointers, n_nodes outside [1, 64], a root or child index out of
 * range, a node reached twice (not a tree), an arity outside [0, 3] or an op of the wrong arity. */
tpp_status tpp_equation_plan(const tpp_eq_node* nodes, int32_t n_nodes, int32_t root,
                             tpp_eq_plan_node* plan, int32_t* n_tmps);

/* One leaf argument: a device tensor of dtype (TPP_DT_F32 or TPP_DT_BF16), its leading dimension
 * (used by TPP_BC_NONE: ld >= m) and its broadcast form. */
typedef struct {
  const void* ptr;
  int64_t ld;
  int32_t dtype;
  int32_t bcast;
} tpp_eq_arg;

/* Evaluate the equation over an m x n output: out[r + c*ldo] = tree(r, c), fp32 arithmetic in
 * the planned order, rounded once to out_type (TPP_DT_F32 or TPP_DT_BF16, nearest even).  Leaves
 * are widened exactly (bf16 is the top half of an fp32).  Every argument in args is read, also
 * one the tree does not reach, so each must describe a valid tensor.  m == 0 or n == 0 is a
 * no-op.  out must not overlap a leaf tensor unless it is that leaf exactly (same pointer and
 * layout).
 * Errors: those of tpp_equation_plan, plus INVALID_ARG for m, n < 0, ldo < m, a leaf index outside
 * [0, n_args), a NULL or badly described argument, n_args above 16; UNSUPPORTED when the plan
 * needs more than 8 temporaries; HIP if the launch fails. */
tpp_status tpp_equation_execute(const tpp_eq_node* nodes, int32_t n_nodes, int32_t root,
                                int32_t m, int32_t n, const tpp_eq_arg* args, int32_t n_args,
                                void* out, int64_t ldo, int32_t out_type, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* TPP_EQUATION_H */
