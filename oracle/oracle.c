/*
 * oracle.c -- plain, slow CPU reference for the batch-reduce GEMM TPP with its fused epilogue,
 * and for the Reduce TPP.  TEST INFRASTRUCTURE ONLY: the product library never includes, links
 * or calls it.  Every loop is the definition written out in fp64, with no blocking, fusion or
 * reordering beyond what the definition states.  Paper: arXiv 2104.05755 (TPP).
 */
#include "oracle.h"

#include <math.h>
#include <stddef.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static int elem_size(int32_t dtype) { return dtype == ORACLE_F32 ? 4 : 2; }

/* bf16 is the upper 16 bits of an fp32 (Sec. 3.2.2), so widening is a shift and is exact. */
float oracle_bf16_to_f32(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return f;
}

/* fp32 -> bf16, round to nearest, ties to even, on the bit pattern.  NaN stays a (quiet) NaN;
 * values past the largest finite bf16 round to infinity through the carry into the exponent. */
uint16_t oracle_f32_to_bf16(float f) {
  uint32_t u;
  memcpy(&u, &f, sizeof u);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x0040u);
  uint32_t keep = u >> 16;
  uint32_t rest = u & 0xffffu;
  if (rest > 0x8000u || (rest == 0x8000u && (keep & 1u))) keep += 1u;
  return (uint16_t)keep;
}

void oracle_f32_to_bf16_array(const float* in, uint16_t* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = oracle_f32_to_bf16(in[i]);
}

double oracle_widen(const void* base, int64_t idx, int32_t dtype) {
  if (dtype == ORACLE_F32) return (double)((const float*)base)[idx];
  return (double)oracle_bf16_to_f32(((const uint16_t*)base)[idx]);
}

/* Output narrowing: the fp64 value is rounded once to fp32 (the accumulation precision), then,
 * for a bf16 output, once more to bf16.  Both steps are round-to-nearest-even. */
static void store_rounded(void* base, int64_t idx, int32_t dtype, double v) {
  float f = (float)v;
  if (dtype == ORACLE_F32)
    ((float*)base)[idx] = f;
  else
    ((uint16_t*)base)[idx] = oracle_f32_to_bf16(f);
}

/* GELU in its tanh form: 0.5 x (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3))), libm tanh in fp64. */
double oracle_gelu_tanh(double x) {
  const double c = sqrt(2.0 / 3.14159265358979323846);
  return 0.5 * x * (1.0 + tanh(c * (x + 0.044715 * x * x * x)));
}

/* Derivative of that GELU form (the GELU_inv of Table 1, used by back-propagation):
 * with u = sqrt(2/pi) (x + 0.044715 x^3) and t = tanh(u),
 *   d/dx [0.5 x (1 + t)] = 0.5 (1 + t) + 0.5 x (1 - t^2) sqrt(2/pi) (1 + 3 * 0.044715 x^2). */
double oracle_gelu_tanh_grad(double x) {
  const double c = sqrt(2.0 / 3.14159265358979323846);
  const double t = tanh(c * (x + 0.044715 * x * x * x));
  return 0.5 * (1.0 + t) + 0.5 * x * (1.0 - t * t) * c * (1.0 + 3.0 * 0.044715 * x * x);
}

int oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Addresses of the i-th pair of blocks, following the three variants of Sec. 2.3:
 *   address-based: the user gives the block addresses;
 *   offset-based:  address_A_i = address_A + offset_A_i;
 *   stride-based:  address_A_i = address_A_{i-1} + stride_A, starting from address_A.
 * The stride variant is written as the recurrence the paper states (a running address). */
static void pair_addresses(const oracle_desc* d, const void* a, const void* b, int64_t count,
                           const int64_t* offs_a, const int64_t* offs_b,
                           const void* const* ptrs_a, const void* const* ptrs_b,
                           const char** out_a, const char** out_b) {
  const int es = elem_size(d->ab_type);
  if (d->kind == ORACLE_ADDRESS) {
    for (int64_t i = 0; i < count; ++i) {
      out_a[i] = (const char*)ptrs_a[i];
      out_b[i] = (const char*)ptrs_b[i];
    }
  } else if (d->kind == ORACLE_OFFSET) {
    for (int64_t i = 0; i < count; ++i) {
      out_a[i] = (const char*)a + offs_a[i] * es;
      out_b[i] = (const char*)b + offs_b[i] * es;
    }
  } else {
    const char* pa = (const char*)a;
    const char* pb = (const char*)b;
    for (int64_t i = 0; i < count; ++i) {
      if (i > 0) {
        pa += d->stride_a * es;
        pb += d->stride_b * es;
      }
      out_a[i] = pa;
      out_b[i] = pb;
    }
  }
}

static int check_desc(const oracle_desc* d) {
  if (!d || d->m <= 0 || d->n <= 0 || d->k <= 0) return -1;
  const int a_trans = (d->flags & ORACLE_A_TRANS) != 0;
  const int b_trans = (d->flags & ORACLE_B_TRANS) != 0;
  if (d->lda < (a_trans ? d->k : d->m) || d->ldb < (b_trans ? d->n : d->k) || d->ldc < d->m)
    return -1;
  if (d->ab_type != ORACLE_F32 && d->ab_type != ORACLE_BF16) return -1;
  if (d->c_type != ORACLE_F32 && d->c_type != ORACLE_BF16) return -1;
  const uint32_t f = d->flags;
  const uint32_t known = ORACLE_EPI_BIAS | ORACLE_EPI_RELU | ORACLE_EPI_GELU_TANH |
                         ORACLE_EPI_RELU_INV | ORACLE_EPI_GELU_TANH_INV | ORACLE_EPI_SAVE_PREACT |
                         ORACLE_A_TRANS | ORACLE_B_TRANS;
  if (f & ~known) return -1;
  if ((f & ORACLE_EPI_RELU) && (f & ORACLE_EPI_GELU_TANH)) return -1;
  if ((f & ORACLE_EPI_RELU_INV) && (f & ORACLE_EPI_GELU_TANH_INV)) return -1;
  /* an inverse activation multiplies the block by a derivative: no forward activation with it */
  if ((f & (ORACLE_EPI_RELU_INV | ORACLE_EPI_GELU_TANH_INV)) &&
      (f & (ORACLE_EPI_RELU | ORACLE_EPI_GELU_TANH | ORACLE_EPI_SAVE_PREACT)))
    return -1;
  /* the pre-activation is only worth keeping when an activation follows it */
  if ((f & ORACLE_EPI_SAVE_PREACT) && !(f & (ORACLE_EPI_RELU | ORACLE_EPI_GELU_TANH))) return -1;
  if (d->kind < ORACLE_STRIDE || d->kind > ORACLE_ADDRESS) return -1;
  return 0;
}

/* The BRGEMM TPP on already-resolved block addresses, then the fused epilogue, per output
 * element (r, c):
 *   s   = sum_i sum_p A_i(r, p) * B_i(p, c)          (Table 3, Sec. 2.3)
 *   v   = beta * C(r, c) + s                         (C read only when beta != 0)
 *   v  += bias[r]                                    (Add with a column broadcast over n)
 *   aux(r, c) = round(v)                             (SAVE_PREACT: the pre-activation kept for
 *                                                     back-propagation, in C's type and layout)
 *   v   = relu(v) or gelu_tanh(v)                    (unary TPP on the finished block, Alg. 6)
 *   v   = v * act'(z), z = aux(r, c)                 (RELU_INV / GELU_TANH_INV, Table 1: the
 *                                                     incoming gradient times the activation's
 *                                                     derivative at the saved pre-activation)
 *   C(r, c) = round(v)                               (Identity with conversion)
 * ReLU's derivative is taken as 1 for z > 0 and 0 otherwise.                                 */
static void brgemm_resolved(const oracle_desc* d, const char* const* pa, const char* const* pb,
                            int64_t count, void* c, const float* bias, void* aux, double* ref64) {
  const int a_trans = (d->flags & ORACLE_A_TRANS) != 0;
  const int b_trans = (d->flags & ORACLE_B_TRANS) != 0;
  for (int32_t col = 0; col < d->n; ++col) {
    for (int32_t row = 0; row < d->m; ++row) {
      double s = 0.0;
      for (int64_t i = 0; i < count; ++i) {
        for (int32_t p = 0; p < d->k; ++p) {
          /* A_i(row, p): column-major, or transposed (Sec. 3.1's transpose of the block) */
          const int64_t at = a_trans ? (int64_t)row * d->lda + p : (int64_t)row + (int64_t)p * d->lda;
          double x = oracle_widen(pa[i], at, d->ab_type);
          /* B_i(p, col): column-major, or transposed */
          const int64_t bt = b_trans ? (int64_t)p * d->ldb + col : (int64_t)p + (int64_t)col * d->ldb;
          double y = oracle_widen(pb[i], bt, d->ab_type);
          s += x * y;
        }
      }
      const int64_t ci = (int64_t)row + (int64_t)col * d->ldc;
      double v = s;
      if (d->beta != 0.0) v = d->beta * oracle_widen(c, ci, d->c_type) + s;
      if (d->flags & ORACLE_EPI_BIAS) v += (double)bias[row];
      if (d->flags & ORACLE_EPI_SAVE_PREACT) store_rounded(aux, ci, d->c_type, v);
      if (d->flags & ORACLE_EPI_RELU) v = v > 0.0 ? v : 0.0;
      if (d->flags & ORACLE_EPI_GELU_TANH) v = oracle_gelu_tanh(v);
      if (d->flags & ORACLE_EPI_RELU_INV) {
        const double z = oracle_widen(aux, ci, d->c_type);
        v = z > 0.0 ? v : 0.0;
      }
      if (d->flags & ORACLE_EPI_GELU_TANH_INV)
        v = v * oracle_gelu_tanh_grad(oracle_widen(aux, ci, d->c_type));
      if (ref64) ref64[(int64_t)row + (int64_t)col * d->m] = v;
      store_rounded(c, ci, d->c_type, v);
    }
  }
}

static int needs_aux(const oracle_desc* d) {
  return (d->flags & (ORACLE_EPI_RELU_INV | ORACLE_EPI_GELU_TANH_INV | ORACLE_EPI_SAVE_PREACT)) != 0;
}

static int check_pairs(const oracle_desc* d, const void* a, const void* b, int64_t count,
                       const int64_t* offs_a, const int64_t* offs_b,
                       const void* const* ptrs_a, const void* const* ptrs_b) {
  if (count < 0) return -1;
  if (count == 0) return 0;
  if (d->kind == ORACLE_ADDRESS) return (ptrs_a && ptrs_b) ? 0 : -1;
  if (d->kind == ORACLE_OFFSET) return (a && b && offs_a && offs_b) ? 0 : -1;
  return (a && b) ? 0 : -1;
}

/* One call: resolve the count block addresses, then run the definition. */
static int brgemm_one(const oracle_desc* d, const void* a, const void* b, void* c,
                      const float* bias, void* aux, int64_t count, const int64_t* offs_a,
                      const int64_t* offs_b, const void* const* ptrs_a,
                      const void* const* ptrs_b, double* ref64) {
  if (check_pairs(d, a, b, count, offs_a, offs_b, ptrs_a, ptrs_b) != 0) return -1;
  const char** pa = (const char**)malloc(sizeof(char*) * (size_t)(count > 0 ? count : 1));
  const char** pb = (const char**)malloc(sizeof(char*) * (size_t)(count > 0 ? count : 1));
  if (!pa || !pb) {
    free(pa);
    free(pb);
    return -1;
  }
  pair_addresses(d, a, b, count, offs_a, offs_b, ptrs_a, ptrs_b, pa, pb);
  brgemm_resolved(d, pa, pb, count, c, bias, aux, ref64);
  free(pa);
  free(pb);
  return 0;
}

int oracle_brgemm(const oracle_desc* d, const void* a, const void* b, void* c, const float* bias,
                  int64_t count, const int64_t* offs_a, const int64_t* offs_b,
                  const void* const* ptrs_a, const void* const* ptrs_b, double* ref64) {
  if (check_desc(d) != 0 || !c) return -1;
  if ((d->flags & ORACLE_EPI_BIAS) && !bias) return -1;
  if (needs_aux(d)) return -1;   /* single calls carry no aux tensor */
  return brgemm_one(d, a, b, c, bias, NULL, count, offs_a, offs_b, ptrs_a, ptrs_b, ref64);
}

int oracle_brgemm_batched_aux(const oracle_desc* d, const oracle_grid* grid, int64_t G,
                              const int64_t* a_off, const int64_t* b_off, const int64_t* c_off,
                              const int64_t* bias_off,
                              const void* a, const void* b, void* c, void* aux, const float* bias,
                              int64_t count, const int64_t* offs_a, const int64_t* offs_b,
                              const int64_t* begin, const void* const* ptrs_a,
                              const void* const* ptrs_b, int64_t n_sel, const int64_t* sel,
                              double* ref64, int nthreads);

/* The loops around the BRGEMM call that Alg. 6 (FC layer: ib_n, ib_m over output blocks) and
 * Alg. 7 (dilated convolution: pos) write out: G independent calls, each with its own bases.
 * Strided form: instance g = gi_m + gm * gi_n, with
 *   A base  = a + gi_m * a_step_m           B base = b + gi_n * b_step_n
 *   C base  = c + gi_m * c_step_m + gi_n * c_step_n     bias base = bias + gi_m * bias_step_m
 * Explicit form: element offsets a_off[g], b_off[g], c_off[g], bias_off[g].
 * Address variant: instance g reduces pairs begin[g] .. begin[g+1]-1 of the pointer lists. */
int oracle_brgemm_batched(const oracle_desc* d, const oracle_grid* grid, int64_t G,
                          const int64_t* a_off, const int64_t* b_off, const int64_t* c_off,
                          const int64_t* bias_off,
                          const void* a, const void* b, void* c, const float* bias,
                          int64_t count, const int64_t* offs_a, const int64_t* offs_b,
                          const int64_t* begin, const void* const* ptrs_a, const void* const* ptrs_b,
                          int64_t n_sel, const int64_t* sel, double* ref64, int nthreads) {
  if (d && needs_aux(d)) return -1;
  return oracle_brgemm_batched_aux(d, grid, G, a_off, b_off, c_off, bias_off, a, b, c, NULL, bias,
                                   count, offs_a, offs_b, begin, ptrs_a, ptrs_b, n_sel, sel, ref64,
                                   nthreads);
}

/* As oracle_brgemm_batched, with the aux tensor: shaped and laid out as C (same leading
 * dimension, same per-instance offsets) and of C's type. */
int oracle_brgemm_batched_aux(const oracle_desc* d, const oracle_grid* grid, int64_t G,
                              const int64_t* a_off, const int64_t* b_off, const int64_t* c_off,
                              const int64_t* bias_off,
                              const void* a, const void* b, void* c, void* aux, const float* bias,
                              int64_t count, const int64_t* offs_a, const int64_t* offs_b,
                              const int64_t* begin, const void* const* ptrs_a,
                              const void* const* ptrs_b, int64_t n_sel, const int64_t* sel,
                              double* ref64, int nthreads) {
  if (check_desc(d) != 0 || G < 0 || !c) return -1;
  if ((d->flags & ORACLE_EPI_BIAS) && !bias) return -1;
  if (needs_aux(d) && !aux) return -1;
  if (grid && (grid->gm <= 0 || grid->gn <= 0 || grid->gm * grid->gn != G)) return -1;
  if (d->kind == ORACLE_ADDRESS && G > 0 && !begin) return -1;
  if (!sel) n_sel = G;
  for (int64_t s = 0; s < n_sel; ++s) {
    int64_t g = sel ? sel[s] : s;
    if (g < 0 || g >= G) return -1;
  }
  const int es_ab = elem_size(d->ab_type);
  const int es_c = elem_size(d->c_type);
  int failed = 0;
#ifdef _OPENMP
  if (nthreads <= 0) nthreads = omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads) reduction(| : failed)
#endif
  for (int64_t s = 0; s < n_sel; ++s) {
    const int64_t g = sel ? sel[s] : s;
    int64_t ao, bo, co, zo;
    if (grid) {
      const int64_t gi_m = g % grid->gm, gi_n = g / grid->gm;
      ao = gi_m * grid->a_step_m;
      bo = gi_n * grid->b_step_n;
      co = gi_m * grid->c_step_m + gi_n * grid->c_step_n;
      zo = gi_m * grid->bias_step_m;
    } else {
      ao = a_off ? a_off[g] : 0;
      bo = b_off ? b_off[g] : 0;
      co = c_off ? c_off[g] : 0;
      zo = bias_off ? bias_off[g] : 0;
    }
    void* cg = (char*)c + co * es_c;
    void* xg = aux ? (char*)aux + co * es_c : NULL;
    const float* zg = bias ? bias + zo : NULL;
    double* rg = ref64 ? ref64 + s * (int64_t)d->m * d->n : NULL;
    int rc;
    if (d->kind == ORACLE_ADDRESS) {
      const int64_t lo = begin[g], hi = begin[g + 1];
      rc = (hi < lo) ? -1
                     : brgemm_one(d, NULL, NULL, cg, zg, xg, hi - lo, NULL, NULL,
                                  ptrs_a ? ptrs_a + lo : NULL, ptrs_b ? ptrs_b + lo : NULL, rg);
    } else {
      const void* ag = a ? (const char*)a + ao * es_ab : NULL;
      const void* bg = b ? (const char*)b + bo * es_ab : NULL;
      rc = brgemm_one(d, ag, bg, cg, zg, xg, count, offs_a, offs_b, NULL, NULL, rg);
    }
    if (rc != 0) failed |= 1;
  }
  return failed ? -1 : 0;
}

/* Reduce TPP (Table 1): fold rows or columns with SUM / MUL / MIN / MAX, of x or of x*x.
 * SUM starts at 0, MUL at 1; MIN and MAX start from the first element. */
static double fold(int32_t op, double acc, double v) {
  switch (op) {
    case ORACLE_RED_SUM: return acc + v;
    case ORACLE_RED_MUL: return acc * v;
    case ORACLE_RED_MIN: return v < acc ? v : acc;
    default: return v > acc ? v : acc;
  }
}

int oracle_reduce(int32_t m, int32_t n, int64_t ld, int32_t in_type, const void* in,
                  int32_t op, uint32_t flags, double* out_x, double* out_x2) {
  if (m <= 0 || n <= 0 || ld < m || !in) return -1;
  if (in_type != ORACLE_F32 && in_type != ORACLE_BF16) return -1;
  if (op < ORACLE_RED_SUM || op > ORACLE_RED_MAX) return -1;
  const int by_cols = (flags & ORACLE_RED_BY_COLS) != 0;
  const int by_rows = (flags & ORACLE_RED_BY_ROWS) != 0;
  if (by_cols == by_rows) return -1;
  if (!(flags & (ORACLE_RED_X | ORACLE_RED_X2))) return -1;
  if ((flags & ORACLE_RED_X) && !out_x) return -1;
  if ((flags & ORACLE_RED_X2) && !out_x2) return -1;
  const int32_t outer = by_cols ? m : n;
  const int32_t inner = by_cols ? n : m;
  for (int32_t o = 0; o < outer; ++o) {
    double ax = 0.0, ax2 = 0.0;
    for (int32_t t = 0; t < inner; ++t) {
      const int32_t row = by_cols ? o : t;
      const int32_t col = by_cols ? t : o;
      const double x = oracle_widen(in, (int64_t)row + (int64_t)col * ld, in_type);
      if (t == 0) {
        ax = (op == ORACLE_RED_MUL) ? 1.0 : (op == ORACLE_RED_SUM ? 0.0 : x);
        ax2 = (op == ORACLE_RED_MUL) ? 1.0 : (op == ORACLE_RED_SUM ? 0.0 : x * x);
        if (op == ORACLE_RED_MIN || op == ORACLE_RED_MAX) continue;
      }
      ax = fold(op, ax, x);
      ax2 = fold(op, ax2, x * x);
    }
    if (flags & ORACLE_RED_X) out_x[o] = ax;
    if (flags & ORACLE_RED_X2) out_x2[o] = ax2;
  }
  return 0;
}

/* Transform TPP (Table 1; Sec. 3.1 defines the three transformations; the VNNI layout is the
 * [K/alpha][M][alpha] reformatting of Sec. 3.2.2).  Entries are moved as raw bytes. */
static void move_entry(void* out, int64_t oi, const void* in, int64_t ii, int32_t es) {
  memcpy((char*)out + oi * es, (const char*)in + ii * es, (size_t)es);
}

static void zero_entry(void* out, int64_t oi, int32_t es) {
  memset((char*)out + oi * es, 0, (size_t)es);
}

int oracle_transform(int32_t kind, int32_t m, int32_t n, int64_t ld_in, int64_t ld_out,
                     int32_t es, int32_t alpha, const void* in, void* out) {
  if (m < 0 || n < 0 || (es != 2 && es != 4)) return -1;
  if (alpha != 1 && alpha != 2 && alpha != 4) return -1;
  if (kind == ORACLE_TR_TRANSPOSE) {
    if (ld_in < m || ld_out < n) return -1;
  } else if (kind == ORACLE_TR_VNNI) {
    if (ld_in < m || ld_out < (int64_t)m * alpha) return -1;
  } else if (kind == ORACLE_TR_VNNI_TO_VNNI_T) {
    if (ld_in < (int64_t)m * alpha || ld_out < (int64_t)n * alpha) return -1;
  } else {
    return -1;
  }
  if (m == 0 || n == 0) return 0;
  if (!in || !out) return -1;
  if (kind == ORACLE_TR_TRANSPOSE) {
    for (int32_t c = 0; c < n; ++c)
      for (int32_t r = 0; r < m; ++r)
        move_entry(out, (int64_t)c + (int64_t)r * ld_out, in, (int64_t)r + (int64_t)c * ld_in, es);
  } else if (kind == ORACLE_TR_VNNI) {
    const int32_t groups = (n + alpha - 1) / alpha;
    for (int32_t g = 0; g < groups; ++g)
      for (int32_t r = 0; r < m; ++r)
        for (int32_t a = 0; a < alpha; ++a) {
          const int32_t c = g * alpha + a;
          const int64_t oi = (int64_t)g * ld_out + (int64_t)r * alpha + a;
          if (c < n)
            move_entry(out, oi, in, (int64_t)r + (int64_t)c * ld_in, es);
          else
            zero_entry(out, oi, es);
        }
  } else {
    /* output group g holds rows r = alpha*g + a of the input as its columns of n entries */
    const int32_t groups = (m + alpha - 1) / alpha;
    for (int32_t g = 0; g < groups; ++g)
      for (int32_t c = 0; c < n; ++c)
        for (int32_t a = 0; a < alpha; ++a) {
          const int32_t r = g * alpha + a;
          const int64_t oi = (int64_t)g * ld_out + (int64_t)c * alpha + a;
          if (r < m)
            move_entry(out, oi, in, (int64_t)(c / alpha) * ld_in + (int64_t)r * alpha + c % alpha,
                       es);
          else
            zero_entry(out, oi, es);
        }
  }
  return 0;
}

/* The loop Alg. 6 writes around a TPP call, for the Reduce and Transform TPPs: G independent
 * calls on blocks in_stride elements apart, whose results are out_stride elements (outputs)
 * apart. */
int oracle_reduce_batched(int32_t m, int32_t n, int64_t ld, int32_t in_type, const void* in,
                          int64_t G, int64_t in_stride, int32_t op, uint32_t flags,
                          double* out_x, double* out_x2, int64_t out_stride) {
  if (G < 0 || in_stride < 0 || out_stride < 0) return -1;
  const int es = elem_size(in_type);
  for (int64_t g = 0; g < G; ++g) {
    const int rc = oracle_reduce(m, n, ld, in_type, (const char*)in + g * in_stride * es, op,
                                 flags, out_x ? out_x + g * out_stride : NULL,
                                 out_x2 ? out_x2 + g * out_stride : NULL);
    if (rc != 0) return rc;
  }
  return 0;
}

int oracle_transform_batched(int32_t kind, int32_t m, int32_t n, int64_t ld_in, int64_t ld_out,
                             int32_t es, int32_t alpha, const void* in, int64_t in_stride,
                             void* out, int64_t out_stride, int64_t G) {
  if (G < 0 || in_stride < 0 || out_stride < 0) return -1;
  for (int64_t g = 0; g < G; ++g) {
    const int rc = oracle_transform(kind, m, n, ld_in, ld_out, es, alpha,
                                    in ? (const char*)in + g * in_stride * es : NULL,
                                    out ? (char*)out + g * out_stride * es : NULL);
    if (rc != 0) return rc;
  }
  return 0;
}

/* Sparse embedding gather-reduce (Alg. 5): the output row of bag b is o = a^T W with a the
 * multi-hot vector of the bag's indices, i.e. the sum of the table rows the bag lists,
 *   out[b][e] = sum_{j = begin[b]}^{begin[b+1]-1} W[idx[j]][e]      (e < E),
 * a listed index counted as often as it is listed (the loop of Alg. 5 over the indices).  Row r
 * of the table starts at W + r*ldw.  Sums are fp64, rounded once to the output type.  An empty
 * bag gives zeros.  Returns -1 for an index outside [0, M) or a decreasing begin. */
int oracle_embedding_bag(int64_t M, int32_t E, int32_t w_type, const void* W, int64_t ldw,
                         int64_t n_bags, const int64_t* begin, const int64_t* idx,
                         int32_t out_type, void* out, int64_t ldo, double* ref64) {
  if (M < 0 || E <= 0 || n_bags < 0 || ldw < E || ldo < E) return -1;
  if (w_type != ORACLE_F32 && w_type != ORACLE_BF16) return -1;
  if (out_type != ORACLE_F32 && out_type != ORACLE_BF16) return -1;
  if (n_bags == 0) return 0;
  if (!begin || !out) return -1;
  for (int64_t b = 0; b < n_bags; ++b) {
    if (begin[b + 1] < begin[b]) return -1;
    for (int64_t j = begin[b]; j < begin[b + 1]; ++j)
      if (idx[j] < 0 || idx[j] >= M) return -1;
  }
  for (int64_t b = 0; b < n_bags; ++b) {
    for (int32_t e = 0; e < E; ++e) {
      double s = 0.0;
      for (int64_t j = begin[b]; j < begin[b + 1]; ++j)
        s += oracle_widen(W, idx[j] * ldw + e, w_type);
      if (ref64) ref64[b * (int64_t)E + e] = s;
      store_rounded(out, b * ldo + e, out_type, s);
    }
  }
  return 0;
}

/* ---- TPP matrix equations (Sec. 4) ---------------------------------------------------------- */

static int eq_check(const oracle_eq_node* nodes, int32_t n_nodes, int32_t r, int depth) {
  if (r < 0 || r >= n_nodes || depth > n_nodes) return -1;
  const oracle_eq_node* x = &nodes[r];
  if (x->arity < ORACLE_EQ_LEAF || x->arity > ORACLE_EQ_TERNARY) return -1;
  for (int c = 0; c < x->arity; ++c)
    if (eq_check(nodes, n_nodes, x->child[c], depth + 1) != 0) return -1;
  return 0;
}

/* Alg. 3, recursively.  Unary: 1 over a leaf, else the child's score.  Binary: the children's
 * score plus one when they are equal, else the larger.  Ternary: 1 when all three children are
 * leaves, else the largest of 3 and the children's scores (as the algorithm prints it). */
static int32_t eq_score(const oracle_eq_node* nodes, int32_t r, int32_t* score) {
  const oracle_eq_node* x = &nodes[r];
  int32_t v = 0;
  if (x->arity == ORACLE_EQ_UNARY) {
    const int32_t c = eq_score(nodes, x->child[0], score);
    v = nodes[x->child[0]].arity == ORACLE_EQ_LEAF ? 1 : c;
  } else if (x->arity == ORACLE_EQ_BINARY) {
    const int32_t l = eq_score(nodes, x->child[0], score);
    const int32_t rr = eq_score(nodes, x->child[1], score);
    v = l == rr ? l + 1 : (l > rr ? l : rr);
  } else if (x->arity == ORACLE_EQ_TERNARY) {
    const int32_t l = eq_score(nodes, x->child[0], score);
    const int32_t mm = eq_score(nodes, x->child[1], score);
    const int32_t rr = eq_score(nodes, x->child[2], score);
    int all_leaves = 1;
    for (int c = 0; c < 3; ++c) all_leaves &= nodes[x->child[c]].arity == ORACLE_EQ_LEAF;
    if (all_leaves) {
      v = 1;
    } else {
      v = 3;
      if (l > v) v = l;
      if (mm > v) v = mm;
      if (rr > v) v = rr;
    }
  }
  score[r] = v;
  return v;
}

int oracle_eq_scores(const oracle_eq_node* nodes, int32_t n_nodes, int32_t root, int32_t* score) {
  if (!nodes || !score || eq_check(nodes, n_nodes, root, 0) != 0) return -1;
  for (int32_t i = 0; i < n_nodes; ++i) score[i] = 0;
  eq_score(nodes, root, score);
  return 0;
}

/* The pool of temporary tensors of Alg. 4: Reserve_Tmp hands out the lowest free id,
 * Recycle_Tmp returns one (a leaf has none to return). */
typedef struct { int32_t used[64]; int32_t high; } eq_pool;

static int32_t eq_reserve(eq_pool* p) {
  for (int32_t i = 0; i < 64; ++i)
    if (!p->used[i]) {
      p->used[i] = 1;
      if (i + 1 > p->high) p->high = i + 1;
      return i;
    }
  return -1;
}

static void eq_recycle(eq_pool* p, int32_t t) {
  if (t >= 0) p->used[t] = 0;
}

/* Alg. 4, recursively: children in order of decreasing register score (ties: the earlier child
 * first), then the node's timestamp; its tmp is a new one when every child is a leaf, else the tmp
 * of its first non-leaf child in the order Left, Right, Middle, the other children's tmps
 * recycled. */
static void eq_visit(const oracle_eq_node* nodes, int32_t r, const int32_t* score, int32_t* ts,
                     int32_t* tmp, int32_t* clock, eq_pool* pool) {
  const oracle_eq_node* x = &nodes[r];
  if (x->arity == ORACLE_EQ_LEAF) return;
  /* children by decreasing score, the earlier child first among equals */
  int32_t seq[3], nseq = 0, taken[3] = {0, 0, 0};
  for (int k = 0; k < x->arity; ++k) {
    int best = -1;
    for (int c = 0; c < x->arity; ++c)
      if (!taken[c] && (best < 0 || score[x->child[c]] > score[x->child[best]])) best = c;
    taken[best] = 1;
    seq[nseq++] = best;
  }
  for (int k = 0; k < nseq; ++k) eq_visit(nodes, x->child[seq[k]], score, ts, tmp, clock, pool);
  ts[r] = (*clock)++;
  int all_leaves = 1;
  for (int c = 0; c < x->arity; ++c) all_leaves &= nodes[x->child[c]].arity == ORACLE_EQ_LEAF;
  if (all_leaves) {
    tmp[r] = eq_reserve(pool);
    return;
  }
  /* the child whose tmp the node takes: Left, else (ternary) Right, else Middle / Right */
  int keep;
  if (nodes[x->child[0]].arity != ORACLE_EQ_LEAF) {
    keep = 0;
  } else if (x->arity == ORACLE_EQ_TERNARY && nodes[x->child[2]].arity != ORACLE_EQ_LEAF) {
    keep = 2;
  } else {
    keep = 1;
  }
  tmp[r] = tmp[x->child[keep]];
  for (int c = 0; c < x->arity; ++c)
    if (c != keep) eq_recycle(pool, tmp[x->child[c]]);
}

int oracle_eq_plan(const oracle_eq_node* nodes, int32_t n_nodes, int32_t root,
                   const int32_t* score, int32_t* timestamp, int32_t* tmp, int32_t* n_tmps) {
  if (!nodes || !score || !timestamp || !tmp || !n_tmps) return -1;
  if (eq_check(nodes, n_nodes, root, 0) != 0) return -1;
  for (int32_t i = 0; i < n_nodes; ++i) timestamp[i] = tmp[i] = -1;
  eq_pool pool;
  memset(&pool, 0, sizeof pool);
  int32_t clock = 0;
  eq_visit(nodes, root, score, timestamp, tmp, &clock, &pool);
  *n_tmps = pool.high;
  return 0;
}

static double eq_value(const oracle_eq_node* nodes, int32_t r, const oracle_eq_leaf* leaves,
                       int32_t row, int32_t col) {
  const oracle_eq_node* x = &nodes[r];
  if (x->arity == ORACLE_EQ_LEAF) {
    const oracle_eq_leaf* L = &leaves[x->leaf];
    int64_t at = 0;
    if (L->bcast == ORACLE_BC_NONE) at = (int64_t)row + (int64_t)col * L->ld;
    else if (L->bcast == ORACLE_BC_COL) at = row;
    else if (L->bcast == ORACLE_BC_ROW) at = col;
    return oracle_widen(L->ptr, at, L->dtype);
  }
  const double a = eq_value(nodes, x->child[0], leaves, row, col);
  if (x->arity == ORACLE_EQ_UNARY) {
    switch (x->op) {
      case ORACLE_EQ_IDENTITY: return a;
      case ORACLE_EQ_NEG: return -a;
      case ORACLE_EQ_EXP: return exp(a);
      case ORACLE_EQ_TANH: return tanh(a);
      case ORACLE_EQ_RELU: return a > 0.0 ? a : 0.0;
      case ORACLE_EQ_GELU_TANH: return oracle_gelu_tanh(a);
      case ORACLE_EQ_SQRT: return sqrt(a);
      case ORACLE_EQ_RCP: return 1.0 / a;
      case ORACLE_EQ_SQUARE: return a * a;
      default: return 1.0 / (1.0 + exp(-a));   /* sigmoid */
    }
  }
  const double b = eq_value(nodes, x->child[1], leaves, row, col);
  if (x->arity == ORACLE_EQ_BINARY) {
    switch (x->op) {
      case ORACLE_EQ_ADD: return a + b;
      case ORACLE_EQ_SUB: return a - b;
      case ORACLE_EQ_MUL: return a * b;
      case ORACLE_EQ_DIV: return a / b;
      case ORACLE_EQ_MAX: return a > b ? a : b;
      default: return a < b ? a : b;             /* min */
    }
  }
  const double c = eq_value(nodes, x->child[2], leaves, row, col);
  return a * b + c;                               /* muladd */
}

static int eq_op_ok(const oracle_eq_node* x) {
  if (x->arity == ORACLE_EQ_UNARY) return x->op >= ORACLE_EQ_IDENTITY && x->op <= ORACLE_EQ_SIGMOID;
  if (x->arity == ORACLE_EQ_BINARY) return x->op >= ORACLE_EQ_ADD && x->op <= ORACLE_EQ_MIN;
  if (x->arity == ORACLE_EQ_TERNARY) return x->op == ORACLE_EQ_MULADD;
  return 1;
}

int oracle_eq_eval(const oracle_eq_node* nodes, int32_t n_nodes, int32_t root, int32_t m,
                   int32_t n, const oracle_eq_leaf* leaves, int32_t n_leaves, void* out,
                   int64_t ldo, int32_t out_type, double* ref64) {
  if (!nodes || eq_check(nodes, n_nodes, root, 0) != 0 || m < 0 || n < 0 || ldo < m) return -1;
  for (int32_t i = 0; i < n_nodes; ++i) {
    if (!eq_op_ok(&nodes[i])) return -1;
    if (nodes[i].arity == ORACLE_EQ_LEAF && (nodes[i].leaf < 0 || nodes[i].leaf >= n_leaves))
      return -1;
  }
  for (int32_t col = 0; col < n; ++col)
    for (int32_t row = 0; row < m; ++row) {
      const double v = eq_value(nodes, root, leaves, row, col);
      if (ref64) ref64[(int64_t)row + (int64_t)col * m] = v;
      store_rounded(out, (int64_t)row + (int64_t)col * ldo, out_type, v);
    }
  return 0;
}
