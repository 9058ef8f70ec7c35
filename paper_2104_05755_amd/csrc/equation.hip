// equation.hip -- TPP matrix equations (Sec. 4) for gfx950: the planner of Alg. 3 / Alg. 4 on the
// host, and an executor that evaluates the planned instruction list per output element.
//
// Executor (see equation_kernel): eight output elements per thread; each instruction of the plan
// dispatches once and then runs over the eight elements.  The temporaries of the plan are named
// registers, so the plan's reuse of temporaries is register reuse: the paper's Strategy 2.  The
// instruction list lives in the kernel arguments and is read with scalar loads.
#include <hip/hip_runtime.h>

#include <math.h>

#include <vector>

#include "brgemm_device.h"
#include "internal.h"

namespace tpp {

// ---- planner (host) --------------------------------------------------------------------------
namespace {

bool op_fits(int32_t arity, int32_t op) {
  switch (arity) {
    case TPP_EQ_LEAF: return true;
    case TPP_EQ_UNARY: return op >= TPP_EQ_IDENTITY && op <= TPP_EQ_SIGMOID;
    case TPP_EQ_BINARY: return op >= TPP_EQ_ADD && op <= TPP_EQ_MIN;
    case TPP_EQ_TERNARY: return op == TPP_EQ_MULADD;
    default: return false;
  }
}

bool is_leaf(const tpp_eq_node* nodes, int32_t i) { return nodes[i].arity == TPP_EQ_LEAF; }

// Nodes reachable from the root in post-order (children before parents), checking that every
// reachable node is reached once and well formed.  Iterative, with an explicit stack.
const char* post_order(const tpp_eq_node* nodes, int32_t n_nodes, int32_t root,
                       std::vector<int32_t>& order) {
  if (root < 0 || root >= n_nodes) return "root index out of range";
  std::vector<char> seen(n_nodes, 0);
  std::vector<std::pair<int32_t, int32_t>> stack;   // (node, next child to visit)
  stack.push_back({root, 0});
  seen[root] = 1;
  while (!stack.empty()) {
    auto& top = stack.back();
    const tpp_eq_node& x = nodes[top.first];
    if (x.arity < TPP_EQ_LEAF || x.arity > TPP_EQ_TERNARY) return "arity outside [0, 3]";
    if (!op_fits(x.arity, x.op)) return "operation of the wrong arity";
    if (top.second < x.arity) {
      const int32_t c = x.child[top.second++];
      if (c < 0 || c >= n_nodes) return "child index out of range";
      if (seen[c]) return "a node is reached twice (not a tree)";
      seen[c] = 1;
      stack.push_back({c, 0});
    } else {
      order.push_back(top.first);
      stack.pop_back();
    }
  }
  return nullptr;
}

struct TmpPool {
  uint64_t used = 0;
  int32_t high = 0;
  int32_t reserve() {   // the lowest free id
    int32_t i = 0;
    while (used >> i & 1) ++i;
    used |= uint64_t(1) << i;
    if (i + 1 > high) high = i + 1;
    return i;
  }
  void recycle(int32_t t) {
    if (t >= 0) used &= ~(uint64_t(1) << t);
  }
};

void plan_node(const tpp_eq_node* nodes, int32_t r, tpp_eq_plan_node* plan, int32_t& clock,
               TmpPool& pool) {
  const tpp_eq_node& x = nodes[r];
  if (x.arity == TPP_EQ_LEAF) return;
  // children by decreasing score; among equal scores the earlier child first (stable)
  int32_t idx[3] = {0, 1, 2};
  for (int a = 1; a < x.arity; ++a)
    for (int b = a; b > 0 && plan[x.child[idx[b]]].score > plan[x.child[idx[b - 1]]].score; --b) {
      const int32_t t = idx[b];
      idx[b] = idx[b - 1];
      idx[b - 1] = t;
    }
  for (int a = 0; a < x.arity; ++a) plan_node(nodes, x.child[idx[a]], plan, clock, pool);
  plan[r].timestamp = clock++;
  bool all_leaves = true;
  for (int a = 0; a < x.arity; ++a) all_leaves = all_leaves && is_leaf(nodes, x.child[a]);
  if (all_leaves) {
    plan[r].tmp = pool.reserve();
    return;
  }
  // the temporary the node takes over: Left's, else Right's (ternary), else the other child's
  int keep = 1;
  if (!is_leaf(nodes, x.child[0])) keep = 0;
  else if (x.arity == TPP_EQ_TERNARY && !is_leaf(nodes, x.child[2])) keep = 2;
  plan[r].tmp = plan[x.child[keep]].tmp;
  for (int a = 0; a < x.arity; ++a)
    if (a != keep) pool.recycle(plan[x.child[a]].tmp);
}

}  // namespace

const char* equation_plan(const tpp_eq_node* nodes, int32_t n_nodes, int32_t root,
                          tpp_eq_plan_node* plan, int32_t* n_tmps) {
  if (!nodes || !plan || !n_tmps) return "NULL nodes, plan or n_tmps";
  if (n_nodes < 1 || n_nodes > EQ_MAX_NODES) return "n_nodes must be in [1, 64]";
  std::vector<int32_t> order;
  if (const char* err = post_order(nodes, n_nodes, root, order)) return err;
  for (int32_t i = 0; i < n_nodes; ++i) plan[i] = {0, -1, -1};
  // Alg. 3 over the post-order (children are scored before their parent)
  for (int32_t r : order) {
    const tpp_eq_node& x = nodes[r];
    int32_t s = 0;
    if (x.arity == TPP_EQ_UNARY) {
      s = is_leaf(nodes, x.child[0]) ? 1 : plan[x.child[0]].score;
    } else if (x.arity == TPP_EQ_BINARY) {
      const int32_t a = plan[x.child[0]].score, b = plan[x.child[1]].score;
      s = a == b ? a + 1 : (a > b ? a : b);
    } else if (x.arity == TPP_EQ_TERNARY) {
      if (is_leaf(nodes, x.child[0]) && is_leaf(nodes, x.child[1]) && is_leaf(nodes, x.child[2])) {
        s = 1;
      } else {
        s = 3;
        for (int a = 0; a < 3; ++a)
          if (plan[x.child[a]].score > s) s = plan[x.child[a]].score;
      }
    }
    plan[r].score = s;
  }
  // Alg. 4
  int32_t clock = 0;
  TmpPool pool;
  plan_node(nodes, root, plan, clock, pool);
  *n_tmps = pool.high;
  return nullptr;
}

const char* equation_compile(const tpp_eq_node* nodes, int32_t n_nodes, int32_t root,
                             EqProgram& prog, bool* too_many_tmps) {
  *too_many_tmps = false;
  tpp_eq_plan_node plan[EQ_MAX_NODES];
  int32_t n_tmps = 0;
  if (const char* err = equation_plan(nodes, n_nodes, root, plan, &n_tmps)) return err;
  if (nodes[root].arity == TPP_EQ_LEAF) {   // the output is a copy of one leaf
    prog.n_instr = 1;
    prog.instr[0] = {TPP_EQ_IDENTITY, 1, 0, {EQ_LEAF_BASE + nodes[root].leaf, 0, 0}};
    prog.result = 0;
    return nullptr;
  }
  if (n_tmps > EQ_MAX_TMPS) {
    *too_many_tmps = true;
    return "the plan needs more than 8 temporaries";
  }
  int32_t n_instr = 0;
  for (int32_t i = 0; i < n_nodes; ++i)
    if (plan[i].timestamp >= 0) ++n_instr;
  for (int32_t i = 0; i < n_nodes; ++i) {
    const int32_t t = plan[i].timestamp;
    if (t < 0) continue;
    const tpp_eq_node& x = nodes[i];
    EqInstr& in = prog.instr[t];
    in.op = x.op;
    in.arity = x.arity;
    in.dst = plan[i].tmp;
    for (int a = 0; a < 3; ++a) {
      if (a >= x.arity) {
        in.src[a] = 0;
        continue;
      }
      const int32_t c = x.child[a];
      in.src[a] = is_leaf(nodes, c) ? EQ_LEAF_BASE + nodes[c].leaf : plan[c].tmp;
    }
  }
  prog.n_instr = n_instr;
  prog.result = plan[root].tmp;
  return nullptr;
}

// ---- executor (device) -----------------------------------------------------------------------
namespace {

using namespace dev;

constexpr int EQ_T = 256;   // threads per workgroup

constexpr int EPT = 8;   // output elements per thread

// v[k] = op(a[k], b[k], cc[k]) for the EPT elements, one dispatch on op.
#define TPP_EQ_OP_CASE(op, expr) \
  case op: { _Pragma("unroll") for (int k = 0; k < EPT; ++k) v[k] = (expr); } break;
#define TPP_EQ_APPLY(opcode)                                                                    \
  switch (opcode) {                                                                             \
    TPP_EQ_OP_CASE(TPP_EQ_IDENTITY, a[k])                                                       \
    TPP_EQ_OP_CASE(TPP_EQ_NEG, -a[k])                                                           \
    TPP_EQ_OP_CASE(TPP_EQ_EXP, expf(a[k]))                                                      \
    TPP_EQ_OP_CASE(TPP_EQ_TANH, tanhf(a[k]))                                                    \
    TPP_EQ_OP_CASE(TPP_EQ_RELU, a[k] > 0.0f ? a[k] : 0.0f)                                      \
    TPP_EQ_OP_CASE(TPP_EQ_GELU_TANH, gelu_tanh(a[k]))                                           \
    TPP_EQ_OP_CASE(TPP_EQ_SQRT, sqrtf(a[k]))                                                    \
    TPP_EQ_OP_CASE(TPP_EQ_RCP, 1.0f / a[k])                                                     \
    TPP_EQ_OP_CASE(TPP_EQ_SQUARE, a[k] * a[k])                                                  \
    TPP_EQ_OP_CASE(TPP_EQ_SIGMOID, 1.0f / (1.0f + expf(-a[k])))                                 \
    TPP_EQ_OP_CASE(TPP_EQ_ADD, a[k] + b[k])                                                     \
    TPP_EQ_OP_CASE(TPP_EQ_SUB, a[k] - b[k])                                                     \
    TPP_EQ_OP_CASE(TPP_EQ_MUL, a[k] * b[k])                                                     \
    TPP_EQ_OP_CASE(TPP_EQ_DIV, a[k] / b[k])                                                     \
    TPP_EQ_OP_CASE(TPP_EQ_MAX, a[k] > b[k] ? a[k] : b[k])                                       \
    TPP_EQ_OP_CASE(TPP_EQ_MIN, a[k] < b[k] ? a[k] : b[k])                                       \
    TPP_EQ_OP_CASE(TPP_EQ_MULADD, __builtin_fmaf(a[k], b[k], cc[k]))                            \
    default: { _Pragma("unroll") for (int k = 0; k < EPT; ++k) v[k] = 0.0f; } break;            \
  }


// EPT output elements per thread, in column-major element order: element k of thread t in
// workgroup b is e = (b * EPT + k) * EQ_T + t, so for every k a wavefront covers 64 consecutive
// elements (contiguous runs of every full-tensor leaf and of the output, whatever the shape: a
// 1 x n row of statistics as well as a tall tensor).  Each instruction of the plan dispatches
// once on its operands' kind and once on its operation, then runs over the EPT elements without
// further branches: the interpretation cost is shared by EPT elements.  The temporaries are
// named register arrays (the plan's reuse of temporaries is register reuse).  WIDE: m * n does
// not fit 32 bits.
template <bool OUT_BF16, bool WIDE>
__global__ __launch_bounds__(EQ_T) void equation_kernel(EqProgram p) {
  const int64_t total = (int64_t)p.m * p.n;
  const int64_t step = (int64_t)gridDim.x * EPT * EQ_T;
  for (int64_t e0 = (int64_t)blockIdx.x * EPT * EQ_T + threadIdx.x; e0 < total; e0 += step) {
    int32_t r[EPT], c[EPT];
    bool ok[EPT];
#pragma unroll
    for (int k = 0; k < EPT; ++k) {
      const int64_t e = e0 + (int64_t)k * EQ_T;
      ok[k] = e < total;
      const int64_t ee = ok[k] ? e : 0;   // element 0 stands in past the end
      c[k] = WIDE ? (int32_t)(ee / p.m) : (int32_t)((uint32_t)ee / (uint32_t)p.m);
      r[k] = (int32_t)(ee - (int64_t)c[k] * p.m);
    }
    float t0[EPT], t1[EPT], t2[EPT], t3[EPT], t4[EPT], t5[EPT], t6[EPT], t7[EPT];
    // FETCH: operand `code` of all EPT elements into o (a temporary, or a leaf loaded for each
    // element); PUT: v into temporary `code`.  Expanded in place (statement macros), so that
    // every array index is a compile-time constant and the arrays stay in registers.
#define TPP_EQ_TMP_CASE(j, o) \
    case j: { _Pragma("unroll") for (int k = 0; k < EPT; ++k) o[k] = t##j[k]; } break;
#define FETCH(code, o)                                                                          \
    switch (code) {                                                                             \
      TPP_EQ_TMP_CASE(0, o) TPP_EQ_TMP_CASE(1, o) TPP_EQ_TMP_CASE(2, o) TPP_EQ_TMP_CASE(3, o)     \
      TPP_EQ_TMP_CASE(4, o) TPP_EQ_TMP_CASE(5, o) TPP_EQ_TMP_CASE(6, o) TPP_EQ_TMP_CASE(7, o)     \
      default: {                                                                                \
        const EqArg& g = p.arg[(code) - EQ_LEAF_BASE];                                          \
        _Pragma("unroll") for (int k = 0; k < EPT; ++k) {                                       \
          const int64_t at = g.bcast == TPP_BC_NONE ? (int64_t)r[k] + (int64_t)c[k] * g.ld      \
                             : g.bcast == TPP_BC_COL ? r[k] : g.bcast == TPP_BC_ROW ? c[k] : 0; \
          o[k] = g.bf16 ? bf16_bits_to_f32(gld<uint16_t>(static_cast<const uint16_t*>(g.ptr) + at)) \
                        : gld<float>(static_cast<const float*>(g.ptr) + at);                    \
        }                                                                                       \
      } break;                                                                                  \
    }
#define TPP_EQ_PUT_CASE(j) \
    case j: { _Pragma("unroll") for (int k = 0; k < EPT; ++k) t##j[k] = v[k]; } break;
#define PUT(code)                                                                               \
    switch (code) {                                                                             \
      TPP_EQ_PUT_CASE(0) TPP_EQ_PUT_CASE(1) TPP_EQ_PUT_CASE(2) TPP_EQ_PUT_CASE(3)                \
      TPP_EQ_PUT_CASE(4) TPP_EQ_PUT_CASE(5) TPP_EQ_PUT_CASE(6) TPP_EQ_PUT_CASE(7)                \
      default: break;                                                                           \
    }
    for (int32_t i = 0; i < p.n_instr; ++i) {
      const EqInstr& in = p.instr[i];
      float a[EPT], b[EPT], cc[EPT], v[EPT];
      FETCH(in.src[0], a)
      if (in.arity > 1) { FETCH(in.src[1], b) }
      if (in.arity > 2) { FETCH(in.src[2], cc) }
      TPP_EQ_APPLY(in.op)
      PUT(in.dst)
    }
    float res[EPT];
    FETCH(p.result, res)
#undef FETCH
#undef PUT
#undef TPP_EQ_TMP_CASE
#undef TPP_EQ_PUT_CASE
#pragma unroll
    for (int k = 0; k < EPT; ++k) {
      if (!ok[k]) continue;
      const int64_t at = (int64_t)r[k] + (int64_t)c[k] * p.ldo;
      if (OUT_BF16)
        gst<uint16_t>(static_cast<uint16_t*>(p.out) + at, f32_to_bf16_bits(res[k]));
      else
        gst<float>(static_cast<float*>(p.out) + at, res[k]);
    }
  }
}

// Small outputs (at most EQ_SMALL elements, e.g. a 1 x n row of statistics): one element per
// thread, so that the grid has as many workgroups as the elements allow, and every leaf of the
// element loaded before the first instruction runs, so that one memory latency replaces the
// chain of leaf loads the interpreter would otherwise wait for one instruction at a time.  The
// leaves and temporaries are named registers (indices dispatched by switch, never computed).
constexpr int64_t EQ_SMALL = 1 << 16;

__device__ __forceinline__ float eq_apply1(int32_t op, float a, float b, float c) {
  switch (op) {
    case TPP_EQ_IDENTITY: return a;
    case TPP_EQ_NEG: return -a;
    case TPP_EQ_EXP: return expf(a);
    case TPP_EQ_TANH: return tanhf(a);
    case TPP_EQ_RELU: return a > 0.0f ? a : 0.0f;
    case TPP_EQ_GELU_TANH: return gelu_tanh(a);
    case TPP_EQ_SQRT: return sqrtf(a);
    case TPP_EQ_RCP: return 1.0f / a;
    case TPP_EQ_SQUARE: return a * a;
    case TPP_EQ_SIGMOID: return 1.0f / (1.0f + expf(-a));
    case TPP_EQ_ADD: return a + b;
    case TPP_EQ_SUB: return a - b;
    case TPP_EQ_MUL: return a * b;
    case TPP_EQ_DIV: return a / b;
    case TPP_EQ_MAX: return a > b ? a : b;
    case TPP_EQ_MIN: return a < b ? a : b;
    case TPP_EQ_MULADD: return __builtin_fmaf(a, b, c);
    default: return 0.0f;
  }
}

template <bool OUT_BF16>
__global__ __launch_bounds__(EQ_T) void equation_small_kernel(EqProgram p) {
  const int32_t total = p.m * p.n;   // at most EQ_SMALL
  const int32_t e = (int32_t)blockIdx.x * EQ_T + (int32_t)threadIdx.x;
  if (e >= total) return;
  const int32_t c = e / p.m, r = e - c * p.m;
  // every leaf of this element, all loads issued before any is used
  float l0 = 0.0f, l1 = 0.0f, l2 = 0.0f, l3 = 0.0f, l4 = 0.0f, l5 = 0.0f, l6 = 0.0f, l7 = 0.0f;
  float l8 = 0.0f, l9 = 0.0f, l10 = 0.0f, l11 = 0.0f, l12 = 0.0f, l13 = 0.0f, l14 = 0.0f,
        l15 = 0.0f;
  auto leaf = [&](int j) -> float {
    const EqArg& g = p.arg[j];
    const int64_t at = g.bcast == TPP_BC_NONE ? (int64_t)r + (int64_t)c * g.ld
                       : g.bcast == TPP_BC_COL ? r : g.bcast == TPP_BC_ROW ? c : 0;
    return g.bf16 ? bf16_bits_to_f32(gld<uint16_t>(static_cast<const uint16_t*>(g.ptr) + at))
                  : gld<float>(static_cast<const float*>(g.ptr) + at);
  };
#define TPP_EQ_LEAF_LOAD(j) \
  if (j < p.n_args) l##j = leaf(j);
  TPP_EQ_LEAF_LOAD(0) TPP_EQ_LEAF_LOAD(1) TPP_EQ_LEAF_LOAD(2) TPP_EQ_LEAF_LOAD(3)
  TPP_EQ_LEAF_LOAD(4) TPP_EQ_LEAF_LOAD(5) TPP_EQ_LEAF_LOAD(6) TPP_EQ_LEAF_LOAD(7)
  TPP_EQ_LEAF_LOAD(8) TPP_EQ_LEAF_LOAD(9) TPP_EQ_LEAF_LOAD(10) TPP_EQ_LEAF_LOAD(11)
  TPP_EQ_LEAF_LOAD(12) TPP_EQ_LEAF_LOAD(13) TPP_EQ_LEAF_LOAD(14) TPP_EQ_LEAF_LOAD(15)
#undef TPP_EQ_LEAF_LOAD
  static_assert(EQ_MAX_ARGS == 16 && EQ_MAX_TMPS == 8 && EQ_LEAF_BASE == 16,
                "one named register per leaf and temporary");
  float t0 = 0.0f, t1 = 0.0f, t2 = 0.0f, t3 = 0.0f, t4 = 0.0f, t5 = 0.0f, t6 = 0.0f, t7 = 0.0f;
  auto get = [&](int32_t code) -> float {
    switch (code) {
      case 0: return t0; case 1: return t1; case 2: return t2; case 3: return t3;
      case 4: return t4; case 5: return t5; case 6: return t6; case 7: return t7;
      case 16: return l0; case 17: return l1; case 18: return l2; case 19: return l3;
      case 20: return l4; case 21: return l5; case 22: return l6; case 23: return l7;
      case 24: return l8; case 25: return l9; case 26: return l10; case 27: return l11;
      case 28: return l12; case 29: return l13; case 30: return l14; case 31: return l15;
      default: return 0.0f;
    }
  };
  for (int32_t i = 0; i < p.n_instr; ++i) {
    const EqInstr& in = p.instr[i];
    const float a = get(in.src[0]);
    const float b = in.arity > 1 ? get(in.src[1]) : 0.0f;
    const float cc = in.arity > 2 ? get(in.src[2]) : 0.0f;
    const float v = eq_apply1(in.op, a, b, cc);
    switch (in.dst) {
      case 0: t0 = v; break; case 1: t1 = v; break; case 2: t2 = v; break; case 3: t3 = v; break;
      case 4: t4 = v; break; case 5: t5 = v; break; case 6: t6 = v; break; case 7: t7 = v; break;
      default: break;
    }
  }
  const float res = get(p.result);
  const int64_t at = (int64_t)r + (int64_t)c * p.ldo;
  if (OUT_BF16)
    gst<uint16_t>(static_cast<uint16_t*>(p.out) + at, f32_to_bf16_bits(res));
  else
    gst<float>(static_cast<float*>(p.out) + at, res);
}

// Vector path: m a multiple of 8, every full-tensor and column leaf and the output 16-byte
// aligned with whole 16-byte units per column (checked on the host).  A thread takes 8 consecutive
// rows of one column (one index split per thread), loads 8 entries of a full or column leaf with
// 16-byte loads, one entry of a row or scalar leaf, and stores its 8 outputs with 16-byte stores.
// NTMP: the temporaries the plan uses are below NTMP (fewer registers, more waves in flight).
template <bool OUT_BF16, int NTMP>
__global__ __launch_bounds__(EQ_T) void equation_vec_kernel(EqProgram p) {
  const int64_t groups = (int64_t)p.m * p.n / EPT;
  for (int64_t gidx = (int64_t)blockIdx.x * EQ_T + threadIdx.x; gidx < groups;
       gidx += (int64_t)gridDim.x * EQ_T) {
    const int64_t e0 = gidx * EPT;
    const int32_t c = (int32_t)(e0 / p.m);
    const int32_t r = (int32_t)(e0 - (int64_t)c * p.m);
    float t0[EPT], t1[EPT], t2[EPT], t3[EPT], t4[EPT], t5[EPT], t6[EPT], t7[EPT];
#define TPP_EQ_TMP_CASE(j, o) \
    case j: if constexpr (j < NTMP) { _Pragma("unroll") for (int k = 0; k < EPT; ++k) o[k] = t##j[k]; } break;
#define FETCH(code, o)                                                                          \
    switch (code) {                                                                             \
      TPP_EQ_TMP_CASE(0, o) TPP_EQ_TMP_CASE(1, o) TPP_EQ_TMP_CASE(2, o) TPP_EQ_TMP_CASE(3, o)     \
      TPP_EQ_TMP_CASE(4, o) TPP_EQ_TMP_CASE(5, o) TPP_EQ_TMP_CASE(6, o) TPP_EQ_TMP_CASE(7, o)     \
      default: {                                                                                \
        const EqArg& g = p.arg[(code) - EQ_LEAF_BASE];                                          \
        if (g.bcast == TPP_BC_NONE || g.bcast == TPP_BC_COL) {                                  \
          const int64_t at = g.bcast == TPP_BC_NONE ? (int64_t)r + (int64_t)c * g.ld : r;       \
          if (g.bf16) {                                                                         \
            const u32x4 w = gld<u32x4>(static_cast<const uint16_t*>(g.ptr) + at);              \
            _Pragma("unroll") for (int q = 0; q < 4; ++q) {                                     \
              o[2 * q] = __uint_as_float(w[q] << 16);                                           \
              o[2 * q + 1] = __uint_as_float(w[q] & 0xffff0000u);                               \
            }                                                                                   \
          } else {                                                                              \
            const f32x4 lo = gld<f32x4>(static_cast<const float*>(g.ptr) + at);                \
            const f32x4 hi = gld<f32x4>(static_cast<const float*>(g.ptr) + at + 4);            \
            _Pragma("unroll") for (int q = 0; q < 4; ++q) { o[q] = lo[q]; o[q + 4] = hi[q]; }   \
          }                                                                                     \
        } else {                                                                                \
          const int64_t at = g.bcast == TPP_BC_ROW ? c : 0;                                     \
          const float x = g.bf16 ? bf16_bits_to_f32(gld<uint16_t>(static_cast<const uint16_t*>(g.ptr) + at)) \
                                 : gld<float>(static_cast<const float*>(g.ptr) + at);          \
          _Pragma("unroll") for (int k = 0; k < EPT; ++k) o[k] = x;                             \
        }                                                                                       \
      } break;                                                                                  \
    }
#define TPP_EQ_PUT_CASE(j) \
    case j: if constexpr (j < NTMP) { _Pragma("unroll") for (int k = 0; k < EPT; ++k) t##j[k] = v[k]; } break;
#define PUT(code)                                                                               \
    switch (code) {                                                                             \
      TPP_EQ_PUT_CASE(0) TPP_EQ_PUT_CASE(1) TPP_EQ_PUT_CASE(2) TPP_EQ_PUT_CASE(3)                \
      TPP_EQ_PUT_CASE(4) TPP_EQ_PUT_CASE(5) TPP_EQ_PUT_CASE(6) TPP_EQ_PUT_CASE(7)                \
      default: break;                                                                           \
    }
    for (int32_t i = 0; i < p.n_instr; ++i) {
      const EqInstr& in = p.instr[i];
      float a[EPT], b[EPT], cc[EPT], v[EPT];
      FETCH(in.src[0], a)
      if (in.arity > 1) { FETCH(in.src[1], b) }
      if (in.arity > 2) { FETCH(in.src[2], cc) }
      TPP_EQ_APPLY(in.op)
      PUT(in.dst)
    }
    float res[EPT];
    FETCH(p.result, res)
#undef FETCH
#undef PUT
#undef TPP_EQ_TMP_CASE
#undef TPP_EQ_PUT_CASE
    const int64_t at = (int64_t)r + (int64_t)c * p.ldo;
    if (OUT_BF16) {
      gst<u32x4>(static_cast<uint16_t*>(p.out) + at,
                 (u32x4){pack_bf16x2(res[0], res[1]), pack_bf16x2(res[2], res[3]),
                         pack_bf16x2(res[4], res[5]), pack_bf16x2(res[6], res[7])});
    } else {
      float* q = static_cast<float*>(p.out) + at;
      gst<f32x4>(q, (f32x4){res[0], res[1], res[2], res[3]});
      gst<f32x4>(q + 4, (f32x4){res[4], res[5], res[6], res[7]});
    }
  }
}

}  // namespace

// The vector path's conditions: m a multiple of 8; every full-tensor or column leaf and the
// output 16-byte aligned, with column strides of whole 16-byte units.
static bool prog_vec(const EqProgram& p) {
  const auto al = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; };
  if (p.m % EPT != 0 || !al(p.out) || (p.ldo * (p.out_bf16 ? 2 : 4)) % 16 != 0) return false;
  for (int32_t k = 0; k < p.n_args; ++k) {
    const EqArg& g = p.arg[k];
    if (g.bcast != TPP_BC_NONE && g.bcast != TPP_BC_COL) continue;
    if (!al(g.ptr)) return false;
    if (g.bcast == TPP_BC_NONE && (g.ld * (g.bf16 ? 2 : 4)) % 16 != 0) return false;
  }
  return true;
}

hipError_t launch_equation(const EqProgram& prog, hipStream_t stream) {
  if (prog.m == 0 || prog.n == 0) return hipSuccess;
  const int64_t total = (int64_t)prog.m * prog.n;
  // enough workgroups for every element once, at most 8 per CU on the 256 CUs (grid stride
  // beyond)
  int64_t blocks = (total + EPT * EQ_T - 1) / (EPT * EQ_T);
  if (blocks > 8 * 256) blocks = 8 * 256;
  const dim3 grid((unsigned)blocks);
  const bool wide = total > 0xffffffffLL;
  if (prog_vec(prog)) {
    int64_t vblocks = (total / EPT + EQ_T - 1) / EQ_T;
    if (vblocks > 8 * 256) vblocks = 8 * 256;
    int32_t ntmp = prog.result + 1;
    for (int32_t i = 0; i < prog.n_instr; ++i)
      if (prog.instr[i].dst + 1 > ntmp) ntmp = prog.instr[i].dst + 1;
    const dim3 vgrid((unsigned)vblocks);
#define TPP_EQ_VEC(B, N) hipLaunchKernelGGL((equation_vec_kernel<B, N>), vgrid, dim3(EQ_T), 0, stream, prog)
    if (prog.out_bf16) {
      if (ntmp <= 2) TPP_EQ_VEC(true, 2);
      else if (ntmp <= 4) TPP_EQ_VEC(true, 4);
      else TPP_EQ_VEC(true, EQ_MAX_TMPS);
    } else {
      if (ntmp <= 2) TPP_EQ_VEC(false, 2);
      else if (ntmp <= 4) TPP_EQ_VEC(false, 4);
      else TPP_EQ_VEC(false, EQ_MAX_TMPS);
    }
#undef TPP_EQ_VEC
  } else if (total <= EQ_SMALL) {
    const dim3 sgrid((unsigned)((total + EQ_T - 1) / EQ_T));
    if (prog.out_bf16)
      hipLaunchKernelGGL((equation_small_kernel<true>), sgrid, dim3(EQ_T), 0, stream, prog);
    else
      hipLaunchKernelGGL((equation_small_kernel<false>), sgrid, dim3(EQ_T), 0, stream, prog);
  } else if (prog.out_bf16) {
    if (wide) hipLaunchKernelGGL((equation_kernel<true, true>), grid, dim3(EQ_T), 0, stream, prog);
    else hipLaunchKernelGGL((equation_kernel<true, false>), grid, dim3(EQ_T), 0, stream, prog);
  } else {
    if (wide) hipLaunchKernelGGL((equation_kernel<false, true>), grid, dim3(EQ_T), 0, stream, prog);
    else hipLaunchKernelGGL((equation_kernel<false, false>), grid, dim3(EQ_T), 0, stream, prog);
  }
  return hipGetLastError();
}

}  // namespace tpp
