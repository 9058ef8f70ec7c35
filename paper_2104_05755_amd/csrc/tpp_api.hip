// tpp_api.hip -- the C ABI of include/tpp_brgemm.h, include/tpp_transform.h,
// include/tpp_embedding.h and include/tpp_equation.h: argument checks,
// the dispatch cache, kernel selection and launches.  Host code only; the kernels live in
// brgemm_kernels.hip, brgemm_dl_kernels.hip, reduce_kernels.hip, transform_kernels.hip,
// embedding_kernels.hip and equation.hip (which also holds the equation planner).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdlib>
#include <cstdio>
#include <cstring>
#include <memory>
#include <map>
#include <mutex>
#include <tuple>
#include <string>
#include <vector>

#include "internal.h"

struct tpp_brgemm_kernel_s {
  tpp_brgemm_desc desc;
  bool bf16;         // A/B are bf16 (else fp32)
  bool vec_ok;       // descriptor allows the 16-byte load path
  char name[96];
};

namespace {

thread_local std::string g_last_error;

tpp_status fail(tpp_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
tpp_status fail(tpp_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

tpp_status ok() {
  g_last_error.clear();
  return TPP_OK;
}

bool same_desc(const tpp_brgemm_desc& x, const tpp_brgemm_desc& y) {
  return x.m == y.m && x.n == y.n && x.k == y.k && x.lda == y.lda && x.ldb == y.ldb &&
         x.ldc == y.ldc && x.a_type == y.a_type && x.b_type == y.b_type && x.c_type == y.c_type &&
         x.comp_type == y.comp_type && std::memcmp(&x.beta, &y.beta, sizeof(float)) == 0 &&
         x.kind == y.kind && x.stride_a == y.stride_a && x.stride_b == y.stride_b &&
         x.flags == y.flags;
}

std::mutex g_cache_mu;
std::vector<std::unique_ptr<tpp_brgemm_kernel_s>>& cache() {
  static std::vector<std::unique_ptr<tpp_brgemm_kernel_s>> c;
  return c;
}

bool valid_dtype(int32_t t) { return t == TPP_DT_F32 || t == TPP_DT_BF16; }

// The direct-LDS kernels address each operand as a wave-uniform base (the first instance block a
// tile touches) plus a 32-bit per-lane byte offset: they apply when the grid steps are
// non-negative and the byte span one BM x BN tile can reach from that base stays below 2^31.
bool dl_offsets_fit(const tpp_brgemm_kernel_s& h, const tpp::BrgemmParams& p, int bm, int bn) {
  const int64_t m = h.desc.m, n = h.desc.n, k = h.desc.k, lda = h.desc.lda, ldb = h.desc.ldb;
  int64_t span_a, span_b;   // elements
  const int64_t block_a = p.a_trans ? m * lda + k : m + k * lda;   // one A_i block
  const int64_t block_b = p.b_trans ? k * ldb + n : n * ldb + k;   // one B_i block
  if (p.fused) {
    if (p.a_step_m < 0 || p.b_step_n < 0) return false;
    span_a = (bm / m + 2) * p.a_step_m + block_a;
    span_b = (bn / n + 2) * p.b_step_n + block_b;
  } else {
    span_a = block_a;
    span_b = block_b;
  }
  return span_a < (int64_t(1) << 30) && span_b < (int64_t(1) << 30);   // bf16: 2 bytes each
}

// Kernel choice for one launch.  bf16 inputs take a 16-byte-load instance when the descriptor
// and the grid keep every 8-element chunk contiguous and aligned (m, k, lda, ldb and all element
// steps multiples of 8); the tile shape is the largest that still gives two tiles per compute
// unit (512 tiles on the 256 CUs).  Anything else takes the element-load instance.
int32_t choose_kernel(const tpp_brgemm_kernel_s& h, const tpp::BrgemmParams& p) {
  if (!h.bf16) return (p.a_trans || p.b_trans) ? -1 : tpp::K_F32_GENERIC;
  bool vec = h.vec_ok;
  if (p.fused) vec = vec && (p.a_step_m % 8 == 0) && (p.b_step_n % 8 == 0);
  if (p.a_trans || p.b_trans) {
    // transposed operands: the 64-k direct-to-LDS instances only (-1: unsupported); a
    // transposed B moves 8 consecutive columns per 16-byte chunk
    if (!vec || h.desc.k % 64 != 0 || (p.b_trans && h.desc.n % 8 != 0)) return -1;
    const int32_t ids[] = {tpp::K_BF16_DL64K_256x256, tpp::K_BF16_DL64K_128x128,
                           tpp::K_BF16_DL64K_64x64};
    if (const char* env = std::getenv("TPP_FORCE_KERNEL")) {
      const int id = std::atoi(env);
      for (int32_t c : ids)
        if (c == id && dl_offsets_fit(h, p, tpp::kernel_tile_m(c), tpp::kernel_tile_n(c)))
          return id;
    }
    for (int32_t c : ids) {
      const int bm = tpp::kernel_tile_m(c), bn = tpp::kernel_tile_n(c);
      const bool last = bm == 64;
      if (!last && (bm > p.vrows || bn > p.vcols)) continue;
      if (!dl_offsets_fit(h, p, bm, bn)) continue;
      const int64_t tiles = p.groups * ((p.vrows + bm - 1) / bm) * ((p.vcols + bn - 1) / bn);
      const int64_t ktot = h.desc.kind == TPP_BR_ADDRESS ? 0 : p.count * (int64_t)h.desc.k;
      if (tiles >= 512 || last) return c;
      if (bm == 128 && ktot >= 8192 && tiles * 8 >= 512) return c;   // split (see below)
    }
    return -1;
  }
  if (!vec) return tpp::K_BF16_GENERIC;
  // Direct buffer->LDS instances when k is a multiple of 32, with 64-k stages when it is a
  // multiple of 64 (whole 128-byte lines of B per load); pointer lists only with 64-k stages
  // (measured faster than register staging there, slower with 32-k stages); register staging
  // otherwise.
  const bool bk64 = h.desc.k % 64 == 0;
  const bool dl_kind = h.desc.k % 32 == 0 && (h.desc.kind != TPP_BR_ADDRESS || bk64);
  if (const char* env = std::getenv("TPP_FORCE_KERNEL")) {
    const int id = std::atoi(env);
    const bool is_dl = tpp::kernel_k_step(id) > 1;
    if (id >= 0 && id < tpp::K_COUNT && id != tpp::K_BF16_GENERIC && id != tpp::K_F32_GENERIC &&
        (!is_dl || (h.desc.k % tpp::kernel_k_step(id) == 0 &&
                    dl_offsets_fit(h, p, tpp::kernel_tile_m(id), tpp::kernel_tile_n(id)))))
      return id;
  }
  struct Cand { int32_t dl_id, vec_id; int bm, bn; };
  const Cand cands[] = {
      {bk64 ? tpp::K_BF16_DL64K_256x256 : tpp::K_BF16_PP_256x256, tpp::K_BF16_256x256, 256, 256},
      {bk64 ? tpp::K_BF16_DL64K_128x128 : tpp::K_BF16_DL_128x128, tpp::K_BF16_128x128, 128, 128},
      {bk64 ? tpp::K_BF16_DL64K_64x64 : tpp::K_BF16_DL_64x64, tpp::K_BF16_64x64, 64, 64}};
  // total k of one instance's batch reduction (address kind: per instance, not known here)
  const int64_t ktot = h.desc.kind == TPP_BR_ADDRESS ? 0 : p.count * (int64_t)h.desc.k;
  for (const Cand& c : cands) {
    // never pad a virtual C out to a larger tile (the 64x64 tile is the floor)
    const bool last = c.bm == 64;
    if (!last && (c.bm > p.vrows || c.bn > p.vcols)) continue;
    const int64_t tiles = p.groups * ((p.vrows + c.bm - 1) / c.bm) * ((p.vcols + c.bn - 1) / c.bn);
    const bool dl = dl_kind && dl_offsets_fit(h, p, c.bm, c.bn);
    // two tiles per compute unit: one workgroup's barriers and epilogue overlap the other's MFMAs
    if (tiles >= 512 || last) return dl ? c.dl_id : c.vec_id;
    // a long batch reduction (weight gradients: all token blocks) makes up the parallelism by
    // splitting its stage list instead (see plan_launch): 128x128 tiles, two workgroups per
    // compute unit (measured on the MLP weight gradients, 1024 x 4096 outputs of 128 pairs: 87 us
    // against 94 unsplit and 96-101 for 256x256 tiles split 4)
    if (dl && bk64 && c.bm == 128 && ktot >= 8192 && tiles * 8 >= 512) return c.dl_id;
  }
  return tpp::K_BF16_64x64;
}

// Device work buffers for partial results, one per (device, stream, purpose) so that calls on
// different streams never share one; allocated on first use, grown when a call needs more (after
// a device synchronisation, since queued work may still use the old one), kept until exit.  The
// caller keeps `hold` (the cache's lock) until its kernels are enqueued, so another host thread
// cannot free the buffer between the lookup and the launch that uses it.
enum WorkPurpose { WORK_REDUCE = 0, WORK_SPLIT = 1 };
struct WorkBuffer {
  float* ptr = nullptr;
  int64_t floats = 0;
};
std::mutex g_work_mu;
std::map<std::tuple<int, void*, int>, WorkBuffer> g_work;

tpp_status work_buffer(int purpose, void* stream, int64_t floats, float** out,
                       std::unique_lock<std::mutex>& hold) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return fail(TPP_ERR_HIP, "hipGetDevice failed");
  hold = std::unique_lock<std::mutex>(g_work_mu);
  WorkBuffer& wb = g_work[std::make_tuple(dev, stream, purpose)];
  if (wb.floats < floats) {
    if (wb.ptr) {
      if (hipDeviceSynchronize() != hipSuccess || hipFree(wb.ptr) != hipSuccess)
        return fail(TPP_ERR_HIP, "could not release the old work buffer");
      wb.ptr = nullptr;
      wb.floats = 0;
    }
    void* ptr = nullptr;
    if (hipMalloc(&ptr, (size_t)floats * sizeof(float)) != hipSuccess)
      return fail(TPP_ERR_NO_MEMORY, "work buffer of %lld floats", (long long)floats);
    wb.ptr = static_cast<float*>(ptr);
    wb.floats = floats;
  }
  *out = wb.ptr;
  return TPP_OK;
}

// What one launch runs: the kernel instance, the split of its stage (or pair) list and the
// floats of work space the split's partial tiles need (0 without a split).  Host-only; no device
// work and no allocation.
struct LaunchPlan {
  int32_t id = -1;
  int32_t split = 1;
  int64_t ws_floats = 0;
};

tpp_status plan_launch(const tpp_brgemm_kernel_s* h, tpp::BrgemmParams& p, LaunchPlan& lp) {
  // the kernels count stages (pairs x k-steps of 32 or 64) and tiles in 32 bits
  const int64_t ksteps = (h->desc.k + 31) / 32;
  if (p.kind != TPP_BR_ADDRESS && p.count * ksteps >= (1LL << 31))
    return fail(TPP_ERR_UNSUPPORTED, "count * ceil(k/32) must be below 2^31");
  // Stride kind: every pair base is a + i*stride_a (+ an instance step), so 16-byte alignment of
  // all of them follows from the base pointers and the element steps, checked here once.
  if (p.kind == TPP_BR_STRIDE) {
    const auto al = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; };
    p.aligned = al(p.a) && al(p.b) && p.stride_a % 8 == 0 && p.stride_b % 8 == 0 &&
                (p.fused || !p.grid_form || (p.a_step_m % 8 == 0 && p.b_step_n % 8 == 0)) &&
                (p.fused || p.grid_form || (!p.a_off && !p.b_off));
  }
  const int32_t id = choose_kernel(*h, p);
  if (id < 0)
    return fail(TPP_ERR_UNSUPPORTED,
                "A_TRANS / B_TRANS need bf16, k %% 64 == 0, m, n, lda, ldb and element steps "
                "multiples of 8 and operand spans below 2^30 elements");
  lp = LaunchPlan();
  lp.id = id;
  const int bm = tpp::kernel_tile_m(id), bn = tpp::kernel_tile_n(id);
  if (id == tpp::K_F32_GENERIC && p.kind != TPP_BR_ADDRESS && p.count >= 2 &&
      !(p.flags & tpp::EPI_AUX_MASK)) {
    // A grid of few 64 x 64 tiles leaves most of the GPU idle while each workgroup walks the
    // whole pair list: split the list into chunks reduced by separate workgroups (about 256 in
    // all) and sum the chunks in a finishing kernel.
    const int64_t tiles = p.groups * ((p.vrows + 63) / 64) * ((p.vcols + 63) / 64);
    if (tiles < 128) {
      int64_t split = 256 / tiles;
      if (const char* env = std::getenv("TPP_SPLIT")) split = std::atoi(env);   // override
      if (split > p.count) split = p.count;
      if (split > 1) {
        lp.split = (int32_t)split;
        lp.ws_floats = tpp::f32_split_ws_floats(lp.split, tiles);
      }
    }
  }
  if (lp.split == 1 && tpp::kernel_k_step(id) > 1 && p.kind != TPP_BR_ADDRESS && p.count > 0) {
    // Direct-to-LDS kernel on a grid of too few tiles: split every tile's stage list into chunks
    // reduced by separate workgroups (about 512 in all for 128x128 tiles, two per compute unit,
    // else about 256; at least 8 stages each) and add the chunks in a finishing kernel.
    // TPP_SPLIT overrides the count.
    const int64_t tiles = p.groups * ((p.vrows + bm - 1) / bm) * ((p.vcols + bn - 1) / bn);
    const int64_t stages = p.count * (h->desc.k / tpp::kernel_k_step(id));
    const int64_t target = bm == 128 ? 512 : 256;
    int64_t split = 1;
    if (tiles < target && stages >= 16) {
      split = target / tiles;
      if (split > 8) split = 8;
      if (split > stages / 8) split = stages / 8;
    }
    if (const char* env = std::getenv("TPP_SPLIT")) split = std::atoi(env);
    if (split > stages) split = stages;
    if (split > 1) {
      lp.split = (int32_t)split;
      lp.ws_floats = split * tiles * (int64_t)bm * bn;
    }
  }
  return TPP_OK;
}

// Work space given by the caller of launch(): `floats` floats at `ptr` (ptr may be null when
// floats is 0).
struct FixedWorkspace {
  float* ptr;
  int64_t floats;
};

// Plan and launch.  fixed == nullptr: a split's work space comes from the per-stream work buffer
// (allocated or grown here); otherwise only from *fixed, and a plan that needs more is refused
// without launching anything.
tpp_status launch(const tpp_brgemm_kernel_s* h, tpp::BrgemmParams& p, void* stream,
                  const FixedWorkspace* fixed = nullptr) {
  LaunchPlan lp;
  if (tpp_status s = plan_launch(h, p, lp)) return s;
  p.split = lp.split;
  p.ws = nullptr;
  std::unique_lock<std::mutex> work_hold;   // held from a work-buffer lookup to the launch
  if (lp.split > 1) {
    if (fixed) {
      if (lp.ws_floats > fixed->floats || !fixed->ptr)
        return fail(TPP_ERR_UNSUPPORTED,
                    "this launch splits its reduction %d ways and needs %lld floats of work "
                    "space; the caller's holds %lld",
                    lp.split, (long long)lp.ws_floats, (long long)fixed->floats);
      p.ws = fixed->ptr;
    } else {
      const tpp_status st = work_buffer(WORK_SPLIT, stream, lp.ws_floats, &p.ws, work_hold);
      if (st != TPP_OK) return st;
    }
  }
  if (std::getenv("TPP_LOG")) {
    std::string name;
    tpp::BrgemmParams q = p;
    (void)tpp::launch_brgemm(q, lp.id, nullptr, &name);
    std::fprintf(stderr, "[tpp] %s: G=%lld vrows=%d vcols=%d fused=%d split=%d -> %s\n", h->name,
                 (long long)p.groups, p.vrows, p.vcols, p.fused, p.split, name.c_str());
  }
  const hipError_t e = tpp::launch_brgemm(p, lp.id, static_cast<hipStream_t>(stream));
  if (e != hipSuccess)
    return fail(TPP_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

void fill_common(const tpp_brgemm_kernel_s* h, tpp::BrgemmParams& p) {
  std::memset(&p, 0, sizeof p);
  const tpp_brgemm_desc& d = h->desc;
  p.m = d.m; p.n = d.n; p.k = d.k;
  p.lda = d.lda; p.ldb = d.ldb; p.ldc = d.ldc;
  p.beta = d.beta;
  // the layout bits travel as a_trans / b_trans
  p.flags = d.flags & ~(uint32_t)(TPP_LAYOUT_A_TRANS | TPP_LAYOUT_B_TRANS);
  p.a_trans = (d.flags & TPP_LAYOUT_A_TRANS) != 0;
  p.b_trans = (d.flags & TPP_LAYOUT_B_TRANS) != 0;
  p.c_bf16 = d.c_type == TPP_DT_BF16;
  p.kind = d.kind;
  p.stride_a = d.stride_a;
  p.stride_b = d.stride_b;
}

tpp_status check_handle(tpp_brgemm_handle h) {
  if (!h) return fail(TPP_ERR_INVALID_ARG, "NULL handle");
  return TPP_OK;
}

tpp_status check_bias(const tpp_brgemm_kernel_s* h, const float* bias) {
  if ((h->desc.flags & TPP_EPI_BIAS) && !bias)
    return fail(TPP_ERR_INVALID_ARG, "TPP_EPI_BIAS set but bias is NULL");
  return TPP_OK;
}

// The calls without an aux argument cannot run a handle whose epilogue reads or writes one.
tpp_status check_no_aux(const tpp_brgemm_kernel_s* h) {
  if (h->desc.flags & tpp::EPI_AUX_MASK)
    return fail(TPP_ERR_INVALID_ARG,
                "the handle's epilogue uses an aux tensor: call tpp_brgemm_execute_batched_aux");
  return TPP_OK;
}

// Single call = a batched call with one instance of a 1x1 strided grid.
tpp_status run_single(const tpp_brgemm_kernel_s* h, tpp::BrgemmParams& p, void* stream) {
  p.fused = 1;
  p.gm = p.gn = 1;
  p.groups = 1;
  p.vrows = p.m;
  p.vcols = p.n;
  return launch(h, p, stream);
}

}  // namespace

extern "C" {

const char* tpp_status_string(tpp_status s) {
  switch (s) {
    case TPP_OK: return "TPP_OK";
    case TPP_ERR_INVALID_ARG: return "TPP_ERR_INVALID_ARG";
    case TPP_ERR_UNSUPPORTED: return "TPP_ERR_UNSUPPORTED";
    case TPP_ERR_HIP: return "TPP_ERR_HIP";
    case TPP_ERR_NO_MEMORY: return "TPP_ERR_NO_MEMORY";
  }
  return "TPP_ERR_UNKNOWN";
}

const char* tpp_last_error_message(void) { return g_last_error.c_str(); }

tpp_status tpp_brgemm_dispatch(const tpp_brgemm_desc* desc, tpp_brgemm_handle* out) {
  if (!desc || !out) return fail(TPP_ERR_INVALID_ARG, "NULL desc or out");
  *out = nullptr;
  const tpp_brgemm_desc& d = *desc;
  if (d.m <= 0 || d.n <= 0 || d.k <= 0)
    return fail(TPP_ERR_INVALID_ARG, "m, n, k must be > 0 (got %d, %d, %d)", d.m, d.n, d.k);
  const bool a_trans = (d.flags & TPP_LAYOUT_A_TRANS) != 0;
  const bool b_trans = (d.flags & TPP_LAYOUT_B_TRANS) != 0;
  if (d.lda < (a_trans ? d.k : d.m) || d.ldb < (b_trans ? d.n : d.k) || d.ldc < d.m)
    return fail(TPP_ERR_INVALID_ARG, "leading dimension too small (lda %lld < m (k with A_TRANS), ldb %lld < k (n with "
                "B_TRANS) or ldc %lld < m)",
                (long long)d.lda, (long long)d.ldb, (long long)d.ldc);
  if (!valid_dtype(d.a_type) || !valid_dtype(d.b_type) || !valid_dtype(d.c_type) ||
      !valid_dtype(d.comp_type))
    return fail(TPP_ERR_INVALID_ARG, "unknown datatype code");
  if (d.a_type != d.b_type)
    return fail(TPP_ERR_UNSUPPORTED, "A and B must share a datatype");
  if (d.comp_type != TPP_DT_F32)
    return fail(TPP_ERR_UNSUPPORTED, "accumulation is fp32 only");
  if (d.kind != TPP_BR_STRIDE && d.kind != TPP_BR_OFFSET && d.kind != TPP_BR_ADDRESS)
    return fail(TPP_ERR_INVALID_ARG, "unknown batch kind %d", d.kind);
  if (d.flags & ~(uint32_t)(TPP_EPI_BIAS | TPP_EPI_RELU | TPP_EPI_GELU_TANH | tpp::EPI_AUX_MASK |
                            TPP_LAYOUT_A_TRANS | TPP_LAYOUT_B_TRANS))
    return fail(TPP_ERR_INVALID_ARG, "unknown flag bits 0x%x", d.flags);
  if ((d.flags & TPP_EPI_RELU) && (d.flags & TPP_EPI_GELU_TANH))
    return fail(TPP_ERR_INVALID_ARG, "RELU and GELU_TANH exclude each other");
  const uint32_t inv = TPP_EPI_RELU_INV | TPP_EPI_GELU_TANH_INV;
  if ((d.flags & inv) == inv)
    return fail(TPP_ERR_INVALID_ARG, "RELU_INV and GELU_TANH_INV exclude each other");
  if ((d.flags & inv) && (d.flags & (TPP_EPI_RELU | TPP_EPI_GELU_TANH | TPP_EPI_SAVE_PREACT)))
    return fail(TPP_ERR_INVALID_ARG,
                "an inverse activation excludes RELU, GELU_TANH and SAVE_PREACT");
  if ((d.flags & TPP_EPI_SAVE_PREACT) && !(d.flags & (TPP_EPI_RELU | TPP_EPI_GELU_TANH)))
    return fail(TPP_ERR_INVALID_ARG, "SAVE_PREACT needs RELU or GELU_TANH");
  if (!std::isfinite(d.beta)) return fail(TPP_ERR_INVALID_ARG, "beta must be finite");

  std::lock_guard<std::mutex> lock(g_cache_mu);
  for (auto& h : cache()) {
    if (same_desc(h->desc, d)) {
      *out = h.get();
      return ok();
    }
  }
  auto h = std::make_unique<tpp_brgemm_kernel_s>();
  h->desc = d;
  h->bf16 = d.a_type == TPP_DT_BF16;
  h->vec_ok = h->bf16 && d.m % 8 == 0 && d.k % 8 == 0 && d.lda % 8 == 0 && d.ldb % 8 == 0 &&
              (d.kind != TPP_BR_STRIDE || (d.stride_a % 8 == 0 && d.stride_b % 8 == 0));
  static const char* kinds[] = {"stride", "offset", "address"};
  std::snprintf(h->name, sizeof h->name, "brgemm_%s_%s_m%d_n%d_k%d_%s%s%s", h->bf16 ? "bf16" : "f32",
                d.c_type == TPP_DT_BF16 ? "bf16out" : "f32out", d.m, d.n, d.k, kinds[d.kind],
                h->vec_ok ? "_vec" : "_generic", a_trans ? (b_trans ? "_atrans_btrans" : "_atrans")
                                                 : (b_trans ? "_btrans" : ""));
  *out = h.get();
  cache().push_back(std::move(h));
  return ok();
}

void tpp_brgemm_release(tpp_brgemm_handle) {}

tpp_status tpp_brgemm_describe(tpp_brgemm_handle h, char* buf, size_t len) {
  if (tpp_status s = check_handle(h)) return s;
  if (!buf || len == 0) return fail(TPP_ERR_INVALID_ARG, "NULL buffer");
  std::snprintf(buf, len, "%s", h->name);
  return ok();
}

tpp_status tpp_brgemm_execute_stride(tpp_brgemm_handle h, const void* a, const void* b, void* c,
                                     const float* bias, int64_t count, void* stream) {
  if (tpp_status s = check_handle(h)) return s;
  if (h->desc.kind != TPP_BR_STRIDE)
    return fail(TPP_ERR_INVALID_ARG, "handle is not a stride-based BRGEMM");
  if (count < 0) return fail(TPP_ERR_INVALID_ARG, "count < 0");
  if (!c) return fail(TPP_ERR_INVALID_ARG, "NULL c");
  if (count > 0 && (!a || !b)) return fail(TPP_ERR_INVALID_ARG, "NULL a or b");
  if (tpp_status s = check_bias(h, bias)) return s;
  if (tpp_status s = check_no_aux(h)) return s;
  tpp::BrgemmParams p;
  fill_common(h, p);
  p.a = a; p.b = b; p.c = c; p.bias = bias;
  p.count = count;
  return run_single(h, p, stream);
}

tpp_status tpp_brgemm_execute_offset(tpp_brgemm_handle h, const void* a, const void* b,
                                     const int64_t* offs_a, const int64_t* offs_b, void* c,
                                     const float* bias, int64_t count, void* stream) {
  if (tpp_status s = check_handle(h)) return s;
  if (h->desc.kind != TPP_BR_OFFSET)
    return fail(TPP_ERR_INVALID_ARG, "handle is not an offset-based BRGEMM");
  if (count < 0) return fail(TPP_ERR_INVALID_ARG, "count < 0");
  if (!c) return fail(TPP_ERR_INVALID_ARG, "NULL c");
  if (count > 0 && (!a || !b || !offs_a || !offs_b))
    return fail(TPP_ERR_INVALID_ARG, "NULL a, b or offset array");
  if (tpp_status s = check_bias(h, bias)) return s;
  if (tpp_status s = check_no_aux(h)) return s;
  tpp::BrgemmParams p;
  fill_common(h, p);
  p.a = a; p.b = b; p.c = c; p.bias = bias;
  p.offs_a = offs_a; p.offs_b = offs_b;
  p.count = count;
  return run_single(h, p, stream);
}

tpp_status tpp_brgemm_execute_address(tpp_brgemm_handle h, const void* const* ptrs_a,
                                      const void* const* ptrs_b, void* c, const float* bias,
                                      int64_t count, void* stream) {
  if (tpp_status s = check_handle(h)) return s;
  if (h->desc.kind != TPP_BR_ADDRESS)
    return fail(TPP_ERR_INVALID_ARG, "handle is not an address-based BRGEMM");
  if (count < 0) return fail(TPP_ERR_INVALID_ARG, "count < 0");
  if (!c) return fail(TPP_ERR_INVALID_ARG, "NULL c");
  if (count > 0 && (!ptrs_a || !ptrs_b)) return fail(TPP_ERR_INVALID_ARG, "NULL pointer list");
  if (tpp_status s = check_bias(h, bias)) return s;
  if (tpp_status s = check_no_aux(h)) return s;
  tpp::BrgemmParams p;
  fill_common(h, p);
  p.c = c; p.bias = bias;
  p.ptrs_a = ptrs_a; p.ptrs_b = ptrs_b;
  // The kernel reads an address-kind pair list through begin[]; a single call is the list
  // [0, count), kept in the kernel arguments (no device array needed).
  p.kind = TPP_BR_ADDRESS;
  p.count = count;
  p.begin = nullptr;
  return run_single(h, p, stream);
}

}  // extern "C"

namespace {

// The arguments of a batched call checked and resolved into p.  *empty is set (and p left
// unfilled) for G == 0, which is a no-op.
tpp_status prepare_batched(tpp_brgemm_handle h, const tpp_grid_strided* grid, int64_t G,
                           const int64_t* d_a_off, const int64_t* d_b_off, const int64_t* d_c_off,
                           const int64_t* d_bias_off, const void* a, const void* b, void* c,
                           void* aux, const float* bias, int64_t count, const int64_t* d_offs_a,
                           const int64_t* d_offs_b, const int64_t* d_begin,
                           const void* const* d_ptrs_a, const void* const* d_ptrs_b,
                           tpp::BrgemmParams& p, bool* empty) {
  *empty = false;
  const tpp_brgemm_desc& d = h->desc;
  if (G < 0) return fail(TPP_ERR_INVALID_ARG, "G < 0");
  if (grid) {
    if (grid->gm <= 0 || grid->gn <= 0) return fail(TPP_ERR_INVALID_ARG, "grid gm, gn must be > 0");
    if (grid->gm * grid->gn != G)
      return fail(TPP_ERR_INVALID_ARG, "grid gm*gn (%lld) != G (%lld)",
                  (long long)(grid->gm * grid->gn), (long long)G);
    if (d_a_off || d_b_off || d_c_off || d_bias_off)
      return fail(TPP_ERR_INVALID_ARG, "offset arrays given together with a strided grid");
  }
  if (G == 0) {
    *empty = true;
    return ok();
  }
  if (!c) return fail(TPP_ERR_INVALID_ARG, "NULL c");
  if (tpp_status s = check_bias(h, bias)) return s;
  if ((d.flags & tpp::EPI_AUX_MASK) && !aux)
    return fail(TPP_ERR_INVALID_ARG, "the handle's epilogue needs the aux tensor (NULL aux)");
  if (d.kind == TPP_BR_ADDRESS) {
    if (!d_begin) return fail(TPP_ERR_INVALID_ARG, "address kind needs d_begin");
    if (!d_ptrs_a || !d_ptrs_b) return fail(TPP_ERR_INVALID_ARG, "NULL pointer list");
  } else {
    if (count < 0) return fail(TPP_ERR_INVALID_ARG, "count < 0");
    if (count > 0 && (!a || !b)) return fail(TPP_ERR_INVALID_ARG, "NULL a or b");
    if (d.kind == TPP_BR_OFFSET && count > 0 && (!d_offs_a || !d_offs_b))
      return fail(TPP_ERR_INVALID_ARG, "NULL offset array");
  }
  fill_common(h, p);
  p.a = a; p.b = b; p.c = c; p.bias = bias;
  p.count = count;
  p.offs_a = d_offs_a; p.offs_b = d_offs_b;
  p.begin = d_begin; p.ptrs_a = d_ptrs_a; p.ptrs_b = d_ptrs_b;
  p.a_off = d_a_off; p.b_off = d_b_off; p.c_off = d_c_off; p.bias_off = d_bias_off;
  p.aux = (d.flags & tpp::EPI_AUX_MASK) ? aux : nullptr;
  if (grid) {
    p.gm = grid->gm; p.gn = grid->gn;
    p.a_step_m = grid->a_step_m; p.b_step_n = grid->b_step_n;
    p.c_step_m = grid->c_step_m; p.c_step_n = grid->c_step_n;
    p.bias_step_m = grid->bias_step_m;
  }
  // A strided grid of stride/offset kind is fused into one virtual C when that C fits int32
  // indexing; address kind (one pair list per instance) and explicit grids tile per instance.
  const int64_t vr = grid ? grid->gm * (int64_t)d.m : d.m;
  const int64_t vc = grid ? grid->gn * (int64_t)d.n : d.n;
  const int64_t lim = (1LL << 31) - 512;
  if (grid && d.kind != TPP_BR_ADDRESS && vr < lim && vc < lim) {
    p.fused = 1;
    p.groups = 1;
    p.vrows = (int32_t)vr;
    p.vcols = (int32_t)vc;
  } else {
    p.fused = 0;
    p.grid_form = grid ? 1 : 0;
    p.groups = G;
    p.vrows = d.m;
    p.vcols = d.n;
  }
  return TPP_OK;
}

tpp_status execute_batched(tpp_brgemm_handle h, const tpp_grid_strided* grid, int64_t G,
                           const int64_t* d_a_off, const int64_t* d_b_off, const int64_t* d_c_off,
                           const int64_t* d_bias_off, const void* a, const void* b, void* c,
                           void* aux, const float* bias, int64_t count, const int64_t* d_offs_a,
                           const int64_t* d_offs_b, const int64_t* d_begin,
                           const void* const* d_ptrs_a, const void* const* d_ptrs_b,
                           void* stream, const FixedWorkspace* fixed = nullptr) {
  tpp::BrgemmParams p;
  bool empty = false;
  if (tpp_status s = prepare_batched(h, grid, G, d_a_off, d_b_off, d_c_off, d_bias_off, a, b, c,
                                     aux, bias, count, d_offs_a, d_offs_b, d_begin, d_ptrs_a,
                                     d_ptrs_b, p, &empty))
    return s;
  if (empty) return ok();
  return launch(h, p, stream, fixed);
}

// Scratch of the allocation-free batched call: the partial tiles of a split reduction.  One copy
// per GPU, held from the library's load until the process ends; every allocation-free call on a
// GPU uses that GPU's copy, so such calls that overlap in time on one GPU race.  Host code never
// uses the array's name as an address (in host code it is a stand-in, not device memory): the
// device address comes from hipGetSymbolAddress, once per device, with that device current.
constexpr int64_t kNoAllocScratchFloats = TPP_BRGEMM_NOALLOC_SCRATCH_BYTES / 4;
static __device__ __align__(256) float scratch[kNoAllocScratchFloats];

std::mutex g_scratch_mu;
std::map<int, float*> g_scratch_ptr;   // device -> address of that device's scratch

tpp_status scratch_address(float** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return fail(TPP_ERR_HIP, "hipGetDevice failed");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  auto it = g_scratch_ptr.find(dev);
  if (it == g_scratch_ptr.end()) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
      return fail(TPP_ERR_HIP, "hipGetSymbolAddress of the scratch array failed on device %d: %s",
                  dev, hipGetErrorString(e));
    it = g_scratch_ptr.emplace(dev, static_cast<float*>(ptr)).first;
  }
  *out = it->second;
  return TPP_OK;
}


}  // namespace

extern "C" {

tpp_status tpp_brgemm_execute_batched(tpp_brgemm_handle h, const tpp_grid_strided* grid,
                                      int64_t G, const int64_t* d_a_off, const int64_t* d_b_off,
                                      const int64_t* d_c_off, const int64_t* d_bias_off,
                                      const void* a, const void* b, void* c, const float* bias,
                                      int64_t count, const int64_t* d_offs_a,
                                      const int64_t* d_offs_b, const int64_t* d_begin,
                                      const void* const* d_ptrs_a, const void* const* d_ptrs_b,
                                      void* stream) {
  if (tpp_status s = check_handle(h)) return s;
  if (tpp_status s = check_no_aux(h)) return s;
  return execute_batched(h, grid, G, d_a_off, d_b_off, d_c_off, d_bias_off, a, b, c, nullptr,
                         bias, count, d_offs_a, d_offs_b, d_begin, d_ptrs_a, d_ptrs_b, stream);
}

tpp_status tpp_brgemm_execute_batched_aux(tpp_brgemm_handle h, const tpp_grid_strided* grid,
                                          int64_t G, const int64_t* d_a_off,
                                          const int64_t* d_b_off, const int64_t* d_c_off,
                                          const int64_t* d_bias_off, const void* a,
                                          const void* b, void* c, void* aux, const float* bias,
                                          int64_t count, const int64_t* d_offs_a,
                                          const int64_t* d_offs_b, const int64_t* d_begin,
                                          const void* const* d_ptrs_a,
                                          const void* const* d_ptrs_b, void* stream) {
  if (tpp_status s = check_handle(h)) return s;
  return execute_batched(h, grid, G, d_a_off, d_b_off, d_c_off, d_bias_off, a, b, c, aux, bias,
                         count, d_offs_a, d_offs_b, d_begin, d_ptrs_a, d_ptrs_b, stream);
}

tpp_status tpp_brgemm_execute_batched_noalloc(
    tpp_brgemm_handle h, const tpp_grid_strided* grid, int64_t G, const int64_t* d_a_off,
    const int64_t* d_b_off, const int64_t* d_c_off, const int64_t* d_bias_off, const void* a,
    const void* b, void* c, const float* bias, int64_t count, const int64_t* d_offs_a,
    const int64_t* d_offs_b, const int64_t* d_begin, const void* const* d_ptrs_a,
    const void* const* d_ptrs_b, void* stream) {
  if (tpp_status s = check_handle(h)) return s;
  if (tpp_status s = check_no_aux(h)) return s;
  tpp::BrgemmParams p;
  bool empty = false;
  if (tpp_status s = prepare_batched(h, grid, G, d_a_off, d_b_off, d_c_off, d_bias_off, a, b, c,
                                     nullptr, bias, count, d_offs_a, d_offs_b, d_begin, d_ptrs_a,
                                     d_ptrs_b, p, &empty))
    return s;
  if (empty) return ok();
  // The plan first (host only): a split that needs more than the scratch array is refused before
  // anything touches the device; a launch without a split never looks the array up.
  LaunchPlan lp;
  tpp::BrgemmParams q = p;
  if (tpp_status s = plan_launch(h, q, lp)) return s;
  float* ws = nullptr;
  if (lp.split > 1) {
    if (lp.ws_floats > kNoAllocScratchFloats)
      return fail(TPP_ERR_UNSUPPORTED,
                  "this launch splits its reduction %d ways and needs %lld bytes of scratch; the "
                  "allocation-free call holds %lld",
                  lp.split, (long long)lp.ws_floats * 4, (long long)kNoAllocScratchFloats * 4);
    if (tpp_status s = scratch_address(&ws)) return s;
  }
  const FixedWorkspace fixed = {ws, ws ? kNoAllocScratchFloats : 0};
  return launch(h, p, stream, &fixed);
}

tpp_status tpp_brgemm_describe_launch(
    tpp_brgemm_handle h, const tpp_grid_strided* grid, int64_t G, const int64_t* d_a_off,
    const int64_t* d_b_off, const int64_t* d_c_off, const int64_t* d_bias_off, const void* a,
    const void* b, void* c, const float* bias, int64_t count, const int64_t* d_offs_a,
    const int64_t* d_offs_b, const int64_t* d_begin, const void* const* d_ptrs_a,
    const void* const* d_ptrs_b, char* buf, size_t len) {
  if (tpp_status s = check_handle(h)) return s;
  if (!buf || len == 0) return fail(TPP_ERR_INVALID_ARG, "NULL buffer");
  buf[0] = 0;
  // a stand-in for the aux tensor: only its presence is checked, nothing is launched
  void* aux = (h->desc.flags & tpp::EPI_AUX_MASK) ? c : nullptr;
  tpp::BrgemmParams p;
  bool empty = false;
  if (tpp_status s = prepare_batched(h, grid, G, d_a_off, d_b_off, d_c_off, d_bias_off, a, b, c,
                                     aux, bias, count, d_offs_a, d_offs_b, d_begin, d_ptrs_a,
                                     d_ptrs_b, p, &empty))
    return s;
  std::string name;
  if (!empty) {
    LaunchPlan lp;
    if (tpp_status s = plan_launch(h, p, lp)) return s;
    p.split = lp.split;
    if (tpp::launch_brgemm(p, lp.id, nullptr, &name) != hipSuccess)
      return fail(TPP_ERR_UNSUPPORTED, "no kernel instance for this launch");
  }
  std::snprintf(buf, len, "%s", name.c_str());
  return ok();
}

}  // extern "C"

namespace {

tpp_status reduce_impl(int32_t m, int32_t n, int64_t ld, int32_t in_type, const void* in,
                       int64_t G, int64_t in_stride, int32_t op, uint32_t flags, float* out_x,
                       float* out_x2, int64_t out_stride, void* stream) {
  if (m <= 0 || n <= 0) return fail(TPP_ERR_INVALID_ARG, "m, n must be > 0");
  if (G < 0 || in_stride < 0 || out_stride < 0)
    return fail(TPP_ERR_INVALID_ARG, "G, in_stride and out_stride must be >= 0");
  if (ld < m) return fail(TPP_ERR_INVALID_ARG, "ld < m");
  if (!valid_dtype(in_type)) return fail(TPP_ERR_INVALID_ARG, "unknown datatype code");
  if (!in) return fail(TPP_ERR_INVALID_ARG, "NULL input");
  if (op < TPP_RED_SUM || op > TPP_RED_MAX) return fail(TPP_ERR_INVALID_ARG, "unknown op %d", op);
  if (flags & ~(uint32_t)(TPP_RED_BY_COLS | TPP_RED_BY_ROWS | TPP_RED_X | TPP_RED_X2))
    return fail(TPP_ERR_INVALID_ARG, "unknown reduce flag bits");
  const bool by_cols = flags & TPP_RED_BY_COLS, by_rows = flags & TPP_RED_BY_ROWS;
  if (by_cols == by_rows) return fail(TPP_ERR_INVALID_ARG, "set exactly one of BY_COLS, BY_ROWS");
  if (!(flags & (TPP_RED_X | TPP_RED_X2))) return fail(TPP_ERR_INVALID_ARG, "set X and/or X2");
  if ((flags & TPP_RED_X) && !out_x) return fail(TPP_ERR_INVALID_ARG, "NULL out_x");
  if ((flags & TPP_RED_X2) && !out_x2) return fail(TPP_ERR_INVALID_ARG, "NULL out_x2");
  if (G == 0) return ok();
  tpp::ReduceParams p{in, m, n, ld, in_type == TPP_DT_BF16, op, flags, out_x, out_x2,
                      G, in_stride, out_stride};
  const int64_t need = tpp::reduce_work_floats(p);
  if (need < 0) return fail(TPP_ERR_UNSUPPORTED, "reduce needs more than 2^31 - 1 workgroups");
  float* work = nullptr;
  std::unique_lock<std::mutex> work_hold;   // held from the work-buffer lookup to the launch
  if (need > 0) {
    const tpp_status st = work_buffer(WORK_REDUCE, stream, need, &work, work_hold);
    if (st != TPP_OK) return st;
  }
  const hipError_t e = tpp::launch_reduce(p, work, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(TPP_ERR_HIP, "reduce launch failed: %s", hipGetErrorString(e));
  return ok();
}

tpp_status transform_impl(int32_t kind, int32_t m, int32_t n, int64_t ld_in, int64_t ld_out,
                          int32_t dtype, int32_t alpha, const void* in, int64_t in_stride,
                          void* out, int64_t out_stride, int64_t G, void* stream) {
  if (G < 0 || in_stride < 0 || out_stride < 0)
    return fail(TPP_ERR_INVALID_ARG, "G, in_stride and out_stride must be >= 0");
  if (kind < TPP_TR_TRANSPOSE || kind > TPP_TR_VNNI_TO_VNNI_T)
    return fail(TPP_ERR_INVALID_ARG, "unknown transform kind %d", kind);
  if (!valid_dtype(dtype)) return fail(TPP_ERR_INVALID_ARG, "unknown datatype code");
  if (m < 0 || n < 0) return fail(TPP_ERR_INVALID_ARG, "m, n must be >= 0");
  if (kind == TPP_TR_TRANSPOSE) {
    alpha = 1;
    if (ld_in < m || ld_out < n) return fail(TPP_ERR_INVALID_ARG, "ld_in < m or ld_out < n");
  } else {
    if (alpha != 1 && alpha != 2 && alpha != 4)
      return fail(TPP_ERR_INVALID_ARG, "alpha must be 1, 2 or 4");
    if (kind == TPP_TR_VNNI && (ld_in < m || ld_out < (int64_t)m * alpha))
      return fail(TPP_ERR_INVALID_ARG, "VNNI needs ld_in >= m and ld_out >= m * alpha");
    if (kind == TPP_TR_VNNI_TO_VNNI_T &&
        (ld_in < (int64_t)m * alpha || ld_out < (int64_t)n * alpha))
      return fail(TPP_ERR_INVALID_ARG,
                  "VNNI to VNNI-transpose needs ld_in >= m * alpha and ld_out >= n * alpha");
  }
  if (m == 0 || n == 0 || G == 0) return ok();
  if (!in || !out) return fail(TPP_ERR_INVALID_ARG, "NULL input or output");
  const int32_t es = dtype == TPP_DT_F32 ? 4 : 2;
  // the 16-byte paths need every block of the batch aligned: the bases, the leading dimensions
  // and (for G > 1) the block strides in whole 16-byte units
  const bool vec = ((reinterpret_cast<uintptr_t>(in) | reinterpret_cast<uintptr_t>(out)) & 15) == 0 &&
                   (ld_in * es) % 16 == 0 && (ld_out * es) % 16 == 0 &&
                   (G == 1 || ((in_stride * es) % 16 == 0 && (out_stride * es) % 16 == 0));
  tpp::TransformParams p{in, out, kind, m, n, ld_in, ld_out, es, alpha, vec ? 1 : 0, 0,
                         G, in_stride, out_stride};
  const hipError_t e = tpp::launch_transform(p, static_cast<hipStream_t>(stream));
  if (e == hipErrorInvalidConfiguration)
    return fail(TPP_ERR_UNSUPPORTED, "transform needs more than 2^31 - 1 workgroups");
  if (e != hipSuccess) return fail(TPP_ERR_HIP, "transform launch failed: %s", hipGetErrorString(e));
  return ok();
}

}  // namespace

extern "C" {

tpp_status tpp_reduce(int32_t m, int32_t n, int64_t ld, int32_t in_type, const void* in,
                      int32_t op, uint32_t flags, float* out_x, float* out_x2, void* stream) {
  return reduce_impl(m, n, ld, in_type, in, 1, 0, op, flags, out_x, out_x2, 0, stream);
}

tpp_status tpp_reduce_batched(int32_t m, int32_t n, int64_t ld, int32_t in_type, const void* in,
                              int64_t G, int64_t in_stride, int32_t op, uint32_t flags,
                              float* out_x, float* out_x2, int64_t out_stride, void* stream) {
  return reduce_impl(m, n, ld, in_type, in, G, in_stride, op, flags, out_x, out_x2, out_stride,
                     stream);
}

tpp_status tpp_transform(int32_t kind, int32_t m, int32_t n, int64_t ld_in, int64_t ld_out,
                         int32_t dtype, int32_t alpha, const void* in, void* out, void* stream) {
  return transform_impl(kind, m, n, ld_in, ld_out, dtype, alpha, in, 0, out, 0, 1, stream);
}

tpp_status tpp_embedding_bag(int64_t M, int32_t E, int32_t w_type, const void* W, int64_t ldw,
                             int64_t n_bags, const int64_t* d_begin, const int64_t* d_idx,
                             int32_t out_type, void* out, int64_t ldo, void* stream) {
  if (M < 0 || E <= 0 || n_bags < 0)
    return fail(TPP_ERR_INVALID_ARG, "M, n_bags must be >= 0 and E > 0");
  if (ldw < E || ldo < E) return fail(TPP_ERR_INVALID_ARG, "ldw and ldo must be >= E");
  if (!valid_dtype(w_type) || !valid_dtype(out_type))
    return fail(TPP_ERR_INVALID_ARG, "unknown datatype code");
  if (n_bags == 0) return ok();
  if (!d_begin || !out || (M > 0 && (!W || !d_idx)))
    return fail(TPP_ERR_INVALID_ARG, "NULL table, list or output");
  tpp::EmbeddingParams p{M, E, w_type == TPP_DT_BF16, out_type == TPP_DT_BF16, W, ldw, n_bags,
                         d_begin, d_idx, out, ldo};
  const hipError_t e = tpp::launch_embedding(p, static_cast<hipStream_t>(stream));
  if (e == hipErrorInvalidConfiguration)
    return fail(TPP_ERR_UNSUPPORTED, "embedding needs more than 2^31 - 1 workgroups");
  if (e != hipSuccess) return fail(TPP_ERR_HIP, "embedding launch failed: %s", hipGetErrorString(e));
  return ok();
}

tpp_status tpp_equation_plan(const tpp_eq_node* nodes, int32_t n_nodes, int32_t root,
                             tpp_eq_plan_node* plan, int32_t* n_tmps) {
  if (const char* err = tpp::equation_plan(nodes, n_nodes, root, plan, n_tmps))
    return fail(TPP_ERR_INVALID_ARG, "equation: %s", err);
  return ok();
}

tpp_status tpp_equation_execute(const tpp_eq_node* nodes, int32_t n_nodes, int32_t root,
                                int32_t m, int32_t n, const tpp_eq_arg* args, int32_t n_args,
                                void* out, int64_t ldo, int32_t out_type, void* stream) {
  if (m < 0 || n < 0) return fail(TPP_ERR_INVALID_ARG, "m, n must be >= 0");
  if (ldo < m) return fail(TPP_ERR_INVALID_ARG, "ldo < m");
  if (!valid_dtype(out_type)) return fail(TPP_ERR_INVALID_ARG, "unknown output datatype");
  if (n_args < 0 || n_args > tpp::EQ_MAX_ARGS || (n_args > 0 && !args))
    return fail(TPP_ERR_INVALID_ARG, "n_args must be in [0, 16] with a non-NULL args");
  tpp::EqProgram prog;
  std::memset(&prog, 0, sizeof prog);
  bool too_many = false;
  if (const char* err = tpp::equation_compile(nodes, n_nodes, root, prog, &too_many))
    return fail(too_many ? TPP_ERR_UNSUPPORTED : TPP_ERR_INVALID_ARG, "equation: %s", err);
  // every leaf the tree reaches names a well-described argument
  for (int32_t t = 0; t < prog.n_instr; ++t)
    for (int a = 0; a < prog.instr[t].arity; ++a) {
      const int32_t code = prog.instr[t].src[a];
      if (code < tpp::EQ_LEAF_BASE) continue;
      const int32_t k = code - tpp::EQ_LEAF_BASE;
      if (k >= n_args) return fail(TPP_ERR_INVALID_ARG, "leaf argument %d of %d", k, n_args);
    }
  for (int32_t k = 0; k < n_args; ++k) {
    const tpp_eq_arg& g = args[k];
    if (!valid_dtype(g.dtype) || g.bcast < TPP_BC_NONE || g.bcast > TPP_BC_SCALAR)
      return fail(TPP_ERR_INVALID_ARG, "argument %d: unknown datatype or broadcast", k);
    if (g.bcast == TPP_BC_NONE && g.ld < m)
      return fail(TPP_ERR_INVALID_ARG, "argument %d: ld < m", k);
    if (!g.ptr && m > 0 && n > 0) return fail(TPP_ERR_INVALID_ARG, "argument %d: NULL", k);
    prog.arg[k] = {g.ptr, g.ld, g.dtype == TPP_DT_BF16 ? 1 : 0, g.bcast};
  }
  if (m == 0 || n == 0) return ok();
  if (!out) return fail(TPP_ERR_INVALID_ARG, "NULL out");
  prog.n_args = n_args;
  prog.m = m;
  prog.n = n;
  prog.ldo = ldo;
  prog.out = out;
  prog.out_bf16 = out_type == TPP_DT_BF16;
  const hipError_t e = tpp::launch_equation(prog, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(TPP_ERR_HIP, "equation launch failed: %s", hipGetErrorString(e));
  return ok();
}

tpp_status tpp_transform_batched(int32_t kind, int32_t m, int32_t n, int64_t ld_in,
                                 int64_t ld_out, int32_t dtype, int32_t alpha, const void* in,
                                 int64_t in_stride, void* out, int64_t out_stride, int64_t G,
                                 void* stream) {
  return transform_impl(kind, m, n, ld_in, ld_out, dtype, alpha, in, in_stride, out, out_stride,
                        G, stream);
}

}  // extern "C"
