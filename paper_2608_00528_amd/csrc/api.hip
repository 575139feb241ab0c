// C ABI of the S^4R library: argument validation, workspace carving and the
// launch sequence of each entry point.  All validation happens on the host
// before anything is launched; see include/s4r.h for the contract.
#include <algorithm>
#include <atomic>
#include <climits>
#include <cmath>
#include <cstdarg>
#include <cstddef>
#include <cstdio>
#include <mutex>
#include <string>
#include <vector>

#include "s4r_device.h"
#include "s4r_internal.h"
#include "select_key.h"

static_assert(sizeof(s4r_config) == 80 && offsetof(s4r_config, capacity) == 56 &&
                  offsetof(s4r_config, rank_v) == 72,
              "s4r_config layout is part of the ABI");

namespace s4r {
namespace {

thread_local std::string g_err;

s4r_status fail(s4r_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

s4r_status ok() {
  g_err.clear();
  return S4R_OK;
}

constexpr int kMaxExtraTok = 1024 + 64;   // sinks + exact window rows in the combine kernel

s4r_status make_problem(const s4r_config* c, Problem& P) {
  if (!c) return fail(S4R_ERR_NULL_ARG, "cfg is NULL");
  if (c->batch < 1) return fail(S4R_ERR_BAD_SHAPE, "batch must be >= 1 (got %d)", c->batch);
  if (c->n_q_heads < 1 || c->n_kv_heads < 1)
    return fail(S4R_ERR_BAD_SHAPE, "head counts must be >= 1 (h_q=%d, h_kv=%d)", c->n_q_heads, c->n_kv_heads);
  if (c->n_q_heads % c->n_kv_heads)
    return fail(S4R_ERR_BAD_SHAPE, "n_q_heads %d is not a multiple of n_kv_heads %d", c->n_q_heads, c->n_kv_heads);
  if (c->head_dim != 64 && c->head_dim != 128)
    return fail(S4R_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", c->head_dim);
  if (c->basis_groups < 1 || c->n_kv_heads % c->basis_groups)
    return fail(S4R_ERR_BAD_SHAPE, "basis_groups %d must divide n_kv_heads %d", c->basis_groups, c->n_kv_heads);
  const int Dp = c->n_kv_heads * c->head_dim;
  const int Dg = Dp / c->basis_groups;
  if (c->rank < 1 || c->rank > Dg)
    return fail(S4R_ERR_BAD_SHAPE, "rank %d must be in [1, Dp/basis_groups = %d]", c->rank, Dg);
  if (Dg > kQMaxChunks * kPChunk)
    return fail(S4R_ERR_UNSUPPORTED, "Dp / basis_groups = %d > %d not supported", Dg, kQMaxChunks * kPChunk);
  // storage widths: the configured ranks rounded up to 32 columns (Dg is a
  // multiple of 64, so the rounded rank still fits the basis group)
  const int rank_s = (c->rank + 31) / 32 * 32;
  const int R = rank_s * c->basis_groups;
  if (R > 256) return fail(S4R_ERR_UNSUPPORTED, "latent width %d (rank stride %d) > 256 not supported", R, rank_s);
  const int rank_v_cfg = c->rank_v ? c->rank_v : c->rank;
  if (rank_v_cfg < 1 || rank_v_cfg > Dg)
    return fail(S4R_ERR_BAD_SHAPE, "rank_v %d must be 0 or in [1, Dp/basis_groups = %d]", c->rank_v, Dg);
  const int rank_v = (rank_v_cfg + 31) / 32 * 32;
  if (rank_v * c->basis_groups > 256)
    return fail(S4R_ERR_UNSUPPORTED, "value latent width %d > 256 not supported", rank_v * c->basis_groups);
  if (c->n_sink < 0 || c->n_sink > 1024) return fail(S4R_ERR_BAD_SHAPE, "n_sink %d outside [0, 1024]", c->n_sink);
  if (c->window < 0) return fail(S4R_ERR_BAD_SHAPE, "window %d < 0", c->window);
  if (c->q_window < 1) return fail(S4R_ERR_BAD_SHAPE, "q_window %d < 1", c->q_window);
  if (c->topk < 0) return fail(S4R_ERR_BAD_SHAPE, "topk %d < 0", c->topk);
  if (c->pool_kernel < 1 || c->pool_kernel % 2 == 0)
    return fail(S4R_ERR_BAD_SHAPE, "pool_kernel %d must be odd and >= 1", c->pool_kernel);
  if (c->pool_kernel > 65) return fail(S4R_ERR_UNSUPPORTED, "pool_kernel %d > 65", c->pool_kernel);
  if (c->pool_mode != S4R_POOL_MAX && c->pool_mode != S4R_POOL_AVG)
    return fail(S4R_ERR_BAD_SHAPE, "pool_mode %d invalid", c->pool_mode);
  if (c->group_agg != S4R_AGG_MEAN && c->group_agg != S4R_AGG_MAX)
    return fail(S4R_ERR_BAD_SHAPE, "group_agg %d invalid", c->group_agg);
  const int G = c->n_q_heads / c->n_kv_heads;
  if (G > kMaxG) return fail(S4R_ERR_UNSUPPORTED, "G = n_q_heads / n_kv_heads = %d > %d not supported", G, kMaxG);
  if ((int64_t)G * c->q_window > kMaxGW)
    return fail(S4R_ERR_UNSUPPORTED, "G * q_window = %lld > %d not supported", (long long)G * c->q_window, kMaxGW);
  if (c->capacity < 16 || c->capacity % 16)
    return fail(S4R_ERR_BAD_SHAPE, "capacity %lld must be a positive multiple of 16", (long long)c->capacity);
  if (c->capacity > (int64_t)kMaxSelGroups * kSelChunk)
    return fail(S4R_ERR_UNSUPPORTED, "capacity %lld > %lld", (long long)c->capacity,
                (long long)kMaxSelGroups * kSelChunk);
  if (!(c->rope_theta >= 0.f) || !std::isfinite(c->rope_theta))
    return fail(S4R_ERR_BAD_SHAPE, "rope_theta must be finite and >= 0");
  if (c->dtype != S4R_FP32 && c->dtype != S4R_BF16) return fail(S4R_ERR_BAD_SHAPE, "dtype %d invalid", c->dtype);
  if (c->bases_shared != 0 && c->bases_shared != 1) return fail(S4R_ERR_BAD_SHAPE, "bases_shared must be 0 or 1");

  P.B = c->batch;
  P.hq = c->n_q_heads;
  P.hkv = c->n_kv_heads;
  P.dh = c->head_dim;
  P.G = G;
  P.Dp = Dp;
  P.nb = c->basis_groups;
  P.rank = rank_s;
  P.R = R;
  P.rank_v = rank_v;
  P.Rv = rank_v * c->basis_groups;
  P.rank_cfg = c->rank;
  P.rank_v_cfg = rank_v_cfg;
  P.R_cfg = c->rank * c->basis_groups;
  P.Dg = Dg;
  P.s = c->n_sink;
  P.W = c->window;
  P.Wq = c->q_window;
  P.k = c->topk;
  P.kappa = c->pool_kernel;
  P.pool_mode = c->pool_mode;
  P.agg = c->group_agg;
  P.bases_shared = c->bases_shared;
  P.dtype = c->dtype;
  P.cap = c->capacity;
  P.theta = c->rope_theta;
  P.GW = G * c->q_window;
  P.nruns_max = c->capacity / kTileTok;
  P.nwg_max = (P.nruns_max + kScoreWaves - 1) / kScoreWaves;   // tiles per wave >= 1
  P.lens.n = 0;
  P.m_max = std::min<int64_t>(c->topk, std::max<int64_t>(c->capacity - c->window, 0)) +
            std::min<int64_t>(c->window, c->capacity);
  return S4R_OK;
}

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

size_t elem_size(const Problem& P) { return P.dtype == S4R_BF16 ? 2 : 4; }

enum Region {
  kQimg, kQcoef, kE, kRunM, kWgStats, kAtilde, kHist, kCand, kBitmap, kIdx, kPartMl, kPartO, kAttnLogits,
  kCandCount, kAboveCount, kSelInfo, kColStats, kRegions
};
struct Layout {
  size_t off[kRegions];
  size_t total;
};

Layout layout(const Problem& P) {
  const size_t B = P.B, GW = P.GW, cap = P.cap;
  size_t sizes[kRegions];
  sizes[kQimg] = B * col_blocks(P) * qimg_mfmas(P) * 16 * (size_t)P.R * 2;
  sizes[kQcoef] = B * P.G * (size_t)P.R * 4;
  sizes[kE] = B * (size_t)gw_padded(P) * cap * 4;
  sizes[kRunM] = B * (size_t)gw_padded(P) * P.nruns_max * 4;
  sizes[kWgStats] = B * GW * P.nwg_max * 2 * 8;
  sizes[kAtilde] = B * cap * 4;
  sizes[kHist] = B * kHistStride * 4;
  sizes[kCand] = B * cand_stride(P) * 8;
  sizes[kBitmap] = B * bitmap_words(cap) * 4;
  sizes[kIdx] = B * P.m_max * 4;
  sizes[kPartMl] = B * P.hq * kMaxSplit * 2 * 4;
  sizes[kPartO] = B * P.hq * kMaxSplit * P.dh * 4;
  sizes[kAttnLogits] = B * P.hq * (P.s + P.m_max) * 4;
  sizes[kCandCount] = B * sel_groups_max(P) * 4;
  sizes[kAboveCount] = B * sel_groups_max(P) * 4;
  sizes[kSelInfo] = B * 4 * 4;
  sizes[kColStats] = B * GW * 2 * 8;
  Layout l;
  size_t o = 0;
  for (int i = 0; i < kRegions; ++i) {
    l.off[i] = o;
    o = align256(o + sizes[i]);
  }
  l.total = o;
  return l;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

#define S4R_REQ(ptr)                                                                     \
  do {                                                                                   \
    if (!(ptr)) return fail(S4R_ERR_NULL_ARG, "%s is NULL", #ptr);                       \
    if (!aligned16(ptr)) return fail(S4R_ERR_MISALIGNED, "%s is not 16-byte aligned", #ptr); \
  } while (0)
#define S4R_OPT(ptr)                                                                     \
  do {                                                                                   \
    if ((ptr) && !aligned16(ptr)) return fail(S4R_ERR_MISALIGNED, "%s is not 16-byte aligned", #ptr); \
  } while (0)

s4r_status check_ws(const Problem& P, void* ws, size_t ws_bytes) {
  if (!ws) return fail(S4R_ERR_NULL_ARG, "ws is NULL");
  if (((uintptr_t)ws & 255) != 0) return fail(S4R_ERR_MISALIGNED, "ws is not 256-byte aligned");
  const size_t need = layout(P).total;
  if (ws_bytes < need)
    return fail(S4R_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu required", ws_bytes, need);
  return S4R_OK;
}

s4r_status check_L(const Problem& P, int64_t L) {
  if (L < 1 || L > P.cap) return fail(S4R_ERR_BAD_SHAPE, "L = %lld outside [1, capacity = %lld]", (long long)L, (long long)P.cap);
  if (P.Wq > L) return fail(S4R_ERR_BAD_SHAPE, "q_window %d > L = %lld", P.Wq, (long long)L);
  return S4R_OK;
}

s4r_status hip_status(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(S4R_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return ok();
}

// ---- kernel timing ------------------------------------------------------------------
struct Timing {
  std::mutex mu;
  std::atomic<bool> enabled{false};   // read without the lock on every step call
  std::vector<hipEvent_t> start, stop;   // [steps][S4R_TIMED_KERNELS]
  int steps = 0;
  int used = 0;
} g_timing;

// ---- scratch for the step without a caller workspace -------------------------------
// A file-scope device array that s4r_decode_step_noalloc uses as its
// workspace.  In host code `scratch` names a host-side stand-in, not device
// memory: its device address is taken once per device with
// hipGetSymbolAddress (with that device current) and only that address is
// handed to kernels.  Each device that runs the entry point keeps its copy
// until the process ends.
constexpr size_t kScratchBytes = size_t(64) << 20;
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;                                   // first lookup per device only
std::atomic<void*> g_scratch_addr[kMaxScratchDevices];

}  // namespace

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

// the device address of this device's `scratch` (looked up on the first call
// on the device; later calls read the cached address without locking)
s4r_status scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(S4R_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxScratchDevices)
    return fail(S4R_ERR_UNSUPPORTED, "device %d outside the %d devices the scratch table holds", dev,
                kMaxScratchDevices);
  void* p = g_scratch_addr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    p = g_scratch_addr[dev].load(std::memory_order_relaxed);
    if (!p) {
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !p)
        return fail(S4R_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
      g_scratch_addr[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return S4R_OK;
}

}  // namespace

Workspace carve_workspace(const Problem& P, void* base) {
  const Layout l = layout(P);
  char* b = (char*)base;
  Workspace w;
  w.qimg = (uint16_t*)(b + l.off[kQimg]);
  w.qcoef = (float*)(b + l.off[kQcoef]);
  w.e = (float*)(b + l.off[kE]);
  w.run_m = (float*)(b + l.off[kRunM]);
  w.wg_stats = (double*)(b + l.off[kWgStats]);
  w.atilde = (float*)(b + l.off[kAtilde]);
  w.hist = (uint32_t*)(b + l.off[kHist]);
  w.cand = (uint64_t*)(b + l.off[kCand]);
  w.bitmap = (uint32_t*)(b + l.off[kBitmap]);
  w.idx = (int32_t*)(b + l.off[kIdx]);
  w.part_ml = (float*)(b + l.off[kPartMl]);
  w.part_o = (float*)(b + l.off[kPartO]);
  w.attn_logits = (float*)(b + l.off[kAttnLogits]);
  w.cand_count = (uint32_t*)(b + l.off[kCandCount]);
  w.above_count = (uint32_t*)(b + l.off[kAboveCount]);
  w.sel_info = (uint32_t*)(b + l.off[kSelInfo]);
  w.col_stats = (double*)(b + l.off[kColStats]);
  w.total = l.total;
  return w;
}

}  // namespace s4r

using namespace s4r;

extern "C" {

const char* s4r_last_error(void) { return g_err.c_str(); }

const char* s4r_version(void) { return "s4r-gfx950 0.1.0"; }

s4r_status s4r_workspace_size(const s4r_config* cfg, size_t* bytes) {
  Problem P;
  s4r_status st = make_problem(cfg, P);
  if (st) return st;
  if (!bytes) return fail(S4R_ERR_NULL_ARG, "bytes is NULL");
  *bytes = layout(P).total;
  return ok();
}

int32_t s4r_num_selected(const s4r_config* cfg, int64_t L) {
  Problem P;
  if (make_problem(cfg, P)) return -1;
  if (L < 1 || L > P.cap) {
    fail(S4R_ERR_BAD_SHAPE, "L = %lld outside [1, capacity]", (long long)L);
    return -1;
  }
  ok();
  return (int32_t)(std::min<int64_t>(P.k, std::max<int64_t>(L - P.W, 0)) + std::min<int64_t>(P.W, L));
}

s4r_status s4r_score_latent(const s4r_config* cfg, int64_t L, const void* q, const float* qwin_prev,
                            const void* bases_k, const void* coef_k, float* scores, float* qcoef_out, void* ws,
                            size_t ws_bytes, hipStream_t stream) {
  Problem P;
  s4r_status st = make_problem(cfg, P);
  if (st) return st;
  if ((st = check_L(P, L))) return st;
  S4R_REQ(q);
  S4R_REQ(bases_k);
  S4R_REQ(coef_k);
  S4R_REQ(scores);
  S4R_OPT(qcoef_out);
  if (P.Wq > 1) S4R_REQ(qwin_prev);
  else if (qwin_prev) return fail(S4R_ERR_BAD_SHAPE, "qwin_prev must be NULL when q_window == 1");
  if ((st = check_ws(P, ws, ws_bytes))) return st;
  Workspace w = carve_workspace(P, ws);
  hipError_t e = launch_project_query(P, w, q, bases_k, qwin_prev, qcoef_out, true, stream);
  if (e == hipSuccess) e = launch_score_stream(P, w, L, coef_k, stream);
  if (e == hipSuccess) e = launch_relevance(P, w, L, scores, stream);
  return hip_status(e, "s4r_score_latent launch");
}

s4r_status s4r_select_topk(const s4r_config* cfg, int64_t L, const float* scores, int32_t* idx, void* ws,
                           size_t ws_bytes, hipStream_t stream) {
  Problem P;
  s4r_status st = make_problem(cfg, P);
  if (st) return st;
  if (L < 1 || L > P.cap) return fail(S4R_ERR_BAD_SHAPE, "L = %lld outside [1, capacity]", (long long)L);
  S4R_REQ(scores);
  S4R_REQ(idx);
  if ((st = check_ws(P, ws, ws_bytes))) return st;
  Workspace w = carve_workspace(P, ws);
  hipError_t e = launch_hist_only(P, w, L, scores, stream);
  if (e == hipSuccess) e = launch_select(P, w, L, scores, L, idx, nullptr, stream);
  return hip_status(e, "s4r_select_topk launch");
}

s4r_status s4r_reconstruct(const s4r_config* cfg, int64_t L, int32_t m, const int32_t* idx, const void* bases_k,
                           const void* bases_v, const void* coef_k, const void* coef_v, float* k_hat, float* v_hat,
                           hipStream_t stream) {
  Problem P;
  s4r_status st = make_problem(cfg, P);
  if (st) return st;
  if (L < 1 || L > P.cap) return fail(S4R_ERR_BAD_SHAPE, "L = %lld outside [1, capacity]", (long long)L);
  if (m < 0) return fail(S4R_ERR_BAD_SHAPE, "m = %d < 0", m);
  if (P.rank_v != P.rank)
    return fail(S4R_ERR_UNSUPPORTED, "explicit reconstruction is built for equal key and value ranks");
  if (m == 0) return ok();
  S4R_REQ(idx);
  S4R_REQ(bases_k);
  S4R_REQ(bases_v);
  S4R_REQ(coef_k);
  S4R_REQ(coef_v);
  S4R_REQ(k_hat);
  S4R_REQ(v_hat);
  return hip_status(launch_reconstruct(P, L, m, idx, bases_k, bases_v, coef_k, coef_v, k_hat, v_hat, stream),
                    "s4r_reconstruct launch");
}

s4r_status s4r_sparse_attn(const s4r_config* cfg, int64_t L, int32_t m, const void* q, const void* sink_k,
                           const void* sink_v, const int32_t* idx, const float* k_sel, const float* v_sel, float* out,
                           void* ws, size_t ws_bytes, hipStream_t stream) {
  Problem P;
  s4r_status st = make_problem(cfg, P);
  if (st) return st;
  if (L < 1 || L > P.cap) return fail(S4R_ERR_BAD_SHAPE, "L = %lld outside [1, capacity]", (long long)L);
  if (m < 0 || m > P.m_max) return fail(S4R_ERR_BAD_SHAPE, "m = %d outside [0, %lld]", m, (long long)P.m_max);
  if (m + P.s < 1) return fail(S4R_ERR_BAD_SHAPE, "attention over an empty set (m + n_sink == 0)");
  S4R_REQ(q);
  S4R_REQ(out);
  if (P.s > 0) {
    S4R_REQ(sink_k);
    S4R_REQ(sink_v);
  }
  if (m > 0) {
    S4R_REQ(idx);
    S4R_REQ(k_sel);
    S4R_REQ(v_sel);
  }
  if ((st = check_ws(P, ws, ws_bytes))) return st;
  Workspace w = carve_workspace(P, ws);
  return hip_status(launch_sparse_attn(P, w, L, m, q, sink_k, sink_v, idx, k_sel, v_sel, out, stream),
                    "s4r_sparse_attn launch");
}

s4r_status s4r_prefill_project(const s4r_config* cfg, int64_t n_rows, const void* s_k, const void* s_v,
                               const void* bases_k, const void* bases_v, void* coef_k, void* coef_v, void* ws,
                               size_t ws_bytes, hipStream_t stream) {
  Problem P;
  s4r_status st = make_problem(cfg, P);
  if (st) return st;
  if (P.dtype != S4R_BF16) return fail(S4R_ERR_UNSUPPORTED, "the bulk projection is built for bf16 storage only");
  if (P.rank_v != P.rank)
    return fail(S4R_ERR_UNSUPPORTED, "the bulk projection is built for equal key and value ranks");
  if (P.rank / 32 < 1 || P.rank / 32 > 6)
    return fail(S4R_ERR_UNSUPPORTED, "the bulk projection is built for rank 32 .. 192 (rank %d)", P.rank);
  if ((P.hkv * P.dh / P.nb) % 32)
    return fail(S4R_ERR_UNSUPPORTED, "basis group width %d is not a multiple of 32", P.hkv * P.dh / P.nb);
  if (n_rows < 1 || n_rows > P.cap)
    return fail(S4R_ERR_BAD_SHAPE, "n_rows = %lld outside [1, capacity = %lld]", (long long)n_rows,
                (long long)P.cap);
  S4R_REQ(s_k);
  S4R_REQ(s_v);
  S4R_REQ(bases_k);
  S4R_REQ(bases_v);
  S4R_REQ(coef_k);
  S4R_REQ(coef_v);
  if ((st = check_ws(P, ws, ws_bytes))) return st;     // the transposed bases use its first bytes
  if (prefill_ws_bytes(P) > layout(P).total) return fail(S4R_ERR_WORKSPACE, "workspace too small for the bases");
  return hip_status(launch_prefill_project(P, n_rows, s_k, s_v, bases_k, bases_v, coef_k, coef_v, ws, stream),
                    "s4r_prefill_project launch");
}

s4r_status s4r_dense_decode(const s4r_config* cfg, int64_t N, const void* q, const void* k_cache,
                            const void* v_cache, float* out, void* ws, size_t ws_bytes, hipStream_t stream) {
  Problem P;
  s4r_status st = make_problem(cfg, P);
  if (st) return st;
  if (P.dtype != S4R_BF16) return fail(S4R_ERR_UNSUPPORTED, "the dense comparator is built for bf16 caches only");
  if (P.dh != 128) return fail(S4R_ERR_UNSUPPORTED, "the dense comparator is built for head_dim 128 only");
  if (P.G > 8) return fail(S4R_ERR_UNSUPPORTED, "the dense comparator is built for G <= 8");
  if (N < 1 || N > P.cap) return fail(S4R_ERR_BAD_SHAPE, "N = %lld outside [1, capacity = %lld]", (long long)N,
                                      (long long)P.cap);
  S4R_REQ(q);
  S4R_REQ(k_cache);
  S4R_REQ(v_cache);
  S4R_REQ(out);
  if ((st = check_ws(P, ws, ws_bytes))) return st;
  Workspace w = carve_workspace(P, ws);
  return hip_status(launch_dense_decode(P, w, N, q, k_cache, v_cache, out, stream), "s4r_dense_decode launch");
}

s4r_status s4r_full_recon_decode(const s4r_config* cfg, int64_t L, const void* q, const void* sink_k,
                                 const void* sink_v, const void* bases_k, const void* bases_v, const void* coef_k,
                                 const void* coef_v, float* out, void* ws, size_t ws_bytes, hipStream_t stream) {
  Problem P;
  s4r_status st = make_problem(cfg, P);
  if (st) return st;
  if ((st = check_L(P, L))) return st;
  if (P.dtype != S4R_BF16 || (P.dh != 64 && P.dh != 128) || P.G > 8 || !attention_supported(P))
    return fail(S4R_ERR_UNSUPPORTED, "full reconstruction is built for bf16 storage, head_dim 64 or 128, G <= 8 and "
                                     "the ranks of the fused attention kernel");
  S4R_REQ(q);
  S4R_REQ(bases_k);
  S4R_REQ(bases_v);
  S4R_REQ(coef_k);
  S4R_REQ(coef_v);
  S4R_REQ(out);
  if (P.s > 0) {
    S4R_REQ(sink_k);
    S4R_REQ(sink_v);
  }
  if ((st = check_ws(P, ws, ws_bytes))) return st;
  Workspace w = carve_workspace(P, ws);
  return hip_status(launch_full_recon(P, w, L, q, sink_k, sink_v, bases_k, bases_v, coef_k, coef_v, out, stream),
                    "s4r_full_recon_decode launch");
}

s4r_status s4r_project_queries(const s4r_config* cfg, int64_t n_rows, const void* q_rows, const void* bases_k,
                               float* qcoef_out, void* ws, size_t ws_bytes, hipStream_t stream) {
  Problem P;
  s4r_status st = make_problem(cfg, P);
  if (st) return st;
  if (n_rows < 1 || n_rows > 4096) return fail(S4R_ERR_BAD_SHAPE, "n_rows = %lld outside [1, 4096]", (long long)n_rows);
  S4R_REQ(q_rows);
  S4R_REQ(bases_k);
  S4R_REQ(qcoef_out);
  if ((st = check_ws(P, ws, ws_bytes))) return st;
  Workspace w = carve_workspace(P, ws);
  return hip_status(launch_project_queries(P, w, n_rows, q_rows, bases_k, qcoef_out, stream),
                    "s4r_project_queries launch");
}

// ---- basis construction of the prefill ------------------------------------------------
static s4r_status check_bases_args(const s4r_config* cfg, int64_t n_rows, double eta, Problem& P, int* nu, int* nr) {
  s4r_status st = make_problem(cfg, P);
  if (st) return st;
  if (P.dtype != S4R_BF16) return fail(S4R_ERR_UNSUPPORTED, "basis construction is built for bf16 storage only");
  if (P.bases_shared) return fail(S4R_ERR_BAD_SHAPE, "basis construction writes per-sequence bases (bases_shared = 0)");
  if (P.Dg % 256) return fail(S4R_ERR_UNSUPPORTED, "basis construction needs Dp / basis_groups %% 256 == 0");
  if (n_rows < 1 || n_rows > INT32_MAX) return fail(S4R_ERR_BAD_SHAPE, "n_rows = %lld outside [1, 2^31)", (long long)n_rows);
  if (!(eta > 0.0 && eta <= 1.0)) return fail(S4R_ERR_BAD_SHAPE, "eta must lie in (0, 1]");
  bases_sample_counts(n_rows, eta, nu, nr);
  if (*nu + *nr < std::max(P.rank, P.rank_v))
    return fail(S4R_ERR_BAD_SHAPE, "%d sampled rows cannot give %d singular vectors", *nu + *nr,
                std::max(P.rank, P.rank_v));
  return S4R_OK;
}

int64_t s4r_prefill_num_samples(int64_t n_rows, double eta) {
  if (n_rows < 1 || !(eta > 0.0 && eta <= 1.0)) return -1;
  int nu = 0, nr = 0;
  bases_sample_counts(n_rows, eta, &nu, &nr);
  return nu + nr;
}

s4r_status s4r_prefill_bases_workspace_size(const s4r_config* cfg, int64_t n_rows, double eta, size_t* bytes) {
  Problem P;
  int nu = 0, nr = 0;
  s4r_status st = check_bases_args(cfg, n_rows, eta, P, &nu, &nr);
  if (st) return st;
  if (!bytes) return fail(S4R_ERR_NULL_ARG, "bytes is NULL");
  return hip_status(prefill_bases_ws_bytes(P, nu + nr, bytes), "s4r_prefill_bases_workspace_size");
}

s4r_status s4r_prefill_bases(const s4r_config* cfg, int64_t n_rows, const void* s_k, const void* s_v, double eta,
                             int32_t center, void* bases_k, void* bases_v, int32_t* sample_idx_out, void* ws,
                             size_t ws_bytes, hipStream_t stream) {
  Problem P;
  int nu = 0, nr = 0;
  s4r_status st = check_bases_args(cfg, n_rows, eta, P, &nu, &nr);
  if (st) return st;
  S4R_REQ(s_k);
  S4R_REQ(s_v);
  S4R_REQ(bases_k);
  S4R_REQ(bases_v);
  S4R_REQ(ws);
  if (center != 0 && center != 1) return fail(S4R_ERR_BAD_SHAPE, "center must be 0 or 1");
  size_t need = 0;
  if ((st = hip_status(prefill_bases_ws_bytes(P, nu + nr, &need), "s4r_prefill_bases workspace query"))) return st;
  if (ws_bytes < need)
    return fail(S4R_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu required", ws_bytes, need);
  return hip_status(launch_prefill_bases(P, n_rows, s_k, s_v, nu, nr, center, sample_idx_out, bases_k, bases_v, ws,
                                         ws_bytes, stream),
                    "s4r_prefill_bases launch");
}

// the fused step for a uniform (P.lens.n == 0) or ragged batch; L is the
// largest length, already checked against the capacity
// state (windowed step, q_window > 1): the window state replaces qwin_prev;
// only the newest query row is projected and scored
static s4r_status decode_step_impl(const Problem& P, int64_t L, const void* q, const float* qwin_prev,
                                   const void* sink_k, const void* sink_v, const void* win_k, const void* win_v,
                                   const void* bases_k, const void* bases_v, void* coef_k, void* coef_v,
                                   const void* k_new, const void* v_new, float* out, int32_t* idx_out,
                                   float* scores_out, void* ws, size_t ws_bytes, hipStream_t stream,
                                   float* state = nullptr) {
  s4r_status st = S4R_OK;
  if (!attention_supported(P))
    return fail(S4R_ERR_UNSUPPORTED, "fused attention not built for G = %d, rank = %d", P.G, P.rank);
  S4R_REQ(q);
  S4R_REQ(bases_k);
  S4R_REQ(bases_v);
  S4R_REQ(coef_k);
  S4R_REQ(coef_v);
  S4R_REQ(out);
  S4R_OPT(idx_out);
  S4R_OPT(scores_out);
  if (P.s > 0) {
    S4R_REQ(sink_k);
    S4R_REQ(sink_v);
  }
  if (state) {
    if (P.Wq < 2) return fail(S4R_ERR_BAD_SHAPE, "the windowed step needs q_window >= 2 (got %d)", P.Wq);
    if (P.lens.n) return fail(S4R_ERR_UNSUPPORTED, "the windowed step takes a uniform batch");
    S4R_REQ(state);
  } else if (P.Wq > 1) {
    S4R_REQ(qwin_prev);
  } else if (qwin_prev) {
    return fail(S4R_ERR_BAD_SHAPE, "qwin_prev must be NULL when q_window == 1");
  }
  if ((win_k == nullptr) != (win_v == nullptr)) return fail(S4R_ERR_NULL_ARG, "win_k and win_v must both be given or both NULL");
  if ((k_new == nullptr) != (v_new == nullptr)) return fail(S4R_ERR_NULL_ARG, "k_new and v_new must both be given or both NULL");
  S4R_OPT(win_k);
  S4R_OPT(win_v);
  S4R_OPT(k_new);
  S4R_OPT(v_new);
  const int64_t n_hist = std::max<int64_t>(L - P.W, 0);
  const int k_eff = (int)std::min<int64_t>(P.k, n_hist);
  const int m = (int)(k_eff + std::min<int64_t>(P.W, L));
  if (m + P.s < 1) return fail(S4R_ERR_BAD_SHAPE, "attention over an empty set (m + n_sink == 0)");
  if ((int64_t)m > (int64_t)kMaxSplit * kMaxTilesPerSplit * 16)
    return fail(S4R_ERR_UNSUPPORTED, "m = %d selected tokens exceeds %d", m, kMaxSplit * kMaxTilesPerSplit * 16);
  if (P.rank_v != P.rank && (int64_t)m > (int64_t)kMaxSplit * kTileMax * 16)
    return fail(S4R_ERR_UNSUPPORTED, "m = %d selected tokens exceeds %d with asymmetric ranks", m,
                kMaxSplit * kTileMax * 16);
  if (win_k && P.s + std::min<int64_t>(P.W, L) > kMaxExtraTok)
    return fail(S4R_ERR_UNSUPPORTED, "n_sink + window = %lld > %d with exact window KV", (long long)(P.s + P.W), kMaxExtraTok);
  if ((st = check_ws(P, ws, ws_bytes))) return st;
  Workspace w = carve_workspace(P, ws);

  // the timing state is locked only while timing is enabled: untimed steps
  // from several host threads do not serialise on it
  std::unique_lock<std::mutex> lk;
  if (g_timing.enabled.load(std::memory_order_acquire)) lk = std::unique_lock<std::mutex>(g_timing.mu);
  const bool timed = lk.owns_lock() && g_timing.enabled && g_timing.used < g_timing.steps;
  const int slot = timed ? g_timing.used * S4R_TIMED_KERNELS : 0;
  auto mark = [&](hipError_t e, int kernel, bool start) -> hipError_t {
    if (e != hipSuccess || !timed) return e;
    return hipEventRecord(start ? g_timing.start[slot + kernel] : g_timing.stop[slot + kernel], stream);
  };
  // the projection and scoring problem: the whole window, or (windowed) the
  // newest row alone, whose G columns see every key
  Problem PS = P;
  if (state) {
    PS.Wq = 1;
    PS.GW = P.G;
  }
  hipError_t e = mark(hipSuccess, 0, true);
  if (e == hipSuccess && k_new)   // the new token's rows with the query coefficients: the scoring pass reads row L - 1
    e = launch_project_step(PS, w, q, bases_k, bases_v, k_new, v_new, coef_k, coef_v, state ? nullptr : qwin_prev,
                            L - 1, stream);
  else if (e == hipSuccess)
    e = launch_project_query(PS, w, q, bases_k, state ? nullptr : qwin_prev, nullptr, true, stream);
  e = mark(e, 0, false);
  e = mark(e, 1, true);
  if (e == hipSuccess) e = launch_score_stream(PS, w, L, coef_k, stream);
  e = mark(e, 1, false);
  e = mark(e, 2, true);
  if (e == hipSuccess)
    e = state ? launch_relevance_windowed(PS, w, L, scores_out, state, P.Wq, stream)
              : launch_relevance(P, w, L, scores_out, stream);
  e = mark(e, 2, false);
  e = mark(e, 3, true);
  // the key the relevance kernel built the histogram with
  if (e == hipSuccess)
    e = launch_select_keyed(P, w, L, w.atilde, P.cap, w.idx, idx_out, fused_key_shift(P, L),
                            relevance_hist_copies(state ? PS : P, L, state ? P.Wq : 0), stream);
  e = mark(e, 3, false);
  if (e == hipSuccess)
    e = launch_attention(P, w, L, m, k_eff, q, sink_k, sink_v, win_k, win_v, bases_k, bases_v, coef_k, coef_v, out,
                         stream, timed ? &g_timing.start[slot + 4] : nullptr,
                         timed ? &g_timing.stop[slot + 4] : nullptr);
  if (timed) g_timing.used++;
  return hip_status(e, "s4r_decode_step launch");
}

s4r_status s4r_decode_step(const s4r_config* cfg, int64_t L, const void* q, const float* qwin_prev,
                           const void* sink_k, const void* sink_v, const void* win_k, const void* win_v,
                           const void* bases_k, const void* bases_v, void* coef_k, void* coef_v, const void* k_new,
                           const void* v_new, float* out, int32_t* idx_out, float* scores_out, void* ws,
                           size_t ws_bytes, hipStream_t stream) {
  Problem P;
  s4r_status st = make_problem(cfg, P);
  if (st) return st;
  if ((st = check_L(P, L))) return st;
  return decode_step_impl(P, L, q, qwin_prev, sink_k, sink_v, win_k, win_v, bases_k, bases_v, coef_k, coef_v, k_new,
                          v_new, out, idx_out, scores_out, ws, ws_bytes, stream);
}

s4r_status s4r_window_state_size(const s4r_config* cfg, size_t* bytes) {
  Problem P;
  s4r_status st = make_problem(cfg, P);
  if (st) return st;
  if (!bytes) return fail(S4R_ERR_NULL_ARG, "bytes is NULL");
  if (P.Wq < 2) return fail(S4R_ERR_BAD_SHAPE, "the window state needs q_window >= 2 (got %d)", P.Wq);
  *bytes = window_state_bytes(P);
  return ok();
}

s4r_status s4r_window_state_init(const s4r_config* cfg, int64_t L, const float* qwin_prev, const void* coef_k,
                                 float* state, void* ws, size_t ws_bytes, hipStream_t stream) {
  Problem P;
  s4r_status st = make_problem(cfg, P);
  if (st) return st;
  if (P.Wq < 2) return fail(S4R_ERR_BAD_SHAPE, "the window state needs q_window >= 2 (got %d)", P.Wq);
  if ((st = check_L(P, L))) return st;
  S4R_REQ(qwin_prev);
  S4R_REQ(coef_k);
  S4R_REQ(state);
  if ((st = check_ws(P, ws, ws_bytes))) return st;
  Workspace w = carve_workspace(P, ws);
  // the window's W_q - 1 older rows as a query window of their own, scored
  // to length L - 1: row r's causal limit is then key L - W_q + r, its own
  Problem P0 = P;
  P0.Wq = P.Wq - 1;
  P0.GW = P.G * P0.Wq;
  hipError_t e = launch_query_image_rows(P0, w, qwin_prev, stream);
  if (e == hipSuccess) e = launch_score_stream(P0, w, L - 1, coef_k, stream);
  if (e == hipSuccess) e = launch_window_store(P0, w, L, state, P.Wq, stream);
  return hip_status(e, "s4r_window_state_init launch");
}

s4r_status s4r_decode_step_windowed(const s4r_config* cfg, int64_t L, const void* q, float* state,
                                    const void* sink_k, const void* sink_v, const void* win_k, const void* win_v,
                                    const void* bases_k, const void* bases_v, void* coef_k, void* coef_v,
                                    const void* k_new, const void* v_new, float* out, int32_t* idx_out,
                                    float* scores_out, void* ws, size_t ws_bytes, hipStream_t stream) {
  Problem P;
  s4r_status st = make_problem(cfg, P);
  if (st) return st;
  if ((st = check_L(P, L))) return st;
  if (!state) return fail(S4R_ERR_NULL_ARG, "state is NULL");
  return decode_step_impl(P, L, q, nullptr, sink_k, sink_v, win_k, win_v, bases_k, bases_v, coef_k, coef_v, k_new,
                          v_new, out, idx_out, scores_out, ws, ws_bytes, stream, state);
}

s4r_status s4r_decode_step_ragged(const s4r_config* cfg, const int64_t* lengths, const void* q,
                                  const float* qwin_prev, const void* sink_k, const void* sink_v, const void* win_k,
                                  const void* win_v, const void* bases_k, const void* bases_v, void* coef_k,
                                  void* coef_v, const void* k_new, const void* v_new, float* out, int32_t* idx_out,
                                  float* scores_out, void* ws, size_t ws_bytes, hipStream_t stream) {
  Problem P;
  s4r_status st = make_problem(cfg, P);
  if (st) return st;
  if (!lengths) return fail(S4R_ERR_NULL_ARG, "lengths is NULL");
  if (P.B > kMaxRaggedB) return fail(S4R_ERR_UNSUPPORTED, "ragged batch of %d sequences exceeds %d", P.B, kMaxRaggedB);
  int64_t L = 0, m0 = -1;
  P.lens.n = P.B;
  for (int b = 0; b < P.B; ++b) {
    const int64_t Lb = lengths[b];
    if ((st = check_L(P, Lb))) return st;
    // every sequence selects the same number of tokens (the index rows share a stride)
    const int64_t mb = std::min<int64_t>(P.k, std::max<int64_t>(Lb - P.W, 0)) + std::min<int64_t>(P.W, Lb);
    if (m0 >= 0 && mb != m0)
      return fail(S4R_ERR_BAD_SHAPE, "ragged lengths must give every sequence the same selected count (%lld vs %lld at b = %d)",
                  (long long)m0, (long long)mb, b);
    m0 = mb;
    L = std::max(L, Lb);
    P.lens.v[b] = (int32_t)Lb;
  }
  return decode_step_impl(P, L, q, qwin_prev, sink_k, sink_v, win_k, win_v, bases_k, bases_v, coef_k, coef_v, k_new,
                          v_new, out, idx_out, scores_out, ws, ws_bytes, stream);
}

s4r_status s4r_decode_step_noalloc(const s4r_config* cfg, int64_t L, const void* q, const float* qwin_prev,
                                   const void* sink_k, const void* sink_v, const void* win_k, const void* win_v,
                                   const void* bases_k, const void* bases_v, void* coef_k, void* coef_v,
                                   const void* k_new, const void* v_new, float* out, int32_t* idx_out,
                                   float* scores_out, hipStream_t stream) {
  Problem P;
  s4r_status st = make_problem(cfg, P);
  if (st) return st;
  if ((st = check_L(P, L))) return st;
  const size_t need = layout(P).total;
  if (need > kScratchBytes)
    return fail(S4R_ERR_WORKSPACE, "this configuration needs %zu bytes of scratch, more than the %zu the library "
                "holds per device; use s4r_decode_step with a workspace", need, kScratchBytes);
  void* ws = nullptr;
  if ((st = scratch_address(&ws))) return st;
  return decode_step_impl(P, L, q, qwin_prev, sink_k, sink_v, win_k, win_v, bases_k, bases_v, coef_k, coef_v, k_new,
                          v_new, out, idx_out, scores_out, ws, kScratchBytes, stream);
}

s4r_status s4r_project_append(const s4r_config* cfg, int64_t row, const void* k_new, const void* v_new,
                              const void* bases_k, const void* bases_v, void* coef_k, void* coef_v,
                              hipStream_t stream) {
  Problem P;
  s4r_status st = make_problem(cfg, P);
  if (st) return st;
  if (row < 0 || row >= P.cap) return fail(S4R_ERR_BAD_SHAPE, "row %lld outside [0, capacity)", (long long)row);
  S4R_REQ(k_new);
  S4R_REQ(v_new);
  S4R_REQ(bases_k);
  S4R_REQ(bases_v);
  S4R_REQ(coef_k);
  S4R_REQ(coef_v);
  return hip_status(launch_project_rows(P, bases_k, bases_v, k_new, v_new, coef_k, coef_v, row, stream),
                    "s4r_project_append launch");
}

static s4r_status pack_common(const s4r_config* cfg, int64_t n_rows, const void* src, void* dst, bool to_tiled,
                              hipStream_t stream) {
  Problem P;
  s4r_status st = make_problem(cfg, P);
  if (st) return st;
  if (n_rows < 0 || n_rows > P.cap)
    return fail(S4R_ERR_BAD_SHAPE, "n_rows %lld outside [0, capacity]", (long long)n_rows);
  S4R_REQ(src);
  S4R_REQ(dst);
  return hip_status(launch_pack(P, n_rows, src, dst, to_tiled, stream), "s4r_pack launch");
}

s4r_status s4r_pack_coef(const s4r_config* cfg, int64_t n_rows, const void* src_rowmajor, void* dst_tiled,
                         hipStream_t stream) {
  return pack_common(cfg, n_rows, src_rowmajor, dst_tiled, true, stream);
}

s4r_status s4r_unpack_coef(const s4r_config* cfg, int64_t n_rows, const void* src_tiled, void* dst_rowmajor,
                           hipStream_t stream) {
  return pack_common(cfg, n_rows, src_tiled, dst_rowmajor, false, stream);
}

int64_t s4r_read_bandwidth_sink_len(void) { return read_bandwidth_threads(); }

s4r_status s4r_read_bandwidth(const void* buf, int64_t bytes, uint32_t* sink, hipStream_t stream) {
  S4R_REQ(buf);
  S4R_REQ(sink);
  if (bytes <= 0 || bytes % 16) return fail(S4R_ERR_BAD_SHAPE, "bytes %lld must be a positive multiple of 16",
                                             (long long)bytes);
  return hip_status(launch_read_all(buf, bytes / 16, sink, stream), "s4r_read_bandwidth launch");
}

s4r_status s4r_timing_enable(int32_t max_steps) {
  std::lock_guard<std::mutex> lk(g_timing.mu);
  if (max_steps < 1 || max_steps > 10000) return fail(S4R_ERR_BAD_SHAPE, "max_steps %d outside [1, 10000]", max_steps);
  for (auto ev : g_timing.start) (void)hipEventDestroy(ev);
  for (auto ev : g_timing.stop) (void)hipEventDestroy(ev);
  const int n = max_steps * S4R_TIMED_KERNELS;
  g_timing.start.assign(n, nullptr);
  g_timing.stop.assign(n, nullptr);
  for (int i = 0; i < n; ++i) {
    if (hipEventCreate(&g_timing.start[i]) != hipSuccess || hipEventCreate(&g_timing.stop[i]) != hipSuccess)
      return fail(S4R_ERR_HIP, "hipEventCreate failed");
  }
  g_timing.steps = max_steps;
  g_timing.used = 0;
  g_timing.enabled = true;
  return ok();
}

s4r_status s4r_timing_read(double* total_ms, int64_t* steps) {
  std::lock_guard<std::mutex> lk(g_timing.mu);
  if (!total_ms || !steps) return fail(S4R_ERR_NULL_ARG, "total_ms / steps is NULL");
  for (int k = 0; k < S4R_TIMED_KERNELS; ++k) total_ms[k] = 0.0;
  for (int i = 0; i < g_timing.used; ++i) {
    for (int k = 0; k < S4R_TIMED_KERNELS; ++k) {
      float ms = 0.f;
      const int s = i * S4R_TIMED_KERNELS + k;
      if (hipEventSynchronize(g_timing.stop[s]) != hipSuccess ||
          hipEventElapsedTime(&ms, g_timing.start[s], g_timing.stop[s]) != hipSuccess)
        return fail(S4R_ERR_HIP, "reading kernel timing events failed");
      total_ms[k] += ms;
    }
  }
  *steps = g_timing.used;
  for (auto ev : g_timing.start) (void)hipEventDestroy(ev);
  for (auto ev : g_timing.stop) (void)hipEventDestroy(ev);
  g_timing.start.clear();
  g_timing.stop.clear();
  g_timing.steps = 0;
  g_timing.used = 0;
  g_timing.enabled = false;
  return ok();
}

}  // extern "C"
