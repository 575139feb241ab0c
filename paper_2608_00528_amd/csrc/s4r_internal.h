// Host-side internals of the S^4R library: the validated problem description,
// the workspace carving, and the launchers each kernel file provides.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/s4r.h"

namespace s4r {

constexpr int kRunTiles = 4;          // coefficient tiles per softmax run (64 tokens)
constexpr int kRunTok = kRunTiles * 16;
constexpr int kScoreWaves = 4;        // waves per scoring workgroup
constexpr int kHistBins = 4096;       // top-12-bit radix histogram of the scores
constexpr int kHistShift = 20;
constexpr int kRelChunk = 1024;       // tokens per relevance workgroup
constexpr int kSelChunk = 2048;       // tokens per selection workgroup (multiple of 32)
constexpr int kCandCap = 4096;        // boundary candidates sorted in LDS
constexpr int kMaxSplit = 64;         // attention splits per (sequence, kv head)
constexpr int kMaxGW = 16;            // G * W_q columns handled by one MFMA block
constexpr int kCounters = 8;          // per-sequence counters in the workspace

struct Problem {
  int B, hq, hkv, dh, G, Dp;
  int nb, rank, R, Dg;                // basis groups, rank per group, R = nb*rank, Dg = Dp/nb
  int s, W, Wq, k, kappa, pool_mode, agg;
  int bases_shared, dtype;
  int64_t cap;
  float theta;
  int GW;                             // G * Wq
  int64_t nruns_max;                  // softmax runs at L = cap
  int64_t m_max;                      // selected tokens at L = cap
};

struct Workspace {
  uint16_t* cq_split;   // [B][3][GW][R] bf16 bits: hi, mid, lo of the query coefficients
  float* e;             // [B][GW][cap]   exp(z - run max), fp32
  double* run_m;        // [B][GW][nruns] run maxima of z
  double* run_s;        // [B][GW][nruns] run sums of e
  double* gstat;        // [B][GW][2]     global max M and normaliser S
  float* atilde;        // [B][cap]       relevance scores
  uint32_t* hist;       // [B][kHistBins]
  uint32_t* counters;   // [B][kCounters]
  uint64_t* cand;       // [B][cap]       boundary candidates (key << 32 | ~index)
  uint32_t* bitmap;     // [B][cap / 32]  selected global positions
  int32_t* idx;         // [B][m_max]
  float* part_ml;       // [B][hq][kMaxSplit][2]   split partial (max, sum)
  float* part_o;        // [B][hq][kMaxSplit][dh]  split partial outputs
  float* attn_logits;   // [B][hq][s + m_max]      explicit-attention scratch
  size_t total;
};

Workspace carve_workspace(const Problem& P, void* base);

// ---- launchers (each returns hipGetLastError() after its launches) --------
hipError_t launch_prepare(const Problem& P, const Workspace& ws, int64_t L, const void* q,
                          const float* qwin_prev, const void* bases_k, const void* bases_v,
                          const void* k_new, const void* v_new, void* coef_k, void* coef_v,
                          int64_t append_row, float* qcoef_out, bool do_query, bool clear,
                          hipStream_t st);
hipError_t launch_score_stream(const Problem& P, const Workspace& ws, int64_t L,
                               const void* coef_k, hipStream_t st);
hipError_t launch_relevance(const Problem& P, const Workspace& ws, int64_t L, float* scores_out,
                            hipStream_t st);
hipError_t launch_hist_only(const Problem& P, const Workspace& ws, int64_t L, const float* scores,
                            hipStream_t st);
hipError_t launch_select(const Problem& P, const Workspace& ws, int64_t L, const float* scores,
                         int64_t score_stride, int32_t* idx, int32_t* idx_copy, hipStream_t st);
hipError_t launch_attention(const Problem& P, const Workspace& ws, int64_t L, int m, int k_eff,
                            const void* q, const void* sink_k, const void* sink_v,
                            const void* win_k, const void* win_v, const void* bases_k,
                            const void* bases_v, const void* coef_k, const void* coef_v,
                            float* out, hipStream_t st, hipEvent_t* t0, hipEvent_t* t1);
hipError_t launch_reconstruct(const Problem& P, int64_t L, int m, const int32_t* idx,
                              const void* bases_k, const void* bases_v, const void* coef_k,
                              const void* coef_v, float* k_hat, float* v_hat, hipStream_t st);
hipError_t launch_sparse_attn(const Problem& P, const Workspace& ws, int64_t L, int m,
                              const void* q, const void* sink_k, const void* sink_v,
                              const int32_t* idx, const float* k_sel, const float* v_sel,
                              float* out, hipStream_t st);
bool attention_supported(const Problem& P);
hipError_t launch_pack(const Problem& P, int64_t n_rows, const void* src, void* dst, bool to_tiled,
                       hipStream_t st);

}  // namespace s4r
