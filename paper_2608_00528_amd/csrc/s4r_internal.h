// Host-side internals of the S^4R library: the validated problem description,
// the workspace carving, and the launchers each kernel file provides.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <cmath>

#include "s4r.h"

namespace s4r {

constexpr int kScoreWaves = 4;        // waves per scoring workgroup
constexpr int kHistBins = 2048;       // top-11-bit radix histogram of the scores
constexpr int kHistShift = 21;
// copies of the top-level histogram: workgroup i of a sequence adds into copy
// i mod nc and the selection sums the nc copies.  Global atomics on one address
// from hundreds of workgroups serialise (about 4 us for 469 workgroups
// flushing 32 bins into one copy on MI355X, none measurable with 8 copies).
constexpr int kHistCopies = 8;
constexpr int kHistStride = (kHistCopies + 1) * kHistBins;   // per sequence: the copies, then level 2
// copies for a histogram that `wgs` workgroups per sequence flush: one per 64
// workgroups, a power of two up to kHistCopies
inline int hist_copies(int64_t wgs) {
  int nc = 1;
  while (nc < kHistCopies && wgs > 64 * nc) nc *= 2;
  return nc;
}
constexpr int kHistChunk = 2048;      // tokens per histogram workgroup (standalone selection)
constexpr int kSelChunk = 2048;       // tokens per selection workgroup (multiple of 32)
constexpr int kMaxSelGroups = 4096;   // classify workgroups per sequence (capacity <= 4096 * kSelChunk)
constexpr int kMaxSplit = 64;         // attention splits per (sequence, kv head)
constexpr int kMaxTilesPerSplit = 512; // 16-token tiles per split (index list staged in LDS)
constexpr int kTileMax = 32;          // tiles per workgroup of the MFMA attention kernel (index list in LDS)
constexpr int kMaxG = 16;             // query groups G = h_q / h_kv
constexpr int kColBlk = 16;           // query columns (G * W_q) per scoring workgroup
constexpr int kMaxGW = 128;           // G * W_q: up to 8 column blocks
constexpr int kPChunk = 256;          // basis rows per projection chunk (one per thread)
constexpr int kQMaxChunks = 8;        // row chunks per basis group (Dp / basis_groups <= 2048)

// per-sequence lengths of a ragged batch, passed to the kernels by value
// (n = 0: every sequence has the call's L)
constexpr int kMaxRaggedB = 64;
struct Lens {
  int32_t n;
  int32_t v[kMaxRaggedB];
};
__host__ __device__ inline int64_t len_of(const Lens& l, int b, int64_t L) { return l.n ? (int64_t)l.v[b] : L; }

// the (key, value) rank pairs the kernel is built for, in 32-column blocks:
// equal ranks 32 .. 256 (224 holds the paper's r = 204 of Appendix B.4), and
// the value-heavy pairs near 1:1.5 and 1:2 of Appendix D.2 for the totals
// 2 r = 256, 320 and 384
constexpr bool tiles_rank_pair(int rbk, int rbv) {
  return (rbk == rbv && rbk >= 1 && rbk <= 8) || (rbk == 3 && rbv == 5) ||
         (rbk == 2 && rbv == 6) || (rbk == 4 && rbv == 6) || (rbk == 3 && rbv == 7) || (rbk == 5 && rbv == 7) ||
         (rbk == 4 && rbv == 8);
}

struct Problem {
  int B, hq, hkv, dh, G, Dp;
  int nb, rank, R, Dg;                // basis groups, rank per group, R = nb*rank, Dg = Dp/nb; rank is
                                      // the storage width (the configured rank rounded up to 32)
  int rank_v, Rv;                     // the value side's (= rank, R unless asymmetric)
  int rank_cfg, rank_v_cfg;           // the configured ranks (columns past them are zero padding)
  int R_cfg;                          // nb * rank_cfg: the latent width of the 1 / sqrt(R) scale
  int s, W, Wq, k, kappa, pool_mode, agg;
  int bases_shared, dtype;
  int64_t cap;
  float theta;
  int GW;                             // G * Wq
  int64_t nruns_max;                  // 16-token tiles at L = cap (one softmax reference each)
  int64_t nwg_max;                    // scoring workgroups per sequence, any L <= cap
  int64_t m_max;                      // selected tokens at L = cap
  Lens lens;                          // ragged batch (n = 0: uniform)
};

struct Workspace {
  uint16_t* qimg;       // [B][column blocks][qimg_mfmas][16][R] the scoring kernel's A operands (bf16 parts)
  float* qcoef;         // [B][G][R] the step's query coefficients c_t^Q (fp32)
  float* e;             // [B][cap][GWP]  exp(z - running max), fp32, token-major
  float* run_m;         // [B][cap / 16][GWP] per-tile softmax reference (running max of z)
  double* wg_stats;     // [B][GW][nwg_max][2] per scoring workgroup (max, sum)
  double* col_stats;    // [B][GW][2]     global (max, 1 / sum) per query column, when folded by k_fold_stats
  float* atilde;        // [B][cap]       relevance scores
  uint32_t* hist;       // [B][kHistCopies + 1][kHistBins]  selection histograms: copies of the top 11 key bits, next 11 of the boundary bin
  uint64_t* cand;       // [B][cand_stride]  per-classify-workgroup candidate regions (key << 32 | ~index)
  uint32_t* cand_count; // [B][sel_groups_max] candidates found by each classify workgroup
  uint32_t* above_count; // [B][sel_groups_max] positions above the boundary bin per classify workgroup
  uint32_t* sel_info;   // [B][4] boundary bin and the count above it
  uint32_t* bitmap;     // [B][bitmap_words(cap)]  selected global positions
  int32_t* idx;         // [B][m_max]
  float* part_ml;       // [B][hq][kMaxSplit][2]   split partial (max, sum)
  float* part_o;        // [B][hq][kMaxSplit][dh]  split partial outputs
  float* attn_logits;   // [B][hq][s + m_max]      explicit-attention scratch
  size_t total;
};

Workspace carve_workspace(const Problem& P, void* base);
int score_workgroups(const Problem& P, int64_t L);
// bitmap words of one sequence (rounded up: a capacity that is an odd
// multiple of 16 ends in half a word)
__host__ __device__ inline int64_t bitmap_words(int64_t cap) { return (cap + 31) / 32; }
inline int64_t sel_groups_max(const Problem& P) { return (P.cap + kSelChunk - 1) / kSelChunk; }
inline int64_t cand_stride(const Problem& P) { return sel_groups_max(P) * kSelChunk; }
// query columns G * W_q rounded up to a multiple of 4 (one 16-byte group per
// MFMA of the scoring kernel): the column stride of the exp values
inline int gw_padded(const Problem& P) { return P.GW <= kColBlk ? (P.GW + 3) / 4 * 4 : (P.GW + kColBlk - 1) / kColBlk * kColBlk; }
// column blocks of the scoring pass (one per kColBlk query columns)
inline int col_blocks(const Problem& P) { return (P.GW + kColBlk - 1) / kColBlk; }
// MFMAs (4 query columns each) per column block of the scoring pass
inline int qimg_mfmas(const Problem& P) { return std::min((P.GW + 3) / 4, kColBlk / 4); }
// RoPE: ratio of consecutive frequencies theta^(-2 / d_h) (0 when RoPE is off)
inline double rope_ratio(const Problem& P) { return P.theta == 0.f ? 0.0 : pow((double)P.theta, -2.0 / P.dh); }

// ---- launchers (each returns hipGetLastError() after its launches) --------

// coefficient projections of Section 3.2.1: the query groups (fp32 c_t^Q
// into ws.qcoef and qcoef_out when given; with `image`, the scoring kernel's
// operand image ws.qimg, the window's older rows from qwin_prev) and a new
// token's key and value rows (into row `row` of the caches)
hipError_t launch_project_query(const Problem& P, const Workspace& ws, const void* q, const void* bases_k,
                                const float* qwin_prev, float* qcoef_out, bool image, hipStream_t st);
hipError_t launch_project_rows(const Problem& P, const void* bases_k, const void* bases_v, const void* k_new,
                               const void* v_new, void* coef_k, void* coef_v, int64_t row, hipStream_t st);
// the operand image of a window given as coefficient rows [B][G][Wq][R] (P0.Wq rows)
hipError_t launch_query_image_rows(const Problem& P0, const Workspace& ws, const float* rows, hipStream_t st);
// windowed relevance (P1: the newest row's G columns, Wq = 1): the older rows'
// softmax from the window state [B][wrows][G][cap], the newest stored in its slot
// window state: [B][W_q][G][cap] fp32 softmax rows; with more than
// kWinDirectRows rows also the older rows' running sum [2][B][G][cap] fp64
// (per step 20 bytes per position and group instead of 4 per older row)
constexpr int kWinDirectRows = 5;
inline size_t window_state_bytes(const Problem& P) {
  size_t n = (size_t)P.B * P.Wq * P.G * P.cap * sizeof(float);
  if (P.Wq > kWinDirectRows) n += (size_t)2 * P.B * P.G * P.cap * sizeof(double);
  return n;
}
inline double* window_rsum(const Problem& P, float* state, int wrows) {
  return wrows > kWinDirectRows ? reinterpret_cast<double*>(state + (size_t)P.B * wrows * P.G * P.cap) : nullptr;
}
hipError_t launch_relevance_windowed(const Problem& P1, const Workspace& ws, int64_t L, float* scores_out,
                                     float* state, int wrows, hipStream_t st);
// window state of the older rows from a stream over them (P0: wrows - 1 rows, length L - 1)
hipError_t launch_window_store(const Problem& P0, const Workspace& ws, int64_t L, float* state, int wrows,
                               hipStream_t st);
hipError_t launch_score_stream(const Problem& P, const Workspace& ws, int64_t L, const void* coef_k, hipStream_t st);
hipError_t launch_relevance(const Problem& P, const Workspace& ws, int64_t L, float* scores_out,
                            hipStream_t st);
// histogram copies the step's relevance kernel flushes into (wrows >= 2: the
// windowed kernel over P with W_q = 1)
int relevance_hist_copies(const Problem& P, int64_t L, int wrows);
hipError_t launch_hist_only(const Problem& P, const Workspace& ws, int64_t L, const float* scores,
                            hipStream_t st);
hipError_t launch_select(const Problem& P, const Workspace& ws, int64_t L, const float* scores,
                         int64_t score_stride, int32_t* idx, int32_t* idx_copy, hipStream_t st);
hipError_t launch_full_recon(const Problem& P, const Workspace& ws, int64_t L, const void* q, const void* sink_k,
                             const void* sink_v, const void* bases_k, const void* bases_v, const void* coef_k,
                             const void* coef_v, float* out, hipStream_t st);
// basis construction of the prefill (bases.hip)
void bases_sample_counts(int64_t T, double eta, int* n_uniform, int* n_recent);
hipError_t prefill_bases_ws_bytes(const Problem& P, int n_s, size_t* bytes);
hipError_t launch_prefill_bases(const Problem& P, int64_t n_rows, const void* s_k, const void* s_v, int n_uniform,
                                int n_recent, int center, int32_t* idx_out, void* bases_k, void* bases_v, void* ws,
                                size_t ws_bytes, hipStream_t st);
hipError_t launch_project_queries(const Problem& P, const Workspace& ws, int64_t n_rows, const void* q_rows,
                                  const void* bases_k, float* out, hipStream_t st);
hipError_t launch_dense_decode(const Problem& P, const Workspace& ws, int64_t N, const void* q, const void* k_cache,
                               const void* v_cache, float* out, hipStream_t st);
hipError_t launch_project_step(const Problem& P, const Workspace& ws, const void* q, const void* bases_k,
                               const void* bases_v, const void* k_new, const void* v_new, void* coef_k, void* coef_v,
                               const float* qwin_prev, int64_t row, hipStream_t st);
size_t prefill_ws_bytes(const Problem& P);
hipError_t launch_prefill_project(const Problem& P, int64_t n_rows, const void* s_k, const void* s_v,
                                  const void* bases_k, const void* bases_v, void* coef_k, void* coef_v, void* ws,
                                  hipStream_t st);
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
// read-bandwidth reference: XOR of every word, one value per thread in sink
int read_bandwidth_threads();
hipError_t launch_read_all(const void* buf, int64_t n16, uint32_t* sink, hipStream_t st);
hipError_t launch_pack(const Problem& P, int64_t n_rows, const void* src, void* dst, bool to_tiled,
                       hipStream_t st);

}  // namespace s4r
