/*
 * s4r.h - C ABI of the S^4R decode-step library for AMD MI355X (gfx950).
 *
 * S^4R (arxiv 2608.00528) keeps a layer's KV cache as full-precision sink
 * tokens plus low-rank coefficients of every other token on per-sequence key
 * and value bases (Section 3.1).  One decode step (Section 3.2) scores every
 * cached token in the latent space, keeps the local window plus the top-k
 * tokens, reconstructs only those as coefficients times basis, applies RoPE
 * at their original positions and runs GQA softmax attention over sinks and
 * reconstructed tokens.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Array pointers are DEVICE pointers, 16-byte aligned, densely packed in
 *    the layouts stated below.  The caller owns all memory; the library does
 *    not allocate device memory on any compute call (the exceptions are named
 *    where they apply: the rocBLAS handle of the basis construction and the
 *    fixed scratch array of s4r_decode_step_noalloc).  Scratch lives in the
 *    caller's workspace, whose
 *    size s4r_workspace_size() returns; its initial contents do not matter.
 *  - Every call is asynchronous on the caller's hipStream_t and performs no
 *    host synchronisation.  Calls that share a workspace must not overlap.
 *  - Arguments are validated on the host before anything is launched.  On
 *    error nothing is launched, no output is touched, the status code says
 *    what class of problem it was and s4r_last_error() (thread-local) says
 *    which argument.  A failed launch returns S4R_ERR_HIP.
 *  - Storage dtype (cfg.dtype) applies to q, sinks, window KV, new K/V rows,
 *    bases and coefficient caches.  Query coefficients and all outputs are
 *    fp32; indices are int32.
 *
 * Notation (paper): B batch, h_q / h_kv query / KV heads, G = h_q / h_kv,
 * d_h head dim, Dp = h_kv * d_h, R = basis_groups * rank (latent width r of
 * the paper), s sinks, W local window, W_q query-coefficient rows, k global
 * budget, L the current non-sink length (the token appended this step
 * included), m = min(k, max(L - W, 0)) + min(W, L) selected tokens.
 *
 * Rank stride: every latent axis is stored rank_s = 32 * ceil(rank / 32)
 * columns wide per basis group (the coefficient layout works in 32-column
 * blocks).  When rank is not a multiple of 32 (the paper's r = 204 of
 * Appendix B.4 is stored in 224 columns), group beta's columns are
 * beta * rank_s .. beta * rank_s + rank - 1 and the rest of its rank_s
 * columns must hold zeros in the bases (the library's own basis construction
 * writes them; projections from zero-padded bases write zero coefficients).
 * Below, R stands for basis_groups * rank_s in every layout; the 1 / sqrt(R)
 * scale of the latent logits (Section 3.2.2) takes the configured
 * basis_groups * rank.
 *
 * Layouts
 * -------
 *  q          [B, h_q, d_h]            pre-RoPE query, head h reads KV head h / G
 *  sink_k/v   [B, s, Dp]               pre-RoPE sink keys / values (Section 3.1.1)
 *  win_k/v    [B, W, Dp]               exact KV of positions L-W .. L-1 (optional)
 *  bases_k/v  [B or 1, basis_groups, Dp / basis_groups, rank], rank fastest
 *             (bases_v: rank_v when set).
 *             Group beta spans KV heads beta*h_kv/basis_groups onward; the
 *             paper's single basis over Dp is basis_groups = 1 (Eq. svd).
 *  coef_k/v   per sequence a [capacity, R] matrix (the value cache
 *             [capacity, R_V] when rank_v is set) in the TILED layout:
 *             element (t, c) of sequence b is at
 *               b*capacity*R + (t/16)*16*R + (c/32)*512 + (t%16)*32 + (c%32)
 *             i.e. 16-token tiles, each split into 32-column blocks of
 *             16 x 32 elements, token-major inside a block.  capacity % 16 == 0
 *             and R % 32 == 0.  s4r_pack_coef / s4r_unpack_coef convert from /
 *             to row-major [B, n, R].
 *  qwin_prev  [B, G, W_q - 1, R] fp32  older query coefficients, oldest first
 *  qcoef_out  [B, G, R] fp32           c_t^Q of this step (for the caller's FIFO)
 *  scores     [B, L] fp32              relevance A~ of every non-sink token
 *  idx        [B, m] int32             selected non-sink positions: the global
 *                                      picks ascending, then the window ascending
 *  k_hat/v_hat[B, m, Dp] fp32          reconstructed pre-RoPE keys / values
 *  out        [B, h_q, d_h] fp32       attention output O_t
 */
#ifndef S4R_H
#define S4R_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  S4R_OK = 0,
  S4R_ERR_NULL_ARG = 1,     /* a required pointer is NULL                      */
  S4R_ERR_BAD_SHAPE = 2,    /* sizes inconsistent (e.g. L > capacity, h_q % h_kv) */
  S4R_ERR_UNSUPPORTED = 3,  /* valid but outside what the kernels implement     */
  S4R_ERR_WORKSPACE = 4,    /* workspace smaller than s4r_workspace_size()      */
  S4R_ERR_MISALIGNED = 5,   /* a pointer is not 16-byte aligned                 */
  S4R_ERR_HIP = 6           /* a HIP call or kernel launch failed               */
} s4r_status;

enum { S4R_FP32 = 0, S4R_BF16 = 1 };          /* storage dtype                    */
enum { S4R_POOL_MAX = 0, S4R_POOL_AVG = 1 };  /* F_P of Section 3.2.3 (default max)  */
enum { S4R_AGG_MEAN = 0, S4R_AGG_MAX = 1 };   /* F_G of Section 3.2.3 (default mean) */

typedef struct {
  int32_t batch;         /* B                                                      */
  int32_t n_q_heads;     /* h_q, a multiple of n_kv_heads                          */
  int32_t n_kv_heads;    /* h_kv                                                   */
  int32_t head_dim;      /* d_h: 64 or 128                                         */
  int32_t basis_groups;  /* 1 = one basis over Dp (paper); must divide n_kv_heads  */
  int32_t rank;          /* rank per basis group, <= Dp/basis_groups, stored in
                            32 * ceil(rank / 32) columns (the rank stride above);
                            the key rank r^K when rank_v is set                    */
  int32_t n_sink;        /* s, sink tokens kept at full precision (Section 3.1.1)  */
  int32_t window;        /* W, local window always kept (Section 3.2.3)            */
  int32_t q_window;      /* W_q >= 1 query-coefficient rows used for scoring (3.2.2);
                            G * W_q <= 128 (the paper's W_q = 32 at G = 4), G <= 16 */
  int32_t topk;          /* k, global budget; clamped to max(L - W, 0)             */
  int32_t pool_kernel;   /* kappa, odd, 1 = no pooling                             */
  int32_t pool_mode;     /* S4R_POOL_MAX | S4R_POOL_AVG                            */
  int32_t group_agg;     /* S4R_AGG_MEAN | S4R_AGG_MAX                             */
  int32_t bases_shared;  /* 1: bases have no batch axis (one basis for all sequences) */
  int64_t capacity;      /* token rows allocated in each coefficient cache, % 16 == 0 */
  float rope_theta;      /* RoPE base; 0 disables RoPE                             */
  int32_t dtype;         /* S4R_FP32 | S4R_BF16                                    */
  int32_t rank_v;        /* 0: values share `rank`; else the value rank r^V per basis
                            group (Appendix D.2: r^K <= r^V), <= Dp/basis_groups,
                            stored with its own rank stride.  The value cache and basis are then
                            [.., R_V = basis_groups * rank_v] wide; asymmetric
                            ranks run on the bf16 matrix-core path for the rank
                            pairs s4r_decode_step lists                            */
} s4r_config;

/* Bytes of workspace any call with this config needs (host only, no GPU). */
s4r_status s4r_workspace_size(const s4r_config* cfg, size_t* bytes);

/* m = min(k, max(L - W, 0)) + min(W, L) (Section 3.3); -1 if cfg or L is invalid. */
int32_t s4r_num_selected(const s4r_config* cfg, int64_t L);

/* Thread-local description of the last error ("" after success). */
const char* s4r_last_error(void);

/* Library version string. */
const char* s4r_version(void);

/*
 * Latent relevance (Section 3.2.2 and the pooling / group-aggregation
 * equations of 3.2.3): c_t^Q = s_t^Q B^K per group, C^Q = [qwin_prev; c_t^Q],
 * Z = C^Q (C^K)^T / sqrt(R) over the L non-sink tokens, causal mask, softmax
 * over L, mean over the W_q rows, pooling with kernel kappa, aggregation
 * over G -> scores[b, l].  qwin_prev may be NULL only when W_q == 1;
 * qcoef_out may be NULL.
 */
s4r_status s4r_score_latent(const s4r_config* cfg, int64_t L, const void* q,
                            const float* qwin_prev, const void* bases_k,
                            const void* coef_k, float* scores, float* qcoef_out,
                            void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Index selection (Section 3.2.3): I_local = [max(L - W, 0), L),
 * I_global = the k_eff largest scores[b, 0 : L - W] (equal scores go to the
 * lower position), idx[b] = sorted(I_global) followed by I_local.  Bit-exact
 * and deterministic for a given scores array.  Scores must be non-negative
 * and finite (as the relevance A~ is); their order is taken from their bits.
 */
s4r_status s4r_select_topk(const s4r_config* cfg, int64_t L, const float* scores,
                           int32_t* idx, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Sparse reconstruction (Section 3.2.3): k_hat[b, n] = C^K[b, idx[b, n]] (B^K)^T,
 * v_hat likewise, per basis group, pre-RoPE, fp32.  idx entries must lie in
 * [0, L); m is the number of indices per sequence.  Equal key and value ranks
 * only (rank_v set to another rank: S4R_ERR_UNSUPPORTED).
 */
s4r_status s4r_reconstruct(const s4r_config* cfg, int64_t L, int32_t m, const int32_t* idx,
                           const void* bases_k, const void* bases_v, const void* coef_k,
                           const void* coef_v, float* k_hat, float* v_hat, hipStream_t stream);

/*
 * Final attention (Section 3.2.3): K* = [sink_k; k_sel], V* = [sink_v; v_sel]
 * at positions [0 .. s-1, s + idx], query at s + L - 1, RoPE on q and K*,
 * out[b, h] = softmax(RoPE(q_h) RoPE(K*_j)^T / sqrt(d_h)) V*_j with j = h / G.
 * k_sel / v_sel are fp32 [B, m, Dp] pre-RoPE rows (e.g. from s4r_reconstruct).
 */
s4r_status s4r_sparse_attn(const s4r_config* cfg, int64_t L, int32_t m, const void* q,
                           const void* sink_k, const void* sink_v, const int32_t* idx,
                           const float* k_sel, const float* v_sel, float* out,
                           void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * One fused decode step of one layer (Section 3.2): optional cache update
 * (k_new / v_new [B, Dp] projected and written into coefficient row L - 1,
 * Section 3.2.1), latent scoring, selection, reconstruction of the selected
 * keys and values, RoPE and attention.  Reconstructed keys and values stay
 * on chip and are never written to memory.  win_k / win_v
 * may be NULL (the paper: the window is reconstructed like every selected
 * token); if given they replace the window rows with exact KV.  idx_out
 * [B, m] and scores_out [B, L] are optional copies of the selection.
 * coef_k / coef_v are written only when k_new / v_new are given.
 * Asymmetric ranks (rank_v set, Appendix D.2) run for bf16 storage, head_dim
 * 64 or 128, G <= 8, m <= 32768 and the (rank, rank_v) pairs (96, 160),
 * (64, 192), (128, 192), (96, 224), (160, 224), (128, 256); other settings
 * return S4R_ERR_UNSUPPORTED.
 */
s4r_status s4r_decode_step(const s4r_config* cfg, int64_t L, const void* q,
                           const float* qwin_prev, const void* sink_k, const void* sink_v,
                           const void* win_k, const void* win_v, const void* bases_k,
                           const void* bases_v, void* coef_k, void* coef_v,
                           const void* k_new, const void* v_new, float* out,
                           int32_t* idx_out, float* scores_out, void* ws, size_t ws_bytes,
                           hipStream_t stream);

/*
 * s4r_decode_step without a caller workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Arguments, outputs and errors are those
 * of s4r_decode_step without ws / ws_bytes.  The workspace is a 64 MiB array
 * the library holds on each device that runs this call (from its first call
 * on the device until the process ends); the call itself allocates nothing.
 * A configuration whose s4r_workspace_size exceeds 64 MiB returns
 * S4R_ERR_WORKSPACE before anything is launched.  The stream must belong to
 * the current device.  Every call on a device shares that device's array and
 * leaves its contents behind (the step clears what it needs cleared itself):
 * calls that overlap on one device, from several streams or host threads,
 * race on it and must be serialised by the caller.
 */
s4r_status s4r_decode_step_noalloc(const s4r_config* cfg, int64_t L, const void* q,
                                   const float* qwin_prev, const void* sink_k, const void* sink_v,
                                   const void* win_k, const void* win_v, const void* bases_k,
                                   const void* bases_v, void* coef_k, void* coef_v,
                                   const void* k_new, const void* v_new, float* out,
                                   int32_t* idx_out, float* scores_out, hipStream_t stream);

/*
 * Windowed decode (Section 3.2.2 with q_window >= 2): the latent scores of
 * query row i of the window are the softmax over keys 0 .. L - W_q + i, and
 * that key range and those keys' coefficients are the same at every later
 * step the row stays in the window (the cache only grows by appended rows).
 * The row's softmax over its keys therefore never changes once it has been
 * computed, so a caller that keeps it on the device needs to score only the
 * newest query row at each step.  The window state holds, per sequence, the
 * softmax of the last W_q query rows over their keys:
 *   state [B, q_window, G, capacity] fp32 (device, caller-owned, 16-byte
 *   aligned, s4r_window_state_size bytes in all); the row that was the newest
 *   at length L_r (it covers keys 0 .. L_r - 1) sits in slot L_r mod q_window.
 *   With q_window > 5 the older rows' sum per key follows, as fp64
 *   [2, B, G, capacity] (two buffers chosen by the parity of L): each step
 *   reads one, writes the other with the newest row added and the row leaving
 *   the window subtracted, so a step reads 20 bytes per key and group instead
 *   of 4 per older row.  The state's contents are the library's.
 *
 * s4r_window_state_init fills the state for the q_window - 1 older rows of
 * the window of a step at length L, from their coefficient rows qwin_prev
 * [B, G, q_window - 1, R] fp32 (the qwin_prev of s4r_decode_step) and the
 * coefficient cache (rows 0 .. L - 2 read).  s4r_decode_step_windowed then
 * equals s4r_decode_step at length L with that qwin_prev (up to the rounding
 * of the older rows' coefficients and of the summation order of the window
 * mean), and stores the newest row's softmax in slot L mod q_window, so the
 * next call, at length L + 1, finds the window of the step after: a sequence
 * of windowed steps must run at consecutive lengths L, L + 1, ... (one
 * appended token per step, as decoding does); the state is not valid for any
 * other length.  Arguments and outputs of s4r_decode_step_windowed are those
 * of s4r_decode_step with state in place of qwin_prev; q_window >= 2 and a
 * uniform batch, else S4R_ERR_BAD_SHAPE / S4R_ERR_UNSUPPORTED.
 */
s4r_status s4r_window_state_size(const s4r_config* cfg, size_t* bytes);
s4r_status s4r_window_state_init(const s4r_config* cfg, int64_t L, const float* qwin_prev,
                                 const void* coef_k, float* state, void* ws, size_t ws_bytes,
                                 hipStream_t stream);
s4r_status s4r_decode_step_windowed(const s4r_config* cfg, int64_t L, const void* q, float* state,
                                    const void* sink_k, const void* sink_v, const void* win_k,
                                    const void* win_v, const void* bases_k, const void* bases_v,
                                    void* coef_k, void* coef_v, const void* k_new, const void* v_new,
                                    float* out, int32_t* idx_out, float* scores_out, void* ws,
                                    size_t ws_bytes, hipStream_t stream);

/*
 * The fused decode step over a ragged batch (Section 3.2, each sequence at
 * its own length): lengths[b] (host memory, B entries, read before the call
 * returns) is sequence b's L, counted with the appended token when k_new /
 * v_new are given, each in [q_window, capacity].  Every other argument is as
 * for s4r_decode_step with L = max_b lengths[b]: coefficient rows past
 * lengths[b] are never read, the new token goes into row lengths[b] - 1 of
 * its sequence, the query sits at position n_sink + lengths[b] - 1,
 * idx_out is [B, m] and scores_out [B, max L] (row b written up to
 * lengths[b]).  Every sequence must select the same number of tokens
 * m = min(topk, L_b - window) + min(window, L_b) (true whenever every
 * L_b >= window + topk), else S4R_ERR_BAD_SHAPE; B <= 64, else
 * S4R_ERR_UNSUPPORTED.
 */
s4r_status s4r_decode_step_ragged(const s4r_config* cfg, const int64_t* lengths, const void* q,
                                  const float* qwin_prev, const void* sink_k, const void* sink_v,
                                  const void* win_k, const void* win_v, const void* bases_k,
                                  const void* bases_v, void* coef_k, void* coef_v,
                                  const void* k_new, const void* v_new, float* out,
                                  int32_t* idx_out, float* scores_out, void* ws, size_t ws_bytes,
                                  hipStream_t stream);

/*
 * Comparator (Appendix B.1, "full reconstruction"; not the method): the
 * cache is stored as coefficients like S^4R's, but every one of the L
 * non-sink tokens is reconstructed, K^ = C^K (B^K)^T and V^ = C^V (B^V)^T,
 * and attention runs over the sinks and all of them: out[b, h] =
 * softmax(RoPE(q_h) RoPE(K*_j)^T / sqrt(d_h)) V*_j, K* = [sink_k; K^],
 * j = h / G, query at position n_sink + L - 1.  The reconstructed rows stay
 * on chip (the MFMA kernel of s4r_decode_step over every token, no index
 * list).  Arguments as for s4r_decode_step; out [B, h_q, d_h] fp32.  bf16
 * storage, head_dim 64 or 128, G <= 8 and the fused kernel's ranks only
 * (otherwise S4R_ERR_UNSUPPORTED).
 */
s4r_status s4r_full_recon_decode(const s4r_config* cfg, int64_t L, const void* q, const void* sink_k,
                                 const void* sink_v, const void* bases_k, const void* bases_v,
                                 const void* coef_k, const void* coef_v, float* out, void* ws,
                                 size_t ws_bytes, hipStream_t stream);

/*
 * Query coefficients of several queries (Section 3.2.1, c^Q = s^Q B^K per
 * query group; Section 3.1 builds the initial query window C^Q this way from
 * the prompt's last queries): q_rows [B, n_rows, h_q, d_h] pre-RoPE queries in
 * the storage dtype, row i of every sequence projected like the query of a
 * decode step; qcoef_out [B, G, n_rows, R] fp32, the layout of qwin_prev when
 * n_rows = W_q - 1 (oldest first).  fp64 sums in the order the scoring kernel
 * uses, rounded once to fp32.  ws / ws_bytes: the decode workspace.
 * 1 <= n_rows <= 4096.
 */
s4r_status s4r_project_queries(const s4r_config* cfg, int64_t n_rows, const void* q_rows,
                               const void* bases_k, float* qcoef_out, void* ws, size_t ws_bytes,
                               hipStream_t stream);

/*
 * Basis construction of the prefill stage (Section 3.1.2, Eq. svd), per
 * sequence, key/value and basis group: the hybrid sample of the n_rows
 * non-sink rows (T' = max(1, floor(eta * n_rows)) rows: the most recent
 * round(0.7 T') as a contiguous block, the rest spaced uniformly over the
 * earlier positions, numpy's linspace then round-half-even), each sampled
 * row's group slice L2-normalised, optionally mean-centred (center = 1),
 * and the right singular vectors of the `rank` largest singular values
 * (rank_v for the values), largest first, written as bases_k / bases_v
 * [B, basis_groups, Dp / basis_groups, rank_s] in the storage dtype (columns
 * from rank to the rank stride rank_s are written as zeros).  Signs of
 * the singular vectors are arbitrary (the decode step depends on B B^T only).
 * s_k / s_v: [B, n_rows, Dp] raw pre-RoPE rows, bf16.  sample_idx_out
 * (optional, device, s4r_prefill_num_samples entries) receives the sample.
 * The Gram matrices are formed in fp64 by this library's kernels; their
 * symmetric eigenproblems run in rocSOLVER (fp64, divide and conquer) within
 * the caller's workspace of s4r_prefill_bases_workspace_size bytes; the first
 * call on a device (this one, or s4r_prefill_bases_workspace_size) creates
 * one rocBLAS handle, kept until the process ends (host threads calling on
 * one device are serialised around it).  Creating the handle is the one
 * place where the library may allocate device memory itself (rocBLAS's own
 * handle state; the solver's workspace is always the caller's).  The call
 * stays asynchronous: the solver's per-matrix convergence flag is consumed
 * on the device, where a matrix that did not converge writes quiet-NaN bases
 * for its (sequence, side, basis group), so the failure reaches the caller
 * through the output instead of passing silently.
 * bf16 storage, bases_shared = 0, (Dp / basis_groups) % 256 == 0 and at least
 * max(rank, rank_v) sampled rows (otherwise S4R_ERR_UNSUPPORTED /
 * S4R_ERR_BAD_SHAPE).
 */
int64_t s4r_prefill_num_samples(int64_t n_rows, double eta);
s4r_status s4r_prefill_bases_workspace_size(const s4r_config* cfg, int64_t n_rows, double eta,
                                            size_t* bytes);
s4r_status s4r_prefill_bases(const s4r_config* cfg, int64_t n_rows, const void* s_k, const void* s_v,
                             double eta, int32_t center, void* bases_k, void* bases_v,
                             int32_t* sample_idx_out, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Bulk projection of the prefill stage (Section 3.1, the coefficient
 * equation): C^K = S^K B^K and C^V = S^V B^V per basis group for the prompt's
 * non-sink rows, written into rows [0, n_rows) of the tiled coefficient caches
 * (other rows untouched).  s_k / s_v: [B, n_rows, Dp] raw pre-RoPE rows, row
 * t = non-sink token t, row-major, storage dtype; bases as in
 * s4r_score_latent.  Products of the bf16 inputs are exact, sums are fp32 on
 * the matrix cores, rounded once to bf16 (a coefficient can differ by one
 * bf16 ulp from the fp64-rounded value where the fp32 sum lies next to a
 * rounding boundary).  bf16 storage, rank 32..192 and equal key and value
 * ranks only (otherwise S4R_ERR_UNSUPPORTED).  ws / ws_bytes: the workspace
 * of s4r_decode_step (s4r_workspace_size); its first B * 2 * Dp * rank * 2
 * bytes hold the bases transposed while the call runs.  The bases themselves
 * come from a truncated SVD of sampled, normalised rows (Section 3.1), which
 * s4r_prefill_bases computes.
 */
s4r_status s4r_prefill_project(const s4r_config* cfg, int64_t n_rows, const void* s_k,
                               const void* s_v, const void* bases_k, const void* bases_v,
                               void* coef_k, void* coef_v, void* ws, size_t ws_bytes,
                               hipStream_t stream);

/*
 * Comparator: dense GQA decode attention over an uncompressed KV cache, the
 * "Full KV" baseline of the efficiency comparison (Section 4.2, Table
 * "efficiency"; the full-attention term of Appendix B.1).  Not part of the
 * S^4R step; it exists so the method and the full cache are measured on the
 * same GPU.  k_cache / v_cache: [B, capacity, Dp] bf16, row n of sequence b
 * holding token n (keys already rotated by RoPE at position n, as a plain KV
 * cache stores them); the N tokens 0..N-1 are attended, the query q
 * [B, h_q, d_h] (pre-RoPE) is rotated at position N - 1.
 * out[b, h] = softmax(RoPE(q_h) K_j^T / sqrt(d_h)) V_j with j = h / G, fp32.
 * Uses cfg's batch, head counts, head_dim, capacity, rope_theta and dtype only;
 * bf16, head_dim 128 and G <= 8 (otherwise S4R_ERR_UNSUPPORTED); the workspace
 * is the same as for s4r_decode_step.
 */
s4r_status s4r_dense_decode(const s4r_config* cfg, int64_t N, const void* q, const void* k_cache,
                            const void* v_cache, float* out, void* ws, size_t ws_bytes,
                            hipStream_t stream);

/*
 * Compressed cache update alone (Section 3.2.1): c^K = k_new B^K and
 * c^V = v_new B^V, rounded to the storage dtype (fp64 accumulation, then
 * fp32 and bf16 round-to-nearest-even), written into coefficient row `row`.
 */
s4r_status s4r_project_append(const s4r_config* cfg, int64_t row, const void* k_new,
                              const void* v_new, const void* bases_k, const void* bases_v,
                              void* coef_k, void* coef_v, hipStream_t stream);

/* Layout conversion of a coefficient cache: row-major [B, n_rows, R] <-> tiled
 * [B, capacity, R] (rows 0 .. n_rows-1; other rows of dst are left as they are).
 * The width is R = basis_groups * rank: convert a value cache of rank_v with a
 * configuration whose rank is rank_v. */
s4r_status s4r_pack_coef(const s4r_config* cfg, int64_t n_rows, const void* src_rowmajor,
                         void* dst_tiled, hipStream_t stream);
s4r_status s4r_unpack_coef(const s4r_config* cfg, int64_t n_rows, const void* src_tiled,
                           void* dst_rowmajor, hipStream_t stream);

/*
 * Kernel timing for measurement.  While enabled, s4r_decode_step records a
 * hipEvent pair around each of its kernels on the caller's stream, for up to
 * `max_steps` calls.  Kernels, in launch order (S4R_TIMED_KERNELS of them):
 *   0 cache update + query projection   1 latent-score stream over C^K
 *   2 relevance + histogram             3 top-k selection
 *   4 reconstruction + split attention  5 split combine
 * s4r_timing_read waits for the recorded events, writes the summed time of
 * each kernel (ms, array of S4R_TIMED_KERNELS) and the number of timed
 * steps, and disables timing.  Events are created in s4r_timing_enable only.
 */
#define S4R_TIMED_KERNELS 6
s4r_status s4r_timing_enable(int32_t max_steps);
s4r_status s4r_timing_read(double* total_ms, int64_t* steps);

/*
 * Read-bandwidth reference for roofline calibration (not part of the method):
 * reads `bytes` (a positive multiple of 16) from the device buffer `buf` once
 * with non-temporal 16-byte loads, each workgroup reading one contiguous range
 * of the buffer (the fastest read pattern measured on this GPU; grid-stride
 * patterns were slower).  `sink` (device, uint32,
 * s4r_read_bandwidth_sink_len() entries) receives one XOR of the words each
 * thread read; the XOR of all entries is the XOR of every 32-bit word of
 * the buffer.  buf must be 16-byte aligned.
 */
int64_t s4r_read_bandwidth_sink_len(void);
s4r_status s4r_read_bandwidth(const void* buf, int64_t bytes, uint32_t* sink, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* S4R_H */
