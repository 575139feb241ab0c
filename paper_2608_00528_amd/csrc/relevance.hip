// Section 3.2.2 softmax / window mean and the pooling and group-aggregation
// equations of Section 3.2.3 on gfx950: k_relevance turns the stream's exp
// values and statistics into A~ (fp32) and adds to the sequence's radix
// histogram; k_hist_scores builds it for caller-given scores.
#include "s4r_device.h"
#include "s4r_internal.h"
#include "select_key.h"

namespace s4r {

// ---------------------------------------------------------------------------
// K2: relevance A~ and its radix histogram
// ---------------------------------------------------------------------------
// grid (ceil(L / chunk), B), 256 threads; chunk = 1024 / 512 tokens for
// G <= 8 / 16.  The stream's exp values are stored token-major,
// e[b][x][c] for query column c = g * W_q + i (GWP = G * W_q rounded up to a
// multiple of 4, padding columns zero), with one reference per 16-token tile,
// tref[b][tile][c].  One memory latency: the scoring workgroups' statistics,
// the chunk's tile references and its exp values (plus the pooling halo) are
// all requested before any is used.  Then each wave folds query columns'
// statistics into the global (M, S), sums in fp64 (the same fixed order in
// every workgroup, so A~ is deterministic), and the per-tile factors
// exp(ref - M) / S; every exponential there takes its fp64 argument through
// exp_neg_accurate (fp64 range reduction, hardware exp2 of the fraction: about
// one fp32 ulp), far cheaper than an fp64 exp per scoring workgroup and
// column in every workgroup.  Per staged position the window mean
// over the W_q rows is formed once (fp32 products of values exact to about an
// ulp; the max-pooling that follows is exact), staged in LDS, and every thread
// pools outputs t, t + 256, ... (consecutive lanes read consecutive words: no
// bank conflicts) and sums the groups in fp64.
constexpr int kRelThreads = 256;
// scoring-workgroup statistics per lane that the relevance kernel folds itself
// (KSP, all requested together): 2 (up to 128 scoring workgroups), or 8 (up to
// 512) with one query column per wave: the paper's batch-1 setting at 120k
// has 469, whose separate fold launch cost 4.6 us, while eight per lane cost
// the 128-workgroup shapes 0.5 us.  Beyond that k_fold_stats folds them first.
constexpr int kRelStatPer = 2, kRelStatWide = 8;
template <int NQ>
constexpr int rel_stat_max() {
  return 64 * (NQ == 1 ? kRelStatWide : kRelStatPer);
}
constexpr int kRelMaxTiles = 1024 / kTileTok + 8;   // tiles touched by a chunk and its halo (h <= 32)

// tokens per workgroup: 1024 (G <= 8) or 512, halved (down to 256) while the
// grid would give fewer than four workgroups per CU.  Measured at 1024, 512
// and 256 tokens: about 1024 workgroups is best at batch 4 (512-token chunks,
// relevance 11.9 -> 10.5 us at 128k), batch 8 and batch 32 (1024-token
// chunks; 512 costs 2.7 and 1 us there).  The histogram copies keep the
// flush atomics of more workgroups from serialising.
constexpr int kRelMinWg = 1024;
int relevance_chunk(const Problem& P, int64_t L) {
  int c = P.G <= 8 ? 1024 : 512;
  while (c > 256 && (int64_t)P.B * ((L + c - 1) / c) < kRelMinWg) c >>= 1;
  return c;
}

// Pooling (kappa = 2H + 1, stride 1, same length) and aggregation over the G
// groups for outputs t, t + 256, ... of a chunk.  With H known at compile time
// every window value is requested from LDS before any is combined, so the
// reads overlap; H < 0 is the generic (slower) path for wide kernels.
template <int H, int TPT, int GMAX>
__device__ __forceinline__ void pool_aggregate(const float* __restrict__ vs, int span, int t, int G, int kappa,
                                               int pool_mode, int agg, float (&af)[TPT]) {
  const int h = (H >= 0) ? H : kappa / 2;
#pragma unroll
  for (int j = 0; j < TPT; ++j) {
    const int o = t + j * kRelThreads;                     // window of output o: vs[g][o .. o + 2h]
    double acc = (agg == S4R_AGG_MEAN) ? 0.0 : -INFINITY;
    if constexpr (H >= 0) {
      float w[GMAX][2 * (H > 0 ? H : 0) + 1];
#pragma unroll
      for (int g = 0; g < GMAX; ++g)
#pragma unroll
        for (int d = 0; d <= 2 * H; ++d) w[g][d] = vs[min(g, G - 1) * span + o + d];   // unguarded: overlapped
#pragma unroll
      for (int g = 0; g < GMAX; ++g) {
        if (g < G) {
          float a;
          if (pool_mode == S4R_POOL_MAX) {
            a = w[g][0];
#pragma unroll
            for (int d = 1; d <= 2 * H; ++d) a = fmaxf(a, w[g][d]);
          } else {
            double sa = 0.0;
#pragma unroll
            for (int d = 0; d <= 2 * H; ++d) sa += (double)w[g][d];
            a = (float)(sa / kappa);
          }
          acc = (agg == S4R_AGG_MEAN) ? acc + (double)a : fmax(acc, (double)a);
        }
      }
    } else {
      for (int g = 0; g < G; ++g) {
        const float* v = vs + g * span + o;
        float a = v[0];
        double sa = (double)v[0];
        for (int d = 1; d <= 2 * h; ++d) {
          a = fmaxf(a, v[d]);
          sa += (double)v[d];
        }
        if (pool_mode != S4R_POOL_MAX) a = (float)(sa / kappa);
        acc = (agg == S4R_AGG_MEAN) ? acc + (double)a : fmax(acc, (double)a);
      }
    }
    af[j] = (float)((agg == S4R_AGG_MEAN) ? acc / G : acc);
  }
}

// WIN (windowed step, query window of wrows rows): the stream scored only
// the newest query row (its G columns, Wq = 1 here); the softmax of each
// older row over its own keys comes from the window state
// [B][wrows][G][cap], row slot L_r mod wrows for the row that was newest at
// length L_r (it covers keys < L_r).  This kernel adds the newest row's
// softmax to the older rows' for the window mean and stores it in its slot.
// With a running sum (rsum, longer windows) the older rows' sum per position
// is kept in fp64 as well, in two buffers [2][B][G][cap] by the parity of L:
// the step reads buffer L & 1 and writes buffer (L + 1) & 1 = that sum plus
// the newest row minus the row leaving the window (the one newest at
// L - wrows + 1, masked at its key limit), for the positions it owns.
template <int NQ, int TPT, bool WQ1, bool WIN, int KSP>
__global__ __launch_bounds__(kRelThreads) void k_relevance(
    const float* __restrict__ e, const float* __restrict__ tref, const double* __restrict__ wg_stats,
    const double* __restrict__ col_stats, float* __restrict__ atilde, uint32_t* __restrict__ hist, float* __restrict__ scores_out,
    int64_t cap, int L, int n_hist, int G, int Wq, int kappa, int pool_mode, int agg, int ntiles_cap, int nwg,
    Lens lens, int key_shift, float* __restrict__ state, int wrows, double* __restrict__ rsum, int hist_nc) {
  constexpr int GWP = 4 * NQ;
  constexpr int CHUNK = kRelThreads * TPT;
  constexpr int SPAN_MAX = CHUNK + 64;
  constexpr int PPT = (SPAN_MAX + kRelThreads - 1) / kRelThreads;   // staged positions per thread
  const int b = blockIdx.y;
  const int score_stride = L;                      // scores_out rows are [B, L] with the call's (largest) L
  {                                                // this sequence's length (ragged batch: n_hist shifts with it)
    const int Lb = (int)len_of(lens, b, L);
    n_hist += Lb - L;
    L = Lb;
  }
  if ((int)blockIdx.x * kRelThreads * TPT >= L) return;   // past this sequence's end
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int GW = G * Wq;
  const int h = kappa / 2;
  const int t0 = blockIdx.x * CHUNK;
  const int x0 = t0 - h;                                   // first staged position
  const int span = CHUNK + 2 * h;
  const int tile_lo = max(x0, 0) / kTileTok;
  const int tile_hi = (min(t0 + CHUNK + h, L) - 1) / kTileTok;
  const int ntl = tile_hi - tile_lo + 1;                   // <= kRelMaxTiles

  __shared__ uint32_t hl[kHistBins];
  __shared__ double sM[GWP], sInvS[GWP];
  __shared__ float fac[kRelMaxTiles][GWP];                 // exp(ref - M) / S per tile and column
  extern __shared__ float vs[];                            // [G][span]: window mean at x0 + i

  // ---- all global reads of this workgroup, issued before any is used ----------
  // statistics: wave w folds columns w, w + 4, ...; two batches of 64 lanes in flight
  // (or, with many scoring workgroups, the global statistics k_fold_stats formed)
  double2 st[NQ][KSP];
  const double2* stats = reinterpret_cast<const double2*>(wg_stats) + (int64_t)b * GW * nwg;
  double2 cs = make_double2(0.0, 0.0);
  if (col_stats) {
    cs = reinterpret_cast<const double2*>(col_stats)[(int64_t)b * GW + min(t, GW - 1)];
  } else {
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int c = min(wave + 4 * q, GW - 1);
#pragma unroll
      for (int k = 0; k < KSP; ++k) st[q][k] = stats[(int64_t)c * nwg + min(lane + 64 * k, nwg - 1)];
    }
  }
  // tile references: thread t loads tile tile_lo + t (all columns)
  float4 rf[NQ];
  {
    const float4* tp = reinterpret_cast<const float4*>(tref + ((int64_t)b * ntiles_cap + tile_lo + min(t, ntl - 1)) * GWP);
#pragma unroll
    for (int q = 0; q < NQ; ++q) rf[q] = tp[q];
  }
  // exp values of the staged positions (clamped into [0, L); masked later)
  float4 ev[PPT][NQ];
#pragma unroll
  for (int k = 0; k < PPT; ++k) {
    const int x = min(max(x0 + t + k * kRelThreads, 0), L - 1);
    const float4* ep = reinterpret_cast<const float4*>(e + ((int64_t)b * cap + x) * GWP);
#pragma unroll
    for (int q = 0; q < NQ; ++q) ev[k][q] = ep[q];
  }
  for (int i = t; i < kHistBins; i += kRelThreads) hl[i] = 0;

  // ---- global (M, S) of each query column ---------------------------------------------
  if (col_stats) {
    if (t < GW) {
      sM[t] = cs.x;
      sInvS[t] = cs.y;
    }
  }
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int c = wave + 4 * q;
    if (!col_stats && c < GW) {                            // wave-uniform
      const double* srow = wg_stats + ((int64_t)b * GW + c) * nwg * 2;
      double M = -INFINITY, S = 0.0;
      for (int base = 0; base < nwg; base += 64 * KSP) {
        double2 s2[KSP];
#pragma unroll
        for (int k = 0; k < KSP; ++k) {
          if (base == 0) {
            s2[k] = st[q][k];
          } else {                                         // more than 128 scoring workgroups
            const int w = min(base + lane + 64 * k, nwg - 1);
            s2[k] = make_double2(srow[2 * w], srow[2 * w + 1]);
          }
        }
        double m = -INFINITY;
#pragma unroll
        for (int k = 0; k < KSP; ++k)
          if (base + lane + 64 * k < nwg) m = fmax(m, s2[k].x);
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) m = fmax(m, shfl_xor_d(m, o));
        double s = 0.0;
#pragma unroll
        for (int k = 0; k < KSP; ++k)
          if (base + lane + 64 * k < nwg && s2[k].x != -INFINITY) s += s2[k].y * (double)exp_neg_accurate(s2[k].x - m);
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) s += shfl_xor_d(s, o);
        if (m != -INFINITY) {
          const double Mn = fmax(M, m);
          S = ((M == -INFINITY) ? 0.0 : S * (double)exp_neg_accurate(M - Mn)) + s * (double)exp_neg_accurate(m - Mn);
          M = Mn;
        }
      }
      if (lane == 0) {
        sM[c] = M;
        sInvS[c] = 1.0 / S;
      }
    }
  }
  __syncthreads();
  // ---- per-tile factors ---------------------------------------------------------------
  if (t < ntl) {
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const float r4[4] = {rf[q].x, rf[q].y, rf[q].z, rf[q].w};
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int c = 4 * q + u;
        fac[t][c] = (c < GW && r4[u] != -INFINITY)
                        ? (float)((double)exp_neg_accurate((double)r4[u] - sM[c]) * sInvS[c]) : 0.f;
      }
    }
  }
  __syncthreads();
  // ---- window mean over the W_q rows of every staged position -------------------------
  const float pad = (pool_mode == S4R_POOL_MAX) ? -INFINITY : 0.f;
  const float inv_wq = 1.f / (float)(WIN ? wrows : Wq);
#pragma unroll
  for (int k = 0; k < PPT; ++k) {
    const int i = t + k * kRelThreads;
    if (i < span) {
      const int x = x0 + i;
      const bool in = x >= 0 && x < L;
      const float* fr = fac[min(max(x, 0), L - 1) / kTileTok - tile_lo];
      float ex[GWP];
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        ex[4 * q] = ev[k][q].x;
        ex[4 * q + 1] = ev[k][q].y;
        ex[4 * q + 2] = ev[k][q].z;
        ex[4 * q + 3] = ev[k][q].w;
      }
      if constexpr (WIN) {
        // the newest row's softmax: into its slot (own chunk) and into LDS;
        // the older rows are added from the running sum, else below
        float* sb = state + (int64_t)b * wrows * G * cap;
        const int slot_new = L % wrows;
        const bool own = in && x >= t0 && x < t0 + CHUNK;
        if (rsum) {
          const double* scur = rsum + ((int64_t)(L & 1) * gridDim.y + b) * G * cap;
          double* snext = rsum + ((int64_t)((L + 1) & 1) * gridDim.y + b) * G * cap;
          const int Lo = L - wrows + 1;                        // the leaving row was newest at Lo
          const float* sold = sb + (int64_t)((Lo % wrows + wrows) % wrows) * G * cap;
          const int xc = min(max(x, 0), (int)cap - 1);
#pragma unroll
          for (int c = 0; c < GWP; ++c) {
            if (c < G) {
              const float pn = in ? ex[c] * fr[c] : 0.f;
              const double so = scur[(int64_t)c * cap + xc];
              const float po = sold[(int64_t)c * cap + xc];
              if (own) {
                sb[((int64_t)slot_new * G + c) * cap + x] = pn;
                snext[(int64_t)c * cap + x] = (so + (double)pn) - (x < Lo ? (double)po : 0.0);
              }
              vs[c * span + i] = in ? (float)((so + (double)pn) * (double)inv_wq) : pad;
            }
          }
        } else {
#pragma unroll
          for (int c = 0; c < GWP; ++c) {
            if (c < G) {
              const float pn = in ? ex[c] * fr[c] : 0.f;
              if (own) sb[((int64_t)slot_new * G + c) * cap + x] = pn;
              vs[c * span + i] = pn;
            }
          }
        }
      } else if constexpr (WQ1) {
#pragma unroll
        for (int c = 0; c < GWP; ++c)
          if (c < G) vs[c * span + i] = in ? ex[c] * fr[c] : pad;
      } else {
        for (int g = 0; g < G; ++g) {
          float sum = 0.f;
#pragma unroll
          for (int c = 0; c < GWP; ++c)
            if (c >= g * Wq && c < (g + 1) * Wq) sum += ex[c] * fr[c];
          vs[g * span + i] = in ? sum * inv_wq : pad;
        }
      }
    }
  }
  __syncthreads();
  if (WIN && !rsum) {
    // ---- older rows of the window: row of age a = 1 .. wrows - 1 covers keys
    // < L - a, in slot (L - a) mod wrows.  Unit u = four consecutive positions
    // 4 (u0 + u) .. + 3 (16-byte loads, unconditional at clamped positions,
    // masked after) of group g; eight rows in flight per batch
    const float* sb = state + (int64_t)b * wrows * G * cap;
    const int u0 = (x0 >= 0 ? x0 : x0 - 3) / 4;         // floor(x0 / 4)
    const int nu = (x0 + span + 3) / 4 - u0;             // units covering the staged positions
    for (int w = t; w < G * nu; w += kRelThreads) {
      const int g = w / nu, xu = 4 * (u0 + w % nu);      // first position of the unit
      const int xl = min(max(xu, 0), (int)(cap - 4));
      float4 sum = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int a0 = 1; a0 < wrows; a0 += 8) {
        float4 o[8];
#pragma unroll
        for (int v = 0; v < 8; ++v) {
          const int a = min(a0 + v, wrows - 1);
          const int slot = ((L - a) % wrows + wrows) % wrows;   // L - a < 0 early on: masked below
          o[v] = *reinterpret_cast<const float4*>(sb + ((int64_t)slot * G + g) * cap + xl);
        }
#pragma unroll
        for (int v = 0; v < 8; ++v) {
          const int lim = L - (a0 + v);                  // keys of this row
          if (a0 + v < wrows) {
            if (xl + 0 < lim) sum.x += o[v].x;
            if (xl + 1 < lim) sum.y += o[v].y;
            if (xl + 2 < lim) sum.z += o[v].z;
            if (xl + 3 < lim) sum.w += o[v].w;
          }
        }
      }
      const float sv[4] = {sum.x, sum.y, sum.z, sum.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int x = xu + j, i = x - x0;
        if (i >= 0 && i < span) {
          const bool in = x >= 0 && x < L && xl == xu;
          vs[g * span + i] = in ? (vs[g * span + i] + sv[j]) * inv_wq : pad;
        }
      }
    }
    __syncthreads();                                       // (wave-uniform: rsum is a kernel argument)
  }
  // ---- pooling (kappa, stride 1, same length) and aggregation over G -------------------
  float af[TPT];
  switch (h) {
    case 0: pool_aggregate<0, TPT, GWP>(vs, span, t, G, kappa, pool_mode, agg, af); break;
    case 1: pool_aggregate<1, TPT, GWP>(vs, span, t, G, kappa, pool_mode, agg, af); break;
    case 2: pool_aggregate<2, TPT, GWP>(vs, span, t, G, kappa, pool_mode, agg, af); break;
    case 3: pool_aggregate<3, TPT, GWP>(vs, span, t, G, kappa, pool_mode, agg, af); break;
    case 4: pool_aggregate<4, TPT, GWP>(vs, span, t, G, kappa, pool_mode, agg, af); break;
    default: pool_aggregate<-1, TPT, GWP>(vs, span, t, G, kappa, pool_mode, agg, af); break;
  }
#pragma unroll
  for (int j = 0; j < TPT; ++j) {
    const int x = t0 + t + j * kRelThreads;
    if (x < L) {
      atilde[(int64_t)b * cap + x] = af[j];
      if (scores_out) scores_out[(int64_t)b * score_stride + x] = af[j];
    }
    if (x < n_hist) atomicAdd(&hl[selection_key_shift(af[j], key_shift) >> kHistShift], 1u);
  }
  __syncthreads();
  // this workgroup's histogram into the sequence's (zeroed by the query
  // projection earlier in the step): one global atomic per non-empty bin
  uint32_t* hs = hist + (int64_t)b * kHistStride + (blockIdx.x & (hist_nc - 1)) * kHistBins;
  for (int i = t; i < kHistBins; i += kRelThreads) {
    const uint32_t c = hl[i];
    if (c) atomicAdd(&hs[i], c);
  }
}

// K2 for more than 16 query columns (G * W_q up to 128, the paper's tied
// W_q = W = 32): grid (ceil(L / 256), B), 256 threads, 256 tokens per
// workgroup.  The global (M, 1 / S) of every column comes from k_fold_stats;
// the per-tile factors exp(ref - M) / S of the chunk's tiles (and halo) go to
// LDS; thread (position, group) forms the window mean of its group's W_q
// columns from the exp values (contiguous per position) with an fp64 sum of
// the fp32 products, then pooling and group aggregation run as in k_relevance.
constexpr int kWideChunk = kRelThreads;
constexpr int kWideMaxTiles = (kWideChunk + 64) / kTileTok + 2;

template <int GMAX>
__global__ __launch_bounds__(kRelThreads) void k_relevance_wide(
    const float* __restrict__ e, const float* __restrict__ tref, const double* __restrict__ col_stats,
    float* __restrict__ atilde, uint32_t* __restrict__ hist, float* __restrict__ scores_out, int64_t cap, int L,
    int n_hist, int G, int Wq, int gwp, int kappa, int pool_mode, int agg, int ntiles_cap, Lens lens, int key_shift,
    int hist_nc) {
  const int b = blockIdx.y;
  const int score_stride = L;
  {
    const int Lb = (int)len_of(lens, b, L);
    n_hist += Lb - L;
    L = Lb;
  }
  if ((int)blockIdx.x * kWideChunk >= L) return;
  const int t = threadIdx.x;
  const int GW = G * Wq;
  const int h = kappa / 2;
  const int t0 = blockIdx.x * kWideChunk;
  const int x0 = t0 - h;
  const int span = kWideChunk + 2 * h;
  const int tile_lo = max(x0, 0) / kTileTok;
  const int tile_hi = (min(t0 + kWideChunk + h, L) - 1) / kTileTok;
  const int ntl = tile_hi - tile_lo + 1;                   // <= kWideMaxTiles

  __shared__ uint32_t hl[kHistBins];
  __shared__ __align__(16) float fac[kWideMaxTiles * kMaxGW];   // [tile][column]
  extern __shared__ float vs[];                            // [G][span]
  for (int i = t; i < kHistBins; i += kRelThreads) hl[i] = 0;
  const double2* cs = reinterpret_cast<const double2*>(col_stats) + (int64_t)b * GW;
  for (int i = t; i < ntl * GW; i += kRelThreads) {
    const int tl = i / GW, c = i % GW;
    const float r = tref[((int64_t)b * ntiles_cap + tile_lo + tl) * gwp + c];
    const double2 st = cs[c];
    fac[tl * GW + c] = (r != -INFINITY) ? (float)((double)exp_neg_accurate((double)r - st.x) * st.y) : 0.f;
  }
  __syncthreads();
  // window mean over the W_q rows of group g at every staged position
  const float pad = (pool_mode == S4R_POOL_MAX) ? -INFINITY : 0.f;
  const double inv_wq = 1.0 / (double)Wq;
  for (int i = t; i < span * G; i += kRelThreads) {
    const int xi = i / G, g = i % G;
    const int x = x0 + xi;
    float v = pad;
    if (x >= 0 && x < L) {
      const float* ep = e + ((int64_t)b * cap + x) * gwp + g * Wq;
      const float* fr = fac + (x / kTileTok - tile_lo) * GW + g * Wq;
      double sum = 0.0;                            // W_q products summed in fp64
      if ((Wq & 3) == 0) {                         // 16-byte loads (rows of gwp, a multiple of 16, floats)
        const float4* e4 = reinterpret_cast<const float4*>(ep);
        const float4* f4 = reinterpret_cast<const float4*>(fr);
        for (int c = 0; c < Wq / 4; ++c) {
          const float4 a = e4[c], f = f4[c];
          sum += (double)a.x * (double)f.x + (double)a.y * (double)f.y + (double)a.z * (double)f.z +
                 (double)a.w * (double)f.w;
        }
      } else {
        for (int c = 0; c < Wq; ++c) sum += (double)ep[c] * (double)fr[c];
      }
      v = (float)(sum * inv_wq);
    }
    vs[g * span + xi] = v;
  }
  __syncthreads();
  float af[1];
  switch (h) {
    case 0: pool_aggregate<0, 1, GMAX>(vs, span, t, G, kappa, pool_mode, agg, af); break;
    case 1: pool_aggregate<1, 1, GMAX>(vs, span, t, G, kappa, pool_mode, agg, af); break;
    case 2: pool_aggregate<2, 1, GMAX>(vs, span, t, G, kappa, pool_mode, agg, af); break;
    case 3: pool_aggregate<3, 1, GMAX>(vs, span, t, G, kappa, pool_mode, agg, af); break;
    case 4: pool_aggregate<4, 1, GMAX>(vs, span, t, G, kappa, pool_mode, agg, af); break;
    default: pool_aggregate<-1, 1, GMAX>(vs, span, t, G, kappa, pool_mode, agg, af); break;
  }
  const int x = t0 + t;
  if (x < L) {
    atilde[(int64_t)b * cap + x] = af[0];
    if (scores_out) scores_out[(int64_t)b * score_stride + x] = af[0];
  }
  if (x < n_hist) atomicAdd(&hl[selection_key_shift(af[0], key_shift) >> kHistShift], 1u);
  __syncthreads();
  uint32_t* hs = hist + (int64_t)b * kHistStride + (blockIdx.x & (hist_nc - 1)) * kHistBins;
  for (int i = t; i < kHistBins; i += kRelThreads) {
    const uint32_t c = hl[i];
    if (c) atomicAdd(&hs[i], c);
  }
}

// histogram of caller-provided scores (standalone selection), into a
// histogram zeroed by k_zero_hist
__global__ __launch_bounds__(256) void k_zero_hist(uint32_t* __restrict__ hist, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) hist[i] = 0u;
}

__global__ __launch_bounds__(256) void k_hist_scores(const float* __restrict__ scores, uint32_t* __restrict__ hist,
                                                     int L, int n_hist, int hist_nc) {
  const int b = blockIdx.y;
  __shared__ uint32_t hl[kHistBins];
  for (int i = threadIdx.x; i < kHistBins; i += blockDim.x) hl[i] = 0;
  __syncthreads();
  const int t0 = blockIdx.x * kHistChunk;
  for (int i = threadIdx.x; i < kHistChunk; i += blockDim.x) {
    const int x = t0 + i;
    if (x < n_hist) atomicAdd(&hl[selection_key(scores[(int64_t)b * L + x]) >> kHistShift], 1u);
  }
  __syncthreads();
  uint32_t* hs = hist + (int64_t)b * kHistStride + (blockIdx.x & (hist_nc - 1)) * kHistBins;
  for (int i = threadIdx.x; i < kHistBins; i += blockDim.x) {
    const uint32_t c = hl[i];
    if (c) atomicAdd(&hs[i], c);
  }
}

// Global (max, 1 / sum) of every query column's softmax over the length,
// folded once from the scoring workgroups' (max, sum) pairs when there are
// more than the relevance kernel folds itself (rel_stat_max): grid (GW,
// B), thread t folds pairs t, t + 256, ... in order, then a fixed-order tree
// across the threads (deterministic).
__global__ __launch_bounds__(256) void k_fold_stats(const double* __restrict__ wg_stats, double* __restrict__ col_stats,
                                                    int GW, int nwg) {
  const int c = blockIdx.x, b = blockIdx.y, t = threadIdx.x;
  const double2* row = reinterpret_cast<const double2*>(wg_stats) + ((int64_t)b * GW + c) * nwg;
  __shared__ double sm[256], ss[256];
  auto merge = [](double& M, double& S, double m, double s) {
    if (m == -INFINITY) return;
    const double Mn = fmax(M, m);
    S = ((M == -INFINITY) ? 0.0 : S * (double)exp_neg_accurate(M - Mn)) + s * (double)exp_neg_accurate(m - Mn);
    M = Mn;
  };
  double M = -INFINITY, S = 0.0;
  for (int w0 = 0; w0 < nwg; w0 += 4 * 256) {
    double2 v[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = row[min(w0 + k * 256 + t, nwg - 1)];
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (w0 + k * 256 + t < nwg) merge(M, S, v[k].x, v[k].y);
  }
  sm[t] = M;
  ss[t] = S;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (t < o) {
      double M2 = sm[t], S2 = ss[t];
      merge(M2, S2, sm[t + o], ss[t + o]);
      sm[t] = M2;
      ss[t] = S2;
    }
    __syncthreads();
  }
  if (t == 0) reinterpret_cast<double2*>(col_stats)[(int64_t)b * GW + c] = make_double2(sm[0], 1.0 / ss[0]);
}

template <int NQ, int TPT>
static void launch_rel_t(const Problem& P, const Workspace& ws, int64_t L, float* scores_out, hipStream_t st) {
  const int n_hist = (int)std::max<int64_t>(L - P.W, 0);
  constexpr int chunk = kRelThreads * TPT;
  const size_t lds = (size_t)P.G * (chunk + 2 * (P.kappa / 2)) * sizeof(float);
  dim3 grid((unsigned)((L + chunk - 1) / chunk), P.B);
  const int nwg = score_workgroups(P, L);
  const bool fold = nwg > rel_stat_max<NQ>();
  constexpr int KW = NQ == 1 ? kRelStatWide : kRelStatPer;   // (only one column per wave folds 512)
  auto kern = nwg > 64 * kRelStatPer && !fold
                  ? (P.Wq == 1 ? k_relevance<NQ, TPT, true, false, KW> : k_relevance<NQ, TPT, false, false, KW>)
                  : (P.Wq == 1 ? k_relevance<NQ, TPT, true, false, kRelStatPer>
                               : k_relevance<NQ, TPT, false, false, kRelStatPer>);
  if (fold) hipLaunchKernelGGL(k_fold_stats, dim3(P.GW, P.B), dim3(256), 0, st, ws.wg_stats, ws.col_stats, P.GW, nwg);
  hipLaunchKernelGGL(kern, grid, dim3(kRelThreads), lds, st, ws.e, ws.run_m, ws.wg_stats,
                     fold ? ws.col_stats : nullptr, ws.atilde, ws.hist, scores_out, P.cap, (int)L, n_hist, P.G, P.Wq, P.kappa, P.pool_mode, P.agg,
                     (int)(P.cap / kTileTok), nwg, P.lens, fused_key_shift(P, L), nullptr, 1, nullptr,
                     hist_copies(grid.x));
}

template <int NQ>
static void launch_rel_nq(const Problem& P, const Workspace& ws, int64_t L, float* scores_out, hipStream_t st) {
  switch (relevance_chunk(P, L)) {
    case 1024: launch_rel_t<NQ, 4>(P, ws, L, scores_out, st); break;
    case 512: launch_rel_t<NQ, 2>(P, ws, L, scores_out, st); break;
    default: launch_rel_t<NQ, 1>(P, ws, L, scores_out, st); break;
  }
}

// more than 16 query columns: the statistics are always folded first
static void launch_rel_wide(const Problem& P, const Workspace& ws, int64_t L, float* scores_out, hipStream_t st) {
  const int n_hist = (int)std::max<int64_t>(L - P.W, 0);
  const int nwg = score_workgroups(P, L);
  hipLaunchKernelGGL(k_fold_stats, dim3(P.GW, P.B), dim3(256), 0, st, ws.wg_stats, ws.col_stats, P.GW, nwg);
  const size_t lds = (size_t)P.G * (kWideChunk + 2 * (P.kappa / 2)) * sizeof(float);
  dim3 grid((unsigned)((L + kWideChunk - 1) / kWideChunk), P.B);
  auto kern = P.G <= 4 ? k_relevance_wide<4> : (P.G <= 8 ? k_relevance_wide<8> : k_relevance_wide<16>);
  hipLaunchKernelGGL(kern, grid, dim3(kRelThreads), lds, st, ws.e, ws.run_m, ws.col_stats, ws.atilde, ws.hist,
                     scores_out, P.cap, (int)L, n_hist, P.G, P.Wq, gw_padded(P), P.kappa, P.pool_mode, P.agg,
                     (int)(P.cap / kTileTok), P.lens, fused_key_shift(P, L), hist_copies(grid.x));
}

hipError_t launch_relevance(const Problem& P, const Workspace& ws, int64_t L, float* scores_out, hipStream_t st) {
  if (P.GW > kColBlk) {
    launch_rel_wide(P, ws, L, scores_out, st);
    return hipGetLastError();
  }
  switch (gw_padded(P) / 4) {
    case 1: launch_rel_nq<1>(P, ws, L, scores_out, st); break;
    case 2: launch_rel_nq<2>(P, ws, L, scores_out, st); break;
    case 3: launch_rel_nq<3>(P, ws, L, scores_out, st); break;
    default: launch_rel_nq<4>(P, ws, L, scores_out, st); break;
  }
  return hipGetLastError();
}

template <int NQ, int TPT>
static void launch_rel_win_t(const Problem& P1, const Workspace& ws, int64_t L, float* scores_out, float* state,
                             int wrows, hipStream_t st) {
  const int n_hist = (int)std::max<int64_t>(L - P1.W, 0);
  constexpr int chunk = kRelThreads * TPT;
  const size_t lds = (size_t)P1.G * (chunk + 2 * (P1.kappa / 2)) * sizeof(float);
  dim3 grid((unsigned)((L + chunk - 1) / chunk), P1.B);
  const int nwg = score_workgroups(P1, L);
  const bool fold = nwg > rel_stat_max<NQ>();
  if (fold) hipLaunchKernelGGL(k_fold_stats, dim3(P1.GW, P1.B), dim3(256), 0, st, ws.wg_stats, ws.col_stats, P1.GW, nwg);
  constexpr int KW = NQ == 1 ? kRelStatWide : kRelStatPer;
  auto kern = nwg > 64 * kRelStatPer && !fold ? k_relevance<NQ, TPT, true, true, KW>
                                              : k_relevance<NQ, TPT, true, true, kRelStatPer>;
  hipLaunchKernelGGL(kern, grid, dim3(kRelThreads), lds, st, ws.e, ws.run_m, ws.wg_stats,
                     fold ? ws.col_stats : nullptr, ws.atilde, ws.hist, scores_out, P1.cap, (int)L, n_hist, P1.G, 1,
                     P1.kappa, P1.pool_mode, P1.agg, (int)(P1.cap / kTileTok), nwg, P1.lens, fused_key_shift(P1, L),
                     state, wrows, window_rsum(P1, state, wrows), hist_copies(grid.x));
}

int relevance_hist_copies(const Problem& P, int64_t L, int wrows) {
  const int chunk = (wrows < 2 && P.GW > kColBlk) ? kWideChunk : relevance_chunk(P, L);
  return hist_copies((L + chunk - 1) / chunk);
}

template <int NQ>
static void launch_rel_win_nq(const Problem& P1, const Workspace& ws, int64_t L, float* scores_out, float* state,
                              int wrows, hipStream_t st) {
  switch (relevance_chunk(P1, L)) {
    case 1024: launch_rel_win_t<NQ, 4>(P1, ws, L, scores_out, state, wrows, st); break;
    case 512: launch_rel_win_t<NQ, 2>(P1, ws, L, scores_out, state, wrows, st); break;
    default: launch_rel_win_t<NQ, 1>(P1, ws, L, scores_out, state, wrows, st); break;
  }
}

hipError_t launch_relevance_windowed(const Problem& P1, const Workspace& ws, int64_t L, float* scores_out,
                                     float* state, int wrows, hipStream_t st) {
  switch (gw_padded(P1) / 4) {
    case 1: launch_rel_win_nq<1>(P1, ws, L, scores_out, state, wrows, st); break;
    case 2: launch_rel_win_nq<2>(P1, ws, L, scores_out, state, wrows, st); break;
    case 3: launch_rel_win_nq<3>(P1, ws, L, scores_out, state, wrows, st); break;
    default: launch_rel_win_nq<4>(P1, ws, L, scores_out, state, wrows, st); break;
  }
  return hipGetLastError();
}

// window state of the W_q - 1 older rows from a stream over them (P0: those
// rows as the query window, scored to length L - 1): row r < wrows - 1 covers
// keys < L_r = L - (wrows - 1 - r) and goes to slot L_r mod wrows.  grid
// (ceil(cap / 256), B); the softmax probability of (row, group, key) is its
// exp value times exp(ref - M) / S of its tile and column (fp64 argument, as
// in the relevance kernel).  With a running sum, buffer L & 1 gets the older
// rows' fp64 sum (oldest row first; 0 where no row covers the key) and buffer
// (L + 1) & 1 zeros, over the whole capacity.
__global__ __launch_bounds__(256) void k_window_store(const float* __restrict__ e, const float* __restrict__ tref,
                                                      const double* __restrict__ col_stats, float* __restrict__ state,
                                                      double* __restrict__ rsum, int64_t cap, int L, int G, int wrows,
                                                      int gwp, int ntiles_cap) {
  const int b = blockIdx.y, x = blockIdx.x * 256 + threadIdx.x;
  const int w0 = wrows - 1;                       // rows in the stream, column c = g * w0 + r
  if (x >= cap) return;
  for (int g = 0; g < G; ++g) {
    double sum = 0.0;
    for (int r = 0; r < w0; ++r) {
      const int Lr = L - (w0 - r);
      if (x >= Lr) continue;
      const int c = g * w0 + r;
      const double2 cs = reinterpret_cast<const double2*>(col_stats)[(int64_t)b * G * w0 + c];
      const float ref = tref[((int64_t)b * ntiles_cap + x / kTileTok) * gwp + c];
      const float fac = (ref != -INFINITY) ? (float)((double)exp_neg_accurate((double)ref - cs.x) * cs.y) : 0.f;
      const float p = e[((int64_t)b * cap + x) * gwp + c] * fac;
      state[(((int64_t)b * wrows + Lr % wrows) * G + g) * cap + x] = p;
      sum += (double)p;
    }
    if (rsum) {
      rsum[(((int64_t)(L & 1) * gridDim.y + b) * G + g) * cap + x] = sum;
      rsum[(((int64_t)((L + 1) & 1) * gridDim.y + b) * G + g) * cap + x] = 0.0;
    }
  }
}

hipError_t launch_window_store(const Problem& P0, const Workspace& ws, int64_t L, float* state, int wrows,
                               hipStream_t st) {
  const int nwg = score_workgroups(P0, L - 1);
  hipLaunchKernelGGL(k_fold_stats, dim3(P0.GW, P0.B), dim3(256), 0, st, ws.wg_stats, ws.col_stats, P0.GW, nwg);
  hipLaunchKernelGGL(k_window_store, dim3((unsigned)((P0.cap + 255) / 256), P0.B), dim3(256), 0, st, ws.e,
                     ws.run_m, ws.col_stats, state, window_rsum(P0, state, wrows), P0.cap, (int)L, P0.G, wrows,
                     gw_padded(P0), (int)(P0.cap / kTileTok));
  return hipGetLastError();
}

hipError_t launch_hist_only(const Problem& P, const Workspace& ws, int64_t L, const float* scores, hipStream_t st) {
  const int n_hist = (int)std::max<int64_t>(L - P.W, 0);
  const int ng = std::max(1, (n_hist + kHistChunk - 1) / kHistChunk);
  hipLaunchKernelGGL(k_zero_hist, dim3((P.B * kHistStride + 255) / 256), dim3(256), 0, st, ws.hist,
                     P.B * kHistStride);
  hipLaunchKernelGGL(k_hist_scores, dim3(ng, P.B), dim3(256), 0, st, scores, ws.hist, (int)L, n_hist,
                     hist_copies(ng));
  return hipGetLastError();
}

}  // namespace s4r
