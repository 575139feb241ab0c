// Section 3.2.2 softmax / window mean and the pooling and group-aggregation
// equations of Section 3.2.3 on gfx950: k_relevance turns the stream's exp
// values and statistics into A~ (fp32) and adds to the sequence's radix
// histogram; k_hist_scores builds it for caller-given scores.
#include "s4r_device.h"
#include "s4r_internal.h"

namespace s4r {

// ---------------------------------------------------------------------------
// K2: relevance A~ and its radix histogram
// ---------------------------------------------------------------------------
// grid (ceil(L / chunk), B), 1024 threads (16 waves, one query row each for
// the statistics).  One memory latency: the scoring
// workgroups' statistics of this workgroup's query rows, the per-run maxima
// of its chunk and the chunk's exp values (plus the pooling halo) are all
// requested before any of them is used.  Then each wave folds its query rows'
// statistics into the global (M, S) (the same fixed order in every workgroup,
// so A~ is deterministic) and the per-run factors exp(run max - M) / S; the
// window mean of every staged position is formed once; each thread pools and
// aggregates 2 consecutive outputs from a register window.

constexpr int kRelThreads = 1024;
constexpr int kRelStatPer = 4;                // statistics pairs per lane per batch
constexpr int kRelRunPer = 3;                 // tile references per lane (chunk <= 2048)
constexpr int kRelPerThr = 2;                 // outputs per thread

template <int H>
__device__ __forceinline__ void pool_window(const double* __restrict__ v, int pool_mode, int kappa, double (&p)[kRelPerThr]) {
  // v points at the window of output 0; outputs j read v[j .. j + 2H]
  double w[kRelPerThr + 2 * H];
#pragma unroll
  for (int i = 0; i < kRelPerThr + 2 * H; ++i) w[i] = v[i];
#pragma unroll
  for (int j = 0; j < kRelPerThr; ++j) {
    double a = w[j];
#pragma unroll
    for (int o = 1; o <= 2 * H; ++o) a = (pool_mode == S4R_POOL_MAX) ? fmax(a, w[j + o]) : a + w[j + o];
    p[j] = (pool_mode == S4R_POOL_MAX) ? a : a / kappa;
  }
}

__global__ __launch_bounds__(kRelThreads) void k_relevance(
    const float* __restrict__ e, const double* __restrict__ run_m, const double* __restrict__ wg_stats,
    float* __restrict__ atilde, uint32_t* __restrict__ hist, float* __restrict__ scores_out,
    int64_t cap, int L, int n_hist, int G, int Wq, int kappa, int pool_mode, int agg, int ntiles_cap, int nwg,
    int chunk) {
  const int b = blockIdx.y;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int GW = G * Wq;
  const int h = kappa / 2;
  const int HP = (h + 3) & ~3;                              // halo slot rounded to 16 bytes
  const int SP = chunk + 2 * HP;                            // staged row stride (floats)
  const int t0 = blockIdx.x * chunk;
  const int span = chunk + 2 * h;
  const int x0 = t0 - h;                                    // first staged position
  const int r_first = max(x0, 0) / kTileTok;               // tiles with a softmax reference
  const int r_last = (min(t0 + chunk + h, L) - 1) / kTileTok;
  const int nr = r_last - r_first + 1;                      // <= chunk / 16 + 2 <= 64 * kRelRunPer
  const int nrc = chunk / kTileTok + 4;                     // tile slots per query row

  // dynamic LDS: histogram, per-run factors, window means, exp values
  extern __shared__ __align__(16) unsigned char lds[];
  uint32_t* hl = reinterpret_cast<uint32_t*>(lds);
  double* fac = reinterpret_cast<double*>(hl + kHistBins);  // [GW][nrc]: exp(run max - M) / S
  double* vs = fac + GW * nrc;                              // [G][span]: window mean at x0 + i
  float* e_s = reinterpret_cast<float*>(vs + G * span);     // [GW][SP]: x at [HP + x - t0]

  // ---- all global reads of this workgroup, issued before any is used ----------
  const double2* stats = reinterpret_cast<const double2*>(wg_stats) + (int64_t)b * GW * nwg;
  double2 st[kRelStatPer];
  double rm[kRelRunPer];
  {
    const int gi = min(wave, GW - 1);            // waves >= GW re-read the last row (unused)
#pragma unroll
    for (int k = 0; k < kRelStatPer; ++k) st[k] = stats[(int64_t)gi * nwg + min(lane + 64 * k, nwg - 1)];
#pragma unroll
    for (int k = 0; k < kRelRunPer; ++k) rm[k] = run_m[((int64_t)b * GW + gi) * ntiles_cap + min(r_first + lane + 64 * k, r_last)];
  }
  {
    // pooling halo (4-byte items, GW * 2h <= kRelThreads): one per thread,
    // loaded before the main batch so that batch's wait covers it
    const int nh = GW * 2 * h;
    float halo_v = 0.f;
    int halo_o = 0;
    if (nh > 0) {
      const int i = min(t, nh - 1);
      const int gi = i / (2 * h), k = i % (2 * h);
      const int x = (k < h) ? t0 - h + k : t0 + chunk + (k - h);
      halo_v = e[((int64_t)b * GW + gi) * cap + min(max(x, 0), L - 1)];   // out-of-range halo is never used
      halo_o = gi * SP + ((k < h) ? HP - h + k : HP + chunk + (k - h));
    }
    // the chunk itself: 16-byte items, chunk / 4 of them per query row (a power
    // of two), clamped to the row's valid part (t0 is a multiple of 4;
    // rounding L - t0 up to 4 stays below the capacity, a multiple of 16)
    const int lc4 = __builtin_ctz(chunk / 4);
    const int c4 = (min(chunk, L - t0) + 3) / 4;
    batched_copy16<2>(
        GW << lc4,
        [&](int i) {
          return reinterpret_cast<const uint4*>(e + ((int64_t)b * GW + (i >> lc4)) * cap + t0) +
                 min(i & ((1 << lc4) - 1), c4 - 1);
        },
        [&](int i) {
          return reinterpret_cast<uint4*>(e_s + (i >> lc4) * SP + HP) + min(i & ((1 << lc4) - 1), c4 - 1);
        });
    if (nh > 0) e_s[halo_o] = halo_v;            // threads past nh rewrite item nh - 1
  }
  for (int i = t; i < kHistBins; i += blockDim.x) hl[i] = 0;

  // ---- global (M, S) of each query row and the per-run factors (one wave per row)
  if (wave < GW) {
    const int gi = wave;
    const double* srow = wg_stats + ((int64_t)b * GW + gi) * nwg * 2;
    double M = -INFINITY, S = 0.0;
    for (int base = 0; base < nwg; base += 64 * kRelStatPer) {
      double2 s2[kRelStatPer];
      if (base == 0) {
#pragma unroll
        for (int k = 0; k < kRelStatPer; ++k) s2[k] = st[k];
      } else {                                              // more than 256 scoring workgroups: reload
#pragma unroll
        for (int k = 0; k < kRelStatPer; ++k) {
          const int w = min(base + lane + 64 * k, nwg - 1);
          s2[k] = make_double2(srow[2 * w], srow[2 * w + 1]);
        }
      }
      double m = -INFINITY;
#pragma unroll
      for (int k = 0; k < kRelStatPer; ++k)
        if (base + lane + 64 * k < nwg) m = fmax(m, s2[k].x);
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) m = fmax(m, shfl_xor_d(m, o));
      double s = 0.0;
#pragma unroll
      for (int k = 0; k < kRelStatPer; ++k)
        if (base + lane + 64 * k < nwg && s2[k].x != -INFINITY) s += s2[k].y * exp(s2[k].x - m);
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) s += shfl_xor_d(s, o);
      if (m != -INFINITY) {                                 // merge this batch into (M, S)
        const double Mn = fmax(M, m);
        S = ((M == -INFINITY) ? 0.0 : S * exp(M - Mn)) + s * exp(m - Mn);
        M = Mn;
      }
    }
    const double inv_s = 1.0 / S;
#pragma unroll
    for (int k = 0; k < kRelRunPer; ++k)
      if (lane + 64 * k < nr) fac[gi * nrc + lane + 64 * k] = (rm[k] == -INFINITY) ? 0.0 : exp(rm[k] - M) * inv_s;
  }
  __syncthreads();

  // ---- window mean over the W_q rows of every staged position --------------------
  const double pad = (pool_mode == S4R_POOL_MAX) ? -INFINITY : 0.0;
  const double inv_wq = 1.0 / Wq;
  for (int g = 0; g < G; ++g) {
    for (int i = t; i < span; i += blockDim.x) {
      const int x = x0 + i;
      const int xr = min(max(x, max(x0, 0)), L - 1) / kTileTok - r_first;
      double sum = 0.0;
      for (int wi = 0; wi < Wq; ++wi) {
        const int gi = g * Wq + wi;
        sum += (double)e_s[gi * SP + HP - h + i] * fac[gi * nrc + xr];
      }
      vs[g * span + i] = (x >= 0 && x < L) ? ((Wq == 1) ? sum : sum * inv_wq) : pad;
    }
  }
  __syncthreads();

  // ---- pooling (kappa) and aggregation over G, 2 outputs per thread -----------
  const int own = t * kRelPerThr;                           // first output (chunk-relative)
  double acc[kRelPerThr];
#pragma unroll
  for (int j = 0; j < kRelPerThr; ++j) acc[j] = (agg == S4R_AGG_MEAN) ? 0.0 : -INFINITY;
  if (own < chunk) {
    for (int g = 0; g < G; ++g) {
      const double* v = vs + g * span + own;                // window of output j: v[j .. j + 2h]
      double p[kRelPerThr];
      switch (h) {
        case 0: pool_window<0>(v, pool_mode, kappa, p); break;
        case 1: pool_window<1>(v, pool_mode, kappa, p); break;
        case 2: pool_window<2>(v, pool_mode, kappa, p); break;
        case 3: pool_window<3>(v, pool_mode, kappa, p); break;
        case 4: pool_window<4>(v, pool_mode, kappa, p); break;
        default:
#pragma unroll
          for (int j = 0; j < kRelPerThr; ++j) {
            double a = v[j];
            for (int o = 1; o < kappa; ++o) a = (pool_mode == S4R_POOL_MAX) ? fmax(a, v[j + o]) : a + v[j + o];
            p[j] = (pool_mode == S4R_POOL_MAX) ? a : a / kappa;
          }
      }
#pragma unroll
      for (int j = 0; j < kRelPerThr; ++j) acc[j] = (agg == S4R_AGG_MEAN) ? acc[j] + p[j] : fmax(acc[j], p[j]);
    }
  }
#pragma unroll
  for (int j = 0; j < kRelPerThr; ++j) {
    const int x = t0 + own + j;
    const bool valid = own < chunk && x < L;
    const float af = (float)((agg == S4R_AGG_MEAN) ? acc[j] / G : acc[j]);
    if (valid) {
      atilde[(int64_t)b * cap + x] = af;
      if (scores_out) scores_out[(int64_t)b * L + x] = af;
    }
    if (valid && x < n_hist) atomicAdd(&hl[score_key(af) >> kHistShift], 1u);
  }
  __syncthreads();
  // this workgroup's histogram into the sequence's (zeroed by the query
  // projection earlier in the step): one global atomic per non-empty bin
  uint32_t* hs = hist + (int64_t)b * kHistBins;
  for (int i = t; i < kHistBins; i += blockDim.x) {
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
                                                     int L, int n_hist) {
  const int b = blockIdx.y;
  __shared__ uint32_t hl[kHistBins];
  for (int i = threadIdx.x; i < kHistBins; i += blockDim.x) hl[i] = 0;
  __syncthreads();
  const int t0 = blockIdx.x * kHistChunk;
  for (int i = threadIdx.x; i < kHistChunk; i += blockDim.x) {
    const int x = t0 + i;
    if (x < n_hist) atomicAdd(&hl[score_key(scores[(int64_t)b * L + x]) >> kHistShift], 1u);
  }
  __syncthreads();
  uint32_t* hs = hist + (int64_t)b * kHistBins;
  for (int i = threadIdx.x; i < kHistBins; i += blockDim.x) {
    const uint32_t c = hl[i];
    if (c) atomicAdd(&hs[i], c);
  }
}

int relevance_chunk(int GW) { return GW <= 4 ? 2048 : (GW <= 8 ? 1024 : 512); }   // <= kRelThreads * kRelPerThr

size_t relevance_lds(int G, int GW, int chunk, int kappa) {
  const int h = kappa / 2;
  const int span = chunk + 2 * h;
  const int SP = chunk + 2 * ((h + 3) & ~3);
  const int nrc = chunk / kTileTok + 4;
  return kHistBins * 4 + (size_t)(GW * nrc + (size_t)G * span) * 8 + (size_t)GW * SP * 4 + 16;
}

hipError_t launch_relevance(const Problem& P, const Workspace& ws, int64_t L, float* scores_out, hipStream_t st) {
  const int n_hist = (int)std::max<int64_t>(L - P.W, 0);
  const int chunk = relevance_chunk(P.GW);
  const size_t lds = relevance_lds(P.G, P.GW, chunk, P.kappa);
  dim3 grid((unsigned)((L + chunk - 1) / chunk), P.B);
  hipLaunchKernelGGL(k_relevance, grid, dim3(kRelThreads), lds, st, ws.e, ws.run_m, ws.wg_stats, ws.atilde, ws.hist,
                     scores_out, P.cap, (int)L, n_hist, P.G, P.Wq, P.kappa, P.pool_mode, P.agg,
                     (int)(P.cap / kTileTok), score_workgroups(P, L), chunk);
  return hipGetLastError();
}

hipError_t launch_hist_only(const Problem& P, const Workspace& ws, int64_t L, const float* scores, hipStream_t st) {
  const int n_hist = (int)std::max<int64_t>(L - P.W, 0);
  const int ng = std::max(1, (n_hist + kHistChunk - 1) / kHistChunk);
  hipLaunchKernelGGL(k_zero_hist, dim3((P.B * kHistBins + 255) / 256), dim3(256), 0, st, ws.hist, P.B * kHistBins);
  hipLaunchKernelGGL(k_hist_scores, dim3(ng, P.B), dim3(256), 0, st, scores, ws.hist, (int)L, n_hist);
  return hipGetLastError();
}

}  // namespace s4r
