// Latent relevance of every cached token (Section 3.2.1 cache update,
// Section 3.2.2 latent logits / softmax / window mean, and the pooling and
// group-aggregation equations of Section 3.2.3), for gfx950.
//
//   k_prepare      c_t^Q = s_t^Q B^K for each query group (fp64 accumulation),
//                  split into three bf16 parts for the MFMA stream; optional
//                  projection of the new token's K/V into coefficient row L-1.
//   k_score_stream streams C^K once (the HBM-bound pass), Z = C^Q C^K^T/sqrt(R)
//                  on bf16 MFMA with per-block fp64 accumulation, writes
//                  exp(z - run max) and per-run (max, sum); the last
//                  workgroup of each sequence folds the runs into (M, S).
//   k_relevance    p = e * exp(run max - M) / S, mean over the W_q rows,
//                  pooling with kernel kappa, aggregation over G -> A~ (fp32),
//                  plus the 4096-bin radix histogram used by the selection.
//   k_pack         row-major <-> tiled coefficient layout.
#include "s4r_device.h"
#include "s4r_internal.h"

namespace s4r {

// ---------------------------------------------------------------------------
// K0: query projection, FIFO assembly, cache update, scratch clearing
// ---------------------------------------------------------------------------
// grid (R/64 chunks, B, 2 = {key basis, value basis}), 256 threads.  Lane =
// latent column inside the chunk, wave w = quarter of the basis group's rows.
constexpr int kPrepMaxVec = kMaxGW + 1;   // G query groups + the new key

template <typename T>
__global__ __launch_bounds__(256) void k_prepare(
    const T* __restrict__ q, const float* __restrict__ qwin_prev, const T* __restrict__ bases_k,
    const T* __restrict__ bases_v, const T* __restrict__ k_new, const T* __restrict__ v_new,
    T* __restrict__ coef_k, T* __restrict__ coef_v, int64_t append_row, float* __restrict__ qcoef_out,
    uint16_t* __restrict__ cq_split, uint32_t* __restrict__ hist, uint32_t* __restrict__ counters,
    int hq, int hkv, int dh, int G, int nb, int rank, int R, int Wq, int bases_shared,
    int64_t cap, int do_query, int clear) {
  const int chunk = blockIdx.x, b = blockIdx.y, which = blockIdx.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int Dp = hkv * dh, Dg = Dp / nb;
  const int r = chunk * 64 + lane;
  const bool r_ok = r < R;
  const int grp = r_ok ? r / rank : 0, rr = r_ok ? r % rank : 0;

  if (clear && chunk == 0 && which == 0) {
    for (int i = threadIdx.x; i < kHistBins; i += blockDim.x) hist[(int64_t)b * kHistBins + i] = 0;
    if (threadIdx.x < kCounters) counters[b * kCounters + threadIdx.x] = 0;
  }

  // vectors projected by this workgroup
  const T* vec_new = which == 0 ? k_new : v_new;
  const int nq = (which == 0 && do_query) ? G : 0;
  const int nvec = nq + (vec_new ? 1 : 0);
  if (nvec == 0) return;

  constexpr int kSlice = 256;                       // basis rows staged per pass
  __shared__ float xs[kPrepMaxVec][kSlice];
  __shared__ double red[4][kPrepMaxVec][64];

  const T* bases = (which == 0 ? bases_k : bases_v) + (bases_shared ? 0 : (int64_t)b * Dp * rank);
  double acc[kPrepMaxVec];
#pragma unroll
  for (int v = 0; v < kPrepMaxVec; ++v) acc[v] = 0.0;

  // the chunk's 64 columns may span two basis groups (rank = 32); walk the
  // groups touched and let each lane accumulate only its own
  const int g_first = (chunk * 64) / rank;
  const int g_last = min(nb - 1, (chunk * 64 + 63) / rank);
  for (int gg = g_first; gg <= g_last; ++gg) {
    for (int d0 = 0; d0 < Dg; d0 += kSlice) {
      const int nrow = min(kSlice, Dg - d0);
      __syncthreads();
      for (int i = threadIdx.x; i < nvec * nrow; i += blockDim.x) {
        const int v = i / nrow, d = i % nrow, dd = gg * Dg + d0 + d;   // feature index in Dp
        float x;
        if (v < nq) {  // group query v: head j*G + v, j = dd / dh
          const int j = dd / dh;
          x = load_elem(q, ((int64_t)b * hq + (int64_t)j * G + v) * dh + dd % dh);
        } else {
          x = load_elem(vec_new, (int64_t)b * Dp + dd);
        }
        xs[v][d] = x;
      }
      __syncthreads();
      if (r_ok && grp == gg) {
        const T* bp = bases + ((int64_t)gg * Dg + d0) * rank + rr;
        for (int d = wave; d < nrow; d += 4) {
          const double bv = (double)load_elem(bp, (int64_t)d * rank);
#pragma unroll
          for (int v = 0; v < kPrepMaxVec; ++v)
            if (v < nvec) acc[v] = fma((double)xs[v][d], bv, acc[v]);
        }
      }
    }
  }
#pragma unroll
  for (int v = 0; v < kPrepMaxVec; ++v) red[wave][v][lane] = acc[v];
  __syncthreads();
  if (wave != 0 || !r_ok) return;
  for (int v = 0; v < nvec; ++v) {
    double x = red[0][v][lane] + red[1][v][lane] + red[2][v][lane] + red[3][v][lane];
    if (v < nq) {
      // current query coefficients are the newest FIFO row (i = Wq - 1)
      const int gi = v * Wq + (Wq - 1);
      Split3 sp = split3(x);
      const int64_t base = ((int64_t)b * 3) * (G * Wq) * R;
      cq_split[base + ((int64_t)0 * G * Wq + gi) * R + r] = sp.hi;
      cq_split[base + ((int64_t)1 * G * Wq + gi) * R + r] = sp.mid;
      cq_split[base + ((int64_t)2 * G * Wq + gi) * R + r] = sp.lo;
      if (qcoef_out) qcoef_out[((int64_t)b * G + v) * R + r] = (float)x;
    } else {
      T* coef = which == 0 ? coef_k : coef_v;
      store_elem(coef, (int64_t)b * cap * R + tiled_offset(append_row, r, R), x);
    }
  }
  if (which == 0 && do_query) {
    // older FIFO rows come from the caller, fp32, oldest first
    for (int g = 0; g < G; ++g)
      for (int i = 0; i < Wq - 1; ++i) {
        double x = (double)qwin_prev[(((int64_t)b * G + g) * (Wq - 1) + i) * R + r];
        Split3 sp = split3(x);
        const int gi = g * Wq + i;
        const int64_t base = ((int64_t)b * 3) * (G * Wq) * R;
        cq_split[base + ((int64_t)0 * G * Wq + gi) * R + r] = sp.hi;
        cq_split[base + ((int64_t)1 * G * Wq + gi) * R + r] = sp.mid;
        cq_split[base + ((int64_t)2 * G * Wq + gi) * R + r] = sp.lo;
      }
  }
}

// ---------------------------------------------------------------------------
// K1: the coefficient stream
// ---------------------------------------------------------------------------
// grid (workgroups per sequence, B), 256 threads = 4 waves.  A wave owns whole
// runs of kRunTiles tiles (16 tokens each); each 16x32 block of C^K is one
// coalesced 1 KiB wave load that lands directly in MFMA A-operand layout.
// The B operand holds the query-coefficient columns (G*W_q <= 16), as hi,
// mid and lo bf16 parts accumulated into the same fp32 MFMA result, which is
// folded into fp64 after every 32-column block.

template <typename T>
struct ALoad;

template <>
struct ALoad<uint16_t> {  // 8 bf16 = one 16-byte load
  static constexpr int kParts = 1;
  __device__ __forceinline__ static void load(const uint16_t* p, Op8 (&a)[1]) {
    a[0].u = *reinterpret_cast<const uint4*>(p);
  }
};

template <>
struct ALoad<float> {  // 8 fp32 = two 16-byte loads, split into 3 bf16 parts
  static constexpr int kParts = 3;
  __device__ __forceinline__ static void load(const float* p, Op8 (&a)[3]) {
    float x[8];
    *reinterpret_cast<float4*>(&x[0]) = *reinterpret_cast<const float4*>(p);
    *reinterpret_cast<float4*>(&x[4]) = *reinterpret_cast<const float4*>(p + 4);
    split_f32x8(x, a[0], a[1], a[2]);
  }
};

template <typename T, int RB>
__global__ __launch_bounds__(256) void k_score_stream(
    const T* __restrict__ coef_k, const uint16_t* __restrict__ cq_split, float* __restrict__ e_out,
    double* __restrict__ run_m, double* __restrict__ run_s, double* __restrict__ gstat,
    uint32_t* __restrict__ counters, int64_t cap, int L, int GW, int Wq, int nruns,
    int runs_per_wave, double scale) {
  constexpr int R = RB * kBlkCol;
  constexpr int NP = ALoad<T>::kParts;
  const int b = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 15, kg = lane >> 4;       // MFMA column / k-group of this lane
  const T* cb = coef_k + (int64_t)b * cap * R;

  // B operands: column col = query row gi, k-group kg, three bf16 parts
  Op8 bop[RB][3];
  {
    const uint16_t* cs = cq_split + (int64_t)b * 3 * GW * R;
#pragma unroll
    for (int kb = 0; kb < RB; ++kb)
#pragma unroll
      for (int p = 0; p < 3; ++p) {
        if (col < GW)
          bop[kb][p].u = *reinterpret_cast<const uint4*>(cs + ((int64_t)p * GW + col) * R + kb * 32 + kg * 8);
        else
          bop[kb][p].u = make_uint4(0, 0, 0, 0);
      }
  }
  // causal limit of this column's query row (Section 3.2.2): keys l <= L - Wq + i
  const int i_row = col % Wq;
  const int lim = (col < GW) ? (L - Wq + i_row) : -1;
  const int ntiles = (L + 15) / 16;

  const int run0 = (blockIdx.x * kScoreWaves + wave) * runs_per_wave;
  for (int ri = 0; ri < runs_per_wave; ++ri) {
    const int run = run0 + ri;
    if (run >= nruns) break;
    double z[kRunTiles][4];
#pragma unroll
    for (int t = 0; t < kRunTiles; ++t) {
      const int tile = run * kRunTiles + t;
      double acc[4] = {0.0, 0.0, 0.0, 0.0};
      if (tile < ntiles) {
        const T* tp = cb + (int64_t)tile * 16 * R + col * 32 + kg * 8;
        Op8 a[RB][NP];
#pragma unroll
        for (int kb = 0; kb < RB; ++kb) ALoad<T>::load(tp + kb * 512, a[kb]);
#pragma unroll
        for (int kb = 0; kb < RB; ++kb) {
          floatx4 d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int pa = 0; pa < NP; ++pa) {
            d = mfma16x16x32(a[kb][pa], bop[kb][0], d);
            d = mfma16x16x32(a[kb][pa], bop[kb][1], d);
            d = mfma16x16x32(a[kb][pa], bop[kb][2], d);
          }
#pragma unroll
          for (int v = 0; v < 4; ++v) acc[v] += (double)d[v];
        }
      }
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int tok = tile * 16 + kg * 4 + v;
        z[t][v] = (tile < ntiles && tok < L && tok <= lim) ? acc[v] * scale : -INFINITY;
      }
    }
    // run maximum of this column (lanes col, col+16, col+32, col+48)
    double m = -INFINITY;
#pragma unroll
    for (int t = 0; t < kRunTiles; ++t)
#pragma unroll
      for (int v = 0; v < 4; ++v) m = fmax(m, z[t][v]);
    m = fmax(m, shfl_xor_d(m, 16));
    m = fmax(m, shfl_xor_d(m, 32));
    double s = 0.0;
#pragma unroll
    for (int t = 0; t < kRunTiles; ++t) {
      float ev[4];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        ev[v] = (z[t][v] == -INFINITY) ? 0.f : expf((float)(z[t][v] - m));
        s += (double)ev[v];
      }
      const int tile = run * kRunTiles + t;
      if (col < GW && tile < ntiles) {
        float* dst = e_out + ((int64_t)b * GW + col) * cap + (int64_t)tile * 16 + kg * 4;
        *reinterpret_cast<float4*>(dst) = make_float4(ev[0], ev[1], ev[2], ev[3]);
      }
    }
    s += shfl_xor_d(s, 16);
    s += shfl_xor_d(s, 32);
    if (kg == 0 && col < GW) {
      run_m[((int64_t)b * GW + col) * nruns + run] = m;
      run_s[((int64_t)b * GW + col) * nruns + run] = s;
    }
  }

  // the last workgroup of this sequence folds the runs into (M, S)
  __shared__ int last;
  __shared__ double red[256];
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned t = atomicAdd(&counters[b * kCounters + 0], 1u);
    last = (t == gridDim.x - 1);
  }
  __syncthreads();
  if (!last) return;
  __threadfence();
  for (int gi = 0; gi < GW; ++gi) {
    const double* rm = run_m + ((int64_t)b * GW + gi) * nruns;
    const double* rs = run_s + ((int64_t)b * GW + gi) * nruns;
    double m = -INFINITY;
    for (int i = threadIdx.x; i < nruns; i += blockDim.x) m = fmax(m, rm[i]);
    red[threadIdx.x] = m;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
      if (threadIdx.x < w) red[threadIdx.x] = fmax(red[threadIdx.x], red[threadIdx.x + w]);
      __syncthreads();
    }
    const double M = red[0];
    __syncthreads();
    double s = 0.0;
    for (int i = threadIdx.x; i < nruns; i += blockDim.x) {
      double mi = rm[i];
      if (mi != -INFINITY) s += rs[i] * exp(mi - M);
    }
    red[threadIdx.x] = s;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
      if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
      __syncthreads();
    }
    if (threadIdx.x == 0) {
      gstat[((int64_t)b * GW + gi) * 2 + 0] = M;
      gstat[((int64_t)b * GW + gi) * 2 + 1] = red[0];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) counters[b * kCounters + 0] = 0;
}

// ---------------------------------------------------------------------------
// K2: relevance A~ and its radix histogram
// ---------------------------------------------------------------------------
// grid (ceil(L / kRelChunk), B), 256 threads.
constexpr int kMaxHalo = 32;   // pool_kernel <= 65

__global__ __launch_bounds__(256) void k_relevance(
    const float* __restrict__ e, const double* __restrict__ run_m, const double* __restrict__ gstat,
    float* __restrict__ atilde, uint32_t* __restrict__ hist, float* __restrict__ scores_out,
    int64_t cap, int L, int n_hist, int G, int Wq, int kappa, int pool_mode, int agg, int nruns) {
  const int b = blockIdx.y;
  const int GW = G * Wq;
  const int h = kappa / 2;
  const int t0 = blockIdx.x * kRelChunk;
  const int span = kRelChunk + 2 * h;
  const int r_first = max(t0 - h, 0) / kRunTok;
  const int r_last = min(t0 + kRelChunk + h, L) / kRunTok;   // inclusive bound, may exceed
  const int nr = r_last - r_first + 1;

  __shared__ double fac[kMaxGW][kRelChunk / kRunTok + 4];   // exp(run max - M) / S
  __shared__ double aq[kRelChunk + 2 * kMaxHalo];           // window-mean relevance of one group
  __shared__ double agg_acc[kRelChunk];
  __shared__ uint32_t hl[kHistBins];

  for (int i = threadIdx.x; i < kHistBins; i += blockDim.x) hl[i] = 0;
  for (int i = threadIdx.x; i < GW * nr; i += blockDim.x) {
    const int gi = i / nr, rr = r_first + i % nr;
    double f = 0.0;
    if (rr < nruns) {
      const double M = gstat[((int64_t)b * GW + gi) * 2 + 0];
      const double S = gstat[((int64_t)b * GW + gi) * 2 + 1];
      const double mr = run_m[((int64_t)b * GW + gi) * nruns + rr];
      f = (mr == -INFINITY) ? 0.0 : exp(mr - M) / S;
    }
    fac[gi][i % nr] = f;
  }
  for (int i = threadIdx.x; i < kRelChunk; i += blockDim.x) agg_acc[i] = (agg == S4R_AGG_MEAN) ? 0.0 : -INFINITY;
  __syncthreads();

  for (int g = 0; g < G; ++g) {
    // window mean over the W_q query rows, on [t0 - h, t0 + chunk + h)
    for (int i = threadIdx.x; i < span; i += blockDim.x) {
      const int x = t0 - h + i;
      double v;
      if (x < 0 || x >= L) {
        v = (pool_mode == S4R_POOL_MAX) ? -INFINITY : 0.0;
      } else {
        double sum = 0.0;
        for (int wi = 0; wi < Wq; ++wi) {
          const int gi = g * Wq + wi;
          sum += (double)e[((int64_t)b * GW + gi) * cap + x] * fac[gi][x / kRunTok - r_first];
        }
        v = sum / Wq;
      }
      aq[i] = v;
    }
    __syncthreads();
    for (int i = threadIdx.x; i < kRelChunk; i += blockDim.x) {
      double p;
      if (pool_mode == S4R_POOL_MAX) {
        p = -INFINITY;
        for (int o = 0; o < kappa; ++o) p = fmax(p, aq[i + o]);
      } else {
        p = 0.0;
        for (int o = 0; o < kappa; ++o) p += aq[i + o];
        p = p / kappa;
      }
      if (agg == S4R_AGG_MEAN) agg_acc[i] += p;
      else agg_acc[i] = fmax(agg_acc[i], p);
    }
    __syncthreads();
  }
  for (int i = threadIdx.x; i < kRelChunk; i += blockDim.x) {
    const int x = t0 + i;
    if (x >= L) continue;
    double a = agg_acc[i];
    if (agg == S4R_AGG_MEAN) a = a / G;
    const float af = (float)a;
    atilde[(int64_t)b * cap + x] = af;
    if (scores_out) scores_out[(int64_t)b * L + x] = af;
    if (x < n_hist) atomicAdd(&hl[score_key(af) >> kHistShift], 1u);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < kHistBins; i += blockDim.x)
    if (hl[i]) atomicAdd(&hist[(int64_t)b * kHistBins + i], hl[i]);
}

// histogram of caller-provided scores (standalone selection); clears first
__global__ __launch_bounds__(256) void k_clear(uint32_t* __restrict__ hist, uint32_t* __restrict__ counters,
                                               int B) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < B * kHistBins; i += gridDim.x * blockDim.x) hist[i] = 0;
  if (blockIdx.x == 0 && threadIdx.x < B * kCounters) counters[threadIdx.x] = 0;
}

__global__ __launch_bounds__(256) void k_hist_scores(const float* __restrict__ scores, uint32_t* __restrict__ hist,
                                                     int L, int n_hist) {
  const int b = blockIdx.y;
  __shared__ uint32_t hl[kHistBins];
  for (int i = threadIdx.x; i < kHistBins; i += blockDim.x) hl[i] = 0;
  __syncthreads();
  const int t0 = blockIdx.x * kRelChunk;
  for (int i = threadIdx.x; i < kRelChunk; i += blockDim.x) {
    const int x = t0 + i;
    if (x < n_hist) atomicAdd(&hl[score_key(scores[(int64_t)b * L + x]) >> kHistShift], 1u);
  }
  __syncthreads();
  for (int i = threadIdx.x; i < kHistBins; i += blockDim.x)
    if (hl[i]) atomicAdd(&hist[(int64_t)b * kHistBins + i], hl[i]);
}

// ---------------------------------------------------------------------------
// layout conversion
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void k_pack(const T* __restrict__ src, T* __restrict__ dst, int64_t n_rows,
                                              int R, int64_t cap, int to_tiled) {
  const int b = blockIdx.y;
  const int64_t n = n_rows * R;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t t = i / R;
    const int c = (int)(i % R);
    const int64_t ro = (int64_t)b * n_rows * R + i;
    const int64_t to = (int64_t)b * cap * R + tiled_offset(t, c, R);
    if (to_tiled) dst[to] = src[ro];
    else dst[ro] = src[to];
  }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
hipError_t launch_prepare(const Problem& P, const Workspace& ws, int64_t L, const void* q,
                          const float* qwin_prev, const void* bases_k, const void* bases_v,
                          const void* k_new, const void* v_new, void* coef_k, void* coef_v,
                          int64_t append_row, float* qcoef_out, bool do_query, bool clear,
                          hipStream_t st) {
  (void)L;
  dim3 grid((P.R + 63) / 64, P.B, 2);
  if (P.dtype == S4R_BF16)
    hipLaunchKernelGGL(k_prepare<uint16_t>, grid, dim3(256), 0, st, (const uint16_t*)q, qwin_prev,
                       (const uint16_t*)bases_k, (const uint16_t*)bases_v, (const uint16_t*)k_new,
                       (const uint16_t*)v_new, (uint16_t*)coef_k, (uint16_t*)coef_v, append_row, qcoef_out,
                       ws.cq_split, ws.hist, ws.counters, P.hq, P.hkv, P.dh, P.G, P.nb, P.rank, P.R, P.Wq,
                       P.bases_shared, P.cap, (int)do_query, (int)clear);
  else
    hipLaunchKernelGGL(k_prepare<float>, grid, dim3(256), 0, st, (const float*)q, qwin_prev,
                       (const float*)bases_k, (const float*)bases_v, (const float*)k_new, (const float*)v_new,
                       (float*)coef_k, (float*)coef_v, append_row, qcoef_out, ws.cq_split, ws.hist,
                       ws.counters, P.hq, P.hkv, P.dh, P.G, P.nb, P.rank, P.R, P.Wq, P.bases_shared, P.cap,
                       (int)do_query, (int)clear);
  return hipGetLastError();
}

template <typename T, int RB>
static void launch_stream_t(const Problem& P, const Workspace& ws, int64_t L, const void* coef_k, hipStream_t st) {
  const int ntiles = (int)((L + 15) / 16);
  const int nruns = (ntiles + kRunTiles - 1) / kRunTiles;
  // a handful of runs per wave keeps per-wave setup small and the grid large
  int rpw = 1;
  while (rpw < 8 && (int64_t)nruns / (rpw * 2 * kScoreWaves) >= 2 * 256) rpw *= 2;
  const int nwg = (nruns + rpw * kScoreWaves - 1) / (rpw * kScoreWaves);
  hipLaunchKernelGGL((k_score_stream<T, RB>), dim3(nwg, P.B), dim3(256), 0, st, (const T*)coef_k, ws.cq_split,
                     ws.e, ws.run_m, ws.run_s, ws.gstat, ws.counters, P.cap, (int)L, P.GW, P.Wq, nruns, rpw,
                     1.0 / sqrt((double)P.R));
}

template <typename T>
static bool dispatch_rb(const Problem& P, const Workspace& ws, int64_t L, const void* coef_k, hipStream_t st) {
  switch (P.R / 32) {
    case 1: launch_stream_t<T, 1>(P, ws, L, coef_k, st); return true;
    case 2: launch_stream_t<T, 2>(P, ws, L, coef_k, st); return true;
    case 3: launch_stream_t<T, 3>(P, ws, L, coef_k, st); return true;
    case 4: launch_stream_t<T, 4>(P, ws, L, coef_k, st); return true;
    case 5: launch_stream_t<T, 5>(P, ws, L, coef_k, st); return true;
    case 6: launch_stream_t<T, 6>(P, ws, L, coef_k, st); return true;
    case 7: launch_stream_t<T, 7>(P, ws, L, coef_k, st); return true;
    case 8: launch_stream_t<T, 8>(P, ws, L, coef_k, st); return true;
    default: return false;
  }
}

hipError_t launch_score_stream(const Problem& P, const Workspace& ws, int64_t L, const void* coef_k,
                               hipStream_t st) {
  bool ok = P.dtype == S4R_BF16 ? dispatch_rb<uint16_t>(P, ws, L, coef_k, st)
                                : dispatch_rb<float>(P, ws, L, coef_k, st);
  if (!ok) return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_relevance(const Problem& P, const Workspace& ws, int64_t L, float* scores_out, hipStream_t st) {
  const int n_hist = (int)std::max<int64_t>(L - P.W, 0);
  const int ntiles = (int)((L + 15) / 16);
  const int nruns = (ntiles + kRunTiles - 1) / kRunTiles;
  dim3 grid((unsigned)((L + kRelChunk - 1) / kRelChunk), P.B);
  hipLaunchKernelGGL(k_relevance, grid, dim3(256), 0, st, ws.e, ws.run_m, ws.gstat, ws.atilde, ws.hist, scores_out,
                     P.cap, (int)L, n_hist, P.G, P.Wq, P.kappa, P.pool_mode, P.agg, nruns);
  return hipGetLastError();
}

hipError_t launch_hist_only(const Problem& P, const Workspace& ws, int64_t L, const float* scores, hipStream_t st) {
  hipLaunchKernelGGL(k_clear, dim3(16), dim3(256), 0, st, ws.hist, ws.counters, P.B);
  const int n_hist = (int)std::max<int64_t>(L - P.W, 0);
  if (n_hist > 0) {
    dim3 grid((unsigned)((n_hist + kRelChunk - 1) / kRelChunk), P.B);
    hipLaunchKernelGGL(k_hist_scores, grid, dim3(256), 0, st, scores, ws.hist, (int)L, n_hist);
  }
  return hipGetLastError();
}

hipError_t launch_pack(const Problem& P, int64_t n_rows, const void* src, void* dst, bool to_tiled, hipStream_t st) {
  if (n_rows <= 0) return hipSuccess;
  const int64_t n = n_rows * P.R;
  dim3 grid((unsigned)std::min<int64_t>((n + 255) / 256, 4096), P.B);
  if (P.dtype == S4R_BF16)
    hipLaunchKernelGGL(k_pack<uint16_t>, grid, dim3(256), 0, st, (const uint16_t*)src, (uint16_t*)dst, n_rows, P.R,
                       P.cap, (int)to_tiled);
  else
    hipLaunchKernelGGL(k_pack<float>, grid, dim3(256), 0, st, (const float*)src, (float*)dst, n_rows, P.R, P.cap,
                       (int)to_tiled);
  return hipGetLastError();
}

}  // namespace s4r
