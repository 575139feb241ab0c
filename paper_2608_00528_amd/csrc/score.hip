// Latent relevance of every cached token (Section 3.2.1 cache update,
// Section 3.2.2 latent logits / softmax / window mean, and the pooling and
// group-aggregation equations of Section 3.2.3), for gfx950.
//
//   k_prepare      c_t^Q = s_t^Q B^K for each query group (fp64 accumulation),
//                  split into three bf16 parts for the MFMA stream; optional
//                  projection of the new token's K/V into coefficient row L-1.
//   k_score_stream streams C^K once (the HBM-bound pass), Z = C^Q C^K^T/sqrt(R)
//                  on bf16 MFMA with per-block fp64 accumulation, writes
//                  exp(z - run max), per-run (max, sum) and per-workgroup
//                  (max, sum) statistics.
//   k_relevance    p = e * exp(run max - M) / S, mean over the W_q rows,
//                  pooling with kernel kappa, aggregation over G -> A~ (fp32),
//                  plus the 2048-bin radix histogram used by the selection.
//   k_pack         row-major <-> tiled coefficient layout.
#include "s4r_device.h"
#include "s4r_internal.h"

namespace s4r {

// ---------------------------------------------------------------------------
// K0: query projection, FIFO assembly, cache update
// ---------------------------------------------------------------------------
// grid (R/16 column blocks, B, 2 = {key basis, value basis}), 256 threads =
// 64 row groups x 4 column groups of 4 latent columns.  A workgroup owns 16
// columns of one basis group over all of its Dg rows (no cross-workgroup
// reduction).  Each thread issues the loads of all its rows of a 1024-row
// slice before using them; partial sums are reduced over the row groups with
// shuffles and then across the four waves in a fixed order (deterministic).
constexpr int kPrepVec = 8;       // vectors per pass
constexpr int kPrepMaxVec = kMaxGW + 1;   // query groups + the new row
constexpr int kPrepSlice = 1024;  // basis rows staged per pass

template <typename T>
struct Load4;
template <>
struct Load4<uint16_t> {
  __device__ __forceinline__ static void load(const uint16_t* p, float (&x)[4]) {
    const uint2 u = *reinterpret_cast<const uint2*>(p);
    x[0] = bf16_bits_to_f32(u.x & 0xFFFFu);
    x[1] = bf16_bits_to_f32(u.x >> 16);
    x[2] = bf16_bits_to_f32(u.y & 0xFFFFu);
    x[3] = bf16_bits_to_f32(u.y >> 16);
  }
};
template <>
struct Load4<float> {
  __device__ __forceinline__ static void load(const float* p, float (&x)[4]) {
    const float4 v = *reinterpret_cast<const float4*>(p);
    x[0] = v.x;
    x[1] = v.y;
    x[2] = v.z;
    x[3] = v.w;
  }
};

template <typename T>
__device__ __forceinline__ void write_qsplit(uint16_t* cq_split, int b, int G, int Wq, int R, int gi, int r, double x) {
  const Split3 sp = split3(x);
  const int64_t base = (int64_t)b * 3 * (G * Wq) * R;
  cq_split[base + ((int64_t)0 * G * Wq + gi) * R + r] = sp.hi;
  cq_split[base + ((int64_t)1 * G * Wq + gi) * R + r] = sp.mid;
  cq_split[base + ((int64_t)2 * G * Wq + gi) * R + r] = sp.lo;
}

template <typename T>
__global__ __launch_bounds__(256) void k_prepare(
    const T* __restrict__ q, const float* __restrict__ qwin_prev, const T* __restrict__ bases_k,
    const T* __restrict__ bases_v, const T* __restrict__ k_new, const T* __restrict__ v_new,
    T* __restrict__ coef_k, T* __restrict__ coef_v, int64_t append_row, float* __restrict__ qcoef_out,
    uint16_t* __restrict__ cq_split, int hq, int hkv, int dh, int G, int nb, int rank, int R, int Wq,
    int bases_shared, int64_t cap, int do_query) {
  const int cb = blockIdx.x, b = blockIdx.y, which = blockIdx.z;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int cg = t & 3, rg = t >> 2;              // 4 columns per thread, 64 row groups
  const int Dp = hkv * dh, Dg = Dp / nb;
  const int c0 = cb * 16;                         // first latent column of the block
  const int grp = c0 / rank, cc0 = c0 - grp * rank + cg * 4;

  const T* vec_new = which == 0 ? k_new : v_new;
  const int nq = (which == 0 && do_query) ? G : 0;
  const int nvec = nq + (vec_new ? 1 : 0);

  if (which == 0 && do_query && t < 16) {
    // older FIFO rows come from the caller, fp32, oldest first
    const int r = c0 + t;
    for (int g = 0; g < G; ++g)
      for (int i = 0; i < Wq - 1; ++i)
        write_qsplit<T>(cq_split, b, G, Wq, R, g * Wq + i, r,
                        (double)qwin_prev[(((int64_t)b * G + g) * (Wq - 1) + i) * R + r]);
  }
  if (nvec == 0) return;

  __shared__ float xs[kPrepVec][kPrepSlice];
  __shared__ double red[4][kPrepVec][16];
  const T* bases = (which == 0 ? bases_k : bases_v) + (bases_shared ? 0 : (int64_t)b * Dp * rank) +
                   (int64_t)grp * Dg * rank + cc0;

  for (int v0 = 0; v0 < nvec; v0 += kPrepVec) {
    const int nv = min(kPrepVec, nvec - v0);
    double acc[kPrepVec][4];
#pragma unroll
    for (int v = 0; v < kPrepVec; ++v)
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[v][c] = 0.0;
    for (int s0 = 0; s0 < Dg; s0 += kPrepSlice) {
      const int nrow = min(kPrepSlice, Dg - s0);
      constexpr int kPer = kPrepSlice / 64;         // rows per thread per slice
      float bv[kPer][4];
#pragma unroll
      for (int i = 0; i < kPer; ++i) {
        const int d = rg + 64 * i;
        if (d < nrow) Load4<T>::load(bases + (int64_t)(s0 + d) * rank, bv[i]);
      }
      __syncthreads();
      batched_copy4<16>(
          nv * nrow,
          [&](int i) -> float {
            const int v = v0 + i / nrow, dd = grp * Dg + s0 + i % nrow;   // feature index in Dp
            if (v < nq)  // group query v: head j*G + v, j = dd / dh
              return load_elem(q, ((int64_t)b * hq + (int64_t)(dd / dh) * G + v) * dh + dd % dh);
            return load_elem(vec_new, (int64_t)b * Dp + dd);
          },
          [&](int i, float x) { xs[i / nrow][i % nrow] = x; });
      __syncthreads();
#pragma unroll
      for (int i = 0; i < kPer; ++i) {
        const int d = rg + 64 * i;
        if (d < nrow) {
#pragma unroll
          for (int v = 0; v < kPrepVec; ++v) {
            if (v < nv) {
              const double xv = (double)xs[v][d];
#pragma unroll
              for (int c = 0; c < 4; ++c) acc[v][c] = fma(xv, (double)bv[i][c], acc[v][c]);
            }
          }
        }
      }
    }
    // reduce over the 16 row groups of this wave (lane bits 2..5), then the 4 waves
#pragma unroll
    for (int v = 0; v < kPrepVec; ++v)
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        double a = acc[v][c];
        a += shfl_xor_d(a, 4);
        a += shfl_xor_d(a, 8);
        a += shfl_xor_d(a, 16);
        a += shfl_xor_d(a, 32);
        if (lane < 4) red[wave][v][lane * 4 + c] = a;   // lane == cg here
      }
    __syncthreads();
    if (t < 16 * nv) {
      const int v = t / 16, col = t % 16;
      const double x = ((red[0][v][col] + red[1][v][col]) + red[2][v][col]) + red[3][v][col];
      const int r = c0 + col;
      const int vv = v0 + v;
      if (vv < nq) {
        // the current query's coefficients are the newest FIFO row (i = Wq - 1)
        write_qsplit<T>(cq_split, b, G, Wq, R, vv * Wq + (Wq - 1), r, x);
        if (qcoef_out) qcoef_out[((int64_t)b * G + vv) * R + r] = (float)x;
      } else {
        T* coef = which == 0 ? coef_k : coef_v;
        store_elem(coef, (int64_t)b * cap * R + tiled_offset(append_row, r, R), x);
      }
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// K0 for the fused step: the same projections as k_prepare in two short
// kernels.  k_project_partial: one workgroup per (64-row chunk of a basis
// group, sequence, basis); thread = latent column of the group, all 64 row
// loads issued before use; fp64 partial sums to the workspace.
// k_project_finish: adds the row-chunk partials in a fixed order and writes
// the query splits, qcoef_out and the appended coefficient row.
// ---------------------------------------------------------------------------
constexpr int kPartRows = 64;

template <typename T>
__global__ __launch_bounds__(256) void k_project_partial(
    const T* __restrict__ q, const T* __restrict__ bases_k, const T* __restrict__ bases_v,
    const T* __restrict__ k_new, const T* __restrict__ v_new, double* __restrict__ partial, int hq, int hkv,
    int dh, int G, int nb, int rank, int R, int bases_shared, int do_query, int nchunk) {
  const int cz = blockIdx.x, b = blockIdx.y, which = blockIdx.z;
  const int t = threadIdx.x;
  const int Dp = hkv * dh, Dg = Dp / nb;
  const int grp = cz / nchunk, ch = cz % nchunk;
  const int d0 = ch * kPartRows;
  const int nrow = min(kPartRows, Dg - d0);
  const T* vec_new = which == 0 ? k_new : v_new;
  const int nq = (which == 0 && do_query) ? G : 0;
  const int nvec = nq + (vec_new ? 1 : 0);
  if (nvec == 0) return;

  __shared__ float xs[kPrepMaxVec][kPartRows];
  const T* bases = (which == 0 ? bases_k : bases_v) + (bases_shared ? 0 : (int64_t)b * Dp * rank) +
                   ((int64_t)grp * Dg + d0) * rank;
  float bv[kPartRows];
  {
    const int tc = min(t, rank - 1);            // every lane loads (threads past rank re-read a column)
#pragma unroll
    for (int i = 0; i < kPartRows; ++i) bv[i] = load_elem(bases, (int64_t)min(i, nrow - 1) * rank + tc);
#pragma unroll
    for (int i = 0; i < kPartRows; ++i) bv[i] = (i < nrow) ? bv[i] : 0.f;
  }
  batched_copy4<8>(
      nvec * kPartRows,
      [&](int i) -> float {
        const int v = i / kPartRows, d = min(i % kPartRows, nrow - 1);   // rows past nrow meet zero bases
        const int dd = grp * Dg + d0 + d;                       // feature index in Dp
        const int64_t oq = ((int64_t)b * hq + (int64_t)(dd / dh) * G + min(v, G - 1)) * dh + dd % dh;
        const int64_t on = (int64_t)b * Dp + dd;
        return (v < nq) ? load_elem(q, oq) : load_elem(vec_new ? vec_new : q, vec_new ? on : oq);
      },
      [&](int i, float x) { xs[i / kPartRows][i % kPartRows] = x; });
  __syncthreads();
  if (t >= rank) return;
  double* out = partial + (((int64_t)(b * 2 + which) * nb * nchunk + cz) * kPrepMaxVec) * R + grp * rank + t;
  for (int v = 0; v < nvec; ++v) {
    double acc = 0.0;
#pragma unroll
    for (int i = 0; i < kPartRows; ++i) acc = fma((double)xs[v][i], (double)bv[i], acc);
    out[(int64_t)v * R] = acc;
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_project_finish(
    const double* __restrict__ partial, const float* __restrict__ qwin_prev, const T* __restrict__ k_new,
    const T* __restrict__ v_new, T* __restrict__ coef_k, T* __restrict__ coef_v, int64_t append_row,
    float* __restrict__ qcoef_out, uint16_t* __restrict__ cq_split, int G, int nb, int rank, int R, int Wq,
    int64_t cap, int do_query, int nchunk) {
  const int b = blockIdx.y, which = blockIdx.z;
  const T* vec_new = which == 0 ? k_new : v_new;
  const int nq = (which == 0 && do_query) ? G : 0;
  const int nvec = nq + (vec_new ? 1 : 0);
  const int i = blockIdx.x * blockDim.x + threadIdx.x;     // (vector, latent column)
  if (which == 0 && do_query && i < G * (Wq - 1) * R) {
    // older FIFO rows come from the caller, fp32, oldest first
    const int r = i % R, gi_old = i / R, g = gi_old / (Wq - 1), k = gi_old % (Wq - 1);
    write_qsplit<T>(cq_split, b, G, Wq, R, g * Wq + k, r,
                    (double)qwin_prev[(((int64_t)b * G + g) * (Wq - 1) + k) * R + r]);
  }
  if (i >= nvec * R) return;
  const int v = i / R, r = i % R, grp = r / rank;
  const double* src = partial + (((int64_t)(b * 2 + which) * nb * nchunk + grp * nchunk) * kPrepMaxVec + v) * R + r;
  double p[16];
  double x = 0.0;
  for (int c0 = 0; c0 < nchunk; c0 += 16) {
#pragma unroll
    for (int c = 0; c < 16; ++c) p[c] = src[(int64_t)min(c0 + c, nchunk - 1) * kPrepMaxVec * R];
#pragma unroll
    for (int c = 0; c < 16; ++c) x += (c0 + c < nchunk) ? p[c] : 0.0;
  }
  if (v < nq) {
    // the current query's coefficients are the newest FIFO row (i = Wq - 1)
    write_qsplit<T>(cq_split, b, G, Wq, R, v * Wq + (Wq - 1), r, x);
    if (qcoef_out) qcoef_out[((int64_t)b * G + v) * R + r] = (float)x;
  } else {
    T* coef = which == 0 ? coef_k : coef_v;
    store_elem(coef, (int64_t)b * cap * R + tiled_offset(append_row, r, R), x);
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

// Loads are unconditional (the tile index is clamped to the last tile of the
// sequence) so the compiler can count outstanding loads exactly and keep the
// prefetched tile in flight while the current one is consumed.
template <typename T, int RB>
__device__ __forceinline__ void load_a_tile(const T* cb, int tile, int ntiles, int col, int kg,
                                            Op8 (&a)[RB][ALoad<T>::kParts]) {
  constexpr int R = RB * kBlkCol;
  const T* tp = cb + (int64_t)min(tile, ntiles - 1) * 16 * R + col * 32 + kg * 8;
#pragma unroll
  for (int kb = 0; kb < RB; ++kb) ALoad<T>::load(tp + kb * 512, a[kb]);
}

template <typename T, int RB>
__global__ __launch_bounds__(256, 2) void k_score_stream(
    const T* __restrict__ coef_k, const uint16_t* __restrict__ cq_split, float* __restrict__ e_out,
    double* __restrict__ run_m, double* __restrict__ run_s, double* __restrict__ wg_stats, int64_t cap, int L,
    int GW, int Wq, int nruns, int runs_per_wave, int nwg, double scale) {
  constexpr int R = RB * kBlkCol;
  constexpr int NP = ALoad<T>::kParts;
  const int b = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 15, kg = lane >> 4;       // MFMA column / k-group of this lane
  const T* cb = coef_k + (int64_t)b * cap * R;

  // B operands (query-coefficient columns, hi/mid/lo bf16 parts) staged once
  // per workgroup in LDS; rows are padded by 16 bytes so the 16-byte reads of
  // one MFMA operand hit distinct banks
  constexpr int RS = R + 8;                        // padded row stride (elements)
  __shared__ __align__(16) uint16_t bsh[3][16][RS];
  {
    const uint16_t* cs = cq_split + (int64_t)b * 3 * GW * R;
    constexpr int K8 = R / 8;
    for (int i = threadIdx.x; i < 3 * (16 - GW) * K8; i += blockDim.x) {   // zero columns >= GW
      const int p = i / ((16 - GW) * K8), rem = i % ((16 - GW) * K8);
      *reinterpret_cast<uint4*>(&bsh[p][GW + rem / K8][(rem % K8) * 8]) = make_uint4(0, 0, 0, 0);
    }
    batched_copy16<4>(
        3 * GW * K8,
        [&](int i) { return reinterpret_cast<const uint4*>(cs + (int64_t)(i / K8) * R + (i % K8) * 8); },
        [&](int i) {
          const int pc = i / K8;            // p * GW + c
          return reinterpret_cast<uint4*>(&bsh[pc / GW][pc % GW][(i % K8) * 8]);
        });
    __syncthreads();
  }
  auto bop = [&](int kb, int p) -> Op8 {
    Op8 o;
    o.u = *reinterpret_cast<const uint4*>(&bsh[p][col][kb * 32 + kg * 8]);
    return o;
  };
  // causal limit of this column's query row (Section 3.2.2): keys l <= L - Wq + i
  const int lim = (col < GW) ? (L - Wq + col % Wq) : -1;
  const int ntiles = (L + 15) / 16;

  const int run0 = (blockIdx.x * kScoreWaves + wave) * runs_per_wave;
  const int run1 = min(run0 + runs_per_wave, nruns);
  const int tile_end = run1 * kRunTiles;
  double Mw = -INFINITY, Sw = 0.0;                 // this wave's running (max, sum) for column col

  Op8 abuf[2][RB][NP];
  load_a_tile<T, RB>(cb, run0 * kRunTiles + 0, ntiles, col, kg, abuf[0]);
  load_a_tile<T, RB>(cb, run0 * kRunTiles + 1, ntiles, col, kg, abuf[1]);
  for (int run = run0; run < run1; ++run) {
    double z[kRunTiles][4];
#pragma unroll
    for (int t = 0; t < kRunTiles; ++t) {
      const int tile = run * kRunTiles + t;
      double acc[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
      for (int kb = 0; kb < RB; ++kb) {
        floatx4 d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int pa = 0; pa < NP; ++pa) {
          d = mfma16x16x32(abuf[t & 1][kb][pa], bop(kb, 0), d);
          d = mfma16x16x32(abuf[t & 1][kb][pa], bop(kb, 1), d);
          d = mfma16x16x32(abuf[t & 1][kb][pa], bop(kb, 2), d);
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[v] += (double)d[v];
      }
      // prefetch two tiles ahead into the buffer just consumed (past the end of
      // this wave's range the load is a harmless re-read of the last tile)
      load_a_tile<T, RB>(cb, min(tile + 2, tile_end - 1), ntiles, col, kg, abuf[t & 1]);
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int tok = tile * 16 + kg * 4 + v;
        z[t][v] = (tile < ntiles && tok <= lim && tok < L) ? acc[v] * scale : -INFINITY;
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
    if (m != -INFINITY) {
      const double mn = fmax(Mw, m);
      Sw = (Mw == -INFINITY ? 0.0 : Sw * exp(Mw - mn)) + s * exp(m - mn);
      Mw = mn;
    }
  }
  // workgroup statistics: the four waves' (max, sum) folded in a fixed order
  __shared__ double wm[kScoreWaves][16], wsum[kScoreWaves][16];
  if (kg == 0) {
    wm[wave][col] = Mw;
    wsum[wave][col] = Sw;
  }
  __syncthreads();
  if (wave == 0 && kg == 0 && col < GW) {
    double M = -INFINITY, S = 0.0;
    for (int w = 0; w < kScoreWaves; ++w) {
      const double mw = wm[w][col];
      if (mw == -INFINITY) continue;
      const double mn = fmax(M, mw);
      S = (M == -INFINITY ? 0.0 : S * exp(M - mn)) + wsum[w][col] * exp(mw - mn);
      M = mn;
    }
    double* ws2 = wg_stats + (((int64_t)b * GW + col) * nwg + blockIdx.x) * 2;
    ws2[0] = M;
    ws2[1] = S;
  }
}

// ---------------------------------------------------------------------------
// K2: relevance A~ and its radix histogram
// ---------------------------------------------------------------------------
// grid (ceil(L / chunk), B), 256 threads.  Every workgroup folds the
// scoring workgroups' statistics into the global (M, S) per query row (the
// same fixed order everywhere), stages the exp values of its chunk plus the
// pooling halo in LDS with independent loads, then pools and aggregates.

__global__ __launch_bounds__(256) void k_relevance(
    const float* __restrict__ e, const double* __restrict__ run_m, const double* __restrict__ wg_stats,
    float* __restrict__ atilde, uint32_t* __restrict__ hist_wg, float* __restrict__ scores_out,
    int64_t cap, int L, int n_hist, int G, int Wq, int kappa, int pool_mode, int agg, int nruns, int nwg,
    int chunk, int64_t hist_stride) {
  const int b = blockIdx.y;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int GW = G * Wq;
  const int h = kappa / 2;
  const int HP = (h + 3) & ~3;                              // halo slot rounded to 16 bytes
  const int SP = chunk + 2 * HP;                            // staged row stride (floats)
  const int t0 = blockIdx.x * chunk;
  const int span = chunk + 2 * h;
  const int x0 = t0 - h;                                    // first staged position
  const int r_first = max(x0, 0) / kRunTok;
  const int r_last = (min(t0 + chunk + h, L) - 1) / kRunTok;
  const int nr = r_last - r_first + 1;
  const int nrc = chunk / kRunTok + 4;                      // run slots per query row

  // dynamic LDS: histogram, per-run factors, (M, S), pooled input, aggregate, exp values
  extern __shared__ __align__(16) unsigned char lds[];
  uint32_t* hl = reinterpret_cast<uint32_t*>(lds);
  double* fac = reinterpret_cast<double*>(hl + kHistBins);  // [GW][nrc]: exp(run max - M) / S
  double* MS = fac + GW * nrc;                              // [GW][2]
  double* aq = MS + 2 * GW;                                 // [chunk + 2h]
  float* e_s = reinterpret_cast<float*>(aq + span + (span & 1));   // [GW][SP]: x at [HP + x - t0]

  // staged exp values: 16-byte loads of the chunk's valid part (t0 is a
  // multiple of 4; rounding L - t0 up to 4 stays below the capacity, a
  // multiple of 16) and 4-byte loads of the halos, all issued before use
  {
    const int c4 = (min(chunk, L - t0) + 3) / 4;
    batched_copy16<8>(
        GW * c4, [&](int i) { return reinterpret_cast<const uint4*>(e + ((int64_t)b * GW + i / c4) * cap + t0) + i % c4; },
        [&](int i) { return reinterpret_cast<uint4*>(e_s + (i / c4) * SP + HP) + i % c4; });
    batched_copy4<2>(
        GW * 2 * h,
        [&](int i) -> float {
          const int gi = i / (2 * h), k = i % (2 * h);
          const int x = (k < h) ? t0 - h + k : t0 + chunk + (k - h);
          return e[((int64_t)b * GW + gi) * cap + min(max(x, 0), L - 1)];   // out-of-range halo is never used
        },
        [&](int i, float v) {
          const int gi = i / (2 * h), k = i % (2 * h);
          const int o = (k < h) ? HP - h + k : HP + chunk + (k - h);
          e_s[gi * SP + o] = v;
        });
  }
  for (int i = t; i < kHistBins; i += blockDim.x) hl[i] = 0;
  // global (M, S) per query row: one wave per row, lanes stride the workgroups
  for (int gi = wave; gi < GW; gi += blockDim.x / 64) {
    const double* st = wg_stats + ((int64_t)b * GW + gi) * nwg * 2;
    double m = -INFINITY;
    for (int i = lane; i < nwg; i += 64) m = fmax(m, st[2 * i]);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m = fmax(m, shfl_xor_d(m, o));
    double sum = 0.0;
    for (int i = lane; i < nwg; i += 64) {
      const double mi = st[2 * i];
      if (mi != -INFINITY) sum += st[2 * i + 1] * exp(mi - m);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) sum += shfl_xor_d(sum, o);
    if (lane == 0) {
      MS[2 * gi] = m;
      MS[2 * gi + 1] = sum;
    }
  }
  __syncthreads();
  for (int i = t; i < GW * nr; i += blockDim.x) {
    const int gi = i / nr, rr = r_first + i % nr;
    const double mr = run_m[((int64_t)b * GW + gi) * nruns + rr];
    fac[gi * nrc + i % nr] = (mr == -INFINITY) ? 0.0 : exp(mr - MS[2 * gi]) / MS[2 * gi + 1];
  }
  __syncthreads();

  // each thread owns kPerThr consecutive output positions; the window mean of
  // every staged position is computed once per group, the pooling reads its
  // kappa window offsets as independent LDS loads, and the group aggregate
  // stays in registers
  constexpr int kPerThr = 8;
  const int own = t * kPerThr;                              // first output (chunk-relative)
  const bool active = own < chunk;
  const int nspan = (span + blockDim.x - 1) / blockDim.x;   // staged positions per thread
  double acc[kPerThr];
#pragma unroll
  for (int j = 0; j < kPerThr; ++j) acc[j] = (agg == S4R_AGG_MEAN) ? 0.0 : -INFINITY;
  const double pad = (pool_mode == S4R_POOL_MAX) ? -INFINITY : 0.0;
  for (int g = 0; g < G; ++g) {
    // window mean over the W_q query rows, on [t0 - h, t0 + chunk + h)
    for (int k0 = 0; k0 < nspan; k0 += 4) {
      double v[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int i = (k0 + q) * blockDim.x + t;
        const int x = x0 + i;
        const bool ok = i < span && x >= 0 && x < L;
        const int ic = min(i, span - 1);                      // clamped: LDS reads stay unguarded
        const int xr = min(max(x, max(x0, 0)), L - 1) / kRunTok - r_first;
        double sum = 0.0;
        for (int wi = 0; wi < Wq; ++wi) {
          const int gi = g * Wq + wi;
          sum += (double)e_s[gi * SP + HP - h + ic] * fac[gi * nrc + xr];
        }
        v[q] = ok ? ((Wq == 1) ? sum : sum / Wq) : pad;
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int i = (k0 + q) * blockDim.x + t;
        if (i < span) aq[i] = v[q];
      }
    }
    __syncthreads();
    if (active) {
      double p[kPerThr];
#pragma unroll
      for (int j = 0; j < kPerThr; ++j) p[j] = (pool_mode == S4R_POOL_MAX) ? -INFINITY : 0.0;
      for (int o = 0; o < kappa; ++o) {
        double w[kPerThr];
#pragma unroll
        for (int j = 0; j < kPerThr; ++j) w[j] = aq[own + j + o];
#pragma unroll
        for (int j = 0; j < kPerThr; ++j) p[j] = (pool_mode == S4R_POOL_MAX) ? fmax(p[j], w[j]) : p[j] + w[j];
      }
#pragma unroll
      for (int j = 0; j < kPerThr; ++j) {
        const double pj = (pool_mode == S4R_POOL_MAX) ? p[j] : p[j] / kappa;
        acc[j] = (agg == S4R_AGG_MEAN) ? acc[j] + pj : fmax(acc[j], pj);
      }
    }
    __syncthreads();
  }
  if (active) {
#pragma unroll
    for (int j = 0; j < kPerThr; ++j) {
      const int x = t0 + own + j;
      if (x >= L) continue;
      const float af = (float)((agg == S4R_AGG_MEAN) ? acc[j] / G : acc[j]);
      atilde[(int64_t)b * cap + x] = af;
      if (scores_out) scores_out[(int64_t)b * L + x] = af;
      if (x < n_hist) atomicAdd(&hl[score_key(af) >> kHistShift], 1u);
    }
  }
  __syncthreads();
  // this workgroup's histogram, written whole (summed by k_hist_reduce)
  uint32_t* hw = hist_wg + ((int64_t)b * hist_stride + blockIdx.x) * kHistBins;
  for (int i = t; i < kHistBins; i += blockDim.x) hw[i] = hl[i];
}

// histogram of caller-provided scores (standalone selection)
__global__ __launch_bounds__(256) void k_hist_scores(const float* __restrict__ scores, uint32_t* __restrict__ hist_wg,
                                                     int L, int n_hist, int64_t hist_stride) {
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
  uint32_t* hw = hist_wg + ((int64_t)b * hist_stride + blockIdx.x) * kHistBins;
  for (int i = threadIdx.x; i < kHistBins; i += blockDim.x) hw[i] = hl[i];
}

// per-workgroup histograms -> one histogram per sequence, fixed summation order
__global__ __launch_bounds__(256) void k_hist_reduce(const uint32_t* __restrict__ hist_wg, uint32_t* __restrict__ hist,
                                                     int ngroups, int64_t hist_stride) {
  const int b = blockIdx.y;
  const int bin = blockIdx.x * blockDim.x + threadIdx.x;
  const uint32_t* hw = hist_wg + (int64_t)b * hist_stride * kHistBins + bin;
  uint32_t sum = 0;
  for (int g0 = 0; g0 < ngroups; g0 += 16) {
    uint32_t v[16];
#pragma unroll
    for (int g = 0; g < 16; ++g) v[g] = hw[(int64_t)min(g0 + g, ngroups - 1) * kHistBins];
#pragma unroll
    for (int g = 0; g < 16; ++g) sum += (g0 + g < ngroups) ? v[g] : 0u;
  }
  hist[(int64_t)b * kHistBins + bin] = sum;
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
  (void)clear;
  dim3 grid(P.R / 16, P.B, 2);
  if (P.dtype == S4R_BF16)
    hipLaunchKernelGGL(k_prepare<uint16_t>, grid, dim3(256), 0, st, (const uint16_t*)q, qwin_prev,
                       (const uint16_t*)bases_k, (const uint16_t*)bases_v, (const uint16_t*)k_new,
                       (const uint16_t*)v_new, (uint16_t*)coef_k, (uint16_t*)coef_v, append_row, qcoef_out,
                       ws.cq_split, P.hq, P.hkv, P.dh, P.G, P.nb, P.rank, P.R, P.Wq, P.bases_shared, P.cap,
                       (int)do_query);
  else
    hipLaunchKernelGGL(k_prepare<float>, grid, dim3(256), 0, st, (const float*)q, qwin_prev,
                       (const float*)bases_k, (const float*)bases_v, (const float*)k_new, (const float*)v_new,
                       (float*)coef_k, (float*)coef_v, append_row, qcoef_out, ws.cq_split, P.hq, P.hkv, P.dh,
                       P.G, P.nb, P.rank, P.R, P.Wq, P.bases_shared, P.cap, (int)do_query);
  return hipGetLastError();
}

hipError_t launch_project(const Problem& P, const Workspace& ws, const void* q, const float* qwin_prev,
                          const void* bases_k, const void* bases_v, const void* k_new, const void* v_new,
                          void* coef_k, void* coef_v, int64_t append_row, float* qcoef_out, hipStream_t st) {
  const int nchunk = (P.Dg + kPartRows - 1) / kPartRows;
  dim3 g1(P.nb * nchunk, P.B, 2);
  const int nfin = std::max(kPrepMaxVec * P.R, P.G * std::max(P.Wq - 1, 0) * P.R);
  dim3 g2((nfin + 255) / 256, P.B, 2);
  if (P.dtype == S4R_BF16) {
    hipLaunchKernelGGL(k_project_partial<uint16_t>, g1, dim3(256), 0, st, (const uint16_t*)q, (const uint16_t*)bases_k,
                       (const uint16_t*)bases_v, (const uint16_t*)k_new, (const uint16_t*)v_new, ws.proj_partial,
                       P.hq, P.hkv, P.dh, P.G, P.nb, P.rank, P.R, P.bases_shared, 1, nchunk);
    hipLaunchKernelGGL(k_project_finish<uint16_t>, g2, dim3(256), 0, st, ws.proj_partial, qwin_prev,
                       (const uint16_t*)k_new, (const uint16_t*)v_new, (uint16_t*)coef_k, (uint16_t*)coef_v,
                       append_row, qcoef_out, ws.cq_split, P.G, P.nb, P.rank, P.R, P.Wq, P.cap, 1, nchunk);
  } else {
    hipLaunchKernelGGL(k_project_partial<float>, g1, dim3(256), 0, st, (const float*)q, (const float*)bases_k,
                       (const float*)bases_v, (const float*)k_new, (const float*)v_new, ws.proj_partial, P.hq,
                       P.hkv, P.dh, P.G, P.nb, P.rank, P.R, P.bases_shared, 1, nchunk);
    hipLaunchKernelGGL(k_project_finish<float>, g2, dim3(256), 0, st, ws.proj_partial, qwin_prev,
                       (const float*)k_new, (const float*)v_new, (float*)coef_k, (float*)coef_v, append_row,
                       qcoef_out, ws.cq_split, P.G, P.nb, P.rank, P.R, P.Wq, P.cap, 1, nchunk);
  }
  return hipGetLastError();
}

// runs per wave and scoring workgroups per sequence for a given length: aim at
// about three resident waves per SIMD over the whole batch
static int runs_per_wave(const Problem& P, int64_t L) {
  const int64_t nruns = (L + kRunTok - 1) / kRunTok;
  const int64_t waves = 3 * 1024;
  return (int)std::max<int64_t>(1, (P.B * nruns + waves - 1) / waves);
}

int score_workgroups(const Problem& P, int64_t L) {
  const int64_t nruns = (L + kRunTok - 1) / kRunTok;
  const int rpw = runs_per_wave(P, L);
  return (int)((nruns + rpw * kScoreWaves - 1) / (rpw * kScoreWaves));
}

template <typename T, int RB>
static void launch_stream_t(const Problem& P, const Workspace& ws, int64_t L, const void* coef_k, hipStream_t st) {
  const int nruns = (int)((L + kRunTok - 1) / kRunTok);
  const int rpw = runs_per_wave(P, L);
  const int nwg = score_workgroups(P, L);
  hipLaunchKernelGGL((k_score_stream<T, RB>), dim3(nwg, P.B), dim3(256), 0, st, (const T*)coef_k, ws.cq_split,
                     ws.e, ws.run_m, ws.run_s, ws.wg_stats, P.cap, (int)L, P.GW, P.Wq, nruns, rpw, nwg,
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

int relevance_chunk(int GW) { return GW <= 4 ? 2048 : (GW <= 8 ? 1024 : 512); }

size_t relevance_lds(int GW, int chunk, int kappa) {
  const int h = kappa / 2;
  const int span = chunk + 2 * h;
  const int SP = chunk + 2 * ((h + 3) & ~3);
  const int nrc = chunk / kRunTok + 4;
  return kHistBins * 4 + (size_t)(GW * nrc + 2 * GW + span + 1) * 8 + (size_t)GW * SP * 4 + 16;
}

hipError_t launch_relevance(const Problem& P, const Workspace& ws, int64_t L, float* scores_out, hipStream_t st) {
  const int n_hist = (int)std::max<int64_t>(L - P.W, 0);
  const int nruns = (int)((L + kRunTok - 1) / kRunTok);
  const int chunk = relevance_chunk(P.GW);
  const size_t lds = relevance_lds(P.GW, chunk, P.kappa);
  dim3 grid((unsigned)((L + chunk - 1) / chunk), P.B);
  hipLaunchKernelGGL(k_relevance, grid, dim3(256), lds, st, ws.e, ws.run_m, ws.wg_stats, ws.atilde, ws.hist_wg,
                     scores_out, P.cap, (int)L, n_hist, P.G, P.Wq, P.kappa, P.pool_mode, P.agg, nruns,
                     score_workgroups(P, L), chunk, rel_groups_max(P));
  return launch_hist_reduce(P, ws, (int)grid.x, st);
}

hipError_t launch_hist_reduce(const Problem& P, const Workspace& ws, int ngroups, hipStream_t st) {
  hipLaunchKernelGGL(k_hist_reduce, dim3(kHistBins / 256, P.B), dim3(256), 0, st, ws.hist_wg, ws.hist, ngroups,
                     rel_groups_max(P));
  return hipGetLastError();
}

hipError_t launch_hist_only(const Problem& P, const Workspace& ws, int64_t L, const float* scores, hipStream_t st) {
  const int n_hist = (int)std::max<int64_t>(L - P.W, 0);
  const int ng = std::max(1, (n_hist + kHistChunk - 1) / kHistChunk);
  hipLaunchKernelGGL(k_hist_scores, dim3(ng, P.B), dim3(256), 0, st, scores, ws.hist_wg, (int)L, n_hist,
                     rel_groups_max(P));
  return launch_hist_reduce(P, ws, ng, st);
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
