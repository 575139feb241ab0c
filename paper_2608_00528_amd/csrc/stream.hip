// Section 3.2.2 latent logits on gfx950: k_score_stream streams C^K once (the
// HBM-bound pass), Z = C^Q C^K^T / sqrt(R) on bf16 MFMA with per-block fp64
// accumulation, and writes exp(z - run max), per-run (max, sum) and
// per-workgroup (max, sum) statistics of the softmax over the length.
#include "s4r_device.h"
#include "s4r_internal.h"

namespace s4r {

// ---------------------------------------------------------------------------
// K1: the coefficient stream
// ---------------------------------------------------------------------------
// grid (workgroups per sequence, B), 256 threads = 4 waves.  A wave owns a
// contiguous range of 16-token tiles; each 16x32 block of C^K is one
// coalesced 1 KiB wave load that lands directly in MFMA A-operand layout, and
// four tiles (bf16) are in flight per wave.  The B operand holds the
// query-coefficient columns (G*W_q <= 16), as hi, mid and lo bf16 parts
// accumulated into the same fp32 MFMA result, which is folded into fp64
// after every 32-column block.  Each tile's exp values are taken against the
// wave's running maximum of z (recorded per tile), so no z outlives its tile.

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
    const T* __restrict__ coef_k, const double* __restrict__ qpart, const float* __restrict__ qwin_prev,
    float* __restrict__ qcoef_out, float* __restrict__ e_out, double* __restrict__ run_m,
    double* __restrict__ wg_stats, int64_t cap, int L, int G, int Wq, int nch, int ntiles_cap, int tiles_per_wave,
    int nwg, double scale) {
  constexpr int R = RB * kBlkCol;
  constexpr int NP = ALoad<T>::kParts;
  const int b = blockIdx.y;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int col = lane & 15, kg = lane >> 4;       // MFMA column / k-group of this lane
  const int GW = G * Wq;
  const T* cb = coef_k + (int64_t)b * cap * R;
  const int ntiles = (L + 15) / 16;

  // this wave's tiles; the count is a multiple of the prefetch depth and tiles
  // past the sequence are computed on a clamped tile and masked.  The first
  // tiles are requested before the query coefficients are prepared.
  // tiles in flight per wave, as many as fit in 256 registers without spilling
  constexpr int PF = (NP == 1) ? (RB <= 6 ? 4 : 2) : (RB <= 3 ? 2 : 1);
  const int tile0 = (blockIdx.x * kScoreWaves + wave) * tiles_per_wave;
  const int tile1 = min(tile0 + tiles_per_wave, ntiles);
  Op8 abuf[PF][RB][NP];
#pragma unroll
  for (int p = 0; p < PF; ++p) load_a_tile<T, RB>(cb, min(tile0 + p, tile1 - 1), ntiles, col, kg, abuf[p]);

  // B operands: column gi = g * Wq + i holds query-coefficient row i of group
  // g (oldest first).  The newest row is the sum of the projection's row-chunk
  // partials (fixed order); older rows come from the caller.  Each value is
  // split into hi, mid and lo bf16 parts, staged once per workgroup in LDS;
  // rows are padded by 16 bytes so the 16-byte reads of one MFMA operand hit
  // distinct banks.
  constexpr int RS = R + 8;                        // padded row stride (elements)
  __shared__ __align__(16) uint16_t bsh[3][16][RS];
  {
    constexpr int K8 = R / 8;
    for (int i = t; i < 3 * 16 * K8; i += blockDim.x) {   // zero columns >= GW
      const int p = i / (16 * K8), c = (i / K8) % 16;
      if (c >= GW) *reinterpret_cast<uint4*>(&bsh[p][c][(i % K8) * 8]) = make_uint4(0, 0, 0, 0);
    }
    const double* qp = qpart + (int64_t)b * nch * G * R;
    // older rows from the caller; with W_q = 1 there are none and the load
    // below re-reads a partial sum (unused) so it needs no branch
    const float* qw = (Wq > 1) ? qwin_prev + (int64_t)b * G * (Wq - 1) * R : reinterpret_cast<const float*>(qp);
    for (int i0 = 0; i0 < GW * R; i0 += 2 * (int)blockDim.x) {
      double part[2][kQMaxChunks];
      float old[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int i = min(i0 + u * (int)blockDim.x + t, GW * R - 1);
        const int gi = i / R, r = i % R, g = gi / Wq, wi = gi % Wq;
#pragma unroll
        for (int c = 0; c < kQMaxChunks; ++c) part[u][c] = qp[((int64_t)min(c, nch - 1) * G + g) * R + r];
        old[u] = qw[(Wq > 1) ? ((int64_t)g * (Wq - 1) + min(wi, Wq - 2)) * R + r : 0];
      }
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int i = i0 + u * (int)blockDim.x + t;
        if (i >= GW * R) break;
        const int gi = i / R, r = i % R, g = gi / Wq, wi = gi % Wq;
        double x = part[u][0];
#pragma unroll
        for (int c = 1; c < kQMaxChunks; ++c)
          if (c < nch) x += part[u][c];
        if (wi < Wq - 1) x = (double)old[u];
        const Split3 sp = split3(x);
        bsh[0][gi][r] = sp.hi;
        bsh[1][gi][r] = sp.mid;
        bsh[2][gi][r] = sp.lo;
        if (qcoef_out && blockIdx.x == 0 && wi == Wq - 1) qcoef_out[((int64_t)b * G + g) * R + r] = (float)x;
      }
    }
    __syncthreads();
  }
  auto bop = [&](int kb, int p) -> Op8 {
    Op8 o;
    o.u = *reinterpret_cast<const uint4*>(&bsh[p][col][kb * 32 + kg * 8]);
    return o;
  };
  // causal limit of this column's query row (Section 3.2.2): keys l <= L - Wq + i
  const int lim = (col < GW) ? (L - Wq + col % Wq) : -1;

  double Mw = -INFINITY, Sw = 0.0;                 // running (max, sum) of column col over this wave's tiles
  for (int tb = tile0; tb < tile1; tb += PF) {
#pragma unroll
    for (int p = 0; p < PF; ++p) {
      const int tile = tb + p;
      double acc[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
      for (int kb = 0; kb < RB; ++kb) {
        floatx4 d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int pa = 0; pa < NP; ++pa) {
          d = mfma16x16x32(abuf[p][kb][pa], bop(kb, 0), d);
          d = mfma16x16x32(abuf[p][kb][pa], bop(kb, 1), d);
          d = mfma16x16x32(abuf[p][kb][pa], bop(kb, 2), d);
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[v] += (double)d[v];
      }
      // prefetch PF tiles ahead into the buffer just consumed (past the end of
      // this wave's range the load is a harmless re-read of its last tile)
      load_a_tile<T, RB>(cb, min(tile + PF, tile1 - 1), ntiles, col, kg, abuf[p]);
      double z[4];
      double m = -INFINITY;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int tok = tile * 16 + kg * 4 + v;
        z[v] = (tile < tile1 && tok <= lim && tok < L) ? acc[v] * scale : -INFINITY;
        m = fmax(m, z[v]);
      }
      // tile maximum of this column (lanes col, col+16, col+32, col+48); the
      // tile's exp values are taken against the running maximum, which is the
      // reference recorded for the tile
      m = fmax(m, shfl_xor_d(m, 16));
      m = fmax(m, shfl_xor_d(m, 32));
      const double ref = fmax(Mw, m);
      float ev[4];
      double s = 0.0;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        ev[v] = (z[v] == -INFINITY) ? 0.f : expf((float)(z[v] - ref));
        s += (double)ev[v];
      }
      s += shfl_xor_d(s, 16);
      s += shfl_xor_d(s, 32);
      if (col < GW && tile < tile1) {
        float* dst = e_out + ((int64_t)b * GW + col) * cap + (int64_t)tile * 16 + kg * 4;
        *reinterpret_cast<float4*>(dst) = make_float4(ev[0], ev[1], ev[2], ev[3]);
        if (kg == 0) run_m[((int64_t)b * GW + col) * ntiles_cap + tile] = ref;
      }
      if (ref > Mw && Mw != -INFINITY) Sw *= exp(Mw - ref);   // the running maximum grew
      Sw += s;
      Mw = ref;
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


// every workgroup gets the same number of tiles (a multiple of the prefetch
// depth), sized so the whole grid is about one round of 2 workgroups (8 waves)
// per CU on the 256 CUs
static int tiles_per_wave(const Problem& P, int64_t L) {
  const int64_t ntiles = (L + kTileTok - 1) / kTileTok;
  const int64_t waves = 256 * 2 * kScoreWaves;
  const int64_t t = std::max<int64_t>(1, (P.B * ntiles + waves - 1) / waves);
  return (int)((t + 3) / 4 * 4);
}

int score_workgroups(const Problem& P, int64_t L) {
  const int64_t ntiles = (L + kTileTok - 1) / kTileTok;
  const int tpw = tiles_per_wave(P, L);
  return (int)((ntiles + tpw * kScoreWaves - 1) / (tpw * kScoreWaves));
}

template <typename T, int RB>
static void launch_stream_t(const Problem& P, const Workspace& ws, int64_t L, const void* coef_k,
                            const float* qwin_prev, float* qcoef_out, hipStream_t st) {
  const int tpw = tiles_per_wave(P, L);
  const int nwg = score_workgroups(P, L);
  hipLaunchKernelGGL((k_score_stream<T, RB>), dim3(nwg, P.B), dim3(256), 0, st, (const T*)coef_k, ws.qpart,
                     qwin_prev, qcoef_out, ws.e, ws.run_m, ws.wg_stats, P.cap, (int)L, P.G, P.Wq, project_chunks(P),
                     (int)(P.cap / kTileTok), tpw, nwg, 1.0 / sqrt((double)P.R));
}

template <typename T>
static bool dispatch_rb(const Problem& P, const Workspace& ws, int64_t L, const void* coef_k, const float* qwin_prev,
                        float* qcoef_out, hipStream_t st) {
  switch (P.R / 32) {
    case 1: launch_stream_t<T, 1>(P, ws, L, coef_k, qwin_prev, qcoef_out, st); return true;
    case 2: launch_stream_t<T, 2>(P, ws, L, coef_k, qwin_prev, qcoef_out, st); return true;
    case 3: launch_stream_t<T, 3>(P, ws, L, coef_k, qwin_prev, qcoef_out, st); return true;
    case 4: launch_stream_t<T, 4>(P, ws, L, coef_k, qwin_prev, qcoef_out, st); return true;
    case 5: launch_stream_t<T, 5>(P, ws, L, coef_k, qwin_prev, qcoef_out, st); return true;
    case 6: launch_stream_t<T, 6>(P, ws, L, coef_k, qwin_prev, qcoef_out, st); return true;
    case 7: launch_stream_t<T, 7>(P, ws, L, coef_k, qwin_prev, qcoef_out, st); return true;
    case 8: launch_stream_t<T, 8>(P, ws, L, coef_k, qwin_prev, qcoef_out, st); return true;
    default: return false;
  }
}

hipError_t launch_score_stream(const Problem& P, const Workspace& ws, int64_t L, const void* coef_k,
                               const float* qwin_prev, float* qcoef_out, hipStream_t st) {
  bool ok = P.dtype == S4R_BF16 ? dispatch_rb<uint16_t>(P, ws, L, coef_k, qwin_prev, qcoef_out, st)
                                : dispatch_rb<float>(P, ws, L, coef_k, qwin_prev, qcoef_out, st);
  if (!ok) return hipErrorInvalidValue;
  return hipGetLastError();
}


}  // namespace s4r
