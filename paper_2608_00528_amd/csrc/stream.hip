// Section 3.2.2 latent logits on gfx950: k_score_stream streams C^K once (the
// HBM-bound pass), Z = C^Q C^K^T / sqrt(R) on bf16 MFMA with per-block fp64
// accumulation, and writes exp(z - running max) per token, the running max
// per 16-token tile and per-workgroup (max, sum) statistics of the softmax
// over the length.
#include "s4r_device.h"
#include "s4r_internal.h"

namespace s4r {

// ---------------------------------------------------------------------------
// K1: the coefficient stream
// ---------------------------------------------------------------------------
// grid (workgroups per sequence, B) with one block of query columns, else a
// 1-D grid over (token range, column block); 256 threads = 4 waves.  A wave
// owns a contiguous range of 16-token tiles; a workgroup scores them against
// one block of up to 16 query columns (more than one block only when
// G * W_q > 16, the blocks re-reading the tiles from L2 / MALL).  Each 16x32
// block of C^K is one coalesced 1 KiB wave load that is used directly as the
// B operand of a 16x16x32 bf16 MFMA (lane l: token l%16, latent columns
// 8*(l/16)..+7).  The A operand holds the query-coefficient columns, four per
// MFMA, each as its hi / mid / lo bf16 parts in rows 4*c + part (row 4*c + 3
// is zero), as the projection kernel wrote them into the operand image, so lane
// (token t, k-group c) receives the three partial products of query column c
// against token t.  The MFMA rounds once per instruction, like an fp32 sum
// aligned to its largest term; the parts of every 32-column block are folded
// into an fp64 accumulator, so z carries no fp32 accumulation across blocks.
// Each tile's exp values are taken against the running maximum of z over the
// wave's tiles (recorded per tile, fp32) with fp64 argument reduction, and
// the running (max, sum) of every query column is kept per wave.

template <typename T>
struct BLoad;

template <>
struct BLoad<uint16_t> {  // 8 bf16 = one 16-byte streaming load
  static constexpr int kParts = 1;
  __device__ __forceinline__ static void load(const uint16_t* p, Op8 (&a)[1]) {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
    a[0].u = make_uint4(v.x, v.y, v.z, v.w);
  }
};

template <>
struct BLoad<float> {  // 8 fp32 = two 16-byte streaming loads, split into 3 bf16 parts
  static constexpr int kParts = 3;
  __device__ __forceinline__ static void load(const float* p, Op8 (&a)[3]) {
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    const f32x4 u = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
    const f32x4 w = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p + 4));
    const float x[8] = {u.x, u.y, u.z, u.w, w.x, w.y, w.z, w.w};
    split_f32x8(x, a[0], a[1], a[2]);
  }
};

// Loads are unconditional (the tile index is clamped to the last tile of the
// sequence) so the compiler can count outstanding loads exactly and keep the
// prefetched tiles in flight while the current one is consumed.
template <typename T, int RB>
__device__ __forceinline__ void load_b_tile(const T* cb, int tile, int ntiles, int slot, int kg,
                                            Op8 (&a)[RB][BLoad<T>::kParts]) {
  constexpr int R = RB * kBlkCol;
  const T* tp = cb + (int64_t)min(tile, ntiles - 1) * 16 * R + slot * 32 + kg * 8;
#pragma unroll
  for (int kb = 0; kb < RB; ++kb) BLoad<T>::load(tp + kb * 512, a[kb]);
}

template <typename T, int RB, int NM>
__global__ __launch_bounds__(256, 2) void k_score_stream(
    const T* __restrict__ coef_k, const uint16_t* __restrict__ qimg, float* __restrict__ e_out,
    float* __restrict__ tref, double* __restrict__ wg_stats, int64_t cap, int L, int G, int Wq, int ntiles_cap,
    int tiles_per_wave,
    int nwg, int gwp, int ncb, int B, double scale, Lens lens) {
  constexpr int R = RB * kBlkCol;
  constexpr int NP = BLoad<T>::kParts;
  // work item (token workgroup x of sequence b, column block cb).  One column
  // block: grid (nwg, B).  Several: a 1-D grid in which the column blocks of
  // one token range are 8 ids apart, so they run on one XCD (workgroup id i
  // goes to XCD i % 8) at about the same time and share its L2 copy of the tiles
  int xw, b, cbk;
  if (ncb == 1) {
    xw = blockIdx.x;
    b = blockIdx.y;
    cbk = 0;
  } else {
    const int id = blockIdx.x, rest = id >> 3;
    const int tw = (rest / ncb) * 8 + (id & 7);
    if (tw >= nwg * B) return;                     // padding of the last group of 8
    cbk = rest % ncb;
    b = tw / nwg;
    xw = tw % nwg;
  }
  L = (int)len_of(lens, b, L);                     // this sequence's length (ragged batch)
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int slot = lane & 15, kg = lane >> 4;      // token slot / k-group (= query column within an MFMA)
  const int GW = G * Wq;
  const int c0 = cbk * kColBlk;                    // first query column of this workgroup's block
  const int GWl = min(GW - c0, 4 * NM);            // its columns
  const T* cb = coef_k + (int64_t)b * cap * R;
  const int ntiles = (L + 15) / 16;

  // tiles in flight per wave and whether the A operands stay in registers:
  // as much as fits in 256 registers without spilling
  constexpr bool A_REG = NM * RB * NP <= 10;
  constexpr int PF = (NP == 1) ? ((NM <= 2 && RB * (A_REG ? 1 + NM / 2 : 1) <= 6) ? 4
                                  : (!A_REG ? (RB <= 5 ? 4 : 2) : (NM * RB <= 16 ? 2 : 1)))
                                : ((NM <= 2 && RB <= 3) ? 2 : 1);
  const int tile0 = (xw * kScoreWaves + wave) * tiles_per_wave;
  const int tile1 = min(tile0 + tiles_per_wave, ntiles);

  // A operands: query column gi = g * Wq + i (row i of group g's window, oldest
  // first) sits in MFMA m = gi / 4, rows 4 * (gi % 4) + part, as the bf16
  // parts the projection kernel wrote into the operand image.  Staged once per
  // workgroup in LDS (rows padded by 16 bytes so the 16-byte operand reads of
  // one MFMA hit distinct banks); rows of no query column, and each column's
  // fourth row, are zero.  The image is requested before the coefficient
  // tiles, so it does not queue behind the streaming loads.
  constexpr int K8 = R / 8;                        // 16-byte units per operand row
  constexpr int kQU = (NM * 16 * K8 + 255) / 256;  // units per thread (<= 8)
  const uint4* qi = reinterpret_cast<const uint4*>(qimg + ((int64_t)b * ncb + cbk) * (NM * 16) * R);
  uint4 qv[kQU];
#pragma unroll
  for (int u = 0; u < kQU; ++u) {
    const int i = min(u * 256 + t, NM * 16 * K8 - 1), row = i / K8;   // row = 16 m + 4 c + part
    const bool used = (row & 3) != 3 && (row >> 2) < GWl;
    qv[u] = used ? qi[i] : make_uint4(0, 0, 0, 0);
  }

  // the first tile now, the rest of the prefetch once the query is staged: the
  // two workgroups of a CU then start streaming together (a full prefetch here
  // would queue the second workgroup's first tiles behind the first's)
  Op8 bbuf[PF][RB][NP];
  load_b_tile<T, RB>(cb, min(tile0, tile1 - 1), ntiles, slot, kg, bbuf[0]);

  constexpr int RS = R + 8;
  __shared__ __align__(16) uint16_t qsh[NM][16][RS];
#pragma unroll
  for (int u = 0; u < kQU; ++u) {
    const int i = u * 256 + t;
    if (i < NM * 16 * K8) *reinterpret_cast<uint4*>(&qsh[0][0][0] + (i / K8) * RS + (i % K8) * 8) = qv[u];
  }
  lds_barrier();                                   // the tile requested above stays in flight
#pragma unroll
  for (int p = 1; p < PF; ++p) load_b_tile<T, RB>(cb, min(tile0 + p, tile1 - 1), ntiles, slot, kg, bbuf[p]);
  // the A operands stay in registers when they fit, else they are re-read from LDS
  Op8 areg[A_REG ? NM : 1][A_REG ? RB : 1];
  if constexpr (A_REG) {
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int kb = 0; kb < RB; ++kb) areg[m][kb].u = *reinterpret_cast<const uint4*>(&qsh[m][slot][kb * 32 + kg * 8]);
  }
  // (re-read per tile: `aoff` is redefined by an empty asm statement in every
  // tile iteration, so the reads are not hoisted out of the loop into
  // NM * RB * 4 live registers)
  int aoff = kg * 8;
  auto aop = [&](int m, int kb) -> Op8 {
    if constexpr (A_REG) {
      return areg[m][kb];
    } else {
      Op8 o;
      o.u = *reinterpret_cast<const uint4*>(&qsh[m][slot][kb * 32 + aoff]);
      return o;
    }
  };

  // per query column of this lane (gi = 4 m + kg): causal limit of its query
  // row (Section 3.2.2: keys l <= L - Wq + i) and the running (max, sum)
  int lim[NM];
  float Mrun[NM];
  double Srun[NM];
#pragma unroll
  for (int m = 0; m < NM; ++m) {
    const int gi = c0 + 4 * m + kg;
    lim[m] = (gi < GW) ? (L - Wq + gi % Wq) : -1;
    Mrun[m] = -INFINITY;
    Srun[m] = 0.0;
  }

  for (int tb = tile0; tb < tile1; tb += PF) {
#pragma unroll
    for (int p = 0; p < PF; ++p) {
      const int tile = tb + p;
      if constexpr (!A_REG) asm volatile("" : "+v"(aoff));
      double acc[NM];
#pragma unroll
      for (int m = 0; m < NM; ++m) acc[m] = 0.0;
#pragma unroll
      for (int kb = 0; kb < RB; ++kb) {
#pragma unroll
        for (int m = 0; m < NM; ++m) {
          floatx4 d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int pb = 0; pb < NP; ++pb) d = mfma16x16x32(aop(m, kb), bbuf[p][kb][pb], d);
          acc[m] += (double)d[0] + (double)(d[1] + d[2]);
        }
      }
      // prefetch PF tiles ahead into the buffer just consumed (past the end of
      // this wave's range the load is a harmless re-read of its last tile)
      load_b_tile<T, RB>(cb, min(tile + PF, tile1 - 1), ntiles, slot, kg, bbuf[p]);
      const int tok = tile * 16 + slot;
#pragma unroll
      for (int m = 0; m < NM; ++m) {
        const double z = (tile < tile1 && tok <= lim[m] && tok < L) ? acc[m] * scale : -INFINITY;
        // running maximum over this wave's tiles (all 16 lanes of the row agree)
        const float ref = fmaxf(slot_max16((float)z), Mrun[m]);
        const float ev = (z == -INFINITY) ? 0.f : exp_neg_accurate(z - (double)ref);
        const float ts = slot_sum16(ev);
        // token-major stores: with one column block the wave's tile is one
        // contiguous run of 16 * 4 * NM values (padding columns hold exp(-inf) = 0)
        if (tile < tile1) {
          e_out[((int64_t)b * cap + tok) * gwp + c0 + 4 * m + kg] = ev;
          if (slot == 0) tref[((int64_t)b * ntiles_cap + tile) * gwp + c0 + 4 * m + kg] = ref;
        }
        if (ref > Mrun[m]) {                       // the running maximum grew
          if (Mrun[m] != -INFINITY) Srun[m] *= (double)exp_neg_accurate((double)Mrun[m] - (double)ref);
          Mrun[m] = ref;
        }
        Srun[m] += (double)ts;
      }
    }
  }
  // workgroup statistics: the four waves' (max, sum) folded in a fixed order
  __shared__ double wm[kScoreWaves][kColBlk], wsum[kScoreWaves][kColBlk];
  if (slot == 0) {
#pragma unroll
    for (int m = 0; m < NM; ++m) {
      wm[wave][4 * m + kg] = (double)Mrun[m];
      wsum[wave][4 * m + kg] = Srun[m];
    }
  }
  __syncthreads();
  if (t < GWl) {
    const int col = c0 + t;
    double M = -INFINITY, S = 0.0;
    for (int w = 0; w < kScoreWaves; ++w) {
      const double mw = wm[w][t];
      if (mw == -INFINITY) continue;
      const double mn = fmax(M, mw);
      S = (M == -INFINITY ? 0.0 : S * exp(M - mn)) + wsum[w][t] * exp(mw - mn);
      M = mn;
    }
    double* ws2 = wg_stats + (((int64_t)b * GW + col) * nwg + xw) * 2;
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
  const int64_t t = std::max<int64_t>(1, (P.B * ntiles * col_blocks(P) + waves - 1) / waves);
  return (int)((t + 3) / 4 * 4);
}

int score_workgroups(const Problem& P, int64_t L) {
  const int64_t ntiles = (L + kTileTok - 1) / kTileTok;
  const int tpw = tiles_per_wave(P, L);
  return (int)((ntiles + tpw * kScoreWaves - 1) / (tpw * kScoreWaves));
}

template <typename T, int RB, int NM>
static void launch_stream_nm(const Problem& P, const Workspace& ws, int64_t L, const void* coef_k, hipStream_t st) {
  const int tpw = tiles_per_wave(P, L);
  const int nwg = score_workgroups(P, L);
  const int ncb = col_blocks(P);
  const dim3 grid = ncb == 1 ? dim3(nwg, P.B) : dim3(8 * ncb * ((nwg * P.B + 7) / 8));
  // the scale takes the configured latent width (storage columns past it are zero)
  hipLaunchKernelGGL((k_score_stream<T, RB, NM>), grid, dim3(256), 0, st, (const T*)coef_k, ws.qimg, ws.e,
                     ws.run_m, ws.wg_stats, P.cap, (int)L, P.G, P.Wq, (int)(P.cap / kTileTok), tpw, nwg, gw_padded(P), ncb, P.B, 1.0 / sqrt((double)P.R_cfg), P.lens);
}

template <typename T, int RB>
static void launch_stream_t(const Problem& P, const Workspace& ws, int64_t L, const void* coef_k, hipStream_t st) {
  switch (qimg_mfmas(P)) {                          // the operand image's MFMAs per column block
    case 1: launch_stream_nm<T, RB, 1>(P, ws, L, coef_k, st); break;
    case 2: launch_stream_nm<T, RB, 2>(P, ws, L, coef_k, st); break;
    case 3: launch_stream_nm<T, RB, 3>(P, ws, L, coef_k, st); break;
    default: launch_stream_nm<T, RB, 4>(P, ws, L, coef_k, st); break;
  }
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

hipError_t launch_score_stream(const Problem& P, const Workspace& ws, int64_t L, const void* coef_k, hipStream_t st) {
  bool ok = P.dtype == S4R_BF16 ? dispatch_rb<uint16_t>(P, ws, L, coef_k, st)
                                : dispatch_rb<float>(P, ws, L, coef_k, st);
  if (!ok) return hipErrorInvalidValue;
  return hipGetLastError();
}


}  // namespace s4r
