// Dense GQA decode attention over an uncompressed bf16 KV cache: the "Full
// KV" baseline the paper compares S^4R against (Section 4.2, Table
// "efficiency"; the full attention term of Appendix B.1), built here so the
// two are measured on the same GPU.  Keys are stored after RoPE, as a plain KV
// cache holds them; the query is rotated at its position N - 1.
//
// Split-K flash decode, HBM-bound (2 B of K plus 2 B of V per cached element):
// grid (split, KV head j, sequence b), 4 waves.  A wave walks the 16-token
// tiles t0 + w, t0 + w + 4, ... of its split with the next tile's K and V
// loads in flight while the current one is consumed:
//   logits  bf16 MFMA 16x16x32: A = the rotated query's hi / lo bf16 parts in
//           rows 4 h + part, B = the key rows as loaded (lane: token l % 16,
//           dims 8 (l / 16) .. + 7 of a 32-dim block), 4 MFMAs per tile, so
//           lane (token t, k-group h) receives head h's logit of token t;
//   softmax online per (token slot, head), one running maximum per head;
//   P V     on the VALU: P and the rescale factors go through the wave's own
//           LDS slice; lane (dim group g, token phase s) owns dims 8 g .. + 7
//           of tokens s, s + 4, s + 8, s + 12 of every tile (16-byte value
//           loads, 256 contiguous bytes per token row across 16 lanes).
// The four waves' (max, sum, output) are merged in LDS and written as the
// split's partial; k_attn_combine merges the splits.
#include "attn_common.h"

namespace s4r {

constexpr int kDenseWaves = 4;
constexpr int kDenseDh = 128;

template <int NMH>
__global__ __launch_bounds__(kDenseWaves * 64) void k_dense_decode(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc, const uint16_t* __restrict__ vc,
    float* __restrict__ part_ml, float* __restrict__ part_o, int N, int tps, int G, int hq, int hkv, int64_t cap,
    double rope_ratio) {
  constexpr int DH = kDenseDh;
  constexpr int NH = 4 * NMH;                      // head slots (heads >= G stay empty)
  const int split = blockIdx.x, j = blockIdx.y, b = blockIdx.z;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int slot = lane & 15, kg = lane >> 4;      // logits: token slot / head within a row group
  const int dg = lane & 15, ts = lane >> 4;        // P V: dim group / token phase
  const int Dp = hkv * DH;
  const int ntile = (N + 15) / 16;
  const int tile0 = split * tps, tile1 = min(tile0 + tps, ntile);

  __shared__ float qrot[NH][DH];
  __shared__ float pw[kDenseWaves][16][NH];        // P of the wave's current tile
  __shared__ float aw[kDenseWaves][NH];            // rescale factor per head
  __shared__ float wm[kDenseWaves][NH], wl[kDenseWaves][NH];
  __shared__ float wo[kDenseWaves][NH][DH];

  // ---- rotated query of every head of the group (fp32, LDS) ----------------------------
  for (int i = t; i < NH * (DH / 2); i += kDenseWaves * 64) {
    const int h = i / (DH / 2), d = i % (DH / 2);
    float xl = 0.f, xh = 0.f;
    if (h < G) {
      const uint16_t* qp = q + ((int64_t)b * hq + (int64_t)j * G + h) * DH;
      xl = bf16_bits_to_f32(qp[d]);
      xh = bf16_bits_to_f32(qp[d + DH / 2]);
    }
    uint64_t F[4];
    rope_freqs_fixed(rope_ratio, d, F);
    float c, s;
    rope_cs_fixed((int64_t)N - 1, F[0], c, s);
    qrot[h][d] = xl * c - xh * s;
    qrot[h][d + DH / 2] = xh * c + xl * s;
  }
  __syncthreads();
  // A operands: row slot = 4 h + part of row group mh, k = dims kb * 32 + 8 kg .. + 7
  Op8 aq[NMH][DH / 32];
#pragma unroll
  for (int mh = 0; mh < NMH; ++mh)
#pragma unroll
    for (int kb = 0; kb < DH / 32; ++kb) {
      const int h = 4 * mh + (slot >> 2), part = slot & 3;
      Op8 hi, lo;
      split2_f32x8(&qrot[h][kb * 32 + 8 * kg], hi, lo);
      aq[mh][kb].u = part == 0 ? hi.u : (part == 1 ? lo.u : make_uint4(0, 0, 0, 0));
    }

  const uint16_t* kb_ = kc + (int64_t)b * cap * Dp + (int64_t)j * DH;
  const uint16_t* vb_ = vc + (int64_t)b * cap * Dp + (int64_t)j * DH;
  auto load_tile = [&](int tile, uint4 (&kk)[DH / 32], uint4 (&vv)[4]) __attribute__((always_inline)) {
    const int n0 = tile * 16;
    const int64_t rk = min(n0 + slot, N - 1);
#pragma unroll
    for (int kb = 0; kb < DH / 32; ++kb) kk[kb] = *reinterpret_cast<const uint4*>(kb_ + rk * Dp + kb * 32 + 8 * kg);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t rv = min(n0 + ts + 4 * i, N - 1);
      vv[i] = *reinterpret_cast<const uint4*>(vb_ + rv * Dp + 8 * dg);
    }
  };

  const float inv_sqrt_d = 1.0f / sqrtf((float)DH);
  float Mrun[NMH], lrun[NMH];
  float o[NH][8];
#pragma unroll
  for (int mh = 0; mh < NMH; ++mh) {
    Mrun[mh] = -INFINITY;
    lrun[mh] = 0.f;
  }
#pragma unroll
  for (int h = 0; h < NH; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) o[h][e] = 0.f;

  uint4 kk[DH / 32], vv[4];
  int tile = tile0 + w;
  if (tile < tile1) load_tile(tile, kk, vv);
  for (; tile < tile1; tile += kDenseWaves) {
    uint4 kn[DH / 32], vn[4];
    const bool more = tile + kDenseWaves < tile1;
    if (more) load_tile(tile + kDenseWaves, kn, vn);
    const int n0 = tile * 16;
    // logits of the tile
#pragma unroll
    for (int mh = 0; mh < NMH; ++mh) {
      floatx4 dl = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < DH / 32; ++kb) {
        Op8 bk;
        bk.u = kk[kb];
        dl = mfma16x16x32(aq[mh][kb], bk, dl);
      }
      const bool valid = n0 + slot < N && 4 * mh + kg < G;
      const float s = valid ? (dl[0] + dl[1]) * inv_sqrt_d : -INFINITY;
      const float pmax = slot_max16(s);
      float alpha = 1.f;
      if (pmax > Mrun[mh]) {                        // uniform within the row of head kg
        alpha = __expf(Mrun[mh] - pmax);            // 0 when the maximum was -inf
        lrun[mh] *= alpha;
        Mrun[mh] = pmax;
      }
      const float p = valid ? __expf(s - Mrun[mh]) : 0.f;
      lrun[mh] += p;
      pw[w][slot][4 * mh + kg] = p;
      if (slot == 0) aw[w][4 * mh + kg] = alpha;
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_s_waitcnt(0xC07F);             // this wave's LDS writes are done
    __builtin_amdgcn_wave_barrier();
    // rescale, then P V for tokens ts, ts + 4, ts + 8, ts + 12
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      const float a = aw[w][h];
#pragma unroll
      for (int e = 0; e < 8; ++e) o[h][e] *= a;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int tk = ts + 4 * i;
      float vf[8];
      const uint32_t vw[4] = {vv[i].x, vv[i].y, vv[i].z, vv[i].w};
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) {
        vf[2 * e2] = __uint_as_float(vw[e2] << 16);
        vf[2 * e2 + 1] = __uint_as_float(vw[e2] & 0xFFFF0000u);
      }
#pragma unroll
      for (int h = 0; h < NH; ++h) {
        const float ph = pw[w][tk][h];
#pragma unroll
        for (int e = 0; e < 8; ++e) o[h][e] = fmaf(ph, vf[e], o[h][e]);
      }
    }
    __builtin_amdgcn_wave_barrier();               // P of this tile read before the next overwrites it
    if (more) {
#pragma unroll
      for (int kb = 0; kb < DH / 32; ++kb) kk[kb] = kn[kb];
#pragma unroll
      for (int i = 0; i < 4; ++i) vv[i] = vn[i];
    }
  }

  // ---- the wave's state: sums over token slots and token phases ------------------------
#pragma unroll
  for (int mh = 0; mh < NMH; ++mh) {
    const float ls = slot_sum16(lrun[mh]);
    if (slot == 0) {
      wm[w][4 * mh + kg] = Mrun[mh];
      wl[w][4 * mh + kg] = ls;
    }
  }
#pragma unroll
  for (int h = 0; h < NH; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float x = o[h][e];
      x += shfl_xor_f(x, 16);
      x += shfl_xor_f(x, 32);
      o[h][e] = x;
    }
  if (ts == 0) {
#pragma unroll
    for (int h = 0; h < NH; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) wo[w][h][8 * dg + e] = o[h][e];
  }
  __syncthreads();
  // ---- merge the four waves into the split's partial -----------------------------------
  for (int i = t; i < G * DH; i += kDenseWaves * 64) {
    const int h = i / DH, d = i % DH;
    float M = -INFINITY;
#pragma unroll
    for (int ww = 0; ww < kDenseWaves; ++ww) M = fmaxf(M, wm[ww][h]);
    float l = 0.f, acc = 0.f;
#pragma unroll
    for (int ww = 0; ww < kDenseWaves; ++ww) {
      const float a = (wm[ww][h] == -INFINITY) ? 0.f : __expf(wm[ww][h] - M);
      l += a * wl[ww][h];
      acc += a * wo[ww][h][d];
    }
    const int64_t pb = ((int64_t)b * hq + (int64_t)j * G + h) * kMaxSplit + split;
    part_o[pb * DH + d] = acc;
    if (d == 0) {
      part_ml[pb * 2 + 0] = M;
      part_ml[pb * 2 + 1] = l;
    }
  }
}

hipError_t launch_combine_only(const Problem& P, const Workspace& ws, int64_t L, int nsplit, const void* q, float* out,
                               hipStream_t st);

hipError_t launch_dense_decode(const Problem& P, const Workspace& ws, int64_t N, const void* q, const void* k_cache,
                               const void* v_cache, float* out, hipStream_t st) {
  const int ntile = (int)((N + 15) / 16);
  // about four workgroups per CU, at most kMaxSplit splits, at least one tile per wave
  int nsplit = (4 * 256 + P.B * P.hkv - 1) / (P.B * P.hkv);
  nsplit = std::max(1, std::min({nsplit, kMaxSplit, (ntile + kDenseWaves - 1) / kDenseWaves}));
  const int tps = (ntile + nsplit - 1) / nsplit;
  nsplit = (ntile + tps - 1) / tps;
  dim3 grid(nsplit, P.hkv, P.B);
  if (P.G > 4)
    hipLaunchKernelGGL(k_dense_decode<2>, grid, dim3(kDenseWaves * 64), 0, st, (const uint16_t*)q,
                       (const uint16_t*)k_cache, (const uint16_t*)v_cache, ws.part_ml, ws.part_o, (int)N, tps, P.G,
                       P.hq, P.hkv, P.cap, rope_ratio(P));
  else
    hipLaunchKernelGGL(k_dense_decode<1>, grid, dim3(kDenseWaves * 64), 0, st, (const uint16_t*)q,
                       (const uint16_t*)k_cache, (const uint16_t*)v_cache, ws.part_ml, ws.part_o, (int)N, tps, P.G,
                       P.hq, P.hkv, P.cap, rope_ratio(P));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_combine_only(P, ws, N, nsplit, q, out, st);
}

}  // namespace s4r
