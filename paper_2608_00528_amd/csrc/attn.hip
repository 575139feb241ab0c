// Sparse reconstruction and final attention of Section 3.2.3 on gfx950.
//
//   k_attn_split  one workgroup per (split, kv head j, sequence).  Wave w owns
//                 the dimension pair blocks {w, w + d_h/32} of head j (16 dims
//                 each, so every RoPE pair (i, i + d_h/2) sits in one lane).
//                 Per 16-token tile of the index list it gathers the selected
//                 coefficient rows (64-byte pieces of the tiled cache) as MFMA
//                 B operands and forms K^T = B^K_j C^T and V^T = B^V_j C^T with
//                 bf16 MFMA (basis rows as A operands, held in registers), so a
//                 lane ends with 8 dims of one token.  RoPE is applied to the
//                 fp32 accumulators, partial logits are summed over the lane's
//                 k-group and across the waves through LDS, and each lane runs
//                 an online softmax for its token slot.  Reconstructed K/V never
//                 leave registers.  The split's (max, sum, output) is written
//                 once after merging the 16 token slots.
//   k_attn_combine one workgroup per (query head, sequence): sink tokens and
//                 the optional exact window KV (full precision, fp32 VALU) and
//                 the merge of all splits into O_t.
//   k_reconstruct / k_sparse_attn: the separately callable reconstruction
//                 (fp32 K^, V^ written out) and attention over given rows.
#include "s4r_device.h"
#include "s4r_internal.h"

namespace s4r {

// RoPE angle of `pos` at frequency index f: returns cos / sin.  The angle is
// pos * theta^(-2f/d_h); it is reduced in fp64 revolutions and evaluated
// with the hardware sine / cosine (argument in revolutions).
__device__ __forceinline__ double rope_rev_freq(float theta, int f, int dh) {
  if (theta == 0.f) return 0.0;
  return exp2(-2.0 * f / dh * log2((double)theta)) * 0.15915494309189535;  // / (2 pi)
}
__device__ __forceinline__ void rope_cs(int64_t pos, double rev_freq, float& c, float& s) {
  double a = (double)pos * rev_freq;
  a -= floor(a);
  const float x = (float)a;
  c = __builtin_amdgcn_cosf(x);
  s = __builtin_amdgcn_sinf(x);
}

// operand loaders: 8 consecutive elements -> bf16 parts
template <typename T>
struct Parts;
template <>
struct Parts<uint16_t> {
  static constexpr int n = 1;
  __device__ __forceinline__ static void load(const uint16_t* p, Op8* o) { o[0].u = *reinterpret_cast<const uint4*>(p); }
};
template <>
struct Parts<float> {
  static constexpr int n = 3;
  __device__ __forceinline__ static void load(const float* p, Op8* o) {
    float x[8];
    *reinterpret_cast<float4*>(&x[0]) = *reinterpret_cast<const float4*>(p);
    *reinterpret_cast<float4*>(&x[4]) = *reinterpret_cast<const float4*>(p + 4);
    split_f32x8(x, o[0], o[1], o[2]);
  }
};

// accumulate A*B over all part pairs whose combined weight is above ~2^-24
template <int NA, int NB>
__device__ __forceinline__ floatx4 mfma_parts(const Op8* a, const Op8* b, floatx4 d) {
#pragma unroll
  for (int i = 0; i < NA; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j)
      if (i + j < 3) d = mfma16x16x32(a[i], b[j], d);
  return d;
}


template <typename T, int RBH, int DH, int G>
__global__ __launch_bounds__(DH * 2) void k_attn_split(
    const T* __restrict__ q, const T* __restrict__ bases_k, const T* __restrict__ bases_v,
    const T* __restrict__ coef_k, const T* __restrict__ coef_v, const int32_t* __restrict__ idx_all,
    int64_t idx_stride, float* __restrict__ part_ml, float* __restrict__ part_o, int n_proc, int nsplit,
    int hq, int hkv, int nb, int rank, int R, int s_sink, int64_t L, int64_t cap, int bases_shared,
    float theta) {
  constexpr int NP = Parts<T>::n;
  constexpr int NWAVE = DH / 32;          // waves per workgroup
  constexpr int HALF_MB = DH / 32;        // pair offset in 16-dim blocks
  const int split = blockIdx.x, j = blockIdx.y, b = blockIdx.z;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int slot = lane & 15, kg = lane >> 4;
  const int Dp = hkv * DH, Dg = Dp / nb;
  const int grp = j / (hkv / nb);
  const int row0 = (j % (hkv / nb)) * DH;          // first basis row of head j in its group
  const int kb0 = grp * rank / 32;                 // first latent block of the group

  // ---- basis operands (A): rows d = 16*mb + slot, k-group kg ------------------
  Op8 ak[2][RBH][NP], av[2][RBH][NP];
  {
    const int64_t boff = (bases_shared ? 0 : (int64_t)b * Dp * rank) + (int64_t)grp * Dg * rank;
#pragma unroll
    for (int hm = 0; hm < 2; ++hm) {
      const int d = 16 * (w + hm * HALF_MB) + slot;
#pragma unroll
      for (int kb = 0; kb < RBH; ++kb) {
        const int64_t o = boff + (int64_t)(row0 + d) * rank + kb * 32 + kg * 8;
        Parts<T>::load(bases_k + o, ak[hm][kb]);
        Parts<T>::load(bases_v + o, av[hm][kb]);
      }
    }
  }
  // ---- rotated query for this lane's 8 dims -------------------------------------
  const int64_t pos_q = s_sink + L - 1;
  double rf[4];
  float qr[G][8];
#pragma unroll
  for (int v = 0; v < 4; ++v) rf[v] = rope_rev_freq(theta, 16 * w + 4 * kg + v, DH);
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    float c, sn;
    rope_cs(pos_q, rf[v], c, sn);
    const int dlo = 16 * w + 4 * kg + v, dhi = dlo + DH / 2;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if (g < G) {
        const int64_t qo = ((int64_t)b * hq + (int64_t)j * G + g) * DH;
        const float xl = load_elem(q, qo + dlo), xh = load_elem(q, qo + dhi);
        qr[g][v] = xl * c - xh * sn;
        qr[g][4 + v] = xh * c + xl * sn;
      }
    }
  }

  // ---- split range ------------------------------------------------------------------
  const int ntile = (n_proc + 15) / 16;
  const int tps = (ntile + nsplit - 1) / nsplit;
  const int tile0 = split * tps, tile1 = min(ntile, tile0 + tps);
  const int32_t* idx = idx_all + (int64_t)b * idx_stride;
  const T* ckb = coef_k + (int64_t)b * cap * R;
  const T* cvb = coef_v + (int64_t)b * cap * R;
  const float inv_sqrt_d = 1.0f / sqrtf((float)DH);

  __shared__ float xlog[2][NWAVE][G][16];

  float mrun[G], lrun[G], oacc[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    mrun[g] = -INFINITY;
    lrun[g] = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) oacc[g][i] = 0.f;
  }

  for (int tile = tile0; tile < tile1; ++tile) {
    const int n = tile * 16 + slot;
    const bool valid = n < n_proc;
    const int64_t tok = valid ? (int64_t)idx[n] : 0;
    // gathered coefficient rows of this token (B operands)
    Op8 bk[RBH][NP], bvv[RBH][NP];
    const int64_t co = (tok >> 4) * 16 * (int64_t)R + (tok & 15) * 32 + kg * 8;
#pragma unroll
    for (int kb = 0; kb < RBH; ++kb) {
      Parts<T>::load(ckb + co + (int64_t)(kb0 + kb) * 512, bk[kb]);
      Parts<T>::load(cvb + co + (int64_t)(kb0 + kb) * 512, bvv[kb]);
    }
    floatx4 dk[2], dv[2];
#pragma unroll
    for (int hm = 0; hm < 2; ++hm) {
      dk[hm] = floatx4{0.f, 0.f, 0.f, 0.f};
      dv[hm] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < RBH; ++kb) {
        dk[hm] = mfma_parts<NP, NP>(ak[hm][kb], bk[kb], dk[hm]);
        dv[hm] = mfma_parts<NP, NP>(av[hm][kb], bvv[kb], dv[hm]);
      }
    }
    // RoPE at the token's original position s + idx
    float kr[8];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      float c, sn;
      rope_cs(s_sink + tok, rf[v], c, sn);
      const float xl = dk[0][v], xh = dk[1][v];
      kr[v] = xl * c - xh * sn;
      kr[4 + v] = xh * c + xl * sn;
    }
    // partial logits over this lane's 8 dims, then over the k-group lanes
    float part[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if (g < G) {
        float a = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) a = fmaf(qr[g][i], kr[i], a);
        a += shfl_xor_f(a, 16);
        a += shfl_xor_f(a, 32);
        part[g] = a;
      }
    }
    const int buf = tile & 1;
    if (kg == 0) {
#pragma unroll
      for (int g = 0; g < G; ++g)
        if (g < G) xlog[buf][w][g][slot] = part[g];
    }
    __syncthreads();
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if (g < G) {
        float sfull = 0.f;
#pragma unroll
        for (int ww = 0; ww < NWAVE; ++ww) sfull += xlog[buf][ww][g][slot];
        const float sc = valid ? sfull * inv_sqrt_d : -INFINITY;
        if (sc != -INFINITY) {
          const float mn = fmaxf(mrun[g], sc);
          const float alpha = __expf(mrun[g] - mn);   // 0 when mrun is -inf
          const float p = __expf(sc - mn);
          lrun[g] = lrun[g] * alpha + p;
          oacc[g][0] = oacc[g][0] * alpha + p * dv[0][0];
          oacc[g][1] = oacc[g][1] * alpha + p * dv[0][1];
          oacc[g][2] = oacc[g][2] * alpha + p * dv[0][2];
          oacc[g][3] = oacc[g][3] * alpha + p * dv[0][3];
          oacc[g][4] = oacc[g][4] * alpha + p * dv[1][0];
          oacc[g][5] = oacc[g][5] * alpha + p * dv[1][1];
          oacc[g][6] = oacc[g][6] * alpha + p * dv[1][2];
          oacc[g][7] = oacc[g][7] * alpha + p * dv[1][3];
          mrun[g] = mn;
        }
      }
    }
  }

  // ---- merge the 16 token slots (lanes with the same k-group) -----------------------
#pragma unroll
  for (int g = 0; g < G; ++g) {
    if (g >= G) continue;
#pragma unroll
    for (int msk = 1; msk < 16; msk <<= 1) {
      const float m2 = shfl_xor_f(mrun[g], msk);
      const float l2 = shfl_xor_f(lrun[g], msk);
      const float mn = fmaxf(mrun[g], m2);
      const float a1 = (mrun[g] == -INFINITY) ? 0.f : __expf(mrun[g] - mn);
      const float a2 = (m2 == -INFINITY) ? 0.f : __expf(m2 - mn);
      lrun[g] = lrun[g] * a1 + l2 * a2;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float o2 = shfl_xor_f(oacc[g][i], msk);
        oacc[g][i] = oacc[g][i] * a1 + o2 * a2;
      }
      mrun[g] = mn;
    }
  }
  if (slot == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if (g >= G) continue;
      const int h = j * G + g;
      const int64_t pb = ((int64_t)b * hq + h) * kMaxSplit + split;
      if (w == 0 && kg == 0) {
        part_ml[pb * 2 + 0] = mrun[g];
        part_ml[pb * 2 + 1] = lrun[g];
      }
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int dlo = 16 * w + 4 * kg + v;
        part_o[pb * DH + dlo] = oacc[g][v];
        part_o[pb * DH + dlo + DH / 2] = oacc[g][4 + v];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// combine: sinks, exact window, splits -> O_t
// ---------------------------------------------------------------------------
constexpr int kMaxExtra = 1024 + 64;   // sinks + exact window rows

template <typename T>
__global__ __launch_bounds__(256) void k_attn_combine(
    const T* __restrict__ q, const T* __restrict__ sink_k, const T* __restrict__ sink_v,
    const T* __restrict__ win_k, const T* __restrict__ win_v, const float* __restrict__ part_ml,
    const float* __restrict__ part_o, float* __restrict__ out, int nsplit, int hq, int hkv, int dh,
    int s_sink, int W, int64_t L, float theta) {
  const int h = blockIdx.x, b = blockIdx.y;
  const int G = hq / hkv, j = h / G;
  const int Dp = hkv * dh;
  const int t = threadIdx.x;
  const int64_t pos_q = s_sink + L - 1;
  const int n_win = win_k ? (int)min<int64_t>(W, L) : 0;
  const int n_extra = s_sink + n_win;

  __shared__ float qr[128];
  __shared__ double rfs[64];
  __shared__ float lg[kMaxExtra];
  __shared__ float red[256];
  __shared__ float s_mx, s_sum;

  if (t < dh / 2) rfs[t] = rope_rev_freq(theta, t, dh);
  if (t < dh / 2) {
    float c, sn;
    rope_cs(pos_q, rfs[t], c, sn);
    const int64_t qo = ((int64_t)b * hq + h) * dh;
    const float xl = load_elem(q, qo + t), xh = load_elem(q, qo + t + dh / 2);
    qr[t] = xl * c - xh * sn;
    qr[t + dh / 2] = xh * c + xl * sn;
  }
  __syncthreads();
  // logits of the full-precision tokens: sinks at positions 0..s-1, exact
  // window rows at s + (L - n_win + w)
  for (int e = t; e < n_extra; e += blockDim.x) {
    const T* kp;
    int64_t pos;
    if (e < s_sink) {
      kp = sink_k + ((int64_t)b * s_sink + e) * Dp + (int64_t)j * dh;
      pos = e;
    } else {
      const int wi = e - s_sink;                       // row of the window block
      kp = win_k + ((int64_t)b * W + (W - n_win) + wi) * Dp + (int64_t)j * dh;
      pos = s_sink + (L - n_win) + wi;
    }
    float acc = 0.f;
    for (int f = 0; f < dh / 2; ++f) {
      float c, sn;
      rope_cs(pos, rfs[f], c, sn);
      const float xl = load_elem(kp, f), xh = load_elem(kp, f + dh / 2);
      acc = fmaf(qr[f], xl * c - xh * sn, acc);
      acc = fmaf(qr[f + dh / 2], xh * c + xl * sn, acc);
    }
    lg[e] = acc / sqrtf((float)dh);
  }
  __syncthreads();
  // max / sum of the extra tokens
  float mx = -INFINITY;
  for (int e = t; e < n_extra; e += blockDim.x) mx = fmaxf(mx, lg[e]);
  red[t] = mx;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (t < o) red[t] = fmaxf(red[t], red[t + o]);
    __syncthreads();
  }
  if (t == 0) s_mx = red[0];
  __syncthreads();
  const float m_e = s_mx;
  float sm = 0.f;
  for (int e = t; e < n_extra; e += blockDim.x) sm += __expf(lg[e] - m_e);
  red[t] = sm;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (t < o) red[t] += red[t + o];
    __syncthreads();
  }
  if (t == 0) s_sum = red[0];
  __syncthreads();
  const float l_e = s_sum;

  // global max over the extra tokens and the splits
  const int64_t pb = ((int64_t)b * hq + h) * kMaxSplit;
  float M = m_e;
  for (int sp = 0; sp < nsplit; ++sp) M = fmaxf(M, part_ml[(pb + sp) * 2]);
  if (t < dh) {
    const int d = t;
    float num = 0.f, den = 0.f;
    if (n_extra > 0) {
      const float a = __expf(m_e - M);
      float o = 0.f;
      for (int e = 0; e < n_extra; ++e) {
        const T* vp;
        if (e < s_sink) vp = sink_v + ((int64_t)b * s_sink + e) * Dp + (int64_t)j * dh;
        else vp = win_v + ((int64_t)b * W + (W - n_win) + (e - s_sink)) * Dp + (int64_t)j * dh;
        o = fmaf(__expf(lg[e] - m_e), load_elem(vp, d), o);
      }
      num += o * a;
      den += l_e * a;
    }
    for (int sp = 0; sp < nsplit; ++sp) {
      const float ms = part_ml[(pb + sp) * 2];
      if (ms == -INFINITY) continue;
      const float a = __expf(ms - M);
      num += part_o[(pb + sp) * dh + d] * a;
      den += part_ml[(pb + sp) * 2 + 1] * a;
    }
    out[((int64_t)b * hq + h) * dh + d] = num / den;
  }
}

// ---------------------------------------------------------------------------
// explicit reconstruction: K^[b, n, :] = C^K[b, idx[b, n]] (B^K)^T (fp32 out)
// ---------------------------------------------------------------------------
// grid (ceil(m / 16), h_kv, B), one wave: 16 tokens x d_h dims of head j.
template <typename T, int RBH>
__global__ __launch_bounds__(64) void k_reconstruct(
    const int32_t* __restrict__ idx_all, const T* __restrict__ bases_k, const T* __restrict__ bases_v,
    const T* __restrict__ coef_k, const T* __restrict__ coef_v, float* __restrict__ k_hat,
    float* __restrict__ v_hat, int m, int hkv, int dh, int nb, int rank, int R, int64_t L, int64_t cap,
    int bases_shared) {
  constexpr int NP = Parts<T>::n;
  const int tile = blockIdx.x, j = blockIdx.y, b = blockIdx.z;
  const int lane = threadIdx.x, slot = lane & 15, kg = lane >> 4;
  const int Dp = hkv * dh, Dg = Dp / nb;
  const int grp = j / (hkv / nb), row0 = (j % (hkv / nb)) * dh, kb0 = grp * rank / 32;
  const int n = tile * 16 + slot;
  int64_t tok = (n < m) ? (int64_t)idx_all[(int64_t)b * m + n] : 0;
  const bool bad = (n < m) && (tok < 0 || tok >= L);
  if (bad) tok = 0;
  const int64_t co = (tok >> 4) * 16 * (int64_t)R + (tok & 15) * 32 + kg * 8;
  const int64_t boff = (bases_shared ? 0 : (int64_t)b * Dp * rank) + (int64_t)grp * Dg * rank;
  for (int which = 0; which < 2; ++which) {
    const T* cb = (which == 0 ? coef_k : coef_v) + (int64_t)b * cap * R;
    const T* bb = (which == 0 ? bases_k : bases_v) + boff;
    float* dst = which == 0 ? k_hat : v_hat;
    Op8 a[RBH][NP];
#pragma unroll
    for (int kb = 0; kb < RBH; ++kb) Parts<T>::load(cb + co + (int64_t)(kb0 + kb) * 512, a[kb]);
    for (int nbk = 0; nbk < dh / 16; ++nbk) {
      floatx4 d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < RBH; ++kb) {
        Op8 bo[NP];
        Parts<T>::load(bb + (int64_t)(row0 + nbk * 16 + slot) * rank + kb * 32 + kg * 8, bo);
        d = mfma_parts<NP, NP>(a[kb], bo, d);
      }
      // lane holds rows (tokens) 4*kg + v of the tile, column (dim) slot
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int nn = tile * 16 + kg * 4 + v;
        if (nn < m) dst[((int64_t)b * m + nn) * Dp + (int64_t)j * dh + nbk * 16 + slot] = d[v];
      }
    }
  }
  // rows with an out-of-range index are set to NaN instead of being read
  if (bad) {
    for (int d = 0; d < dh; ++d) {
      k_hat[((int64_t)b * m + n) * Dp + (int64_t)j * dh + d] = __int_as_float(0x7fc00000);
      v_hat[((int64_t)b * m + n) * Dp + (int64_t)j * dh + d] = __int_as_float(0x7fc00000);
    }
  }
}

// ---------------------------------------------------------------------------
// explicit attention over given fp32 rows (plus sinks)
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void k_sparse_attn(
    const T* __restrict__ q, const T* __restrict__ sink_k, const T* __restrict__ sink_v,
    const int32_t* __restrict__ idx_all, const float* __restrict__ k_sel, const float* __restrict__ v_sel,
    float* __restrict__ out, float* __restrict__ logits_all, int m, int hq, int hkv, int dh, int s_sink,
    int64_t L, int64_t logit_stride, float theta) {
  const int h = blockIdx.x, b = blockIdx.y, t = threadIdx.x;
  const int G = hq / hkv, j = h / G, Dp = hkv * dh;
  const int n_all = s_sink + m;
  float* lg = logits_all + ((int64_t)b * hq + h) * logit_stride;
  __shared__ float qr[128];
  __shared__ double rfs[64];
  __shared__ float red[256];
  __shared__ float s_mx, s_sum;
  if (t < dh / 2) rfs[t] = rope_rev_freq(theta, t, dh);
  if (t < dh / 2) {
    float c, sn;
    rope_cs(s_sink + L - 1, rfs[t], c, sn);
    const int64_t qo = ((int64_t)b * hq + h) * dh;
    const float xl = load_elem(q, qo + t), xh = load_elem(q, qo + t + dh / 2);
    qr[t] = xl * c - xh * sn;
    qr[t + dh / 2] = xh * c + xl * sn;
  }
  __syncthreads();
  for (int e = t; e < n_all; e += blockDim.x) {
    float acc = 0.f;
    int64_t pos;
    if (e < s_sink) {
      pos = e;
      const T* kp = sink_k + ((int64_t)b * s_sink + e) * Dp + (int64_t)j * dh;
      for (int f = 0; f < dh / 2; ++f) {
        float c, sn;
        rope_cs(pos, rfs[f], c, sn);
        const float xl = load_elem(kp, f), xh = load_elem(kp, f + dh / 2);
        acc = fmaf(qr[f], xl * c - xh * sn, acc);
        acc = fmaf(qr[f + dh / 2], xh * c + xl * sn, acc);
      }
    } else {
      const int n = e - s_sink;
      pos = s_sink + (int64_t)idx_all[(int64_t)b * m + n];
      const float* kp = k_sel + ((int64_t)b * m + n) * Dp + (int64_t)j * dh;
      for (int f = 0; f < dh / 2; ++f) {
        float c, sn;
        rope_cs(pos, rfs[f], c, sn);
        const float xl = kp[f], xh = kp[f + dh / 2];
        acc = fmaf(qr[f], xl * c - xh * sn, acc);
        acc = fmaf(qr[f + dh / 2], xh * c + xl * sn, acc);
      }
    }
    lg[e] = acc / sqrtf((float)dh);
  }
  __syncthreads();
  float mx = -INFINITY;
  for (int e = t; e < n_all; e += blockDim.x) mx = fmaxf(mx, lg[e]);
  red[t] = mx;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (t < o) red[t] = fmaxf(red[t], red[t + o]);
    __syncthreads();
  }
  if (t == 0) s_mx = red[0];
  __syncthreads();
  float sm = 0.f;
  for (int e = t; e < n_all; e += blockDim.x) sm += __expf(lg[e] - s_mx);
  red[t] = sm;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (t < o) red[t] += red[t + o];
    __syncthreads();
  }
  if (t == 0) s_sum = red[0];
  __syncthreads();
  if (t < dh) {
    float o = 0.f;
    for (int e = 0; e < n_all; ++e) {
      const float p = __expf(lg[e] - s_mx);
      const float v = (e < s_sink) ? load_elem(sink_v, ((int64_t)b * s_sink + e) * Dp + (int64_t)j * dh + t)
                                   : v_sel[((int64_t)b * m + (e - s_sink)) * Dp + (int64_t)j * dh + t];
      o = fmaf(p, v, o);
    }
    out[((int64_t)b * hq + h) * dh + t] = o / s_sum;
  }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
static int choose_splits(const Problem& P, int n_proc) {
  const int ntile = (n_proc + 15) / 16;
  int ns = (ntile + 3) / 4;                                  // ~4 tiles per split
  const int cap_wg = std::max(1, 1024 / std::max(1, P.B * P.hkv));
  ns = std::min(ns, cap_wg);
  ns = std::min(ns, kMaxSplit);
  return std::max(ns, 1);
}

template <typename T, int RBH, int DH, int G>
static void launch_split_t(const Problem& P, const Workspace& ws, int64_t L, int m, int n_proc, int nsplit,
                           const void* q, const void* bases_k, const void* bases_v, const void* coef_k,
                           const void* coef_v, hipStream_t st) {
  hipLaunchKernelGGL((k_attn_split<T, RBH, DH, G>), dim3(nsplit, P.hkv, P.B), dim3(DH * 2), 0, st, (const T*)q,
                     (const T*)bases_k, (const T*)bases_v, (const T*)coef_k, (const T*)coef_v, ws.idx,
                     (int64_t)m, ws.part_ml, ws.part_o, n_proc, nsplit, P.hq, P.hkv, P.nb, P.rank, P.R,
                     P.s, L, P.cap, P.bases_shared, P.theta);
}

#define S4R_SPLIT_ARGS P, ws, L, m, n_proc, nsplit, q, bk, bv, ck, cv, st

template <typename T, int DH, int G>
static bool dispatch_split_rb(const Problem& P, const Workspace& ws, int64_t L, int m, int n_proc, int nsplit,
                              const void* q, const void* bk, const void* bv, const void* ck, const void* cv,
                              hipStream_t st) {
  switch (P.rank / 32) {
    case 1: launch_split_t<T, 1, DH, G>(S4R_SPLIT_ARGS); return true;
    case 2: launch_split_t<T, 2, DH, G>(S4R_SPLIT_ARGS); return true;
    case 3: launch_split_t<T, 3, DH, G>(S4R_SPLIT_ARGS); return true;
    case 4: launch_split_t<T, 4, DH, G>(S4R_SPLIT_ARGS); return true;
    case 5: launch_split_t<T, 5, DH, G>(S4R_SPLIT_ARGS); return true;
    case 6: launch_split_t<T, 6, DH, G>(S4R_SPLIT_ARGS); return true;
    case 8: launch_split_t<T, 8, DH, G>(S4R_SPLIT_ARGS); return true;
    default: return false;
  }
}

template <typename T, int DH>
static bool dispatch_split_g(const Problem& P, const Workspace& ws, int64_t L, int m, int n_proc, int nsplit,
                             const void* q, const void* bk, const void* bv, const void* ck, const void* cv,
                             hipStream_t st) {
  switch (P.G) {
    case 1: return dispatch_split_rb<T, DH, 1>(S4R_SPLIT_ARGS);
    case 2: return dispatch_split_rb<T, DH, 2>(S4R_SPLIT_ARGS);
    case 4: return dispatch_split_rb<T, DH, 4>(S4R_SPLIT_ARGS);
    case 7: return dispatch_split_rb<T, DH, 7>(S4R_SPLIT_ARGS);
    case 8: return dispatch_split_rb<T, DH, 8>(S4R_SPLIT_ARGS);
    default: return false;
  }
}

// which (G, rank) pairs the fused attention kernel is built for
bool attention_supported(const Problem& P) {
  const int rb = P.rank / 32;
  const bool g_ok = P.G == 1 || P.G == 2 || P.G == 4 || P.G == 7 || P.G == 8;
  const bool rb_ok = (rb >= 1 && rb <= 6) || rb == 8;
  return g_ok && rb_ok && (P.dh == 64 || P.dh == 128);
}

hipError_t launch_attention(const Problem& P, const Workspace& ws, int64_t L, int m, int k_eff, const void* q,
                            const void* sink_k, const void* sink_v, const void* win_k, const void* win_v,
                            const void* bases_k, const void* bases_v, const void* coef_k, const void* coef_v,
                            float* out, hipStream_t st, hipEvent_t* t0, hipEvent_t* t1) {
  (void)t0;
  (void)t1;
  const int n_proc = win_k ? k_eff : m;      // exact window rows go to the combine kernel
  const int nsplit = choose_splits(P, n_proc);
  bool ok = true;
  if (n_proc > 0) {
    const void *bk = bases_k, *bv = bases_v, *ck = coef_k, *cv = coef_v;
    if (P.dtype == S4R_BF16)
      ok = P.dh == 128 ? dispatch_split_g<uint16_t, 128>(S4R_SPLIT_ARGS) : dispatch_split_g<uint16_t, 64>(S4R_SPLIT_ARGS);
    else
      ok = P.dh == 128 ? dispatch_split_g<float, 128>(S4R_SPLIT_ARGS) : dispatch_split_g<float, 64>(S4R_SPLIT_ARGS);
  }
  if (!ok) return hipErrorInvalidValue;
  const int ns_used = n_proc > 0 ? nsplit : 0;
  if (P.dtype == S4R_BF16)
    hipLaunchKernelGGL(k_attn_combine<uint16_t>, dim3(P.hq, P.B), dim3(256), 0, st, (const uint16_t*)q,
                       (const uint16_t*)sink_k, (const uint16_t*)sink_v, (const uint16_t*)win_k,
                       (const uint16_t*)win_v, ws.part_ml, ws.part_o, out, ns_used, P.hq, P.hkv, P.dh, P.s, P.W, L,
                       P.theta);
  else
    hipLaunchKernelGGL(k_attn_combine<float>, dim3(P.hq, P.B), dim3(256), 0, st, (const float*)q,
                       (const float*)sink_k, (const float*)sink_v, (const float*)win_k, (const float*)win_v,
                       ws.part_ml, ws.part_o, out, ns_used, P.hq, P.hkv, P.dh, P.s, P.W, L, P.theta);
  return hipGetLastError();
}

template <typename T, int RBH>
static void launch_rec_t(const Problem& P, int64_t L, int m, const int32_t* idx, const void* bk, const void* bv,
                         const void* ck, const void* cv, float* kh, float* vh, hipStream_t st) {
  hipLaunchKernelGGL((k_reconstruct<T, RBH>), dim3((m + 15) / 16, P.hkv, P.B), dim3(64), 0, st, idx, (const T*)bk,
                     (const T*)bv, (const T*)ck, (const T*)cv, kh, vh, m, P.hkv, P.dh, P.nb, P.rank, P.R, L, P.cap,
                     P.bases_shared);
}

template <typename T>
static bool dispatch_rec(const Problem& P, int64_t L, int m, const int32_t* idx, const void* bk, const void* bv,
                         const void* ck, const void* cv, float* kh, float* vh, hipStream_t st) {
  switch (P.rank / 32) {
    case 1: launch_rec_t<T, 1>(P, L, m, idx, bk, bv, ck, cv, kh, vh, st); return true;
    case 2: launch_rec_t<T, 2>(P, L, m, idx, bk, bv, ck, cv, kh, vh, st); return true;
    case 3: launch_rec_t<T, 3>(P, L, m, idx, bk, bv, ck, cv, kh, vh, st); return true;
    case 4: launch_rec_t<T, 4>(P, L, m, idx, bk, bv, ck, cv, kh, vh, st); return true;
    case 5: launch_rec_t<T, 5>(P, L, m, idx, bk, bv, ck, cv, kh, vh, st); return true;
    case 6: launch_rec_t<T, 6>(P, L, m, idx, bk, bv, ck, cv, kh, vh, st); return true;
    case 7: launch_rec_t<T, 7>(P, L, m, idx, bk, bv, ck, cv, kh, vh, st); return true;
    case 8: launch_rec_t<T, 8>(P, L, m, idx, bk, bv, ck, cv, kh, vh, st); return true;
    default: return false;
  }
}

hipError_t launch_reconstruct(const Problem& P, int64_t L, int m, const int32_t* idx, const void* bases_k,
                              const void* bases_v, const void* coef_k, const void* coef_v, float* k_hat,
                              float* v_hat, hipStream_t st) {
  if (m <= 0) return hipSuccess;
  bool ok = P.dtype == S4R_BF16
                ? dispatch_rec<uint16_t>(P, L, m, idx, bases_k, bases_v, coef_k, coef_v, k_hat, v_hat, st)
                : dispatch_rec<float>(P, L, m, idx, bases_k, bases_v, coef_k, coef_v, k_hat, v_hat, st);
  if (!ok) return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_sparse_attn(const Problem& P, const Workspace& ws, int64_t L, int m, const void* q,
                              const void* sink_k, const void* sink_v, const int32_t* idx, const float* k_sel,
                              const float* v_sel, float* out, hipStream_t st) {
  const int64_t stride = P.s + P.m_max;
  if (P.dtype == S4R_BF16)
    hipLaunchKernelGGL(k_sparse_attn<uint16_t>, dim3(P.hq, P.B), dim3(256), 0, st, (const uint16_t*)q,
                       (const uint16_t*)sink_k, (const uint16_t*)sink_v, idx, k_sel, v_sel, out, ws.attn_logits, m,
                       P.hq, P.hkv, P.dh, P.s, L, stride, P.theta);
  else
    hipLaunchKernelGGL(k_sparse_attn<float>, dim3(P.hq, P.B), dim3(256), 0, st, (const float*)q,
                       (const float*)sink_k, (const float*)sink_v, idx, k_sel, v_sel, out, ws.attn_logits, m, P.hq,
                       P.hkv, P.dh, P.s, L, stride, P.theta);
  return hipGetLastError();
}

}  // namespace s4r
