// Sparse reconstruction and final attention of Section 3.2.3 on gfx950.
//
//   k_attn_split  one workgroup per (split, kv head j, sequence).  Wave w owns
//                 the dimension pair blocks {w, w + d_h/32} of head j (16 dims
//                 each, so every RoPE pair (i, i + d_h/2) sits in one lane).
//                 Per 16-token tile of the index list it gathers the selected
//                 coefficient rows (64-byte pieces of the tiled cache) as MFMA
//                 B operands and forms K^T = B^K_j C^T and V^T = B^V_j C^T with
//                 bf16 MFMA (basis rows as A operands: the key basis staged in LDS,
//                 the value basis in registers), so a
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
#include "attn_common.h"

namespace s4r {

// ---------------------------------------------------------------------------
// combine: sinks, exact window, splits -> O_t
// ---------------------------------------------------------------------------
// One workgroup per (query head, sequence).  Every split's (max, sum, output)
// is requested up front (thread t holds float4 t, t + 256, ... of the splits'
// outputs, i.e. dims 4 t % d_h .. + 3 of several splits), together with the key and value rows
// of the first kPreTok extra full-precision tokens (the sinks; further rows
// of an optional exact window are loaded as they are reached).  The extra
// tokens are attended on the VALU with the same fixed-point RoPE phases, and
// the partials are merged with the usual max rescaling.
constexpr int kMaxExtra = 1024 + 64;   // sinks + exact window rows
constexpr int kCombVec = kMaxSplit * 128 / (4 * 256);   // float4 of split outputs per thread
constexpr int kPreTok = 4;             // extra tokens whose rows come with the first loads

// CV: float4 of split outputs per thread, the smallest of 1, 2, 4, kCombVec
// that covers nsplit * d_h / 4 (the launch picks it)
template <typename T, int CV>
__global__ __launch_bounds__(256) void k_attn_combine(
    const T* __restrict__ q, const T* __restrict__ sink_k, const T* __restrict__ sink_v,
    const T* __restrict__ win_k, const T* __restrict__ win_v, const float* __restrict__ part_ml,
    const float* __restrict__ part_o, float* __restrict__ out, int nsplit, int hq, int hkv, int dh,
    int s_sink, int W, int64_t L, double rope_ratio, Lens lens) {
  const int h = blockIdx.x, b = blockIdx.y;
  L = len_of(lens, b, L);
  const int G = hq / hkv, j = h / G;
  const int Dp = hkv * dh;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int64_t pos_q = s_sink + L - 1;
  const int n_win = win_k ? (int)min<int64_t>(W, L) : 0;
  const int n_extra = s_sink + n_win;
  const int half = dh / 2;
  const int64_t pb = ((int64_t)b * hq + h) * kMaxSplit;

  __shared__ float qr[128];
  __shared__ uint64_t fq[64];
  __shared__ float lg[kMaxExtra];
  __shared__ float s_as[kMaxSplit];
  __shared__ float red[1024];
  __shared__ float s_me, s_den, s_ae;

  // ---- every load of the split partials and the query, issued together -----------------
  const int ne4 = nsplit * dh / 4;                // float4 of split outputs (d_h is a multiple of 4)
  const int ldh = __builtin_ctz(dh);               // head_dim is a power of two
  float4 po[CV];
  const float4* po4 = reinterpret_cast<const float4*>(part_o + pb * dh);
#pragma unroll
  for (int i = 0; i < CV; ++i) po[i] = po4[max(min(t + 256 * i, ne4 - 1), 0)];   // masked below
  float2 ml = make_float2(-INFINITY, 0.f);
  if (t < nsplit) ml = reinterpret_cast<const float2*>(part_ml)[pb + t];
  float xl = 0.f, xh = 0.f;
  if (t < half) {
    const int64_t qo = ((int64_t)b * hq + h) * dh;
    xl = load_elem(q, qo + t);
    xh = load_elem(q, qo + t + half);
  }
  auto krow = [&](int e) -> const T* {
    if (e < s_sink) return sink_k + ((int64_t)b * s_sink + e) * Dp + (int64_t)j * dh;
    return win_k + ((int64_t)b * W + (W - n_win) + (e - s_sink)) * Dp + (int64_t)j * dh;
  };
  auto vrow = [&](int e) -> const T* {
    if (e < s_sink) return sink_v + ((int64_t)b * s_sink + e) * Dp + (int64_t)j * dh;
    return win_v + ((int64_t)b * W + (W - n_win) + (e - s_sink)) * Dp + (int64_t)j * dh;
  };
  auto kpos = [&](int e) -> int64_t { return e < s_sink ? (int64_t)e : (int64_t)s_sink + (L - n_win) + (e - s_sink); };
  // key row of extra token `wave` (lane = RoPE pair) and value rows of the
  // first kPreTok extra tokens (thread t < d_h = dim t)
  float pkl = 0.f, pkh = 0.f;
  if (wave < n_extra && lane < half) {
    const T* kp = krow(wave);
    pkl = load_elem(kp, lane);
    pkh = load_elem(kp, lane + half);
  }
  float pv[kPreTok];
#pragma unroll
  for (int e = 0; e < kPreTok; ++e) pv[e] = (e < n_extra && t < dh) ? load_elem(vrow(e), t) : 0.f;

  // ---- rotated query ----------------------------------------------------------------------
  if (t < half) {
    uint64_t F[4];
    rope_freqs_fixed(rope_ratio, t, F);
    fq[t] = F[0];
    float c, sn;
    rope_cs_fixed(pos_q, F[0], c, sn);
    qr[t] = xl * c - xh * sn;
    qr[t + half] = xh * c + xl * sn;
  }
  __syncthreads();
  // ---- logits of the full-precision tokens: one wave per token, lane = RoPE pair ---------
  for (int e = wave; e < n_extra; e += 4) {
    float part = 0.f;
    if (lane < half) {
      const T* kp = krow(e);
      const float kl = (e == wave) ? pkl : load_elem(kp, lane), kh = (e == wave) ? pkh : load_elem(kp, lane + half);
      float c, sn;
      rope_cs_fixed(kpos(e), fq[lane], c, sn);
      part = qr[lane] * (kl * c - kh * sn) + qr[lane + half] * (kh * c + kl * sn);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) part += shfl_xor_f(part, o);
    if (lane == 0) lg[e] = part / sqrtf((float)dh);
  }
  __syncthreads();
  // ---- (max, sum) of the extra tokens, global maximum, split weights (wave 0) ------------
  if (wave == 0) {
    float mx = -INFINITY;
    for (int e = lane; e < n_extra; e += 64) mx = fmaxf(mx, lg[e]);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, shfl_xor_f(mx, o));
    float sm = 0.f;
    for (int e = lane; e < n_extra; e += 64) sm += __expf(lg[e] - mx);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) sm += shfl_xor_f(sm, o);
    float M = mx;
    float ms = (lane < nsplit) ? ml.x : -INFINITY;
    float m2 = ms;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m2 = fmaxf(m2, shfl_xor_f(m2, o));
    M = fmaxf(M, m2);
    const float ae = (n_extra > 0) ? __expf(mx - M) : 0.f;
    const float a = (lane < nsplit && ms != -INFINITY) ? __expf(ms - M) : 0.f;   // empty split: weight 0
    // denominator: the splits' weighted sums (lane = split) plus the extra tokens'
    float den = (lane < nsplit) ? a * ml.y : 0.f;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) den += shfl_xor_f(den, o);
    if (lane == 0) {
      s_me = mx;
      s_ae = ae;
      s_den = den + ae * sm;
    }
    if (lane < kMaxSplit) s_as[lane] = a;
  }
  __syncthreads();
  // ---- weighted split outputs: thread t holds dims 4 t % dh .. + 3 -----------------------
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int i = 0; i < CV; ++i) {
    const int e4 = t + 256 * i;
    if (e4 < ne4) {
      const float a = s_as[(4 * e4) >> ldh];
      acc.x += po[i].x * a;
      acc.y += po[i].y * a;
      acc.z += po[i].z * a;
      acc.w += po[i].w * a;
    }
  }
  *reinterpret_cast<float4*>(&red[4 * t]) = acc;   // red[e] holds dim e % dh
  __syncthreads();
  if (t < dh) {
    float num = 0.f;
    for (int k = t; k < 1024; k += dh) num += red[k];
    if (n_extra > 0) {
      const float me = s_me;
      float o = 0.f;
#pragma unroll
      for (int e = 0; e < kPreTok; ++e)
        if (e < n_extra) o = fmaf(__expf(lg[e] - me), pv[e], o);
#pragma unroll 4
      for (int e = kPreTok; e < n_extra; ++e) o = fmaf(__expf(lg[e] - me), load_elem(vrow(e), t), o);
      num += o * s_ae;
    }
    out[((int64_t)b * hq + h) * dh + t] = num / s_den;
  }
}

// the split merge of nsplit partials per (query head, sequence) with the extra
// full-precision tokens (sinks, optional exact window) attended beside them
template <typename T>
static void launch_combine_t(const Problem& P, const Workspace& ws, int64_t L, int nsplit, const void* q,
                             const void* sink_k, const void* sink_v, const void* win_k, const void* win_v, int s_sink,
                             int W, float* out, hipStream_t st) {
  const int need = (nsplit * P.dh + 1023) / 1024;
  auto kern = need <= 1 ? k_attn_combine<T, 1>
              : need <= 2 ? k_attn_combine<T, 2> : need <= 4 ? k_attn_combine<T, 4> : k_attn_combine<T, kCombVec>;
  hipLaunchKernelGGL(kern, dim3(P.hq, P.B), dim3(256), 0, st, (const T*)q, (const T*)sink_k, (const T*)sink_v,
                     (const T*)win_k, (const T*)win_v, ws.part_ml, ws.part_o, out, nsplit, P.hq, P.hkv, P.dh, s_sink,
                     W, L, rope_ratio(P), P.lens);
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
  __shared__ float red[1024];
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
  // about two workgroups per CU over the whole batch, at least two tiles each,
  // and an index list that fits comfortably in LDS
  const int ntile = (n_proc + 15) / 16;
  const int pairs = std::max(1, P.B * P.hkv);
  int ns = std::max(1, 512 / pairs);
  ns = std::min(ns, std::max(1, ntile / 2));
  ns = std::min(ns, kMaxSplit);
  while ((ntile + ns - 1) / ns > kMaxTilesPerSplit && ns < kMaxSplit) ++ns;
  return std::max(ns, 1);
}

// per-(dtype, head dim) instantiations live in attn_split_*.hip
bool launch_split_bf16_128(const Problem&, const Workspace&, int64_t, int, int, int, const void*, const void*,
                           const void*, const void*, const void*, hipStream_t);
bool launch_split_bf16_64(const Problem&, const Workspace&, int64_t, int, int, int, const void*, const void*,
                          const void*, const void*, const void*, hipStream_t);
bool launch_split_f32_128(const Problem&, const Workspace&, int64_t, int, int, int, const void*, const void*,
                          const void*, const void*, const void*, hipStream_t);
bool launch_split_f32_64(const Problem&, const Workspace&, int64_t, int, int, int, const void*, const void*,
                         const void*, const void*, const void*, hipStream_t);

bool launch_tiles_bf16_128(const Problem&, const Workspace&, int64_t, int, int, const void*, const void*,
                           const void*, const void*, const void*, hipStream_t, int*, bool);
bool launch_tiles_bf16_64(const Problem&, const Workspace&, int64_t, int, int, const void*, const void*,
                          const void*, const void*, const void*, hipStream_t, int*, bool);

// which (G, rank) pairs the fused attention kernel is built for (asymmetric
// key / value ranks: the bf16 MFMA kernel only)
bool attention_supported(const Problem& P) {
  if (P.rank_v != P.rank)
    return P.dtype == S4R_BF16 && (P.dh == 64 || P.dh == 128) && P.G <= 8 &&
           tiles_rank_pair(P.rank / 32, P.rank_v / 32);
  const int rb = P.rank / 32;
  const bool g_ok = P.G == 1 || P.G == 2 || P.G == 4 || P.G == 7 || P.G == 8;
  // seven blocks (rank 224, the padded r = 204) only on the bf16 MFMA kernel
  const bool rb_ok = (rb >= 1 && rb <= 6) || rb == 8 || (rb == 7 && P.dtype == S4R_BF16);
  return g_ok && rb_ok && (P.dh == 64 || P.dh == 128);
}

hipError_t launch_attention(const Problem& P, const Workspace& ws, int64_t L, int m, int k_eff, const void* q,
                            const void* sink_k, const void* sink_v, const void* win_k, const void* win_v,
                            const void* bases_k, const void* bases_v, const void* coef_k, const void* coef_v,
                            float* out, hipStream_t st, hipEvent_t* t0, hipEvent_t* t1) {
  const int n_proc = win_k ? k_eff : m;      // exact window rows go to the combine kernel
  int nsplit = choose_splits(P, n_proc);
  bool ok = true;
  if (t0 && hipEventRecord(t0[0], st) != hipSuccess) return hipErrorUnknown;
  bool tiles = false;                        // bf16: the MFMA kernel when it covers the configuration
  if (n_proc > 0 && P.dtype == S4R_BF16) {
    int ns = 0;
    tiles = P.dh == 128
                ? launch_tiles_bf16_128(P, ws, L, m, n_proc, q, bases_k, bases_v, coef_k, coef_v, st, &ns, false)
                : launch_tiles_bf16_64(P, ws, L, m, n_proc, q, bases_k, bases_v, coef_k, coef_v, st, &ns, false);
    if (tiles) nsplit = ns;
  }
  if (n_proc > 0 && !tiles && P.rank_v != P.rank) return hipErrorInvalidValue;   // MFMA kernel only
  if (n_proc > 0 && !tiles) {
    if (P.dtype == S4R_BF16)
      ok = P.dh == 128 ? launch_split_bf16_128(P, ws, L, m, n_proc, nsplit, q, bases_k, bases_v, coef_k, coef_v, st)
                       : launch_split_bf16_64(P, ws, L, m, n_proc, nsplit, q, bases_k, bases_v, coef_k, coef_v, st);
    else
      ok = P.dh == 128 ? launch_split_f32_128(P, ws, L, m, n_proc, nsplit, q, bases_k, bases_v, coef_k, coef_v, st)
                       : launch_split_f32_64(P, ws, L, m, n_proc, nsplit, q, bases_k, bases_v, coef_k, coef_v, st);
  }
  if (!ok) return hipErrorInvalidValue;
  if (t1 && hipEventRecord(t1[0], st) != hipSuccess) return hipErrorUnknown;
  if (t0 && hipEventRecord(t0[1], st) != hipSuccess) return hipErrorUnknown;
  const int ns_used = n_proc > 0 ? nsplit : 0;
  if (P.dtype == S4R_BF16)
    launch_combine_t<uint16_t>(P, ws, L, ns_used, q, sink_k, sink_v, win_k, win_v, P.s, P.W, out, st);
  else
    launch_combine_t<float>(P, ws, L, ns_used, q, sink_k, sink_v, win_k, win_v, P.s, P.W, out, st);
  hipError_t e = hipGetLastError();
  if (e == hipSuccess && t1) e = hipEventRecord(t1[1], st);
  return e;
}

// full reconstruction (Appendix B.1): attention over the sinks and all L
// tokens, each reconstructed from its coefficients: the bf16 MFMA kernel in
// its every-token mode, then the split merge with the sinks
hipError_t launch_full_recon(const Problem& P, const Workspace& ws, int64_t L, const void* q, const void* sink_k,
                             const void* sink_v, const void* bases_k, const void* bases_v, const void* coef_k,
                             const void* coef_v, float* out, hipStream_t st) {
  int ns = 0;
  const bool ok =
      P.dh == 128
          ? launch_tiles_bf16_128(P, ws, L, (int)L, (int)L, q, bases_k, bases_v, coef_k, coef_v, st, &ns, true)
          : launch_tiles_bf16_64(P, ws, L, (int)L, (int)L, q, bases_k, bases_v, coef_k, coef_v, st, &ns, true);
  if (!ok) return hipErrorInvalidValue;
  launch_combine_t<uint16_t>(P, ws, L, ns, q, sink_k, sink_v, nullptr, nullptr, P.s, P.W, out, st);
  return hipGetLastError();
}

// the split merge alone (no extra full-precision tokens), for kernels that
// leave split partials in the workspace
hipError_t launch_combine_only(const Problem& P, const Workspace& ws, int64_t L, int nsplit, const void* q, float* out,
                               hipStream_t st) {
  launch_combine_t<uint16_t>(P, ws, L, nsplit, q, nullptr, nullptr, nullptr, nullptr, 0, 0, out, st);
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
