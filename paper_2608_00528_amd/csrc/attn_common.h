// Device helpers shared by the attention kernels (RoPE, operand parts) and
// the fused reconstruction + split attention kernel template.
#pragma once

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

// RoPE phase of integer position pos at a frequency given as a 0.64
// fixed-point number of revolutions per position: the fractional revolution
// pos * F mod 1 is exact in 64-bit integer arithmetic
__device__ __forceinline__ void rope_cs_fixed(int64_t pos, uint64_t F, float& c, float& s) {
  // high word of the low 64 bits of pos * F (positions are below 2^31): two
  // 32-bit multiplies and an add
  const uint32_t p = (uint32_t)pos, flo = (uint32_t)F, fhi = (uint32_t)(F >> 32);
  const uint32_t hi = (uint32_t)(((uint64_t)p * flo) >> 32) + p * fhi;
  const float x = (float)hi * 2.3283064365386963e-10f;          // 2^-32 revolutions, rounded to 24 bits
  c = __builtin_amdgcn_cosf(x);
  s = __builtin_amdgcn_sinf(x);
}
// revolutions per position of frequencies f0 .. f0 + 3, as 0.64 fixed point:
// theta^(-2 f / d_h) / (2 pi) = ratio^f / (2 pi) with ratio = theta^(-2 / d_h)
// (computed once on the host in fp64; ratio 0 disables RoPE).  ratio^f0 by
// repeated squaring: about 2^-50 relative, so the phase stays exact to about
// 2^-32 revolutions for any position below 2^18.
__device__ __forceinline__ void rope_freqs_fixed(double ratio, int f0, uint64_t (&F)[4]) {
  double p = 1.0, base = ratio;
  for (int e = f0; e > 0; e >>= 1) {
    if (e & 1) p *= base;
    base *= base;
  }
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    F[v] = (ratio == 0.0) ? 0ull : (uint64_t)(p * 0.15915494309189535 * 18446744073709551616.0);
    p *= ratio;
  }
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


// two workgroups per CU (at most 256 registers per lane) where the
// instantiation fits without spilling: bf16 storage with
// 24 * (rank / 32) + 19 * (G - 1) <= 186, from the compiled register counts
template <typename T, int RBH, int G>
constexpr int attn_split_occupancy() {
  return (sizeof(T) == 2 && 24 * RBH + 19 * (G - 1) <= 186) ? 2 : 1;
}

template <typename T, int RBH, int DH, int G>
__global__ __launch_bounds__(DH * 2, (attn_split_occupancy<T, RBH, G>())) void k_attn_split(
    const T* __restrict__ q, const T* __restrict__ bases_k, const T* __restrict__ bases_v,
    const T* __restrict__ coef_k, const T* __restrict__ coef_v, const int32_t* __restrict__ idx_all,
    int64_t idx_stride, float* __restrict__ part_ml, float* __restrict__ part_o, int n_proc, int nsplit,
    int hq, int hkv, int nb, int rank, int R, int s_sink, int64_t L, int64_t cap, int bases_shared,
    float theta, Lens lens) {
  constexpr int NP = Parts<T>::n;
  constexpr int NWAVE = DH / 32;          // waves per workgroup
  constexpr int HALF_MB = DH / 32;        // pair offset in 16-dim blocks
  const int split = blockIdx.x, j = blockIdx.y, b = blockIdx.z;
  L = len_of(lens, b, L);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int slot = lane & 15, kg = lane >> 4;
  const int Dp = hkv * DH, Dg = Dp / nb;
  const int grp = j / (hkv / nb);
  const int row0 = (j % (hkv / nb)) * DH;          // first basis row of head j in its group
  const int kb0 = grp * rank / 32;                 // first latent block of the group

  // ---- prologue: every global read of the workgroup's setup is requested
  // before any is used (value basis and query into registers, the split's
  // index list and the key basis into LDS), so it costs one round trip.
  const int ntile = (n_proc + 15) / 16;
  const int tps = (ntile + nsplit - 1) / nsplit;
  const int tile0 = split * tps, tile1 = min(ntile, tile0 + tps);
  const int32_t* idx = idx_all + (int64_t)b * idx_stride;
  const T* ckb = coef_k + (int64_t)b * cap * R;
  const T* cvb = coef_v + (int64_t)b * cap * R;
  const float inv_sqrt_d = 1.0f / sqrtf((float)DH);
  extern __shared__ int32_t sidx[];                 // [tps * 16] token positions of the split
  __shared__ float xlog[2][NWAVE][G][16];

  // basis operands (A): rows d = 16*mb + slot, k-group kg.  bf16: the key
  // basis slice of every wave sits in LDS (rows padded by 16 bytes: the
  // 16-byte operand reads of one MFMA hit distinct banks) and the value basis
  // in registers; fp32 (three bf16 parts each) keeps both in registers.
  constexpr bool KB_LDS = (NP == 1);
  constexpr int KS = RBH * 32 + 8;                 // padded LDS row (elements)
  __shared__ __align__(16) uint16_t kbase[KB_LDS ? NWAVE : 1][2][16][KB_LDS ? KS : 8];
  Op8 ak[KB_LDS ? 1 : 2][KB_LDS ? 1 : RBH][NP], av[2][RBH][NP];
  const int64_t boff = (bases_shared ? 0 : (int64_t)b * Dp * rank) + (int64_t)grp * Dg * rank;
#pragma unroll
  for (int hm = 0; hm < 2; ++hm) {
    const int d = 16 * (w + hm * HALF_MB) + slot;
#pragma unroll
    for (int kb = 0; kb < RBH; ++kb) {
      const int64_t o = boff + (int64_t)(row0 + d) * rank + kb * 32 + kg * 8;
      if constexpr (!KB_LDS) Parts<T>::load(bases_k + o, ak[hm][kb]);
      Parts<T>::load(bases_v + o, av[hm][kb]);
    }
  }
  // the query at this lane's 8 dims (rotated below)
  float qx[G][8];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int dlo = 16 * w + 4 * kg + v, dhi = dlo + DH / 2;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int64_t qo = ((int64_t)b * hq + (int64_t)j * G + g) * DH;
      qx[g][v] = load_elem(q, qo + dlo);
      qx[g][4 + v] = load_elem(q, qo + dhi);
    }
  }
  // the split's index list (one item per thread for up to 16 tiles)
  const int nsi = (tile1 - tile0) * 16;
  int32_t si0 = 0;
  if (nsi > 0) si0 = idx[min(tile0 * 16 + min((int)threadIdx.x, nsi - 1), n_proc - 1)];
  if constexpr (KB_LDS) {
    // whole workgroup copies the K rows of all waves: [wave][hm][16 rows][RBH*32]
    const int per_row = RBH * 4;                 // 16-byte pieces per row
    batched_copy16<(NWAVE * 2 * 16 * RBH * 4 + DH * 2 - 1) / (DH * 2)>(
        NWAVE * 2 * 16 * per_row,
        [&](int i) {
          const int ww = i / (2 * 16 * per_row), rem = i % (2 * 16 * per_row);
          const int hm = rem / (16 * per_row), rem2 = rem % (16 * per_row);
          const int d = 16 * (ww + hm * HALF_MB) + rem2 / per_row;
          return reinterpret_cast<const uint4*>(bases_k + boff + (int64_t)(row0 + d) * rank + (rem2 % per_row) * 8);
        },
        [&](int i) {
          const int ww = i / (2 * 16 * per_row), rem = i % (2 * 16 * per_row);
          const int hm = rem / (16 * per_row), rem2 = rem % (16 * per_row);
          return reinterpret_cast<uint4*>(&kbase[ww][hm][rem2 / per_row][(rem2 % per_row) * 8]);
        });
  }
  if (nsi > 0) {
    const int i = min((int)threadIdx.x, nsi - 1);   // threads past nsi rewrite item nsi - 1
    sidx[i] = (tile0 * 16 + i < n_proc) ? si0 : -1;
  }
  for (int i = (int)blockDim.x + (int)threadIdx.x; i < nsi; i += (int)blockDim.x)   // splits over 16 tiles
    sidx[i] = (tile0 * 16 + i < n_proc) ? idx[tile0 * 16 + i] : -1;
  auto akop = [&](int hm, int kb) -> const Op8* {
    if constexpr (KB_LDS) {
      return reinterpret_cast<const Op8*>(&kbase[w][hm][slot][kb * 32 + kg * 8]);
    } else {
      return ak[hm][kb];
    }
  };
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
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float xl = qx[g][v], xh = qx[g][4 + v];
      qr[g][v] = xl * c - xh * sn;
      qr[g][4 + v] = xh * c + xl * sn;
    }
  }
  __syncthreads();

  float mrun[G], lrun[G], oacc[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    mrun[g] = -INFINITY;
    lrun[g] = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) oacc[g][i] = 0.f;
  }

  // coefficient row offset of this lane's token in a tile (0 for padding slots)
  auto tok_of = [&](int tile) -> int64_t {
    const int32_t x = sidx[(tile - tile0) * 16 + slot];
    return x < 0 ? 0 : (int64_t)x;
  };
  auto row_off = [&](int64_t tok) -> int64_t { return (tok >> 4) * 16 * (int64_t)R + (tok & 15) * 32 + kg * 8; };
  auto issue = [&](const T* base, int64_t tok, Op8 (&dst)[RBH][NP]) {
    const int64_t co = row_off(tok);
#pragma unroll
    for (int kb = 0; kb < RBH; ++kb) Parts<T>::load(base + co + (int64_t)(kb0 + kb) * 512, dst[kb]);
  };

  // one tile's reconstruction, RoPE, logits and online softmax from gathered
  // coefficient operands bk / bv (this lane: token slot, k-group kg)
  auto compute_tile = [&](int tile, const Op8 (&bk)[RBH][NP], const Op8 (&bv)[RBH][NP]) {
    const bool valid = sidx[(tile - tile0) * 16 + slot] >= 0;
    const int64_t tok = tok_of(tile);
    floatx4 dk[2];
#pragma unroll
    for (int hm = 0; hm < 2; ++hm) {
      dk[hm] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < RBH; ++kb) {
        if constexpr (KB_LDS) {
          Op8 a0;
          a0.u = *reinterpret_cast<const uint4*>(akop(hm, kb));
          dk[hm] = mfma16x16x32(a0, bk[kb][0], dk[hm]);
        } else {
          dk[hm] = mfma_parts<NP, NP>(akop(hm, kb), bk[kb], dk[hm]);
        }
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
      float a = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) a = fmaf(qr[g][i], kr[i], a);
      a += shfl_xor_f(a, 16);
      a += shfl_xor_f(a, 32);
      part[g] = a;
    }
    const int buf = tile & 1;
    if (kg == 0) {
#pragma unroll
      for (int g = 0; g < G; ++g) xlog[buf][w][g][slot] = part[g];
    }
    floatx4 dv[2];
#pragma unroll
    for (int hm = 0; hm < 2; ++hm) {
      dv[hm] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < RBH; ++kb) dv[hm] = mfma_parts<NP, NP>(av[hm][kb], bv[kb], dv[hm]);
    }
    lds_barrier();   // logit exchange; gathers in flight stay in flight
    // online softmax with one running maximum per query head shared by the 16
    // token slots: the tile's maximum comes from a reduction over the slots,
    // and the accumulators are rescaled only when it raises the running
    // maximum (a uniform branch), so most tiles need no rescale
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float sfull = 0.f;
#pragma unroll
      for (int ww = 0; ww < NWAVE; ++ww) sfull += xlog[buf][ww][g][slot];
      const float sc = valid ? sfull * inv_sqrt_d : -INFINITY;
      const float tmax = slot_max16(sc);
      if (tmax > mrun[g]) {
        const float alpha = __expf(mrun[g] - tmax);   // 0 when mrun is -inf
        lrun[g] *= alpha;
#pragma unroll
        for (int i = 0; i < 8; ++i) oacc[g][i] *= alpha;
        mrun[g] = tmax;
      }
      const float p = valid ? __expf(sc - mrun[g]) : 0.f;
      lrun[g] += p;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        oacc[g][v] = fmaf(p, dv[0][v], oacc[g][v]);
        oacc[g][4 + v] = fmaf(p, dv[1][v], oacc[g][4 + v]);
      }
    }
  };

  // gathers into registers, the next tile's issued before this tile's compute
  // and kept in flight across its LDS-only barrier
  Op8 bka[RBH][NP], bkb[RBH][NP], bva[RBH][NP], bvb[RBH][NP];
  if (tile0 < tile1) {
    issue(ckb, tok_of(tile0), bka);
    issue(cvb, tok_of(tile0), bva);
  }
  for (int tile = tile0; tile < tile1; tile += 2) {
    {
      const int64_t tn = tok_of(min(tile + 1, tile1 - 1));
      issue(ckb, tn, bkb);
      issue(cvb, tn, bvb);
    }
    compute_tile(tile, bka, bva);
    if (tile + 1 < tile1) {
      const int64_t tn = tok_of(min(tile + 2, tile1 - 1));
      issue(ckb, tn, bka);
      issue(cvb, tn, bva);
      compute_tile(tile + 1, bkb, bvb);
    }
  }

  // ---- merge the 16 token slots (they share the running maximum) ------------------
#pragma unroll
  for (int g = 0; g < G; ++g) {
    lrun[g] = slot_sum16(lrun[g]);
#pragma unroll
    for (int i = 0; i < 8; ++i) oacc[g][i] = slot_sum16(oacc[g][i]);
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

// two fp32 values -> packed bf16 (round to nearest even; one v_cvt_pk_bf16_f32)
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  const f32x2_t v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

// 8 fp32 values -> one bf16 operand (round to nearest even)
__device__ __forceinline__ void round_f32x8(const float* x, Op8& o) {
  o.u = make_uint4(pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]), pack_bf16x2(x[4], x[5]),
                   pack_bf16x2(x[6], x[7]));
}

// 8 fp32 values -> bf16 hi and lo parts (x ~= hi + lo to about 2^-17)
__device__ __forceinline__ void split2_f32x8(const float* x, Op8& hi, Op8& lo) {
  uint32_t ph[4], pl[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    ph[i] = pack_bf16x2(x[2 * i], x[2 * i + 1]);
    const float r0 = x[2 * i] - __uint_as_float(ph[i] << 16);
    const float r1 = x[2 * i + 1] - __uint_as_float(ph[i] & 0xFFFF0000u);
    pl[i] = pack_bf16x2(r0, r1);
  }
  hi.u = make_uint4(ph[0], ph[1], ph[2], ph[3]);
  lo.u = make_uint4(pl[0], pl[1], pl[2], pl[3]);
}

}  // namespace s4r
