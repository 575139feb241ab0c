// Fused sparse reconstruction + split attention for bf16 storage on gfx950
// (Section 3.2.3): every contraction on bf16 MFMA, every gather issued up front.
//
// One workgroup per (split, HPW KV heads, sequence), NW = d_h / 32 waves,
// TPW tiles of 16 selected tokens; HPW heads of one basis group reuse the
// gathered rows.  The work items are laid out over a 1-D grid so
// that the workgroups of one (sequence, split) land on the same XCD
// (workgroup i runs on XCD i % 8): the gathered coefficient rows are then
// fetched from HBM once per XCD and re-read from its L2 by the other heads.
//
//   1. the split's index list goes to LDS; every selected token's C^K and
//      C^V row pieces are requested at once with 16-byte global->LDS loads
//      (lane l of a wave load lands at byte 16 l of the destination, so one
//      wave load writes one 16-token x 32-column block in MFMA operand
//      layout);
//   2. wave w owns the dimension blocks {w, w + NW} (16 dims each), so each
//      RoPE pair (i, i + d_h/2) is in one lane; its bases stay in registers;
//   3. per tile: K^ = B^K_j C^T (D[dim][token]), RoPE at the token's
//      original position, then the wave's partial logits against the
//      rotated query on MFMA: the query's hi / lo bf16 parts sit in A rows
//      4 h + part, so lane (token t, k-group h) receives the parts for head h
//      and token t, and K~ enters as hi / lo bf16 parts;
//   4. the NW partial logits are summed through LDS; lane (t, h) runs the
//      online softmax of (token t, head h) with one running maximum per head
//      shared by the 16 token slots;
//   5. V^ = C^V B^V_j^T (D[token][dim]) of two tiles, as hi / lo bf16 parts,
//      forms the B operand of P V^, with P's hi / lo bf16 parts (staged
//      through LDS) as A rows 4 h + part; the output rows of head h land in
//      the lanes that own head h's softmax state, which rescale them when
//      its maximum grows.  Every operand pair carries about 16 significant
//      bits, so the fused step tracks the fp32 path to about 1e-5.
//
// Each split writes its (max, sum) and unnormalised output per head.
#pragma once

#include "attn_common.h"

namespace s4r {

// two fp32 values -> packed bf16 (round to nearest even; one v_cvt_pk_bf16_f32)
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  const f32x2_t v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
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

// occupancy target: three workgroups per CU (at most 168 registers per lane)
// where the gathered rows of three fit in LDS, else two
template <int RBH, int TPW>
constexpr int attn_tiles_waves_per_simd() {
  return (RBH <= 5 && 3 * 2 * TPW * RBH * 1024 <= 150 * 1024) ? 3 : 2;
}

template <int RBH, int NW, int NMH, int TPW, int HPW>
__global__ __launch_bounds__(NW * 64, (attn_tiles_waves_per_simd<RBH, TPW>())) void k_attn_tiles(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ bases_k, const uint16_t* __restrict__ bases_v,
    const uint16_t* __restrict__ coef_k, const uint16_t* __restrict__ coef_v, const int32_t* __restrict__ idx_all,
    int64_t idx_stride, float* __restrict__ part_ml, float* __restrict__ part_o, int n_proc, int nsplit, int ngroups,
    int G, int hq, int hkv, int nb, int rank, int R, int s_sink, int64_t L, int64_t cap, int bases_shared,
    double rope_ratio) {
  constexpr int DH = NW * 32;                      // NMH = ceil(G / 4): 4 heads per MFMA row group
  static_assert(TPW % 2 == 0, "tiles are processed in pairs");
  // ---- work item: HPW consecutive KV heads of group (sequence, split); the
  // workgroups of one group share an XCD ---------------------------------------------------
  const int id = blockIdx.x;
  const int nhp = hkv / HPW;
  const int xcd = id & 7, r8 = id >> 3;
  const int hp = r8 % nhp;
  const int grp_id = (r8 / nhp) * 8 + xcd;
  if (grp_id >= ngroups) return;
  const int b = grp_id / nsplit, split = grp_id % nsplit;

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int slot = lane & 15, kg = lane >> 4;
  const int Dp = hkv * DH, Dg = Dp / nb;
  const int bgrp = (hp * HPW) / (hkv / nb);        // the HPW heads share one basis group
  const int kb0 = bgrp * rank / 32;                // first latent block of the group
  const int tile0 = split * TPW;
  const int ntile = (n_proc + 15) / 16;
  const int nt = min(TPW, ntile - tile0);          // >= 1 (nsplit = ceil(ntile / TPW))

  __shared__ __align__(16) uint16_t gk[TPW][RBH][512];   // gathered C^K blocks: [token slot][32 columns]
  __shared__ __align__(16) uint16_t gv[TPW][RBH][512];
  __shared__ int32_t sidx[TPW * 16];
  __shared__ float xl[2][NW][NMH][4][16];                // partial logits [tile of pair][wave][mh][head][slot]
  __shared__ __align__(16) uint16_t ps[2][NMH][4][2][16]; // P parts [tile of pair][mh][head][hi|lo][slot]

  // ---- 1. index list, then every gather of the workgroup ---------------------------------
  const int32_t* idx = idx_all + (int64_t)b * idx_stride;
  for (int i = threadIdx.x; i < TPW * 16; i += NW * 64)
    sidx[i] = (tile0 * 16 + i < n_proc) ? idx[tile0 * 16 + i] : -1;
  // the query dims of this lane's k-group: f_v = 16 w + 4 kg + v and f_v + d_h / 2
  const int fq = 16 * w + 4 * kg;
  uint64_t Ff[4];
  rope_freqs_fixed(rope_ratio, fq, Ff);
  const int64_t pos_q = s_sink + L - 1;
  const int64_t boff = (bases_shared ? 0 : (int64_t)b * Dp * rank) + (int64_t)bgrp * Dg * rank;
  lds_barrier();                                   // sidx visible
  {
    // wave w gathers tiles w, w + NW, ...: per tile one row offset, then the
    // 2 x RBH wave loads of 1 KiB at constant distances
    const uint16_t* ckb = coef_k + (int64_t)b * cap * R + (int64_t)kb0 * 512;
    const uint16_t* cvb = coef_v + (int64_t)b * cap * R + (int64_t)kb0 * 512;
    const int tq = lane >> 2, quarter = lane & 3;
#pragma unroll
    for (int t0 = 0; t0 < TPW; t0 += NW) {
      const int t = t0 + w;
      if (t < TPW) {                               // wave-uniform
        const int32_t x = sidx[t * 16 + tq];
        const uint32_t tok = x < 0 ? 0u : (uint32_t)x;
        const int64_t off = (int64_t)(tok >> 4) * 16 * R + (tok & 15) * 32 + quarter * 8;
#pragma unroll
        for (int kb = 0; kb < RBH; ++kb) {
          // (destinations through local pointers: the builtin's LDS operand
          // must be a plain pointer for the host pass to keep the kernel stub)
          uint16_t* dk = &gk[t][kb][0];
          uint16_t* dvp = &gv[t][kb][0];
          __builtin_amdgcn_global_load_lds(ckb + off + kb * 512, dk, 16, 0, 0);
          __builtin_amdgcn_global_load_lds(cvb + off + kb * 512, dvp, 16, 0, 0);
        }
      }
    }
  }
  const float inv_sqrt_d = 1.0f / sqrtf((float)DH);

  for (int jj = 0; jj < HPW; ++jj) {
  const int j = hp * HPW + jj;
  const int row0 = (j % (hkv / nb)) * DH;          // first basis row of head j in its group
  // bases (registers): A operands of K^ (row = dim) and B operands of V^
  // (column = dim) read the same 16 bytes
  Op8 bk[2][RBH], bv[2][RBH];
#pragma unroll
  for (int m = 0; m < 2; ++m) {
    const int d = 16 * (w + m * NW) + slot;
#pragma unroll
    for (int kb = 0; kb < RBH; ++kb) {
      const int64_t o = boff + (int64_t)(row0 + d) * rank + kb * 32 + kg * 8;
      bk[m][kb].u = *reinterpret_cast<const uint4*>(bases_k + o);
      bv[m][kb].u = *reinterpret_cast<const uint4*>(bases_v + o);
    }
  }
  uint2 qlo[NMH], qhi[NMH];
#pragma unroll
  for (int mh = 0; mh < NMH; ++mh) {
    const int h = min(4 * mh + (slot >> 2), G - 1);
    const uint16_t* qp = q + ((int64_t)b * hq + (int64_t)j * G + h) * DH + fq;
    qlo[mh] = *reinterpret_cast<const uint2*>(qp);
    qhi[mh] = *reinterpret_cast<const uint2*>(qp + DH / 2);
  }
  // ---- 2. rotated query as the A operand of the logits (overlaps the gathers) ------------
  Op8 aq[NMH];
  {
    const int part = slot & 3;
#pragma unroll
    for (int mh = 0; mh < NMH; ++mh) {
      const bool live = (4 * mh + (slot >> 2) < G) && part < 2;
      const uint32_t lo4[2] = {qlo[mh].x, qlo[mh].y}, hi4[2] = {qhi[mh].x, qhi[mh].y};
      float xr[8];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const float xl0 = bf16_bits_to_f32((lo4[v >> 1] >> (16 * (v & 1))) & 0xFFFFu);
        const float xh0 = bf16_bits_to_f32((hi4[v >> 1] >> (16 * (v & 1))) & 0xFFFFu);
        float c, s;
        rope_cs_fixed(pos_q, Ff[v], c, s);
        xr[v] = xl0 * c - xh0 * s;
        xr[4 + v] = xh0 * c + xl0 * s;
      }
      Op8 hi, lo;
      split2_f32x8(xr, hi, lo);
      aq[mh].u = live ? (part == 0 ? hi.u : lo.u) : make_uint4(0, 0, 0, 0);
    }
  }
  float Mrun[NMH], lrun[NMH];
  floatx4 oacc[NMH][2];
#pragma unroll
  for (int mh = 0; mh < NMH; ++mh) {
    Mrun[mh] = -INFINITY;
    lrun[mh] = 0.f;
    oacc[mh][0] = floatx4{0.f, 0.f, 0.f, 0.f};
    oacc[mh][1] = floatx4{0.f, 0.f, 0.f, 0.f};
  }
  if (jj == 0) {
    __builtin_amdgcn_s_waitcnt(0);                 // this wave's gathers have landed
    __syncthreads();                               // everyone's
  }

  // ---- 3-5. tile pairs ----------------------------------------------------------------
  for (int tp = 0; tp < nt; tp += 2) {
    floatx4 dv[2][2];                              // V^ of the pair: [tile][dim block]
    float sl[2][NMH];
    int32_t tokv[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int t = tp + u;
      tokv[u] = sidx[t * 16 + slot];
      // K^ for the wave's two dimension blocks: lane (token slot, kg) gets dims 4 kg + v
      floatx4 dk[2];
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        dk[m] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < RBH; ++kb) {
          Op8 c;
          c.u = *reinterpret_cast<const uint4*>(&gk[t][kb][slot * 32 + kg * 8]);
          dk[m] = mfma16x16x32(bk[m][kb], c, dk[m]);
        }
      }
      // RoPE at the token's original position
      const int64_t pos = s_sink + (tokv[u] < 0 ? 0 : (int64_t)tokv[u]);
      float kr[8];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        float c, s;
        rope_cs_fixed(pos, Ff[v], c, s);
        kr[v] = dk[0][v] * c - dk[1][v] * s;
        kr[4 + v] = dk[1][v] * c + dk[0][v] * s;
      }
      Op8 khi, klo;
      split2_f32x8(kr, khi, klo);
      // partial logits over this wave's 32 dims: lane (slot, kg) <- head 4 mh + kg
#pragma unroll
      for (int mh = 0; mh < NMH; ++mh) {
        floatx4 dl = mfma16x16x32(aq[mh], khi, floatx4{0.f, 0.f, 0.f, 0.f});
        dl = mfma16x16x32(aq[mh], klo, dl);
        xl[u][w][mh][kg][slot] = dl[0] + dl[1];
      }
      // V^ of this tile: lane (dim, kg) gets tokens 4 kg + v
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        dv[u][m] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < RBH; ++kb) {
          Op8 c;
          c.u = *reinterpret_cast<const uint4*>(&gv[t][kb][slot * 32 + kg * 8]);
          dv[u][m] = mfma16x16x32(c, bv[m][kb], dv[u][m]);
        }
      }
    }
    lds_barrier();                                 // partial logits of every wave
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int mh = 0; mh < NMH; ++mh) {
        float s = 0.f;
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) s += xl[u][ww][mh][kg][slot];
        const bool valid = tokv[u] >= 0 && 4 * mh + kg < G;
        sl[u][mh] = valid ? s * inv_sqrt_d : -INFINITY;
      }
    // online softmax of (token slot, head 4 mh + kg); the 16 slots share the maximum
#pragma unroll
    for (int mh = 0; mh < NMH; ++mh) {
      const float pmax = slot_max16(fmaxf(sl[0][mh], sl[1][mh]));
      if (pmax > Mrun[mh]) {                       // uniform within the row of head kg
        const float alpha = __expf(Mrun[mh] - pmax);   // 0 when the maximum was -inf
        lrun[mh] *= alpha;
        oacc[mh][0] *= alpha;
        oacc[mh][1] *= alpha;
        Mrun[mh] = pmax;
      }
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const float p = (sl[u][mh] == -INFINITY) ? 0.f : __expf(sl[u][mh] - Mrun[mh]);
        lrun[mh] += p;
        if (w == 0) {                              // one wave stages P for all
          const uint32_t ph = pack_bf16x2(p, 0.f);
          ps[u][mh][kg][0][slot] = (uint16_t)ph;
          ps[u][mh][kg][1][slot] = (uint16_t)pack_bf16x2(p - __uint_as_float(ph << 16), 0.f);
        }
      }
    }
    lds_barrier();                                 // P staged
    // P V^: A = P parts (row 4 h + part, k = tokens 4 kg + v of both tiles), B = V^ as
    // hi / lo bf16 parts
    Op8 vhi[2], vlo[2];
#pragma unroll
    for (int m = 0; m < 2; ++m) {
      const float x[8] = {dv[0][m][0], dv[0][m][1], dv[0][m][2], dv[0][m][3],
                          dv[1][m][0], dv[1][m][1], dv[1][m][2], dv[1][m][3]};
      split2_f32x8(x, vhi[m], vlo[m]);
    }
#pragma unroll
    for (int mh = 0; mh < NMH; ++mh) {
      const int hh = slot >> 2, part = slot & 3;
      Op8 ap;
      if (part < 2) {
        const uint2 a0 = *reinterpret_cast<const uint2*>(&ps[0][mh][hh][part][4 * kg]);
        const uint2 a1 = *reinterpret_cast<const uint2*>(&ps[1][mh][hh][part][4 * kg]);
        ap.u = make_uint4(a0.x, a0.y, a1.x, a1.y);
      } else {
        ap.u = make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        oacc[mh][m] = mfma16x16x32(ap, vhi[m], oacc[mh][m]);
        oacc[mh][m] = mfma16x16x32(ap, vlo[m], oacc[mh][m]);
      }
    }
  }

  // ---- partial results of the split --------------------------------------------------
#pragma unroll
  for (int mh = 0; mh < NMH; ++mh) {
    const float lsum = slot_sum16(lrun[mh]);
    const int hl = 4 * mh + kg;                    // head within the group of this lane's row
    if (hl < G) {
      const int h = j * G + hl;
      const int64_t pb = ((int64_t)b * hq + h) * kMaxSplit + split;
      if (w == 0 && slot == 0) {
        part_ml[pb * 2 + 0] = Mrun[mh];
        part_ml[pb * 2 + 1] = lsum;
      }
#pragma unroll
      for (int m = 0; m < 2; ++m) part_o[pb * DH + 16 * (w + m * NW) + slot] = oacc[mh][m][0] + oacc[mh][m][1];
    }
  }
  }   // heads of the workgroup
}

}  // namespace s4r

namespace s4r {

// which configurations the MFMA attention kernel covers (bf16 storage)
inline int attn_tiles_per_wg(int ntile) { return ntile <= kMaxSplit * 4 ? 4 : (ntile <= kMaxSplit * 8 ? 8 : 0); }

template <int RBH, int NW, int NMH, int TPW, int HPW>
static void launch_tiles_h(const Problem& P, const Workspace& ws, int64_t L, int m, int n_proc, const void* q,
                           const void* bk, const void* bv, const void* ck, const void* cv, hipStream_t st,
                           int* nsplit_out) {
  const int ntile = (n_proc + 15) / 16;
  const int nsplit = (ntile + TPW - 1) / TPW;
  const int ngroups = P.B * nsplit;
  const int nwg = 8 * (P.hkv / HPW) * ((ngroups + 7) / 8);
  hipLaunchKernelGGL((k_attn_tiles<RBH, NW, NMH, TPW, HPW>), dim3(nwg), dim3(NW * 64), 0, st, (const uint16_t*)q,
                     (const uint16_t*)bk, (const uint16_t*)bv, (const uint16_t*)ck, (const uint16_t*)cv, ws.idx,
                     (int64_t)m, ws.part_ml, ws.part_o, n_proc, nsplit, ngroups, P.G, P.hq, P.hkv, P.nb, P.rank, P.R,
                     P.s, L, P.cap, P.bases_shared, rope_ratio(P));
  *nsplit_out = nsplit;
}

// one KV head per workgroup: a workgroup that walks two heads over the same
// gathered rows halves the gather traffic but doubles its critical path, and
// measured slower on MI355X (the HPW parameter keeps that variant available)
template <int RBH, int NW, int NMH, int TPW>
static void launch_tiles_t(const Problem& P, const Workspace& ws, int64_t L, int m, int n_proc, const void* q,
                           const void* bk, const void* bv, const void* ck, const void* cv, hipStream_t st,
                           int* nsplit_out) {
  launch_tiles_h<RBH, NW, NMH, TPW, 1>(P, ws, L, m, n_proc, q, bk, bv, ck, cv, st, nsplit_out);
}

template <int NW, int NMH, int TPW>
static bool dispatch_tiles_rb(const Problem& P, const Workspace& ws, int64_t L, int m, int n_proc, const void* q,
                              const void* bk, const void* bv, const void* ck, const void* cv, hipStream_t st,
                              int* ns) {
  switch (P.rank / 32) {
    case 1: launch_tiles_t<1, NW, NMH, TPW>(P, ws, L, m, n_proc, q, bk, bv, ck, cv, st, ns); return true;
    case 2: launch_tiles_t<2, NW, NMH, TPW>(P, ws, L, m, n_proc, q, bk, bv, ck, cv, st, ns); return true;
    case 3: launch_tiles_t<3, NW, NMH, TPW>(P, ws, L, m, n_proc, q, bk, bv, ck, cv, st, ns); return true;
    case 4: launch_tiles_t<4, NW, NMH, TPW>(P, ws, L, m, n_proc, q, bk, bv, ck, cv, st, ns); return true;
    case 5: launch_tiles_t<5, NW, NMH, TPW>(P, ws, L, m, n_proc, q, bk, bv, ck, cv, st, ns); return true;
    case 6: launch_tiles_t<6, NW, NMH, TPW>(P, ws, L, m, n_proc, q, bk, bv, ck, cv, st, ns); return true;
    case 8: launch_tiles_t<8, NW, NMH, TPW>(P, ws, L, m, n_proc, q, bk, bv, ck, cv, st, ns); return true;
    default: return false;
  }
}

// launches the split kernel for head dim 32 * NW; returns false when the
// configuration is not covered (the caller then uses the general kernel)
template <int NW>
static bool launch_tiles_dh(const Problem& P, const Workspace& ws, int64_t L, int m, int n_proc, const void* q,
                            const void* bk, const void* bv, const void* ck, const void* cv, hipStream_t st,
                            int* ns) {
  const int tpw = attn_tiles_per_wg((n_proc + 15) / 16);
  if (P.G > 8 || tpw == 0) return false;
  const bool two = P.G > 4;
  if (tpw == 4)
    return two ? dispatch_tiles_rb<NW, 2, 4>(P, ws, L, m, n_proc, q, bk, bv, ck, cv, st, ns)
               : dispatch_tiles_rb<NW, 1, 4>(P, ws, L, m, n_proc, q, bk, bv, ck, cv, st, ns);
  return two ? dispatch_tiles_rb<NW, 2, 8>(P, ws, L, m, n_proc, q, bk, bv, ck, cv, st, ns)
             : dispatch_tiles_rb<NW, 1, 8>(P, ws, L, m, n_proc, q, bk, bv, ck, cv, st, ns);
}

}  // namespace s4r
