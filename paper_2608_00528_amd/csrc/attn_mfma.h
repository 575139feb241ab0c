// Fused sparse reconstruction + split attention for bf16 storage on gfx950
// (Section 3.2.3): every contraction on bf16 MFMA.
//
// One workgroup per (split, KV head, sequence), NW = d_h / 32 waves, tpw
// tiles of 16 selected tokens (tpw chosen so that all workgroups fit in one
// round of the chip).  The work items are laid out over a 1-D grid so that the
// workgroups of one (sequence, split) land on the same XCD (workgroup i runs
// on XCD i % 8): the gathered coefficient rows are then fetched from HBM once
// per XCD and re-read from its L2 by the other heads.
//
//   1. the split's index list goes to LDS; the tiles are gathered in pairs
//      into two LDS buffers (even pairs in one, odd pairs in the other) with
//      16-byte buffer->LDS loads (lane l of a wave load lands at byte 16 l of
//      the destination, so one wave load writes one 16-token x 32-column block;
//      lane l fetches quarter (l % 4) ^ ((l / 8) % 4) of token l / 4's row, an
//      XOR swizzle that keeps the operand reads free of bank conflicts).  One
//      32-bit lane offset per tile serves all of a tile's blocks, whose 1 KiB
//      steps go in the scalar offset: no 64-bit address arithmetic per block.
//      Pairs 0 and 1 are requested up front; pair
//      p + 2 as soon as every wave has read pair p, so the gathers overlap
//      the arithmetic of pair p + 1;
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
//   5. V^ = C^V B^V_j^T (D[token][dim]) of two tiles, rounded once to bf16,
//      forms the B operand of P V^, with P rounded once to bf16 (moved
//      between lanes with permutes) as A rows 4 h; the output rows of
//      head h land in the lanes that own head h's softmax state, which
//      rescale them when its maximum grows.
// Steps 3-5 are software-pipelined over the tile pairs: after one barrier
// per pair, a wave runs the softmax and P V^ of pair p (from the partial
// logits every wave wrote, double-buffered by pair parity) and then K^, RoPE,
// the partial logits and V^ of pair p + 1, so the two chains' instructions
// are independent within one basic block (the rescale is branch-free).
//
// Precision: the logits' operands carry about 16 significant bits each (the
// rotated query and K~ as hi / lo parts), since a logit error enters the
// weights through the exponential: with heavy-tailed coefficients logits
// reach tens, where a bf16 K~ (relative error 2^-9 per element) moved the
// output by 1.3e-2, most of the 2e-2 bound for bf16 storage.  V^ enters the
// output linearly, so it is rounded once to bf16 (at most 2^-9 relative per
// element, a few 1e-3 at the output), and so is P (each weight within 2^-9
// relative; the normaliser sums the unrounded weights): the largest output
// error over the parity cases went from 4e-3 to 6e-3; every sum is fp32.
//
// Each split writes its (max, sum) and unnormalised output per head.
#pragma once

#include <type_traits>

#include "attn_common.h"

namespace s4r {

// occupancy target (workgroups per CU = waves per SIMD): three (at most 168
// registers per lane; the four tile slots of a workgroup take 4 * (RBH + RBV)
// KiB of LDS) while the operands fit without spilling, else two (one for the
// widest eight-head case)
constexpr int attn_tiles_waves(int rbh, int rbv, int nmh) {
  if (nmh == 1) return (rbh + rbv <= 10 && rbh <= 6 && rbv <= 6) ? 3 : 2;
  return rbh + rbv <= 6 ? 3 : (rbh + rbv < 16 ? 2 : 1);
}
template <int RBH, int RBV, int NMH>
constexpr int attn_tiles_waves_per_simd() {
  return attn_tiles_waves(RBH, RBV, NMH);
}

// s_waitcnt vmcnt(N) alone (gfx9 encoding: expcnt and lgkmcnt not waited)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is six bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// one wave's gather of one 16-token tile into slot u of a pair buffer: its RBH
// 1 KiB blocks of C^K and RBV of C^V as 16-byte buffer->LDS loads through the
// resources rsk / rsv (lane l: token l / 4, quarter (l % 4) ^ ((l / 8) % 4) of
// the 32 columns, stored at byte 16 l; a token past the list reads row 0,
// never used).  T is the tile's number within the workgroup.  The LDS
// destinations are named directly (LDS pointers for the builtin).
#define S4R_GATHER_TILE(GK, GV, U, T)                                                       \
  do {                                                                                       \
    const int32_t x_ = tok_at((T) * 16 + (lane >> 2));                                       \
    const uint32_t tok_ = x_ < 0 ? 0u : (uint32_t)x_;                                        \
    const uint32_t in_ = ((tok_ & 15) * 32 + (((lane & 3) ^ ((lane >> 3) & 3)) * 8)) * 2;   \
    const uint32_t offk_ = (tok_ >> 4) * (32u * R) + in_;                                    \
    const uint32_t offv_ = (tok_ >> 4) * (32u * Rv) + in_;                                   \
    _Pragma("unroll") for (int kb = 0; kb < RBH; ++kb)                                       \
      __builtin_amdgcn_raw_ptr_buffer_load_lds(                                              \
          rsk, (__attribute__((address_space(3))) void*)&GK[U][kb][0], 16, offk_, kb * 1024, 0, 0); \
    _Pragma("unroll") for (int kb = 0; kb < RBV; ++kb)                                       \
      __builtin_amdgcn_raw_ptr_buffer_load_lds(                                              \
          rsv, (__attribute__((address_space(3))) void*)&GV[U][kb][0], 16, offv_, kb * 1024, 0, 0); \
  } while (0)

// IDENT: every token of the sequence in order (full reconstruction,
// Appendix B.1): token i of the workgroup's tiles is tile0 * 16 + i, no index
// list is read and the tiles per workgroup are not bounded by its LDS slot.
// RBH / RBV: 32-column blocks of one head's key / value basis group (they
// differ when the ranks are asymmetric, Appendix D.2).
template <int RBH, int RBV, int NW, int NMH, bool IDENT>
__global__ __launch_bounds__(NW * 64, (attn_tiles_waves_per_simd<RBH, RBV, NMH>())) void k_attn_tiles(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ bases_k, const uint16_t* __restrict__ bases_v,
    const uint16_t* __restrict__ coef_k, const uint16_t* __restrict__ coef_v, const int32_t* __restrict__ idx_all,
    int64_t idx_stride, float* __restrict__ part_ml, float* __restrict__ part_o, int n_proc, int tpw, int nsplit,
    int ngroups, int G, int hq, int hkv, int nb, int rank, int R, int rank_v, int Rv, int s_sink, int64_t L,
    int64_t cap,
    int bases_shared, double rope_ratio, Lens lens) {
  constexpr int DH = NW * 32;                      // NMH = ceil(G / 4): 4 heads per MFMA row group
  static_assert(NW >= 2, "a tile pair is gathered by two waves");
  // ---- work item: KV head j of group (sequence, split); the workgroups of
  // one group share an XCD ------------------------------------------------------------------
  const int id = blockIdx.x;
  const int xcd = id & 7, r8 = id >> 3;
  const int j = r8 % hkv;
  const int grp_id = (r8 / hkv) * 8 + xcd;
  if (grp_id >= ngroups) return;
  const int b = grp_id / nsplit, split = grp_id % nsplit;
  L = len_of(lens, b, L);

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int slot = lane & 15, kg = lane >> 4;
  // where token slot's k-group kg sits in a gathered block: quarter
  // kg ^ ((slot >> 1) & 3) of its 64-byte row (the gathers store it there), so
  // the eight lanes of one 128-byte LDS read cycle hit eight distinct bank
  // groups instead of two
  const int kq = slot * 32 + (kg ^ ((slot >> 1) & 3)) * 8;   // element offset in a block
  const int Dp = hkv * DH, Dg = Dp / nb;
  const int bgrp = j / (hkv / nb);                 // basis group of head j
  const int kb0 = bgrp * rank / 32;                // its first latent block (keys)
  const int kbv0 = bgrp * rank_v / 32;             // (values)
  const int row0 = (j % (hkv / nb)) * DH;          // first basis row of head j in its group
  const int tile0 = split * tpw;
  const int ntile = (n_proc + 15) / 16;
  const int nt = min(tpw, ntile - tile0);          // >= 1 (nsplit = ceil(ntile / tpw))
  const int npair = (nt + 1) >> 1;

  // two pair buffers (even pairs in A, odd pairs in B) of gathered C^K / C^V
  // blocks [tile of pair][block][token slot][32 columns]: separate arrays, so
  // the loads refilling one buffer never hold up the reads of the other
  __shared__ __align__(16) uint16_t gkA[2][RBH][512], gvA[2][RBV][512];
  __shared__ __align__(16) uint16_t gkB[2][RBH][512], gvB[2][RBV][512];
  __shared__ int32_t sidx[kTileMax * 16];
  __shared__ float xl[2][2][NW][NMH][4][16];             // partial logits [pair & 1][tile of pair][wave][mh][head][slot]

  // ---- 1. index list, bases and query requested; then the first two pairs' gathers ---------
  int32_t xi[kTileMax * 16 / (NW * 64)];
  if constexpr (!IDENT) {
    const int32_t* idx = idx_all + (int64_t)b * idx_stride;
#pragma unroll
    for (int k = 0; k < kTileMax * 16 / (NW * 64); ++k) {
      const int i = threadIdx.x + k * NW * 64;
      xi[k] = idx[min(tile0 * 16 + i, n_proc - 1)];
    }
  }
  // token of slot i of this workgroup's tiles (-1: past the list)
  auto tok_at = [&](int i) __attribute__((always_inline)) -> int32_t {
    if constexpr (IDENT) {
      const int x = tile0 * 16 + i;
      return (i < nt * 16 && x < n_proc) ? x : -1;
    } else {
      return sidx[i];
    }
  };
  // bases (registers): A operands of K^ (row = dim) and B operands of V^
  // (column = dim) read the same 16-byte pattern of their basis
  const int64_t boff = (bases_shared ? 0 : (int64_t)b * Dp * rank) + (int64_t)bgrp * Dg * rank;
  const int64_t boffv = (bases_shared ? 0 : (int64_t)b * Dp * rank_v) + (int64_t)bgrp * Dg * rank_v;
  Op8 bk[2][RBH], bv[2][RBV];
#pragma unroll
  for (int m = 0; m < 2; ++m) {
    const int d = 16 * (w + m * NW) + slot;
#pragma unroll
    for (int kb = 0; kb < RBH; ++kb)
      bk[m][kb].u = *reinterpret_cast<const uint4*>(bases_k + boff + (int64_t)(row0 + d) * rank + kb * 32 + kg * 8);
#pragma unroll
    for (int kb = 0; kb < RBV; ++kb)
      bv[m][kb].u =
          *reinterpret_cast<const uint4*>(bases_v + boffv + (int64_t)(row0 + d) * rank_v + kb * 32 + kg * 8);
  }
  // the query dims of this lane's k-group: f_v = 16 w + 4 kg + v and f_v + d_h / 2
  const int fq = 16 * w + 4 * kg;
  uint2 qlo[NMH], qhi[NMH];
#pragma unroll
  for (int mh = 0; mh < NMH; ++mh) {
    const int h = min(4 * mh + (slot >> 2), G - 1);
    const uint16_t* qp = q + ((int64_t)b * hq + (int64_t)j * G + h) * DH + fq;
    qlo[mh] = *reinterpret_cast<const uint2*>(qp);
    qhi[mh] = *reinterpret_cast<const uint2*>(qp + DH / 2);
  }
  if constexpr (!IDENT) {
#pragma unroll
    for (int k = 0; k < kTileMax * 16 / (NW * 64); ++k) {
      const int i = threadIdx.x + k * NW * 64;
      sidx[i] = (i < nt * 16 && tile0 * 16 + i < n_proc) ? xi[k] : -1;
    }
  }
  uint64_t Ff[4];
  rope_freqs_fixed(rope_ratio, fq, Ff);
  const int64_t pos_q = s_sink + L - 1;
  lds_barrier();                                   // sidx visible
  const uint16_t* ckb = coef_k + (int64_t)b * cap * R + (int64_t)kb0 * 512;
  const uint16_t* cvb = coef_v + (int64_t)b * cap * Rv + (int64_t)kbv0 * 512;
  // buffer resources over the sequence's caches (byte offsets below cap * R * 2
  // <= 2^32 by the capacity limit; no range check): one 32-bit lane offset per
  // tile row serves every 32-column block, whose 1 KiB steps go in the scalar offset
  const __amdgpu_buffer_rsrc_t rsk = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(ckb), (short)0, -1, 0x00020000);
  const __amdgpu_buffer_rsrc_t rsv = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(cvb), (short)0, -1, 0x00020000);
  // tile t is gathered by wave t % NW; pairs 0 and 1 now (every wave issues
  // the same number of loads), pair p + 2 once pair p has been read
#pragma unroll
  for (int t0 = 0; t0 < 4; t0 += NW) {
    const int t = t0 + w;
    if (t < 2)
      S4R_GATHER_TILE(gkA, gvA, t, t);
    else
      S4R_GATHER_TILE(gkB, gvB, t - 2, t);
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
  const float inv_sqrt_d = 1.0f / sqrtf((float)DH);

  // ---- 3-5. software-pipelined over tile pairs: the softmax and P V^ of pair p
  // run beside the reconstruction of pair p + 1, with one barrier per pair ------------------
  // stage: K^, RoPE and the wave's partial logits of pair q (buffer BUF) -> xl[q & 1]; V^ -> dv
  auto stage_pair = [&](const int q, auto buf, floatx4 (&dv)[2][2], int32_t (&tokv)[2])
                        __attribute__((always_inline)) {
    constexpr int BUF = decltype(buf)::value;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      tokv[u] = tok_at((2 * q + u) * 16 + slot);
      // K^ for the wave's two dimension blocks: lane (token slot, kg) gets dims 4 kg + v
      floatx4 dk[2];
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        dk[m] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < RBH; ++kb) {
          Op8 c;
          c.u = *reinterpret_cast<const uint4*>(BUF == 0 ? &gkA[u][kb][kq] : &gkB[u][kb][kq]);
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
        xl[q & 1][u][w][mh][kg][slot] = dl[0] + dl[1];
      }
      // V^ of this tile: lane (dim, kg) gets tokens 4 kg + v
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        dv[u][m] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < RBV; ++kb) {
          Op8 c;
          c.u = *reinterpret_cast<const uint4*>(BUF == 0 ? &gvA[u][kb][kq] : &gvB[u][kb][kq]);
          dv[u][m] = mfma16x16x32(c, bv[m][kb], dv[u][m]);
        }
      }
    }
  };
  // finish: online softmax of pair q from every wave's partial logits, then P V^
  auto finish_pair = [&](const int q, const floatx4 (&dv)[2][2], const int32_t (&tokv)[2])
                         __attribute__((always_inline)) {
    float sl[2][NMH];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int mh = 0; mh < NMH; ++mh) {
        float s = 0.f;
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) s += xl[q & 1][u][ww][mh][kg][slot];
        const bool valid = tokv[u] >= 0 && 4 * mh + kg < G;
        sl[u][mh] = valid ? s * inv_sqrt_d : -INFINITY;
      }
    // online softmax of (token slot, head 4 mh + kg); the 16 slots share the maximum
    uint32_t phi[NMH];
#pragma unroll
    for (int mh = 0; mh < NMH; ++mh) {
      // rescale without a branch (the pair's finish and the next pair's staging
      // stay one basic block, so their instructions can interleave)
      const float mnew = fmaxf(Mrun[mh], slot_max16(fmaxf(sl[0][mh], sl[1][mh])));
      const float alpha = (mnew == -INFINITY) ? 1.f : __expf(Mrun[mh] - mnew);   // 0 when the maximum was -inf
      lrun[mh] *= alpha;
      oacc[mh][0] *= alpha;
      oacc[mh][1] *= alpha;
      Mrun[mh] = mnew;
      float pr[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        pr[u] = (sl[u][mh] == -INFINITY) ? 0.f : __expf(sl[u][mh] - Mrun[mh]);
        lrun[mh] += pr[u];
      }
      // P of both tiles rounded to bf16, packed (tile 0 low half, tile 1 high half)
      phi[mh] = pack_bf16x2(pr[0], pr[1]);
    }
    // P V^: A = P (row 4 h, k = tokens 4 kg + v of both tiles; rows 4 h + 1..3
    // zero), B = V^ rounded to bf16.  Every wave builds its own A operand from
    // the softmax lanes with lane permutes (lane (row 4 h, k-group c) takes
    // token 4 c + v, head h from lane (4 c + v) + 16 h), so P never goes
    // through LDS and needs no barrier
    Op8 vb16[2];
#pragma unroll
    for (int m = 0; m < 2; ++m) {
      const float x[8] = {dv[0][m][0], dv[0][m][1], dv[0][m][2], dv[0][m][3],
                          dv[1][m][0], dv[1][m][1], dv[1][m][2], dv[1][m][3]};
      round_f32x8(x, vb16[m]);
    }
    const int hh = slot >> 2, part = slot & 3;
#pragma unroll
    for (int mh = 0; mh < NMH; ++mh) {
      uint32_t r[4];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int src = ((4 * kg + v) + 16 * hh) << 2;
        const uint32_t rh = (uint32_t)__builtin_amdgcn_ds_bpermute(src, (int)phi[mh]);
        r[v] = part == 0 ? rh : 0u;
      }
      Op8 ap;
      ap.u = make_uint4((r[0] & 0xFFFFu) | (r[1] << 16), (r[2] & 0xFFFFu) | (r[3] << 16),
                        (r[0] >> 16) | (r[1] & 0xFFFF0000u), (r[2] >> 16) | (r[3] & 0xFFFF0000u));
#pragma unroll
      for (int m = 0; m < 2; ++m) oacc[mh][m] = mfma16x16x32(ap, vb16[m], oacc[mh][m]);
    }
  };
  // refill the buffer of pair q - 2 (free once every wave staged it) with pair q
  auto refill = [&](const int q, auto buf) __attribute__((always_inline)) {
    constexpr int BUF = decltype(buf)::value;
    if (q < npair) {
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int t = 2 * q + u;
        if (t % NW == w) {
          if constexpr (BUF == 0)
            S4R_GATHER_TILE(gkA, gvA, u, t);
          else
            S4R_GATHER_TILE(gkB, gvB, u, t);
        }
      }
    }
  };
  // iteration p: pair p + 1's rows have landed (the only gathers in flight),
  // every wave has staged pair p (xl[p & 1] complete, buffer of pair p free)
  auto iterate = [&](const int p, auto buf, floatx4 (&dv)[2][2], int32_t (&tokv)[2])
                     __attribute__((always_inline)) {
    constexpr int BUF = decltype(buf)::value;    // buffer of pair p
    wait_vmcnt<0>();
    lds_barrier();
    refill(p + 2, buf);
    floatx4 dvn[2][2];
    int32_t tokn[2];
    finish_pair(p, dv, tokv);
    stage_pair(p + 1, std::integral_constant<int, 1 - BUF>(), dvn, tokn);
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      tokv[u] = tokn[u];
#pragma unroll
      for (int m = 0; m < 2; ++m) dv[u][m] = dvn[u][m];
    }
  };
  // pair 0's rows (pair 1's gathers may stay in flight), then stage it
  if ((2 % NW) == w || (3 % NW) == w)
    wait_vmcnt<RBH + RBV>();                       // one tile's gathers
  else
    wait_vmcnt<0>();
  lds_barrier();
  floatx4 dvc[2][2];
  int32_t tokc[2];
  stage_pair(0, std::integral_constant<int, 0>(), dvc, tokc);
  int p = 0;
  for (; p + 2 < npair; p += 2) {
    iterate(p, std::integral_constant<int, 0>(), dvc, tokc);
    iterate(p + 1, std::integral_constant<int, 1>(), dvc, tokc);
  }
  if (p + 1 < npair) {
    iterate(p, std::integral_constant<int, 0>(), dvc, tokc);
    ++p;
  }
  lds_barrier();                                   // xl of the last pair complete
  finish_pair(p, dvc, tokc);
  wait_vmcnt<0>();                                 // no gather left in flight (a second pair that
                                                   // was never used when there is one pair only)

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
}

}  // namespace s4r

namespace s4r {

// tiles per workgroup: the smallest even count whose workgroups fit in one
// round of the chip (the kernel's workgroups per CU), at most kMaxSplit
// splits; with an index list, 0 when the list needs more than kTileMax tiles
// per workgroup (the general kernel then runs)
inline int attn_tiles_per_wg(const Problem& P, int ntile, bool ident) {
  const int slots = 256 * attn_tiles_waves(P.rank / 32, P.rank_v / 32, P.G > 4 ? 2 : 1);
  const int ns_target = std::max(1, slots / std::max(1, P.B * P.hkv));
  int tpw = (ntile + ns_target - 1) / ns_target;
  tpw = std::max(2, (tpw + 1) / 2 * 2);
  while ((ntile + tpw - 1) / tpw > kMaxSplit) tpw += 2;
  return (ident || tpw <= kTileMax) ? tpw : 0;
}

template <int RBH, int RBV, int NW, int NMH, bool IDENT>
static void launch_tiles_t(const Problem& P, const Workspace& ws, int64_t L, int m, int n_proc, int tpw,
                           const void* q, const void* bk, const void* bv, const void* ck, const void* cv,
                           hipStream_t st, int* nsplit_out) {
  const int ntile = (n_proc + 15) / 16;
  const int nsplit = (ntile + tpw - 1) / tpw;
  const int ngroups = P.B * nsplit;
  const int nwg = 8 * P.hkv * ((ngroups + 7) / 8);
  hipLaunchKernelGGL((k_attn_tiles<RBH, RBV, NW, NMH, IDENT>), dim3(nwg), dim3(NW * 64), 0, st, (const uint16_t*)q,
                     (const uint16_t*)bk, (const uint16_t*)bv, (const uint16_t*)ck, (const uint16_t*)cv, ws.idx,
                     (int64_t)m, ws.part_ml, ws.part_o, n_proc, tpw, nsplit, ngroups, P.G, P.hq, P.hkv, P.nb,
                     P.rank, P.R, P.rank_v, P.Rv, P.s, L, P.cap, P.bases_shared, rope_ratio(P), P.lens);
  *nsplit_out = nsplit;
}

template <int NW, int NMH, bool IDENT>
static bool dispatch_tiles_rb(const Problem& P, const Workspace& ws, int64_t L, int m, int n_proc, int tpw,
                              const void* q, const void* bk, const void* bv, const void* ck, const void* cv,
                              hipStream_t st, int* ns) {
#define S4R_TILES_CASE(RK, RV)                                                                         \
  if (P.rank / 32 == RK && P.rank_v / 32 == RV) {                                                     \
    static_assert(tiles_rank_pair(RK, RV), "pair not in the list");                                  \
    launch_tiles_t<RK, RV, NW, NMH, IDENT>(P, ws, L, m, n_proc, tpw, q, bk, bv, ck, cv, st, ns);       \
    return true;                                                                                      \
  }
  S4R_TILES_CASE(1, 1)
  S4R_TILES_CASE(2, 2)
  S4R_TILES_CASE(3, 3)
  S4R_TILES_CASE(4, 4)
  S4R_TILES_CASE(5, 5)
  S4R_TILES_CASE(6, 6)
  S4R_TILES_CASE(7, 7)
  S4R_TILES_CASE(8, 8)
  S4R_TILES_CASE(3, 5)
  S4R_TILES_CASE(2, 6)
  S4R_TILES_CASE(4, 6)
  S4R_TILES_CASE(3, 7)
  S4R_TILES_CASE(5, 7)
  S4R_TILES_CASE(4, 8)
#undef S4R_TILES_CASE
  return false;
}

// launches the split kernel for head dim 32 * NW over the index list in the
// workspace (ident: over every token); returns false when the configuration
// is not covered (the caller then uses the general kernel)
template <int NW>
static bool launch_tiles_dh(const Problem& P, const Workspace& ws, int64_t L, int m, int n_proc, const void* q,
                            const void* bk, const void* bv, const void* ck, const void* cv, hipStream_t st,
                            int* ns, bool ident) {
  const int tpw = attn_tiles_per_wg(P, (n_proc + 15) / 16, ident);
  if (P.G > 8 || tpw == 0) return false;
  if (ident)
    return P.G > 4 ? dispatch_tiles_rb<NW, 2, true>(P, ws, L, m, n_proc, tpw, q, bk, bv, ck, cv, st, ns)
                   : dispatch_tiles_rb<NW, 1, true>(P, ws, L, m, n_proc, tpw, q, bk, bv, ck, cv, st, ns);
  return P.G > 4 ? dispatch_tiles_rb<NW, 2, false>(P, ws, L, m, n_proc, tpw, q, bk, bv, ck, cv, st, ns)
                 : dispatch_tiles_rb<NW, 1, false>(P, ws, L, m, n_proc, tpw, q, bk, bv, ck, cv, st, ns);
}

}  // namespace s4r
