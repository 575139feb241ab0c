// Index selection of Section 3.2.3 on gfx950:
//   I_local  = [max(L - W, 0), L)
//   I_global = the k_eff = min(k, max(L - W, 0)) largest scores of
//              [0, L - W), equal scores going to the lower position
//   idx      = sorted(I_global) ++ I_local
//
// Scores are non-negative fp32, so their bit patterns (sign bit shifted out)
// order like the values;
// a candidate is the composite (key << 32) | ~position, unique, and larger
// exactly when it goes first (higher score, then lower position).
//
// A 2048-bin histogram of the top 11 key bits (built by the relevance kernel
// or k_hist_scores) fixes the boundary bin b1: count(bins > b1) < k_eff <=
// count(bins >= b1).  Then two kernels, both one workgroup per 2048 positions:
//   k_select_classify  marks the positions above b1 in a bitmap (its words
//                      built with lane shuffles), counts them per chunk,
//                      lists the chunk's b1 candidates and adds their next 11
//                      key bits to a second histogram (global atomics);
//   k_select_finish    every workgroup derives the same rule from the second
//                      histogram: candidates above the boundary sub-bin b2
//                      are chosen, and of those in b2 (usually a handful: only
//                      exact ties share all 22 bits) the need3 largest
//                      composites, ranked exactly (a radix select when there
//                      are many).  Counting the chosen candidates per chunk
//                      gives every chunk's output offset; the workgroup
//                      writes its own chunk's positions in ascending order.
// Integer work on the given scores: bit-exact and deterministic.
#include "s4r_device.h"
#include "s4r_internal.h"
#include "select_key.h"

namespace s4r {

constexpr int kSelThreads = 256;
constexpr int kSelPer = kSelChunk / kSelThreads;   // consecutive positions per thread (8)
constexpr int kS3Cap = 1024;                       // level-3 candidates ranked by counting
constexpr int kSubShift = kHistShift - 11;         // the next 11 key bits (level 2)

// block-wide exclusive prefix sum of one value per thread (wave shuffles,
// then the wave totals through LDS); returns the block total
__device__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* scratch /* >= 4 */, uint32_t& excl) {
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  uint32_t x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = (uint32_t)__builtin_amdgcn_ds_bpermute(max(lane - o, 0) << 2, (int)x);
    if (lane >= o) x += y;
  }
  if (lane == 63) scratch[wave] = x;
  lds_barrier();
  uint32_t off = 0, total = 0;
#pragma unroll
  for (int w = 0; w < kSelThreads / 64; ++w) {
    const uint32_t sw = scratch[w];
    if (w < wave) off += sw;
    total += sw;
  }
  excl = off + x - v;
  lds_barrier();
  return total;
}

// boundary bin of a 2048-bin histogram held as nc <= NC copies (summed here):
// the highest bin b with count(bins >= b) >= kk; `above` = count(bins > b).
// The bins are loaded with independent 16-byte loads (8 consecutive bins of
// every copy per thread, thread 0 = top bins; copies past nc repeat the last
// one's address, cache hits, and are not added).
template <int NC>
__device__ void find_boundary(const uint32_t* __restrict__ hist, int nc, uint32_t kk, uint32_t* scratch, int& b1,
                              uint32_t& above) {
  constexpr int per = kHistBins / kSelThreads;
  static_assert(per == 8, "two 16-byte loads per copy");
  const int t = threadIdx.x;
  const int lo = kHistBins - per * (t + 1);          // this thread's lowest bin
  uint4 part[NC][2];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const uint4* hp = reinterpret_cast<const uint4*>(hist + min(c, nc - 1) * kHistBins + lo);
    part[c][0] = hp[0];
    part[c][1] = hp[1];
  }
  uint32_t cnt[per];                                 // cnt[i]: bin kHistBins - 1 - (t * per + i)
#pragma unroll
  for (int i = 0; i < per; ++i) cnt[i] = 0u;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const uint32_t v[per] = {part[c][0].x, part[c][0].y, part[c][0].z, part[c][0].w,
                             part[c][1].x, part[c][1].y, part[c][1].z, part[c][1].w};
#pragma unroll
    for (int i = 0; i < per; ++i)
      if (c < nc) cnt[i] += v[per - 1 - i];
  }
  uint32_t sum = 0;
#pragma unroll
  for (int i = 0; i < per; ++i) sum += cnt[i];
  uint32_t excl;
  block_exclusive_scan(sum, scratch, excl);          // count strictly above this thread's bins
  __shared__ int s_b1;
  __shared__ uint32_t s_above;
  if (excl < kk && excl + sum >= kk) {
    uint32_t run = excl;
#pragma unroll
    for (int i = 0; i < per; ++i) {
      if (run < kk && run + cnt[i] >= kk) {
        s_b1 = kHistBins - 1 - (t * per + i);
        s_above = run;
      }
      run += cnt[i];
    }
  }
  lds_barrier();
  b1 = s_b1;
  above = s_above;
  lds_barrier();
}

// ---------------------------------------------------------------------------
// classify: one workgroup per 2048 positions
// ---------------------------------------------------------------------------
template <int NC>   // copies of the top-level histogram (a power of two, at most kHistCopies)
__global__ __launch_bounds__(kSelThreads) void k_select_classify(
    const float* __restrict__ scores, int64_t score_stride, uint32_t* __restrict__ hist_all,
    uint64_t* __restrict__ cand_all, uint32_t* __restrict__ bitmap_all, uint32_t* __restrict__ cand_count,
    uint32_t* __restrict__ above_count, uint32_t* __restrict__ sel_info, int64_t cand_stride, int64_t cnt_stride,
    int64_t cap, int L, int W, int k, Lens lens, int key_shift) {
  const int b = blockIdx.y, c = blockIdx.x;
  L = (int)len_of(lens, b, L);
  const int t = threadIdx.x, lane = t & 63;
  const int n_hist = max(L - W, 0);
  const int k_eff = min(k, n_hist);
  if (k_eff == 0 || c * kSelChunk >= n_hist) return;   // (a shorter sequence of a ragged batch)
  uint32_t* hist1 = hist_all + (int64_t)b * kHistStride;
  uint32_t* hist2 = hist1 + kHistCopies * kHistBins;
  uint64_t* cand = cand_all + (int64_t)b * cand_stride + (int64_t)c * kSelChunk;
  const float* sc = scores + (int64_t)b * score_stride;
  const int c0 = c * kSelChunk;

  __shared__ uint32_t scratch[kSelThreads / 64];
  __shared__ uint32_t h2[kHistBins];
  __shared__ uint32_t s_count;
  // this thread's 8 consecutive scores (unguarded: masked below)
  float v[kSelPer];
#pragma unroll
  for (int i = 0; i < kSelPer; ++i) v[i] = sc[min(c0 + t * kSelPer + i, n_hist - 1)];
  for (int i = t; i < kHistBins; i += kSelThreads) h2[i] = 0u;
  if (t == 0) s_count = 0u;
  int b1;
  uint32_t above1;
  find_boundary<NC>(hist1, NC, (uint32_t)k_eff, scratch, b1, above1);
  if (c == 0 && t == 0) {
    sel_info[b * 4 + 0] = (uint32_t)b1;
    sel_info[b * 4 + 1] = above1;
  }
  uint32_t mask8 = 0u;
#pragma unroll
  for (int i = 0; i < kSelPer; ++i) {
    const int x = c0 + t * kSelPer + i;
    const uint32_t key = selection_key_shift(v[i], key_shift);
    const int bin = (int)(key >> kHistShift);
    const bool valid = x < n_hist;
    if (valid && bin > b1) mask8 |= 1u << i;
    const bool is_cand = valid && bin == b1;
    const uint32_t slot = wave_append(&s_count, is_cand);
    if (is_cand) {
      cand[slot] = ((uint64_t)key << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)x);
      atomicAdd(&h2[(key >> kSubShift) & (kHistBins - 1)], 1u);
    }
  }
  // a bitmap word covers 4 threads' bytes: lane 4q gathers lanes 4q..4q+3
  const uint32_t m1 = (uint32_t)__shfl_down((int)mask8, 1), m2 = (uint32_t)__shfl_down((int)mask8, 2),
                 m3 = (uint32_t)__shfl_down((int)mask8, 3);
  const uint32_t word = mask8 | (m1 << 8) | (m2 << 16) | (m3 << 24);
  const int wi = t >> 2;                                // word index within the chunk
  if ((lane & 3) == 0 && c0 + wi * 32 < n_hist) bitmap_all[b * bitmap_words(cap) + c0 / 32 + wi] = word;
  uint32_t excl;
  const uint32_t n_above = block_exclusive_scan((uint32_t)__popc(mask8), scratch, excl);
  __syncthreads();                                      // s_count and h2 complete
  if (t == 0) {
    above_count[(int64_t)b * cnt_stride + c] = n_above;
    cand_count[(int64_t)b * cnt_stride + c] = s_count;
  }
  for (int i = t; i < kHistBins; i += kSelThreads) {
    const uint32_t n = h2[i];
    if (n) atomicAdd(&hist2[i], n);
  }
}

// ---------------------------------------------------------------------------
// finish: one workgroup per 2048 positions
// ---------------------------------------------------------------------------
// per-chunk counters per thread: NCP (a template parameter, the smallest of
// 1, 2, 4, 16 with 256 NCP >= the sequence's chunks), so a 128k sequence's 64
// chunks cost one load per thread and counter instead of 16
constexpr int kFinCntMax = kMaxSelGroups / kSelThreads;    // 16
constexpr int kFinBatch = 8;                              // candidates per thread per batch

// candidate i of the sequence, the chunks' lists concatenated in chunk order
// (cpre = exclusive prefix of the chunks' candidate counts, cpre[nch] = total)
__device__ __forceinline__ int cand_chunk_of(const uint32_t* cpre, int nch, int top, int i) {
  int g = 0;
  for (int step = top >> 1; step > 0; step >>= 1) {
    const int cc = g + step;
    if (cpre[min(cc, nch)] <= (uint32_t)i) g = cc;
  }
  return g;
}

template <int NCP>
__global__ __launch_bounds__(kSelThreads) void k_select_finish(
    const uint32_t* __restrict__ hist_all, const uint64_t* __restrict__ cand_all,
    const uint32_t* __restrict__ bitmap_all, const uint32_t* __restrict__ cand_count,
    const uint32_t* __restrict__ above_count, const uint32_t* __restrict__ sel_info, int32_t* __restrict__ idx_all,
    int32_t* __restrict__ idx_copy, int64_t idx_stride, int64_t cand_stride, int64_t cnt_stride, int64_t cap, int L,
    int W, int k, Lens lens) {
  constexpr uint64_t kLow42 = (1ull << 42) - 1;          // low 10 key bits + position bits
  const int b = blockIdx.y, c = blockIdx.x;
  L = (int)len_of(lens, b, L);
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int n_hist = max(L - W, 0);
  const int k_eff = min(k, n_hist);
  const int nch = (n_hist + kSelChunk - 1) / kSelChunk;
  int32_t* idx = idx_all + (int64_t)b * idx_stride;
  int32_t* idx2 = idx_copy ? idx_copy + (int64_t)b * idx_stride : nullptr;
  // the window goes to the workgroup of the last chunk (chunk 0 when there is none)
  if (c == max(nch, 1) - 1) {
    for (int i = t; i < L - n_hist; i += kSelThreads) {
      idx[k_eff + i] = n_hist + i;
      if (idx2) idx2[k_eff + i] = n_hist + i;
    }
  }
  if (k_eff == 0 || c >= max(nch, 1)) return;          // (a shorter sequence of a ragged batch)
  const uint32_t* hist2 = hist_all + (int64_t)b * kHistStride + kHistCopies * kHistBins;
  const uint64_t* cand_b = cand_all + (int64_t)b * cand_stride;

  __shared__ uint32_t scratch[kSelThreads / 64];
  __shared__ uint32_t cpre[kMaxSelGroups + 1];
  __shared__ uint32_t chosen[kMaxSelGroups];
  __shared__ uint64_t s3[kS3Cap];
  __shared__ uint32_t own[kSelChunk / 32];
  __shared__ uint32_t s_n3, s_digit, s_rem;
  __shared__ uint32_t dh[256];

  // ---- every load the workgroup needs first, issued together ---------------------------
  const uint32_t b1 = sel_info[b * 4 + 0], above1 = sel_info[b * 4 + 1];
  uint32_t cc[NCP], ac[NCP];
#pragma unroll
  for (int i = 0; i < NCP; ++i) {
    const int g = min(t * NCP + i, nch - 1);
    cc[i] = cand_count[(int64_t)b * cnt_stride + g];
    ac[i] = above_count[(int64_t)b * cnt_stride + g];
  }
  const int wbase = c * (kSelChunk / 32);
  const int nwords = (n_hist + 31) / 32;
  uint32_t myword = 0u;
  if (t < kSelChunk / 32) myword = bitmap_all[b * bitmap_words(cap) + min(wbase + t, nwords - 1)];
  const uint32_t need = (uint32_t)k_eff - above1;        // >= 1
  int b2;
  uint32_t above2;
  find_boundary<1>(hist2, 1, need, scratch, b2, above2);
  const uint32_t need3 = need - above2;                  // >= 1, taken from sub-bin b2
  // prefix of the candidate counts (chunk order), chosen counters cleared
  uint32_t csum = 0;
#pragma unroll
  for (int i = 0; i < NCP; ++i) csum += (t * NCP + i < nch) ? cc[i] : 0u;
  uint32_t cex;
  const uint32_t n_cand = block_exclusive_scan(csum, scratch, cex);
  {
    uint32_t run = cex;
#pragma unroll
    for (int i = 0; i < NCP; ++i) {
      const int g = t * NCP + i;
      if (g < nch) cpre[g] = run;
      run += (g < nch) ? cc[i] : 0u;
      if (g < nch) chosen[g] = 0u;
    }
  }
  if (t == 0) {
    cpre[nch] = n_cand;
    s_n3 = 0u;
  }
  if (t < kSelChunk / 32) own[t] = (wbase + t < nwords) ? myword : 0u;
  __syncthreads();
  int top = 1;
  while (top < nch) top <<= 1;

  // ---- candidates: above b2 chosen, b2 to level 3 ----------------------------------------
  auto mark = [&](uint64_t comp) {
    const uint32_t x = 0xFFFFFFFFu - (uint32_t)comp;
    const int g = (int)(x / kSelChunk);
    atomicAdd(&chosen[g], 1u);
    if (g == c) atomicOr(&own[(x % kSelChunk) >> 5], 1u << (x & 31));
  };
  for (int base = 0; base < (int)n_cand; base += kFinBatch * kSelThreads) {
    int ii[kFinBatch], gg[kFinBatch];
    uint64_t r[kFinBatch];
#pragma unroll
    for (int q = 0; q < kFinBatch; ++q) {
      ii[q] = min(base + q * kSelThreads + t, (int)n_cand - 1);
      gg[q] = cand_chunk_of(cpre, nch, top, ii[q]);
    }
#pragma unroll
    for (int q = 0; q < kFinBatch; ++q) r[q] = cand_b[(int64_t)gg[q] * kSelChunk + (ii[q] - (int)cpre[gg[q]])];
#pragma unroll
    for (int q = 0; q < kFinBatch; ++q) {
      const bool live = base + q * kSelThreads + t < (int)n_cand;
      const int sb = (int)((uint32_t)(r[q] >> 32) >> kSubShift) & (kHistBins - 1);
      if (live && sb > b2) mark(r[q]);
      const bool lev3 = live && sb == b2;
      const uint32_t slot = wave_append(&s_n3, lev3);
      if (lev3 && slot < (uint32_t)kS3Cap) s3[slot] = r[q];
    }
  }
  __syncthreads();
  const uint32_t n3 = s_n3;
  if (n3 <= (uint32_t)kS3Cap) {
    // exact rank among the level-3 candidates by counting larger composites
    for (int i0 = 0; i0 < (int)n3; i0 += kSelThreads) {
      const int i = i0 + t;
      const uint64_t x = s3[min(i, (int)n3 - 1)];
      uint32_t rank = 0;
      for (uint32_t j = 0; j < n3; ++j) rank += (s3[j] > x) ? 1u : 0u;
      if (i < (int)n3 && rank < need3) mark(x);
    }
  } else {
    // many exact ties: radix select (8-bit digits, top down) of the need3-th
    // largest low-42-bit value among the sub-bin b2 candidates, scanning the
    // candidate lists in place; then mark those at or above it
    const uint32_t keytop = (b1 << 11) | (uint32_t)b2;   // key bits 31..10 shared by level 3
    uint64_t prefix = 0, pmask = 0;
    uint32_t remaining = need3;
    for (int shift = 34; shift >= -6; shift -= 8) {
      const int sh = shift < 0 ? 0 : shift;
      const int nbits = shift < 0 ? 8 + shift : 8;
      const uint64_t dmask = ((1ull << nbits) - 1) << sh;
      dh[t] = 0u;
      __syncthreads();
      for (int base = 0; base < (int)n_cand; base += kFinBatch * kSelThreads) {
        int ii[kFinBatch], gg[kFinBatch];
        uint64_t r[kFinBatch];
#pragma unroll
        for (int q = 0; q < kFinBatch; ++q) {
          ii[q] = min(base + q * kSelThreads + t, (int)n_cand - 1);
          gg[q] = cand_chunk_of(cpre, nch, top, ii[q]);
        }
#pragma unroll
        for (int q = 0; q < kFinBatch; ++q) r[q] = cand_b[(int64_t)gg[q] * kSelChunk + (ii[q] - (int)cpre[gg[q]])];
#pragma unroll
        for (int q = 0; q < kFinBatch; ++q) {
          const bool live = base + q * kSelThreads + t < (int)n_cand;
          const uint64_t low = r[q] & kLow42;
          if (live && (uint32_t)(r[q] >> 42) == keytop && (low & pmask) == prefix)
            atomicAdd(&dh[(low & dmask) >> sh], 1u);
        }
      }
      __syncthreads();
      if (t == 0) {
        uint32_t run = 0;
        int d = (1 << nbits) - 1;
        for (; d > 0; --d) {
          if (run + dh[d] >= remaining) break;
          run += dh[d];
        }
        s_digit = (uint32_t)d;
        s_rem = remaining - run;
      }
      __syncthreads();
      prefix |= (uint64_t)s_digit << sh;
      pmask |= dmask;
      remaining = s_rem;
      __syncthreads();
    }
    for (int base = 0; base < (int)n_cand; base += kFinBatch * kSelThreads) {
      int ii[kFinBatch], gg[kFinBatch];
      uint64_t r[kFinBatch];
#pragma unroll
      for (int q = 0; q < kFinBatch; ++q) {
        ii[q] = min(base + q * kSelThreads + t, (int)n_cand - 1);
        gg[q] = cand_chunk_of(cpre, nch, top, ii[q]);
      }
#pragma unroll
      for (int q = 0; q < kFinBatch; ++q) r[q] = cand_b[(int64_t)gg[q] * kSelChunk + (ii[q] - (int)cpre[gg[q]])];
#pragma unroll
      for (int q = 0; q < kFinBatch; ++q) {
        const bool live = base + q * kSelThreads + t < (int)n_cand;
        if (live && (uint32_t)(r[q] >> 42) == keytop && (r[q] & kLow42) >= prefix) mark(r[q]);
      }
    }
  }
  __syncthreads();

  // ---- output offset of this chunk: positions selected in earlier chunks ------------------
  uint32_t before = 0;
#pragma unroll
  for (int i = 0; i < NCP; ++i) {
    const int g = t * NCP + i;
    if (g < c) before += ac[i] + chosen[g];
  }
  uint32_t bex;
  const uint32_t off = block_exclusive_scan(before, scratch, bex);
  // ---- this chunk's positions, ascending: 64 words expanded by one wave -------------------
  if (wave == 0) {
    const uint32_t wv = own[lane];
    const uint32_t pc = (uint32_t)__popc(wv);
    uint32_t x = pc;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t y = (uint32_t)__builtin_amdgcn_ds_bpermute(max(lane - o, 0) << 2, (int)x);
      if (lane >= o) x += y;
    }
    uint32_t pos = off + x - pc;
    uint32_t rem = wv;
    while (rem) {
      const int bit = __ffs(rem) - 1;
      rem &= rem - 1;
      const int32_t p = (int32_t)(c * kSelChunk + lane * 32 + bit);
      idx[pos] = p;
      if (idx2) idx2[pos] = p;
      ++pos;
    }
  }
}

hipError_t launch_select(const Problem& P, const Workspace& ws, int64_t L, const float* scores,
                         int64_t score_stride, int32_t* idx, int32_t* idx_copy, hipStream_t st) {
  const int64_t n_hist = std::max<int64_t>(L - P.W, 0);
  const int ng = (int)std::max<int64_t>(1, (n_hist + kHistChunk - 1) / kHistChunk);   // k_hist_scores' workgroups
  return launch_select_keyed(P, ws, L, scores, score_stride, idx, idx_copy, 1, hist_copies(ng), st);
}

hipError_t launch_select_keyed(const Problem& P, const Workspace& ws, int64_t L, const float* scores,
                               int64_t score_stride, int32_t* idx, int32_t* idx_copy, int key_shift, int hist_nc,
                               hipStream_t st) {
  const int64_t n_hist = std::max<int64_t>(L - P.W, 0);
  const int m = (int)(std::min<int64_t>(P.k, n_hist) + std::min<int64_t>(P.W, L));
  const int nch = (int)((n_hist + kSelChunk - 1) / kSelChunk);
  if (std::min<int64_t>(P.k, n_hist) > 0) {
    static_assert(kHistCopies == 8, "classify instances for 1, 2, 4 and 8 copies");
    auto cls = hist_nc == 1 ? k_select_classify<1>
               : hist_nc == 2 ? k_select_classify<2> : hist_nc == 4 ? k_select_classify<4> : k_select_classify<8>;
    hipLaunchKernelGGL(cls, dim3(nch, P.B), dim3(kSelThreads), 0, st, scores, score_stride, ws.hist, ws.cand,
                       ws.bitmap, ws.cand_count, ws.above_count, ws.sel_info, cand_stride(P), sel_groups_max(P), P.cap,
                       (int)L, P.W, P.k, P.lens, key_shift);
  }
  auto fin = nch <= kSelThreads ? k_select_finish<1>
             : nch <= 2 * kSelThreads ? k_select_finish<2>
             : nch <= 4 * kSelThreads ? k_select_finish<4> : k_select_finish<kFinCntMax>;
  hipLaunchKernelGGL(fin, dim3(std::max(nch, 1), P.B), dim3(kSelThreads), 0, st, ws.hist, ws.cand, ws.bitmap,
                     ws.cand_count, ws.above_count, ws.sel_info, idx, idx_copy, (int64_t)m, cand_stride(P),
                     sel_groups_max(P), P.cap, (int)L, P.W, P.k, P.lens);
  return hipGetLastError();
}

}  // namespace s4r
