// Index selection of Section 3.2.3 on gfx950:
//   I_local  = [max(L - W, 0), L)
//   I_global = the k_eff = min(k, max(L - W, 0)) largest scores of
//              [0, L - W), equal scores going to the lower position
//   idx      = sorted(I_global) ++ I_local
//
// Scores are non-negative fp32, so their bit patterns order like the values.
// A 2048-bin histogram of the top 11 bits (built by the relevance kernel or
// k_hist_scores) fixes the boundary bin.  Then:
//   - every workgroup owns 2048 consecutive positions (64 bitmap words):
//     positions above the boundary bin are set in a bitmap, positions inside
//     it are appended to a candidate list as (key << 32 | ~position), a
//     composite that is unique and orders "higher score, then lower position"
//     first;
//   - a second kernel, one workgroup per sequence, picks the remaining candidates
//     (a second 11-bit histogram level in LDS, then exact ranks by counting,
//     or an exact radix select when there are too many equal keys), and turns
//     the bitmap into the sorted index list with block-wide prefix sums, then
//     appends the window.
// Everything is integer work on the given scores: the result is bit-exact
// and deterministic.
#include "s4r_device.h"
#include "s4r_internal.h"

namespace s4r {

constexpr int kSelThreads = 256;
constexpr int kL3Cap = 1024;     // level-3 candidates ranked by counting
constexpr int kSegWords = 4096;  // bitmap words staged in LDS per segment (131072 positions)

// block-wide exclusive prefix sum of one value per thread (wave shuffles,
// then the four wave totals through LDS); returns the block total
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

// boundary bin of the histogram: the highest bin b1 with count(bins >= b1) >= k_eff
__device__ void find_boundary(const uint32_t* __restrict__ hist, int k_eff, uint32_t* scratch, int& b1,
                              uint32_t& above) {
  constexpr int per = kHistBins / kSelThreads;   // bins per thread, thread 0 = top bins
  const int t = threadIdx.x;
  uint32_t cnt[per];
  uint32_t sum = 0;
#pragma unroll
  for (int i = 0; i < per; ++i) {
    cnt[i] = hist[kHistBins - 1 - (t * per + i)];
    sum += cnt[i];
  }
  uint32_t excl;
  block_exclusive_scan(sum, scratch, excl);      // count strictly above this thread's bins
  __shared__ int s_b1;
  __shared__ uint32_t s_above;
  if (excl < (uint32_t)k_eff && excl + sum >= (uint32_t)k_eff) {
    uint32_t run = excl;
#pragma unroll
    for (int i = 0; i < per; ++i) {
      if (run < (uint32_t)k_eff && run + cnt[i] >= (uint32_t)k_eff) {
        s_b1 = kHistBins - 1 - (t * per + i);
        s_above = run;
      }
      run += cnt[i];
    }
  }
  __syncthreads();
  b1 = s_b1;
  above = s_above;
  __syncthreads();
}

// one workgroup per 2048 positions: bitmap words above the boundary bin,
// candidates inside it
__global__ __launch_bounds__(kSelThreads) void k_select_classify(
    const float* __restrict__ scores, int64_t score_stride, const uint32_t* __restrict__ hist_all,
    uint64_t* __restrict__ cand_all, uint32_t* __restrict__ bitmap_all, uint32_t* __restrict__ cand_count,
    int64_t cand_stride, int64_t cnt_stride, int64_t cap, int L, int W, int k) {
  const int b = blockIdx.y;
  const int t = threadIdx.x;
  const int n_hist = max(L - W, 0);
  const int k_eff = min(k, n_hist);
  if (k_eff == 0) return;
  const uint32_t* hist = hist_all + (int64_t)b * kHistBins;
  // this workgroup's own candidate region and count: no cross-workgroup atomics
  uint64_t* cand = cand_all + (int64_t)b * cand_stride + (int64_t)blockIdx.x * kSelChunk;
  uint32_t* bitmap = bitmap_all + (int64_t)b * (cap / 32);
  const float* sc = scores + (int64_t)b * score_stride;

  __shared__ uint32_t scratch[kSelThreads];
  __shared__ uint32_t words[kSelChunk / 32];
  __shared__ uint32_t s_count;

  int b1;
  uint32_t above;
  find_boundary(hist, k_eff, scratch, b1, above);

  const int c0 = blockIdx.x * kSelChunk;
  if (t < kSelChunk / 32) words[t] = 0;
  if (t == 0) s_count = 0;
  __syncthreads();
  constexpr int per = kSelChunk / kSelThreads;   // 8 consecutive positions per thread
  float v[per];
#pragma unroll
  for (int i = 0; i < per; ++i) v[i] = sc[min(c0 + t * per + i, n_hist - 1)];   // unguarded: masked below
#pragma unroll
  for (int i = 0; i < per; ++i) {
    const int x = c0 + t * per + i;
    const uint32_t key = score_key(v[i]);
    const int bin = (int)(key >> kHistShift);
    const bool valid = x < n_hist;
    if (valid && bin > b1) atomicOr(&words[(t * per + i) >> 5], 1u << ((t * per + i) & 31));
    const bool is_cand = valid && bin == b1;
    const uint32_t slot = wave_append(&s_count, is_cand);
    if (is_cand) cand[slot] = ((uint64_t)key << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)x);
  }
  __syncthreads();
  if (t < kSelChunk / 32 && c0 + t * 32 < n_hist) bitmap[c0 / 32 + t] = words[t];
  if (t == 0) cand_count[(int64_t)b * cnt_stride + blockIdx.x] = s_count;
}

// exact radix select over n composites in `list` (global or LDS) restricted to
// entries matching (c & fmask) == fval: returns the `need`-th largest value of
// the low 52 bits.  One workgroup; dh is a 256-entry LDS histogram.
__device__ uint64_t radix_select52(const uint64_t* list, uint32_t n, uint64_t fmask, uint64_t fval, uint32_t need,
                                   uint32_t* dh, uint32_t* s_digit, uint32_t* s_rem) {
  const int t = threadIdx.x;
  uint64_t prefix = 0, pmask = 0;
  uint32_t remaining = need;
  for (int shift = 44; shift >= -4; shift -= 8) {
    const int sh = shift < 0 ? 0 : shift;
    const int nbits = shift < 0 ? 8 + shift : 8;
    const uint64_t dmask = ((1ull << nbits) - 1) << sh;
    dh[t] = 0;
    __syncthreads();
    for (uint32_t i = t; i < n; i += kSelThreads) {
      const uint64_t c = list[i];
      if ((c & fmask) == fval && (c & pmask) == prefix) atomicAdd(&dh[(c & dmask) >> sh], 1u);
    }
    __syncthreads();
    if (t == 0) {
      uint32_t run = 0;
      int d = (1 << nbits) - 1;
      for (; d > 0; --d) {
        if (run + dh[d] >= remaining) break;
        run += dh[d];
      }
      *s_digit = (uint32_t)d;
      *s_rem = remaining - run;
    }
    __syncthreads();
    prefix |= (uint64_t)(*s_digit) << sh;
    pmask |= dmask;
    remaining = *s_rem;
    __syncthreads();
  }
  return prefix;
}

// one workgroup per sequence: resolve the boundary bin, emit the index list
__global__ __launch_bounds__(kSelThreads) void k_select_finish(
    const uint32_t* __restrict__ hist_all, const uint64_t* __restrict__ cand_all, uint32_t* __restrict__ bitmap_all,
    const uint32_t* __restrict__ cand_count, uint64_t* __restrict__ cand2_all, int64_t cand_stride,
    int64_t cnt_stride, int32_t* __restrict__ idx_all, int32_t* __restrict__ idx_copy, int64_t idx_stride,
    int64_t cap, int L, int W, int k) {
  constexpr uint64_t kLow52 = 0xFFFFFFFFFFFFFull;
  constexpr int kSub = 32 + kHistShift - 11;     // shift of the level-2 key bits in a composite
  const int b = blockIdx.x;
  const int t = threadIdx.x;
  const int n_hist = max(L - W, 0);
  const int k_eff = min(k, n_hist);
  const uint32_t* hist = hist_all + (int64_t)b * kHistBins;
  const uint64_t* cand_b = cand_all + (int64_t)b * cand_stride;
  uint64_t* cand = cand2_all + (int64_t)b * cand_stride;     // compacted list (overflow path)
  uint32_t* bitmap = bitmap_all + (int64_t)b * (cap / 32);
  int32_t* idx = idx_all + (int64_t)b * idx_stride;
  int32_t* idx2 = idx_copy ? idx_copy + (int64_t)b * idx_stride : nullptr;
  const int ncw = (n_hist + kSelChunk - 1) / kSelChunk;        // classify workgroups

  __shared__ uint32_t scratch[kSelThreads];
  __shared__ uint32_t h2[kHistBins];
  __shared__ uint64_t lcand[kCandCap];           // candidates; chosen ones stacked from the top
  __shared__ uint64_t l3[kL3Cap];
  __shared__ uint32_t segw[kSegWords];
  __shared__ uint32_t woff[kSegWords];           // bit offset of each non-empty word
  __shared__ uint32_t wlist[kSegWords];          // index of each non-empty word
  __shared__ uint32_t s_digit, s_rem, s_n3, s_nchosen;
  __shared__ uint32_t s_off[kMaxSelGroups + 1];

  int b1 = -1;
  uint32_t above = 0;
  if (k_eff > 0) find_boundary(hist, k_eff, scratch, b1, above);
  const uint32_t need = (k_eff > 0) ? (uint32_t)k_eff - above : 0u;
  uint32_t n_cand = 0;
  if (need > 0) {
    // offsets of the classify workgroups' candidate regions (fixed order)
    uint32_t run = 0;
    for (int g0 = 0; g0 < ncw; g0 += kSelThreads) {
      const int g = g0 + t;
      const uint32_t cl = cand_count[(int64_t)b * cnt_stride + min(g, ncw - 1)];
      const uint32_t c = (g < ncw) ? cl : 0u;
      uint32_t excl;
      const uint32_t tot = block_exclusive_scan(c, scratch, excl);
      if (g < ncw) s_off[g] = run + excl;
      run += tot;
    }
    if (t == 0) s_off[ncw] = run;
    __syncthreads();
    n_cand = s_off[ncw];
  }
  if (t == 0) {
    s_nchosen = 0;
    s_n3 = 0;
  }
  __syncthreads();

  // candidates in (group, slot) order: the source group of entry i is the
  // last g with s_off[g] <= i, found by a fixed-step binary search that 16
  // entries per thread run interleaved (s_off[ncw] = n_cand ends every search)
  int top = 1;
  while (top < ncw) top <<= 1;
  auto gather = [&](uint64_t* dst) {
    for (int base = 0; base < (int)n_cand; base += 16 * kSelThreads) {
      int ii[16], g[16];
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        ii[q] = min(base + q * kSelThreads + t, (int)n_cand - 1);
        g[q] = 0;
      }
      for (int step = top >> 1; step > 0; step >>= 1) {
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int c = g[q] + step;
          if (s_off[min(c, ncw)] <= (uint32_t)ii[q]) g[q] = c;
        }
      }
      uint64_t r[16];
#pragma unroll
      for (int q = 0; q < 16; ++q) r[q] = cand_b[(int64_t)g[q] * kSelChunk + (ii[q] - (int)s_off[g[q]])];
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int i = base + q * kSelThreads + t;
        if (i < (int)n_cand) dst[i] = r[q];
      }
    }
  };
  // chosen candidates are stacked into lcand from the top end
  auto choose = [&](uint64_t c, bool pred) {
    const uint32_t slot = wave_append(&s_nchosen, pred);
    if (pred) lcand[kCandCap - 1 - slot] = c;
  };

  if (need > 0 && n_cand <= (uint32_t)kCandCap) {
    gather(lcand);
    // level 2: histogram of the next 11 key bits among the candidates
    for (int i = t; i < kHistBins; i += kSelThreads) h2[i] = 0;
    __syncthreads();
    for (int i0 = 0; i0 < (int)n_cand; i0 += kSelThreads) {
      const int i = i0 + t;
      if (i < (int)n_cand) atomicAdd(&h2[(uint32_t)(lcand[i] >> kSub) & (kHistBins - 1)], 1u);
    }
    __syncthreads();
    int b2;
    uint32_t above2;
    find_boundary(h2, (int)need, scratch, b2, above2);
    const uint32_t need3 = need - above2;
    // sub-bins above b2 are chosen, sub-bin b2 goes to level 3; every thread
    // first copies its candidates to registers because chosen entries are
    // stacked into lcand from the top end
    uint64_t mine[kCandCap / kSelThreads];
#pragma unroll
    for (int q = 0; q < kCandCap / kSelThreads; ++q) {
      const int i = q * kSelThreads + t;
      mine[q] = (i < (int)n_cand) ? lcand[i] : 0ull;
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kCandCap / kSelThreads; ++q) {
      const int i = q * kSelThreads + t;
      const uint64_t c = mine[q];
      const int sb = (int)((uint32_t)(c >> kSub) & (kHistBins - 1));
      const bool valid = i < (int)n_cand;
      choose(c, valid && sb > b2);
      const bool lev3 = valid && sb == b2;
      const uint32_t slot = wave_append(&s_n3, lev3);
      if (lev3 && slot < (uint32_t)kL3Cap) l3[slot] = c;
    }
    __syncthreads();
    const uint32_t n3 = s_n3;
    if (n3 <= (uint32_t)kL3Cap) {
      // level 3: exact rank of each remaining candidate by counting larger composites
      for (int i0 = 0; i0 < (int)n3; i0 += kSelThreads) {
        const int i = i0 + t;
        const uint64_t c = l3[min(i, (int)n3 - 1)];
        uint32_t rank = 0;
        for (uint32_t j = 0; j < n3; ++j) rank += (l3[j] > c) ? 1u : 0u;
        choose(c, i < (int)n3 && rank < need3);
      }
    } else {
      // many equal keys in sub-bin b2: exact radix select among them (the
      // unchosen candidates are still in their own thread's registers: write
      // the sub-bin b2 ones to the global list first)
      for (int q = 0; q < kCandCap / kSelThreads; ++q) {
        const int i = q * kSelThreads + t;
        if (i < (int)n_cand) cand[i] = mine[q];
      }
      __syncthreads();
      // key bits 31..10 shared by sub-bin b2 (l3[0] is one of its candidates)
      const uint64_t fmask = ~kLow52 | (((uint64_t)(kHistBins - 1)) << kSub);
      const uint64_t fval = l3[0] & fmask;
      const uint64_t thr = radix_select52(cand, n_cand, fmask, fval, need3, scratch, &s_digit, &s_rem);
      for (int i0 = 0; i0 < (int)n_cand; i0 += kSelThreads) {
        const int i = i0 + t;
        const uint64_t c = cand[min(i, (int)n_cand - 1)];
        choose(c, i < (int)n_cand && (c & fmask) == fval && (c & kLow52) >= thr);
      }
    }
    __syncthreads();
  } else if (need > 0) {
    // more boundary candidates than fit in LDS (massive ties): exact radix
    // select of the need-th largest composite over the compacted global list;
    // the chosen positions are OR-ed into the global bitmap directly
    gather(cand);
    __syncthreads();
    const uint64_t thr = radix_select52(cand, n_cand, 0ull, 0ull, need, scratch, &s_digit, &s_rem);
    for (uint32_t i = t; i < n_cand; i += kSelThreads) {
      const uint64_t c = cand[i];
      if ((c & kLow52) >= thr) {
        const uint32_t x = 0xFFFFFFFFu - (uint32_t)(c & 0xFFFFFFFFull);
        atomicOr(&bitmap[x >> 5], 1u << (x & 31));
      }
    }
    __syncthreads();
  }
  const uint32_t nchosen = s_nchosen;
  // the global bitmap was written by the classify kernel; only the overflow
  // path above adds to it from this kernel, and then reads it back atomically
  const bool overflow = need > 0 && n_cand > (uint32_t)kCandCap;

  // ---- bitmap (+ chosen positions) -> ascending positions, by segments in LDS -----
  // Per segment: bit offsets of the words by a block scan of popcounts, the
  // non-empty words compacted by a second scan, then the non-empty words are
  // expanded, dealt out round-robin over the threads.  Positions
  // are staged in LDS (lcand is free once the chosen candidates are merged
  // into the segment) and written out with coalesced stores when they fit.
  const int nwords = (n_hist + 31) / 32;
  constexpr int kOutCap = kCandCap * 2;
  uint32_t* lout = reinterpret_cast<uint32_t*>(lcand);
  const bool stage = k_eff <= kOutCap && nwords <= kSegWords;
  constexpr int kWPT = kSegWords / kSelThreads;   // words per thread per segment
  uint32_t base = 0;
  if (k_eff > 0) {
    for (int s0 = 0; s0 < nwords; s0 += kSegWords) {
      const int nw = min(kSegWords, nwords - s0);
      for (int b0 = 0; b0 < nw; b0 += 8 * kSelThreads) {
        uint32_t r[8];
        if (overflow) {
#pragma unroll
          for (int q = 0; q < 8; ++q)
            r[q] = __hip_atomic_load(&bitmap[s0 + min(b0 + q * kSelThreads + t, nw - 1)], __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT);
        } else {
#pragma unroll
          for (int q = 0; q < 8; ++q) r[q] = bitmap[s0 + min(b0 + q * kSelThreads + t, nw - 1)];
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) segw[min(b0 + q * kSelThreads + t, nw - 1)] = r[q];   // past nw: same value again
      }
      for (int i = nw + t; i < kSegWords; i += kSelThreads) segw[i] = 0u;
      __syncthreads();
      for (uint32_t i = t; i < nchosen; i += kSelThreads) {
        const uint32_t x = 0xFFFFFFFFu - (uint32_t)(lcand[kCandCap - 1 - i] & 0xFFFFFFFFull);
        const int w = (int)(x >> 5) - s0;
        if (w >= 0 && w < nw) atomicOr(&segw[w], 1u << (x & 31));
      }
      __syncthreads();
      // thread t owns words [t * kWPT, (t + 1) * kWPT) of the segment
      uint32_t cnt = 0, ne = 0;
#pragma unroll
      for (int i = 0; i < kWPT; ++i) {
        const uint32_t v = segw[t * kWPT + i];
        cnt += __popc(v);
        ne += v ? 1u : 0u;
      }
      uint32_t bexcl, nexcl;
      const uint32_t total = block_exclusive_scan(cnt, scratch, bexcl);
      const uint32_t n_ne = block_exclusive_scan(ne, scratch, nexcl);
      {
        uint32_t pos = base + bexcl, slot = nexcl;
#pragma unroll
        for (int i = 0; i < kWPT; ++i) {
          const int w = t * kWPT + i;
          const uint32_t v = segw[w];
          if (v) {
            woff[slot] = pos;
            wlist[slot] = (uint32_t)w;
            ++slot;
          }
          pos += __popc(v);
        }
      }
      __syncthreads();
      // expansion: the non-empty words are dealt out round-robin, so every
      // thread gets words from all over the segment and clustered selections
      // do not pile up on one thread
      for (uint32_t j = t; j < n_ne; j += kSelThreads) {
        const uint32_t w = wlist[j];
        uint32_t v = segw[w];
        uint32_t pos = woff[j];
        while (v) {
          const int bit = __ffs(v) - 1;
          v &= v - 1;
          const int32_t x = (int32_t)((s0 + (int)w) * 32 + bit);
          if (stage) {
            lout[pos] = (uint32_t)x;
          } else {
            idx[pos] = x;
            if (idx2) idx2[pos] = x;
          }
          ++pos;
        }
      }
      base += total;
      __syncthreads();
    }
  }
  if (k_eff > 0 && stage) {
    for (int i = t; i < k_eff; i += kSelThreads) {   // the segment loop ended with a barrier
      const int32_t v = (int32_t)lout[i];
      idx[i] = v;
      if (idx2) idx2[i] = v;
    }
  }
  for (int i = t; i < L - n_hist; i += kSelThreads) {
    idx[k_eff + i] = n_hist + i;
    if (idx2) idx2[k_eff + i] = n_hist + i;
  }
}

hipError_t launch_select(const Problem& P, const Workspace& ws, int64_t L, const float* scores,
                         int64_t score_stride, int32_t* idx, int32_t* idx_copy, hipStream_t st) {
  const int64_t n_hist = std::max<int64_t>(L - P.W, 0);
  const int m = (int)(std::min<int64_t>(P.k, n_hist) + std::min<int64_t>(P.W, L));
  if (std::min<int64_t>(P.k, n_hist) > 0) {
    dim3 grid((unsigned)((n_hist + kSelChunk - 1) / kSelChunk), P.B);
    hipLaunchKernelGGL(k_select_classify, grid, dim3(kSelThreads), 0, st, scores, score_stride, ws.hist, ws.cand,
                       ws.bitmap, ws.cand_count, cand_stride(P), sel_groups_max(P), P.cap, (int)L, P.W, P.k);
  }
  hipLaunchKernelGGL(k_select_finish, dim3(P.B), dim3(kSelThreads), 0, st, ws.hist, ws.cand, ws.bitmap,
                     ws.cand_count, ws.cand2, cand_stride(P), sel_groups_max(P), idx, idx_copy, (int64_t)m, P.cap,
                     (int)L, P.W, P.k);
  return hipGetLastError();
}

}  // namespace s4r
