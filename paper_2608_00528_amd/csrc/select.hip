// Index selection of Section 3.2.3 on gfx950:
//   I_local  = [max(L - W, 0), L)
//   I_global = the k_eff = min(k, max(L - W, 0)) largest scores of
//              [0, L - W), equal scores going to the lower position
//   idx      = sorted(I_global) ++ I_local
//
// Scores are non-negative fp32, so their bit patterns order like the values.
// A 4096-bin histogram of the top 12 bits (built by the relevance kernel or
// k_hist_scores) fixes the boundary bin.  k_select then runs one pass:
//   - every workgroup owns 2048 consecutive positions (64 bitmap words):
//     positions above the boundary bin are set in a bitmap, positions inside
//     it are appended to a candidate list as (key << 32 | ~position), a
//     composite that is unique and orders "higher score, then lower position"
//     first;
//   - the last workgroup of each sequence picks the remaining candidates
//     (bitonic sort in LDS, or an exact radix select over the list when it is
//     too long for LDS), sets their bits and turns the bitmap into the sorted
//     index list with a block-wide prefix sum, then appends the window.
// Everything is integer work on the given scores: the result is bit-exact
// and deterministic.
#include "s4r_device.h"
#include "s4r_internal.h"

namespace s4r {

constexpr int kSelThreads = 256;

// block-wide exclusive prefix sum of one value per thread; returns the total
__device__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* scratch /* >= 256 */, uint32_t& excl) {
  const int t = threadIdx.x;
  scratch[t] = v;
  __syncthreads();
  for (int off = 1; off < kSelThreads; off <<= 1) {
    uint32_t add = (t >= off) ? scratch[t - off] : 0u;
    __syncthreads();
    scratch[t] += add;
    __syncthreads();
  }
  const uint32_t incl = scratch[t];
  const uint32_t total = scratch[kSelThreads - 1];
  excl = incl - v;
  __syncthreads();
  return total;
}

// boundary bin of the histogram: the highest bin b1 with count(bins >= b1) >= k_eff
__device__ void find_boundary(const uint32_t* __restrict__ hist, int k_eff, uint32_t* scratch, int& b1,
                              uint32_t& above) {
  constexpr int per = kHistBins / kSelThreads;   // 16 bins per thread, thread 0 = top bins
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

// bitonic sort, descending, of n (power of two) 64-bit keys in LDS
__device__ void bitonic_desc(uint64_t* a, int n) {
  for (int size = 2; size <= n; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = threadIdx.x; i < n / 2; i += blockDim.x) {
        const int lo = 2 * i - (i & (stride - 1));
        const int hi = lo + stride;
        const bool desc = ((lo & size) == 0);
        const uint64_t x = a[lo], y = a[hi];
        if ((x < y) == desc) {
          a[lo] = y;
          a[hi] = x;
        }
      }
      __syncthreads();
    }
  }
}

__global__ __launch_bounds__(kSelThreads) void k_select(
    const float* __restrict__ scores, int64_t score_stride, const uint32_t* __restrict__ hist_all,
    uint64_t* __restrict__ cand_all, uint32_t* __restrict__ bitmap_all, uint32_t* __restrict__ counters,
    int32_t* __restrict__ idx_all, int32_t* __restrict__ idx_copy, int64_t idx_stride, int64_t cap, int L, int W,
    int k) {
  const int b = blockIdx.y;
  const int t = threadIdx.x;
  const int n_hist = max(L - W, 0);
  const int k_eff = min(k, n_hist);
  const uint32_t* hist = hist_all + (int64_t)b * kHistBins;
  uint64_t* cand = cand_all + (int64_t)b * cap;
  uint32_t* bitmap = bitmap_all + (int64_t)b * (cap / 32);
  uint32_t* ctr = counters + b * kCounters;
  const float* sc = scores + (int64_t)b * score_stride;

  __shared__ uint32_t scratch[kSelThreads];
  __shared__ uint32_t words[kSelChunk / 32];
  __shared__ uint64_t lcand[kCandCap];           // also the local candidate buffer
  __shared__ uint32_t s_count, s_base;
  __shared__ int s_last;

  int b1 = -1;
  uint32_t above = 0;
  if (k_eff > 0) find_boundary(hist, k_eff, scratch, b1, above);

  // ---- classify this workgroup's positions --------------------------------
  const int c0 = blockIdx.x * kSelChunk;
  if (t < kSelChunk / 32) words[t] = 0;
  if (t == 0) s_count = 0;
  __syncthreads();
  if (k_eff > 0) {
    constexpr int per = kSelChunk / kSelThreads;   // 8 consecutive positions per thread
    for (int i = 0; i < per; ++i) {
      const int x = c0 + t * per + i;
      if (x >= n_hist) break;
      const uint32_t key = score_key(sc[x]);
      const int bin = (int)(key >> kHistShift);
      if (bin > b1) {
        atomicOr(&words[(t * per + i) >> 5], 1u << ((t * per + i) & 31));
      } else if (bin == b1) {
        const uint32_t slot = atomicAdd(&s_count, 1u);
        lcand[slot] = ((uint64_t)key << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)x);
      }
    }
  }
  __syncthreads();
  if (t < kSelChunk / 32 && c0 + t * 32 < n_hist) bitmap[c0 / 32 + t] = words[t];
  if (t == 0 && s_count) s_base = atomicAdd(&ctr[2], s_count);
  __syncthreads();
  for (uint32_t i = t; i < s_count; i += kSelThreads) cand[s_base + i] = lcand[i];

  // ---- the last workgroup of the sequence finishes --------------------------
  __threadfence();
  __syncthreads();
  if (t == 0) s_last = (atomicAdd(&ctr[1], 1u) == gridDim.x - 1);
  __syncthreads();
  if (!s_last) return;
  __threadfence();

  int32_t* idx = idx_all + (int64_t)b * idx_stride;
  int32_t* idx2 = idx_copy ? idx_copy + (int64_t)b * idx_stride : nullptr;
  const uint32_t n_cand = ctr[2];
  const uint32_t need = (k_eff > 0) ? (uint32_t)k_eff - above : 0u;

  if (need > 0) {
    if (n_cand <= (uint32_t)kCandCap) {
      int n2 = 1;
      while (n2 < (int)n_cand) n2 <<= 1;
      for (int i = t; i < n2; i += kSelThreads) lcand[i] = (i < (int)n_cand) ? cand[i] : 0ull;
      __syncthreads();
      bitonic_desc(lcand, n2);
      for (uint32_t i = t; i < need; i += kSelThreads) {
        const uint32_t x = 0xFFFFFFFFu - (uint32_t)(lcand[i] & 0xFFFFFFFFull);
        atomicOr(&bitmap[x >> 5], 1u << (x & 31));
      }
    } else {
      // exact radix select of the need-th largest composite over the list;
      // all candidates share the top 12 key bits, so 52 bits remain
      uint64_t prefix = 0, pmask = 0;
      uint32_t remaining = need;
      uint32_t* dh = scratch;                     // 256-bin digit histogram
      for (int shift = 44; shift >= -4; shift -= 8) {
        const int sh = shift < 0 ? 0 : shift;
        const int nbits = shift < 0 ? 8 + shift : 8;
        const uint64_t dmask = ((1ull << nbits) - 1) << sh;
        dh[t] = 0;
        __syncthreads();
        for (uint32_t i = t; i < n_cand; i += kSelThreads) {
          const uint64_t c = cand[i];
          if ((c & pmask) == prefix) atomicAdd(&dh[(c & dmask) >> sh], 1u);
        }
        __syncthreads();
        if (t == 0) {
          uint32_t run = 0;
          int d = (1 << nbits) - 1;
          for (; d > 0; --d) {
            if (run + dh[d] >= remaining) break;
            run += dh[d];
          }
          s_count = (uint32_t)d;
          s_base = remaining - run;
        }
        __syncthreads();
        prefix |= (uint64_t)s_count << sh;
        pmask |= dmask;
        remaining = s_base;
        __syncthreads();
      }
      // prefix is now the need-th largest composite (composites are unique)
      for (uint32_t i = t; i < n_cand; i += kSelThreads) {
        const uint64_t c = cand[i];
        if ((c & 0xFFFFFFFFFFFFFull) >= (prefix & 0xFFFFFFFFFFFFFull)) {
          const uint32_t x = 0xFFFFFFFFu - (uint32_t)(c & 0xFFFFFFFFull);
          atomicOr(&bitmap[x >> 5], 1u << (x & 31));
        }
      }
    }
  }
  __threadfence();
  __syncthreads();

  // ---- bitmap -> ascending positions ------------------------------------------
  const int nwords = (n_hist + 31) / 32;
  uint32_t base = 0;
  if (k_eff > 0) {
    for (int w0 = 0; w0 < nwords; w0 += kSelThreads * 8) {
      uint32_t wv[8];
      uint32_t cnt = 0;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int w = w0 + t * 8 + i;
        wv[i] = (w < nwords) ? bitmap[w] : 0u;
        cnt += __popc(wv[i]);
      }
      uint32_t excl;
      const uint32_t total = block_exclusive_scan(cnt, scratch, excl);
      uint32_t pos = base + excl;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        uint32_t v = wv[i];
        const int w = w0 + t * 8 + i;
        while (v) {
          const int bit = __ffs(v) - 1;
          v &= v - 1;
          if (idx2) idx2[pos] = w * 32 + bit;
          idx[pos++] = w * 32 + bit;
        }
      }
      base += total;
    }
  }
  for (int i = t; i < L - n_hist; i += kSelThreads) {
    idx[k_eff + i] = n_hist + i;
    if (idx2) idx2[k_eff + i] = n_hist + i;
  }
  if (t == 0) {
    ctr[1] = 0;
    ctr[2] = 0;
  }
}

hipError_t launch_select(const Problem& P, const Workspace& ws, int64_t L, const float* scores,
                         int64_t score_stride, int32_t* idx, int32_t* idx_copy, hipStream_t st) {
  const int64_t n_hist = std::max<int64_t>(L - P.W, 0);
  const int m = (int)(std::min<int64_t>(P.k, n_hist) + std::min<int64_t>(P.W, L));
  dim3 grid((unsigned)std::max<int64_t>(1, (n_hist + kSelChunk - 1) / kSelChunk), P.B);
  hipLaunchKernelGGL(k_select, grid, dim3(kSelThreads), 0, st, scores, score_stride, ws.hist, ws.cand, ws.bitmap,
                     ws.counters, idx, idx_copy, (int64_t)m, P.cap, (int)L, P.W, P.k);
  return hipGetLastError();
}

}  // namespace s4r
