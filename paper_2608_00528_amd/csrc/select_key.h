// Order-preserving keys of relevance scores for the selection histograms
// (Section 3.2.3's top-k): scores are non-negative, so the fp32 bit pattern
// with the (always clear) sign bit shifted out orders like the values, and the
// 11-bit histogram levels resolve 8 exponent and 3 mantissa bits.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "s4r_internal.h"

namespace s4r {

__device__ __forceinline__ uint32_t selection_key(float s) { return __float_as_uint(s) << 1; }

// the same for scores in [0, 1] (the fused step's relevance: means and maxima
// of softmax probabilities): exponent bit 30 is clear too, so two bits shift
// out and the levels resolve 4 mantissa bits; a value above 1, which the
// relevance cannot produce, would tie with 1 instead of wrapping round
__device__ __forceinline__ uint32_t selection_key_unit(float s) { return min(__float_as_uint(s), 0x3F800000u) << 2; }

// key_shift 2: scores in [0, 1] (selection_key_unit); 1: any non-negative
// scores (selection_key)
__device__ __forceinline__ uint32_t selection_key_shift(float s, int key_shift) {
  return key_shift == 2 ? selection_key_unit(s) : selection_key(s);
}

// the fused step's key (the relevance kernel's histogram and the selection
// kernels use the same): the [0, 1] key where the top-k is a large share of
// the positions (its boundary bin then holds many candidates: 10.9k instead
// of 5.5k at k = 0.2 L), else the plain key (fewer non-empty histogram bins
// for the relevance kernel to flush: 2.8 us less at k = 0.016 L)
inline int fused_key_shift(const Problem& P, int64_t L) {
  const int64_t n_hist = std::max<int64_t>(L - P.W, 0);
  return std::min<int64_t>(P.k, n_hist) * 16 >= n_hist ? 2 : 1;
}

// the selection kernels with the key the scores' range allows
// (hist_nc: the copies of the top-level histogram that its producer flushed into)
hipError_t launch_select_keyed(const Problem& P, const Workspace& ws, int64_t L, const float* scores,
                               int64_t score_stride, int32_t* idx, int32_t* idx_copy, int key_shift, int hist_nc,
                               hipStream_t st);

}  // namespace s4r
