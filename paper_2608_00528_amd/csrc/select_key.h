// Order-preserving key of a relevance score for the selection histograms
// (Section 3.2.3's top-k): scores are non-negative, so the fp32 bit pattern
// with the (always clear) sign bit shifted out orders like the values, and the
// 11-bit histogram levels resolve 8 exponent and 3 mantissa bits.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace s4r {

__device__ __forceinline__ uint32_t selection_key(float s) { return __float_as_uint(s) << 1; }

}  // namespace s4r
