// Row-major <-> tiled coefficient layout conversion (s4r_pack_coef /
// s4r_unpack_coef).
#include "s4r_device.h"
#include "s4r_internal.h"

namespace s4r {

// ---------------------------------------------------------------------------
// layout conversion
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void k_pack(const T* __restrict__ src, T* __restrict__ dst, int64_t n_rows,
                                              int R, int64_t cap, int to_tiled) {
  const int b = blockIdx.y;
  const int64_t n = n_rows * R;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t t = i / R;
    const int c = (int)(i % R);
    const int64_t ro = (int64_t)b * n_rows * R + i;
    const int64_t to = (int64_t)b * cap * R + tiled_offset(t, c, R);
    if (to_tiled) dst[to] = src[ro];
    else dst[ro] = src[to];
  }
}


hipError_t launch_pack(const Problem& P, int64_t n_rows, const void* src, void* dst, bool to_tiled, hipStream_t st) {
  if (n_rows <= 0) return hipSuccess;
  const int64_t n = n_rows * P.R;
  dim3 grid((unsigned)std::min<int64_t>((n + 255) / 256, 4096), P.B);
  if (P.dtype == S4R_BF16)
    hipLaunchKernelGGL(k_pack<uint16_t>, grid, dim3(256), 0, st, (const uint16_t*)src, (uint16_t*)dst, n_rows, P.R,
                       P.cap, (int)to_tiled);
  else
    hipLaunchKernelGGL(k_pack<float>, grid, dim3(256), 0, st, (const float*)src, (float*)dst, n_rows, P.R, P.cap,
                       (int)to_tiled);
  return hipGetLastError();
}

}  // namespace s4r
