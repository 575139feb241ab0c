// Read-bandwidth reference for roofline calibration: one pass over a buffer
// with 16-byte loads, twenty per lane in flight, grid-stride over the whole
// chip (s4r_read_bandwidth).  It computes an XOR of every 32-bit word so the
// loads cannot be dropped; the value is returned per thread.
#include "s4r_device.h"
#include "s4r_internal.h"

namespace s4r {

constexpr int kCeilPer = 20;

__global__ __launch_bounds__(256) void k_read_all(const uint4* __restrict__ src, int64_t n16,
                                                  uint32_t* __restrict__ sink) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  uint32_t acc = 0;
  for (int64_t base = gid; base < n16; base += kCeilPer * stride) {
    uint4 v[kCeilPer];
#pragma unroll
    for (int k = 0; k < kCeilPer; ++k) v[k] = src[min(base + k * stride, n16 - 1)];
#pragma unroll
    for (int k = 0; k < kCeilPer; ++k) {
      const uint32_t x = v[k].x ^ v[k].y ^ v[k].z ^ v[k].w;
      acc ^= (base + k * stride < n16) ? x : 0u;   // clamped re-reads do not count
    }
  }
  sink[gid] = acc;
}

int read_bandwidth_threads() { return 256 * 2048; }

hipError_t launch_read_all(const void* buf, int64_t n16, uint32_t* sink, hipStream_t st) {
  hipLaunchKernelGGL(k_read_all, dim3(2048), dim3(256), 0, st, (const uint4*)buf, n16, sink);
  return hipGetLastError();
}

}  // namespace s4r
