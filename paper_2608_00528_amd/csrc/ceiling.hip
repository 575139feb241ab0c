// Read-bandwidth reference for roofline calibration (s4r_read_bandwidth): one
// pass over a buffer in the access pattern that measured fastest on MI355X --
// every workgroup streams one contiguous range with 16-byte non-temporal
// loads, eight per lane in flight, 2048 workgroups.  It computes an XOR of
// every 32-bit word so the loads cannot be dropped; one value per thread.
#include "s4r_device.h"
#include "s4r_internal.h"

namespace s4r {

constexpr int kCeilPer = 8;
constexpr int kCeilGrid = 2048;

__global__ __launch_bounds__(256) void k_read_all(const uint4* __restrict__ src, int64_t n16,
                                                  uint32_t* __restrict__ sink) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  const int64_t chunk = (n16 + gridDim.x - 1) / gridDim.x;
  const int64_t c0 = (int64_t)blockIdx.x * chunk;
  const int64_t c1 = min(c0 + chunk, n16);
  uint32_t acc = 0;
  for (int64_t base = c0 + threadIdx.x; base < c1; base += kCeilPer * 256) {
    u32x4 v[kCeilPer];
#pragma unroll
    for (int k = 0; k < kCeilPer; ++k)
      v[k] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src + min(base + k * 256, c1 - 1)));
#pragma unroll
    for (int k = 0; k < kCeilPer; ++k) {
      const uint32_t x = v[k].x ^ v[k].y ^ v[k].z ^ v[k].w;
      acc ^= (base + k * 256 < c1) ? x : 0u;   // clamped re-reads do not count
    }
  }
  sink[(int64_t)blockIdx.x * 256 + threadIdx.x] = acc;
}

int read_bandwidth_threads() { return 256 * kCeilGrid; }

hipError_t launch_read_all(const void* buf, int64_t n16, uint32_t* sink, hipStream_t st) {
  hipLaunchKernelGGL(k_read_all, dim3(kCeilGrid), dim3(256), 0, st, (const uint4*)buf, n16, sink);
  return hipGetLastError();
}

}  // namespace s4r
