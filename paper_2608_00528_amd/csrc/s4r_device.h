// Device-side helpers shared by the gfx950 kernels of the S^4R library:
// storage-format conversions, the tiled coefficient layout, bf16 MFMA
// wrappers and wave-level shuffles.  CDNA4 only (wave64, MFMA 16x16x32 bf16).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace s4r {

constexpr int kWave = 64;
constexpr int kTileTok = 16;   // tokens per coefficient tile
constexpr int kBlkCol = 32;    // latent columns per coefficient block

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// storage formats
// ---------------------------------------------------------------------------
struct BF16 {  // bf16 stored as its 16-bit pattern
  using storage = uint16_t;
};
struct F32 {
  using storage = float;
};

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

// fp32 -> bf16 bits, round to nearest even (finite inputs)
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ float load_elem(const uint16_t* p, int64_t i) {
  return bf16_bits_to_f32(p[i]);
}
__device__ __forceinline__ float load_elem(const float* p, int64_t i) { return p[i]; }

__device__ __forceinline__ void store_elem(uint16_t* p, int64_t i, double v) {
  p[i] = (uint16_t)f32_to_bf16_bits((float)v);
}
__device__ __forceinline__ void store_elem(float* p, int64_t i, double v) { p[i] = (float)v; }

// ---------------------------------------------------------------------------
// tiled coefficient layout: element (t, c) of one sequence's [cap, R] block
// ---------------------------------------------------------------------------
__device__ __forceinline__ int64_t tiled_offset(int64_t t, int c, int R) {
  return (t >> 4) * (int64_t)(kTileTok * R) + (int64_t)(c >> 5) * (kTileTok * kBlkCol) +
         (int64_t)(t & 15) * kBlkCol + (c & 31);
}

// ---------------------------------------------------------------------------
// bf16 splits: x ~= hi + mid + lo, each a bf16 value (~24 significant bits)
// ---------------------------------------------------------------------------
struct Split3 {
  uint16_t hi, mid, lo;
};

__device__ __forceinline__ Split3 split3(double x) {
  Split3 s;
  uint32_t h = f32_to_bf16_bits((float)x);
  double r1 = x - (double)bf16_bits_to_f32(h);
  uint32_t m = f32_to_bf16_bits((float)r1);
  double r2 = r1 - (double)bf16_bits_to_f32(m);
  uint32_t l = f32_to_bf16_bits((float)r2);
  s.hi = (uint16_t)h;
  s.mid = (uint16_t)m;
  s.lo = (uint16_t)l;
  return s;
}

// ---------------------------------------------------------------------------
// MFMA operand packing.  An operand is 8 bf16 values held in 4 VGPRs.
// ---------------------------------------------------------------------------
union Op8 {
  uint4 u;
  bf16x8 v;
  uint16_t h[8];
};

// 8 fp32 values -> three bf16 operands (hi, mid, lo)
__device__ __forceinline__ void split_f32x8(const float* x, Op8& hi, Op8& mid, Op8& lo) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    uint32_t h = f32_to_bf16_bits(x[i]);
    float r1 = x[i] - bf16_bits_to_f32(h);   // exact in fp32
    uint32_t m = f32_to_bf16_bits(r1);
    float r2 = r1 - bf16_bits_to_f32(m);     // exact in fp32
    hi.h[i] = (uint16_t)h;
    mid.h[i] = (uint16_t)m;
    lo.h[i] = (uint16_t)f32_to_bf16_bits(r2);
  }
}

// D = A * B + C for 16x16x32 bf16 (gfx950).  Lane l supplies row l%16 of A
// and column l%16 of B for the k-group l/16 (8 values each); it receives
// D[4*(l/16) + v][l%16], v = 0..3.  The k order inside a group is the same for
// A and B, so any consistent assignment of contraction indices works.
__device__ __forceinline__ floatx4 mfma16x16x32(const Op8& a, const Op8& b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v, b.v, c, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// wave shuffles (ds_bpermute based, full 64-lane)
// ---------------------------------------------------------------------------
__device__ __forceinline__ float shfl_xor_f(float v, int mask) {
  int lane = __lane_id();
  return __int_as_float(__builtin_amdgcn_ds_bpermute((lane ^ mask) << 2, __float_as_int(v)));
}
__device__ __forceinline__ double shfl_xor_d(double v, int mask) {
  int lane = __lane_id();
  int lo = __double2loint(v), hi = __double2hiint(v);
  lo = __builtin_amdgcn_ds_bpermute((lane ^ mask) << 2, lo);
  hi = __builtin_amdgcn_ds_bpermute((lane ^ mask) << 2, hi);
  return __hiloint2double(hi, lo);
}

// Copy n items (16 bytes each) with the whole block: every thread issues PER
// loads before its first store, so a staging pass costs one memory latency per
// PER * blockDim items instead of one per item.  src_of(i) / dst_of(i) map an
// item index to its source and destination.  Neither loads nor stores are
// guarded by a condition: slots past n re-read item n - 1 and write that same
// value to item n - 1's destination.  (A guarded load makes the compiler wait
// for it before the branch joins, and a guarded store lets it sink the load
// into the branch; either serialises the batch.)
template <int PER, typename SrcOf, typename DstOf>
__device__ __forceinline__ void batched_copy16(int n, SrcOf src_of, DstOf dst_of) {
  if (n <= 0) return;
  for (int base = 0; base < n; base += PER * (int)blockDim.x) {
    uint4 r[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) r[k] = *src_of(min(base + k * (int)blockDim.x + (int)threadIdx.x, n - 1));
#pragma unroll
    for (int k = 0; k < PER; ++k) *dst_of(min(base + k * (int)blockDim.x + (int)threadIdx.x, n - 1)) = r[k];
  }
}

// same for 4-byte items; src_of(i) returns the value, dst_of(i, v) stores it
template <int PER, typename SrcOf, typename DstOf>
__device__ __forceinline__ void batched_copy4(int n, SrcOf src_of, DstOf dst_of) {
  if (n <= 0) return;
  for (int base = 0; base < n; base += PER * (int)blockDim.x) {
    float r[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) r[k] = src_of(min(base + k * (int)blockDim.x + (int)threadIdx.x, n - 1));
#pragma unroll
    for (int k = 0; k < PER; ++k) dst_of(min(base + k * (int)blockDim.x + (int)threadIdx.x, n - 1), r[k]);
  }
}

// reductions over the 16 token slots of a wave (lane bits 0..3) with DPP:
// quad_perm swaps for bits 0 and 1, row rotations by 4 and 8 for bits 2 and 3
template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float slot_max16(float x) {
  x = fmaxf(x, dpp_f<0xB1>(x));    // quad_perm [1,0,3,2]
  x = fmaxf(x, dpp_f<0x4E>(x));    // quad_perm [2,3,0,1]
  x = fmaxf(x, dpp_f<0x124>(x));   // row_ror:4
  x = fmaxf(x, dpp_f<0x128>(x));   // row_ror:8
  return x;
}
__device__ __forceinline__ float slot_sum16(float x) {
  x += dpp_f<0xB1>(x);
  x += dpp_f<0x4E>(x);
  x += dpp_f<0x124>(x);
  x += dpp_f<0x128>(x);
  return x;
}

// Workgroup barrier for LDS exchange only: waits for this wave's LDS traffic
// (lgkmcnt) but not for outstanding global loads (vmcnt), so prefetched
// global data stays in flight across the barrier.  (__syncthreads() waits for
// every outstanding memory operation.)  The signal fences keep the compiler
// from moving memory accesses across it.
__device__ __forceinline__ void lds_barrier() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0xC07F);   // gfx9 encoding: lgkmcnt(0), vmcnt/expcnt not waited
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Wave-aggregated append.  Lanes of one wave that hit the same LDS word in one
// atomic instruction are serialised by the hardware; this issues one atomic
// per wave instead.  Every active lane of the wave must make the call
// (inactive lanes simply do not take part).

// reserves one slot of *counter for every active lane with pred; returns the
// lane's slot (in lane order within the wave), undefined where pred is false
__device__ __forceinline__ uint32_t wave_append(uint32_t* counter, bool pred) {
  const uint64_t m = __ballot(pred);
  if (m == 0) return 0u;
  const int leader = __ffsll((unsigned long long)m) - 1;
  uint32_t base = 0u;
  if (__lane_id() == leader) base = atomicAdd(counter, (uint32_t)__popcll(m));
  base = (uint32_t)__shfl((int)base, leader);
  const int lane = __lane_id();
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  return base + (uint32_t)__popcll(m & below);
}

// exp(x) for x <= 0 given in fp64: 2^(x log2 e) with the integer part split off
// in fp64, the fraction evaluated by the hardware exp2 (relative error about
// one fp32 ulp for any x)
__device__ __forceinline__ float exp_neg_accurate(double x) {
  const double y = x * 1.4426950408889634;
  const double n = rint(y);
  const float f = (float)(y - n);
  return ldexpf(__builtin_amdgcn_exp2f(f), (int)fmax(n, -300.0));
}

}  // namespace s4r
