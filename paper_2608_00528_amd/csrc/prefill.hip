// Bulk projection of the prefill stage (Section 3.1, the coefficient
// equation): C = S B for every non-sink prompt row, per basis group, written
// into the tiled coefficient cache (bf16 storage).
//
// k_transpose_bases first writes every basis group transposed, [column][dim],
// into the workspace.  k_prefill_project: grid (128-row blocks, basis group x
// {key, value}, sequence), 4 waves; wave w owns 2 tiles of 16 rows.  The
// product runs on bf16 MFMA 16x16x32 with fp32 accumulation in the MFMA
// accumulators: A = the prompt rows as loaded (lane: row l % 16, dims
// 8 (l / 16) .. + 7 of a 32-dim block), B = the transposed basis slice of the
// block (one 16-byte LDS read per operand), brought into a ring of LDS buffers
// by 16-byte global->LDS loads two blocks ahead (lane l of a wave load lands
// at byte 16 l: 16 columns x 32 dims per instruction); the rows of the next
// block are in flight in registers.  bf16 inputs make every product exact; the
// fp32 sums are rounded once to bf16.
#include "s4r_device.h"
#include "s4r_internal.h"

namespace s4r {

constexpr int kPfWaves = 4;
constexpr int kPfTiles = 2;                       // 16-row tiles per wave (two waves per SIMD:
                                                  // 737 us at the headline shape, 931 with four
                                                  // tiles at one wave per SIMD, 864 with one tile)
constexpr int kPfRows = kPfWaves * kPfTiles * 16;  // rows per workgroup

// s_waitcnt vmcnt(N) alone (gfx9 encoding: expcnt and lgkmcnt not waited)
template <int N>
__device__ __forceinline__ void pf_wait_vmcnt() {
  static_assert(N >= 0 && N < 16, "small counts only");
  __builtin_amdgcn_s_waitcnt(N | (7 << 4) | (15 << 8));
}

// bases [B|1][nb][Dg][rank] -> bt [B][2][nb][rank][Dg]: grid (Dg / 32, 2 nb, B),
// one 32-row x rank block per workgroup through LDS
__global__ __launch_bounds__(256) void k_transpose_bases(const uint16_t* __restrict__ bases_k,
                                                         const uint16_t* __restrict__ bases_v,
                                                         uint16_t* __restrict__ bt, int Dg, int nb, int rank,
                                                         int bases_shared) {
  const int d0 = blockIdx.x * 32, gz = blockIdx.y, b = blockIdx.z;
  const int grp = gz >> 1, which = gz & 1;
  const int Dp = Dg * nb;
  const uint16_t* src = (which == 0 ? bases_k : bases_v) + (bases_shared ? 0 : (int64_t)b * Dp * rank) +
                        (int64_t)grp * Dg * rank;
  uint16_t* dst = bt + (((int64_t)b * 2 + which) * nb + grp) * (int64_t)rank * Dg;
  __shared__ uint16_t tile[32][256 + 2];
  for (int i = threadIdx.x; i < 32 * rank; i += blockDim.x) tile[i / rank][i % rank] = src[(int64_t)(d0 + i / rank) * rank + i % rank];
  __syncthreads();
  for (int i = threadIdx.x; i < 32 * rank; i += blockDim.x) {
    const int c = i / 32, d = i % 32;
    dst[(int64_t)c * Dg + d0 + d] = tile[d][c];
  }
}

template <int RBH>
__global__ __launch_bounds__(kPfWaves * 64) void k_prefill_project(
    const uint16_t* __restrict__ s_k, const uint16_t* __restrict__ s_v, const uint16_t* __restrict__ bt_all,
    uint16_t* __restrict__ coef_k, uint16_t* __restrict__ coef_v, int64_t n_rows, int hkv, int dh, int nb, int R,
    int64_t cap) {
  constexpr int RANK = RBH * 32;
  constexpr int NCB = RANK / 16;                  // 16-column blocks of the group
  constexpr int NBUF = 3;                         // slice buffers: two blocks ahead
  const int blk = blockIdx.x, gz = blockIdx.y, b = blockIdx.z;
  const int grp = gz >> 1, which = gz & 1;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int slot = lane & 15, kq = lane >> 4;
  const int Dp = hkv * dh, Dg = Dp / nb;
  const int nkb = Dg / 32;
  const uint16_t* S = (which == 0 ? s_k : s_v) + (int64_t)b * n_rows * Dp + (int64_t)grp * Dg;
  const uint16_t* Bt = bt_all + (((int64_t)b * 2 + which) * nb + grp) * (int64_t)RANK * Dg;
  uint16_t* C = (which == 0 ? coef_k : coef_v) + (int64_t)b * cap * R;

  __shared__ __align__(16) uint16_t bt[NBUF][RANK][32];

  const int64_t row0 = (int64_t)blk * kPfRows + (w * kPfTiles) * 16;
  // slice kb: NCB wave loads of 16 columns x 32 dims, shared out over the waves
  // (lane l: column 16 n + l / 4, dims 8 (l % 4) .. + 7 -> LDS byte 16 l)
  // (a macro, the LDS destination through a plain local pointer: with the
  // array expression passed to the builtin directly the host pass drops the
  // kernel's launch stub)
#define S4R_PF_ISSUE_SLICE(KB)                                                                           \
  do {                                                                                                   \
    _Pragma("unroll") for (int n0 = 0; n0 < NCB; n0 += kPfWaves) {                                       \
      const int n_ = n0 + w;                                                                             \
      if (n_ < NCB) {                                                                                    \
        uint16_t* dst_ = &bt[(KB) % NBUF][16 * n_][0];                                                   \
        __builtin_amdgcn_global_load_lds(Bt + (int64_t)(16 * n_ + (lane >> 2)) * Dg + (KB) * 32 + (lane & 3) * 8, \
                                         dst_, 16, 0, 0);                                                \
      }                                                                                                  \
    }                                                                                                    \
  } while (0)
  // this wave's share of a slice's wave loads (n = w, w + 4, ... < NCB)
  const int my_slice_loads = w < NCB ? (NCB - w + kPfWaves - 1) / kPfWaves : 0;
  auto load_rows = [&](int kb, Op8 (&a)[kPfTiles]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < kPfTiles; ++i) {
      const int64_t r = min(row0 + i * 16 + slot, n_rows - 1);
      a[i].u = *reinterpret_cast<const uint4*>(S + r * Dp + kb * 32 + kq * 8);
    }
  };

  floatx4 acc[kPfTiles][NCB];
#pragma unroll
  for (int i = 0; i < kPfTiles; ++i)
#pragma unroll
    for (int n = 0; n < NCB; ++n) acc[i][n] = floatx4{0.f, 0.f, 0.f, 0.f};

  // issue order per wave: slice 0, rows 0, slice 1, then in iteration kb rows
  // kb + 1 before slice kb + 2; so at the top of iteration kb only the loads of
  // slice kb + 1 may still be in flight
  Op8 a[kPfTiles];
  S4R_PF_ISSUE_SLICE(0);
  load_rows(0, a);
  if (nkb > 1) S4R_PF_ISSUE_SLICE(1);
  for (int kb = 0; kb < nkb; ++kb) {
    // rows kb and this wave's part of slice kb have landed; then every wave's
    if (kb + 1 < nkb) {
      switch (my_slice_loads) {
        case 0: pf_wait_vmcnt<0>(); break;
        case 1: pf_wait_vmcnt<1>(); break;
        case 2: pf_wait_vmcnt<2>(); break;
        default: pf_wait_vmcnt<3>(); break;
      }
    } else {
      pf_wait_vmcnt<0>();
    }
    __syncthreads();
    const bool more = kb + 1 < nkb;
    Op8 an[kPfTiles];
    if (more) load_rows(kb + 1, an);
    if (kb + 2 < nkb) S4R_PF_ISSUE_SLICE(kb + 2);  // its buffer was last read before this barrier
#pragma unroll
    for (int n = 0; n < NCB; ++n) {
      Op8 bop;
      bop.u = *reinterpret_cast<const uint4*>(&bt[kb % NBUF][n * 16 + slot][kq * 8]);
#pragma unroll
      for (int i = 0; i < kPfTiles; ++i) acc[i][n] = mfma16x16x32(a[i], bop, acc[i][n]);
    }
    if (more) {
#pragma unroll
      for (int i = 0; i < kPfTiles; ++i) a[i] = an[i];
    }
  }
#undef S4R_PF_ISSUE_SLICE
  // D layout: lane (column slot, row group kq) holds rows 4 kq + v of the tile
  const int c0 = grp * RANK;
#pragma unroll
  for (int i = 0; i < kPfTiles; ++i)
#pragma unroll
    for (int n = 0; n < NCB; ++n)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t r = row0 + i * 16 + 4 * kq + v;
        const int c = c0 + n * 16 + slot;
        if (r < n_rows) C[tiled_offset(r, c, R)] = (uint16_t)f32_to_bf16_bits(acc[i][n][v]);
      }
}

template <int RBH>
static void launch_pf(const Problem& P, int64_t n_rows, const void* s_k, const void* s_v, const uint16_t* bt,
                      void* coef_k, void* coef_v, hipStream_t st) {
  dim3 grid((unsigned)((n_rows + kPfRows - 1) / kPfRows), 2 * P.nb, P.B);
  hipLaunchKernelGGL(k_prefill_project<RBH>, grid, dim3(kPfWaves * 64), 0, st, (const uint16_t*)s_k,
                     (const uint16_t*)s_v, bt, (uint16_t*)coef_k, (uint16_t*)coef_v, n_rows, P.hkv, P.dh, P.nb, P.R,
                     P.cap);
}

size_t prefill_ws_bytes(const Problem& P) { return (size_t)P.B * 2 * P.hkv * P.dh * P.rank * 2; }

hipError_t launch_prefill_project(const Problem& P, int64_t n_rows, const void* s_k, const void* s_v,
                                  const void* bases_k, const void* bases_v, void* coef_k, void* coef_v, void* ws,
                                  hipStream_t st) {
  uint16_t* bt = (uint16_t*)ws;
  const int Dg = P.hkv * P.dh / P.nb;
  hipLaunchKernelGGL(k_transpose_bases, dim3(Dg / 32, 2 * P.nb, P.B), dim3(256), 0, st, (const uint16_t*)bases_k,
                     (const uint16_t*)bases_v, bt, Dg, P.nb, P.rank, P.bases_shared);
  switch (P.rank / 32) {
    case 1: launch_pf<1>(P, n_rows, s_k, s_v, bt, coef_k, coef_v, st); break;
    case 2: launch_pf<2>(P, n_rows, s_k, s_v, bt, coef_k, coef_v, st); break;
    case 3: launch_pf<3>(P, n_rows, s_k, s_v, bt, coef_k, coef_v, st); break;
    case 4: launch_pf<4>(P, n_rows, s_k, s_v, bt, coef_k, coef_v, st); break;
    case 5: launch_pf<5>(P, n_rows, s_k, s_v, bt, coef_k, coef_v, st); break;
    case 6: launch_pf<6>(P, n_rows, s_k, s_v, bt, coef_k, coef_v, st); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace s4r
