// Basis construction of the prefill stage (Section 3.1.2, Eq. svd): the
// hybrid token sample, token-wise L2 normalisation of the sampled rows (each
// basis group's slice on its own), optional mean-centring, and the top-rank
// right singular vectors of the sampled matrix X [n_s, Dg] per (sequence,
// key/value, basis group).
//
// The right singular vectors of X are the eigenvectors of its Gram matrix
// M = X^T X (centred: X^T X - n_s mu mu^T).  M is formed here in fp64 from the
// stored bf16 rows (64 x 64 output tiles per workgroup, upper triangle only,
// written to both halves); the symmetric eigenproblem of every M runs in
// rocSOLVER's batched divide-and-conquer solver (fp64) inside the caller's
// workspace; the eigenvectors of the `rank` largest eigenvalues, largest
// first, become the bases in the storage format.
#include <rocblas/rocblas.h>
#include <rocsolver/rocsolver.h>

#include <algorithm>
#include <cmath>
#include <mutex>

#include "s4r_device.h"
#include "s4r_internal.h"

namespace s4r {

constexpr int kGramTile = 64;     // output tile of the Gram kernel
constexpr int kGramChunk = 32;    // samples staged per LDS round
constexpr int kMeanChunks = 32;   // partial column sums (fixed-order merge)

// ---- sampling -------------------------------------------------------------------------
// uniformly spaced early positions (numpy linspace over [0, E - 1], num
// points, rounded half to even), then the recent block [E, T)
__global__ void k_sample_hybrid(int32_t* __restrict__ idx, int64_t T, int n_uniform, int n_recent) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t E = T - n_recent;
  if (i < n_uniform) {
    int64_t v = 0;
    if (n_uniform > 1) {
      if (i == n_uniform - 1) {
        v = E - 1;
      } else {
        const double step = (double)(E - 1) / (double)(n_uniform - 1);
        v = (int64_t)rint((double)i * step);
      }
    }
    idx[i] = (int32_t)v;
  } else if (i < (int64_t)n_uniform + n_recent) {
    idx[i] = (int32_t)(E + (i - n_uniform));
  }
}

// ---- normalisation ----------------------------------------------------------------------
// inv[mat][s] = 1 / ||row slice|| (1 for an all-zero slice); mat = (b * 2 + side) * nb + g.
// One wave per sampled row: grid (ceil(n_s / 4), 2 nb, B), 256 threads.
__global__ __launch_bounds__(256) void k_row_norms(const uint16_t* __restrict__ s_k, const uint16_t* __restrict__ s_v,
                                                   const int32_t* __restrict__ idx, double* __restrict__ inv,
                                                   int64_t n_rows, int n_s, int Dp, int nb) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int s = blockIdx.x * 4 + wave;
  const int side = blockIdx.y & 1, g = blockIdx.y >> 1, b = blockIdx.z;
  if (s >= n_s) return;
  const int Dg = Dp / nb;
  const uint16_t* row = (side ? s_v : s_k) + ((int64_t)b * n_rows + idx[s]) * Dp + (int64_t)g * Dg;
  double acc = 0.0;
  for (int d = lane; d < Dg; d += 64) {
    const double x = (double)bf16_bits_to_f32(row[d]);
    acc = fma(x, x, acc);
  }
  for (int o = 32; o > 0; o >>= 1) acc += shfl_xor_d(acc, o);
  if (lane == 0) {
    const int mat = (b * 2 + side) * nb + g;
    inv[(int64_t)mat * n_s + s] = acc > 0.0 ? 1.0 / sqrt(acc) : 1.0;
  }
}

// partial column sums of the normalised samples: part[mat][chunk][d], chunk c
// covering samples c, c + kMeanChunks, ...; grid (Dg / 256, 2 nb * kMeanChunks, B)
__global__ __launch_bounds__(256) void k_col_partial(const uint16_t* __restrict__ s_k, const uint16_t* __restrict__ s_v,
                                                     const int32_t* __restrict__ idx, const double* __restrict__ inv,
                                                     double* __restrict__ part, int64_t n_rows, int n_s, int Dp,
                                                     int nb) {
  const int d = blockIdx.x * 256 + threadIdx.x;
  const int sg = blockIdx.y / kMeanChunks, c = blockIdx.y % kMeanChunks;
  const int side = sg & 1, g = sg >> 1, b = blockIdx.z;
  const int Dg = Dp / nb;
  const int mat = (b * 2 + side) * nb + g;
  const uint16_t* base = (side ? s_v : s_k) + (int64_t)b * n_rows * Dp + (int64_t)g * Dg + d;
  double acc = 0.0;
  for (int s = c; s < n_s; s += kMeanChunks)
    acc = fma((double)bf16_bits_to_f32(base[(int64_t)idx[s] * Dp]), inv[(int64_t)mat * n_s + s], acc);
  part[((int64_t)mat * kMeanChunks + c) * Dg + d] = acc;
}

// ---- Gram matrix --------------------------------------------------------------------------
// M[mat] (column-major Dg x Dg) = sum_s xh_s xh_s^T (- n_s mu mu^T when centred).
// Grid (T (T + 1) / 2 upper tiles, 2 nb, B) with T = Dg / 64; 256 threads.
// The samples of a round (32 of them, both 64-column ranges, weighted by the
// row norms' inverses) are staged in LDS as fp64, the next round's requested
// while the current one is multiplied; wave w accumulates the
// 32 x 32 quadrant (w / 2, w % 2) of the tile on the fp64 matrix cores
// (16x16x4: lane l holds A[row l % 16][sample l / 16] and B[sample l / 16]
// [column l % 16], and receives D rows l / 16 + 4 i of column l % 16, as
// probed on gfx950), four 16 x 16 blocks per wave, four samples per step.
typedef double double4_t __attribute__((ext_vector_type(4)));
__global__ __launch_bounds__(256) void k_gram(const uint16_t* __restrict__ s_k, const uint16_t* __restrict__ s_v,
                                              const int32_t* __restrict__ idx, const double* __restrict__ inv,
                                              const double* __restrict__ part, double* __restrict__ M,
                                              int64_t n_rows, int n_s, int Dp, int nb, int center) {
  const int Dg = Dp / nb;
  const int nt = Dg / kGramTile;
  // upper-triangle tile (ti <= tj) of linear index blockIdx.x
  int ti = 0, rem = blockIdx.x;
  while (rem >= nt - ti) {
    rem -= nt - ti;
    ++ti;
  }
  const int tj = ti + rem;
  const int side = blockIdx.y & 1, g = blockIdx.y >> 1, b = blockIdx.z;
  const int mat = (b * 2 + side) * nb + g;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int lr = lane & 15, lk = lane >> 4;       // MFMA operand row / column, sample within the step
  const int qr = (wave >> 1) * 32, qc = (wave & 1) * 32;   // the wave's quadrant
  const uint16_t* base = (side ? s_v : s_k) + (int64_t)b * n_rows * Dp + (int64_t)g * Dg;
  const double* inv_m = inv + (int64_t)mat * n_s;
  __shared__ double xa[kGramChunk][kGramTile + 1], xb[kGramChunk][kGramTile + 1];
  double4_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = double4_t{0.0, 0.0, 0.0, 0.0};
  const int i0 = ti * kGramTile, j0 = tj * kGramTile;
  // the next round's sample values are requested before this round's MFMAs
  // run and written to LDS after them (8 per thread and column range)
  constexpr int kPer = kGramChunk * kGramTile / 256;
  uint16_t ra[kPer], rb[kPer];
  double rw[kPer];
  auto fetch = [&](int s0) __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int e = t + k * 256, r = e / kGramTile, col = e % kGramTile;
      const int s = min(s0 + r, n_s - 1);
      const uint16_t* row = base + (int64_t)idx[s] * Dp;
      ra[k] = row[i0 + col];
      rb[k] = row[j0 + col];
      rw[k] = (s0 + r < n_s) ? inv_m[s] : 0.0;
    }
  };
  auto stage = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int e = t + k * 256, r = e / kGramTile, col = e % kGramTile;
      xa[r][col] = (double)bf16_bits_to_f32(ra[k]) * rw[k];
      xb[r][col] = (double)bf16_bits_to_f32(rb[k]) * rw[k];
    }
  };
  fetch(0);
  stage();
  __syncthreads();
  for (int s0 = 0; s0 < n_s; s0 += kGramChunk) {
    if (s0 + kGramChunk < n_s) fetch(s0 + kGramChunk);
#pragma unroll
    for (int k4 = 0; k4 < kGramChunk; k4 += 4) {
      double a[2], bb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) a[i] = xa[k4 + lk][qr + 16 * i + lr];
#pragma unroll
      for (int j = 0; j < 2; ++j) bb[j] = xb[k4 + lk][qc + 16 * j + lr];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[i], bb[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
    if (s0 + kGramChunk < n_s) {
      stage();
      __syncthreads();
    }
  }
  double* Mm = M + (int64_t)mat * Dg * Dg;
  const double* pm = part + (int64_t)mat * kMeanChunks * Dg;
  const double inv_n = 1.0 / (double)n_s;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int gj = j0 + qc + 16 * j + lr;
    double mj = 0.0;
    if (center)
      for (int c = 0; c < kMeanChunks; ++c) mj += pm[(int64_t)c * Dg + gj];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int gi = i0 + qr + 16 * i + lk + 4 * e;
        double v = acc[i][j][e];
        if (center) {
          double mi = 0.0;
          for (int c = 0; c < kMeanChunks; ++c) mi += pm[(int64_t)c * Dg + gi];
          v -= (mi * inv_n) * (mj * inv_n) * (double)n_s;
        }
        Mm[gi + (int64_t)gj * Dg] = v;
        Mm[gj + (int64_t)gi * Dg] = v;
      }
  }
}

// ---- bases ----------------------------------------------------------------------------------
// bases[b][g][d][c] = eigenvector (Dg - 1 - c) of M[(b * 2 + side) * nb + g],
// component d (eigenvalues ascending), in the storage format, for the
// configured rank's columns c < rank_*; the padding columns up to the storage
// width (stride_*) are zero.  A matrix whose eigensolve did not converge
// (info != 0) gets quiet-NaN bases, so the failure reaches the caller.
template <typename T>
__global__ __launch_bounds__(256) void k_write_bases(const double* __restrict__ V, const rocblas_int* __restrict__ info,
                                                     T* __restrict__ bases_k, T* __restrict__ bases_v, int B, int nb,
                                                     int Dg, int stride_k, int stride_v, int rank_k, int rank_v) {
  const int side = blockIdx.y;
  const int stride = side ? stride_v : stride_k, rank = side ? rank_v : rank_k;
  const int64_t n = (int64_t)B * nb * Dg * stride;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x) {
    const int c = (int)(e % stride);
    const int d = (int)((e / stride) % Dg);
    const int g = (int)((e / ((int64_t)stride * Dg)) % nb);
    const int b = (int)(e / ((int64_t)stride * Dg * nb));
    const int mat = (b * 2 + side) * nb + g;
    const double v = c < rank ? V[(int64_t)mat * Dg * Dg + d + (int64_t)(Dg - 1 - c) * Dg] : 0.0;
    store_elem(side ? bases_v : bases_k, e, info[mat] == 0 ? v : __builtin_nan(""));
  }
}

// ---- host side -----------------------------------------------------------------------------

// one rocBLAS handle per device, created on first use and kept until the
// process ends (its workspace is always the caller's); handle_mutex(dev)
// serialises the set-stream / set-workspace / solve sequence of host threads
static std::mutex g_handle_mu[64];
static rocblas_handle device_handle(hipError_t& err) {
  static std::mutex mu;
  static rocblas_handle handles[64] = {};
  int dev = 0;
  err = hipGetDevice(&dev);
  if (err != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  std::lock_guard<std::mutex> lk(mu);
  if (!handles[dev] && rocblas_create_handle(&handles[dev]) != rocblas_status_success) {
    err = hipErrorUnknown;
    return nullptr;
  }
  return handles[dev];
}

void bases_sample_counts(int64_t T, double eta, int* n_uniform, int* n_recent) {
  const int64_t n = std::max<int64_t>(1, (int64_t)std::floor(eta * (double)T));
  const int64_t nr = std::min<int64_t>(T, (int64_t)std::nearbyint(0.7 * (double)n));
  const int64_t nu = n - nr;
  const int64_t E = T - nr;
  *n_recent = (int)nr;
  *n_uniform = (nu > 0 && E > 0) ? (int)std::min<int64_t>(nu, E) : 0;
}

namespace {
struct BasesLayout {
  size_t m, d, e, info, inv, part, idx, solver, total;
};
BasesLayout bases_layout(const Problem& P, int n_s, size_t solver_bytes) {
  auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
  const size_t nmat = (size_t)P.B * 2 * P.nb, Dg = P.Dg;
  BasesLayout l;
  size_t o = 0;
  l.m = o;
  o = al(o + nmat * Dg * Dg * 8);
  l.d = o;
  o = al(o + nmat * Dg * 8);
  l.e = o;
  o = al(o + nmat * Dg * 8);
  l.info = o;
  o = al(o + nmat * sizeof(rocblas_int));
  l.inv = o;
  o = al(o + nmat * (size_t)n_s * 8);
  l.part = o;
  o = al(o + nmat * kMeanChunks * Dg * 8);
  l.idx = o;
  o = al(o + (size_t)n_s * 4);
  l.solver = o;
  o = al(o + solver_bytes);
  l.total = o;
  return l;
}

// device memory rocSOLVER asks for (a size query: nothing runs)
hipError_t solver_bytes(const Problem& P, size_t* bytes) {
  hipError_t err = hipSuccess;
  rocblas_handle h = device_handle(err);
  if (!h) return err == hipSuccess ? hipErrorUnknown : err;
  const int nmat = P.B * 2 * P.nb, Dg = P.Dg;
  double* dummy = reinterpret_cast<double*>(256);   // never dereferenced in a size query
  int dev = 0;
  if ((err = hipGetDevice(&dev)) != hipSuccess) return err;
  std::lock_guard<std::mutex> lk(g_handle_mu[dev]);
  if (rocblas_start_device_memory_size_query(h) != rocblas_status_success) return hipErrorUnknown;
  rocsolver_dsyevd_strided_batched(h, rocblas_evect_original, rocblas_fill_upper, Dg, dummy, Dg,
                                   (rocblas_stride)Dg * Dg, dummy, Dg, dummy, Dg,
                                   reinterpret_cast<rocblas_int*>(dummy), nmat);
  size_t sz = 0;
  if (rocblas_stop_device_memory_size_query(h, &sz) != rocblas_status_success) return hipErrorUnknown;
  *bytes = sz;
  return hipSuccess;
}
}  // namespace

hipError_t prefill_bases_ws_bytes(const Problem& P, int n_s, size_t* bytes) {
  size_t sb = 0;
  hipError_t e = solver_bytes(P, &sb);
  if (e != hipSuccess) return e;
  *bytes = bases_layout(P, n_s, sb).total;
  return hipSuccess;
}

hipError_t launch_prefill_bases(const Problem& P, int64_t n_rows, const void* s_k, const void* s_v, int n_uniform,
                                int n_recent, int center, int32_t* idx_out, void* bases_k, void* bases_v, void* ws,
                                size_t ws_bytes, hipStream_t st) {
  const int n_s = n_uniform + n_recent;
  size_t sb = 0;
  hipError_t e = solver_bytes(P, &sb);
  if (e != hipSuccess) return e;
  const BasesLayout l = bases_layout(P, n_s, sb);
  if (ws_bytes < l.total) return hipErrorInvalidValue;
  char* w = static_cast<char*>(ws);
  double* M = reinterpret_cast<double*>(w + l.m);
  double* D = reinterpret_cast<double*>(w + l.d);
  double* E = reinterpret_cast<double*>(w + l.e);
  rocblas_int* info = reinterpret_cast<rocblas_int*>(w + l.info);
  double* inv = reinterpret_cast<double*>(w + l.inv);
  double* part = reinterpret_cast<double*>(w + l.part);
  int32_t* idx = reinterpret_cast<int32_t*>(w + l.idx);
  const int nb = P.nb, Dg = P.Dg, Dp = P.Dp;
  const uint16_t* sk = static_cast<const uint16_t*>(s_k);
  const uint16_t* sv = static_cast<const uint16_t*>(s_v);

  hipLaunchKernelGGL(k_sample_hybrid, dim3((n_s + 255) / 256), dim3(256), 0, st, idx, n_rows, n_uniform, n_recent);
  hipLaunchKernelGGL(k_row_norms, dim3((n_s + 3) / 4, 2 * nb, P.B), dim3(256), 0, st, sk, sv, idx, inv, n_rows, n_s,
                     Dp, nb);
  if (center)
    hipLaunchKernelGGL(k_col_partial, dim3(Dg / 256, 2 * nb * kMeanChunks, P.B), dim3(256), 0, st, sk, sv, idx, inv,
                       part, n_rows, n_s, Dp, nb);
  const int nt = Dg / kGramTile;
  hipLaunchKernelGGL(k_gram, dim3(nt * (nt + 1) / 2, 2 * nb, P.B), dim3(256), 0, st, sk, sv, idx, inv, part, M,
                     n_rows, n_s, Dp, nb, center);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  rocblas_handle h = device_handle(e);
  if (!h) return e == hipSuccess ? hipErrorUnknown : e;
  int dev = 0;
  if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
  std::lock_guard<std::mutex> lk(g_handle_mu[dev]);
  if (rocblas_set_stream(h, st) != rocblas_status_success) return hipErrorUnknown;
  if (rocblas_set_workspace(h, w + l.solver, sb) != rocblas_status_success) return hipErrorUnknown;
  const rocblas_status rs = rocsolver_dsyevd_strided_batched(
      h, rocblas_evect_original, rocblas_fill_upper, Dg, M, Dg, (rocblas_stride)Dg * Dg, D, Dg, E, Dg, info,
      P.B * 2 * nb);
  // the handle must not keep pointing into the caller's memory
  rocblas_set_workspace(h, nullptr, 0);
  if (rs != rocblas_status_success) return hipErrorUnknown;
  const int64_t nel = (int64_t)P.B * nb * Dg * std::max(P.rank, P.rank_v);
  const dim3 grid((unsigned)std::min<int64_t>((nel + 255) / 256, 4096), 2);
  if (P.dtype == S4R_BF16)
    hipLaunchKernelGGL(k_write_bases<uint16_t>, grid, dim3(256), 0, st, M, info, (uint16_t*)bases_k,
                       (uint16_t*)bases_v, P.B, nb, Dg, P.rank, P.rank_v, P.rank_cfg, P.rank_v_cfg);
  else
    hipLaunchKernelGGL(k_write_bases<float>, grid, dim3(256), 0, st, M, info, (float*)bases_k, (float*)bases_v, P.B,
                       nb, Dg, P.rank, P.rank_v, P.rank_cfg, P.rank_v_cfg);
  if (idx_out) e = hipMemcpyAsync(idx_out, idx, (size_t)n_s * 4, hipMemcpyDeviceToDevice, st);
  if (e == hipSuccess) e = hipGetLastError();
  return e;
}

}  // namespace s4r
