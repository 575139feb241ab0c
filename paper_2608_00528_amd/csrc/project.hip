// Section 3.2.1 (compressed cache update) on gfx950: the query coefficients
// c_t^Q = s_t^Q B^K of every query group and the projection of a new token's
// key and value into coefficient row L-1 (c_t^K = s_t^K B^K, c_t^V = s_t^V B^V).
#include "s4r_device.h"
#include "s4r_internal.h"

namespace s4r {

// ---------------------------------------------------------------------------
// Both kernels: 256 threads = 4 column groups of 8 latent columns x 64 row
// groups; a workgroup owns 32 latent columns of one basis group.  A thread
// holds 4 basis rows (rg + 64 i) of its 8 columns in registers, in storage
// format; the projected vectors are staged in LDS as fp32 (their exact
// values).  Products are accumulated in fp64 and reduced over the 64 row
// groups (DPP within 16-lane rows, shuffles across rows, then the 4 waves
// through LDS) in a fixed order, so results are deterministic.
// ---------------------------------------------------------------------------
constexpr int kPRows = 4;                     // basis rows per thread
constexpr int kPVec = 4;                      // vectors accumulated per pass
constexpr int kRowPre = 4;                    // 256-row chunks of a new row's projection loaded together

// 8 consecutive basis elements, kept in their storage format until used
struct Raw8bf16 {
  uint4 u;
  __device__ __forceinline__ void load(const uint16_t* p) { u = *reinterpret_cast<const uint4*>(p); }
  __device__ __forceinline__ float operator[](int c) const {
    const uint32_t w = (c >> 1) == 0 ? u.x : (c >> 1) == 1 ? u.y : (c >> 1) == 2 ? u.z : u.w;
    return (c & 1) ? __uint_as_float(w & 0xFFFF0000u) : __uint_as_float(w << 16);
  }
};
struct Raw8f32 {
  float4 a, b;
  __device__ __forceinline__ void load(const float* p) {
    a = *reinterpret_cast<const float4*>(p);
    b = *reinterpret_cast<const float4*>(p + 4);
  }
  __device__ __forceinline__ float operator[](int c) const {
    const float4& h = (c < 4) ? a : b;
    const int k = c & 3;
    return k == 0 ? h.x : k == 1 ? h.y : k == 2 ? h.z : h.w;
  }
};
template <typename T>
struct Raw8;
template <>
struct Raw8<uint16_t> {
  using type = Raw8bf16;
};
template <>
struct Raw8<float> {
  using type = Raw8f32;
};

// fp64 move within 16-lane rows (row_ror)
template <int CTRL>
__device__ __forceinline__ double dpp_move_d(double x) {
  const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(x), CTRL, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(x), CTRL, 0xF, 0xF, false);
  return __hiloint2double(hi, lo);
}
// sum over the 16 lanes of a wave that share (lane & 3)
__device__ __forceinline__ double wave_sum16(double a) {
  a += dpp_move_d<0x124>(a);   // row_ror:4
  a += dpp_move_d<0x128>(a);   // row_ror:8
  a += shfl_xor_d(a, 16);
  a += shfl_xor_d(a, 32);
  return a;
}

template <int NV, typename RawT>
__device__ __forceinline__ void accumulate_rows(const RawT (&bw)[kPRows], const float (*xs)[kPChunk], int rg,
                                                double (&acc)[kPVec][8]) {
#pragma unroll
  for (int i = 0; i < kPRows; ++i) {
    const int r = rg + 64 * i;
    double xv[NV];
#pragma unroll
    for (int v = 0; v < NV; ++v) xv[v] = (double)xs[v][r];
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const double bc = (double)bw[i][c];
#pragma unroll
      for (int v = 0; v < NV; ++v) acc[v][c] = fma(xv[v], bc, acc[v][c]);
    }
  }
}

// per-thread sums (NV vectors x 8 columns) -> per-wave sums in red[wave][v][32]
template <int NV>
__device__ __forceinline__ void reduce_rows(double (&acc)[kPVec][8], double (*red)[kPVec][32], int wave, int lane,
                                            int cg) {
#pragma unroll
  for (int v = 0; v < NV; ++v)
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[v][c] = wave_sum16(acc[v][c]);
  if (lane < 4) {
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int c = 0; c < 8; ++c) red[wave][v][cg * 8 + c] = acc[v][c];
  }
}

// ---------------------------------------------------------------------------
// query coefficients: grid (R / 32, ceil(Dg / 256) row chunks, B).  Each
// workgroup writes the partial sums of its 256-row chunk for all G query
// groups to qpart [B][chunks][G][R] (fp64); the scoring kernel adds the
// chunks in a fixed order.  Splitting the rows over workgroups keeps every
// thread's work to one load round trip and a short fp64 dot product.
// ---------------------------------------------------------------------------
template <typename T>
__device__ __forceinline__ void project_query_body(const T* __restrict__ q, const T* __restrict__ bases_k,
                                                   double* __restrict__ qpart, uint32_t* __restrict__ hist, int hq,
                                                   int hkv, int dh, int G, int nb, int rank, int R, int bases_shared,
                                                   int cblk, int ch, int b, int nch) {
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int cg = t & 3, rg = t >> 2;
  const int Dp = hkv * dh, Dg = Dp / nb;
  const int ldh = __builtin_ctz(dh);              // head_dim is a power of two
  const int c0 = cblk * 32;                       // first latent column of the block
  const int grp = c0 / rank;                      // its basis group
  const int r0 = ch * kPChunk;                    // first row of the chunk in the group
  const int nrow = min(kPChunk, Dg - r0);
  // the step's two selection histograms start from zero (the relevance and
  // classify kernels add to them later in the step)
  if (cblk == 0 && ch == 0)
    for (int i = t; i < 2 * kHistBins; i += blockDim.x) hist[(int64_t)b * 2 * kHistBins + i] = 0u;

  __shared__ float xs[kMaxG][kPChunk];
  __shared__ double red[4][kPVec][32];
  const T* bases = bases_k + (bases_shared ? 0 : (int64_t)b * Dp * rank) + ((int64_t)grp * Dg + r0) * rank +
                   (c0 - grp * rank) + cg * 8;
  // basis rows rg + 64 i (addresses clamped; rows past nrow meet x = 0) and
  // the chunk of every group query, all requested before any is used
  typename Raw8<T>::type bw[kPRows];
#pragma unroll
  for (int i = 0; i < kPRows; ++i) bw[i].load(bases + (int64_t)min(rg + 64 * i, nrow - 1) * rank);
  batched_copy4<kMaxG * kPChunk / 256>(
      G * kPChunk,
      [&](int i) -> float {
        const int v = i >> 8, d = grp * Dg + r0 + min(i & (kPChunk - 1), nrow - 1);   // feature index in Dp
        return load_elem(q, ((int64_t)b * hq + (int64_t)(d >> ldh) * G + v) * dh + (d & (dh - 1)));
      },
      [&](int i, float x) { xs[i >> 8][min(i & (kPChunk - 1), nrow - 1)] = x; });
  if (nrow < kPChunk)
    for (int i = t; i < G * kPChunk; i += blockDim.x)
      if ((i & (kPChunk - 1)) >= nrow) xs[i >> 8][i & (kPChunk - 1)] = 0.f;
  __syncthreads();

  for (int v0 = 0; v0 < G; v0 += kPVec) {
    const int nv = min(kPVec, G - v0);
    double acc[kPVec][8];
#pragma unroll
    for (int v = 0; v < kPVec; ++v)
#pragma unroll
      for (int c = 0; c < 8; ++c) acc[v][c] = 0.0;
    const float(*xv)[kPChunk] = xs + v0;
    switch (nv) {
      case 1: accumulate_rows<1>(bw, xv, rg, acc); reduce_rows<1>(acc, red, wave, lane, cg); break;
      case 2: accumulate_rows<2>(bw, xv, rg, acc); reduce_rows<2>(acc, red, wave, lane, cg); break;
      case 3: accumulate_rows<3>(bw, xv, rg, acc); reduce_rows<3>(acc, red, wave, lane, cg); break;
      default: accumulate_rows<4>(bw, xv, rg, acc); reduce_rows<4>(acc, red, wave, lane, cg); break;
    }
    __syncthreads();
    if (t < nv * 32) {
      const int v = t >> 5, c = t & 31;
      const double x = ((red[0][v][c] + red[1][v][c]) + red[2][v][c]) + red[3][v][c];
      qpart[(((int64_t)b * nch + ch) * G + v0 + v) * R + c0 + c] = x;
    }
    __syncthreads();                              // red is reused by the next pass
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_project_query(const T* __restrict__ q, const T* __restrict__ bases_k,
                                                       double* __restrict__ qpart, uint32_t* __restrict__ hist,
                                                       int hq, int hkv, int dh, int G, int nb, int rank, int R,
                                                       int bases_shared) {
  project_query_body<T>(q, bases_k, qpart, hist, hq, hkv, dh, G, nb, rank, R, bases_shared, blockIdx.x, blockIdx.y,
                        blockIdx.z, gridDim.y);
}

// ---------------------------------------------------------------------------
// new token's coefficient rows: grid (R / 32, B, 2 = {key, value}).  The
// workgroup loops over 256-row chunks of its basis group and writes the full
// sums into row append_row of the cache (rounded to the storage format).
// ---------------------------------------------------------------------------
template <typename T>
__device__ __forceinline__ void project_rows_body(const T* __restrict__ bases_k, const T* __restrict__ bases_v,
                                                  const T* __restrict__ k_new, const T* __restrict__ v_new,
                                                  T* __restrict__ coef_k, T* __restrict__ coef_v, int64_t append_row,
                                                  int hkv, int dh, int nb, int rank, int R, int bases_shared,
                                                  int64_t cap, int cblk, int b, int which) {
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int cg = t & 3, rg = t >> 2;
  const int Dp = hkv * dh, Dg = Dp / nb;
  const int c0 = cblk * 32;
  const int grp = c0 / rank;
  const T* x_new = which == 0 ? k_new : v_new;
  T* coef = which == 0 ? coef_k : coef_v;

  __shared__ float xs[kRowPre][kPChunk];
  __shared__ double red[4][kPVec][32];
  const T* bases = (which == 0 ? bases_k : bases_v) + (bases_shared ? 0 : (int64_t)b * Dp * rank) +
                   (int64_t)grp * Dg * rank + (c0 - grp * rank) + cg * 8;
  double acc[kPVec][8];
#pragma unroll
  for (int v = 0; v < kPVec; ++v)
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[v][c] = 0.0;
  // kRowPre chunks of 256 rows at a time: every basis row and vector element
  // of the group is requested before any is used (one memory latency for a
  // basis group of up to 1024 rows), then the chunks are summed in order
  for (int r00 = 0; r00 < Dg; r00 += kRowPre * kPChunk) {
    typename Raw8<T>::type bw[kRowPre][kPRows];
    float x[kRowPre];
#pragma unroll
    for (int ci = 0; ci < kRowPre; ++ci) {
      const int r0 = min(r00 + ci * kPChunk, Dg - 1);   // past the group's end: a re-read, never summed
      const int nrow = min(kPChunk, Dg - r0);
#pragma unroll
      for (int i = 0; i < kPRows; ++i) bw[ci][i].load(bases + (int64_t)(r0 + min(rg + 64 * i, nrow - 1)) * rank);
      x[ci] = load_elem(x_new, (int64_t)b * Dp + grp * Dg + r0 + min(t, nrow - 1));
    }
    if (r00 > 0) __syncthreads();                 // previous group's xs reads are done
#pragma unroll
    for (int ci = 0; ci < kRowPre; ++ci) {
      const int r0 = r00 + ci * kPChunk;
      xs[ci][t] = (r0 + t < Dg) ? x[ci] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int ci = 0; ci < kRowPre; ++ci)
      if (r00 + ci * kPChunk < Dg) accumulate_rows<1>(bw[ci], &xs[ci], rg, acc);
  }
  reduce_rows<1>(acc, red, wave, lane, cg);
  __syncthreads();
  if (t < 32) {
    const double v = ((red[0][0][t] + red[1][0][t]) + red[2][0][t]) + red[3][0][t];
    store_elem(coef, (int64_t)b * cap * R + tiled_offset(append_row, c0 + t, R), v);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_project_rows(const T* __restrict__ bases_k, const T* __restrict__ bases_v,
                                                      const T* __restrict__ k_new, const T* __restrict__ v_new,
                                                      T* __restrict__ coef_k, T* __restrict__ coef_v,
                                                      int64_t append_row, int hkv, int dh, int nb, int rank, int R,
                                                      int rank_v, int Rv, int bases_shared, int64_t cap, Lens lens) {
  // the value side has its own width when the ranks are asymmetric
  const int which = blockIdx.z;
  if ((int)blockIdx.x * 32 >= (which ? Rv : R)) return;
  // a ragged batch appends at each sequence's own last row
  const int64_t row = lens.n ? (int64_t)lens.v[blockIdx.y] - 1 : append_row;
  project_rows_body<T>(bases_k, bases_v, k_new, v_new, coef_k, coef_v, row, hkv, dh, nb, which ? rank_v : rank,
                       which ? Rv : R, bases_shared, cap, blockIdx.x, blockIdx.y, which);
}

// both projections of a step that appends a token, in one launch: blocks
// [0, nq) are the query-coefficient workgroups (R / 32 x chunks x B, in that
// order), the rest the new rows' (max(R, R_V) / 32 x B x 2).  They touch disjoint
// memory, and one launch saves a dispatch and a first-read latency.
template <typename T>
__global__ __launch_bounds__(256) void k_project_step(const T* __restrict__ q, const T* __restrict__ bases_k,
                                                      const T* __restrict__ bases_v, const T* __restrict__ k_new,
                                                      const T* __restrict__ v_new, T* __restrict__ coef_k,
                                                      T* __restrict__ coef_v, double* __restrict__ qpart,
                                                      uint32_t* __restrict__ hist, int64_t append_row, int hq,
                                                      int hkv, int dh, int G, int nb, int rank, int R,
                                                      int rank_v, int Rv, int bases_shared, int64_t cap, int B,
                                                      int nch, Lens lens) {
  const int ncb = R / 32;
  const int nq = ncb * nch * B;
  int id = blockIdx.x;
  if (id < nq) {
    const int cblk = id % ncb, ch = (id / ncb) % nch, b = id / (ncb * nch);
    project_query_body<T>(q, bases_k, qpart, hist, hq, hkv, dh, G, nb, rank, R, bases_shared, cblk, ch, b, nch);
  } else {
    id -= nq;
    const int ncr = max(R, Rv) / 32;               // row blocks per (sequence, side)
    const int cblk = id % ncr, b = (id / ncr) % B, which = id / (ncr * B);
    if (cblk * 32 >= (which ? Rv : R)) return;
    const int64_t row = lens.n ? (int64_t)lens.v[b] - 1 : append_row;
    project_rows_body<T>(bases_k, bases_v, k_new, v_new, coef_k, coef_v, row, hkv, dh, nb, which ? rank_v : rank,
                         which ? Rv : R,
                         bases_shared, cap, cblk, b, which);
  }
}

hipError_t launch_project_query(const Problem& P, double* qpart, uint32_t* hist, const void* q, const void* bases_k,
                                hipStream_t st) {
  dim3 grid(P.R / 32, project_chunks(P), P.B);
  if (P.dtype == S4R_BF16)
    hipLaunchKernelGGL(k_project_query<uint16_t>, grid, dim3(256), 0, st, (const uint16_t*)q,
                       (const uint16_t*)bases_k, qpart, hist, P.hq, P.hkv, P.dh, P.G, P.nb, P.rank, P.R,
                       P.bases_shared);
  else
    hipLaunchKernelGGL(k_project_query<float>, grid, dim3(256), 0, st, (const float*)q, (const float*)bases_k, qpart,
                       hist, P.hq, P.hkv, P.dh, P.G, P.nb, P.rank, P.R, P.bases_shared);
  return hipGetLastError();
}

// rows of C^Q from the query-projection partials: out[b][g][row][r] = the fp32
// rounding of the chunk partials summed in chunk order (the order the scoring
// kernel sums them in)
__global__ __launch_bounds__(256) void k_qcoef_row(const double* __restrict__ qpart, float* __restrict__ out, int B,
                                                   int G, int R, int nch, int64_t n_rows, int64_t row) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= B * G * R) return;
  const int b = i / (G * R), g = (i / R) % G, r = i % R;
  double x = qpart[(((int64_t)b * nch) * G + g) * R + r];
  for (int c = 1; c < nch; ++c) x += qpart[(((int64_t)b * nch + c) * G + g) * R + r];
  out[(((int64_t)b * G + g) * n_rows + row) * R + r] = (float)x;
}

// C^Q rows of n_rows queries [B, n_rows, h_q, d_h]: each row staged as
// [B, h_q, d_h] in the workspace, projected, and its partials summed
hipError_t launch_project_queries(const Problem& P, const Workspace& ws, int64_t n_rows, const void* q_rows,
                                  const void* bases_k, float* out, hipStream_t st) {
  const size_t es = P.dtype == S4R_BF16 ? 2 : 4;
  const size_t row_bytes = (size_t)P.hq * P.dh * es;
  void* staged = ws.part_o;                       // >= B * h_q * d_h * 4 bytes
  const int n = P.B * P.G * P.R;
  for (int64_t row = 0; row < n_rows; ++row) {
    hipError_t e = hipMemcpy2DAsync(staged, row_bytes, static_cast<const char*>(q_rows) + row * row_bytes,
                                    (size_t)n_rows * row_bytes, row_bytes, P.B, hipMemcpyDeviceToDevice, st);
    if (e == hipSuccess) e = launch_project_query(P, ws.qpart, ws.hist, staged, bases_k, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_qcoef_row, dim3((n + 255) / 256), dim3(256), 0, st, ws.qpart, out, P.B, P.G, P.R,
                       project_chunks(P), n_rows, row);
  }
  return hipGetLastError();
}

hipError_t launch_project_rows(const Problem& P, const void* bases_k, const void* bases_v, const void* k_new,
                               const void* v_new, void* coef_k, void* coef_v, int64_t row, hipStream_t st) {
  dim3 grid(std::max(P.R, P.Rv) / 32, P.B, 2);
  if (P.dtype == S4R_BF16)
    hipLaunchKernelGGL(k_project_rows<uint16_t>, grid, dim3(256), 0, st, (const uint16_t*)bases_k,
                       (const uint16_t*)bases_v, (const uint16_t*)k_new, (const uint16_t*)v_new, (uint16_t*)coef_k,
                       (uint16_t*)coef_v, row, P.hkv, P.dh, P.nb, P.rank, P.R, P.rank_v, P.Rv, P.bases_shared, P.cap,
                       P.lens);
  else
    hipLaunchKernelGGL(k_project_rows<float>, grid, dim3(256), 0, st, (const float*)bases_k, (const float*)bases_v,
                       (const float*)k_new, (const float*)v_new, (float*)coef_k, (float*)coef_v, row, P.hkv, P.dh,
                       P.nb, P.rank, P.R, P.rank_v, P.Rv, P.bases_shared, P.cap, P.lens);
  return hipGetLastError();
}

hipError_t launch_project_step(const Problem& P, double* qpart, uint32_t* hist, const void* q, const void* bases_k,
                               const void* bases_v, const void* k_new, const void* v_new, void* coef_k, void* coef_v,
                               int64_t row, hipStream_t st) {
  const int nch = project_chunks(P);
  dim3 grid((P.R / 32) * nch * P.B + (std::max(P.R, P.Rv) / 32) * P.B * 2);
  if (P.dtype == S4R_BF16)
    hipLaunchKernelGGL(k_project_step<uint16_t>, grid, dim3(256), 0, st, (const uint16_t*)q, (const uint16_t*)bases_k,
                       (const uint16_t*)bases_v, (const uint16_t*)k_new, (const uint16_t*)v_new, (uint16_t*)coef_k,
                       (uint16_t*)coef_v, qpart, hist, row, P.hq, P.hkv, P.dh, P.G, P.nb, P.rank, P.R,
                       P.rank_v, P.Rv, P.bases_shared, P.cap, P.B, nch, P.lens);
  else
    hipLaunchKernelGGL(k_project_step<float>, grid, dim3(256), 0, st, (const float*)q, (const float*)bases_k,
                       (const float*)bases_v, (const float*)k_new, (const float*)v_new, (float*)coef_k,
                       (float*)coef_v, qpart, hist, row, P.hq, P.hkv, P.dh, P.G, P.nb, P.rank, P.R, P.rank_v, P.Rv,
                       P.bases_shared, P.cap, P.B, nch, P.lens);
  return hipGetLastError();
}

}  // namespace s4r
