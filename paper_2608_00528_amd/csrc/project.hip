// Section 3.2.1 (compressed cache update) on gfx950: the query coefficients
// c_t^Q = s_t^Q B^K of every query group and the projection of a new token's
// key and value into coefficient row L-1 (c_t^K = s_t^K B^K, c_t^V = s_t^V B^V).
#include "s4r_device.h"
#include "s4r_internal.h"

namespace s4r {

// ---------------------------------------------------------------------------
// Both projections are short dot products (a basis group of up to 2048 rows)
// for few vectors, so they are latency-bound: the work is spread over many
// small workgroups, each thread's operands are requested together, and the
// reduction is short.  A workgroup owns 8 latent columns of one basis group;
// thread t holds basis rows t + 256 i (i < NCH, the group's 256-row chunks
// rounded up to a power of two) of its 8 columns in registers, in storage
// format, and the projected vectors' elements of the same rows, read straight
// from memory (no staging).  Products are accumulated in fp64 (exact: a
// bf16 or fp32 basis element times an fp32 vector element) per thread in row
// order, then summed over the wave's 64 lanes (two gfx950 lane swaps that
// halve the values per lane, then DPP within 16-lane rows) and over the 4
// waves through LDS, in a fixed order, so the results are deterministic.
// ---------------------------------------------------------------------------
constexpr int kPCols = 8;                     // latent columns per query workgroup (4 or 8)
constexpr int kQVec = 4;                      // query vectors per pass
// the step kernel's query workgroups: 16 columns, two vectors per pass, so
// its query and new-row workgroups (R / 16 + 2 R / 32 per sequence) fit one
// round of the chip at three waves per SIMD for a 32-sequence batch
constexpr int kSPCols = 16, kSQVec = 2;

// 8 consecutive basis elements, kept in their storage format until used
struct Raw8bf16 {
  uint4 u;
  __device__ __forceinline__ void load(const uint16_t* p) { u = *reinterpret_cast<const uint4*>(p); }
  // an empty asm that "changes" the value: its conversions cannot be hoisted above this point
  __device__ __forceinline__ void opaque() { asm volatile("" : "+v"(u.x), "+v"(u.y), "+v"(u.z), "+v"(u.w)); }
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
  __device__ __forceinline__ void opaque() {
    asm volatile("" : "+v"(a.x), "+v"(a.y), "+v"(a.z), "+v"(a.w), "+v"(b.x), "+v"(b.y), "+v"(b.z), "+v"(b.w));
  }
  __device__ __forceinline__ float operator[](int c) const {
    const float4& h = (c < 4) ? a : b;
    const int k = c & 3;
    return k == 0 ? h.x : k == 1 ? h.y : k == 2 ? h.z : h.w;
  }
};
// 4 consecutive basis elements
struct Raw4bf16 {
  uint2 u;
  __device__ __forceinline__ void load(const uint16_t* p) { u = *reinterpret_cast<const uint2*>(p); }
  __device__ __forceinline__ float operator[](int c) const {
    const uint32_t w = (c >> 1) == 0 ? u.x : u.y;
    return (c & 1) ? __uint_as_float(w & 0xFFFF0000u) : __uint_as_float(w << 16);
  }
};
struct Raw4f32 {
  float4 a;
  __device__ __forceinline__ void load(const float* p) { a = *reinterpret_cast<const float4*>(p); }
  __device__ __forceinline__ float operator[](int c) const {
    return c == 0 ? a.x : c == 1 ? a.y : c == 2 ? a.z : a.w;
  }
};
// 16 consecutive basis elements (the step projection's 16-column workgroups)
struct Raw16bf16 {
  Raw8bf16 a, b;
  __device__ __forceinline__ void load(const uint16_t* p) {
    a.load(p);
    b.load(p + 8);
  }
  __device__ __forceinline__ void opaque() {
    a.opaque();
    b.opaque();
  }
  __device__ __forceinline__ float operator[](int c) const { return c < 8 ? a[c] : b[c - 8]; }
};
struct Raw16f32 {
  Raw8f32 a, b;
  __device__ __forceinline__ void load(const float* p) {
    a.load(p);
    b.load(p + 8);
  }
  __device__ __forceinline__ void opaque() {
    a.opaque();
    b.opaque();
  }
  __device__ __forceinline__ float operator[](int c) const { return c < 8 ? a[c] : b[c - 8]; }
};
template <typename T, int N>
struct RawN;
template <>
struct RawN<uint16_t, 8> {
  using type = Raw8bf16;
};
template <>
struct RawN<float, 8> {
  using type = Raw8f32;
};
template <>
struct RawN<uint16_t, 16> {
  using type = Raw16bf16;
};
template <>
struct RawN<float, 16> {
  using type = Raw16f32;
};
template <>
struct RawN<uint16_t, 4> {
  using type = Raw4bf16;
};
template <>
struct RawN<float, 4> {
  using type = Raw4f32;
};

// fp64 move within 16-lane rows (DPP)
template <int CTRL>
__device__ __forceinline__ double dpp_move_d(double x) {
  const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(x), CTRL, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(x), CTRL, 0xF, 0xF, false);
  return __hiloint2double(hi, lo);
}

// x + y after the gfx950 lane swaps: permlane32_swap exchanges lanes 32..63 of
// its first operand with lanes 0..31 of its second, permlane16_swap the odd
// 16-lane rows of the first with the even rows of the second (each dword of
// the fp64 values the same way).  Afterwards the lower half (even rows) holds
// the first operand summed over the lane pair, the upper half (odd rows) the
// second.
__device__ __forceinline__ double swap32_add(double x, double y) {
  const auto lo = __builtin_amdgcn_permlane32_swap((unsigned)__double2loint(x), (unsigned)__double2loint(y), false,
                                                   false);
  const auto hi = __builtin_amdgcn_permlane32_swap((unsigned)__double2hiint(x), (unsigned)__double2hiint(y), false,
                                                   false);
  return __hiloint2double((int)hi[0], (int)lo[0]) + __hiloint2double((int)hi[1], (int)lo[1]);
}
__device__ __forceinline__ double swap16_add(double x, double y) {
  const auto lo = __builtin_amdgcn_permlane16_swap((unsigned)__double2loint(x), (unsigned)__double2loint(y), false,
                                                   false);
  const auto hi = __builtin_amdgcn_permlane16_swap((unsigned)__double2hiint(x), (unsigned)__double2hiint(y), false,
                                                   false);
  return __hiloint2double((int)hi[0], (int)lo[0]) + __hiloint2double((int)hi[1], (int)lo[1]);
}

// sums of a[0..N) over the 64 lanes of a wave, written to red[wave][0..N):
// the lane swaps leave row r (lanes 16 r .. 16 r + 15) with values
// r N / 4 .. + N / 4 - 1 summed over the four rows, DPP sums them within the
// row (row_ror 8 and 4, then the quad swaps), and lane 16 r writes them
template <int N>
__device__ __forceinline__ void reduce_wave(double (&a)[N], double (*red)[32], int wave, int lane) {
#pragma unroll
  for (int j = 0; j < N / 2; ++j) a[j] = swap32_add(a[j], a[j + N / 2]);
#pragma unroll
  for (int j = 0; j < N / 4; ++j) a[j] = swap16_add(a[j], a[j + N / 4]);
#pragma unroll
  for (int j = 0; j < N / 4; ++j) {
    a[j] += dpp_move_d<0x128>(a[j]);   // row_ror:8
    a[j] += dpp_move_d<0x124>(a[j]);   // row_ror:4
    a[j] += dpp_move_d<0x4E>(a[j]);    // quad_perm [2,3,0,1]
    a[j] += dpp_move_d<0xB1>(a[j]);    // quad_perm [1,0,3,2]
  }
  if ((lane & 15) == 0) {
#pragma unroll
    for (int j = 0; j < N / 4; ++j) red[wave][(lane >> 4) * (N / 4) + j] = a[j];
  }
}

// image address of query column gi, latent column col (part 0; part q is R further)
__device__ __forceinline__ uint16_t* qimg_at(uint16_t* qimg, int b, int ncb, int nmb, int R, int gi, int col) {
  const int cb = gi / kColBlk, gl = gi % kColBlk;
  return qimg + ((((int64_t)b * ncb + cb) * nmb + (gl >> 2)) * 16 + 4 * (gl & 3)) * R + col;
}

// four consecutive latent columns' parts, packed per part (4 bf16 in 8 bytes)
__device__ __forceinline__ void qimg_pack4(float4 x, uint2 (&pk)[3]) {
  const Split3 s0 = split3((double)x.x), s1 = split3((double)x.y), s2 = split3((double)x.z),
               s3 = split3((double)x.w);
  pk[0] = make_uint2(s0.hi | ((uint32_t)s1.hi << 16), s2.hi | ((uint32_t)s3.hi << 16));
  pk[1] = make_uint2(s0.mid | ((uint32_t)s1.mid << 16), s2.mid | ((uint32_t)s3.mid << 16));
  pk[2] = make_uint2(s0.lo | ((uint32_t)s1.lo << 16), s2.lo | ((uint32_t)s3.lo << 16));
}

// ---------------------------------------------------------------------------
// query coefficients: grid (R / PC, B).  A workgroup forms, for its PC latent
// columns (8 in k_project_query, 16 in the step kernel) and every query
// group g, c^Q[g] = q_g B^K over all rows of the basis group (QV groups per
// pass), and writes it (1) rounded to fp32 into
// qcoef [B][G][R] (and the caller's qcoef_out), (2) as the hi / mid / lo bf16
// parts the scoring kernel's MFMA A operand holds, into the operand image
// qimg [B][column blocks][NMB][16][R] (query column gi = g W_q + i in block
// gi / 16, MFMA (gi % 16) / 4, rows 4 (gi % 4) + part), together with the
// window's older rows from qwin_prev when given.  The image's other rows are
// never read.
// ---------------------------------------------------------------------------
template <typename T, int NCH, int PC = kPCols, int QV = kQVec>
__device__ __forceinline__ void project_query_body(const T* __restrict__ q, const T* __restrict__ bases_k,
                                                   const float* __restrict__ qwin_prev, uint16_t* __restrict__ qimg,
                                                   float* __restrict__ qcoef, float* __restrict__ qcoef_out,
                                                   uint32_t* __restrict__ hist, int hq, int hkv, int dh, int G,
                                                   int Wq, int nb, int rank, int R, int bases_shared, int ncb,
                                                   int nmb, int cblk, int b) {
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int Dp = hkv * dh, Dg = Dp / nb;
  const int ldh = __builtin_ctz(dh);              // head_dim is a power of two
  const int c0 = cblk * PC;                       // first latent column of the block
  const int grp = c0 / rank;                      // its basis group
  // the window's older query rows (oldest first): unit u = t + 256 k is
  // latent columns c0 + 4 (u % U) .. + 3 of older row j = u / U (U = PC / 4
  // units per row), i.e. group j / (W_q - 1), window row j % (W_q - 1)
  // (G (W_q - 1) <= 127 rows: NOU units per thread).  Requested first, written last.
  constexpr int U = PC / 4, NOU = (127 * U + 255) / 256;
  const bool old_rows = qimg && qwin_prev && Wq > 1;
  const int n_old = old_rows ? G * (Wq - 1) : 0;
  float4 oldv[NOU];
#pragma unroll
  for (int k = 0; k < NOU; ++k) {
    const int u = t + 256 * k, jo = u / U;
    oldv[k] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (jo < n_old) {
      const int go = jo / (Wq - 1), wo = jo - go * (Wq - 1);
      oldv[k] = *reinterpret_cast<const float4*>(qwin_prev + (((int64_t)b * G + go) * (Wq - 1) + wo) * R + c0 +
                                                 4 * (u % U));
    }
  }

  // basis rows t + 256 i of the block's columns (rows past the group's end:
  // a re-read of its last row, met by x = 0)
  const T* bases = bases_k + (bases_shared ? 0 : (int64_t)b * Dp * rank) + (int64_t)grp * Dg * rank + (c0 - grp * rank);
  typename RawN<T, PC>::type bw[NCH];
#pragma unroll
  for (int i = 0; i < NCH; ++i) bw[i].load(bases + (int64_t)min(t + 256 * i, Dg - 1) * rank);
  // the group's query elements of those rows, for vectors v0 .. v0 + 3 (the
  // last vector repeated past G)
  float x[QV][NCH];
  auto load_x = [&](int v0) {
#pragma unroll
    for (int v = 0; v < QV; ++v)
#pragma unroll
      for (int i = 0; i < NCH; ++i) {
        const int d = grp * Dg + min(t + 256 * i, Dg - 1);   // feature index in Dp
        x[v][i] = load_elem(q, ((int64_t)b * hq + (int64_t)(d >> ldh) * G + min(v0 + v, G - 1)) * dh + (d & (dh - 1)));
      }
  };
  load_x(0);
  // the step's selection histograms start from zero (the relevance and
  // classify kernels add to them later in the step): the sequence's R / PC
  // workgroups clear a slice each
  {
    const int nblk = R / PC, per = (kHistStride / 4 + nblk - 1) / nblk;
    uint4* hz = reinterpret_cast<uint4*>(hist + (int64_t)b * kHistStride);
    const int i1 = min((cblk + 1) * per, kHistStride / 4);
    for (int i = cblk * per + t; i < i1; i += blockDim.x) hz[i] = make_uint4(0u, 0u, 0u, 0u);
  }

  __shared__ double red[4][32];
  for (int v0 = 0; v0 < G; v0 += QV) {
    if (v0 > 0) load_x(v0);
    double acc[QV * PC];                          // [vector][column]
#pragma unroll
    for (int j = 0; j < QV * PC; ++j) acc[j] = 0.0;
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
      const bool in = t + 256 * i < Dg;
      typename RawN<T, PC>::type bi = bw[i];       // converted here, in every pass
      bi.opaque();
#pragma unroll
      for (int c = 0; c < PC; ++c) {
        const double bc = (double)bi[c];
#pragma unroll
        for (int v = 0; v < QV; ++v) acc[v * PC + c] = fma(in ? (double)x[v][i] : 0.0, bc, acc[v * PC + c]);
      }
    }
    reduce_wave<QV * PC>(acc, red, wave, lane);
    __syncthreads();
    if (t < QV * PC && v0 + t / PC < G) {
      const int g = v0 + t / PC, col = c0 + t % PC;
      const double xq = ((red[0][t] + red[1][t]) + red[2][t]) + red[3][t];
      qcoef[((int64_t)b * G + g) * R + col] = (float)xq;
      if (qcoef_out) qcoef_out[((int64_t)b * G + g) * R + col] = (float)xq;
      if (qimg) {
        const Split3 sp = split3(xq);
        uint16_t* pi = qimg_at(qimg, b, ncb, nmb, R, g * Wq + Wq - 1, col);
        pi[0] = sp.hi;
        pi[R] = sp.mid;
        pi[2 * R] = sp.lo;
      }
    }
    __syncthreads();                              // red is reused by the next pass
  }
#pragma unroll
  for (int k = 0; k < NOU; ++k) {
    const int u = t + 256 * k, jo = u / U;
    if (jo < n_old) {
      const int go = jo / (Wq - 1), wo = jo - go * (Wq - 1);
      uint2 pk[3];
      qimg_pack4(oldv[k], pk);
      uint16_t* p = qimg_at(qimg, b, ncb, nmb, R, go * Wq + wo, c0 + 4 * (u % U));
#pragma unroll
      for (int part = 0; part < 3; ++part) *reinterpret_cast<uint2*>(p + part * R) = pk[part];
    }
  }
}

template <typename T, int NCH>
__global__ __launch_bounds__(256) void k_project_query(const T* __restrict__ q, const T* __restrict__ bases_k,
                                                       const float* __restrict__ qwin_prev, uint16_t* __restrict__ qimg,
                                                       float* __restrict__ qcoef, float* __restrict__ qcoef_out,
                                                       uint32_t* __restrict__ hist, int hq, int hkv, int dh, int G,
                                                       int Wq, int nb, int rank, int R, int bases_shared, int ncb,
                                                       int nmb) {
  project_query_body<T, NCH>(q, bases_k, qwin_prev, qimg, qcoef, qcoef_out, hist, hq, hkv, dh, G, Wq, nb, rank, R,
                             bases_shared, ncb, nmb, blockIdx.x, blockIdx.y);
}

// ---------------------------------------------------------------------------
// new token's coefficient rows: grid (max(R, R_V) / 32, B, 2 = {key, value}).
// One vector per side, so a workgroup takes 32 columns (4 groups of 8 per
// thread, the same 32 sums per lane as a query pass) and writes their full
// sums into row append_row of the cache (rounded to the storage format).
// ---------------------------------------------------------------------------
constexpr int kRCols = 32;                    // latent columns per new-row workgroup

template <typename T, int NCH>
__device__ __forceinline__ void project_rows_body(const T* __restrict__ bases_k, const T* __restrict__ bases_v,
                                                  const T* __restrict__ k_new, const T* __restrict__ v_new,
                                                  T* __restrict__ coef_k, T* __restrict__ coef_v, int64_t append_row,
                                                  int hkv, int dh, int nb, int rank, int R, int bases_shared,
                                                  int64_t cap, int cblk, int b, int which) {
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int Dp = hkv * dh, Dg = Dp / nb;
  const int c0 = cblk * kRCols;
  const int grp = c0 / rank;
  const T* x_new = which == 0 ? k_new : v_new;
  T* coef = which == 0 ? coef_k : coef_v;
  const T* bases = (which == 0 ? bases_k : bases_v) + (bases_shared ? 0 : (int64_t)b * Dp * rank) +
                   (int64_t)grp * Dg * rank + (c0 - grp * rank);
  constexpr int NG = kRCols / 8;                  // column groups of 8
  typename RawN<T, 8>::type bw[NCH][NG];
  float x[NCH];
#pragma unroll
  for (int i = 0; i < NCH; ++i) {
    const int r = min(t + 256 * i, Dg - 1);
#pragma unroll
    for (int k = 0; k < NG; ++k) bw[i][k].load(bases + (int64_t)r * rank + k * 8);
    x[i] = load_elem(x_new, (int64_t)b * Dp + grp * Dg + r);
  }
  __shared__ double red[4][32];
  double acc[kRCols];                             // [column group][column]
#pragma unroll
  for (int j = 0; j < kRCols; ++j) acc[j] = 0.0;
#pragma unroll
  for (int i = 0; i < NCH; ++i) {
    const double xv = t + 256 * i < Dg ? (double)x[i] : 0.0;
#pragma unroll
    for (int k = 0; k < NG; ++k) {
      bw[i][k].opaque();
#pragma unroll
      for (int c = 0; c < 8; ++c) acc[k * 8 + c] = fma(xv, (double)bw[i][k][c], acc[k * 8 + c]);
    }
  }
  reduce_wave<kRCols>(acc, red, wave, lane);
  __syncthreads();
  if (t < kRCols) {
    const double v = ((red[0][t] + red[1][t]) + red[2][t]) + red[3][t];
    store_elem(coef, (int64_t)b * cap * R + tiled_offset(append_row, c0 + t, R), v);
  }
}

template <typename T, int NCH>
__global__ __launch_bounds__(256) void k_project_rows(const T* __restrict__ bases_k, const T* __restrict__ bases_v,
                                                      const T* __restrict__ k_new, const T* __restrict__ v_new,
                                                      T* __restrict__ coef_k, T* __restrict__ coef_v,
                                                      int64_t append_row, int hkv, int dh, int nb, int rank, int R,
                                                      int rank_v, int Rv, int bases_shared, int64_t cap, Lens lens) {
  // the value side has its own width when the ranks are asymmetric
  const int which = blockIdx.z;
  if ((int)blockIdx.x * kRCols >= (which ? Rv : R)) return;
  // a ragged batch appends at each sequence's own last row
  const int64_t row = lens.n ? (int64_t)lens.v[blockIdx.y] - 1 : append_row;
  project_rows_body<T, NCH>(bases_k, bases_v, k_new, v_new, coef_k, coef_v, row, hkv, dh, nb, which ? rank_v : rank,
                            which ? Rv : R, bases_shared, cap, blockIdx.x, blockIdx.y, which);
}

// both projections of a step that appends a token, in one launch: per
// sequence R / 16 query-coefficient workgroups and max(R, R_V) / 32 new-row
// workgroups per side.  They touch disjoint memory, and one launch saves a
// dispatch and a first-read latency.  Every workgroup of sequence b runs on
// XCD b mod 8 (workgroup i is dispatched to XCD i mod 8): the query and key
// workgroups read different columns of the same basis rows (32 and 64 bytes
// of each bf16 row), so a row's cache lines come from HBM once into that
// XCD's L2 instead of once per XCD.
template <typename T, int NCH>
__global__ __launch_bounds__(256) void k_project_step(const T* __restrict__ q, const T* __restrict__ bases_k,
                                                      const T* __restrict__ bases_v, const T* __restrict__ k_new,
                                                      const T* __restrict__ v_new, T* __restrict__ coef_k,
                                                      T* __restrict__ coef_v, const float* __restrict__ qwin_prev,
                                                      uint16_t* __restrict__ qimg, float* __restrict__ qcoef,
                                                      uint32_t* __restrict__ hist, int64_t append_row, int hq,
                                                      int hkv, int dh, int G, int Wq, int nb, int rank, int R,
                                                      int rank_v, int Rv, int bases_shared, int64_t cap, int B,
                                                      int ncb, int nmb, Lens lens) {
  const int ncq = R / kSPCols;
  const int ncr = max(R, Rv) / kRCols;             // row blocks per (sequence, side)
  const int per_seq = ncq + 2 * ncr;
  const int xcd = blockIdx.x & 7, k = blockIdx.x >> 3;
  const int b = xcd + 8 * (k / per_seq), id = k % per_seq;
  if (b >= B) return;
  if (id < ncq) {
    project_query_body<T, NCH, kSPCols, kSQVec>(q, bases_k, qwin_prev, qimg, qcoef, nullptr, hist, hq, hkv, dh, G,
                                                Wq, nb, rank, R, bases_shared, ncb, nmb, id, b);
  } else {
    const int cblk = (id - ncq) % ncr, which = (id - ncq) / ncr;
    if (cblk * kRCols >= (which ? Rv : R)) return;
    const int64_t row = lens.n ? (int64_t)lens.v[b] - 1 : append_row;
    project_rows_body<T, NCH>(bases_k, bases_v, k_new, v_new, coef_k, coef_v, row, hkv, dh, nb,
                              which ? rank_v : rank, which ? Rv : R, bases_shared, cap, cblk, b, which);
  }
}

// 256-row chunks of a basis group, rounded up to a power of two (<= 8)
static int chunk_pow2(const Problem& P) {
  const int nch = (P.Dg + kPChunk - 1) / kPChunk;
  return nch <= 1 ? 1 : nch <= 2 ? 2 : nch <= 4 ? 4 : 8;
}

template <typename T, int NCH>
static void launch_query_t(const Problem& P, const Workspace& ws, const void* q, const void* bases_k,
                           const float* qwin_prev, float* qcoef_out, uint16_t* img, hipStream_t st) {
  hipLaunchKernelGGL((k_project_query<T, NCH>), dim3(P.R / kPCols, P.B), dim3(256), 0, st, (const T*)q,
                     (const T*)bases_k, qwin_prev, img, ws.qcoef, qcoef_out, ws.hist, P.hq, P.hkv, P.dh, P.G, P.Wq,
                     P.nb, P.rank, P.R, P.bases_shared, col_blocks(P), qimg_mfmas(P));
}

template <typename T>
static void launch_query_c(const Problem& P, const Workspace& ws, const void* q, const void* bases_k,
                           const float* qwin_prev, float* qcoef_out, uint16_t* img, hipStream_t st) {
  switch (chunk_pow2(P)) {
    case 1: launch_query_t<T, 1>(P, ws, q, bases_k, qwin_prev, qcoef_out, img, st); break;
    case 2: launch_query_t<T, 2>(P, ws, q, bases_k, qwin_prev, qcoef_out, img, st); break;
    case 4: launch_query_t<T, 4>(P, ws, q, bases_k, qwin_prev, qcoef_out, img, st); break;
    default: launch_query_t<T, 8>(P, ws, q, bases_k, qwin_prev, qcoef_out, img, st); break;
  }
}

hipError_t launch_project_query(const Problem& P, const Workspace& ws, const void* q, const void* bases_k,
                                const float* qwin_prev, float* qcoef_out, bool image, hipStream_t st) {
  uint16_t* img = image ? ws.qimg : nullptr;
  if (P.dtype == S4R_BF16)
    launch_query_c<uint16_t>(P, ws, q, bases_k, qwin_prev, qcoef_out, img, st);
  else
    launch_query_c<float>(P, ws, q, bases_k, qwin_prev, qcoef_out, img, st);
  return hipGetLastError();
}

// the scoring kernel's operand image of a query window given entirely as
// coefficient rows (the window state's set-up): rows [B][G][n_rows][R] fp32,
// one thread per four latent columns of a row
__global__ __launch_bounds__(256) void k_query_image_rows(const float* __restrict__ rows, uint16_t* __restrict__ qimg,
                                                          int B, int G, int n_rows, int R, int ncb, int nmb) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int nu = R / 4;
  if (i >= (int64_t)B * G * n_rows * nu) return;
  const int u = (int)(i % nu), j = (int)((i / nu) % n_rows), g = (int)((i / ((int64_t)nu * n_rows)) % G);
  const int b = (int)(i / ((int64_t)nu * n_rows * G));
  const float4 x = *reinterpret_cast<const float4*>(rows + (((int64_t)b * G + g) * n_rows + j) * R + 4 * u);
  uint2 pk[3];
  qimg_pack4(x, pk);
  uint16_t* p = qimg_at(qimg, b, ncb, nmb, R, g * n_rows + j, 4 * u);
#pragma unroll
  for (int part = 0; part < 3; ++part) *reinterpret_cast<uint2*>(p + part * R) = pk[part];
}

hipError_t launch_query_image_rows(const Problem& P0, const Workspace& ws, const float* rows, hipStream_t st) {
  const int64_t n = (int64_t)P0.B * P0.G * P0.Wq * (P0.R / 4);
  hipLaunchKernelGGL(k_query_image_rows, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, rows, ws.qimg, P0.B,
                     P0.G, P0.Wq, P0.R, col_blocks(P0), qimg_mfmas(P0));
  return hipGetLastError();
}

// row `row` of C^Q for n_rows queries: out[b][g][row][r] = qcoef[b][g][r]
__global__ __launch_bounds__(256) void k_qcoef_row(const float* __restrict__ qcoef, float* __restrict__ out, int B,
                                                   int G, int R, int64_t n_rows, int64_t row) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= B * G * R) return;
  const int b = i / (G * R), g = (i / R) % G, r = i % R;
  out[(((int64_t)b * G + g) * n_rows + row) * R + r] = qcoef[i];
}

// C^Q rows of n_rows queries [B, n_rows, h_q, d_h]: each row staged as
// [B, h_q, d_h] in the workspace, projected (the same fp64 sums as a decode
// step's query, rounded once to fp32) and copied to its row
hipError_t launch_project_queries(const Problem& P, const Workspace& ws, int64_t n_rows, const void* q_rows,
                                  const void* bases_k, float* out, hipStream_t st) {
  const size_t es = P.dtype == S4R_BF16 ? 2 : 4;
  const size_t row_bytes = (size_t)P.hq * P.dh * es;
  void* staged = ws.part_o;                       // >= B * h_q * d_h * 4 bytes
  const int n = P.B * P.G * P.R;
  for (int64_t row = 0; row < n_rows; ++row) {
    hipError_t e = hipMemcpy2DAsync(staged, row_bytes, static_cast<const char*>(q_rows) + row * row_bytes,
                                    (size_t)n_rows * row_bytes, row_bytes, P.B, hipMemcpyDeviceToDevice, st);
    if (e == hipSuccess) e = launch_project_query(P, ws, staged, bases_k, nullptr, nullptr, false, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_qcoef_row, dim3((n + 255) / 256), dim3(256), 0, st, ws.qcoef, out, P.B, P.G, P.R, n_rows,
                       row);
  }
  return hipGetLastError();
}

template <typename T, int NCH>
static void launch_rows_t(const Problem& P, const void* bases_k, const void* bases_v, const void* k_new,
                          const void* v_new, void* coef_k, void* coef_v, int64_t row, hipStream_t st) {
  hipLaunchKernelGGL((k_project_rows<T, NCH>), dim3(std::max(P.R, P.Rv) / kRCols, P.B, 2), dim3(256), 0, st,
                     (const T*)bases_k, (const T*)bases_v, (const T*)k_new, (const T*)v_new, (T*)coef_k, (T*)coef_v,
                     row, P.hkv, P.dh, P.nb, P.rank, P.R, P.rank_v, P.Rv, P.bases_shared, P.cap, P.lens);
}

template <typename T>
static void launch_rows_c(const Problem& P, const void* bases_k, const void* bases_v, const void* k_new,
                          const void* v_new, void* coef_k, void* coef_v, int64_t row, hipStream_t st) {
  switch (chunk_pow2(P)) {
    case 1: launch_rows_t<T, 1>(P, bases_k, bases_v, k_new, v_new, coef_k, coef_v, row, st); break;
    case 2: launch_rows_t<T, 2>(P, bases_k, bases_v, k_new, v_new, coef_k, coef_v, row, st); break;
    case 4: launch_rows_t<T, 4>(P, bases_k, bases_v, k_new, v_new, coef_k, coef_v, row, st); break;
    default: launch_rows_t<T, 8>(P, bases_k, bases_v, k_new, v_new, coef_k, coef_v, row, st); break;
  }
}

hipError_t launch_project_rows(const Problem& P, const void* bases_k, const void* bases_v, const void* k_new,
                               const void* v_new, void* coef_k, void* coef_v, int64_t row, hipStream_t st) {
  if (P.dtype == S4R_BF16)
    launch_rows_c<uint16_t>(P, bases_k, bases_v, k_new, v_new, coef_k, coef_v, row, st);
  else
    launch_rows_c<float>(P, bases_k, bases_v, k_new, v_new, coef_k, coef_v, row, st);
  return hipGetLastError();
}

template <typename T, int NCH>
static void launch_step_t(const Problem& P, const Workspace& ws, const void* q, const void* bases_k,
                          const void* bases_v, const void* k_new, const void* v_new, void* coef_k, void* coef_v,
                          const float* qwin_prev, int64_t row, hipStream_t st) {
  const int per_seq = P.R / kSPCols + 2 * (std::max(P.R, P.Rv) / kRCols);
  const dim3 grid(8 * ((P.B + 7) / 8) * per_seq);  // sequence b on XCD b mod 8
  hipLaunchKernelGGL((k_project_step<T, NCH>), grid, dim3(256), 0, st, (const T*)q, (const T*)bases_k,
                     (const T*)bases_v, (const T*)k_new, (const T*)v_new, (T*)coef_k, (T*)coef_v, qwin_prev, ws.qimg,
                     ws.qcoef, ws.hist, row, P.hq, P.hkv, P.dh, P.G, P.Wq, P.nb, P.rank, P.R, P.rank_v, P.Rv,
                     P.bases_shared, P.cap, P.B, col_blocks(P), qimg_mfmas(P), P.lens);
}

template <typename T>
static void launch_step_c(const Problem& P, const Workspace& ws, const void* q, const void* bases_k,
                          const void* bases_v, const void* k_new, const void* v_new, void* coef_k, void* coef_v,
                          const float* qwin_prev, int64_t row, hipStream_t st) {
  switch (chunk_pow2(P)) {
    case 1: launch_step_t<T, 1>(P, ws, q, bases_k, bases_v, k_new, v_new, coef_k, coef_v, qwin_prev, row, st); break;
    case 2: launch_step_t<T, 2>(P, ws, q, bases_k, bases_v, k_new, v_new, coef_k, coef_v, qwin_prev, row, st); break;
    case 4: launch_step_t<T, 4>(P, ws, q, bases_k, bases_v, k_new, v_new, coef_k, coef_v, qwin_prev, row, st); break;
    default: launch_step_t<T, 8>(P, ws, q, bases_k, bases_v, k_new, v_new, coef_k, coef_v, qwin_prev, row, st); break;
  }
}

hipError_t launch_project_step(const Problem& P, const Workspace& ws, const void* q, const void* bases_k,
                               const void* bases_v, const void* k_new, const void* v_new, void* coef_k, void* coef_v,
                               const float* qwin_prev, int64_t row, hipStream_t st) {
  if (P.dtype == S4R_BF16)
    launch_step_c<uint16_t>(P, ws, q, bases_k, bases_v, k_new, v_new, coef_k, coef_v, qwin_prev, row, st);
  else
    launch_step_c<float>(P, ws, q, bases_k, bases_v, k_new, v_new, coef_k, coef_v, qwin_prev, row, st);
  return hipGetLastError();
}

}  // namespace s4r
