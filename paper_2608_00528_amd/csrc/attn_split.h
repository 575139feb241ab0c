// Launch + dispatch of the fused split attention kernel for one (dtype, head
// dim); included by the attn_split_*.hip translation units.
#pragma once

#include "attn_common.h"

namespace s4r {

template <typename T, int RBH, int DH, int G>
static void launch_split_t(const Problem& P, const Workspace& ws, int64_t L, int m, int n_proc, int nsplit,
                           const void* q, const void* bases_k, const void* bases_v, const void* coef_k,
                           const void* coef_v, hipStream_t st) {
  const int ntile = (n_proc + 15) / 16;
  const size_t lds = (size_t)((ntile + nsplit - 1) / nsplit) * 16 * sizeof(int32_t);
  hipLaunchKernelGGL((k_attn_split<T, RBH, DH, G>), dim3(nsplit, P.hkv, P.B), dim3(DH * 2), lds, st, (const T*)q,
                     (const T*)bases_k, (const T*)bases_v, (const T*)coef_k, (const T*)coef_v, ws.idx,
                     (int64_t)m, ws.part_ml, ws.part_o, n_proc, nsplit, P.hq, P.hkv, P.nb, P.rank, P.R,
                     P.s, L, P.cap, P.bases_shared, P.theta, P.lens);
}

#define S4R_SPLIT_ARGS P, ws, L, m, n_proc, nsplit, q, bk, bv, ck, cv, st

template <typename T, int DH, int G>
static bool dispatch_split_rb(const Problem& P, const Workspace& ws, int64_t L, int m, int n_proc, int nsplit,
                              const void* q, const void* bk, const void* bv, const void* ck, const void* cv,
                              hipStream_t st) {
  switch (P.rank / 32) {
    case 1: launch_split_t<T, 1, DH, G>(S4R_SPLIT_ARGS); return true;
    case 2: launch_split_t<T, 2, DH, G>(S4R_SPLIT_ARGS); return true;
    case 3: launch_split_t<T, 3, DH, G>(S4R_SPLIT_ARGS); return true;
    case 4: launch_split_t<T, 4, DH, G>(S4R_SPLIT_ARGS); return true;
    case 5: launch_split_t<T, 5, DH, G>(S4R_SPLIT_ARGS); return true;
    case 6: launch_split_t<T, 6, DH, G>(S4R_SPLIT_ARGS); return true;
    case 8: launch_split_t<T, 8, DH, G>(S4R_SPLIT_ARGS); return true;
    default: return false;
  }
}

template <typename T, int DH>
static bool dispatch_split_g(const Problem& P, const Workspace& ws, int64_t L, int m, int n_proc, int nsplit,
                             const void* q, const void* bk, const void* bv, const void* ck, const void* cv,
                             hipStream_t st) {
  switch (P.G) {
    case 1: return dispatch_split_rb<T, DH, 1>(S4R_SPLIT_ARGS);
    case 2: return dispatch_split_rb<T, DH, 2>(S4R_SPLIT_ARGS);
    case 4: return dispatch_split_rb<T, DH, 4>(S4R_SPLIT_ARGS);
    case 7: return dispatch_split_rb<T, DH, 7>(S4R_SPLIT_ARGS);
    case 8: return dispatch_split_rb<T, DH, 8>(S4R_SPLIT_ARGS);
    default: return false;
  }
}

template <typename T, int DH>
static bool launch_split_dt(const Problem& P, const Workspace& ws, int64_t L, int m, int n_proc, int nsplit,
                            const void* q, const void* bk, const void* bv, const void* ck, const void* cv,
                            hipStream_t st) {
  return dispatch_split_g<T, DH>(S4R_SPLIT_ARGS);
}

}  // namespace s4r
