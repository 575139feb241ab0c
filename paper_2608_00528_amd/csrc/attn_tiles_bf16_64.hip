// MFMA split attention (bf16 storage), head dim 64.
#include "attn_mfma.h"

namespace s4r {

bool launch_tiles_bf16_64(const Problem& P, const Workspace& ws, int64_t L, int m, int n_proc, const void* q,
                          const void* bk, const void* bv, const void* ck, const void* cv, hipStream_t st,
                          int* nsplit, bool ident) {
  return launch_tiles_dh<2>(P, ws, L, m, n_proc, q, bk, bv, ck, cv, st, nsplit, ident);
}

}  // namespace s4r
