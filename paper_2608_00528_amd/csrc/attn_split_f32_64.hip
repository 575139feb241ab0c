// Fused reconstruction + split attention, f32 storage, head dim 64.
#include "attn_split.h"

namespace s4r {

bool launch_split_f32_64(const Problem& P, const Workspace& ws, int64_t L, int m, int n_proc, int nsplit,
                        const void* q, const void* bk, const void* bv, const void* ck, const void* cv,
                        hipStream_t st) {
  return launch_split_dt<float, 64>(P, ws, L, m, n_proc, nsplit, q, bk, bv, ck, cv, st);
}

}  // namespace s4r
