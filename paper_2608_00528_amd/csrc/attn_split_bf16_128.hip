// Fused reconstruction + split attention, bf16 storage, head dim 128.
#include "attn_split.h"

namespace s4r {

bool launch_split_bf16_128(const Problem& P, const Workspace& ws, int64_t L, int m, int n_proc, int nsplit,
                        const void* q, const void* bk, const void* bv, const void* ck, const void* cv,
                        hipStream_t st) {
  return launch_split_dt<uint16_t, 128>(P, ws, L, m, n_proc, nsplit, q, bk, bv, ck, cv, st);
}

}  // namespace s4r
