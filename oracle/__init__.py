"""Plain CPU oracle of the S^4R decode step (arxiv 2608.00528).

TEST INFRASTRUCTURE ONLY.  This package is a slow, obviously correct, float64
numpy statement of what the paper's decode stage computes, written step by step
in the order of Section 3.2 so that a reader can check it against the paper by
eye.  It exists to prove the GPU path right, never to stand in for it: only the
test suite, the smoke check and the benchmark's CPU-baseline leg may import or
run it.  It shares no code with the HIP library and does not import the input
generators; the GPU path never imports it.

Modules
-------
decode   Section 3.2: compressed cache update, latent relevance, pooling,
         group aggregation, index selection, sparse reconstruction, sinks,
         RoPE and the final attention.
prefill  Section 3.1: sink split, token sampling, token-wise normalisation,
         truncated SVD, coefficient projection, initial query window.  Used to
         turn raw synthetic KV into the stored state the decode step reads.
cost     Section 3.3 memory model and Appendix B decode-time cost model.
storage  Rounding of float64 values to the storage formats (bf16, fp32).

Readings of points the paper leaves open are listed in the module docstrings
where they are applied.  Every function here is pinned by a CPU test against
something other than itself: identities, library routines, brute force, loop
forms written from the equations (group aggregation, the query FIFO and its
causal limits), hand-computed sample positions of the hybrid sampler, and the
worked example of Appendix B.4.  Mutation tests plant plausible mistakes
(a dropped scale, wrong query grouping, pooling off by one, ties to the higher
index, a RoPE sign, a transposed basis, a dropped window row, mean and max
aggregation exchanged, a newest-first query FIFO, a sampler that takes the
first early positions) and check that a pin fails for each.
"""

from . import cost, decode, prefill, storage  # noqa: F401
from .decode import (  # noqa: F401
    aggregate,
    attend,
    causal_mask,
    decode_step,
    group_queries,
    latent_logits,
    num_selected,
    pool,
    project,
    project_append,
    reconstruct,
    rope,
    select,
    softmax_over_length,
    window_mean,
)
