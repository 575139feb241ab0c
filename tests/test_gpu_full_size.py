"""Parity at the full workload sizes, in the launch configuration bench.py
times: the fused s4r_decode_step over tiled caches of capacity ceil16(L), one
workspace, inputs resident on the GPU.

The oracle computes every sequence of the batch in full (float64, about half a
second per 128k-token sequence), so every score, every index and every output
row is compared, with the bars of the other parity tests.  The measured launch
(no idx_out / scores_out) must give bit-identical outputs to the checked one.
"""

import numpy as np
import pytest
import torch

import paper_2608_00528_amd as s4r
import workloads as W
from oracle import decode
from gpu_util import cfg_from_workload, check_selection, oracle_cfg, rel_err_rows, score_tol, to_gpu_state

pytestmark = pytest.mark.gpu

OUT_TOL = {"bf16": 2e-2, "fp32": 1e-4}


@pytest.mark.parametrize("name", ["llama8b_32k", "llama8b_128k", "qwen7b_128k"])
def test_full_size_decode_step(name):
    wl = W.CONFIGS[name]
    print(f"[full-size] {wl.describe()}", flush=True)
    st = W.latent_state(wl, seed=1)
    c = cfg_from_workload(wl)
    g = to_gpu_state(c, st)
    ws = s4r.alloc_workspace(c)
    m = s4r.num_selected(c, wl.L)
    idx = torch.empty((wl.batch, m), dtype=torch.int32, device="cuda")
    scores = torch.empty((wl.batch, wl.L), dtype=torch.float32, device="cuda")
    out = s4r.decode_step(c, wl.L, g["q"], g["sink_k"], g["sink_v"], g["bases_k"], g["bases_v"], g["coef_k"],
                          g["coef_v"], ws, idx_out=idx, scores_out=scores)
    out_bench = s4r.decode_step(c, wl.L, g["q"], g["sink_k"], g["sink_v"], g["bases_k"], g["bases_v"],
                                g["coef_k"], g["coef_v"], ws)
    torch.cuda.synchronize()
    assert torch.equal(out, out_bench), "the timed launch differs from the checked one"

    oc = oracle_cfg(c, wl.pool_mode, wl.group_agg)
    ref = decode.decode_step(oc, wl.L, st["q"], st["sink_k"], st["sink_v"], st["bases_k"], st["bases_v"],
                             st["coef_k"], st["coef_v"])
    a = ref["a_tilde"]
    got = scores.cpu().numpy().astype(np.float64)
    err_s = np.abs(got - a) / np.maximum(np.abs(a), 1e-30)
    tol_s = score_tol(ref["cQ"], st["coef_k"], wl.L, wl.dtype)     # per sequence

    idx_np = idx.cpu().numpy().astype(np.int64)
    flips = check_selection(idx_np, ref["idx"], a, wl.L, wl.window, wl.topk)
    assert np.array_equal(idx_np, decode.select(got, wl.L, wl.window, wl.topk))

    o_ref, _, _ = decode.sparse_attention(st["q"], idx_np, st["sink_k"], st["sink_v"], st["bases_k"],
                                          st["bases_v"], st["coef_k"], st["coef_v"], wl.L, wl.n_kv_heads,
                                          oc["rope_theta"])
    err = rel_err_rows(out.cpu().numpy(), o_ref)
    print(f"[full-size] {name}: score err {err_s.max():.2e} (bound {tol_s.min():.2e}..{tol_s.max():.2e}), "
          f"tie flips {flips}, out err {err:.2e}", flush=True)
    assert err <= OUT_TOL[wl.dtype], f"output rel err {err:.3e} (tie flips {flips})"
    for b in range(wl.batch):
        assert err_s[b].max() <= tol_s[b], f"sequence {b}: score rel err {err_s[b].max():.3e} > {tol_s[b]:.3e}"
