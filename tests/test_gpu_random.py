"""GPU parity of the fused decode step on seeded random configurations.

Each case draws one configuration the library accepts (head_dim, query
group size G, KV heads, basis groups, a rank that is often not a multiple of
32, storage format, batch, length and capacity, sinks, local window, k,
query window with its earlier rows, pooling kernel and mode, group
aggregation, and whether the step appends the new token's key and value,
Section 3.2.1) and compares the step with the oracle's step (Section 3.2) on
the workloads' latent recipe, to the bars of the other parity tests:
selection equal to the oracle's up to near-ties and exactly the top-k of the
step's own scores; outputs within 2e-2 (bf16 storage) or 1e-4 (fp32) of the
oracle attending over the step's own index set (and its own appended rows,
which equal the oracle's up to one storage ulp at a rounding tie).  The draws
are fixed by the case number, so a failure names a reproducible
configuration.
"""

import numpy as np
import pytest
import torch

import paper_2608_00528_amd as s4r
import workloads as W
from oracle import decode
from gpu_util import (cfg_from_workload, check_selection, dev, draw_random_workload, oracle_cfg, rel_err_rows,
                      to_gpu_state, unpad_latent)

pytestmark = pytest.mark.gpu

OUT_TOL = {"bf16": 2e-2, "fp32": 1e-4}
N_CASES = 40


@pytest.mark.parametrize("case", range(N_CASES))
def test_random_configuration(case):
    wl, cap, append = draw_random_workload(case)
    L = wl.L
    print(f"[random {case}] {wl.describe()} rank/group {wl.rank} nb {wl.basis_groups} W_q {wl.q_window} "
          f"kappa {wl.pool_kernel} {wl.pool_mode}/{wl.group_agg} cap {cap} append {append}", flush=True)
    st = W.latent_state(wl, seed=case, capacity=cap, L=L)
    c = cfg_from_workload(wl, capacity=cap)
    g = to_gpu_state(c, st)
    ws = s4r.alloc_workspace(c)
    m = s4r.num_selected(c, L)
    idx = torch.empty((wl.batch, m), dtype=torch.int32, device="cuda")
    scores = torch.empty((wl.batch, L), dtype=torch.float32, device="cuda")
    kw, kw_ref = {}, {}
    if append:
        rng = np.random.default_rng(2000 + case)
        tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
        kn = W.round_storage(rng.standard_normal((wl.batch, wl.Dp)), wl.dtype)
        vn = W.round_storage(rng.standard_normal((wl.batch, wl.Dp)), wl.dtype)
        kw = dict(k_new=dev(kn, tdt), v_new=dev(vn, tdt))
        kw_ref = dict(k_new=kn, v_new=vn)
    out = s4r.decode_step(c, L, g["q"], g["sink_k"], g["sink_v"], g["bases_k"], g["bases_v"], g["coef_k"],
                          g["coef_v"], ws, qwin_prev=g.get("qwin_prev"), idx_out=idx, scores_out=scores, **kw)
    torch.cuda.synchronize()
    stc = dict(st)
    stc["coef_k"], stc["coef_v"] = st["coef_k"][:, :L], st["coef_v"][:, :L]
    ref = decode.decode_step(oracle_cfg(c, wl.pool_mode, wl.group_agg), L, st["q"], st["sink_k"], st["sink_v"],
                             st["bases_k"], st["bases_v"], stc["coef_k"], stc["coef_v"],
                             qwin_prev=st.get("qwin_prev"), **kw_ref)
    if append:
        # the step's own appended rows (row L - 1), every earlier row unchanged
        rows_k = unpad_latent(s4r.unpack_coef(c, L, g["coef_k"]).double().cpu().numpy(), wl.rank, wl.basis_groups)
        rows_v = unpad_latent(s4r.unpack_coef(c, L, g["coef_v"]).double().cpu().numpy(), wl.rank, wl.basis_groups)
        for got, want in ((rows_k, ref["coef_k"]), (rows_v, ref["coef_v"])):
            assert np.array_equal(got[:, :L - 1], want[:, :L - 1])
            ulp = 2.0 ** -7 if wl.dtype == "bf16" else 2.0 ** -23
            assert np.abs(got[:, L - 1] - want[:, L - 1]).max() <= ulp * np.abs(want[:, L - 1]).max()
            assert (got[:, L - 1] == want[:, L - 1]).mean() > 0.99
        stc["coef_k"], stc["coef_v"] = rows_k, rows_v
    idx_np = idx.cpu().numpy().astype(np.int64)
    flips = check_selection(idx_np, ref["idx"], ref["a_tilde"], L, wl.window, wl.topk)
    assert np.array_equal(idx_np, decode.select(scores.cpu().numpy().astype(np.float64), L, wl.window, wl.topk))
    o_ref, _, _ = decode.sparse_attention(st["q"], idx_np, st["sink_k"], st["sink_v"], st["bases_k"],
                                          st["bases_v"], stc["coef_k"], stc["coef_v"], L, wl.n_kv_heads,
                                          oracle_cfg(c)["rope_theta"])
    o = out.cpu().numpy()
    assert np.isfinite(o).all()
    err = rel_err_rows(o, o_ref)
    print(f"[random {case}] out err {err:.2e}, tie flips {flips}", flush=True)
    assert err <= OUT_TOL[wl.dtype], f"output rel err {err:.3e}"
