"""s4r_decode_step_noalloc (the step on the library's own per-device scratch)
against s4r_decode_step with a caller workspace: two calls in a row, the
second on a smaller problem, each bit-identical to the workspace path (same
kernels, same fixed-order arithmetic), through the C ABI."""

import numpy as np
import pytest
import torch

import paper_2608_00528_amd as s4r
import workloads as W
from oracle import decode
from tests.gpu_util import cfg_from_workload, check_selection, oracle_cfg, rel_err_rows, to_gpu_state

pytestmark = pytest.mark.gpu


def _both(wl, seed, append):
    st = W.latent_state(wl, seed=seed)
    c = cfg_from_workload(wl)
    g = to_gpu_state(c, st)
    m = s4r.num_selected(c, wl.L)
    kw = {}
    if append:
        rng = np.random.default_rng(seed + 7)
        kn = W.round_storage(rng.standard_normal((wl.batch, wl.n_kv_heads * wl.head_dim)), wl.dtype)
        vn = W.round_storage(rng.standard_normal((wl.batch, wl.n_kv_heads * wl.head_dim)), wl.dtype)
        dt = s4r.storage_dtype(c)
        kw = dict(k_new=torch.from_numpy(kn).to("cuda", dt), v_new=torch.from_numpy(vn).to("cuda", dt))
    res = []
    for noalloc in (True, False):
        ck, cv = g["coef_k"].clone(), g["coef_v"].clone()      # the append writes row L - 1
        idx = torch.empty((wl.batch, m), dtype=torch.int32, device="cuda")
        sc = torch.empty((wl.batch, wl.L), dtype=torch.float32, device="cuda")
        print(f"[no-alloc] {wl.describe()} append={append} noalloc={noalloc}", flush=True)
        if noalloc:
            out = s4r.decode_step_noalloc(c, wl.L, g["q"], g["sink_k"], g["sink_v"], g["bases_k"], g["bases_v"],
                                          ck, cv, idx_out=idx, scores_out=sc, **kw)
        else:
            ws = s4r.alloc_workspace(c)
            out = s4r.decode_step(c, wl.L, g["q"], g["sink_k"], g["sink_v"], g["bases_k"], g["bases_v"], ck, cv,
                                  ws, idx_out=idx, scores_out=sc, **kw)
        torch.cuda.synchronize()
        res.append((out.cpu(), idx.cpu(), sc.cpu(), ck.cpu(), cv.cpu()))
    for a, b in zip(res[0], res[1]):
        assert torch.equal(a, b)
    return c, st, res[0]


def test_noalloc_matches_workspace_step_twice():
    # first call: two sequences of 16k tokens
    wl1 = W.CONFIGS["llama8b_32k"].scaled(N=16384 + 4, batch=2, topk=512)
    c1, st1, (out1, idx1, _, _, _) = _both(wl1, seed=11, append=False)
    # the first call's result is also the oracle's selection and output
    ref = decode.decode_step(oracle_cfg(c1), wl1.L, st1["q"], st1["sink_k"], st1["sink_v"], st1["bases_k"],
                             st1["bases_v"], st1["coef_k"], st1["coef_v"])
    idx_np = idx1.numpy().astype(np.int64)
    check_selection(idx_np, ref["idx"], ref["a_tilde"], wl1.L, wl1.window, wl1.topk)
    o_ref, _, _ = decode.sparse_attention(st1["q"], idx_np, st1["sink_k"], st1["sink_v"], st1["bases_k"],
                                          st1["bases_v"], st1["coef_k"], st1["coef_v"], wl1.L, wl1.n_kv_heads,
                                          oracle_cfg(c1)["rope_theta"])
    assert rel_err_rows(out1.numpy(), o_ref) <= 2e-2
    # second call: a smaller problem (one sequence, 3k tokens, a new token
    # appended) on the scratch the first call left behind
    wl2 = W.CONFIGS["llama8b_32k"].scaled(N=3000 + 4, batch=1, topk=256)
    _both(wl2, seed=12, append=True)


def test_noalloc_refuses_configurations_beyond_its_scratch():
    wl = W.CONFIGS["llama8b_32L_sustained"]
    c = cfg_from_workload(wl)
    assert s4r.workspace_size(c) > 64 << 20
    q = torch.zeros((wl.batch, wl.n_q_heads, wl.head_dim), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(s4r.S4RError, match="WORKSPACE"):
        s4r.decode_step_noalloc(c, wl.L, q, q, q, q, q, q, q)
