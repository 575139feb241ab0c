"""GPU parity of the windowed and the ragged decode step on seeded random
configurations (the draws of tests/test_gpu_random.py's generator, with
their own case numbers).

Windowed: s4r_window_state_init, then s4r_decode_step_windowed at W_q + 2
consecutive lengths (so the state's ring of slots wraps and, above five
rows, the running sum loses rows as they leave), each step against the
oracle's step with the window's older query rows given explicitly
(Section 3.2.2).  Ragged: every sequence at its own length in one launch
against the oracle's step on that sequence alone, rows past each length
NaN.  Bars as in the other parity tests.
"""

import numpy as np
import pytest
import torch

import paper_2608_00528_amd as s4r
import workloads as W
from oracle import decode
from gpu_util import (cfg_from_workload, check_selection, dev, draw_random_workload, oracle_cfg, rel_err_rows,
                      slice_state, to_gpu_state, unpad_latent)

pytestmark = pytest.mark.gpu

OUT_TOL = {"bf16": 2e-2, "fp32": 1e-4}
SCORE_TOL = 5e-6


@pytest.mark.parametrize("case", range(12))
def test_random_windowed_steps(case):
    wl, _, append = draw_random_workload(100 + case, q_windows=(2, 3, 4, 6, 8, 12), min_len=400, max_len=3000)
    B, wq, L0 = wl.batch, wl.q_window, wl.L
    nsteps = wq + 2
    cap = ((L0 + nsteps + 15) // 16) * 16
    print(f"[random windowed {case}] {wl.describe()} rank/group {wl.rank} nb {wl.basis_groups} W_q {wq} "
          f"kappa {wl.pool_kernel} {wl.pool_mode}/{wl.group_agg} steps {nsteps} append {append}", flush=True)
    st = W.latent_state(wl, seed=case, capacity=cap, L=(L0 if append else cap))
    c = cfg_from_workload(wl, capacity=cap)
    g = to_gpu_state(c, st)
    ws = s4r.alloc_workspace(c)
    dt = s4r.storage_dtype(c)
    oc = oracle_cfg(c, wl.pool_mode, wl.group_agg)
    rng = np.random.default_rng(300 + case)
    rows = [st["qwin_prev"][:, :, i] for i in range(wq - 1)]    # the window's query rows, oldest first
    coef_k, coef_v = st["coef_k"], st["coef_v"]
    state = s4r.alloc_window_state(c)
    s4r.window_state_init(c, L0 + 1, g["qwin_prev"], g["coef_k"], state, ws)
    for t in range(nsteps):
        L = L0 + 1 + t
        q = W.round_storage(st["q"] + 0.3 * np.abs(st["q"]).mean() * rng.standard_normal(st["q"].shape), wl.dtype)
        kn = W.round_storage(rng.standard_normal((B, wl.Dp)), wl.dtype) if append else None
        vn = W.round_storage(rng.standard_normal((B, wl.Dp)), wl.dtype) if append else None
        m = s4r.num_selected(c, L)
        idx = torch.empty((B, m), dtype=torch.int32, device="cuda")
        scores = torch.empty((B, L), dtype=torch.float32, device="cuda")
        out = s4r.decode_step_windowed(c, L, dev(q, dt), state, g["sink_k"], g["sink_v"], g["bases_k"],
                                       g["bases_v"], g["coef_k"], g["coef_v"], ws,
                                       k_new=None if kn is None else dev(kn, dt),
                                       v_new=None if vn is None else dev(vn, dt), idx_out=idx, scores_out=scores)
        torch.cuda.synchronize()
        qwin = np.stack([W.round_storage(r, "fp32") for r in rows[t:t + wq - 1]], axis=2)   # [B, G, wq - 1, R]
        ref = decode.decode_step(oc, L, q, st["sink_k"], st["sink_v"], st["bases_k"], st["bases_v"], coef_k,
                                 coef_v, qwin_prev=qwin, k_new=kn, v_new=vn)
        if append:
            # continue from the rows the GPU appended (equal to the oracle's up
            # to one storage ulp at a rounding tie)
            rk = unpad_latent(s4r.unpack_coef(c, cap, g["coef_k"]).double().cpu().numpy(), wl.rank,
                              wl.basis_groups)
            rv = unpad_latent(s4r.unpack_coef(c, cap, g["coef_v"]).double().cpu().numpy(), wl.rank,
                              wl.basis_groups)
            assert (rk[:, L - 1] == ref["coef_k"][:, L - 1]).mean() > 0.99
            assert (rv[:, L - 1] == ref["coef_v"][:, L - 1]).mean() > 0.99
            coef_k, coef_v = rk, rv
        rows.append(decode.project(decode.group_queries(q, wl.n_kv_heads), st["bases_k"]))
        idx_np = idx.cpu().numpy().astype(np.int64)
        flips = check_selection(idx_np, ref["idx"], ref["a_tilde"], L, wl.window, wl.topk)
        sc = scores.cpu().numpy().astype(np.float64)
        assert np.array_equal(idx_np, decode.select(sc, L, wl.window, wl.topk))
        serr = np.abs(sc - ref["a_tilde"][:, :L]).max() / np.abs(ref["a_tilde"][:, :L]).max()
        o_ref, _, _ = decode.sparse_attention(q, idx_np, st["sink_k"], st["sink_v"], st["bases_k"], st["bases_v"],
                                              coef_k[:, :L], coef_v[:, :L], L, wl.n_kv_heads, oc["rope_theta"])
        err = rel_err_rows(out.cpu().numpy(), o_ref)
        print(f"[random windowed {case}] step {t} L {L}: scores {serr:.2e}, out {err:.2e}, tie flips {flips}",
              flush=True)
        assert serr <= 1e-5
        assert err <= OUT_TOL[wl.dtype]


@pytest.mark.parametrize("case", range(12))
def test_random_ragged_step(case):
    wl, _, append = draw_random_workload(200 + case, min_len=600, max_len=5000)
    rng = np.random.default_rng(400 + case)
    B = int(rng.integers(2, 5))
    wl = wl.scaled(batch=B)
    Lmax = wl.L
    lo = min(Lmax, max(wl.topk + wl.window + 1, 64))   # every sequence selects k + W tokens
    lengths = [int(x) for x in rng.integers(lo, Lmax + 1, size=B)]
    lengths[int(rng.integers(0, B))] = Lmax
    print(f"[random ragged {case}] {wl.describe()} rank/group {wl.rank} nb {wl.basis_groups} W_q {wl.q_window} "
          f"kappa {wl.pool_kernel} {wl.pool_mode}/{wl.group_agg} lengths {lengths} append {append}", flush=True)
    st = W.latent_state(wl, seed=case)
    c = cfg_from_workload(wl)
    st_gpu = dict(st)
    for key in ("coef_k", "coef_v"):
        x = st[key].copy()
        for b, L_b in enumerate(lengths):
            x[b, L_b - (1 if append else 0):] = np.nan
        st_gpu[key] = x
    g = to_gpu_state(c, st_gpu)
    dt = s4r.storage_dtype(c)
    kw = {}
    if append:
        kn = W.round_storage(rng.standard_normal((B, wl.Dp)), wl.dtype)
        vn = W.round_storage(rng.standard_normal((B, wl.Dp)), wl.dtype)
        kw = dict(k_new=dev(kn, dt), v_new=dev(vn, dt))
    ws = s4r.alloc_workspace(c)
    m = s4r.num_selected(c, Lmax)
    idx = torch.empty((B, m), dtype=torch.int32, device="cuda")
    scores = torch.full((B, Lmax), -7.0, dtype=torch.float32, device="cuda")
    out = s4r.decode_step_ragged(c, lengths, g["q"], g["sink_k"], g["sink_v"], g["bases_k"], g["bases_v"],
                                 g["coef_k"], g["coef_v"], ws, qwin_prev=g.get("qwin_prev"), idx_out=idx,
                                 scores_out=scores, **kw)
    torch.cuda.synchronize()
    o = out.cpu().numpy()
    assert np.isfinite(o).all()
    idx_np = idx.cpu().numpy().astype(np.int64)
    sc = scores.cpu().numpy()
    rows_k = unpad_latent(s4r.unpack_coef(c, Lmax, g["coef_k"]).double().cpu().numpy(), wl.rank, wl.basis_groups)
    rows_v = unpad_latent(s4r.unpack_coef(c, Lmax, g["coef_v"]).double().cpu().numpy(), wl.rank, wl.basis_groups)
    oc = oracle_cfg(c, wl.pool_mode, wl.group_agg)
    for b, L_b in enumerate(lengths):
        one = slice_state(st, b, L_b)
        if append:
            ck, cv = decode.project_append(kn[b:b + 1], vn[b:b + 1], one["bases_k"], one["bases_v"], oc["dtype"])
            assert (rows_k[b, L_b - 1] == ck[0]).mean() > 0.99
            assert (rows_v[b, L_b - 1] == cv[0]).mean() > 0.99
            assert np.isnan(rows_k[b, L_b:]).all()
            one["coef_k"], one["coef_v"] = rows_k[b:b + 1, :L_b], rows_v[b:b + 1, :L_b]
        ref = decode.decode_step(oc, L_b, one["q"], one["sink_k"], one["sink_v"], one["bases_k"], one["bases_v"],
                                 one["coef_k"], one["coef_v"], qwin_prev=one["qwin_prev"])
        a_ref = ref["a_tilde"][0]
        err = np.abs(sc[b, :L_b] - a_ref) / np.maximum(np.abs(a_ref), 1e-30)
        assert err.max() <= SCORE_TOL, f"sequence {b} (L = {L_b}): score rel err {err.max():.3e}"
        assert (sc[b, L_b:] == -7.0).all()
        check_selection(idx_np[b:b + 1], ref["idx"], ref["a_tilde"], L_b, wl.window, wl.topk)
        assert np.array_equal(idx_np[b:b + 1], decode.select(sc[b:b + 1, :L_b].astype(np.float64), L_b,
                                                             wl.window, wl.topk))
        o_ref, _, _ = decode.sparse_attention(one["q"], idx_np[b:b + 1], one["sink_k"], one["sink_v"],
                                              one["bases_k"], one["bases_v"], one["coef_k"], one["coef_v"], L_b,
                                              wl.n_kv_heads, oc["rope_theta"])
        err = rel_err_rows(o[b:b + 1], o_ref)
        assert err <= OUT_TOL[wl.dtype], f"sequence {b} (L = {L_b}): output rel err {err:.3e}"
    print(f"[random ragged {case}] ok", flush=True)
