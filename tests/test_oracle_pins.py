"""Pins of the CPU oracle against things other than itself.

Each check below compares the oracle with an independent statement of the
same quantity: a linear-algebra identity, a torch library routine, a brute
force over tiny inputs, or a closed form.  The checks are plain functions so
the mutation tests at the bottom can show that a planted mistake in the
oracle (a dropped term, a wrong sign or index, a transposed operand) makes at
least one of them fail.
"""

import itertools

import numpy as np
import pytest
import torch

import oracle
from oracle import decode, prefill, storage

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


# ----------------------------------------------------------------------------
# small random problems
# ----------------------------------------------------------------------------

def _orth(rng, n, k):
    q, r = np.linalg.qr(rng.standard_normal((n, k)))
    return q * np.sign(np.diag(r))


def small_problem(seed=0, B=2, hkv=2, G=2, dh=8, nb=1, rank=6, L=40, s=3, orthonormal=False):
    rng = np.random.default_rng(seed)
    Dp = hkv * dh
    dg = Dp // nb
    if orthonormal:
        bk = np.stack([np.stack([_orth(rng, dg, rank) for _ in range(nb)]) for _ in range(B)])
        bv = np.stack([np.stack([_orth(rng, dg, rank) for _ in range(nb)]) for _ in range(B)])
    else:
        bk = rng.standard_normal((B, nb, dg, rank))
        bv = rng.standard_normal((B, nb, dg, rank))
    R = nb * rank
    return {
        "q": rng.standard_normal((B, hkv * G, dh)),
        "bases_k": bk, "bases_v": bv,
        "coef_k": rng.standard_normal((B, L, R)),
        "coef_v": rng.standard_normal((B, L, R)),
        "sink_k": rng.standard_normal((B, s, Dp)),
        "sink_v": rng.standard_normal((B, s, Dp)),
        "hkv": hkv, "G": G, "dh": dh, "L": L, "s": s, "R": R, "nb": nb,
    }


def cfg_of(p, W=4, k=5, kappa=3, theta=100.0, pool_mode="max", agg="mean"):
    return dict(n_kv_heads=p["hkv"], window=W, topk=k, pool_kernel=kappa,
                pool_mode=pool_mode, group_agg=agg, rope_theta=theta, dtype="fp32")


def run(p, cfg, **kw):
    return decode.decode_step(cfg, p["L"], p["q"], p["sink_k"], p["sink_v"], p["bases_k"],
                              p["bases_v"], p["coef_k"], p["coef_v"], **kw)


# ----------------------------------------------------------------------------
# independent reference pieces (written from the definitions, loop form)
# ----------------------------------------------------------------------------

def ref_group_query(q, hkv, g):
    """q_g = concat over kv heads j of query head j*G + g (loop form)."""
    B, hq, dh = q.shape
    G = hq // hkv
    return np.stack([np.concatenate([q[b, j * G + g] for j in range(hkv)]) for b in range(B)])


def ref_full_keys(coef, bases):
    """Every reconstructed key, row by row: sum_r c[r] * basis column r."""
    B, L, R = coef.shape
    nb, dg, rank = bases.shape[1:]
    out = np.zeros((B, L, nb * dg))
    for b in range(B):
        for k in range(nb):
            blk = bases[b if bases.shape[0] > 1 else 0, k]            # [dg, rank]
            for rr in range(rank):
                out[b, :, k * dg:(k + 1) * dg] += np.outer(coef[b, :, k * rank + rr], blk[:, rr])
    return out


def ref_rope_complex(x, pos, theta):
    """RoPE as complex multiplication: (x_i + i x_{i+d/2}) * exp(i pos w_i)."""
    if theta == 0:          # RoPE switched off
        return np.array(x, dtype=np.float64)
    d = x.shape[-1]
    half = d // 2
    w = theta ** (-(2.0 * np.arange(half)) / d)
    z = x[..., :half] + 1j * x[..., half:]
    z = z * np.exp(1j * np.asarray(pos, dtype=np.float64)[..., None] * w)
    return np.concatenate([z.real, z.imag], axis=-1)


def torch_gqa_attention(q, K, V, pos_k, pos_q, theta, hkv):
    """Dense GQA attention through torch SDPA (float64) with complex-form RoPE;
    kv heads are repeated with repeat_interleave (head h reads kv head h // G)."""
    B, hq, dh = q.shape
    n = K.shape[1]
    qr = ref_rope_complex(q, np.broadcast_to(np.asarray(pos_q, float)[:, None], (B, hq)), theta)
    Kh = K.reshape(B, n, hkv, dh).transpose(0, 2, 1, 3)                # [B, hkv, n, dh]
    Kr = ref_rope_complex(Kh, np.broadcast_to(np.asarray(pos_k, float)[:, None, :], (B, hkv, n)), theta)
    Vh = V.reshape(B, n, hkv, dh).transpose(0, 2, 1, 3)
    G = hq // hkv
    tq = torch.from_numpy(qr)[:, :, None, :]                          # [B, hq, 1, dh]
    tk = torch.from_numpy(np.ascontiguousarray(Kr)).repeat_interleave(G, dim=1)
    tv = torch.from_numpy(np.ascontiguousarray(Vh)).repeat_interleave(G, dim=1)
    o = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv)
    return o[:, :, 0, :].numpy()


# ----------------------------------------------------------------------------
# pin checks
# ----------------------------------------------------------------------------

def check_latent_identity(seed=0, nb=1):
    """(q_g B)(c)^T / sqrt(R) == q_g . (B c) / sqrt(R) for every token (any B)."""
    p = small_problem(seed, nb=nb, hkv=2 * nb if nb > 1 else 2)
    Z = decode.latent_logits(decode.query_window(p["q"], None, p["bases_k"], p["hkv"]),
                             p["coef_k"], p["L"])
    K = ref_full_keys(p["coef_k"], p["bases_k"])
    for g in range(p["G"]):
        qg = ref_group_query(p["q"], p["hkv"], g)
        ref = np.einsum("bd,bld->bl", qg, K) / np.sqrt(p["R"])
        if not np.allclose(Z[:, g, 0, :], ref, rtol=1e-11, atol=1e-11):
            return False
    return True


def check_rotation_invariance(seed=1):
    """B -> B Q and C -> C Q (Q orthogonal per basis group) change nothing."""
    p = small_problem(seed, nb=2, hkv=2, rank=5, L=50)
    cfg = cfg_of(p, W=4, k=7)
    a = run(p, cfg)
    rng = np.random.default_rng(seed + 100)
    p2 = dict(p)
    bk, bv, ck, cv = (p[x].copy() for x in ("bases_k", "bases_v", "coef_k", "coef_v"))
    rank = bk.shape[-1]
    for b in range(bk.shape[0]):
        for k in range(2):
            Qk = _orth(rng, rank, rank)
            Qv = _orth(rng, rank, rank)
            bk[b, k] = bk[b, k] @ Qk
            bv[b, k] = bv[b, k] @ Qv
            ck[b, :, k * rank:(k + 1) * rank] = ck[b, :, k * rank:(k + 1) * rank] @ Qk
            cv[b, :, k * rank:(k + 1) * rank] = cv[b, :, k * rank:(k + 1) * rank] @ Qv
    p2.update(bases_k=bk, bases_v=bv, coef_k=ck, coef_v=cv)
    b_ = run(p2, cfg)
    return (np.allclose(a["Z"], b_["Z"], rtol=1e-10, atol=1e-12)
            and np.allclose(a["a_tilde"], b_["a_tilde"], rtol=1e-10, atol=1e-15)
            and np.array_equal(a["idx"], b_["idx"])
            and np.allclose(a["out"], b_["out"], rtol=1e-10, atol=1e-12))


def check_pool_vs_torch(seed=2):
    rng = np.random.default_rng(seed)
    x = rng.random((2, 3, 37))
    ok = True
    for kappa in (1, 3, 5, 7, 9):
        t = torch.from_numpy(x)
        mx = torch.nn.functional.max_pool1d(t, kappa, stride=1, padding=kappa // 2).numpy()
        av = torch.nn.functional.avg_pool1d(t, kappa, stride=1, padding=kappa // 2,
                                            count_include_pad=True).numpy()
        ok &= np.allclose(decode.pool(x, kappa, "max"), mx, rtol=0, atol=0)
        ok &= np.allclose(decode.pool(x, kappa, "avg"), av, rtol=1e-14, atol=1e-15)
    return bool(ok)


def check_topk_special_case(seed=3):
    """W_q = 1, kappa = 1, G = 1: softmax is monotone, so the global picks are
    the top-k of q . K^ (reconstructed keys), ties to the lower index."""
    p = small_problem(seed, G=1, hkv=2, L=60)
    W, k = 5, 9
    cfg = cfg_of(p, W=W, k=k, kappa=1)
    r = run(p, cfg)
    K = ref_full_keys(p["coef_k"], p["bases_k"])
    qg = ref_group_query(p["q"], p["hkv"], 0)
    for b in range(p["q"].shape[0]):
        scores = K[b, :p["L"] - W] @ qg[b]
        order = sorted(range(p["L"] - W), key=lambda l: (-scores[l], l))[:k]
        if list(r["idx"][b, :k]) != sorted(order):
            return False
    return True


def brute_select(a, L, W, k):
    n_hist = max(L - W, 0)
    k_eff = min(k, n_hist)
    out = []
    for row in a:
        pairs = sorted(((-row[l], l) for l in range(n_hist)))
        glob = sorted(l for _, l in pairs[:k_eff])
        out.append(glob + list(range(n_hist, L)))
    return np.array(out, dtype=np.int64).reshape(len(a), -1)


def check_select_bruteforce(seed=4):
    rng = np.random.default_rng(seed)
    for L, W, k in [(20, 4, 5), (20, 4, 0), (20, 4, 16), (20, 4, 40), (3, 5, 2), (1, 1, 3),
                    (17, 0, 6), (30, 30, 4), (31, 7, 24)]:
        a = rng.integers(0, 4, size=(3, L)).astype(np.float64)  # many exact ties
        if not np.array_equal(decode.select(a, L, W, k), brute_select(a, L, W, k)):
            return False
        if decode.select(a, L, W, k).shape[1] != decode.num_selected(L, W, k):
            return False
    return True


def check_full_rank_exact(seed=5):
    """R = Dp with a square orthonormal basis: reconstruct(project(S)) == S."""
    rng = np.random.default_rng(seed)
    Dp = 12
    S = rng.standard_normal((2, 9, Dp))
    Bm = np.stack([_orth(rng, Dp, Dp)[None] for _ in range(2)])      # [B, 1, Dp, Dp]
    C = decode.project(S, Bm)
    return np.allclose(decode.reconstruct(C, Bm), S, rtol=0, atol=1e-12)


def check_full_budget_dense(seed=6, theta=100.0, W=3):
    """k >= L - W: the step equals dense GQA attention over [sinks; C B^T]."""
    p = small_problem(seed, hkv=2, G=3, dh=8, L=25, s=2)
    cfg = cfg_of(p, W=W, k=10 ** 6, kappa=5, theta=theta)
    r = run(p, cfg)
    B, L, s = p["q"].shape[0], p["L"], p["s"]
    K = np.concatenate([p["sink_k"], ref_full_keys(p["coef_k"], p["bases_k"])], axis=1)
    V = np.concatenate([p["sink_v"], ref_full_keys(p["coef_v"], p["bases_v"])], axis=1)
    pos_k = np.broadcast_to(np.arange(s + L), (B, s + L))
    ref = torch_gqa_attention(p["q"], K, V, pos_k, np.full(B, s + L - 1), theta, p["hkv"])
    return np.allclose(r["out"], ref, rtol=1e-10, atol=1e-12)


def check_rope_complex(seed=7):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((3, 5, 16))
    pos = rng.integers(0, 10 ** 5, size=(3, 5))
    return np.allclose(decode.rope(x, pos, 500000.0), ref_rope_complex(x, pos, 500000.0),
                       rtol=1e-10, atol=1e-10)


def check_rope_shift_invariance(seed=8):
    """Shifting every position by the same amount leaves the output unchanged."""
    rng = np.random.default_rng(seed)
    B, hq, hkv, dh, n = 2, 4, 2, 8, 11
    q = rng.standard_normal((B, hq, dh))
    K = rng.standard_normal((B, n, hkv * dh))
    V = rng.standard_normal((B, n, hkv * dh))
    pos_k = np.sort(rng.choice(1000, size=(B, n), replace=False), axis=1)
    pos_q = np.full(B, 1000)
    o1 = decode.attend(q, K, V, pos_k, pos_q, 1000.0, hkv)
    o2 = decode.attend(q, K, V, pos_k + 777, pos_q + 777, 1000.0, hkv)
    return np.allclose(o1, o2, rtol=1e-9, atol=1e-10)


def check_plain_gqa(seed=9, theta=10000.0):
    """s = 0, L = W and a full-rank basis: ordinary GQA decode attention over S."""
    rng = np.random.default_rng(seed)
    B, hkv, G, dh, L = 2, 2, 2, 8, 6
    Dp = hkv * dh
    S_k = rng.standard_normal((B, L, Dp))
    S_v = rng.standard_normal((B, L, Dp))
    Bk = np.stack([_orth(rng, Dp, Dp)[None] for _ in range(B)])
    Bv = np.stack([_orth(rng, Dp, Dp)[None] for _ in range(B)])
    q = rng.standard_normal((B, hkv * G, dh))
    cfg = dict(n_kv_heads=hkv, window=L, topk=3, pool_kernel=3, rope_theta=theta, dtype="fp32")
    r = decode.decode_step(cfg, L, q, np.zeros((B, 0, Dp)), np.zeros((B, 0, Dp)), Bk, Bv,
                           decode.project(S_k, Bk), decode.project(S_v, Bv))
    ref = torch_gqa_attention(q, S_k, S_v, np.broadcast_to(np.arange(L), (B, L)),
                              np.full(B, L - 1), theta, hkv)
    return np.allclose(r["out"], ref, rtol=1e-10, atol=1e-11)


def check_causal_window(seed=10):
    """W_q > 1: row i only sees keys up to its own position, rows are averaged."""
    p = small_problem(seed, L=30)
    Wq = 4
    rng = np.random.default_rng(seed)
    qprev = rng.standard_normal((p["q"].shape[0], p["G"], Wq - 1, p["R"]))
    rel = decode.relevance(p["q"], qprev, p["bases_k"], p["coef_k"], p["L"], p["hkv"], 1)
    cQ = rel["cQ"]
    L = p["L"]
    for b in range(cQ.shape[0]):
        for g in range(cQ.shape[1]):
            acc = np.zeros(L)
            for i in range(Wq):
                pos = L - Wq + i
                z = np.array([cQ[b, g, i] @ p["coef_k"][b, l] / np.sqrt(p["R"]) for l in range(pos + 1)])
                e = np.exp(z - z.max())
                acc[:pos + 1] += e / e.sum()
            if not np.allclose(rel["AQ"][b, g], acc / Wq, rtol=1e-12, atol=1e-15):
                return False
    return True


def check_dense_comparator(seed=11):
    """The dense comparator (keys stored after RoPE) equals torch SDPA with
    complex-form RoPE applied to pre-RoPE keys at positions 0..N-1."""
    rng = np.random.default_rng(seed)
    B, hq, hkv, dh, N = 2, 8, 2, 16, 37
    q = rng.standard_normal((B, hq, dh))
    K = rng.standard_normal((B, N, hkv * dh))
    V = rng.standard_normal((B, N, hkv * dh))
    theta = 10000.0
    pos = np.broadcast_to(np.arange(N, dtype=float), (B, N))
    Kst = np.concatenate([ref_rope_complex(K[:, :, j * dh:(j + 1) * dh], pos, theta) for j in range(hkv)], axis=-1)
    got = decode.dense_decode(q, Kst, V, hkv, theta)
    want = torch_gqa_attention(q, K, V, pos, np.full(B, N - 1.0), theta, hkv)
    return np.allclose(got, want, rtol=1e-12, atol=1e-12)


def check_full_reconstruction(seed=12, nb=1, rank_v=5):
    """Full-reconstruction decoding (Appendix B.1) equals torch SDPA over the
    cache rebuilt with torch matrix products, C B^T per basis group, sinks
    first, complex-form RoPE at positions 0..s+L-1 (also with a value rank
    other than the key rank, Appendix D.2)."""
    rng = np.random.default_rng(seed)
    B, hq, hkv, dh, L, s, rank = 2, 8, 2, 16, 23, 3, 5
    Dp = hkv * dh
    Dg = Dp // nb
    q = rng.standard_normal((B, hq, dh))
    bases_k = rng.standard_normal((B, nb, Dg, rank))
    bases_v = rng.standard_normal((B, nb, Dg, rank_v))
    ck = rng.standard_normal((B, L + 4, nb * rank))           # rows past L are never used
    cv = rng.standard_normal((B, L + 4, nb * rank_v))
    sk = rng.standard_normal((B, s, Dp))
    sv = rng.standard_normal((B, s, Dp))
    theta = 10000.0

    def rebuild(c, bases):
        tc = torch.from_numpy(c[:, :L])
        tb = torch.from_numpy(bases)
        r = bases.shape[-1]
        parts = [tc[:, :, g * r:(g + 1) * r] @ tb[:, g].transpose(1, 2) for g in range(nb)]
        return torch.cat(parts, dim=2).numpy()
    K = np.concatenate([sk, rebuild(ck, bases_k)], axis=1)
    V = np.concatenate([sv, rebuild(cv, bases_v)], axis=1)
    pos = np.broadcast_to(np.arange(s + L, dtype=float), (B, s + L))
    want = torch_gqa_attention(q, K, V, pos, np.full(B, s + L - 1.0), theta, hkv)
    got = decode.full_reconstruction_decode(q, sk, sv, bases_k, bases_v, ck, cv, L, hkv, theta)
    return np.allclose(got, want, rtol=1e-12, atol=1e-12)


def ref_relevance_loop(q_rows, pos_rows, bases_k, coef_k, L, hkv, kappa, pool_mode, agg):
    """A~ written out in loops from the equations of Sections 3.2.1-3.2.3.

    q_rows: W_q raw query arrays [B, h_q, d_h], oldest first, the query of row
    i sitting at non-sink position pos_rows[i].  Per group g: the latent query
    of every row (s^Q B^K, group g's heads concatenated over the KV heads), its
    logits against every key l <= its position divided by sqrt(R), a softmax
    over those keys, the mean over the rows, pooling over [l - h, l + h]
    clipped to the sequence (max of the in-range values, or their sum / kappa),
    and the group aggregation: sum over g / G (mean) or the largest (max)."""
    B = coef_k.shape[0]
    G = q_rows[0].shape[1] // hkv
    nb, dg, rank = bases_k.shape[1:]
    R = nb * rank
    h = kappa // 2
    out = np.zeros((B, L))
    for b in range(B):
        bk = bases_k[b if bases_k.shape[0] > 1 else 0]
        pooled = np.zeros((G, L))
        for g in range(G):
            aq = np.zeros(L)
            for qr, pos in zip(q_rows, pos_rows):
                qg = ref_group_query(qr, hkv, g)[b]                  # [Dp]
                cq = np.zeros(R)
                for k in range(nb):
                    for rr in range(rank):
                        cq[k * rank + rr] = sum(qg[k * dg + d] * bk[k, d, rr] for d in range(dg))
                z = [sum(cq[c] * coef_k[b, l, c] for c in range(R)) / np.sqrt(R) for l in range(pos + 1)]
                zmax = max(z)
                e = [np.exp(v - zmax) for v in z]
                tot = sum(e)
                for l in range(pos + 1):
                    aq[l] += e[l] / tot / len(q_rows)
            for l in range(L):
                nbrs = [aq[x] for x in range(l - h, l + h + 1) if 0 <= x < L]
                pooled[g, l] = max(nbrs) if pool_mode == "max" else sum(nbrs) / kappa
        for l in range(L):
            if agg == "mean":
                out[b, l] = sum(pooled[g, l] for g in range(G)) / G
            else:
                best = pooled[0, l]
                for g in range(1, G):
                    if pooled[g, l] > best:
                        best = pooled[g, l]
                out[b, l] = best
    return out


def _agg_problem(seed):
    """G = 3 groups whose softmaxes peak at different positions, so the mean and
    the maximum over the groups rank the tokens differently."""
    p = small_problem(seed, B=2, hkv=2, G=3, dh=4, rank=5, L=18)
    p["q"] = p["q"] * 3.0
    return p


def check_group_aggregation_mean(seed=13):
    """F_G = mean over the G groups (Section 3.2.3) against the loop form."""
    p = _agg_problem(seed)
    got = decode.relevance(p["q"], None, p["bases_k"], p["coef_k"], p["L"], p["hkv"], 3, "max", "mean")["a_tilde"]
    want = ref_relevance_loop([p["q"]], [p["L"] - 1], p["bases_k"], p["coef_k"], p["L"], p["hkv"], 3, "max", "mean")
    return np.allclose(got, want, rtol=1e-12, atol=1e-15)


def check_group_aggregation_max(seed=14):
    """F_G = max over the G groups (the max variant) against the loop form,
    with average pooling."""
    p = _agg_problem(seed)
    got = decode.relevance(p["q"], None, p["bases_k"], p["coef_k"], p["L"], p["hkv"], 3, "avg", "max")["a_tilde"]
    want = ref_relevance_loop([p["q"]], [p["L"] - 1], p["bases_k"], p["coef_k"], p["L"], p["hkv"], 3, "avg", "max")
    return np.allclose(got, want, rtol=1e-12, atol=1e-15)


def check_query_fifo_order(seed=15):
    """The FIFO of Section 3.2.1: W_q raw queries, oldest first, the current one
    last.  The earlier rows are projected here in loop form and handed over as
    qwin_prev; the current query goes in as q.  Row i is the query at position
    L - W_q + i and sees keys up to that position only (Section 3.2.2), so a
    FIFO that put the current query first would mask it at L - W_q and change
    A~.  Also checks that the oracle's C^Q rows are those projections, in order."""
    p = small_problem(seed, B=2, hkv=2, G=2, dh=4, rank=5, L=16)
    rng = np.random.default_rng(seed + 100)
    Wq = 4
    B, hq, dh = p["q"].shape
    rows = [2.0 * rng.standard_normal((B, hq, dh)) for _ in range(Wq - 1)] + [2.0 * p["q"]]
    bk = p["bases_k"]
    rank = bk.shape[-1]
    G = p["G"]
    cq_rows = np.zeros((B, G, Wq, rank))
    for i, qr in enumerate(rows):
        for b in range(B):
            for g in range(G):
                qg = ref_group_query(qr, p["hkv"], g)[b]
                for rr in range(rank):
                    cq_rows[b, g, i, rr] = sum(qg[d] * bk[b, 0, d, rr] for d in range(qg.size))
    rel = decode.relevance(rows[-1], cq_rows[:, :, :Wq - 1], bk, p["coef_k"], p["L"], p["hkv"], 3, "max", "mean")
    if not np.allclose(rel["cQ"], cq_rows, rtol=1e-12, atol=1e-13):
        return False
    pos = [p["L"] - Wq + i for i in range(Wq)]
    want = ref_relevance_loop(rows, pos, bk, p["coef_k"], p["L"], p["hkv"], 3, "max", "mean")
    return np.allclose(rel["a_tilde"], want, rtol=1e-12, atol=1e-15)


ALL_CHECKS = [check_latent_identity, check_rotation_invariance, check_pool_vs_torch,
              check_topk_special_case, check_select_bruteforce, check_full_rank_exact,
              check_full_budget_dense, check_rope_complex, check_rope_shift_invariance,
              check_plain_gqa, check_causal_window, check_dense_comparator, check_full_reconstruction,
              check_group_aggregation_mean, check_group_aggregation_max, check_query_fifo_order]


# ----------------------------------------------------------------------------
# the pins as tests
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("nb", [1, 2])
def test_latent_scores_equal_reconstructed_scores(nb):
    assert check_latent_identity(nb=nb)


def test_rotation_invariance():
    assert check_rotation_invariance()


def test_pooling_matches_torch():
    assert check_pool_vs_torch()


def test_single_query_topk_is_plain_topk():
    assert check_topk_special_case()


def test_select_matches_bruteforce():
    assert check_select_bruteforce()


def test_full_rank_reconstruction_exact():
    assert check_full_rank_exact()


@pytest.mark.parametrize("theta,W", [(100.0, 3), (0.0, 3), (500000.0, 0)])
def test_full_budget_equals_dense_attention(theta, W):
    assert check_full_budget_dense(theta=theta, W=W)


def test_dense_comparator_matches_torch_sdpa():
    assert check_dense_comparator()


@pytest.mark.parametrize("nb,rank_v", [(1, 5), (2, 5), (1, 9), (2, 7)])
def test_full_reconstruction_matches_torch_sdpa(nb, rank_v):
    assert check_full_reconstruction(nb=nb, rank_v=rank_v)


def test_full_reconstruction_over_every_index_is_sparse_attention():
    """With every token selected, S^4R's sparse attention is full
    reconstruction (Section 3.2.3 against Appendix B.1)."""
    rng = np.random.default_rng(13)
    B, hq, hkv, dh, L, s, rank = 2, 4, 2, 8, 19, 2, 4
    Dp = hkv * dh
    args = dict(sink_k=rng.standard_normal((B, s, Dp)), sink_v=rng.standard_normal((B, s, Dp)),
                bases_k=rng.standard_normal((1, 1, Dp, rank)), bases_v=rng.standard_normal((1, 1, Dp, rank)),
                coef_k=rng.standard_normal((B, L, rank)), coef_v=rng.standard_normal((B, L, rank)))
    q = rng.standard_normal((B, hq, dh))
    full = decode.full_reconstruction_decode(q, L=L, n_kv_heads=hkv, theta=500.0, **args)
    idx = np.broadcast_to(np.arange(L), (B, L))
    sparse, _, _ = decode.sparse_attention(q, idx, L=L, n_kv_heads=hkv, rope_theta=500.0, **args)
    assert np.allclose(full, sparse, rtol=1e-12, atol=1e-12)


def test_rope_rotate_half_equals_complex_form():
    assert check_rope_complex()


def test_rope_relative_positions():
    assert check_rope_shift_invariance()


def test_plain_gqa_decode_special_case():
    assert check_plain_gqa()


def test_causal_query_window():
    assert check_causal_window()


@pytest.mark.parametrize("check", [check_group_aggregation_mean, check_group_aggregation_max])
def test_group_aggregation_matches_loop_form(check):
    assert check()


def test_group_aggregation_modes_differ_on_the_pin_inputs():
    """The aggregation pins use inputs on which mean and max give different
    rankings, so exchanging the two modes cannot pass them."""
    p = _agg_problem(13)
    a_mean = decode.relevance(p["q"], None, p["bases_k"], p["coef_k"], p["L"], p["hkv"], 3, "max", "mean")["a_tilde"]
    a_max = decode.relevance(p["q"], None, p["bases_k"], p["coef_k"], p["L"], p["hkv"], 3, "max", "max")["a_tilde"]
    assert not np.allclose(a_mean, a_max)
    assert any(not np.array_equal(np.argsort(-a_mean[b], kind="stable")[:5], np.argsort(-a_max[b], kind="stable")[:5])
               for b in range(a_mean.shape[0]))


def test_query_fifo_oldest_first():
    assert check_query_fifo_order()


def test_exact_window_kv_replaces_reconstruction():
    """With exact window KV equal to the reconstructed window rows the output is
    unchanged; with different rows only attention changes, never selection."""
    p = small_problem(11, L=30)
    W = 5
    cfg = cfg_of(p, W=W, k=6)
    a = run(p, cfg)
    K = ref_full_keys(p["coef_k"], p["bases_k"])
    V = ref_full_keys(p["coef_v"], p["bases_v"])
    L = p["L"]
    same = run(p, cfg, win_k=K[:, L - W:L], win_v=V[:, L - W:L])
    assert np.allclose(same["out"], a["out"], rtol=1e-12, atol=1e-12)
    rng = np.random.default_rng(0)
    other = run(p, cfg, win_k=rng.standard_normal(K[:, L - W:L].shape),
                win_v=rng.standard_normal(V[:, L - W:L].shape))
    assert np.array_equal(other["idx"], a["idx"])
    assert not np.allclose(other["out"], a["out"])


def test_append_projects_and_rounds_new_row():
    p = small_problem(12, L=20)
    rng = np.random.default_rng(1)
    Dp = p["hkv"] * p["dh"]
    kn, vn = rng.standard_normal((2, Dp)), rng.standard_normal((2, Dp))
    cfg = cfg_of(p)
    cfg["dtype"] = "bf16"
    r = run(p, cfg, k_new=kn, v_new=vn)
    # independent: torch matmul per basis group, torch bf16 cast
    ref = torch.einsum("bd,bdr->br", torch.from_numpy(kn), torch.from_numpy(p["bases_k"][:, 0]))
    ref = ref.to(torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(r["coef_k"][:, p["L"] - 1], ref)
    assert np.array_equal(r["coef_k"][:, :p["L"] - 1], p["coef_k"][:, :p["L"] - 1])


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(13)
    x = np.concatenate([rng.standard_normal(10000) * 10.0 ** rng.integers(-30, 30, 10000),
                        np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -9, -0.0, 0.0, 65504.0])])
    ref = torch.from_numpy(x).to(torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(storage.to_bf16(x), ref)


def test_num_selected_formula():
    for L, W, k in itertools.product([0, 1, 5, 64, 100], [0, 1, 4, 64], [0, 1, 10, 1000]):
        if L == 0:
            continue
        a = np.zeros((1, L))
        assert decode.select(a, L, W, k).shape[1] == decode.num_selected(L, W, k)


# ----------------------------------------------------------------------------
# mutation tests: a planted mistake in the oracle must trip a pin
# ----------------------------------------------------------------------------

def _fails(monkeypatch_ctx, target, name, replacement):
    with monkeypatch_ctx.context() as m:
        m.setattr(target, name, replacement)
        return [c.__name__ for c in ALL_CHECKS if not c()]


def test_mutation_dropped_scale(monkeypatch):
    orig = decode.latent_logits

    def bad(cQ, coef_k, L):
        return orig(cQ, coef_k, L) * np.sqrt(np.asarray(coef_k).shape[-1])
    assert _fails(monkeypatch, decode, "latent_logits", bad)


def test_mutation_wrong_query_grouping(monkeypatch):
    def bad(q, n_kv_heads):
        q = np.asarray(q, dtype=np.float64)
        B, hq, dh = q.shape
        return q.reshape(B, hq // n_kv_heads, n_kv_heads * dh)   # plain view: wrong heads
    assert _fails(monkeypatch, decode, "group_queries", bad)


def test_mutation_pool_off_by_one(monkeypatch):
    orig = decode.pool

    def bad(AQ, kappa, mode="max"):
        return np.roll(orig(AQ, kappa, mode), 1, axis=-1)
    assert _fails(monkeypatch, decode, "pool", bad)


def test_mutation_tie_to_higher_index(monkeypatch):
    def bad(a_tilde, L, W, k):
        a = np.asarray(a_tilde, dtype=np.float64)
        n_hist = max(L - W, 0)
        k_eff = min(k, n_hist)
        out = []
        for row in a:
            order = np.argsort(-row[:n_hist][::-1], kind="stable")
            glob = np.sort(n_hist - 1 - order[:k_eff])
            out.append(np.concatenate([glob, np.arange(n_hist, L)]))
        return np.array(out, dtype=np.int64)
    assert "check_select_bruteforce" in _fails(monkeypatch, decode, "select", bad)


def test_mutation_rope_sign(monkeypatch):
    orig = decode.rope

    def bad(x, pos, theta):
        return orig(x, -np.asarray(pos, dtype=np.float64), theta)
    assert _fails(monkeypatch, decode, "rope", bad)


def test_mutation_transposed_basis(monkeypatch):
    def bad(coef_rows, bases):
        bases = np.asarray(bases, dtype=np.float64)
        c = np.asarray(coef_rows, dtype=np.float64)
        # uses the basis rows as if they were columns (only shape-valid when square)
        nb, dg, rank = bases.shape[1:]
        bt = np.swapaxes(bases, -1, -2) if dg == rank else bases[..., ::-1, :]
        cb = c.reshape(c.shape[0], c.shape[1], nb, rank)
        bb = np.broadcast_to(bt, (c.shape[0], nb, dg, rank))
        return np.einsum("bnkr,bkdr->bnkd", cb, bb).reshape(c.shape[0], c.shape[1], nb * dg)
    assert _fails(monkeypatch, decode, "reconstruct", bad)


def test_mutation_window_mean_drops_row(monkeypatch):
    def bad(A):
        return np.mean(A[:, :, 1:, :], axis=2) if A.shape[2] > 1 else np.mean(A, axis=2)
    assert "check_causal_window" in _fails(monkeypatch, decode, "window_mean", bad)


def test_mutation_group_aggregation_swapped(monkeypatch):
    def bad(P, mode="mean"):
        P = np.asarray(P, dtype=np.float64)
        return np.max(P, axis=1) if mode == "mean" else np.mean(P, axis=1)
    failed = _fails(monkeypatch, decode, "aggregate", bad)
    assert "check_group_aggregation_mean" in failed and "check_group_aggregation_max" in failed


def test_mutation_fifo_newest_first(monkeypatch):
    orig = decode.query_window

    def bad(q, qwin_prev, bases_k, n_kv_heads):
        cq = orig(q, None, bases_k, n_kv_heads)
        if qwin_prev is None or np.asarray(qwin_prev).shape[2] == 0:
            return cq
        return np.concatenate([cq, np.asarray(qwin_prev, dtype=np.float64)], axis=2)
    assert "check_query_fifo_order" in _fails(monkeypatch, decode, "query_window", bad)


# ----------------------------------------------------------------------------
# prefill (Section 3.1)
# ----------------------------------------------------------------------------

def test_prefill_bases_orthonormal_and_exact_on_low_rank():
    rng = np.random.default_rng(14)
    B, N, Dp, r_true, s = 2, 200, 16, 5, 4
    F = rng.standard_normal((B, N, r_true))
    P = rng.standard_normal((B, r_true, Dp))
    S = np.einsum("bnr,brd->bnd", F, P)
    st = prefill.prefill(S, S, s, rank=r_true, sample_idx=np.arange(0, N - s, 3), dtype="fp32")
    for b in range(B):
        Bm = st["bases_k"][b, 0]
        assert np.allclose(Bm.T @ Bm, np.eye(r_true), atol=1e-6)
    # rank >= true rank: coefficients reconstruct the raw (un-normalised) rows
    st64 = prefill.prefill(S, S, s, rank=r_true, sample_idx=np.arange(0, N - s, 3), dtype="fp32")
    rec = decode.reconstruct(st64["coef_k"], st64["bases_k"])
    assert np.allclose(rec, S[:, s:], rtol=1e-4, atol=1e-4 * np.abs(S).max())
    assert np.array_equal(st["sink_k"], storage.to_fp32(S[:, :s]))


def test_prefill_normalisation_changes_basis_not_projection():
    """Normalisation only feeds the SVD: the stored coefficients are S B."""
    rng = np.random.default_rng(15)
    S = rng.standard_normal((1, 60, 8)) * rng.random((1, 60, 1)) * 50
    st = prefill.prefill(S, S, 2, rank=3, sample_idx=np.arange(0, 58, 2), dtype="fp32")
    C_ref = np.einsum("td,dr->tr", S[0, 2:], st["bases_k"][0, 0])
    assert np.allclose(st["coef_k"][0], C_ref, rtol=1e-6, atol=1e-5)
    Xn = S[0, 2:][np.arange(0, 58, 2)]
    Xn = Xn / np.linalg.norm(Xn, axis=1, keepdims=True)
    v = np.linalg.svd(Xn)[2][:3].T
    # same subspace as the SVD of the normalised samples
    assert np.allclose(v @ v.T, st["bases_k"][0, 0] @ st["bases_k"][0, 0].T, atol=1e-5)


def test_hybrid_sampler_split():
    idx = prefill.sample_hybrid(1000, eta=0.2)
    assert idx.size == 200
    recent = idx[idx >= 1000 - 140]
    assert recent.size == 140 and recent.max() == 999
    assert np.all(np.diff(idx) > 0)


# Hybrid sampling of Section 3.1.2 with the 7:3 recent-to-uniform split of
# Section 4: T' = floor(eta * T) rows, round(0.7 T') of them the contiguous
# block of the latest positions, the rest spread evenly over the earlier
# positions from the first to the last one before the block (reading: evenly
# spaced real positions, rounded to the nearest integer, halves to even).
# Worked by hand:
#   T = 100, eta = 0.2:  T' = 20, 14 recent = 86..99, 6 uniform over [0, 85]
#                        step 85/5 = 17 -> 0 17 34 51 68 85
#   T = 25, eta = 0.4:   T' = 10, 7 recent = 18..24, 3 uniform over [0, 17]
#                        step 8.5 -> 0, 8.5 -> 8 (half to even), 17
#   T = 61, eta = 0.25:  T' = 15, round(10.5) = 10 recent (half to even) =
#                        51..60, 5 uniform over [0, 50] step 12.5 -> 0, 12.5 -> 12,
#                        25, 37.5 -> 38, 50
#   T = 9, eta = 0.3:    T' = 2, round(1.4) = 1 recent = 8, 1 uniform = 0
HYBRID_CASES = [
    (100, 0.2, [0, 17, 34, 51, 68, 85] + list(range(86, 100))),
    (25, 0.4, [0, 8, 17] + list(range(18, 25))),
    (61, 0.25, [0, 12, 25, 38, 50] + list(range(51, 61))),
    (9, 0.3, [0, 8]),
]


@pytest.mark.parametrize("T,eta,want", HYBRID_CASES)
def test_hybrid_sampler_positions_by_hand(T, eta, want):
    assert prefill.sample_hybrid(T, eta).tolist() == want


def test_mutation_sampler_first_positions(monkeypatch):
    """Taking the first n_uniform early positions instead of spreading them
    over the early part is caught by the hand-computed lists."""
    def bad(T, eta, recent_share=0.7):
        n = max(1, int(np.floor(eta * T)))
        n_recent = min(T, int(round(recent_share * n)))
        return np.concatenate([np.arange(n - n_recent), np.arange(T - n_recent, T)]).astype(np.int64)
    with monkeypatch.context() as m:
        m.setattr(prefill, "sample_hybrid", bad)
        assert any(prefill.sample_hybrid(T, eta).tolist() != want for T, eta, want in HYBRID_CASES)


def test_prefill_initial_query_window_loop_form():
    """The prefill's initial C^Q (Section 3.1, the most recent W queries
    projected on the key basis) row by row against the loop-form grouping and
    an explicit sum over the basis rows."""
    rng = np.random.default_rng(16)
    B, hkv, G, dh, W, N, s, rank = 2, 2, 3, 4, 3, 40, 2, 5
    Dp = hkv * dh
    S = rng.standard_normal((B, N, Dp))
    qr = rng.standard_normal((B, hkv * G, W, dh))
    st = prefill.prefill(S, S, s, rank=rank, dtype="fp32", q_recent=qr, n_kv_heads=hkv)
    bk = st["bases_k"]
    for b in range(B):
        for g in range(G):
            for w in range(W):
                qg = ref_group_query(qr[:, :, w, :], hkv, g)[b]
                want = [sum(qg[d] * bk[b, 0, d, r] for d in range(Dp)) for r in range(rank)]
                assert np.allclose(st["qwin"][b, g, w], want, rtol=1e-6, atol=1e-6)


def test_oracle_package_exports():
    for name in ("decode_step", "select", "pool", "rope", "attend", "reconstruct"):
        assert hasattr(oracle, name)


@pytest.mark.parametrize("pool_mode,agg,wq", [("max", "mean", 1), ("avg", "max", 4), ("max", "max", 2),
                                              ("avg", "mean", 4)])
def test_relevance_lies_in_unit_interval(pool_mode, agg, wq):
    """A~ is a mean or maximum over groups of pooled window means of softmax
    probabilities (Section 3.2.2-3.2.3), so it lies in [0, 1] whatever the
    logits; the selection's finer key for the fused step relies on it."""
    rng = np.random.default_rng(21 + wq)
    B, hq, hkv, dh, L, r = 2, 8, 2, 16, 300, 8
    Dp = hkv * dh
    bases = np.linalg.qr(rng.standard_normal((Dp, r)))[0][None, None]
    for scale in (0.1, 10.0, 1e4):                        # flat to one-hot softmaxes
        q = scale * rng.standard_normal((B, hq, dh))
        coef = rng.standard_normal((B, L, r))
        qwin = scale * rng.standard_normal((B, hq // hkv, wq - 1, r)) if wq > 1 else None
        a = decode.relevance(q, qwin, bases, coef, L, hkv, 7, pool_mode, agg)["a_tilde"]
        assert np.all(a >= 0.0) and np.all(a <= 1.0 + 1e-12), (scale, a.min(), a.max())
        assert a.max() > 0.0
