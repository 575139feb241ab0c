"""S^4R decode step, written out in the order of Section 3.2 (float64, numpy).

Notation follows the paper: B batch, G query-to-KV head ratio, Dp = h_kv*d_h
(the concatenated KV width of one layer), r the latent width of the
coefficient caches, L the current non-sink cache length (the token appended at
this step included), s the number of sink tokens, W the local window, W_q the
number of query-coefficient rows used for scoring, kappa the pooling kernel.

Array layouts (all float64 unless stated):
  q          [B, h_q, d_h]              pre-RoPE query of the current token
  bases      [B or 1, nb, Dp/nb, rank]  nb basis groups; nb = 1 is the paper's
                                        single basis over Dp (Eq. svd)
  coef       [B, >=L, R]                R = nb*rank, row l = non-sink token l
  qwin_prev  [B, G, W_q-1, R]           older query coefficients, oldest first
  sink_k/v   [B, s, Dp]                 pre-RoPE sink keys/values

Readings of points the paper leaves open (each applied where marked):
  R1  GQA grouping.  Query head h belongs to KV head j = h // G and group
      member g = h % G; the group-g query is the concatenation over j of the
      heads j*G + g, a vector of width Dp (the shape of s_t^Q in 3.2.1).
  R2  Scale.  Logits divide by sqrt(R) with R the full latent width (nb*rank);
      per-head bases are the block-diagonal case of one joint basis.
  R3  Query FIFO.  Row i of C^Q (oldest first) is the query at non-sink
      position L - W_q + i; the causal mask keeps keys l <= that position.
  R4  Pooling.  Stride 1, output length equal to input length, window
      [l - kappa//2, l + kappa//2] clipped to [0, L); max ignores the missing
      neighbours, avg divides the in-range sum by kappa.  Pooling runs over
      the full length and precedes the restriction to [0, L - W).
  R5  Top-k.  k_eff = min(k, max(L - W, 0)); equal scores go to the lower
      position.  The index set is the sorted global positions followed by the
      window positions [max(L - W, 0), L).
  R6  Positions.  Sink i sits at position i, non-sink token l at s + l, the
      query at s + L - 1; RoPE is the rotate-half form with angle
      pos * theta^(-2i/d_h), theta = 0 disables it.  Values are not rotated.
  R7  Window source.  By default the local window is reconstructed from its
      coefficients like every other selected token; if exact window KV is
      given it replaces those rows.
"""

import numpy as np

from . import storage


def _f64(x):
    return None if x is None else np.asarray(x, dtype=np.float64)


# ----------------------------------------------------------------------------
# Section 3.2.1: compressed cache update
# ----------------------------------------------------------------------------

def group_queries(q, n_kv_heads):
    """s_t^Q of shape [B, G, Dp] from per-head queries [B, h_q, d_h] (R1)."""
    q = _f64(q)
    B, hq, dh = q.shape
    G = hq // n_kv_heads
    # q[b, j*G + g, :] -> out[b, g, j*dh:(j+1)*dh]
    return q.reshape(B, n_kv_heads, G, dh).transpose(0, 2, 1, 3).reshape(B, G, n_kv_heads * dh)


def project(x, bases):
    """Coefficients x B of Eq. coefficients / the update equations of 3.2.1.

    x: [B, ..., Dp]; bases [B|1, nb, Dp/nb, rank] -> [B, ..., nb*rank].  Each
    basis group projects its own slice of the feature axis.
    """
    x = _f64(x)
    bases = _f64(bases)
    nb, dg, rank = bases.shape[1:]
    lead = x.shape[:-1]
    xb = x.reshape(x.shape[0], -1, nb, dg)
    bb = np.broadcast_to(bases, (x.shape[0], nb, dg, rank))
    c = np.einsum("bnkd,bkdr->bnkr", xb, bb)
    return c.reshape(*lead, nb * rank)


def project_append(k_new, v_new, bases_k, bases_v, dtype):
    """New key/value coefficient rows c_t^K = s_t^K B^K, c_t^V = s_t^V B^V,
    rounded to the cache's storage format (they are written into it)."""
    ck = project(_f64(k_new)[:, None, :], bases_k)[:, 0]
    cv = project(_f64(v_new)[:, None, :], bases_v)[:, 0]
    return storage.round_to(ck, dtype), storage.round_to(cv, dtype)


def query_window(q, qwin_prev, bases_k, n_kv_heads):
    """C^Q after pushing the current query coefficients c_t^Q = s_t^Q B^K onto
    the FIFO (R3): [B, G, W_q, R], oldest first."""
    cq = project(group_queries(q, n_kv_heads), bases_k)  # [B, G, R]
    cq = cq[:, :, None, :]
    if qwin_prev is None or _f64(qwin_prev).shape[2] == 0:
        return cq
    return np.concatenate([_f64(qwin_prev), cq], axis=2)


# ----------------------------------------------------------------------------
# Section 3.2.2: latent-space relevance estimation
# ----------------------------------------------------------------------------

def latent_logits(cQ, coef_k, L):
    """Z = C^Q (C_t^K)^T / sqrt(r) over the L non-sink tokens (R2)."""
    cQ = _f64(cQ)
    CK = _f64(coef_k)[:, :L, :]
    R = CK.shape[-1]
    return np.einsum("bgir,blr->bgil", cQ, CK) / np.sqrt(R)


def causal_mask(Z, L):
    """Mask keys after each query row's own position (R3)."""
    Z = np.array(Z, dtype=np.float64, copy=True)
    Wq = Z.shape[2]
    pos_q = L - Wq + np.arange(Wq)                      # [W_q]
    keys = np.arange(Z.shape[3])                        # [L]
    Z[:, :, keys[None, :] > pos_q[:, None]] = -np.inf   # broadcast over (i, l)
    return Z


def softmax_over_length(Z):
    """softmax along the cache-length axis (max-subtracted)."""
    m = np.max(Z, axis=-1, keepdims=True)
    e = np.exp(Z - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def window_mean(A):
    """A^Q = (1/W_q) sum_i A[:, :, i, :]."""
    return np.mean(A, axis=2)


# ----------------------------------------------------------------------------
# Section 3.2.3: pooling, group aggregation, selection
# ----------------------------------------------------------------------------

def pool(AQ, kappa, mode="max"):
    """Sequence pooling F_P with kernel kappa along the last axis (R4)."""
    AQ = _f64(AQ)
    if kappa % 2 != 1:
        raise ValueError("pool kernel must be odd")
    h = kappa // 2
    L = AQ.shape[-1]
    fill = -np.inf if mode == "max" else 0.0
    padded = np.full(AQ.shape[:-1] + (L + 2 * h,), fill)
    padded[..., h:h + L] = AQ
    views = [padded[..., o:o + L] for o in range(kappa)]
    if mode == "max":
        return np.max(np.stack(views), axis=0)
    if mode == "avg":
        return np.sum(np.stack(views), axis=0) / kappa
    raise ValueError(f"unknown pool mode {mode!r}")


def aggregate(P, mode="mean"):
    """Group aggregation F_G over the G axis -> A~ [B, L]."""
    if mode == "mean":
        return np.mean(P, axis=1)
    if mode == "max":
        return np.max(P, axis=1)
    raise ValueError(f"unknown group aggregation {mode!r}")


def num_selected(L, W, k):
    """m = |I^|: k_eff global tokens plus the (clipped) local window (R5)."""
    return min(k, max(L - W, 0)) + min(W, L)


def select(a_tilde, L, W, k):
    """I^ = I_local U TopK(A~[:, :L-W], k) (R5); int64 [B, m]."""
    a_tilde = _f64(a_tilde)
    B = a_tilde.shape[0]
    n_hist = max(L - W, 0)
    k_eff = min(k, n_hist)
    local = np.arange(n_hist, L, dtype=np.int64)
    out = np.empty((B, k_eff + local.size), dtype=np.int64)
    for b in range(B):
        # stable sort of the negated scores: equal scores keep index order
        order = np.argsort(-a_tilde[b, :n_hist], kind="stable")
        out[b, :k_eff] = np.sort(order[:k_eff])
        out[b, k_eff:] = local
    return out


# ----------------------------------------------------------------------------
# Section 3.2.3: sparse reconstruction, sinks, RoPE, final attention
# ----------------------------------------------------------------------------

def reconstruct(coef_rows, bases):
    """K^ = C[I^] (B)^T (and V^ likewise); coef_rows [B, n, R] -> [B, n, Dp]."""
    c = _f64(coef_rows)
    bases = _f64(bases)
    nb, dg, rank = bases.shape[1:]
    cb = c.reshape(c.shape[0], c.shape[1], nb, rank)
    bb = np.broadcast_to(bases, (c.shape[0], nb, dg, rank))
    return np.einsum("bnkr,bkdr->bnkd", cb, bb).reshape(c.shape[0], c.shape[1], nb * dg)


def rope(x, pos, theta):
    """Rotate-half RoPE on the last axis of x [..., n, d] at positions [..., n] (R6)."""
    x = _f64(x)
    if theta == 0:
        return x.copy()
    d = x.shape[-1]
    half = d // 2
    inv_freq = float(theta) ** (-np.arange(half, dtype=np.float64) * 2.0 / d)
    ang = np.asarray(pos, dtype=np.float64)[..., None] * inv_freq
    cos, sin = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def attend(q, kstar, vstar, pos_k, pos_q, theta, n_kv_heads):
    """O_t = softmax(RoPE(q) RoPE(K*)^T / sqrt(d_h)) V* per query head, with
    query head h reading KV head h // G (R1, R6).  Returns [B, h_q, d_h]."""
    q = _f64(q)
    kstar = _f64(kstar)
    vstar = _f64(vstar)
    B, hq, dh = q.shape
    G = hq // n_kv_heads
    n = kstar.shape[1]
    qr = rope(q, np.broadcast_to(np.asarray(pos_q, dtype=np.float64)[:, None], (B, hq)), theta)
    out = np.empty((B, hq, dh))
    for h in range(hq):
        j = h // G
        kj = rope(kstar[:, :, j * dh:(j + 1) * dh], pos_k, theta)   # [B, n, dh]
        vj = vstar[:, :, j * dh:(j + 1) * dh]
        logits = np.einsum("bd,bnd->bn", qr[:, h], kj) / np.sqrt(dh)
        if n == 0:
            raise ValueError("attention over an empty set")
        p = softmax_over_length(logits)
        out[:, h] = np.einsum("bn,bnd->bd", p, vj)
    return out


# ----------------------------------------------------------------------------
# The whole step
# ----------------------------------------------------------------------------

def dense_decode(q, k_cache, v_cache, n_kv_heads, theta):
    """Comparator, not part of S^4R: the "Full KV" decode attention of the
    efficiency comparison (Section 4.2; the full attention term of Appendix
    B.1).  The cache holds the N = k_cache.shape[1] tokens uncompressed, keys
    already rotated by RoPE at their positions 0..N-1 (as a plain KV cache
    stores them); the query is rotated at position N - 1.  Head h reads KV
    head h // G (R1).  Returns [B, h_q, d_h]."""
    q = _f64(q)
    K = _f64(k_cache)
    V = _f64(v_cache)
    B, hq, dh = q.shape
    N = K.shape[1]
    G = hq // n_kv_heads
    qr = rope(q, np.full((B, hq), float(N - 1)), theta)
    out = np.empty((B, hq, dh))
    for h in range(hq):
        j = h // G
        logits = np.einsum("bd,bnd->bn", qr[:, h], K[:, :, j * dh:(j + 1) * dh]) / np.sqrt(dh)
        out[:, h] = np.einsum("bn,bnd->bd", softmax_over_length(logits), V[:, :, j * dh:(j + 1) * dh])
    return out


def full_reconstruction_decode(q, sink_k, sink_v, bases_k, bases_v, coef_k, coef_v, L, n_kv_heads, theta):
    """Comparator, not S^4R: full-reconstruction low-rank decoding (Appendix
    B.1).  Every cached non-sink token is reconstructed, K = C^K (B^K)^T and
    V = C^V (B^V)^T (rows 0..L-1), the result is laid out as a plain KV cache
    (sinks at positions 0..s-1, token l at s + l, keys rotated at their
    positions, R6) and attended to as in the Full-KV decode, the query at
    s + L - 1.  Returns [B, h_q, d_h]."""
    k_hat = reconstruct(_f64(coef_k)[:, :L], bases_k)
    v_hat = reconstruct(_f64(coef_v)[:, :L], bases_v)
    k_all = np.concatenate([_f64(sink_k), k_hat], axis=1)
    v_all = np.concatenate([_f64(sink_v), v_hat], axis=1)
    B, N, Dp = k_all.shape
    dh = q.shape[2]
    pos = np.broadcast_to(np.arange(N, dtype=np.float64)[None, :, None], (B, N, Dp // dh))
    k_rot = rope(k_all.reshape(B, N, Dp // dh, dh), pos, theta).reshape(B, N, Dp)
    return dense_decode(q, k_rot, v_all, n_kv_heads, theta)


def relevance(q, qwin_prev, bases_k, coef_k, L, n_kv_heads, pool_kernel=7,
              pool_mode="max", group_agg="mean"):
    """Latent relevance A~ of every non-sink token (3.2.2 and the first two
    equations of 3.2.3).  Returns a dict of every intermediate."""
    cQ = query_window(q, qwin_prev, bases_k, n_kv_heads)
    Wq = cQ.shape[2]
    if Wq > L:
        raise ValueError("query window longer than the cache")
    Z = causal_mask(latent_logits(cQ, coef_k, L), L)
    A = softmax_over_length(Z)
    AQ = window_mean(A)
    P = pool(AQ, pool_kernel, pool_mode)
    a_tilde = aggregate(P, group_agg)
    return {"cQ": cQ, "Z": Z, "A": A, "AQ": AQ, "P": P, "a_tilde": a_tilde}


def sparse_attention(q, idx, sink_k, sink_v, bases_k, bases_v, coef_k, coef_v, L,
                     n_kv_heads, rope_theta, win_k=None, win_v=None, W=None):
    """Reconstruct the selected tokens, prepend the sinks, attend (3.2.3)."""
    idx = np.asarray(idx, dtype=np.int64)
    B = idx.shape[0]
    CK = _f64(coef_k)
    CV = _f64(coef_v)
    rows_k = np.stack([CK[b, idx[b]] for b in range(B)])
    rows_v = np.stack([CV[b, idx[b]] for b in range(B)])
    k_hat = reconstruct(rows_k, bases_k)
    v_hat = reconstruct(rows_v, bases_v)
    if win_k is not None:
        # R7: exact window KV replaces the reconstructed window rows.
        # win_k[:, w] holds position L - W + w.
        win_k = _f64(win_k)
        win_v = _f64(win_v)
        for b in range(B):
            for n, l in enumerate(idx[b]):
                w = l - (L - W)
                if l >= L - W and 0 <= w < W:
                    k_hat[b, n] = win_k[b, w]
                    v_hat[b, n] = win_v[b, w]
    sink_k = _f64(sink_k)
    sink_v = _f64(sink_v)
    s = sink_k.shape[1]
    kstar = np.concatenate([sink_k, k_hat], axis=1)
    vstar = np.concatenate([sink_v, v_hat], axis=1)
    pos_k = np.concatenate([np.broadcast_to(np.arange(s), (B, s)), s + idx], axis=1)
    pos_q = np.full(B, s + L - 1)
    out = attend(q, kstar, vstar, pos_k, pos_q, rope_theta, n_kv_heads)
    return out, k_hat, v_hat


def decode_step(cfg, L, q, sink_k, sink_v, bases_k, bases_v, coef_k, coef_v,
                qwin_prev=None, win_k=None, win_v=None, k_new=None, v_new=None):
    """One decode step of one layer.

    cfg keys: n_kv_heads, window, topk, pool_kernel, pool_mode, group_agg,
    rope_theta, dtype (storage format, used for the appended row).
    If k_new/v_new are given they are projected and written into row L - 1 of
    copies of the coefficient caches first (3.2.1).  Returns a dict with
    a_tilde [B, L], idx [B, m], out [B, h_q, d_h] and the intermediates.
    """
    coef_k = np.array(coef_k, dtype=np.float64, copy=True)
    coef_v = np.array(coef_v, dtype=np.float64, copy=True)
    if k_new is not None:
        ck, cv = project_append(k_new, v_new, bases_k, bases_v, cfg.get("dtype", storage.FP32))
        coef_k[:, L - 1] = ck
        coef_v[:, L - 1] = cv
    rel = relevance(q, qwin_prev, bases_k, coef_k, L, cfg["n_kv_heads"],
                    cfg.get("pool_kernel", 7), cfg.get("pool_mode", "max"),
                    cfg.get("group_agg", "mean"))
    idx = select(rel["a_tilde"], L, cfg["window"], cfg["topk"])
    out, k_hat, v_hat = sparse_attention(q, idx, sink_k, sink_v, bases_k, bases_v,
                                         coef_k, coef_v, L, cfg["n_kv_heads"],
                                         cfg.get("rope_theta", 0.0), win_k, win_v,
                                         cfg["window"])
    rel.update({"idx": idx, "out": out, "k_hat": k_hat, "v_hat": v_hat,
                "coef_k": coef_k, "coef_v": coef_v})
    return rel
