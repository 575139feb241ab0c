"""S^4R prefilling stage (Section 3.1), float64 numpy.

Turns a prompt's raw pre-RoPE keys and values into the stored decode state:
full-precision sinks, per-sequence bases B^{K/V} and coefficient caches
C^{K/V} (Eq. svd and Eq. coefficients), plus the initial query window C^Q.

Readings:
  P1  Sampling.  Two samplers are provided: the paper's hybrid sampler
      (uniform over the early positions plus a contiguous recent block, split
      recent:uniform = 7:3, T' = eta * T; Sections 3.1.2 and 4), and a plain
      "every n-th non-sink token" sampler used by the synthetic workloads.
  P2  Normalisation applies to the sampled rows only, before the SVD (3.1.2);
      the coefficients project the raw, un-normalised rows (Eq. coefficients),
      so nothing has to be undone at reconstruction.  With several basis
      groups each group's slice is normalised on its own.
  P3  Optional mean-centring of the normalised samples shapes the basis only;
      no mean vector is stored.
  P4  Storage rounding is applied once to the outputs (sinks, bases,
      coefficients) in the requested format.
"""

import numpy as np

from . import storage


def split_sinks(S, n_sink):
    """First s tokens bypass compression (3.1.1)."""
    return S[:, :n_sink], S[:, n_sink:]


def sample_every(T, step):
    """Every step-th non-sink position."""
    return np.arange(0, T, step, dtype=np.int64)


def sample_hybrid(T, eta, recent_share=0.7):
    """Hybrid sampler of 3.1.2: a contiguous block of the most recent tokens
    plus uniformly spaced early tokens, T' = floor(eta*T) in total, with
    recent:uniform = recent_share : 1 - recent_share."""
    n = max(1, int(np.floor(eta * T)))
    n_recent = min(T, int(round(recent_share * n)))
    n_uniform = n - n_recent
    recent = np.arange(T - n_recent, T, dtype=np.int64)
    early_end = T - n_recent
    if n_uniform > 0 and early_end > 0:
        uniform = np.unique(np.linspace(0, early_end - 1, num=min(n_uniform, early_end)).round().astype(np.int64))
    else:
        uniform = np.zeros(0, dtype=np.int64)
    return np.concatenate([uniform, recent])


def normalize_rows(X):
    """Token-wise L2 normalisation along the feature axis (3.1.2)."""
    n = np.linalg.norm(X, axis=-1, keepdims=True)
    return X / np.where(n > 0, n, 1.0)


def truncated_svd_basis(X, rank):
    """Top-rank right singular vectors of X [T', d] as a [d, rank] basis (Eq. svd)."""
    _, _, vt = np.linalg.svd(X, full_matrices=False)
    return vt[:rank].T.copy()


def build_bases(S_nonsink, sample_idx, rank, n_groups=1, center=False):
    """Bases [B, nb, Dp/nb, rank] from the sampled non-sink rows (P2, P3)."""
    B, T, Dp = S_nonsink.shape
    dg = Dp // n_groups
    out = np.empty((B, n_groups, dg, rank))
    for b in range(B):
        X = S_nonsink[b, sample_idx]
        for k in range(n_groups):
            Xg = normalize_rows(X[:, k * dg:(k + 1) * dg])
            if center:
                Xg = Xg - Xg.mean(axis=0, keepdims=True)
            out[b, k] = truncated_svd_basis(Xg, rank)
    return out


def project_tokens(S_nonsink, bases):
    """C = S B per basis group (Eq. coefficients) -> [B, T, nb*rank]."""
    B, T, Dp = S_nonsink.shape
    nb, dg, rank = bases.shape[1:]
    Sg = S_nonsink.reshape(B, T, nb, dg)
    return np.einsum("btkd,bkdr->btkr", Sg, bases).reshape(B, T, nb * rank)


def prefill(S_k, S_v, n_sink, rank, n_groups=1, sample_idx=None, center=False,
            dtype=storage.FP32, q_recent=None, n_kv_heads=None):
    """Whole prefill stage for one layer.

    S_k, S_v: [B, N, Dp] raw pre-RoPE keys/values of the prompt (sinks first).
    sample_idx: non-sink positions fed to the SVD (default: every 8th).
    q_recent: optional [B, h_q, W, d_h] most recent queries -> initial C^Q.
    Returns a dict of stored (rounded) arrays, all float64.
    """
    S_k = np.asarray(S_k, dtype=np.float64)
    S_v = np.asarray(S_v, dtype=np.float64)
    sink_k, X_k = split_sinks(S_k, n_sink)
    sink_v, X_v = split_sinks(S_v, n_sink)
    T = X_k.shape[1]
    if sample_idx is None:
        sample_idx = sample_every(T, 8)
    rnd = lambda a: storage.round_to(a, dtype)  # noqa: E731
    bk = rnd(build_bases(X_k, sample_idx, rank, n_groups, center))
    bv = rnd(build_bases(X_v, sample_idx, rank, n_groups, center))
    out = {
        "sink_k": rnd(sink_k),
        "sink_v": rnd(sink_v),
        "bases_k": bk,
        "bases_v": bv,
        # the stored (rounded) bases are the ones decode reconstructs with
        "coef_k": rnd(project_tokens(X_k, bk)),
        "coef_v": rnd(project_tokens(X_v, bv)),
    }
    if q_recent is not None:
        qr = np.asarray(q_recent, dtype=np.float64)        # [B, h_q, W, d_h]
        B, hq, W, dh = qr.shape
        G = hq // n_kv_heads
        # group queries per row (same mapping as decode), then project
        qg = qr.reshape(B, n_kv_heads, G, W, dh).transpose(0, 2, 3, 1, 4).reshape(B, G, W, n_kv_heads * dh)
        nb, dg, r = bk.shape[1:]
        cq = np.einsum("bgwkd,bkdr->bgwkr", qg.reshape(B, G, W, nb, dg), bk).reshape(B, G, W, nb * r)
        out["qwin"] = storage.to_fp32(cq)
    return out
