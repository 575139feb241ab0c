"""Helpers shared by the GPU parity tests: move oracle-side stored state onto
the GPU in the library's layouts, and the comparison rules.

Stored state is built on the host (workloads + the oracle's prefill, or the
workloads' latent recipe), already rounded to the storage format, so the GPU
and the oracle read exactly the same values."""

import numpy as np
import torch

import paper_2608_00528_amd as s4r
import workloads as W


def cfg_from_workload(wl, capacity=None, **over):
    kw = dict(batch=wl.batch, n_q_heads=wl.n_q_heads, n_kv_heads=wl.n_kv_heads, head_dim=wl.head_dim,
              rank=wl.rank, basis_groups=wl.basis_groups, n_sink=wl.n_sink, window=wl.window,
              q_window=wl.q_window, topk=wl.topk, pool_kernel=wl.pool_kernel, pool_mode=wl.pool_mode,
              group_agg=wl.group_agg, rope_theta=wl.rope_theta, dtype=wl.dtype, rank_v=wl.rank_v,
              capacity=capacity if capacity is not None else ((wl.L + 15) // 16) * 16)
    kw.update(over)
    return s4r.make_config(**kw)


def oracle_cfg(c, pool_mode="max", group_agg="mean"):
    return dict(n_kv_heads=c.n_kv_heads, window=c.window, topk=c.topk, pool_kernel=c.pool_kernel,
                pool_mode=pool_mode, group_agg=group_agg, rope_theta=float(np.float32(c.rope_theta)),
                dtype="bf16" if c.dtype == 1 else "fp32")


def dev(x, dtype, device="cuda"):
    return torch.from_numpy(np.ascontiguousarray(x)).to(device=device, dtype=dtype)


def to_gpu_state(c, st, device="cuda"):
    """Stored state (float64 numpy, rounded) -> GPU tensors; coefficient caches
    are uploaded row-major and packed into the tiled layout by the library.
    Latent axes are laid out in the library's storage width (a rank that is
    not a multiple of 32 gets zero columns up to the next multiple)."""
    dt = s4r.storage_dtype(c)
    rank_v = c.rank_v or c.rank
    g = {}
    for k in ("q", "sink_k", "sink_v"):
        if k in st and st[k] is not None:
            g[k] = dev(st[k], dt, device)
    for k, r in (("bases_k", c.rank), ("bases_v", rank_v)):
        if k in st and st[k] is not None:
            g[k] = dev(s4r.pad_latent(st[k], r), dt, device)
    for k, r in (("coef_k", c.rank), ("coef_v", rank_v)):
        rm = s4r.pad_latent(st[k], r, c.basis_groups)
        n = rm.shape[1]
        full = np.zeros((rm.shape[0], c.capacity, rm.shape[2]))
        full[:, :n] = rm
        ck = c if k == "coef_k" else s4r.value_config(c)       # the value cache has its own width
        g[k] = s4r.pack_coef(ck, c.capacity, dev(full, dt, device))
    if st.get("qwin_prev") is not None:
        g["qwin_prev"] = dev(s4r.pad_latent(st["qwin_prev"], c.rank, c.basis_groups), torch.float32, device)
    return g


def unpad_latent(x, rank, basis_groups=1):
    """The configured columns of latent data read back in the library's storage
    width (inverse of pad_latent); asserts the padding columns hold zeros
    (NaN rows, which the tests plant past a sequence's end, are left alone)."""
    x = np.asarray(x)
    rs = s4r.rank_stride(rank)
    if rs == rank:
        return x
    assert x.shape[-1] == rs * basis_groups
    parts = []
    for g in range(basis_groups):
        pad = x[..., g * rs + rank:(g + 1) * rs]
        assert np.all((pad == 0) | np.isnan(pad)), "padding columns are not zero"
        parts.append(x[..., g * rs:g * rs + rank])
    return np.concatenate(parts, axis=-1)


def rel_err_rows(gpu, ref):
    """max over rows of ||gpu - ref||_inf / ||ref||_inf (rows = last axis)."""
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    num = np.abs(gpu - ref).max(axis=-1)
    den = np.maximum(np.abs(ref).max(axis=-1), 1e-30)
    return float((num / den).max())


def check_selection(idx_gpu, idx_ref, a_ref, L, W, k, rel_tol=1e-6):
    """Index sets must be equal except for elements whose oracle score lies
    within rel_tol of the k-th largest score (near-ties); the window part must
    match exactly and each row must be strictly ascending per part.
    Returns the number of tolerated differences."""
    n_hist = max(L - W, 0)
    k_eff = min(k, n_hist)
    flips = 0
    for b in range(idx_ref.shape[0]):
        gi, ri = idx_gpu[b], idx_ref[b]
        assert np.array_equal(gi[k_eff:], ri[k_eff:]), "window part differs"
        g, r = gi[:k_eff], ri[:k_eff]
        assert np.all(np.diff(g) > 0), "global part not strictly ascending"
        assert np.all((g >= 0) & (g < n_hist))
        diff = np.setxor1d(g, r)
        if diff.size:
            srt = np.sort(a_ref[b, :n_hist])[::-1]
            kth = srt[k_eff - 1]
            gap = np.abs(a_ref[b, diff] - kth) / max(abs(kth), 1e-300)
            assert np.all(gap <= rel_tol), f"selection differs beyond ties: gaps {gap.max():.3e}"
            flips += diff.size // 2
    return flips


def slice_state(st, b, L_b):
    """Sequence b of a batch state, coefficient rows cut at L_b."""
    one = {}
    for key, x in st.items():
        if key == "needles" or x is None or not isinstance(x, np.ndarray):
            one[key] = x
            continue
        one[key] = x[b:b + 1]
    one["coef_k"], one["coef_v"] = st["coef_k"][b:b + 1, :L_b], st["coef_v"][b:b + 1, :L_b]
    return one


def latent_state_np(wl, seed=0, capacity=None, L=None):
    return W.latent_state(wl, seed=seed, capacity=capacity, L=L)


def score_tol(cq, coef_k, L, dtype):
    """Per-sequence bound on the relative error of the GPU's A~.

    The latent logits are summed by bf16 MFMAs whose 32-product blocks are
    added in fp32 (products exact, then folded into fp64 per block); the
    rounding inside a block is bounded by c * 2^-24 * sum_k |cq_k C_lk| (a
    gfx950 check of random and heavy-tailed blocks measured c <= 4.6; c = 8
    is used for bf16 storage, 16 for fp32 storage, whose coefficients take
    several part products).  An absolute logit error dz becomes a relative
    error dz of exp(z - M); the softmax sum adds at most the largest such
    error again; fp32 storage of the exp values and of A~ adds ~1e-6.
    cq: [B, G, W_q, R] query coefficients, coef_k: [B, >=L, R]."""
    c = 8.0 if dtype == "bf16" else 16.0
    B, R = cq.shape[0], cq.shape[-1]
    tol = np.empty(B)
    for b in range(B):
        s_abs = np.abs(cq[b].reshape(-1, R)) @ np.abs(coef_k[b, :L]).T
        tol[b] = 2.0 * c * 2.0 ** -24 * s_abs.max() / np.sqrt(R) + 1e-6
    return tol


def draw_random_workload(case, q_windows=(1, 1, 2, 3, 4), min_len=300, max_len=5000):
    """A seeded random configuration within the fused attention kernel's
    (G, rank) set (G in {1, 2, 4, 7, 8}, rank stride / 32 in 1..6 or 8, 7 for
    bf16 only): returns (workload, capacity, whether the step appends)."""
    rng = np.random.default_rng(1000 + case)
    dtype = "fp32" if rng.random() < 0.25 else "bf16"
    head_dim = 64 if rng.random() < 0.3 else 128
    G = int(rng.choice([1, 2, 4, 7, 8]))
    hkv = int(rng.choice([1, 2, 4, 8] if G <= 4 else [1, 2, 4]))
    nb = 2 if (hkv >= 2 and rng.random() < 0.3) else 1
    dg = hkv * head_dim // nb
    blocks = [b for b in (1, 2, 3, 4, 5, 6, 7, 8) if (b != 7 or dtype == "bf16") and 32 * b * nb <= 256
              and 32 * (b - 1) + 1 <= dg]
    b = int(rng.choice(blocks))
    rank = int(rng.integers(32 * (b - 1) + 1, min(32 * b, dg) + 1))
    batch = int(rng.integers(1, 4))
    L = int(rng.integers(min_len, max_len))
    n_sink = int(rng.choice([0, 2, 4]))
    window = int(rng.choice([0, 8, 32, 64]))
    q_window = int(rng.choice(q_windows))
    while G * q_window > 128:
        q_window -= 1
    topk = int(rng.integers(1, max(2, (L - window) // 3)))
    wl = W.CONFIGS["llama8b_32k"].scaled(
        name=f"random{case}", batch=batch, n_q_heads=G * hkv, n_kv_heads=hkv, head_dim=head_dim,
        N=L + n_sink, n_sink=n_sink, rank=rank, basis_groups=nb, window=window, topk=topk, dtype=dtype,
        r_true=max(4, (rank * nb * 3) // 4), q_window=q_window, pool_kernel=int(rng.choice([1, 3, 5, 7])),
        pool_mode=str(rng.choice(["max", "avg"])), group_agg=str(rng.choice(["mean", "max"])), n_needles=4,
        outlier_channels=0, recipe="latent")
    cap = ((L + 15) // 16) * 16 + 16 * int(rng.integers(0, 3))
    append = bool(rng.random() < 0.35)
    return wl, cap, append
