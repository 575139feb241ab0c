"""Seeded synthetic workloads for the S^4R decode step.

This module only draws random numbers and lays them out in the shapes of the
paper's long-context workloads (Llama-3.1-8B and Qwen2.5-7B single layers at
32k/128k context, 4 sinks, ~5x compression).  It holds none of the method's
arithmetic: no projection onto a learned basis, no scoring, no selection.  It
is shared by the tests (which turn raw KV into stored state with the oracle's
prefill) and by the benchmark (which draws the stored state directly in latent
coordinates).  It imports neither the oracle nor the GPU package.

Two recipes
-----------
raw_kv(wl, seed)        raw pre-RoPE keys/values [B, N, Dp] and the query:
                        low-rank Gaussian (or Student-t) signal + noise, sinks
                        scaled x10, a few outlier key channels, needles planted
                        along the group-mean query direction.
latent_state(wl, seed)  the stored state directly: per-sequence random
                        orthonormal bases (QR of a Gaussian), coefficient rows
                        drawn as low-rank latent signal with a decaying
                        spectrum + noise, needles in latent coordinates, sinks
                        and a query that lies mostly in the key basis' span.

Seeds come from numpy.random.SeedSequence([workload id, layer, sequence,
stream tag]) so every sequence and every tensor has its own stream.
"""

import dataclasses

import numpy as np
import torch

# stream tags
_T_KEY, _T_VAL, _T_QRY, _T_NEEDLE, _T_SINK, _T_BASIS_K, _T_BASIS_V, _T_STEP, _T_QWIN = range(9)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    wid: int                 # numeric id used in seeds
    batch: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    N: int                   # context length including the sinks
    n_sink: int
    rank: int                # rank per basis group
    basis_groups: int
    window: int
    topk: int
    dtype: str               # "bf16" | "fp32"
    rope_theta: float
    r_true: int
    noise: float
    n_needles: int
    outlier_channels: int = 0
    outlier_scale: float = 1.0
    heavy_tail: bool = False
    q_window: int = 1
    pool_kernel: int = 7
    pool_mode: str = "max"
    group_agg: str = "mean"
    layers: int = 1
    steps: int = 1
    rank_v: int = 0          # value rank per basis group (Appendix D.2); 0 = rank
    recipe: str = "latent"   # how the benchmark draws the stored state: "latent" (latent_state) or
                             # "raw" (raw_kv_device, then the GPU prefill turns it into bases and caches)

    @property
    def G(self):
        return self.n_q_heads // self.n_kv_heads

    @property
    def Dp(self):
        return self.n_kv_heads * self.head_dim

    @property
    def R(self):
        return self.rank * self.basis_groups

    @property
    def rank_value(self):
        return self.rank_v or self.rank

    @property
    def R_v(self):
        return self.rank_value * self.basis_groups

    @property
    def L(self):
        return self.N - self.n_sink

    def scaled(self, **kw):
        return dataclasses.replace(self, **kw)

    def describe(self):
        return (f"{self.name}: B={self.batch} h_q={self.n_q_heads} h_kv={self.n_kv_heads} "
                f"d_h={self.head_dim} N={self.N} s={self.n_sink} r={self.R} W={self.window} "
                f"k={self.topk} {self.dtype}")


# The workloads: one tiny fp32 layer, Llama-3.1-8B-shaped layers at 32k and
# 128k, a Qwen2.5-7B-shaped layer at 128k, the 32-layer sustained run, and
# the paper's own operating points on a Qwen3-4B-shaped layer (32/8 heads,
# d_h = 128, D' = 1024) at a 120k context with reconstruction ratio 0.2, so
# k = floor(0.2 L) - W (Section 3.2.3), and rank 204 (Appendix B.4, the rank
# that the memory-ratio equation gives for eta = 0.2 at D' = 1024): the
# efficiency setting of Section 4.2 with the query window tied to the local
# window W = W_q = 4, and the default setting of Section 4 with W = W_q = 32.
CONFIGS = {
    "tiny_fp32": Workload("tiny_fp32", 1, batch=1, n_q_heads=8, n_kv_heads=2, head_dim=64,
                          N=4096, n_sink=4, rank=32, basis_groups=2, window=64, topk=128,
                          dtype="fp32", rope_theta=10000.0, r_true=24, noise=0.05, n_needles=5),
    "llama8b_32k": Workload("llama8b_32k", 2, batch=1, n_q_heads=32, n_kv_heads=8, head_dim=128,
                            N=32768, n_sink=4, rank=160, basis_groups=1, window=64, topk=1024,
                            dtype="bf16", rope_theta=500000.0, r_true=128, noise=0.05,
                            n_needles=32, outlier_channels=4, outlier_scale=8.0, recipe="raw"),
    "llama8b_128k": Workload("llama8b_128k", 3, batch=4, n_q_heads=32, n_kv_heads=8, head_dim=128,
                             N=131072, n_sink=4, rank=160, basis_groups=1, window=128, topk=2048,
                             dtype="bf16", rope_theta=500000.0, r_true=128, noise=0.05,
                             n_needles=32, outlier_channels=4, outlier_scale=8.0, recipe="raw"),
    "qwen7b_128k": Workload("qwen7b_128k", 4, batch=8, n_q_heads=28, n_kv_heads=4, head_dim=128,
                            N=131072, n_sink=4, rank=96, basis_groups=1, window=64, topk=1024,
                            dtype="bf16", rope_theta=1000000.0, r_true=80, noise=0.1,
                            n_needles=32, heavy_tail=True, recipe="raw"),
    "llama8b_32L_sustained": Workload("llama8b_32L_sustained", 5, batch=32, n_q_heads=32, n_kv_heads=8,
                                      head_dim=128, N=32768, n_sink=4, rank=160, basis_groups=1,
                                      window=64, topk=1024, dtype="bf16", rope_theta=500000.0,
                                      r_true=128, noise=0.05, n_needles=32, outlier_channels=4,
                                      outlier_scale=8.0, layers=32, steps=256),
    "qwen3_4b_120k": Workload("qwen3_4b_120k", 6, batch=1, n_q_heads=32, n_kv_heads=8, head_dim=128,
                              N=120_004, n_sink=4, rank=204, basis_groups=1, window=4,
                              topk=int(0.2 * 120_000) - 4, dtype="bf16", rope_theta=1000000.0, r_true=160,
                              noise=0.05, n_needles=32, q_window=4),
    "qwen3_4b_120k_w32": Workload("qwen3_4b_120k_w32", 7, batch=1, n_q_heads=32, n_kv_heads=8, head_dim=128,
                                  N=120_004, n_sink=4, rank=204, basis_groups=1, window=32,
                                  topk=int(0.2 * 120_000) - 32, dtype="bf16", rope_theta=1000000.0, r_true=160,
                                  noise=0.05, n_needles=32, q_window=32),
}

HEADLINE = "llama8b_128k"


def _rng(wl, seed, layer, seq, tag):
    return np.random.default_rng(np.random.SeedSequence([wl.wid, seed, layer, seq, tag]))


def round_storage(x, dtype):
    """Round float64 data to the storage format with torch's own casts
    (round to nearest even); returns float64 holding representable values."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float64)).to(torch.float32)
    if dtype == "bf16":
        t = t.to(torch.bfloat16).to(torch.float32)
    elif dtype != "fp32":
        raise ValueError(dtype)
    return t.to(torch.float64).numpy()


def _signal(rng, n, r_true, heavy):
    if heavy:
        return rng.standard_t(3.0, size=(n, r_true)) / np.sqrt(3.0)
    return rng.standard_normal((n, r_true))


def _needle_positions(rng, wl, count):
    hi = max(wl.L - wl.window, 1)
    count = min(count, hi)
    return np.sort(rng.choice(hi, size=count, replace=False))


def _query_heads(q_groups, wl):
    """[B, G, Dp] group queries -> [B, h_q, d_h] per-head queries (head j*G+g)."""
    B = q_groups.shape[0]
    return (q_groups.reshape(B, wl.G, wl.n_kv_heads, wl.head_dim)
            .transpose(0, 2, 1, 3).reshape(B, wl.n_q_heads, wl.head_dim))


def raw_kv(wl, seed=0, layer=0):
    """Raw prompt keys/values [B, N, Dp] and the query [B, h_q, d_h] (float64).

    Keys and values are F P / sqrt(r_true) + noise * E with a per-sequence
    mixing matrix P; the first n_sink rows are scaled x10; `outlier_channels`
    key channels are scaled by `outlier_scale`.  The group queries are 0.9 of
    a direction in P's row space plus 0.1 noise, scaled so latent logits have
    a standard deviation of about 1.5.  Needle keys (at positions in
    [0, L - W), non-sink numbering) get the kv-head slice of the mean group
    query direction added with a norm that lifts their logits well above the
    rest.
    """
    B, N, Dp = wl.batch, wl.N, wl.Dp
    S_k = np.empty((B, N, Dp))
    S_v = np.empty((B, N, Dp))
    qg = np.empty((B, wl.G, Dp))
    needles = []
    for b in range(B):
        rk, rv, rq = (_rng(wl, seed, layer, b, t) for t in (_T_KEY, _T_VAL, _T_QRY))
        Pk = rk.standard_normal((wl.r_true, Dp)) / np.sqrt(wl.r_true)
        Pv = rv.standard_normal((wl.r_true, Dp)) / np.sqrt(wl.r_true)
        S_k[b] = _signal(rk, N, wl.r_true, wl.heavy_tail) @ Pk + wl.noise * rk.standard_normal((N, Dp))
        S_v[b] = _signal(rv, N, wl.r_true, wl.heavy_tail) @ Pv + wl.noise * rv.standard_normal((N, Dp))
        if wl.outlier_channels:
            ch = rk.choice(Dp, size=wl.outlier_channels, replace=False)
            S_k[b, :, ch] *= wl.outlier_scale
        S_k[b, :wl.n_sink] *= 10.0
        S_v[b, :wl.n_sink] *= 10.0
        sig = rq.standard_normal((wl.G, wl.r_true)) @ Pk
        sig /= np.linalg.norm(sig, axis=-1, keepdims=True)
        noise = rq.standard_normal((wl.G, Dp))
        noise /= np.linalg.norm(noise, axis=-1, keepdims=True)
        qdir = 0.9 * sig + 0.1 * noise
        qdir /= np.linalg.norm(qdir, axis=-1, keepdims=True)
        qnorm = 1.5 * np.sqrt(wl.R) / (np.linalg.norm(S_k[b, wl.n_sink:], axis=-1).mean() / np.sqrt(wl.r_true))
        qg[b] = qdir * qnorm
        rn = _rng(wl, seed, layer, b, _T_NEEDLE)
        pos = _needle_positions(rn, wl, wl.n_needles)
        needles.append(pos)
        mean_dir = qdir.mean(axis=0)
        for p in pos:
            lift = (10.0 + 4.0 * rn.random()) * np.sqrt(wl.R) / qnorm
            for j in range(wl.n_kv_heads):
                sl = slice(j * wl.head_dim, (j + 1) * wl.head_dim)
                d = mean_dir[sl]
                S_k[b, wl.n_sink + p, sl] += lift * d / max(np.linalg.norm(mean_dir), 1e-12)
    q = round_storage(_query_heads(qg, wl), wl.dtype)
    return {"S_k": S_k, "S_v": S_v, "q": q, "needles": needles}


def _orthonormal(rng, rows, cols):
    a = rng.standard_normal((rows, cols))
    qm, rm = np.linalg.qr(a)
    return qm * np.sign(np.diag(rm))[None, :]


def latent_state(wl, seed=0, layer=0, capacity=None, L=None):
    """Stored decode state drawn directly (already rounded to wl.dtype).

    Returns float64 arrays:
      bases_k/v [B, nb, Dp/nb, rank] orthonormal columns per group,
      coef_k/v  [B, capacity, R] (rows >= L are zero),
      sink_k/v  [B, s, Dp], q [B, h_q, d_h], needles (positions per sequence),
      qwin_prev [B, G, W_q - 1, R] fp32 latent coefficients of the window's
                earlier queries (None when W_q = 1).
    Coefficient rows are F M + noise * E with F Gaussian (Student-t nu=3 when
    heavy_tail) and M a random mixing with a 1/(1 + i/16) column spectrum;
    row norms are about sqrt(Dp).  The query of group g is B^K u_g (+10%
    orthogonal noise) scaled for a latent-logit standard deviation of ~1.5.
    """
    B, Dp, R, nb = wl.batch, wl.Dp, wl.R, wl.basis_groups
    dg = Dp // nb
    L = wl.L if L is None else L
    cap = L if capacity is None else capacity
    out = {k: None for k in ("bases_k", "bases_v", "coef_k", "coef_v", "sink_k", "sink_v", "q", "qwin_prev")}
    bk = np.empty((B, nb, dg, wl.rank))
    bv = np.empty((B, nb, dg, wl.rank_value))
    Rv = wl.R_v
    ck = np.zeros((B, cap, R))
    cv = np.zeros((B, cap, Rv))
    sk = np.empty((B, wl.n_sink, Dp))
    sv = np.empty((B, wl.n_sink, Dp))
    qg = np.empty((B, wl.G, Dp))
    qwin = np.empty((B, wl.G, wl.q_window - 1, R))
    needles = []
    spectrum = 1.0 / (1.0 + np.arange(R) / 16.0)
    spectrum_v = 1.0 / (1.0 + np.arange(Rv) / 16.0)
    for b in range(B):
        rbk = _rng(wl, seed, layer, b, _T_BASIS_K)
        rbv = _rng(wl, seed, layer, b, _T_BASIS_V)
        for g in range(nb):
            bk[b, g] = _orthonormal(rbk, dg, wl.rank)
            bv[b, g] = _orthonormal(rbv, dg, wl.rank_value)
        rk, rv, rq, rs = (_rng(wl, seed, layer, b, t) for t in (_T_KEY, _T_VAL, _T_QRY, _T_SINK))
        scale = np.sqrt(Dp) / np.sqrt((spectrum ** 2).sum())
        scale_v = np.sqrt(Dp) / np.sqrt((spectrum_v ** 2).sum())
        Mk = rk.standard_normal((wl.r_true, R)) * spectrum / np.sqrt(wl.r_true) * scale
        Mv = rv.standard_normal((wl.r_true, Rv)) * spectrum_v / np.sqrt(wl.r_true) * scale_v
        ck[b, :L] = _signal(rk, L, wl.r_true, wl.heavy_tail) @ Mk + wl.noise * scale * rk.standard_normal((L, R)) * spectrum
        cv[b, :L] = (_signal(rv, L, wl.r_true, wl.heavy_tail) @ Mv
                     + wl.noise * scale_v * rv.standard_normal((L, Rv)) * spectrum_v)
        sk[b] = 10.0 * rs.standard_normal((wl.n_sink, Dp))
        sv[b] = 10.0 * rs.standard_normal((wl.n_sink, Dp))
        # query: latent direction u_g in the span of Mk's rows, mapped through B^K
        u = rq.standard_normal((wl.G, wl.r_true)) @ Mk
        u /= np.linalg.norm(u, axis=-1, keepdims=True)
        qlat = np.empty((wl.G, Dp))
        for g in range(nb):
            qlat[:, g * dg:(g + 1) * dg] = u[:, g * wl.rank:(g + 1) * wl.rank] @ bk[b, g].T
        qlat /= np.maximum(np.linalg.norm(qlat, axis=-1, keepdims=True), 1e-12)
        noise = rq.standard_normal((wl.G, Dp))
        noise /= np.linalg.norm(noise, axis=-1, keepdims=True)
        qdir = 0.9 * qlat + 0.1 * noise
        qdir /= np.linalg.norm(qdir, axis=-1, keepdims=True)
        # u is aligned with the high-variance latent directions, so the
        # component of a coefficient row along it is about 2 sqrt(Dp/r_true)
        qnorm = 1.5 * np.sqrt(R) / (2.0 * np.sqrt(Dp) / np.sqrt(wl.r_true))
        qg[b] = qdir * qnorm
        if wl.q_window > 1:
            # the earlier queries of the window, drawn directly as latent query
            # coefficients of the same scale (their own latent directions plus 10% noise)
            rw = _rng(wl, seed, layer, b, _T_QWIN)
            for i in range(wl.q_window - 1):
                uw = rw.standard_normal((wl.G, wl.r_true)) @ Mk
                uw /= np.linalg.norm(uw, axis=-1, keepdims=True)
                nw = rw.standard_normal((wl.G, R))
                nw /= np.linalg.norm(nw, axis=-1, keepdims=True)
                qwin[b, :, i] = (0.9 * uw + 0.1 * nw) * qnorm
        rn = _rng(wl, seed, layer, b, _T_NEEDLE)
        wl_eff = wl.scaled(N=L + wl.n_sink)
        pos = _needle_positions(rn, wl_eff, wl.n_needles)
        needles.append(pos)
        udir = u.mean(axis=0)
        udir /= max(np.linalg.norm(udir), 1e-12)
        for p in pos:
            lift = (10.0 + 4.0 * rn.random()) * np.sqrt(R) / qnorm
            ck[b, p] += lift * udir
    rnd = lambda a: round_storage(a, wl.dtype)  # noqa: E731
    out.update(bases_k=rnd(bk), bases_v=rnd(bv), coef_k=rnd(ck), coef_v=rnd(cv),
               sink_k=rnd(sk), sink_v=rnd(sv), q=rnd(_query_heads(qg, wl)), needles=needles,
               qwin_prev=round_storage(qwin, "fp32") if wl.q_window > 1 else None)
    return out


def step_inputs(wl, seed, layer, step, state=None):
    """Per-step inputs of the sustained run: a fresh query and the new token's
    raw key/value (drawn near the bases' span when a state is given)."""
    r = _rng(wl, seed, layer, step, _T_STEP)
    B, Dp = wl.batch, wl.Dp
    # group-query norm as in latent_state: 1.5 sqrt(R) sqrt(r_true) / sqrt(Dp)
    qnorm = 1.5 * np.sqrt(wl.R) * np.sqrt(wl.r_true) / np.sqrt(Dp)
    q = r.standard_normal((B, wl.n_q_heads, wl.head_dim)) * qnorm / np.sqrt(Dp)
    k_new = r.standard_normal((B, Dp))
    v_new = r.standard_normal((B, Dp))
    rnd = lambda a: round_storage(a, wl.dtype)  # noqa: E731
    return {"q": rnd(q), "k_new": rnd(k_new), "v_new": rnd(v_new)}


def _torch_seed(wl, seed, layer, tag):
    return int(np.random.SeedSequence([wl.wid, seed, layer, tag]).generate_state(1, dtype=np.uint64)[0] >> 1)


def sustained_layer(wl, seed, layer, L0, capacity, steps, device="cuda"):
    """One layer of the sustained multi-layer run, drawn on `device`.

    The stored state is drawn directly in latent coordinates (valid because
    the bases are orthonormal): coefficient rows F M + noise with F Gaussian
    [L0, r_true] and M a random mixing with a 1/(1 + i/16) column spectrum, row
    norms about sqrt(Dp), rows >= L0 zero; per-sequence orthonormal bases by a
    seeded float32 QR on the host; sinks 10x Gaussian.  Per step s (0-based)
    it draws a fresh query, Gaussian per head with a group norm of 1.5 sqrt(R)
    (latent logits of standard deviation about 1.5), and the new token's raw
    key/value, Gaussian.  Everything is rounded once to the storage type.

    Returns a dict of device tensors: bases_k/v [B, nb, Dp/nb, rank],
    coef_k/v row-major [B, capacity, R], sink_k/v [B, s, Dp], and per step
    q [steps, B, h_q, d_h], k_new/v_new [steps, B, Dp].
    """
    if wl.basis_groups != 1:
        raise ValueError("the sustained recipe draws one joint basis per sequence")
    B, Dp, R = wl.batch, wl.Dp, wl.R
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    gh = torch.Generator(device="cpu")
    out = {}
    for key, tag in (("bases_k", _T_BASIS_K), ("bases_v", _T_BASIS_V)):
        gh.manual_seed(_torch_seed(wl, seed, layer, tag))
        a = torch.randn((B, Dp, R), generator=gh, dtype=torch.float32)
        qm, rm = torch.linalg.qr(a)
        qm = qm * torch.sign(torch.diagonal(rm, dim1=-2, dim2=-1))[:, None, :]
        out[key] = qm.reshape(B, 1, Dp, R).to(device=device, dtype=dt).contiguous()
    gd = torch.Generator(device=device)
    spectrum = 1.0 / (1.0 + torch.arange(R, dtype=torch.float32, device=device) / 16.0)
    scale = float(np.sqrt(Dp) / np.sqrt(float((spectrum.double() ** 2).sum())))
    for key, tag in (("coef_k", _T_KEY), ("coef_v", _T_VAL)):
        gd.manual_seed(_torch_seed(wl, seed, layer, tag))
        mix = torch.randn((B, wl.r_true, R), generator=gd, device=device) * (spectrum * (scale / np.sqrt(wl.r_true)))
        c = torch.zeros((B, capacity, R), dtype=dt, device=device)
        for b in range(B):   # one sequence at a time bounds the float32 temporaries
            f = torch.randn((L0, wl.r_true), generator=gd, device=device)
            e = torch.randn((L0, R), generator=gd, device=device)
            c[b, :L0] = (torch.mm(f, mix[b].contiguous()) + e * (spectrum * (wl.noise * scale))).to(dt)
        out[key] = c
    gd.manual_seed(_torch_seed(wl, seed, layer, _T_SINK))
    out["sink_k"] = (10.0 * torch.randn((B, wl.n_sink, Dp), generator=gd, device=device)).to(dt)
    out["sink_v"] = (10.0 * torch.randn((B, wl.n_sink, Dp), generator=gd, device=device)).to(dt)
    gd.manual_seed(_torch_seed(wl, seed, layer, _T_STEP))
    q_std = 1.5 * np.sqrt(R) / np.sqrt(Dp)
    out["q"] = (q_std * torch.randn((steps, B, wl.n_q_heads, wl.head_dim), generator=gd, device=device)).to(dt)
    out["k_new"] = torch.randn((steps, B, Dp), generator=gd, device=device).to(dt)
    out["v_new"] = torch.randn((steps, B, Dp), generator=gd, device=device).to(dt)
    return out


def _student_t3(shape, gen, device):
    """Student-t samples with 3 degrees of freedom, scaled to unit variance:
    a Gaussian over the root of a chi-square(3) / 3 (three squared Gaussians)."""
    z = torch.randn(shape, generator=gen, device=device)
    chi = torch.randn((3,) + tuple(shape), generator=gen, device=device).pow(2).sum(0)
    return z / torch.sqrt(chi / 3.0) / np.sqrt(3.0)


def raw_kv_device(wl, seed=0, layer=0, device="cuda"):
    """The raw_kv recipe drawn on `device` with torch's generator (for the
    full-size workloads, whose float64 host copies would take gigabytes):
    raw pre-RoPE keys / values [B, N, Dp] = F P / sqrt(r_true) + noise * E
    with F Gaussian (Student-t nu = 3 when heavy_tail), `outlier_channels` key
    channels scaled by `outlier_scale`, sinks x10, and the group queries 0.9 of
    a direction in P's row space plus 0.1 noise, scaled for latent logits of
    standard deviation about 1.5; needle keys at seeded positions in
    [0, L - W) get the kv-head slices of the mean group-query direction added.
    Everything is rounded once to the storage dtype.  Returns a dict of device
    tensors S_k, S_v [B, N, Dp], q [B, h_q, d_h] and needles (host arrays)."""
    B, N, Dp = wl.batch, wl.N, wl.Dp
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    S_k = torch.empty((B, N, Dp), dtype=dt, device=device)
    S_v = torch.empty((B, N, Dp), dtype=dt, device=device)
    qg = torch.empty((B, wl.G, Dp), dtype=torch.float32, device=device)
    needles = []
    g = torch.Generator(device=device)
    for b in range(B):
        g.manual_seed(_torch_seed(wl, seed, layer, 1000 * b + _T_KEY))
        Pk = torch.randn((wl.r_true, Dp), generator=g, device=device) / np.sqrt(wl.r_true)
        Pv = torch.randn((wl.r_true, Dp), generator=g, device=device) / np.sqrt(wl.r_true)
        sig = (lambda n: _student_t3((n, wl.r_true), g, device)) if wl.heavy_tail else \
            (lambda n: torch.randn((n, wl.r_true), generator=g, device=device))
        sk = torch.mm(sig(N), Pk) + wl.noise * torch.randn((N, Dp), generator=g, device=device)
        sv = torch.mm(sig(N), Pv) + wl.noise * torch.randn((N, Dp), generator=g, device=device)
        if wl.outlier_channels:
            ch = torch.randperm(Dp, generator=g, device=device)[:wl.outlier_channels]
            sk[:, ch] *= wl.outlier_scale
        sk[:wl.n_sink] *= 10.0
        sv[:wl.n_sink] *= 10.0
        sq = torch.mm(torch.randn((wl.G, wl.r_true), generator=g, device=device), Pk)
        sq /= sq.norm(dim=-1, keepdim=True)
        nq = torch.randn((wl.G, Dp), generator=g, device=device)
        nq /= nq.norm(dim=-1, keepdim=True)
        qdir = 0.9 * sq + 0.1 * nq
        qdir /= qdir.norm(dim=-1, keepdim=True)
        qnorm = 1.5 * np.sqrt(wl.R) / (float(sk[wl.n_sink:].norm(dim=-1).mean()) / np.sqrt(wl.r_true))
        qg[b] = qdir * qnorm
        hi = max(wl.L - wl.window, 1)
        count = min(wl.n_needles, hi)
        pos = torch.sort(torch.randperm(hi, generator=g, device=device)[:count]).values
        lift = (10.0 + 4.0 * torch.rand((count,), generator=g, device=device)) * (np.sqrt(wl.R) / qnorm)
        mean_dir = qdir.mean(dim=0)
        md = mean_dir / torch.clamp(mean_dir.norm(), min=1e-12)
        sk[wl.n_sink + pos] += lift[:, None] * md[None, :]
        needles.append(pos.cpu().numpy())
        S_k[b] = sk.to(dt)
        S_v[b] = sv.to(dt)
        del sk, sv
    q = (qg.reshape(B, wl.G, wl.n_kv_heads, wl.head_dim).transpose(1, 2)
         .reshape(B, wl.n_q_heads, wl.head_dim).to(dt).contiguous())
    return {"S_k": S_k, "S_v": S_v, "q": q, "needles": needles}


def dense_cache(wl, seed=0, device="cuda", n_tokens=None):
    """An uncompressed KV cache of the workload's shape for the dense
    comparator, drawn on `device`: keys and values [B, N, Dp] Gaussian (keys
    taken as already stored after RoPE: a random vector is as good a rotated
    key as any), a Gaussian query [B, h_q, d_h] with logits of standard
    deviation about 1.5, everything rounded once to bf16."""
    N = wl.N if n_tokens is None else n_tokens
    g = torch.Generator(device=device)
    g.manual_seed(_torch_seed(wl, seed, 0, _T_KEY))
    k = torch.randn((wl.batch, N, wl.Dp), generator=g, device=device).to(torch.bfloat16)
    g.manual_seed(_torch_seed(wl, seed, 0, _T_VAL))
    v = torch.randn((wl.batch, N, wl.Dp), generator=g, device=device).to(torch.bfloat16)
    g.manual_seed(_torch_seed(wl, seed, 0, _T_QRY))
    q = (1.5 * torch.randn((wl.batch, wl.n_q_heads, wl.head_dim), generator=g, device=device)).to(torch.bfloat16)
    return {"k": k, "v": v, "q": q}
