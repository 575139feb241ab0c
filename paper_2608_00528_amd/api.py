"""Python binding of the S^4R C ABI (include/s4r.h).

Thin marshalling only: every function checks tensor placement / dtype /
contiguity, allocates outputs with torch when the caller passes none, and
calls the library on torch's current HIP stream.  All arithmetic happens in
the gfx950 kernels of libs4r.so; there is no CPU path.
"""

import ctypes

import torch

from . import _lib as L

_DTYPES = {"bf16": (L.S4R_BF16, torch.bfloat16), "fp32": (L.S4R_FP32, torch.float32)}
_POOL = {"max": L.S4R_POOL_MAX, "avg": L.S4R_POOL_AVG}
_AGG = {"mean": L.S4R_AGG_MEAN, "max": L.S4R_AGG_MAX}


def make_config(*, batch, n_q_heads, n_kv_heads, head_dim, rank, capacity, basis_groups=1, n_sink=4,
                window=64, q_window=1, topk=1024, pool_kernel=7, pool_mode="max", group_agg="mean",
                bases_shared=False, rope_theta=0.0, dtype="bf16", rank_v=0):
    c = L.Config()
    c.batch, c.n_q_heads, c.n_kv_heads, c.head_dim = batch, n_q_heads, n_kv_heads, head_dim
    c.basis_groups, c.rank, c.n_sink, c.window = basis_groups, rank, n_sink, window
    c.q_window, c.topk, c.pool_kernel = q_window, topk, pool_kernel
    c.pool_mode, c.group_agg = _POOL[pool_mode], _AGG[group_agg]
    c.bases_shared = int(bool(bases_shared))
    c.capacity = capacity
    c.rope_theta = float(rope_theta)
    c.dtype = _DTYPES[dtype][0]
    c.rank_v = rank_v
    return c


def value_config(cfg):
    """The configuration whose `rank` is the value rank: the layout helpers
    (pack_coef / unpack_coef) take a cache's width from `rank`, so a value
    cache of an asymmetric configuration is converted with this one."""
    c = L.Config()
    ctypes.pointer(c)[0] = cfg
    if cfg.rank_v:
        c.rank, c.rank_v = cfg.rank_v, 0
    return c


def storage_dtype(cfg):
    return torch.bfloat16 if cfg.dtype == L.S4R_BF16 else torch.float32


def _ptr(t, name, dtype=None, required=True):
    if t is None:
        if required:
            raise ValueError(f"{name} is required")
        return None
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    return ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _cfgp(cfg):
    return ctypes.byref(cfg)


def version():
    return L.load().s4r_version().decode()


def workspace_size(cfg):
    n = ctypes.c_size_t()
    L.check(L.load().s4r_workspace_size(_cfgp(cfg), ctypes.byref(n)))
    return n.value


def alloc_workspace(cfg, device="cuda"):
    return torch.empty(workspace_size(cfg), dtype=torch.uint8, device=device)


def num_selected(cfg, length):
    m = L.load().s4r_num_selected(_cfgp(cfg), length)
    if m < 0:
        raise L.S4RError(L.S4R_ERR_BAD_SHAPE, L.load().s4r_last_error().decode())
    return m


def _G(cfg):
    return cfg.n_q_heads // cfg.n_kv_heads


def rank_stride(rank):
    """Storage width of a rank: the rank rounded up to a multiple of 32 (the
    coefficient layout works in 32-column blocks; the extra columns hold zeros)."""
    return (rank + 31) // 32 * 32


def _R(cfg):
    return rank_stride(cfg.rank) * cfg.basis_groups


def pad_latent(x, rank, basis_groups=1):
    """Lay latent data out in the library's storage width: the last axis of
    `x` holds basis_groups blocks of `rank` columns (bases: one block); each
    block moves to its own rank_stride(rank) columns, the padding columns zero.
    Works on torch tensors and numpy arrays; returns `x` itself when the rank
    is already a multiple of 32."""
    rs = rank_stride(rank)
    if rs == rank:
        return x
    if x.shape[-1] != rank * basis_groups:
        raise ValueError(f"last axis {x.shape[-1]} is not {basis_groups} x rank {rank}")
    shape = tuple(x.shape[:-1]) + (basis_groups * rs,)
    if isinstance(x, torch.Tensor):
        out = torch.zeros(shape, dtype=x.dtype, device=x.device)
    else:
        import numpy as np
        out = np.zeros(shape, dtype=x.dtype)
    for g in range(basis_groups):
        out[..., g * rs:g * rs + rank] = x[..., g * rank:(g + 1) * rank]
    return out


def score_latent(cfg, length, q, bases_k, coef_k, ws, qwin_prev=None, scores=None, qcoef=None):
    dt = storage_dtype(cfg)
    dev = q.device
    if scores is None:
        scores = torch.empty((cfg.batch, length), dtype=torch.float32, device=dev)
    L.check(L.load().s4r_score_latent(
        _cfgp(cfg), length, _ptr(q, "q", dt), _ptr(qwin_prev, "qwin_prev", torch.float32, False),
        _ptr(bases_k, "bases_k", dt), _ptr(coef_k, "coef_k", dt), _ptr(scores, "scores", torch.float32),
        _ptr(qcoef, "qcoef", torch.float32, False), _ptr(ws, "ws", torch.uint8), ws.numel(), _stream()))
    return scores


def select_topk(cfg, length, scores, ws, idx=None):
    if idx is None:
        idx = torch.empty((cfg.batch, num_selected(cfg, length)), dtype=torch.int32, device=scores.device)
    L.check(L.load().s4r_select_topk(_cfgp(cfg), length, _ptr(scores, "scores", torch.float32),
                                     _ptr(idx, "idx", torch.int32), _ptr(ws, "ws", torch.uint8), ws.numel(),
                                     _stream()))
    return idx


def reconstruct(cfg, length, idx, bases_k, bases_v, coef_k, coef_v, k_hat=None, v_hat=None):
    dt = storage_dtype(cfg)
    m = idx.shape[1]
    Dp = cfg.n_kv_heads * cfg.head_dim
    if k_hat is None:
        k_hat = torch.empty((cfg.batch, m, Dp), dtype=torch.float32, device=idx.device)
    if v_hat is None:
        v_hat = torch.empty((cfg.batch, m, Dp), dtype=torch.float32, device=idx.device)
    L.check(L.load().s4r_reconstruct(_cfgp(cfg), length, m, _ptr(idx, "idx", torch.int32),
                                     _ptr(bases_k, "bases_k", dt), _ptr(bases_v, "bases_v", dt),
                                     _ptr(coef_k, "coef_k", dt), _ptr(coef_v, "coef_v", dt),
                                     _ptr(k_hat, "k_hat", torch.float32), _ptr(v_hat, "v_hat", torch.float32),
                                     _stream()))
    return k_hat, v_hat


def sparse_attn(cfg, length, q, sink_k, sink_v, idx, k_sel, v_sel, ws, out=None):
    dt = storage_dtype(cfg)
    m = idx.shape[1] if idx is not None else 0
    if out is None:
        out = torch.empty((cfg.batch, cfg.n_q_heads, cfg.head_dim), dtype=torch.float32, device=q.device)
    need_sink = cfg.n_sink > 0
    L.check(L.load().s4r_sparse_attn(_cfgp(cfg), length, m, _ptr(q, "q", dt),
                                     _ptr(sink_k, "sink_k", dt, need_sink), _ptr(sink_v, "sink_v", dt, need_sink),
                                     _ptr(idx, "idx", torch.int32, m > 0), _ptr(k_sel, "k_sel", torch.float32, m > 0),
                                     _ptr(v_sel, "v_sel", torch.float32, m > 0), _ptr(out, "out", torch.float32),
                                     _ptr(ws, "ws", torch.uint8), ws.numel(), _stream()))
    return out


def decode_step(cfg, length, q, sink_k, sink_v, bases_k, bases_v, coef_k, coef_v, ws, qwin_prev=None,
                win_k=None, win_v=None, k_new=None, v_new=None, out=None, idx_out=None, scores_out=None):
    dt = storage_dtype(cfg)
    if out is None:
        out = torch.empty((cfg.batch, cfg.n_q_heads, cfg.head_dim), dtype=torch.float32, device=q.device)
    need_sink = cfg.n_sink > 0
    L.check(L.load().s4r_decode_step(
        _cfgp(cfg), length, _ptr(q, "q", dt), _ptr(qwin_prev, "qwin_prev", torch.float32, False),
        _ptr(sink_k, "sink_k", dt, need_sink), _ptr(sink_v, "sink_v", dt, need_sink),
        _ptr(win_k, "win_k", dt, False), _ptr(win_v, "win_v", dt, False),
        _ptr(bases_k, "bases_k", dt), _ptr(bases_v, "bases_v", dt), _ptr(coef_k, "coef_k", dt),
        _ptr(coef_v, "coef_v", dt), _ptr(k_new, "k_new", dt, False), _ptr(v_new, "v_new", dt, False),
        _ptr(out, "out", torch.float32), _ptr(idx_out, "idx_out", torch.int32, False),
        _ptr(scores_out, "scores_out", torch.float32, False), _ptr(ws, "ws", torch.uint8), ws.numel(),
        _stream()))
    return out


def window_state_size(cfg):
    """Bytes of the window state: [B, q_window, G, capacity] fp32 softmax rows,
    and for longer windows the older rows' running sum [2, B, G, capacity]
    fp64 after them."""
    n = ctypes.c_size_t()
    L.check(L.load().s4r_window_state_size(_cfgp(cfg), ctypes.byref(n)))
    return n.value


def alloc_window_state(cfg, device="cuda"):
    """A zeroed window state of window_state_size(cfg) bytes (fp32 elements)."""
    return torch.zeros((window_state_size(cfg) // 4,), dtype=torch.float32, device=device)


def window_state_init(cfg, length, qwin_prev, coef_k, state, ws):
    """Softmax rows of the window's q_window - 1 older queries (their
    coefficient rows qwin_prev [B, G, q_window - 1, R]) for a windowed step at
    `length`."""
    dt = storage_dtype(cfg)
    L.check(L.load().s4r_window_state_init(
        _cfgp(cfg), length, _ptr(qwin_prev, "qwin_prev", torch.float32), _ptr(coef_k, "coef_k", dt),
        _ptr(state, "state", torch.float32), _ptr(ws, "ws", torch.uint8), ws.numel(), _stream()))
    return state


def decode_step_windowed(cfg, length, q, state, sink_k, sink_v, bases_k, bases_v, coef_k, coef_v, ws,
                         win_k=None, win_v=None, k_new=None, v_new=None, out=None, idx_out=None, scores_out=None):
    """The fused step with the window state in place of qwin_prev (steps at
    consecutive lengths); the newest query row's softmax is stored in it."""
    dt = storage_dtype(cfg)
    if out is None:
        out = torch.empty((cfg.batch, cfg.n_q_heads, cfg.head_dim), dtype=torch.float32, device=q.device)
    need_sink = cfg.n_sink > 0
    L.check(L.load().s4r_decode_step_windowed(
        _cfgp(cfg), length, _ptr(q, "q", dt), _ptr(state, "state", torch.float32),
        _ptr(sink_k, "sink_k", dt, need_sink), _ptr(sink_v, "sink_v", dt, need_sink),
        _ptr(win_k, "win_k", dt, False), _ptr(win_v, "win_v", dt, False),
        _ptr(bases_k, "bases_k", dt), _ptr(bases_v, "bases_v", dt), _ptr(coef_k, "coef_k", dt),
        _ptr(coef_v, "coef_v", dt), _ptr(k_new, "k_new", dt, False), _ptr(v_new, "v_new", dt, False),
        _ptr(out, "out", torch.float32), _ptr(idx_out, "idx_out", torch.int32, False),
        _ptr(scores_out, "scores_out", torch.float32, False), _ptr(ws, "ws", torch.uint8), ws.numel(),
        _stream()))
    return out


def decode_step_noalloc(cfg, length, q, sink_k, sink_v, bases_k, bases_v, coef_k, coef_v, qwin_prev=None,
                        win_k=None, win_v=None, k_new=None, v_new=None, out=None, idx_out=None, scores_out=None):
    """The fused step on the library's own per-device scratch (no workspace
    argument); configurations needing more than 64 MiB of it are refused."""
    dt = storage_dtype(cfg)
    if out is None:
        out = torch.empty((cfg.batch, cfg.n_q_heads, cfg.head_dim), dtype=torch.float32, device=q.device)
    need_sink = cfg.n_sink > 0
    L.check(L.load().s4r_decode_step_noalloc(
        _cfgp(cfg), length, _ptr(q, "q", dt), _ptr(qwin_prev, "qwin_prev", torch.float32, False),
        _ptr(sink_k, "sink_k", dt, need_sink), _ptr(sink_v, "sink_v", dt, need_sink),
        _ptr(win_k, "win_k", dt, False), _ptr(win_v, "win_v", dt, False),
        _ptr(bases_k, "bases_k", dt), _ptr(bases_v, "bases_v", dt), _ptr(coef_k, "coef_k", dt),
        _ptr(coef_v, "coef_v", dt), _ptr(k_new, "k_new", dt, False), _ptr(v_new, "v_new", dt, False),
        _ptr(out, "out", torch.float32), _ptr(idx_out, "idx_out", torch.int32, False),
        _ptr(scores_out, "scores_out", torch.float32, False), _stream()))
    return out


def decode_step_ragged(cfg, lengths, q, sink_k, sink_v, bases_k, bases_v, coef_k, coef_v, ws, qwin_prev=None,
                       win_k=None, win_v=None, k_new=None, v_new=None, out=None, idx_out=None, scores_out=None):
    """The fused step over a ragged batch: lengths is a sequence of B ints
    (each sequence's L, the appended token included)."""
    dt = storage_dtype(cfg)
    if len(lengths) != cfg.batch:
        raise ValueError(f"lengths has {len(lengths)} entries for a batch of {cfg.batch}")
    lens = (ctypes.c_int64 * cfg.batch)(*[int(x) for x in lengths])
    if out is None:
        out = torch.empty((cfg.batch, cfg.n_q_heads, cfg.head_dim), dtype=torch.float32, device=q.device)
    need_sink = cfg.n_sink > 0
    L.check(L.load().s4r_decode_step_ragged(
        _cfgp(cfg), lens, _ptr(q, "q", dt), _ptr(qwin_prev, "qwin_prev", torch.float32, False),
        _ptr(sink_k, "sink_k", dt, need_sink), _ptr(sink_v, "sink_v", dt, need_sink),
        _ptr(win_k, "win_k", dt, False), _ptr(win_v, "win_v", dt, False),
        _ptr(bases_k, "bases_k", dt), _ptr(bases_v, "bases_v", dt), _ptr(coef_k, "coef_k", dt),
        _ptr(coef_v, "coef_v", dt), _ptr(k_new, "k_new", dt, False), _ptr(v_new, "v_new", dt, False),
        _ptr(out, "out", torch.float32), _ptr(idx_out, "idx_out", torch.int32, False),
        _ptr(scores_out, "scores_out", torch.float32, False), _ptr(ws, "ws", torch.uint8), ws.numel(),
        _stream()))
    return out


def project_queries(cfg, q_rows, bases_k, ws, out=None):
    """C^Q rows [B, G, n, R] fp32 of the queries q_rows [B, n, h_q, d_h] (the
    initial query window of the prefill: qwin_prev for n = W_q - 1)."""
    dt = storage_dtype(cfg)
    n = q_rows.shape[1]
    G = cfg.n_q_heads // cfg.n_kv_heads
    if out is None:
        out = torch.empty((cfg.batch, G, n, _R(cfg)), dtype=torch.float32, device=q_rows.device)
    L.check(L.load().s4r_project_queries(_cfgp(cfg), n, _ptr(q_rows, "q_rows", dt), _ptr(bases_k, "bases_k", dt),
                                         _ptr(out, "out", torch.float32), _ptr(ws, "ws", torch.uint8), ws.numel(),
                                         _stream()))
    return out


def prefill_bases(cfg, n_rows, s_k, s_v, eta=0.2, center=False, bases_k=None, bases_v=None, sample_idx=None,
                  ws=None):
    """Bases of a prompt's non-sink raw K/V rows [B, n_rows, Dp] (hybrid
    sample, token-wise normalisation, truncated SVD; Section 3.1.2).  Returns
    (bases_k, bases_v); sample_idx (int32, num_samples entries) receives the
    sampled positions when given."""
    dt = storage_dtype(cfg)
    lib = L.load()
    dg = cfg.n_kv_heads * cfg.head_dim // cfg.basis_groups
    shape = lambda r: (cfg.batch, cfg.basis_groups, dg, rank_stride(r))  # noqa: E731
    if bases_k is None:
        bases_k = torch.empty(shape(cfg.rank), dtype=dt, device=s_k.device)
    if bases_v is None:
        bases_v = torch.empty(shape(cfg.rank_v or cfg.rank), dtype=dt, device=s_k.device)
    if ws is None:
        ws = torch.empty(prefill_bases_workspace_size(cfg, n_rows, eta), dtype=torch.uint8, device=s_k.device)
    L.check(lib.s4r_prefill_bases(_cfgp(cfg), n_rows, _ptr(s_k, "s_k", dt), _ptr(s_v, "s_v", dt), float(eta),
                                  int(bool(center)), _ptr(bases_k, "bases_k", dt), _ptr(bases_v, "bases_v", dt),
                                  _ptr(sample_idx, "sample_idx", torch.int32, False), _ptr(ws, "ws", torch.uint8),
                                  ws.numel(), _stream()))
    return bases_k, bases_v


def prefill_bases_workspace_size(cfg, n_rows, eta=0.2):
    sz = ctypes.c_size_t()
    L.check(L.load().s4r_prefill_bases_workspace_size(_cfgp(cfg), n_rows, float(eta), ctypes.byref(sz)))
    return sz.value


def num_samples(n_rows, eta=0.2):
    return L.load().s4r_prefill_num_samples(n_rows, float(eta))


def prefill_project(cfg, n_rows, s_k, s_v, bases_k, bases_v, coef_k, coef_v, ws):
    """Bulk projection of a prompt's non-sink raw K/V rows [B, n_rows, Dp]
    into rows [0, n_rows) of the tiled coefficient caches (ws: the decode
    workspace)."""
    dt = storage_dtype(cfg)
    L.check(L.load().s4r_prefill_project(_cfgp(cfg), n_rows, _ptr(s_k, "s_k", dt), _ptr(s_v, "s_v", dt),
                                         _ptr(bases_k, "bases_k", dt), _ptr(bases_v, "bases_v", dt),
                                         _ptr(coef_k, "coef_k", dt), _ptr(coef_v, "coef_v", dt),
                                         _ptr(ws, "ws", torch.uint8), ws.numel(), _stream()))


def prefill(cfg, S_k, S_v, eta=0.2, center=False, ws=None):
    """The prefill stage of Section 3.1 on the GPU for a prompt's raw pre-RoPE
    keys / values S_k, S_v [B, N, Dp] (sinks first): the first n_sink rows
    kept as the sinks, the bases of the non-sink rows (s4r_prefill_bases:
    hybrid sample with ratio eta, token-wise normalisation, optional
    centring, truncated SVD) and their bulk projection into tiled coefficient
    caches of cfg.capacity rows (s4r_prefill_project).  Returns a dict of
    device tensors sink_k, sink_v, bases_k, bases_v, coef_k, coef_v."""
    s = cfg.n_sink
    n = S_k.shape[1] - s
    sink_k, sink_v = S_k[:, :s].contiguous(), S_v[:, :s].contiguous()
    X_k, X_v = S_k[:, s:].contiguous(), S_v[:, s:].contiguous()
    bases_k, bases_v = prefill_bases(cfg, n, X_k, X_v, eta=eta, center=center)
    dt = storage_dtype(cfg)
    coef_k = torch.zeros((cfg.batch, cfg.capacity, _R(cfg)), dtype=dt, device=S_k.device)
    coef_v = torch.zeros((cfg.batch, cfg.capacity, _R(value_config(cfg))), dtype=dt, device=S_k.device)
    if ws is None:
        ws = alloc_workspace(cfg, S_k.device)
    prefill_project(cfg, n, X_k, X_v, bases_k, bases_v, coef_k, coef_v, ws)
    return {"sink_k": sink_k, "sink_v": sink_v, "bases_k": bases_k, "bases_v": bases_v, "coef_k": coef_k,
            "coef_v": coef_v}


def full_recon_decode(cfg, length, q, sink_k, sink_v, bases_k, bases_v, coef_k, coef_v, ws, out=None):
    """Comparator (Appendix B.1): attention over the sinks and every one of
    the `length` tokens reconstructed from the coefficient caches."""
    dt = storage_dtype(cfg)
    if out is None:
        out = torch.empty((cfg.batch, cfg.n_q_heads, cfg.head_dim), dtype=torch.float32, device=q.device)
    need_sink = cfg.n_sink > 0
    L.check(L.load().s4r_full_recon_decode(
        _cfgp(cfg), length, _ptr(q, "q", dt), _ptr(sink_k, "sink_k", dt, need_sink),
        _ptr(sink_v, "sink_v", dt, need_sink), _ptr(bases_k, "bases_k", dt), _ptr(bases_v, "bases_v", dt),
        _ptr(coef_k, "coef_k", dt), _ptr(coef_v, "coef_v", dt), _ptr(out, "out", torch.float32),
        _ptr(ws, "ws", torch.uint8), ws.numel(), _stream()))
    return out


def dense_decode(cfg, n_tokens, q, k_cache, v_cache, ws, out=None):
    """Comparator: dense GQA decode over an uncompressed bf16 KV cache
    [B, capacity, Dp] (keys stored after RoPE) for tokens 0..n_tokens-1."""
    if out is None:
        out = torch.empty((cfg.batch, cfg.n_q_heads, cfg.head_dim), dtype=torch.float32, device=q.device)
    dt = storage_dtype(cfg)
    L.check(L.load().s4r_dense_decode(_cfgp(cfg), n_tokens, _ptr(q, "q", dt), _ptr(k_cache, "k_cache", dt),
                                      _ptr(v_cache, "v_cache", dt), _ptr(out, "out", torch.float32),
                                      _ptr(ws, "ws", torch.uint8), ws.numel(), _stream()))
    return out


def project_append(cfg, row, k_new, v_new, bases_k, bases_v, coef_k, coef_v):
    dt = storage_dtype(cfg)
    L.check(L.load().s4r_project_append(_cfgp(cfg), row, _ptr(k_new, "k_new", dt), _ptr(v_new, "v_new", dt),
                                        _ptr(bases_k, "bases_k", dt), _ptr(bases_v, "bases_v", dt),
                                        _ptr(coef_k, "coef_k", dt), _ptr(coef_v, "coef_v", dt), _stream()))


def pack_coef(cfg, n_rows, src, dst=None):
    dt = storage_dtype(cfg)
    if dst is None:
        dst = torch.zeros((cfg.batch, cfg.capacity, _R(cfg)), dtype=dt, device=src.device)
    L.check(L.load().s4r_pack_coef(_cfgp(cfg), n_rows, _ptr(src, "src", dt), _ptr(dst, "dst", dt), _stream()))
    return dst


def unpack_coef(cfg, n_rows, src, dst=None):
    dt = storage_dtype(cfg)
    if dst is None:
        dst = torch.empty((cfg.batch, n_rows, _R(cfg)), dtype=dt, device=src.device)
    L.check(L.load().s4r_unpack_coef(_cfgp(cfg), n_rows, _ptr(src, "src", dt), _ptr(dst, "dst", dt), _stream()))
    return dst


TIMED_KERNELS = ("prepare", "score_stream", "relevance", "select", "attn_split", "attn_combine")


def timing_enable(max_steps):
    L.check(L.load().s4r_timing_enable(max_steps))


def timing_read():
    """-> ({kernel name: summed ms}, timed steps)"""
    ms = (ctypes.c_double * len(TIMED_KERNELS))()
    n = ctypes.c_int64()
    L.check(L.load().s4r_timing_read(ms, ctypes.byref(n)))
    return dict(zip(TIMED_KERNELS, list(ms))), n.value


def read_bandwidth(buf, sink=None):
    """One read pass over the bytes of GPU tensor `buf` (roofline reference).
    Returns the per-thread XOR sink (uint32 viewed as int32)."""
    lib = L.load()
    if sink is None:
        sink = torch.empty(lib.s4r_read_bandwidth_sink_len(), dtype=torch.int32, device=buf.device)
    L.check(lib.s4r_read_bandwidth(_ptr(buf, "buf"), buf.numel() * buf.element_size(), _ptr(sink, "sink", torch.int32),
                                   _stream()))
    return sink
