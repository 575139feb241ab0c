"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every function include/s4r.h declares, computes sizes, and rejects invalid
arguments with the documented status codes before launching anything.

Every call with a non-NULL fake pointer here is built to fail validation, so
nothing is ever launched with it."""

import ctypes
import os
import re

import pytest
import torch

import paper_2608_00528_amd as s4r
from paper_2608_00528_amd import _lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "s4r.h")
# fake pointers are only ever passed where validation must reject the call;
# skip on GPU machines anyway so no fake pointer can reach a kernel there
pytestmark = pytest.mark.skipif(torch.cuda.is_available(), reason="host-only checks")

FAKE = ctypes.c_void_p(0x10000)        # aligned, never dereferenced
FAKE_MIS = ctypes.c_void_p(0x10004)    # misaligned


def header_functions():
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:s4r_status|int32_t|int64_t|const char\*)\s+(s4r_\w+)\s*\(", txt, re.M)))


def cfg(**kw):
    base = dict(batch=2, n_q_heads=8, n_kv_heads=2, head_dim=64, rank=32, capacity=1024, window=16, topk=32,
                rope_theta=10000.0, dtype="bf16")
    base.update(kw)
    return s4r.make_config(**base)


def test_exports_match_header():
    lib = L.load()
    funcs = header_functions()
    assert len(funcs) == len(L.EXPORTS)
    assert sorted(L.EXPORTS) == funcs
    for f in funcs:
        assert hasattr(lib, f)


def test_config_struct_layout():
    assert ctypes.sizeof(L.Config) == 80
    assert L.Config.capacity.offset == 56 and L.Config.dtype.offset == 68 and L.Config.rank_v.offset == 72


def test_version_and_sizes():
    assert s4r.version().startswith("s4r-gfx950")
    c = cfg()
    ws = s4r.workspace_size(c)
    assert ws > 0 and ws % 256 == 0
    assert s4r.num_selected(c, 1000) == 32 + 16
    assert s4r.num_selected(c, 20) == 4 + 16
    assert s4r.num_selected(c, 10) == 0 + 10
    # workspace grows with capacity
    assert s4r.workspace_size(cfg(capacity=4096)) > ws


@pytest.mark.parametrize("field,value,status", [
    ("batch", 0, L.S4R_ERR_BAD_SHAPE),
    ("n_q_heads", 7, L.S4R_ERR_BAD_SHAPE),
    ("head_dim", 96, L.S4R_ERR_UNSUPPORTED),
    ("basis_groups", 3, L.S4R_ERR_BAD_SHAPE),
    ("rank", 0, L.S4R_ERR_BAD_SHAPE),
    ("rank", 4096, L.S4R_ERR_BAD_SHAPE),
    ("pool_kernel", 4, L.S4R_ERR_BAD_SHAPE),
    ("pool_kernel", 0, L.S4R_ERR_BAD_SHAPE),
    ("q_window", 0, L.S4R_ERR_BAD_SHAPE),
    ("q_window", 33, L.S4R_ERR_UNSUPPORTED),     # G * W_q = 132 > 128
    ("n_q_heads", 34, L.S4R_ERR_UNSUPPORTED),    # G = 17 > 16
    ("capacity", 1000, L.S4R_ERR_BAD_SHAPE),
    ("dtype", 7, L.S4R_ERR_BAD_SHAPE),
    ("topk", -1, L.S4R_ERR_BAD_SHAPE),
    ("window", -1, L.S4R_ERR_BAD_SHAPE),
    ("n_sink", -1, L.S4R_ERR_BAD_SHAPE),
    ("pool_mode", 5, L.S4R_ERR_BAD_SHAPE),
])
def test_config_validation(field, value, status):
    c = cfg()
    setattr(c, field, value)
    n = ctypes.c_size_t()
    st = L.load().s4r_workspace_size(ctypes.byref(c), ctypes.byref(n))
    assert st == status
    assert L.load().s4r_last_error().decode()


@pytest.mark.parametrize("rank_v,status", [(16, L.S4R_OK), (-32, L.S4R_ERR_BAD_SHAPE),
                                           (160, L.S4R_ERR_BAD_SHAPE)])
def test_value_rank_validation(rank_v, status):
    """rank_v: 0 (= rank) or a rank within Dp / basis_groups = 128 (stored
    with its own stride of 32 * ceil(rank_v / 32) columns)."""
    lib = L.load()
    sz = ctypes.c_size_t()
    assert lib.s4r_workspace_size(ctypes.byref(cfg(rank_v=rank_v)), ctypes.byref(sz)) == status
    assert lib.s4r_workspace_size(ctypes.byref(cfg(rank_v=96)), ctypes.byref(sz)) == L.S4R_OK


def test_asymmetric_ranks_support():
    """Asymmetric ranks run on the bf16 matrix-core path for the listed pairs;
    other settings are refused before any launch."""
    lib = L.load()

    def step(c):
        return lib.s4r_decode_step(ctypes.byref(c), 100, FAKE, None, FAKE, FAKE, None, None, FAKE, FAKE, FAKE,
                                   FAKE, None, None, FAKE, None, None, FAKE, 0, None)
    assert step(cfg(rank=32, rank_v=96)) == L.S4R_ERR_UNSUPPORTED             # pair (32, 96) not built
    assert step(cfg(rank=64, rank_v=96, dtype="fp32")) == L.S4R_ERR_UNSUPPORTED
    assert step(cfg(head_dim=128, rank=96, rank_v=160)) == L.S4R_ERR_WORKSPACE  # built: fails on ws only
    assert lib.s4r_reconstruct(ctypes.byref(cfg(head_dim=128, rank=96, rank_v=160)), 100, 4, FAKE, FAKE, FAKE,
                               FAKE, FAKE, FAKE, FAKE, None) == L.S4R_ERR_UNSUPPORTED
    assert lib.s4r_prefill_project(ctypes.byref(cfg(head_dim=128, rank=96, rank_v=160)), 100, FAKE, FAKE, FAKE,
                                   FAKE, FAKE, FAKE, FAKE, 1 << 40, None) == L.S4R_ERR_UNSUPPORTED


def test_null_config():
    n = ctypes.c_size_t()
    assert L.load().s4r_workspace_size(None, ctypes.byref(n)) == L.S4R_ERR_NULL_ARG


def _score(c, Lval, q=FAKE, qwin=None, bk=FAKE, ck=FAKE, sc=FAKE, qo=None, ws=FAKE, wsb=1 << 40):
    return L.load().s4r_score_latent(ctypes.byref(c), Lval, q, qwin, bk, ck, sc, qo, ws, wsb, None)


def test_score_latent_argument_errors():
    c = cfg()
    assert _score(c, 0) == L.S4R_ERR_BAD_SHAPE                  # L < 1
    assert _score(c, 2048) == L.S4R_ERR_BAD_SHAPE               # L > capacity
    assert _score(c, 100, q=None) == L.S4R_ERR_NULL_ARG
    assert _score(c, 100, ck=FAKE_MIS) == L.S4R_ERR_MISALIGNED
    assert _score(c, 100, ws=None) == L.S4R_ERR_NULL_ARG
    assert _score(c, 100, wsb=16) == L.S4R_ERR_WORKSPACE
    assert _score(c, 100, ws=ctypes.c_void_p(0x10010)) == L.S4R_ERR_MISALIGNED   # ws needs 256 B
    assert _score(c, 100, qwin=FAKE) == L.S4R_ERR_BAD_SHAPE     # qwin_prev with W_q == 1
    c2 = cfg(q_window=2)
    assert _score(c2, 100) == L.S4R_ERR_NULL_ARG                 # qwin_prev missing
    assert _score(c2, 1, qwin=FAKE) == L.S4R_ERR_BAD_SHAPE       # W_q > L


def test_decode_step_argument_errors():
    c = cfg()
    lib = L.load()

    def call(Lval=100, k_new=None, v_new=None, win_k=None, win_v=None, sink=FAKE, out=FAKE, wsb=1 << 40, c=c):
        return lib.s4r_decode_step(ctypes.byref(c), Lval, FAKE, None, sink, sink, win_k, win_v, FAKE, FAKE, FAKE,
                                   FAKE, k_new, v_new, out, None, None, FAKE, wsb, None)
    assert call(k_new=FAKE) == L.S4R_ERR_NULL_ARG               # k_new without v_new
    assert call(win_v=FAKE) == L.S4R_ERR_NULL_ARG               # win_v without win_k
    assert call(sink=None) == L.S4R_ERR_NULL_ARG                # sinks required when s > 0
    assert call(out=None) == L.S4R_ERR_NULL_ARG
    assert call(wsb=0) == L.S4R_ERR_WORKSPACE
    assert call(Lval=0) == L.S4R_ERR_BAD_SHAPE
    c3 = cfg(n_q_heads=6, n_kv_heads=2)                          # G = 3: no fused kernel built
    assert call(c=c3) == L.S4R_ERR_UNSUPPORTED
    c0 = cfg(n_sink=0, window=0, topk=0)                         # nothing to attend to
    assert call(c=c0, sink=None) == L.S4R_ERR_BAD_SHAPE


def test_window_state_entry_points():
    """Window state: its size is B * q_window * G * capacity floats (plus the
    running sum's 2 * B * G * capacity doubles above five rows); every
    entry point refuses q_window = 1 and missing or misaligned buffers before
    launching anything, and the windowed step never takes qwin_prev."""
    lib = L.load()
    c1 = cfg()
    cw = cfg(q_window=4)
    n = ctypes.c_size_t()
    assert lib.s4r_window_state_size(ctypes.byref(c1), ctypes.byref(n)) == L.S4R_ERR_BAD_SHAPE
    assert lib.s4r_window_state_size(ctypes.byref(cw), None) == L.S4R_ERR_NULL_ARG
    assert s4r.window_state_size(cw) == 2 * 4 * 4 * 1024 * 4
    # longer windows add the older rows' fp64 running sum in two buffers
    assert s4r.window_state_size(cfg(q_window=5)) == 2 * 5 * 4 * 1024 * 4
    assert s4r.window_state_size(cfg(q_window=6)) == 2 * 6 * 4 * 1024 * 4 + 2 * 2 * 4 * 1024 * 8
    assert lib.s4r_window_state_init(ctypes.byref(c1), 100, FAKE, FAKE, FAKE, FAKE, 1 << 40, None) == L.S4R_ERR_BAD_SHAPE
    assert lib.s4r_window_state_init(ctypes.byref(cw), 100, None, FAKE, FAKE, FAKE, 1 << 40, None) == L.S4R_ERR_NULL_ARG
    assert lib.s4r_window_state_init(ctypes.byref(cw), 100, FAKE, FAKE, None, FAKE, 1 << 40, None) == L.S4R_ERR_NULL_ARG
    assert lib.s4r_window_state_init(ctypes.byref(cw), 100, FAKE, FAKE, FAKE_MIS, FAKE, 1 << 40, None) == \
        L.S4R_ERR_MISALIGNED
    assert lib.s4r_window_state_init(ctypes.byref(cw), 3, FAKE, FAKE, FAKE, FAKE, 1 << 40, None) == L.S4R_ERR_BAD_SHAPE
    assert lib.s4r_window_state_init(ctypes.byref(cw), 100, FAKE, FAKE, FAKE, FAKE, 0, None) == L.S4R_ERR_WORKSPACE

    def step(c=cw, state=FAKE, Lval=100, wsb=1 << 40):
        return lib.s4r_decode_step_windowed(ctypes.byref(c), Lval, FAKE, state, FAKE, FAKE, None, None, FAKE, FAKE,
                                            FAKE, FAKE, None, None, FAKE, None, None, FAKE, wsb, None)
    assert step(state=None) == L.S4R_ERR_NULL_ARG
    assert step(state=FAKE_MIS) == L.S4R_ERR_MISALIGNED
    assert step(c=c1) == L.S4R_ERR_BAD_SHAPE                    # q_window 1: nothing to keep
    assert step(Lval=2) == L.S4R_ERR_BAD_SHAPE                  # fewer keys than window rows
    assert step(wsb=0) == L.S4R_ERR_WORKSPACE


def test_ragged_decode_step_argument_errors():
    lib = L.load()

    def call(lens, c=None, out=FAKE, wsb=1 << 40):
        c = c or cfg()
        arr = None if lens is None else (ctypes.c_int64 * len(lens))(*lens)
        return lib.s4r_decode_step_ragged(ctypes.byref(c), arr, FAKE, None, FAKE, FAKE, None, None, FAKE, FAKE,
                                          FAKE, FAKE, None, None, out, None, None, FAKE, wsb, None)
    assert call(None) == L.S4R_ERR_NULL_ARG                      # no lengths
    assert call([100, 0]) == L.S4R_ERR_BAD_SHAPE                 # a length below 1
    assert call([100, 1025]) == L.S4R_ERR_BAD_SHAPE              # a length past the capacity
    # window 16 + topk 32: a sequence of 40 selects 40, one of 100 selects 48
    assert call([100, 40]) == L.S4R_ERR_BAD_SHAPE
    assert call([100, 48], wsb=0) == L.S4R_ERR_WORKSPACE         # equal counts pass on to the workspace check
    assert call([100, 48], out=None) == L.S4R_ERR_NULL_ARG
    c65 = cfg(batch=65)
    assert call([100] * 65, c=c65) == L.S4R_ERR_UNSUPPORTED      # more sequences than the length table holds


def test_other_entry_point_errors():
    c = cfg()
    lib = L.load()
    assert lib.s4r_select_topk(ctypes.byref(c), 100, None, FAKE, FAKE, 1 << 40, None) == L.S4R_ERR_NULL_ARG
    assert lib.s4r_select_topk(ctypes.byref(c), 5000, FAKE, FAKE, FAKE, 1 << 40, None) == L.S4R_ERR_BAD_SHAPE
    assert lib.s4r_reconstruct(ctypes.byref(c), 100, -1, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == L.S4R_ERR_BAD_SHAPE
    assert lib.s4r_reconstruct(ctypes.byref(c), 100, 0, None, None, None, None, None, None, None, None) == L.S4R_OK
    assert lib.s4r_reconstruct(ctypes.byref(c), 100, 8, FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, None) == L.S4R_ERR_NULL_ARG
    big = s4r.num_selected(c, 1024) + 1
    assert lib.s4r_sparse_attn(ctypes.byref(c), 100, big, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 40,
                               None) == L.S4R_ERR_BAD_SHAPE
    assert lib.s4r_project_append(ctypes.byref(c), 1024, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == L.S4R_ERR_BAD_SHAPE
    assert lib.s4r_project_append(ctypes.byref(c), 3, None, FAKE, FAKE, FAKE, FAKE, FAKE, None) == L.S4R_ERR_NULL_ARG
    assert lib.s4r_pack_coef(ctypes.byref(c), 2048, FAKE, FAKE, None) == L.S4R_ERR_BAD_SHAPE
    assert lib.s4r_unpack_coef(ctypes.byref(c), 10, FAKE_MIS, FAKE, None) == L.S4R_ERR_MISALIGNED
    assert lib.s4r_timing_enable(0) == L.S4R_ERR_BAD_SHAPE
    assert lib.s4r_timing_read(None, None) == L.S4R_ERR_NULL_ARG
    assert s4r.num_selected.__module__   # binding importable
    assert lib.s4r_num_selected(ctypes.byref(c), 0) == -1
    assert lib.s4r_read_bandwidth(FAKE, 100, FAKE, None) == L.S4R_ERR_BAD_SHAPE      # not a multiple of 16
    assert lib.s4r_read_bandwidth(None, 64, FAKE, None) == L.S4R_ERR_NULL_ARG
    assert lib.s4r_read_bandwidth_sink_len() > 0


def test_dense_comparator_argument_errors():
    lib = L.load()

    def call(c, n=100, q=FAKE, k=FAKE, v=FAKE, out=FAKE, ws=FAKE, wsb=1 << 40):
        return lib.s4r_dense_decode(ctypes.byref(c), n, q, k, v, out, ws, wsb, None)
    c = cfg(head_dim=128)
    assert call(c, n=0) == L.S4R_ERR_BAD_SHAPE                      # N < 1
    assert call(c, n=1025) == L.S4R_ERR_BAD_SHAPE                   # N > capacity
    assert call(c, k=None) == L.S4R_ERR_NULL_ARG
    assert call(c, v=FAKE_MIS) == L.S4R_ERR_MISALIGNED
    assert call(c, wsb=16) == L.S4R_ERR_WORKSPACE
    assert call(cfg()) == L.S4R_ERR_UNSUPPORTED                     # head_dim 64
    assert call(cfg(head_dim=128, dtype="fp32")) == L.S4R_ERR_UNSUPPORTED
    assert call(cfg(head_dim=128, n_q_heads=32, n_kv_heads=2)) == L.S4R_ERR_UNSUPPORTED   # G = 16


def test_full_recon_argument_errors():
    lib = L.load()

    def call(c, n=100, q=FAKE, ck=FAKE, sink=FAKE, out=FAKE, wsb=1 << 40):
        return lib.s4r_full_recon_decode(ctypes.byref(c), n, q, sink, sink, FAKE, FAKE, ck, FAKE, out, FAKE, wsb,
                                         None)
    c = cfg()
    assert call(c, n=0) == L.S4R_ERR_BAD_SHAPE
    assert call(c, n=1025) == L.S4R_ERR_BAD_SHAPE
    assert call(c, q=None) == L.S4R_ERR_NULL_ARG
    assert call(c, sink=None) == L.S4R_ERR_NULL_ARG               # sinks required when s > 0
    assert call(c, out=None) == L.S4R_ERR_NULL_ARG
    assert call(c, ck=FAKE_MIS) == L.S4R_ERR_MISALIGNED
    assert call(c, wsb=16) == L.S4R_ERR_WORKSPACE
    assert call(cfg(dtype="fp32")) == L.S4R_ERR_UNSUPPORTED
    assert call(cfg(n_q_heads=6, n_kv_heads=2)) == L.S4R_ERR_UNSUPPORTED     # G = 3
    assert call(cfg(head_dim=32)) == L.S4R_ERR_UNSUPPORTED


def test_project_queries_argument_errors():
    lib = L.load()

    def call(n=3, q=FAKE, out=FAKE, wsb=1 << 40):
        return lib.s4r_project_queries(ctypes.byref(cfg()), n, q, FAKE, out, FAKE, wsb, None)
    assert call(n=0) == L.S4R_ERR_BAD_SHAPE
    assert call(n=5000) == L.S4R_ERR_BAD_SHAPE
    assert call(q=None) == L.S4R_ERR_NULL_ARG
    assert call(out=FAKE_MIS) == L.S4R_ERR_MISALIGNED
    assert call(wsb=16) == L.S4R_ERR_WORKSPACE


def test_prefill_sample_counts_match_oracle():
    """The library's sample count is the length of the oracle's hybrid sample
    (Section 3.1.2) for lengths and ratios around every rounding case."""
    from oracle import prefill
    lib = L.load()
    for T in (1, 2, 3, 7, 10, 15, 16, 100, 101, 999, 3000, 4096, 120000):
        for eta in (0.01, 0.05, 0.1, 0.2, 0.25, 0.5, 0.75, 1.0):
            assert lib.s4r_prefill_num_samples(T, eta) == len(prefill.sample_hybrid(T, eta)), (T, eta)
    assert lib.s4r_prefill_num_samples(0, 0.2) == -1
    assert lib.s4r_prefill_num_samples(100, 0.0) == -1


def test_prefill_bases_argument_errors():
    lib = L.load()

    def call(c, n=1000, eta=0.2, s=FAKE, center=0):
        return lib.s4r_prefill_bases(ctypes.byref(c), n, s, FAKE, eta, center, FAKE, FAKE, None, FAKE, 1 << 40, None)
    c = cfg(head_dim=128)                                                  # Dg = 256
    assert call(cfg(head_dim=128, dtype="fp32")) == L.S4R_ERR_UNSUPPORTED
    assert call(cfg(head_dim=128, bases_shared=True)) == L.S4R_ERR_BAD_SHAPE
    assert call(cfg(head_dim=64)) == L.S4R_ERR_UNSUPPORTED                 # Dg = 128
    assert call(c, n=0) == L.S4R_ERR_BAD_SHAPE
    assert call(c, eta=0.0) == L.S4R_ERR_BAD_SHAPE
    assert call(c, eta=1.5) == L.S4R_ERR_BAD_SHAPE
    assert call(c, n=100) == L.S4R_ERR_BAD_SHAPE                           # 20 samples < rank 32
    sz = ctypes.c_size_t()
    assert lib.s4r_prefill_bases_workspace_size(ctypes.byref(c), 100, 0.2, ctypes.byref(sz)) == L.S4R_ERR_BAD_SHAPE


def test_prefill_projection_argument_errors():
    lib = L.load()

    def call(c, n=100, s=FAKE, cv=FAKE, wsb=1 << 40):
        return lib.s4r_prefill_project(ctypes.byref(c), n, s, FAKE, FAKE, FAKE, FAKE, cv, FAKE, wsb, None)
    c = cfg()
    assert call(c, n=0) == L.S4R_ERR_BAD_SHAPE
    assert call(c, n=1025) == L.S4R_ERR_BAD_SHAPE
    assert call(c, s=None) == L.S4R_ERR_NULL_ARG
    assert call(c, cv=FAKE_MIS) == L.S4R_ERR_MISALIGNED
    assert call(c, wsb=16) == L.S4R_ERR_WORKSPACE
    assert call(cfg(dtype="fp32")) == L.S4R_ERR_UNSUPPORTED
    assert call(cfg(head_dim=128, rank=256)) == L.S4R_ERR_UNSUPPORTED      # rank > 192


def test_noalloc_step_refuses_beyond_its_scratch():
    """The step on the library's own scratch refuses a configuration whose
    workspace exceeds the 64 MiB the library holds, before any HIP call."""
    lib = L.load()
    big = cfg(batch=32, n_q_heads=32, n_kv_heads=8, head_dim=128, rank=160, capacity=40960, window=64, topk=1024)
    assert s4r.workspace_size(big) > 64 << 20
    args = [FAKE] * 15
    st = lib.s4r_decode_step_noalloc(ctypes.byref(big), 40000, *args, None)
    assert st == L.S4R_ERR_WORKSPACE
    assert b"64" in lib.s4r_last_error() or b"67108864" in lib.s4r_last_error()
    # argument errors come first, as for the workspace step
    assert lib.s4r_decode_step_noalloc(None, 10, *args, None) == L.S4R_ERR_NULL_ARG
    assert lib.s4r_decode_step_noalloc(ctypes.byref(cfg()), 0, *args, None) == L.S4R_ERR_BAD_SHAPE


def test_rank_stride_and_query_window_limits():
    """A rank that is not a multiple of 32 is stored at the next multiple (the
    paper's r = 204 in 224 columns): the workspace is that of the stored width;
    a stored width beyond 256 is refused; G * W_q runs up to 128 (the paper's
    W_q = 32 at G = 4)."""
    lib = L.load()
    n48, n64, n = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
    assert lib.s4r_workspace_size(ctypes.byref(cfg(rank=48)), ctypes.byref(n48)) == L.S4R_OK
    assert lib.s4r_workspace_size(ctypes.byref(cfg(rank=64)), ctypes.byref(n64)) == L.S4R_OK
    assert n48.value == n64.value
    paper = dict(n_q_heads=32, n_kv_heads=8, head_dim=128, capacity=120_000, window=32, topk=23_968)
    assert lib.s4r_workspace_size(ctypes.byref(cfg(rank=204, q_window=32, **paper)), ctypes.byref(n)) == L.S4R_OK
    assert lib.s4r_workspace_size(ctypes.byref(cfg(rank=232, **paper)), ctypes.byref(n)) == L.S4R_OK
    assert lib.s4r_workspace_size(ctypes.byref(cfg(rank=260, **paper)), ctypes.byref(n)) == L.S4R_ERR_UNSUPPORTED
    assert lib.s4r_workspace_size(ctypes.byref(cfg(rank=204, q_window=33, **paper)),
                                  ctypes.byref(n)) == L.S4R_ERR_UNSUPPORTED
    assert s4r.rank_stride(204) == 224 and s4r.rank_stride(224) == 224 and s4r.rank_stride(1) == 32


def test_pad_latent_layout():
    """pad_latent moves each basis group's rank columns to its own 32-aligned
    block, zeros elsewhere; multiples of 32 pass through unchanged."""
    import numpy as np
    x = np.arange(2 * 3 * 2 * 40, dtype=np.float64).reshape(2, 3, 80) + 1.0
    y = s4r.pad_latent(x, 40, basis_groups=2)
    assert y.shape == (2, 3, 128)
    assert np.array_equal(y[..., 0:40], x[..., 0:40]) and np.array_equal(y[..., 64:104], x[..., 40:80])
    assert not y[..., 40:64].any() and not y[..., 104:128].any()
    t = torch.from_numpy(x)
    assert torch.equal(s4r.pad_latent(t, 40, 2), torch.from_numpy(y))
    z = np.ones((2, 64))
    assert s4r.pad_latent(z, 32, 2) is z
