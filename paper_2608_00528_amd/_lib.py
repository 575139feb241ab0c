"""ctypes view of libs4r.so (include/s4r.h).  Argument marshalling only."""

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libs4r.so")

S4R_OK, S4R_ERR_NULL_ARG, S4R_ERR_BAD_SHAPE, S4R_ERR_UNSUPPORTED, S4R_ERR_WORKSPACE, \
    S4R_ERR_MISALIGNED, S4R_ERR_HIP = range(7)
STATUS_NAMES = {0: "OK", 1: "NULL_ARG", 2: "BAD_SHAPE", 3: "UNSUPPORTED", 4: "WORKSPACE",
                5: "MISALIGNED", 6: "HIP"}
S4R_FP32, S4R_BF16 = 0, 1
S4R_POOL_MAX, S4R_POOL_AVG = 0, 1
S4R_AGG_MEAN, S4R_AGG_MAX = 0, 1

EXPORTS = (
    "s4r_workspace_size", "s4r_num_selected", "s4r_last_error", "s4r_version",
    "s4r_score_latent", "s4r_select_topk", "s4r_reconstruct", "s4r_sparse_attn",
    "s4r_decode_step", "s4r_project_append", "s4r_pack_coef", "s4r_unpack_coef",
    "s4r_timing_enable", "s4r_timing_read", "s4r_read_bandwidth_sink_len", "s4r_read_bandwidth",
    "s4r_dense_decode", "s4r_prefill_project", "s4r_decode_step_ragged",
    "s4r_full_recon_decode", "s4r_prefill_num_samples", "s4r_prefill_bases_workspace_size", "s4r_prefill_bases",
    "s4r_project_queries", "s4r_decode_step_noalloc",
    "s4r_window_state_size", "s4r_window_state_init", "s4r_decode_step_windowed",
)


class Config(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("basis_groups", ctypes.c_int32),
        ("rank", ctypes.c_int32),
        ("n_sink", ctypes.c_int32),
        ("window", ctypes.c_int32),
        ("q_window", ctypes.c_int32),
        ("topk", ctypes.c_int32),
        ("pool_kernel", ctypes.c_int32),
        ("pool_mode", ctypes.c_int32),
        ("group_agg", ctypes.c_int32),
        ("bases_shared", ctypes.c_int32),
        ("capacity", ctypes.c_int64),
        ("rope_theta", ctypes.c_float),
        ("dtype", ctypes.c_int32),
        ("rank_v", ctypes.c_int32),
    ]


_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_SZ = ctypes.c_size_t
_CFG = ctypes.POINTER(Config)

_SIGS = {
    "s4r_workspace_size": (_I32, [_CFG, ctypes.POINTER(_SZ)]),
    "s4r_num_selected": (_I32, [_CFG, _I64]),
    "s4r_last_error": (ctypes.c_char_p, []),
    "s4r_version": (ctypes.c_char_p, []),
    "s4r_score_latent": (_I32, [_CFG, _I64, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "s4r_select_topk": (_I32, [_CFG, _I64, _P, _P, _P, _SZ, _P]),
    "s4r_reconstruct": (_I32, [_CFG, _I64, _I32, _P, _P, _P, _P, _P, _P, _P, _P]),
    "s4r_sparse_attn": (_I32, [_CFG, _I64, _I32, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "s4r_decode_step": (_I32, [_CFG, _I64, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                               _P, _SZ, _P]),
    "s4r_project_append": (_I32, [_CFG, _I64, _P, _P, _P, _P, _P, _P, _P]),
    "s4r_pack_coef": (_I32, [_CFG, _I64, _P, _P, _P]),
    "s4r_unpack_coef": (_I32, [_CFG, _I64, _P, _P, _P]),
    "s4r_timing_enable": (_I32, [_I32]),
    "s4r_timing_read": (_I32, [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_I64)]),
    "s4r_read_bandwidth_sink_len": (_I64, []),
    "s4r_read_bandwidth": (_I32, [_P, _I64, _P, _P]),
    "s4r_dense_decode": (_I32, [_CFG, _I64, _P, _P, _P, _P, _P, _SZ, _P]),
    "s4r_prefill_project": (_I32, [_CFG, _I64, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "s4r_project_queries": (_I32, [_CFG, _I64, _P, _P, _P, _P, _SZ, _P]),
    "s4r_prefill_num_samples": (_I64, [_I64, ctypes.c_double]),
    "s4r_prefill_bases_workspace_size": (_I32, [_CFG, _I64, ctypes.c_double, ctypes.POINTER(_SZ)]),
    "s4r_prefill_bases": (_I32, [_CFG, _I64, _P, _P, ctypes.c_double, _I32, _P, _P, _P, _P, _SZ, _P]),
    "s4r_full_recon_decode": (_I32, [_CFG, _I64, _P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "s4r_decode_step_noalloc": (_I32, [_CFG, _I64, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                       _P, _P]),
    "s4r_decode_step_ragged": (_I32, [_CFG, ctypes.POINTER(_I64), _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                      _P, _P, _P, _P, _P, _SZ, _P]),
    "s4r_window_state_size": (_I32, [_CFG, ctypes.POINTER(_SZ)]),
    "s4r_window_state_init": (_I32, [_CFG, _I64, _P, _P, _P, _P, _SZ, _P]),
    "s4r_decode_step_windowed": (_I32, [_CFG, _I64, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                        _P, _SZ, _P]),
}

_lib = None


def load():
    """Load libs4r.so once.  Raises if it has not been built: there is no
    fallback implementation."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing; build it with `python -m paper_2608_00528_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    for name, (res, args) in _SIGS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


class S4RError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


def check(status):
    if status != S4R_OK:
        raise S4RError(status, load().s4r_last_error().decode())
    return status
