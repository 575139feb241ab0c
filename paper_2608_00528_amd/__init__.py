"""S^4R decode step (arxiv 2608.00528) for AMD MI355X (gfx950).

The compute path is libs4r.so: hand-written HIP kernels behind the C ABI of
include/s4r.h.  This package is its Python binding (ctypes + torch device
memory and streams) and its build script.  Importing it loads the library and
fails loudly when the library has not been built.
"""

from . import _lib
from ._lib import Config, S4RError  # noqa: F401

_lib.load()

from .api import (  # noqa: E402,F401
    alloc_window_state,
    alloc_workspace,
    decode_step,
    decode_step_noalloc,
    decode_step_ragged,
    decode_step_windowed,
    dense_decode,
    full_recon_decode,
    make_config,
    num_selected,
    pack_coef,
    pad_latent,
    prefill,
    num_samples,
    prefill_bases,
    prefill_project,
    project_append,
    project_queries,
    rank_stride,
    read_bandwidth,
    reconstruct,
    score_latent,
    select_topk,
    sparse_attn,
    storage_dtype,
    timing_enable,
    timing_read,
    unpack_coef,
    window_state_init,
    window_state_size,
    value_config,
    version,
    workspace_size,
)
