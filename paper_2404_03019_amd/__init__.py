"""libgeot_hip: sorted segment reduction and fused gather-weight-scatter on MI355X (gfx950).

The computation lives in hand-written HIP kernels behind the C-ABI of
include/geot.h; this package only builds that library and marshals torch
tensors into it (see ``geot.py``).
"""
from .geot import (  # noqa: F401
    FAMILIES,
    OPS,
    GeotError,
    KernelChoice,
    IndexStats,
    LIB_PATH,
    lib,
    segment_reduce,
    gather_scatter,
    workspace_size,
    segment_reduce_ws,
    gather_scatter_ws,
    segment_reduce_noalloc,
    noalloc_scratch_bytes,
    segment_reduce_backward,
    gather_scatter_backward,
    segment_reduce_max_arg,
    gather_scatter_max_arg,
    segment_reduce_backward_max_arg,
    gather_scatter_backward_max_arg,
    index_stats,
    transpose_edges,
    check_index,
    select,
    last_choice,
    profile_begin,
    profile_end,
    release_scratch,
    version,
)
