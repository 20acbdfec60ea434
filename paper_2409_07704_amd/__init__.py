"""libmas: batched Monotonic Alignment Search for AMD MI355X (gfx950).

The alignment runs in hand-written HIP kernels behind the C ABI of
``include/mas.h``; this package is the thin Python binding with the same
entry-point names.  It never computes an alignment in Python.
"""
from ._native import (  # noqa: F401
    ITEM_BAD_WORKSPACE,
    ITEM_EMPTY,
    ITEM_INFEASIBLE,
    ITEM_OK,
    ITEM_OUT_OF_RANGE,
    ITEM_SYNC_TIMEOUT,
    LIB_PATH,
    STATIC_SCRATCH_BYTES,
    MasError,
    Workspace,
    lib,
    mas_expand_path,
    mas_expand_text,
    mas_forward,
    mas_forward_ex,
    mas_forward_sentinel,
    mas_forward_static,
    mas_loglik,
    mas_search,
    mas_status_string,
    mas_version,
    mas_workspace_bytes,
    mas_workspace_init,
)
