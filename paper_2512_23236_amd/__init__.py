"""MI355X (gfx950) batched multi-table pooled embedding-bag lookup and its
sparse gradient: hand-written HIP kernels behind a C ABI (include/tbe.h),
with a thin Python binding in :mod:`paper_2512_23236_amd.tbe`."""
from . import tbe  # noqa: F401
from .tbe import Plan, SparseGrad, TBEError, backward, backward_workspace_bytes, forward  # noqa: F401
