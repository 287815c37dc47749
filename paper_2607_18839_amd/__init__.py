"""MI355X (gfx950) branch-parallel decode step of hierarchical parallel decoding.

The compute runs in libhpd.so (hand-written HIP kernels behind a C ABI,
include/hpd.h).  This package is the thin Python side: ``_lib`` mirrors the
C entry points one to one, and ``torch_api`` marshals torch tensors (device
memory and streams) into them.
"""
from . import _lib  # noqa: F401
from ._lib import (  # noqa: F401
    HPD_BF16,
    HPD_F32,
    HpdError,
    hpd_branch_attn_step,
    hpd_decode_step,
    hpd_decode_workspace_bytes,
    hpd_plan_create,
    hpd_plan_query,
    hpd_plan_upload,
)
