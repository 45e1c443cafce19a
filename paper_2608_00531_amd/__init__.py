"""libcure: MI355X (gfx950) HIP kernels for CURE's verify-and-repair hot path.

The kernels and the C ABI live in csrc/ and include/cure.h; ``cure`` is the
thin ctypes binding (names match the C entry points).
"""

from .cure import (  # noqa: F401
    cure_margins, cure_margins_accept, cure_margins_noalloc, cure_tree_attn, cure_tree_attn_workspace_size, cure_accept,
    cure_repair_tree, cure_commit, cure_read_ceiling, lib,
    library_path, CureError, CURE_OK, CURE_ERR_INVALID_ARG, CURE_ERR_UNSUPPORTED,
    CURE_ERR_BAD_TREE, CURE_ERR_HIP, CURE_ERR_WORKSPACE, CURE_F32, CURE_BF16,
    CURE_ATTN_FORCE_VALU, CURE_MAX_TREE_NODES,
)
