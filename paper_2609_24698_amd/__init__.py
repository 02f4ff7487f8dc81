"""Tree-structured speculative verification over CSA/HCA compressed attention on MI355X.

The compute path is the gfx950 HIP library ``lib/libtv.so`` (C ABI in
``include/tv.h``); this package is its Python binding.
"""
from .binding import (  # noqa: F401
    EXPORTED,
    DeviceRound,
    LayeredRound,
    TvCache,
    TvDims,
    TvError,
    lib,
    make_cache,
    make_dims,
    status_string,
    tv_branch_compress,
    tv_build_tree_mask,
    tv_commit_accepted_path,
    tv_profile_disable,
    tv_profile_enable,
    tv_profile_read,
    tv_select_accepted_path,
    tv_select_workspace_bytes,
    tv_verify_attention,
    tv_verify_workspace_bytes,
)
