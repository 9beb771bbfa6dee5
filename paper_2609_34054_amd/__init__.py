"""PreLRShared hot path (PReCache, Sec. 3.1) for MI355X / gfx950.

The compute lives in ``libprecache.so`` (hand-written HIP kernels behind the C
ABI declared in ``include/precache.h``); this package is its thin Python
binding.  Torch provides device memory and streams only.
"""
from .binding import (  # noqa: F401
    EXPORTS,
    LrsaDims,
    LrsaPaging,
    PrecacheError,
    lib,
    lr_shared_attention,
    lr_shared_attention_noalloc,
    lr_shared_attention_paged,
    make_dims,
    paged_workspace_size,
    materialize_agent_kv,
    precompute_lr_cache,
    project_kv_and_lr_cache,
    project_kv_and_lr_cache_paged,
    stream_read,
    use_checked_library,
    workspace_size,
)

__version__ = "0.1.0"
