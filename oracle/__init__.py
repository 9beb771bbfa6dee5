"""Plain fp64 CPU oracle for the PreLRShared hot path (test infrastructure only).

This package is test infrastructure.  Only ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` may import it; the GPU product path
never imports, links or calls anything here, and nothing here imports the GPU
path.
"""
from .precache_oracle import (  # noqa: F401
    rope_frequencies,
    rope,
    precompute_lr_cache,
    project_kv_and_lr,
    rebuild_kv,
    attention_scores,
    attention_probs,
    attention,
    materialize_agent_kv,
    lr_shared_attention,
    merge_partials,
)
