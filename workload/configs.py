"""The five workload shapes the hot path is tested and measured on.

Shapes follow the paper's setting (multi-LoRA agents on Llama/Mistral-class
backbones, Sec. 4.1; trajectories of 1.9k-66.4k tokens, Table 5; 3-8 agents,
App. C.5; ranks 4-64, App. D.1; LoRA on k and v as in the QKVO variant,
App. D.2) at the sizes of one transformer layer.
"""
from __future__ import annotations

from dataclasses import dataclass, field


@dataclass(frozen=True)
class Config:
    index: int                 # 1..5, also the seed namespace
    name: str
    hidden: int                # d_in of k_proj / v_proj
    n_q: int
    n_kv: int
    head_dim: int
    theta: float               # RoPE base
    n_agents: int
    rank: int
    context: int               # shared context S already covered by the caches
    prefill_tokens: int        # new query tokens of one prefill chunk (0: none)
    decode_batch: int          # concurrent decode requests (0: none)
    precompute_rows: int       # hidden-state rows of one precompute call
    n_proj: int = 2            # k and v adapted
    layers: int = 1
    extra: dict = field(default_factory=dict)

    @property
    def group(self) -> int:
        return self.n_q // self.n_kv

    @property
    def lr_cols(self) -> int:
        return self.n_proj * self.n_agents * self.rank


CONFIGS = {
    1: Config(1, "tiny single layer", hidden=256, n_q=4, n_kv=4, head_dim=64,
              theta=1e4, n_agents=3, rank=8, context=512, prefill_tokens=16,
              decode_batch=1, precompute_rows=528),
    2: Config(2, "8B-shaped layer, 8k context", hidden=4096, n_q=32, n_kv=8,
              head_dim=128, theta=5e5, n_agents=4, rank=16, context=8192,
              prefill_tokens=512, decode_batch=1, precompute_rows=512),
    3: Config(3, "8B-shaped layer, 32k context", hidden=4096, n_q=32, n_kv=8,
              head_dim=128, theta=5e5, n_agents=8, rank=16, context=32768,
              prefill_tokens=4096, decode_batch=16, precompute_rows=4096),
    4: Config(4, "14B-shaped layer, 64k context", hidden=5120, n_q=40, n_kv=8,
              head_dim=128, theta=5e5, n_agents=6, rank=64, context=65536,
              prefill_tokens=2048, decode_batch=8, precompute_rows=2048),
    5: Config(5, "32-layer 8B-shaped stack, 4k-64k in 4096-token turns",
              hidden=4096, n_q=32, n_kv=8, head_dim=128, theta=5e5,
              n_agents=8, rank=16, context=65536, prefill_tokens=256,
              decode_batch=1, precompute_rows=4096, layers=32,
              extra={"turn_tokens": 4096, "turns": 16, "decode_steps": 128}),
}
