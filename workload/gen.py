"""Seeded generators of synthetic inputs (random draws only, no method arithmetic).

Every tensor is drawn with its own ``torch.Generator`` seeded ``1000*c + k``
(c = workload index, k = tensor index), in float32 and then rounded to bf16
(round to nearest even).  Distributions follow the workload description:
hidden states ``X ~ N(0, 1)``; frozen and LoRA down-projection weights with
variance ``1/hidden``; LoRA up-projections ``B`` with variance 0.02 (the second
argument of N(.,.) is read as a variance); base-cache and query entries
``N(0, 1)`` (the distribution of a rotated projection of unit-scale hidden
states); LR-cache entries ``N(0, 1)`` (the distribution of ``X A`` for such X
and A).

Storage orientation of the LoRA weights is the one the C ABI takes (the PEFT
storage layout): down-projections as rows ``[n_proj*N*r, hidden]`` (row
``(p*N + a)*r + j`` is column j of agent a's ``A`` for projection p) and
up-projections as ``[n_kv*d, r]`` (the transpose of the paper's ``B``).
"""
from __future__ import annotations

import math

import torch

B_VAR = 0.02


def seed_for(config_index: int, k: int) -> int:
    return 1000 * int(config_index) + int(k)


def normal_bf16(shape, std: float, seed: int, device="cpu") -> torch.Tensor:
    """``N(0, std^2)`` draws rounded to bf16, reproducible from ``seed``."""
    g = torch.Generator(device=device).manual_seed(int(seed))
    x = torch.randn(*shape, generator=g, dtype=torch.float32, device=device)
    if std != 1.0:
        x.mul_(std)
    return x.to(torch.bfloat16)


def precompute_case(cfg, rows: int, seed_base: int = 0, device="cpu"):
    """Hidden states of one new segment and the stacked down-projections."""
    c = cfg.index
    X = normal_bf16((rows, cfg.hidden), 1.0, seed_for(c, seed_base + 1), device)
    A_rows = normal_bf16((cfg.lr_cols, cfg.hidden), 1.0 / math.sqrt(cfg.hidden),
                         seed_for(c, seed_base + 2), device)
    return {"X": X, "A_rows": A_rows}


def lora_case(cfg, tokens: int, seed_base: int = 0):
    """The full single-layer generative chain of the tiny workload.

    Returns hidden states ``X [tokens, hidden]``, frozen projections
    ``W_q [hidden, n_q*d]``, ``W_k, W_v [hidden, n_kv*d]`` (paper orientation,
    ``Y = X W``), stacked down-projections ``A_rows`` and per-agent
    up-projections ``Bk_rows, Bv_rows [N, n_kv*d, r]``.
    """
    c, h, d = cfg.index, cfg.hidden, cfg.head_dim
    s = 1.0 / math.sqrt(h)
    return {
        "X": normal_bf16((tokens, h), 1.0, seed_for(c, seed_base + 1)),
        "W_q": normal_bf16((h, cfg.n_q * d), s, seed_for(c, seed_base + 3)),
        "W_k": normal_bf16((h, cfg.n_kv * d), s, seed_for(c, seed_base + 4)),
        "W_v": normal_bf16((h, cfg.n_kv * d), s, seed_for(c, seed_base + 5)),
        "A_rows": normal_bf16((cfg.lr_cols, h), s, seed_for(c, seed_base + 2)),
        "Bk_rows": normal_bf16((cfg.n_agents, cfg.n_kv * d, cfg.rank),
                               math.sqrt(B_VAR), seed_for(c, seed_base + 6)),
        "Bv_rows": normal_bf16((cfg.n_agents, cfg.n_kv * d, cfg.rank),
                               math.sqrt(B_VAR), seed_for(c, seed_base + 7)),
    }


def attention_case(cfg, *, batch: int, n_tok: int, kv_len, positions, s_cap: int,
                   seed_base: int = 0, lr_k: bool = True, lr_v: bool = True,
                   q_std: float = 1.0, b_std: float = math.sqrt(B_VAR),
                   rank: int | None = None, poison_tail: bool = True, device="cpu"):
    """Inputs of one ``lr_shared_attention`` call.

    ``kv_len`` is a list of per-request valid lengths and ``positions`` a
    ``[batch, n_tok]`` nested list of absolute query positions.  Rows at and
    beyond ``kv_len[b]`` of every cache are filled with NaN when
    ``poison_tail`` is set, so any read past the valid range shows up.
    """
    c, d, r = cfg.index, cfg.head_dim, (rank or cfg.rank)
    out = {
        "Q": normal_bf16((batch, n_tok, cfg.n_q, d), q_std, seed_for(c, seed_base + 11), device),
        "K_base": normal_bf16((batch, s_cap, cfg.n_kv, d), 1.0, seed_for(c, seed_base + 12), device),
        "V_base": normal_bf16((batch, s_cap, cfg.n_kv, d), 1.0, seed_for(c, seed_base + 13), device),
        "L_k": normal_bf16((batch, s_cap, r), 1.0, seed_for(c, seed_base + 14), device) if lr_k else None,
        "L_v": normal_bf16((batch, s_cap, r), 1.0, seed_for(c, seed_base + 15), device) if lr_v else None,
        "Bk_rows": normal_bf16((batch, cfg.n_kv * d, r), b_std, seed_for(c, seed_base + 16), device) if lr_k else None,
        "Bv_rows": normal_bf16((batch, cfg.n_kv * d, r), b_std, seed_for(c, seed_base + 17), device) if lr_v else None,
        "positions": torch.tensor(positions, dtype=torch.int32).reshape(batch, n_tok),
        "kv_len": torch.tensor(kv_len, dtype=torch.int32).reshape(batch),
    }
    if poison_tail:
        for name in ("K_base", "V_base", "L_k", "L_v"):
            t = out[name]
            if t is None:
                continue
            for b in range(batch):
                t[b, int(kv_len[b]):] = float("nan")
    return out
