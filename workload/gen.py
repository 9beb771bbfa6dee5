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

Weights are drawn in the orientation of Eq. 1, the one the C ABI takes:
frozen projections ``W [hidden, d_out]``, the stacked down-projections
``A_stack [hidden, n_proj*N*r]`` (columns ``(p*N + a)*r .. + r`` are agent a's
``A`` for projection p) and up-projections ``B [r, n_kv*d]``.
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
    A_stack = normal_bf16((cfg.hidden, cfg.lr_cols), 1.0 / math.sqrt(cfg.hidden),
                          seed_for(c, seed_base + 2), device)
    return {"X": X, "A_stack": A_stack}


def lora_case(cfg, tokens: int, seed_base: int = 0):
    """The full single-layer generative chain of the tiny workload.

    Returns hidden states ``X [tokens, hidden]``, frozen projections
    ``W_q [hidden, n_q*d]``, ``W_k, W_v [hidden, n_kv*d]`` (paper orientation,
    ``Y = X W``), stacked down-projections ``A_stack [hidden, n_proj*N*r]`` and
    per-agent up-projections ``B_k, B_v [N, r, n_kv*d]``.
    """
    c, h, d = cfg.index, cfg.hidden, cfg.head_dim
    s = 1.0 / math.sqrt(h)
    return {
        "X": normal_bf16((tokens, h), 1.0, seed_for(c, seed_base + 1)),
        "W_q": normal_bf16((h, cfg.n_q * d), s, seed_for(c, seed_base + 3)),
        "W_k": normal_bf16((h, cfg.n_kv * d), s, seed_for(c, seed_base + 4)),
        "W_v": normal_bf16((h, cfg.n_kv * d), s, seed_for(c, seed_base + 5)),
        "A_stack": normal_bf16((h, cfg.lr_cols), s, seed_for(c, seed_base + 2)),
        "B_k": normal_bf16((cfg.n_agents, cfg.rank, cfg.n_kv * d),
                           math.sqrt(B_VAR), seed_for(c, seed_base + 6)),
        "B_v": normal_bf16((cfg.n_agents, cfg.rank, cfg.n_kv * d),
                           math.sqrt(B_VAR), seed_for(c, seed_base + 7)),
    }


def attention_case(cfg, *, batch: int, n_tok: int, kv_len, positions, s_cap: int,
                   seed_base: int = 0, lr_k: bool = True, lr_v: bool = True,
                   q_std: float = 1.0, b_std: float = math.sqrt(B_VAR), v_std: float = 1.0,
                   rank: int | None = None, poison_tail: bool = True, device="cpu"):
    """Inputs of one ``lr_shared_attention`` call.

    ``kv_len`` is a list of per-request valid lengths and ``positions`` a
    ``[batch, n_tok]`` nested list of absolute query positions.  Rows at and
    beyond ``kv_len[b]`` of every cache are filled with NaN when
    ``poison_tail`` is set, so any read past the valid range shows up.
    ``v_std`` scales the value side (V_base and B_v) as a whole.
    """
    c, d, r = cfg.index, cfg.head_dim, (rank or cfg.rank)
    out = {
        "Q": normal_bf16((batch, n_tok, cfg.n_q, d), q_std, seed_for(c, seed_base + 11), device),
        "K_base": normal_bf16((batch, s_cap, cfg.n_kv, d), 1.0, seed_for(c, seed_base + 12), device),
        "V_base": normal_bf16((batch, s_cap, cfg.n_kv, d), v_std, seed_for(c, seed_base + 13), device),
        "L_k": normal_bf16((batch, s_cap, r), 1.0, seed_for(c, seed_base + 14), device) if lr_k else None,
        "L_v": normal_bf16((batch, s_cap, r), 1.0, seed_for(c, seed_base + 15), device) if lr_v else None,
        "B_k": normal_bf16((batch, r, cfg.n_kv * d), b_std, seed_for(c, seed_base + 16), device) if lr_k else None,
        "B_v": normal_bf16((batch, r, cfg.n_kv * d), b_std * v_std, seed_for(c, seed_base + 17), device) if lr_v else None,
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


def plant_plan(*, n_tok, n_q, n_kv, positions, kv_len, must, per_query, seed):
    """Choose planted keys: a list of ``(b, i, h, t)``, key t of request b to be
    aimed at query head h of query token i.

    ``positions [B][n_tok]`` and ``kv_len [B]`` give the keys each query may
    see (``t <= positions[b][i]`` and ``t < kv_len[b]``).  ``must[b]`` lists
    positions that should hold a planted key (split and tile boundaries, the
    causal diagonal ...); ``per_query(b, i, h)`` says how many keys (query
    token i, head h) gets, or 0.  The must-positions are handed out first,
    each to a visible (i, h) that still wants keys, then seeded random
    positions fill the rest.  Each (b, t, KV head) slot is used at most once,
    so a planted key serves exactly one query head.  Pure index bookkeeping.
    """
    rng = torch.Generator().manual_seed(int(seed))
    group = n_q // n_kv
    plan = []
    for b in range(len(kv_len)):
        kvl = int(kv_len[b])
        want = {(i, h): int(per_query(b, i, h)) for i in range(n_tok) for h in range(n_q)}
        used = set()                                     # (t, g)
        order = [ih for ih in want if want[ih] > 0]

        def give(i, h, t):
            plan.append((b, i, h, t))
            used.add((t, h // group))
            want[(i, h)] -= 1

        for k, t in enumerate(sorted(set(int(x) for x in must[b]))):
            if not 0 <= t < kvl:
                continue
            # Rotate the starting query head so the must-positions spread over heads.
            for j in range(len(order)):
                i, h = order[(k + j) % len(order)]
                if want[(i, h)] > 0 and t <= positions[b][i] and (t, h // group) not in used:
                    give(i, h, t)
                    break
        for i, h in order:
            vis = min(int(positions[b][i]) + 1, kvl)
            tries = 0
            while want[(i, h)] > 0 and vis > 0 and tries < 64:
                t = int(torch.randint(0, vis, (1,), generator=rng))
                tries += 1
                if (t, h // group) not in used:
                    give(i, h, t)
    return plan


def plant_keys(case, plan, margin: float, n_q: int, n_kv: int):
    """Aim the planted keys: ``K_base[b, t, g] = (margin / sqrt(d)) * Q[b, i, h]``
    (g the KV head of h), rounded to bf16.  With unit-scale queries such a key
    scores about ``margin`` through the base cache alone; the agent's LR key
    term then moves it up or down.  Returns the case (modified in place)."""
    d = case["Q"].shape[-1]
    group = n_q // n_kv
    c = margin / math.sqrt(d)
    for b, i, h, t in plan:
        case["K_base"][b, t, h // group] = (case["Q"][b, i, h].float() * c).to(torch.bfloat16)
    return case
