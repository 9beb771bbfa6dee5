"""The planted-key ("sharp") parity set.

With unit-scale random queries and keys over thousands of tokens, attention is
nearly uniform and every output is a tiny average, so absolute gates see
little.  Here selected keys are aimed at selected query heads
(``K_base[t, g] = c * Q[i, h]``) so that each such query head puts almost all
of its weight on its 1-8 planted keys: its output is O(1) and is decided by
those few keys, their agent's LR key term (which moves their scores by about
+-0.6) and their value rows.  The planted keys sit where a kernel's structure
could go wrong: the first key, every decode split boundary, prefill tile and
split boundaries, the middle and the last key (the causal diagonal).  A fault
confined to one split or one tile then moves some output by O(0.1-1).

Scales: a planted key scores ``log(kv_len) + 4`` through its base part, so it
outweighs all unplanted keys together about 30 times.  The value side (V_base
and B_v) is drawn at half scale, which keeps the outputs unit-scale (mean
|O| 0.3-0.5, max below 3): the gates are stated for unit-scale outputs, and
bf16 storage of an output of size 4-8 alone errs up to 0.016.
"""
from __future__ import annotations

import ctypes
import math

from workload import attention_case
from workload.gen import plant_keys, plant_plan

SHARP_V_STD = 0.5
TILE_DECODE = 32      # tokens per decode KV tile
TILE_PREFILL = 64     # tokens per prefill KV tile


def margin(kv_len: int) -> float:
    return math.log(max(int(kv_len), 2)) + 4.0


def decode_split_tokens(dims) -> int:
    """Tokens per decode split of a call, from its workspace size."""
    from paper_2609_34054_amd.binding import lib
    ws = lib().lr_shared_attention_workspace_size(ctypes.byref(dims))
    r = dims.rank if dims.rank in (8, 16, 32, 64) else 8
    ns = ws // (dims.batch * dims.n_q_heads * (4 + dims.head_dim + r) * 4)
    tiles = -(-dims.s_cap // TILE_DECODE)
    return -(-tiles // ns) * TILE_DECODE


def prefill_split_tokens(dims) -> int:
    """Tokens per KV split of a prefill call (its whole range when unsplit)."""
    from paper_2609_34054_amd.binding import lib
    ws = lib().lr_shared_attention_workspace_size(ctypes.byref(dims))
    tiles = -(-dims.s_cap // TILE_PREFILL)
    if ws == 0:
        return tiles * TILE_PREFILL
    r = dims.rank if dims.rank in (8, 16, 32, 64) else 8
    ns = ws // (dims.batch * dims.n_tok * dims.n_q_heads * (4 + dims.head_dim + r) * 4)
    return -(-tiles // ns) * TILE_PREFILL


def boundary_keys(kv_len: int, step: int, every: int = 1):
    """The keys on both sides of every ``every``-th multiple of ``step``, plus
    the first, middle and last key."""
    out = {0, kv_len // 2, kv_len - 1}
    k = step
    n = 0
    while k < kv_len:
        if n % every == 0:
            out.update((k - 1, k))
        k += step
        n += 1
    return sorted(t for t in out if 0 <= t < kv_len)


def sharp_case(cfg, *, batch, n_tok, kv_len, positions, s_cap, seed, lr="kv", rank=None, must=None,
               per_query=None, poison_tail=True):
    """An attention case with planted keys.  ``must[b]`` lists the keys of
    request b to plant first; ``per_query(b, i, h)`` how many keys each query
    head gets (default 1 + h % 8 for decode, 1 + (i + h) % 4 for prefill)."""
    if per_query is None:
        per_query = (lambda b, i, h: 1 + h % 8) if n_tok == 1 else (lambda b, i, h: 1 + (i + h) % 4)
    if must is None:
        must = [[] for _ in range(batch)]
    c = attention_case(cfg, batch=batch, n_tok=n_tok, kv_len=kv_len, positions=positions, s_cap=s_cap,
                       seed_base=seed, lr_k=lr in ("kv", "k"), lr_v=lr in ("kv", "v"), rank=rank,
                       v_std=SHARP_V_STD, poison_tail=False)
    plan = plant_plan(n_tok=n_tok, n_q=cfg.n_q, n_kv=cfg.n_kv, positions=positions, kv_len=kv_len, must=must,
                      per_query=per_query, seed=seed + 7)
    plant_keys(c, plan, margin(max(kv_len)), cfg.n_q, cfg.n_kv)
    if poison_tail:
        for name in ("K_base", "V_base", "L_k", "L_v"):
            t = c[name]
            if t is not None:
                for b in range(batch):
                    t[b, int(kv_len[b]):] = float("nan")
    c["plan"] = plan
    return c
