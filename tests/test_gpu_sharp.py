"""GPU parity on the planted-key ("sharp") set: O(1) outputs decided by a few
keys placed at split and tile boundaries and on the causal diagonal (see
sharp_cases.py), for every rank and LR wiring at small sizes (every output
checked) and in the launch plans of the 8k, 32k and 64k workloads (sampled
outputs).  Each case also checks the LR-sensitivity gate: the LR terms'
contribution O - O(B = 0) is reproduced to 5e-2 relative."""
import math

import numpy as np
import pytest
import torch

import oracle
from gpu_cases import (ATOL_MAX, ATOL_MEAN, LR_SENS, LSE_ATOL, attn_errors, f64, gpu_attention, lse_error,
                       oracle_attention, to_dev)
from paper_2609_34054_amd import make_dims
from sharp_cases import boundary_keys, decode_split_tokens, prefill_split_tokens, sharp_case
from workload import CONFIGS, Config

pytestmark = pytest.mark.gpu


def mk_cfg(idx, n_q, n_kv, d, r):
    return Config(idx, "sharp", hidden=256, n_q=n_q, n_kv=n_kv, head_dim=d, theta=5e5, n_agents=1, rank=r,
                  context=0, prefill_tokens=0, decode_batch=0, precompute_rows=0)


def zero_b(g):
    z = dict(g)
    for k in ("B_k", "B_v"):
        if z[k] is not None:
            z[k] = torch.zeros_like(z[k])
    return z


def check_lr_sensitivity(O, O0, Oref, O0ref):
    dg, dr = f64(O) - f64(O0), Oref - O0ref
    rel = np.linalg.norm(dg - dr) / np.linalg.norm(dr)
    assert rel <= LR_SENS, rel
    return rel


def plan_dims(cfg, g):
    return make_dims(g["Q"], g["K_base"], g["L_k"], g["L_v"], g["B_k"], g["B_v"], cfg.theta)


# --------------------------------------------------------------- small sizes
# id, d, r, n_q, n_kv, n_tok, kv_lens, lr
SMALL = []
for r in (8, 16, 32, 64):
    for lr in ("kv", "v", "k"):
        SMALL.append((f"decode_r{r}_{lr}", 128, r, 8, 2, 1, [3000, 2999], lr))
        SMALL.append((f"prefill_r{r}_{lr}", 128, r, 8, 2, 16, [530], lr))
        SMALL.append((f"split_prefill_r{r}_{lr}", 128, r, 8, 2, 64, [1100], lr))
SMALL += [
    ("decode_g5_r64", 128, 64, 10, 2, 1, [1500, 700, 64], "kv"),
    ("prefill_g5_r64_ragged", 128, 64, 10, 2, 37, [700, 300], "kv"),
    ("decode_d64_r16", 64, 16, 4, 4, 1, [900], "kv"),
    ("split_prefill_d64_r32", 64, 32, 8, 2, 24, [1300], "kv"),
]


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_sharp_small(case):
    cid, d, r, n_q, n_kv, n_tok, kv_lens, lr = case
    print(f"sharp {cid}", flush=True)
    cfg = mk_cfg(80 + len(cid), n_q, n_kv, d, r)
    B = len(kv_lens)
    pos = [list(range(k - n_tok, k)) for k in kv_lens]
    s_cap = -(-max(kv_lens) // 16) * 16
    # The launch plan decides where splits start: plant keys on their edges.
    probe = sharp_case(cfg, batch=B, n_tok=n_tok, kv_len=kv_lens, positions=pos, s_cap=s_cap, seed=1, lr=lr,
                       per_query=lambda b, i, h: 0, poison_tail=False)
    dims = plan_dims(cfg, probe)
    if n_tok == 1:
        step = decode_split_tokens(dims)
        n_splits = -(-s_cap // step)
        must = [boundary_keys(k, step, every=max(1, n_splits // 10)) for k in kv_lens]
    else:
        step = prefill_split_tokens(dims)
        must = [sorted(set(boundary_keys(k, 64, every=3)) | set(boundary_keys(k, step)) |
                       {k - 1 - j for j in range(0, n_tok, 5)}) for k in kv_lens]
    c = sharp_case(cfg, batch=B, n_tok=n_tok, kv_len=kv_lens, positions=pos, s_cap=s_cap, seed=31 * len(cid),
                   lr=lr, must=must)
    g = to_dev(c)
    O, lse = gpu_attention(g, cfg.theta)
    Oref, lref = oracle_attention(c, cfg.theta)
    mx, mean = attn_errors(O, Oref)
    print(f"  |O| mean {np.abs(Oref).mean():.3f}, max abs err {mx:.2e}, mean abs err {mean:.2e}", flush=True)
    assert mx <= ATOL_MAX and mean <= ATOL_MEAN, (mx, mean)
    assert lse_error(lse, lref) <= LSE_ATOL
    O0, _ = gpu_attention(zero_b(g), cfg.theta)
    O0ref, _ = oracle_attention(c, cfg.theta, zero_b=True)
    check_lr_sensitivity(O, O0, Oref, O0ref)


# ---------------------------------------------------------------- full sizes
def full_batch(cfg, B, n_tok, kv, pos, sampled_toks, must, tag):
    """Device batch built request by request (each seeded on its own), with
    keys planted for the sampled query tokens."""
    g, cases = None, {}
    per_query = (lambda b, i, h: (1 + (h + i) % 8) if i in sampled_toks else 0)
    for b in range(B):
        c = sharp_case(cfg, batch=1, n_tok=n_tok, kv_len=[kv], positions=[pos], s_cap=kv, seed=10_000 * tag + 37 * b,
                       must=[must], per_query=per_query, poison_tail=False)
        if g is None:
            g = {k: (torch.empty((B,) + tuple(v.shape[1:]), dtype=v.dtype, device="cuda") if v is not None else None)
                 for k, v in c.items() if k != "plan"}
        for k, v in c.items():
            if k != "plan" and v is not None:
                g[k][b].copy_(v[0])
        cases[b] = c
    return g, cases


def check_full(cfg, g, cases, reqs, toks):
    O, lse = gpu_attention(g, cfg.theta)
    O0, _ = gpu_attention(zero_b(g), cfg.theta)
    for b in reqs:
        c = cases[b]
        Oref, lref = oracle_attention(c, cfg.theta, toks=toks)
        O0ref, _ = oracle_attention(c, cfg.theta, toks=toks, zero_b=True)
        Og, O0g = O[b:b + 1, toks], O0[b:b + 1, toks]
        mx, mean = attn_errors(Og, Oref)
        rel = check_lr_sensitivity(Og, O0g, Oref, O0ref)
        print(f"  request {b}: |O| mean {np.abs(Oref).mean():.3f}, max abs err {mx:.2e}, mean abs err "
              f"{mean:.2e}, LR-term rel err {rel:.2e}", flush=True)
        assert mx <= ATOL_MAX and mean <= ATOL_MEAN, (b, mx, mean)
        assert lse_error(lse[b:b + 1, toks], lref) <= LSE_ATOL


def test_sharp_c3_decode_batch16_32k():
    """The benchmark's decode: 16 requests at 32768 tokens, 32 splits of 1024
    keys, a planted key on both sides of every split boundary."""
    cfg = CONFIGS[3]
    S, B = cfg.context, cfg.decode_batch
    g, cases = full_batch(cfg, B, 1, S, [S - 1], {0}, boundary_keys(S, 1024), 31)
    assert decode_split_tokens(plan_dims(cfg, g)) == 1024
    check_full(cfg, g, cases, [0, 9, 15], [0])


def test_sharp_c3_prefill_4096_at_32k():
    cfg = CONFIGS[3]
    S, n = cfg.context, cfg.prefill_tokens
    kv = S + n
    toks = [0, 31, 32, 2047, 4064, 4095]
    must = sorted(set(boundary_keys(kv, 64, every=37)) | {S + i for i in toks} | {S + i - 1 for i in toks})
    g, cases = full_batch(cfg, 1, n, kv, list(range(S, kv)), set(toks), must, 32)
    check_full(cfg, g, cases, [0], toks)


def test_sharp_c4_prefill_2048_at_64k():
    """14B shape, rank 64, GQA 5: the prefill splits its KV range."""
    cfg = CONFIGS[4]
    S, n = cfg.context, cfg.prefill_tokens
    kv = S + n
    toks = [0, 25, 26, 1024, 2047]
    probe_dims = make_dims(torch.empty((1, n, cfg.n_q, cfg.head_dim), dtype=torch.bfloat16),
                           torch.empty((1, kv, cfg.n_kv, cfg.head_dim), dtype=torch.bfloat16),
                           torch.empty((1, kv, cfg.rank), dtype=torch.bfloat16), None,
                           torch.empty((1, cfg.rank, cfg.n_kv * cfg.head_dim), dtype=torch.bfloat16), None,
                           cfg.theta)
    step = prefill_split_tokens(probe_dims)
    assert step < kv  # split
    must = sorted(set(boundary_keys(kv, step)) | set(boundary_keys(kv, 64, every=101)) | {S + i for i in toks})
    g, cases = full_batch(cfg, 1, n, kv, list(range(S, kv)), set(toks), must, 33)
    check_full(cfg, g, cases, [0], toks)


def test_sharp_c4_decode_batch8_64k():
    cfg = CONFIGS[4]
    S, B = cfg.context, cfg.decode_batch
    probe = make_dims(torch.empty((B, 1, cfg.n_q, cfg.head_dim), dtype=torch.bfloat16),
                      torch.empty((B, S, cfg.n_kv, cfg.head_dim), dtype=torch.bfloat16),
                      torch.empty((B, S, cfg.rank), dtype=torch.bfloat16), None,
                      torch.empty((B, cfg.rank, cfg.n_kv * cfg.head_dim), dtype=torch.bfloat16), None, cfg.theta)
    step = decode_split_tokens(probe)
    g, cases = full_batch(cfg, B, 1, S, [S - 1], {0}, boundary_keys(S, step, every=2), 34)
    check_full(cfg, g, cases, [0, 7], [0])


def test_sharp_c2_prefill_512_and_decode_at_8k():
    cfg = CONFIGS[2]
    S, n = cfg.context, cfg.prefill_tokens
    kv = S + n
    toks = [0, 1, 255, 300, 511]
    must = sorted(set(boundary_keys(kv, 64, every=11)) | {S + i for i in toks})
    g, cases = full_batch(cfg, 1, n, kv, list(range(S, kv)), set(toks), must, 35)
    check_full(cfg, g, cases, [0], toks)
    g, cases = full_batch(cfg, 1, 1, S, [S - 1], {0}, boundary_keys(S, 32, every=16), 36)
    check_full(cfg, g, cases, [0], [0])
