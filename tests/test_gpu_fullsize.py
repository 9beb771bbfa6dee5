"""Parity at the full workload sizes, in the launch configuration the benchmark
times.  The GPU computes every output; the oracle recomputes sampled requests
and sampled query tokens (each input is regenerated on the host from its seed,
request by request, so the host never holds the whole batch)."""
import numpy as np
import pytest
import torch

import oracle
from gpu_cases import ATOL_MAX, ATOL_MEAN, LSE_ATOL, attn_errors, f64, gpu_attention, lse_error
from workload import CONFIGS, attention_case

pytestmark = pytest.mark.gpu


def request_case(cfg, b, n_tok, kv_len, pos, s_cap, tag, lr_k=True, lr_v=True, rank=None):
    """Inputs of request b alone (batch 1), seeded per request."""
    return attention_case(cfg, batch=1, n_tok=n_tok, kv_len=[kv_len], positions=[pos], s_cap=s_cap,
                          seed_base=10_000 * tag + 37 * b, poison_tail=False, lr_k=lr_k, lr_v=lr_v, rank=rank)


def build_batch(cfg, B, n_tok, kv_len, pos_of, s_cap, tag, **wiring):
    """Device tensors for the whole batch, filled request by request."""
    g = None
    for b in range(B):
        c = request_case(cfg, b, n_tok, kv_len, pos_of(b), s_cap, tag, **wiring)
        if g is None:
            g = {k: (torch.empty((B,) + tuple(v.shape[1:]), dtype=v.dtype, device="cuda") if v is not None else None)
                 for k, v in c.items()}
        for k, v in c.items():
            if v is not None:
                g[k][b].copy_(v[0])
    return g


def check_sampled(cfg, g, O, lse, n_tok, kv_len, pos_of, s_cap, tag, reqs, toks, **wiring):
    for b in reqs:
        c = request_case(cfg, b, n_tok, kv_len, pos_of(b), s_cap, tag, **wiring)
        Q = f64(c["Q"])[:, toks]
        pos = c["positions"].numpy()[:, toks]
        Oref, lref = oracle.lr_shared_attention(Q, f64(c["K_base"]), f64(c["V_base"]), f64(c["L_k"]),
                                                f64(c["L_v"]), f64(c["B_k"]), f64(c["B_v"]),
                                                pos, [kv_len], cfg.theta)
        mx, mean = attn_errors(O[b:b + 1, toks], Oref)
        print(f"  request {b}: max abs {mx:.2e}, mean abs {mean:.2e}", flush=True)
        assert mx <= ATOL_MAX and mean <= ATOL_MEAN, (b, mx, mean)
        assert lse_error(lse[b:b + 1, toks], lref) <= LSE_ATOL


def test_c2_decode_8k():
    cfg = CONFIGS[2]
    S = cfg.context
    g = build_batch(cfg, 1, 1, S, lambda b: [S - 1], S, 2)
    O, lse = gpu_attention(g, cfg.theta)
    check_sampled(cfg, g, O, lse, 1, S, lambda b: [S - 1], S, 2, [0], [0])


def test_c2_prefill_512_at_8k():
    cfg = CONFIGS[2]
    S, n = cfg.context, cfg.prefill_tokens
    pos = list(range(S, S + n))
    g = build_batch(cfg, 1, n, S + n, lambda b: pos, S + n, 3)
    O, lse = gpu_attention(g, cfg.theta)
    check_sampled(cfg, g, O, lse, n, S + n, lambda b: pos, S + n, 3, [0], [0, 1, 127, 128, 255, 300, 510, 511])


def test_c3_decode_batch16_32k():
    cfg = CONFIGS[3]
    S = cfg.context
    g = build_batch(cfg, cfg.decode_batch, 1, S, lambda b: [S - 1], S, 4)
    O, lse = gpu_attention(g, cfg.theta)
    check_sampled(cfg, g, O, lse, 1, S, lambda b: [S - 1], S, 4, [0, 9, 15], [0])


def test_c3_prefill_4096_at_32k():
    cfg = CONFIGS[3]
    S, n = cfg.context, cfg.prefill_tokens
    pos = list(range(S, S + n))
    g = build_batch(cfg, 1, n, S + n, lambda b: pos, S + n, 5)
    O, lse = gpu_attention(g, cfg.theta)
    check_sampled(cfg, g, O, lse, n, S + n, lambda b: pos, S + n, 5, [0], [0, 31, 32, 2047, 4064, 4095])


def test_c4_decode_batch8_64k():
    cfg = CONFIGS[4]
    S = cfg.context
    g = build_batch(cfg, cfg.decode_batch, 1, S, lambda b: [S - 1], S, 6)
    O, lse = gpu_attention(g, cfg.theta)
    check_sampled(cfg, g, O, lse, 1, S, lambda b: [S - 1], S, 6, [0, 7], [0])


def test_c4_prefill_2048_at_64k():
    cfg = CONFIGS[4]
    S, n = cfg.context, cfg.prefill_tokens
    pos = list(range(S, S + n))
    g = build_batch(cfg, 1, n, S + n, lambda b: pos, S + n, 7)
    O, lse = gpu_attention(g, cfg.theta)
    check_sampled(cfg, g, O, lse, n, S + n, lambda b: pos, S + n, 7, [0], [0, 25, 26, 1024, 2047])


@pytest.mark.parametrize("wiring", [dict(lr_k=False, lr_v=True, rank=64), dict(lr_k=False, lr_v=True, rank=32),
                                    dict(lr_k=True, lr_v=True, rank=8), dict(lr_k=True, lr_v=True, rank=64)],
                         ids=["qv_r64", "qv_r32", "kv_r8", "kv_r64"])
def test_c3_prefill_rank_sweep_wirings(wiring):
    # The rank sweep's prefill shapes (4096 queries at 32k, the tile-cache
    # instantiations: values-only LR from rank 32, k and v at ranks 8 and 64).
    cfg = CONFIGS[3]
    S, n = cfg.context, cfg.prefill_tokens
    pos = list(range(S, S + n))
    g = build_batch(cfg, 1, n, S + n, lambda b: pos, S + n, 8, **wiring)
    O, lse = gpu_attention(g, cfg.theta)
    check_sampled(cfg, g, O, lse, n, S + n, lambda b: pos, S + n, 8, [0], [0, 63, 64, 2047, 4031, 4095], **wiring)
