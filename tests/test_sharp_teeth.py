"""The planted-key parity data has teeth (CPU only).

At the full 32k-context shapes, each mistake a kernel could make in one KV
split or one KV tile -- the key LR term rotated at split-relative positions,
the key or value LR term dropped, the split skipped, the causal diagonal
masked -- is planted in the oracle's computation and must move the sampled
outputs past the GPU gates (max abs 2e-2; LR sensitivity 5e-2), so a kernel
making it fails parity.  On the unit-scale random data alone such faults
stayed inside every gate."""
import numpy as np
import pytest

import oracle
from gpu_cases import ATOL_MAX, LR_SENS
from paper_2609_34054_amd.binding import LrsaDims
from sharp_cases import boundary_keys, decode_split_tokens, sharp_case
from workload import CONFIGS

f64 = lambda t: None if t is None else t.double().numpy()


def _decode_case():
    cfg = CONFIGS[3]
    S = cfg.context
    dims = LrsaDims(batch=cfg.decode_batch, n_tok=1, n_q_heads=cfg.n_q, n_kv_heads=cfg.n_kv, head_dim=cfg.head_dim,
                    rank=cfg.rank, s_cap=S, kv_req_stride=S * cfg.n_kv * cfg.head_dim, l_req_stride=S * cfg.rank,
                    b_req_stride=cfg.rank * cfg.n_kv * cfg.head_dim, softmax_scale=0.0, reserved0=0.0,
                    rope_theta=cfg.theta)
    L = decode_split_tokens(dims)
    assert L == 1024  # 32 splits of 32 tiles at batch 16
    c = sharp_case(cfg, batch=1, n_tok=1, kv_len=[S], positions=[[S - 1]], s_cap=S, seed=424242,
                   must=[boundary_keys(S, L)], poison_tail=False)
    return cfg, c, L


def _parts(c, theta):
    K, V = oracle.rebuild_kv(f64(c["K_base"])[0], f64(c["V_base"])[0], f64(c["L_k"])[0], f64(c["L_v"])[0],
                             f64(c["B_k"])[0], f64(c["B_v"])[0], theta)
    return f64(c["Q"])[0], K, V, c["positions"].numpy()[0]


def _caught(O, O_ref, O0_ref=None, O0=None):
    """The GPU gates a kernel producing O would fail."""
    if np.abs(O - O_ref).max() > 2 * ATOL_MAX:
        return True
    if O0 is not None:
        dg, dr = O - O0, O_ref - O0_ref
        return np.linalg.norm(dg - dr) / np.linalg.norm(dr) > 2 * LR_SENS
    return False


@pytest.fixture(scope="module")
def decode():
    cfg, c, L = _decode_case()
    Q, K, V, pos = _parts(c, cfg.theta)
    S = K.shape[0]
    O, _ = oracle.attention(Q, K, V, pos, S)
    return cfg, c, L, Q, K, V, pos, O


@pytest.mark.parametrize("split", [1, 16, 31])
@pytest.mark.parametrize("fault", ["k_split_relative_rotation", "k_lr_dropped", "v_lr_dropped", "split_skipped"])
def test_decode_split_fault_is_caught(decode, split, fault):
    cfg, c, L, Q, K, V, pos, O = decode
    s0, s1 = split * L, (split + 1) * L
    Km, Vm = K.copy(), V.copy()
    Kb, Vb = f64(c["K_base"])[0], f64(c["V_base"])[0]
    if fault == "k_split_relative_rotation":
        # The split's tokens rebuilt as if they started at position 0.
        Km[s0:s1], _ = oracle.rebuild_kv(Kb[s0:s1], Vb[s0:s1], f64(c["L_k"])[0, s0:s1], None,
                                         f64(c["B_k"])[0], None, cfg.theta)
    elif fault == "k_lr_dropped":
        Km[s0:s1] = Kb[s0:s1]
    elif fault == "v_lr_dropped":
        Vm[s0:s1] = Vb[s0:s1]
    if fault == "split_skipped":
        keep = np.r_[0:s0, s1:K.shape[0]]
        Om, _ = oracle.attention(Q, Km[keep], Vm[keep], np.full_like(pos, len(keep) - 1), len(keep))
    else:
        Om, _ = oracle.attention(Q, Km, Vm, pos, K.shape[0])
    assert _caught(Om, O), np.abs(Om - O).max()


def test_decode_diagonal_masked_is_caught(decode):
    cfg, c, L, Q, K, V, pos, O = decode
    S = K.shape[0]
    Om, _ = oracle.attention(Q, K[: S - 1], V[: S - 1], np.full_like(pos, S - 2), S - 1)
    assert _caught(Om, O)


def test_decode_outputs_are_unit_scale_and_lr_driven(decode):
    cfg, c, L, Q, K, V, pos, O = decode
    assert 0.1 < np.abs(O).mean() < 1.0 and np.abs(O).max() < 4.0
    Kb, Vb = f64(c["K_base"])[0], f64(c["V_base"])[0]
    O0, _ = oracle.attention(Q, Kb, Vb, pos, K.shape[0])
    assert np.abs(O - O0).mean() > 0.05  # the LR terms move the outputs by O(0.1)


def test_prefill_tile_fault_is_caught():
    """Sampled queries of the 32k prefill (4096 tokens at 32768..36863): a
    fault in the LR term of one 64-token tile (at a tile boundary holding a
    planted key, or at the causal diagonal) is caught."""
    cfg = CONFIGS[3]
    S, n = cfg.context, cfg.prefill_tokens
    kv = S + n
    toks = [0, 31, 2047, 4095]
    pos = [list(range(S, kv))]
    must = [sorted({64 * 100 - 1, 64 * 100, 64 * 300, S + 31, S + 4095, kv - 1})]
    c = sharp_case(cfg, batch=1, n_tok=n, kv_len=[kv], positions=pos, s_cap=kv, seed=777,
                   must=must, per_query=lambda b, i, h: (1 + (i + h) % 4) if i in toks else 0, poison_tail=False)
    Q, K, V, p = _parts(c, cfg.theta)
    Q, p = Q[toks], p[toks]
    O, _ = oracle.attention(Q, K, V, p, kv)
    planted = sorted({t for (_, i, _, t) in c["plan"]})
    Kb = f64(c["K_base"])[0]
    Vb = f64(c["V_base"])[0]
    for t in (64 * 100, 64 * 300, S + 31, kv - 1):
        assert t in planted
        t0 = (t // 64) * 64
        for fault in ("k", "v"):
            Km, Vm = K.copy(), V.copy()
            if fault == "k":
                Km[t0:t0 + 64] = Kb[t0:t0 + 64]
            else:
                Vm[t0:t0 + 64] = Vb[t0:t0 + 64]
            Om, _ = oracle.attention(Q, Km, Vm, p, kv)
            assert _caught(Om, O), (t, fault, np.abs(Om - O).max())
