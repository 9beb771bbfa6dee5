"""The oracle against the facts that pin it (CPU only)."""
import numpy as np
import pytest

import oracle
import oracle_pins as pins


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    pin(oracle)


@pytest.mark.parametrize("d,theta", [(64, 1e4), (8, 5e5)])
def test_merged_weights_wider_heads(d, theta):
    pins.pin_merged_weights(oracle, seed=11, d=d, theta=theta, S=20, n_new=3)


def test_merged_weights_at_large_positions():
    # The LR term is rotated at each token's absolute position: check the
    # identity near position 65k by shifting the whole trajectory behind a
    # prefix of 65000 zero hidden states.
    pins.pin_merged_weights(oracle, seed=12, d=8, theta=1e4, S=40, n_new=1, t0=65000)


def test_tiny_workload_runs_and_is_finite():
    """The oracle finishes the tiny workload's attention in seconds."""
    from workload import CONFIGS, attention_case
    cfg = CONFIGS[1]
    S = cfg.context + cfg.prefill_tokens
    pos = [list(range(cfg.context, S))]
    case = attention_case(cfg, batch=1, n_tok=cfg.prefill_tokens, kv_len=[S], positions=pos,
                          s_cap=S + 8)
    f = lambda t: None if t is None else t.double().numpy()
    Bk = f(case["B_k"])
    Bv = f(case["B_v"])
    O, lse = oracle.lr_shared_attention(f(case["Q"]), f(case["K_base"]), f(case["V_base"]),
                                        f(case["L_k"]), f(case["L_v"]), Bk, Bv,
                                        case["positions"].numpy(), case["kv_len"].numpy(), cfg.theta)
    assert np.isfinite(O).all() and np.isfinite(lse).all()
