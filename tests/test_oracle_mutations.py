"""Plant plausible mistakes in a copy of the oracle; the pins must catch each.

The mistakes are planted on the CPU, in a private copy of the oracle's source;
the real oracle module is never modified.
"""
import importlib.util
import os
import types

import pytest

import oracle_pins as pins

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "oracle", "precache_oracle.py")

MUTATIONS = {
    "rope_sign": ("lo * c - hi * s", "lo * c + hi * s"),
    "rope_frequency": ("-2.0 * j / d", "-1.0 * j / d"),
    "rope_pairing_interleaved": ("lo, hi = x[..., : d // 2], x[..., d // 2:]",
                                 "lo, hi = x[..., 0::2], x[..., 1::2]"),
    "lr_key_not_rotated": ("K = K + rope(E, t[:, None], theta)", "K = K + E"),
    "lr_key_rotated_at_t_plus_1": ("t = np.arange(S, dtype=np.float64)",
                                   "t = np.arange(1, S + 1, dtype=np.float64)"),
    "lr_value_dropped": ("V = V + (_f64(L_v)[:S] @ _f64(B_v)).reshape(S, n_kv, d)", "V = V"),
    "lr_key_head_split_transposed": ("E = (_f64(L_k)[:S] @ _f64(B_k)).reshape(S, n_kv, d)",
                                     "E = (_f64(L_k)[:S] @ _f64(B_k)).reshape(S, d, n_kv).transpose(0, 2, 1)"),
    "lr_value_head_split_transposed": ("V = V + (_f64(L_v)[:S] @ _f64(B_v)).reshape(S, n_kv, d)",
                                       "V = V + (_f64(L_v)[:S] @ _f64(B_v)).reshape(S, d, n_kv).transpose(0, 2, 1)"),
    "gqa_mapping_modulo": ("K[:kv_len, g, :].T", "K[:kv_len, h % n_kv, :].T"),
    "value_head_mapping": ("V[:kv_len, h // group, :]", "V[:kv_len, h % n_kv, :]"),
    "causal_mask_strict": ("np.arange(kv_len)[None, :] <= np.asarray(positions)",
                           "np.arange(kv_len)[None, :] < np.asarray(positions)"),
    "softmax_scale_1_over_d": ("scale = 1.0 / np.sqrt(d)", "scale = 1.0 / d"),
    "softmax_unnormalised": ("return e / z, (m + np.log(z))[..., 0]", "return e, (m + np.log(z))[..., 0]"),
    "lse_missing_max": ("return e / z, (m + np.log(z))[..., 0]", "return e / z, (np.log(z))[..., 0]"),
    "precompute_agent_major": ("col = (p * n_agents + a) * rank", "col = (a * n_proj + p) * rank"),
    "precompute_transposed_block": ("L[p, a] = X @ A_stack[:, col: col + rank]",
                                    "L[p, a] = X @ A_stack[:, col: col + rank][::-1]"),
    "projection_value_uses_key_weights": ("V = (X @ W_v).reshape(T, n_kv, d)", "V = (X @ W_k).reshape(T, n_kv, d)"),
    "projection_key_unrotated": ("K = rope(K, np.asarray(positions, dtype=np.float64)[:, None], theta)", "K = K"),
    "projection_key_head_split_transposed": ("K = (X @ W_k).reshape(T, n_kv, d)",
                                             "K = (X @ W_k).reshape(T, d, n_kv).transpose(0, 2, 1)"),
    "merge_unshifted_lse": ("return O, m + np.log(z)", "return O, np.log(z)"),
    "merge_unweighted": ("O = sum(w[i][..., None] * np.asarray(p[0], dtype=np.float64)",
                         "O = sum(np.asarray(p[0], dtype=np.float64)"),
}


def _mutant(name, old, new):
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation {name}: target text not found in the oracle"
    mod = types.ModuleType(f"oracle_mutant_{name}")
    exec(compile(src.replace(old, new), f"<mutant {name}>", "exec"), mod.__dict__)
    return mod


def test_unmutated_copy_passes():
    mod = types.ModuleType("oracle_copy")
    exec(compile(open(SRC).read(), "<copy>", "exec"), mod.__dict__)
    for pin in pins.ALL_PINS:
        pin(mod)


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch(name):
    old, new = MUTATIONS[name]
    mod = _mutant(name, old, new)
    caught = []
    for pin in pins.ALL_PINS:
        try:
            pin(mod)
        except (AssertionError, ValueError, IndexError, FloatingPointError):
            caught.append(pin.__name__)
    assert caught, f"no pin detects the planted mistake '{name}'"
