"""The oracle against hand-derived worked cases (tests/golden/worked_cases.json)."""
import json
import math
import os

import numpy as np

import oracle

CASES = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "worked_cases.json")))["cases"]


def _case(name):
    return next(c for c in CASES if c["name"] == name)


def test_golden_attention_cases():
    for c in CASES:
        if "Q" not in c:
            continue
        scale = math.sqrt(2.0) * math.log(3.0)
        Bk = np.array([c["B_k_unit"]]) * scale                   # [r, n_kv*d]
        Bv = np.array(c["B_v"])
        O, lse = oracle.lr_shared_attention(
            np.array(c["Q"])[None], np.array(c["K_base"])[None], np.array(c["V_base"])[None],
            np.array(c["L_k"])[None], np.array(c["L_v"])[None], Bk[None], Bv[None],
            np.array([c["positions"]]), [len(c["K_base"])], c["theta"])
        assert np.allclose(O[0], c["expected_O"], atol=1e-12), (c["name"], O)
        assert np.allclose(lse[0], c["expected_lse"], atol=1e-12), (c["name"], lse)


def test_golden_precompute():
    c = _case("precompute_two_agents")
    L = oracle.precompute_lr_cache(np.array(c["X"]), np.array(c["A_stack"]), 1, 2, 1)
    assert np.array_equal(L, np.array(c["expected_L"]))
