"""The checked build (libprecache_checked.so): device-resident kv_len and
query positions are checked on the device before a call's kernels run.
Valid inputs give the release library's outputs bit for bit; a position
outside [0, kv_len[b]) or a kv_len outside [1, s_cap] returns PRC_EDEVDATA
naming the first offender, and nothing is launched (the outputs keep their
sentinel).  Every invalid case is rejected before any attention kernel runs."""
import pytest
import torch

import paper_2609_34054_amd as prc
from paper_2609_34054_amd.binding import use_checked_library
from workload import CONFIGS, attention_case

pytestmark = pytest.mark.gpu
EDEVDATA = 8


@pytest.fixture
def checked():
    use_checked_library(True)
    assert prc.lib().prc_device_checks() == 1
    yield
    use_checked_library(False)


def _case(n_tok, kv_lens, seed):
    cfg = CONFIGS[1]
    s_cap = -(-max(kv_lens) // 64) * 64
    pos = [list(range(k - n_tok, k)) for k in kv_lens]
    c = attention_case(cfg, batch=len(kv_lens), n_tok=n_tok, kv_len=kv_lens, positions=pos, s_cap=s_cap,
                       seed_base=seed, poison_tail=False)
    return cfg, {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in c.items()}, s_cap


def _call(cfg, g, O=None):
    out, _ = prc.lr_shared_attention(g["Q"], g["K_base"], g["V_base"], g["L_k"], g["L_v"], g["B_k"], g["B_v"],
                                     g["positions"], g["kv_len"], rope_theta=cfg.theta, O=O)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("n_tok,kv_lens", [(1, [700, 333, 64]), (24, [530, 200])], ids=["decode", "prefill"])
def test_checked_build_matches_release_on_valid_inputs(n_tok, kv_lens):
    cfg, g, _ = _case(n_tok, kv_lens, 900 + n_tok)
    ref = _call(cfg, g)
    use_checked_library(True)
    try:
        out = _call(cfg, g)
    finally:
        use_checked_library(False)
    assert torch.equal(out, ref)


@pytest.mark.parametrize("n_tok", [1, 24], ids=["decode", "prefill"])
def test_position_past_kv_len_is_reported(checked, n_tok):
    cfg, g, _ = _case(n_tok, [530, 300], 910 + n_tok)
    # Request 1, token n_tok - 1: one past its last valid key; request 1,
    # token 0 also bad when n_tok > 1 (the lower token is the one reported).
    g["positions"][1, n_tok - 1] = int(g["kv_len"][1])
    if n_tok > 1:
        g["positions"][1, 0] = -3
    O = torch.full_like(g["Q"], 7.0)
    with pytest.raises(prc.PrecacheError) as e:
        _call(cfg, g, O=O)
    assert e.value.status == EDEVDATA
    bad_tok = 0 if n_tok > 1 else n_tok - 1
    assert f"positions[1][{bad_tok}]" in str(e.value)
    assert bool((O == 7.0).all())  # nothing launched


@pytest.mark.parametrize("bad", [0, -5, "over"])
def test_kv_len_out_of_range_is_reported(checked, bad):
    cfg, g, s_cap = _case(1, [400, 300, 200], 920)
    g["kv_len"][2] = s_cap + 1 if bad == "over" else bad
    g["positions"][0, 0] = 10_000  # a position fault in an earlier request ...
    g["kv_len"][0] = 400
    O = torch.full_like(g["Q"], 7.0)
    with pytest.raises(prc.PrecacheError) as e:
        _call(cfg, g, O=O)
    assert e.value.status == EDEVDATA
    assert "positions[0][0]" in str(e.value)  # ... is found first (lowest request)
    g["positions"][0, 0] = 399
    with pytest.raises(prc.PrecacheError) as e:
        _call(cfg, g, O=O)
    assert e.value.status == EDEVDATA and "kv_len[2]" in str(e.value)
    assert bool((O == 7.0).all())


def test_materialize_checks_kv_len(checked):
    cfg, g, s_cap = _case(1, [300, 200], 930)
    g["kv_len"][1] = s_cap + 64
    K = torch.full_like(g["K_base"], 3.0)
    V = torch.full_like(g["V_base"], 3.0)
    with pytest.raises(prc.PrecacheError) as e:
        prc.materialize_agent_kv(g["K_base"], g["V_base"], g["L_k"], g["L_v"], g["B_k"], g["B_v"], g["kv_len"],
                                 rope_theta=cfg.theta, K_full=K, V_full=V)
    assert e.value.status == EDEVDATA and "kv_len[1]" in str(e.value)
    torch.cuda.synchronize()
    assert bool((K == 3.0).all()) and bool((V == 3.0).all())
