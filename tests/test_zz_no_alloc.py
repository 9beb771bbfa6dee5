"""lr_shared_attention_noalloc, the entry point that allocates nothing: its split
partials live in the library's static per-device workspace.  Called through
the C ABI and checked against lr_shared_attention (which takes a caller
workspace) on the same inputs, twice in a row with the second call smaller,
and against the fp64 oracle."""
import ctypes

import pytest
import torch

from gpu_cases import ATOL_MAX, ATOL_MEAN, LSE_ATOL, attn_errors, lse_error, oracle_attention, to_dev
from paper_2609_34054_amd.binding import lib, make_dims
from workload import Config, attention_case

pytestmark = pytest.mark.gpu


def _cfg(idx, n_q, n_kv, d, r):
    return Config(idx, "noalloc", hidden=256, n_q=n_q, n_kv=n_kv, head_dim=d, theta=5e5, n_agents=1, rank=r,
                  context=0, prefill_tokens=0, decode_batch=0, precompute_rows=0)


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _run(noalloc, dims, g):
    O = torch.full_like(g["Q"], float("nan"))
    lse = torch.full(g["Q"].shape[:3], float("nan"), dtype=torch.float32, device="cuda")
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    args = [ctypes.byref(dims), _p(g["Q"]), _p(g["K_base"]), _p(g["V_base"]), _p(g["L_k"]), _p(g["L_v"]),
            _p(g["B_k"]), _p(g["B_v"]), _p(g["positions"]), _p(g["kv_len"]), _p(O), _p(lse)]
    if noalloc:
        st = lib().lr_shared_attention_noalloc(*args, stream)
    else:
        need = lib().lr_shared_attention_workspace_size(ctypes.byref(dims))
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device="cuda")
        st = lib().lr_shared_attention(*args, _p(ws), need, stream)
    assert st == 0, lib().prc_last_error()
    torch.cuda.synchronize()
    return O, lse


# (id, d, r, n_q, n_kv, n_tok, kv_lens, s_cap): each pair runs larger, then smaller.
PAIRS = [
    (("decode_big", 128, 16, 32, 8, 1, [6000, 4100, 5999, 1], 6016),
     ("decode_small", 128, 16, 32, 8, 1, [700, 3], 704)),
    (("split_prefill_big", 128, 64, 10, 2, 20, [2000, 1500], 2048),
     ("split_prefill_small", 128, 64, 10, 2, 7, [1100], 1152)),
]


@pytest.mark.parametrize("pair", PAIRS, ids=[p[0][0] for p in PAIRS])
def test_noalloc_matches_workspace_call(pair):
    for cid, d, r, n_q, n_kv, n_tok, kv_lens, s_cap in pair:
        print(f"noalloc {cid}", flush=True)
        cfg = _cfg(70 + len(cid), n_q, n_kv, d, r)
        pos = [list(range(k - n_tok, k)) for k in kv_lens]
        c = attention_case(cfg, batch=len(kv_lens), n_tok=n_tok, kv_len=kv_lens, positions=pos, s_cap=s_cap,
                           seed_base=31 * len(cid))
        g = to_dev(c)
        dims = make_dims(g["Q"], g["K_base"], g["L_k"], g["L_v"], g["B_k"], g["B_v"], cfg.theta)
        assert lib().lr_shared_attention_workspace_size(ctypes.byref(dims)) > 0  # partials are used
        O_ws, lse_ws = _run(False, dims, g)
        O_na, lse_na = _run(True, dims, g)
        assert torch.equal(O_na, O_ws) and torch.equal(lse_na, lse_ws)
        Oref, lref = oracle_attention(c, cfg.theta)
        mx, mean = attn_errors(O_na, Oref)
        assert mx <= ATOL_MAX and mean <= ATOL_MEAN, (cid, mx, mean)
        assert lse_error(lse_na, lref) <= LSE_ATOL


def test_noalloc_refuses_calls_beyond_its_workspace():
    cfg = _cfg(90, 32, 8, 128, 16)
    c = attention_case(cfg, batch=1, n_tok=1, kv_len=[64], positions=[[63]], s_cap=64, poison_tail=False)
    g = to_dev(c)
    dims = make_dims(g["Q"], g["K_base"], g["L_k"], g["L_v"], g["B_k"], g["B_v"], cfg.theta)
    dims.batch = 4096  # 4096 requests at the same (shared) buffers need far more partials
    dims.kv_req_stride = dims.l_req_stride = dims.b_req_stride = 0
    assert lib().lr_shared_attention_workspace_size(ctypes.byref(dims)) > 32 << 20
    O = torch.empty(1, dtype=torch.bfloat16, device="cuda")
    st = lib().lr_shared_attention_noalloc(ctypes.byref(dims), _p(g["Q"]), _p(g["K_base"]), _p(g["V_base"]),
                                           _p(g["L_k"]), _p(g["L_v"]), _p(g["B_k"]), _p(g["B_v"]),
                                           _p(g["positions"]), _p(g["kv_len"]), _p(O), None, None)
    assert st == 5, st  # PRC_EWORKSPACE, nothing launched
