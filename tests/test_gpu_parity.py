"""GPU parity of every entry point against the fp64 oracle, at sizes the oracle
finishes in seconds (several tiles, ragged tails, GQA groups 1/4/5/8, ranks
8-64, head dims 64/128, every LR wiring), plus edge cases."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_34054_amd as prc
from gpu_cases import (ATOL_MAX, ATOL_MEAN, LR_SENS, LSE_ATOL, PRE_REL, attn_errors, f64,
                       gpu_attention, lse_error, oracle_attention, to_dev)
from workload import CONFIGS, Config, attention_case, precompute_case
from workload.gen import normal_bf16

pytestmark = pytest.mark.gpu


def mk_cfg(idx, n_q, n_kv, d, r, theta=1e4, hidden=256, n_agents=1):
    return Config(idx, "parity", hidden=hidden, n_q=n_q, n_kv=n_kv, head_dim=d, theta=theta,
                  n_agents=n_agents, rank=r, context=0, prefill_tokens=0, decode_batch=0, precompute_rows=0)


# ----------------------------------------------------------------- precompute
PRE_CASES = [
    # id, T, d_in, n_proj, N, r, tok_offset, s_cap
    ("tiny_c1", 528, 256, 2, 3, 8, 0, 528),
    ("ragged_tail", 77, 264, 2, 2, 16, 5, 100),
    ("r32_single_proj", 130, 512, 1, 5, 32, 3, 200),
    ("r64", 64, 128, 2, 1, 64, 0, 64),
    ("one_row", 1, 4096, 2, 8, 16, 31, 32),
    # 1-4 rows take the matrix-vector kernel (one wave per output column).
    ("gemv_t2_r8", 2, 4096, 2, 3, 8, 7, 9),
    ("gemv_t3_ragged_d_in", 3, 264, 2, 2, 16, 5, 100),
    ("gemv_t4_r64", 4, 520, 1, 3, 64, 0, 4),
    ("gemm_t5", 5, 520, 2, 2, 32, 1, 6),
    ("c2_chunk", 512, 4096, 2, 4, 16, 8192, 8704),
    ("c3_segment", 4096, 4096, 2, 8, 16, 32768, 36864),
    ("c4_chunk", 2048, 5120, 2, 6, 64, 0, 2048),
]


@pytest.mark.parametrize("cid,T,d_in,n_proj,N,r,off,s_cap", PRE_CASES, ids=[c[0] for c in PRE_CASES])
def test_precompute(cid, T, d_in, n_proj, N, r, off, s_cap):
    print(f"precompute {cid}", flush=True)
    cfg = mk_cfg(7, 4, 4, 64, r, hidden=d_in, n_agents=N)
    cfg = Config(**{**cfg.__dict__, "n_proj": n_proj})
    pc = precompute_case(cfg, T, seed_base=T)
    sentinel = 3.0
    L = torch.full((n_proj, N, s_cap, r), sentinel, dtype=torch.bfloat16, device="cuda")
    prc.precompute_lr_cache(pc["X"].cuda(), pc["A_stack"].cuda(), n_proj, N, r, L, tok_offset=off)
    torch.cuda.synchronize()
    ref = oracle.precompute_lr_cache(f64(pc["X"]), f64(pc["A_stack"]), n_proj, N, r)
    got = f64(L)
    rel = np.linalg.norm(got[:, :, off:off + T] - ref) / np.linalg.norm(ref)
    assert rel <= PRE_REL, rel
    # Rows outside the segment are untouched.
    assert (got[:, :, :off] == sentinel).all() and (got[:, :, off + T:] == sentinel).all()


def test_precompute_strided_rows():
    """X rows with a row stride larger than d_in (a view into a wider buffer)."""
    cfg = mk_cfg(8, 4, 4, 64, 16, hidden=256, n_agents=2)
    pc = precompute_case(cfg, 100)
    wide = torch.zeros(100, 384, dtype=torch.bfloat16)
    wide[:, :256] = pc["X"]
    L = torch.zeros((2, 2, 100, 16), dtype=torch.bfloat16, device="cuda")
    prc.precompute_lr_cache(wide.cuda()[:, :256], pc["A_stack"].cuda(), 2, 2, 16, L)
    torch.cuda.synchronize()
    ref = oracle.precompute_lr_cache(f64(pc["X"]), f64(pc["A_stack"]), 2, 2, 16)
    assert np.linalg.norm(f64(L) - ref) / np.linalg.norm(ref) <= PRE_REL


# ------------------------------------------------------- fused projection
# id, T, d_in, n_kv, d, n_proj, N, r, tok_offset, s_cap, theta
PROJ_CASES = [
    ("d128_ragged", 100, 256, 2, 128, 2, 3, 8, 5, 128, 5e5),
    ("d64_large_positions", 70, 264, 4, 64, 2, 2, 16, 10000, 10100, 1e4),
    ("single_token_append", 1, 512, 2, 128, 2, 4, 16, 333, 400, 5e5),
    # 1-4 rows take the matrix-vector kernel (keys rotated per RoPE pair).
    ("gemv_t3_d64_far_positions", 3, 264, 4, 64, 2, 2, 16, 60000, 60010, 1e4),
    ("gemv_t4_d128_r64", 4, 4096, 8, 128, 2, 3, 64, 65532, 65536, 5e5),
    ("r64_one_proj", 130, 320, 1, 128, 1, 3, 64, 0, 130, 5e5),
    # Enough 128-wide tiles (16 x 17) for the wide-tile kernel; ragged tokens.
    ("wide_tiles", 2000, 256, 8, 128, 2, 2, 16, 3, 2003, 5e5),
]


@pytest.mark.parametrize("case", PROJ_CASES, ids=[c[0] for c in PROJ_CASES])
def test_project_kv_and_lr(case):
    cid, T, d_in, n_kv, d, n_proj, N, r, off, s_cap, theta = case
    print(f"projection {cid}", flush=True)
    g = 900 + len(cid)
    X = normal_bf16((T, d_in), 1.0, g + 1)
    W = normal_bf16((d_in, 2 * n_kv * d), 1.0 / math.sqrt(d_in), g + 2)
    A_stack = normal_bf16((d_in, n_proj * N * r), 1.0 / math.sqrt(d_in), g + 3)
    sentinel = -7.0
    K = torch.full((s_cap, n_kv, d), sentinel, dtype=torch.bfloat16, device="cuda")
    V = torch.full_like(K, sentinel)
    L = torch.full((n_proj, N, s_cap, r), sentinel, dtype=torch.bfloat16, device="cuda")
    prc.project_kv_and_lr_cache(X.cuda(), W.cuda(), A_stack.cuda(), n_kv, d, n_proj, N, r, K, V, L,
                                rope_theta=theta, tok_offset=off)
    torch.cuda.synchronize()
    Wk, Wv = f64(W[:, : n_kv * d]), f64(W[:, n_kv * d:])
    Kr, Vr, Lr = oracle.project_kv_and_lr(f64(X), Wk, Wv, f64(A_stack), n_kv, n_proj, N, r,
                                          np.arange(off, off + T), theta)
    for name, got, ref in (("K", f64(K)[off:off + T], Kr), ("V", f64(V)[off:off + T], Vr),
                           ("L", f64(L)[:, :, off:off + T], Lr)):
        rel = np.linalg.norm(got - ref) / np.linalg.norm(ref)
        assert rel <= PRE_REL, (name, rel)
        # bf16 output rounding bounds each element by about 2^-8 of its size.
        assert np.max(np.abs(got - ref) - 2 ** -7 * np.abs(ref)) <= 2e-2, name
    # Rows outside the segment are untouched.
    for t in (K, V):
        out = torch.cat([t[:off], t[off + T:]]).float()
        assert (out == sentinel).all()
    out = torch.cat([L[:, :, :off], L[:, :, off + T:]], dim=2).float()
    assert (out == sentinel).all()
    # The LR part agrees with the precompute alone to about the last bf16
    # place: the two may tile the GEMM differently (the narrow one splits k
    # over its waves), so their fp32 sums differ in order, which moves values
    # near zero (cancellations) by a little more than their own ulp.
    L2 = torch.full_like(L, sentinel)
    prc.precompute_lr_cache(X.cuda(), A_stack.cuda(), n_proj, N, r, L2, tok_offset=off)
    torch.cuda.synchronize()
    a, b = L.float(), L2.float()
    assert ((a - b).abs() <= 2 ** -7 * b.abs() + 1e-3 * b.abs().max()).all()


def test_project_base_only():
    """n_agents = 0: the base projection alone (no LR buffers)."""
    T, d_in, n_kv, d, off, s_cap, theta = 65, 128, 2, 64, 7, 80, 5e5
    X = normal_bf16((T, d_in), 1.0, 951)
    W = normal_bf16((d_in, 2 * n_kv * d), 1.0 / math.sqrt(d_in), 952)
    K = torch.zeros((s_cap, n_kv, d), dtype=torch.bfloat16, device="cuda")
    V = torch.zeros_like(K)
    prc.project_kv_and_lr_cache(X.cuda(), W.cuda(), None, n_kv, d, 2, 0, 16, K, V, None, rope_theta=theta,
                                tok_offset=off)
    torch.cuda.synchronize()
    A0 = np.zeros((d_in, 0))
    Kr, Vr, _ = oracle.project_kv_and_lr(f64(X), f64(W[:, : n_kv * d]), f64(W[:, n_kv * d:]), A0, n_kv,
                                         2, 0, 16, np.arange(off, off + T), theta)
    for got, ref in ((f64(K)[off:off + T], Kr), (f64(V)[off:off + T], Vr)):
        assert np.linalg.norm(got - ref) / np.linalg.norm(ref) <= PRE_REL


# ------------------------------------------------------------------ attention
# id, d, r, n_q, n_kv, n_tok, kv_lens, s_cap, lr ("kv"|"v"|"k"|"none"), q_std, pos ("end"|"mid")
ATTN_CASES = [
    ("c1_prefill", 64, 8, 4, 4, 16, [528], 544, "kv", 1.0, "end"),
    ("c1_decode", 64, 8, 4, 4, 1, [528], 544, "kv", 1.0, "end"),
    ("g4_r16_prefill_ragged", 128, 16, 8, 2, 70, [300, 233], 320, "kv", 1.0, "end"),
    ("g4_r16_decode_ragged", 128, 16, 8, 2, 1, [1000, 77, 1], 1024, "kv", 1.0, "end"),
    ("g4_r16_decode_long", 128, 16, 8, 2, 1, [5000], 5000, "kv", 1.0, "end"),
    ("g5_r64_prefill", 128, 64, 10, 2, 37, [200, 150], 256, "kv", 1.0, "end"),
    ("g5_r64_decode", 128, 64, 10, 2, 1, [700, 64], 704, "kv", 1.0, "end"),
    ("g8_r32_prefill", 128, 32, 16, 2, 20, [150], 160, "kv", 1.0, "end"),
    ("g8_r32_decode", 128, 32, 16, 2, 1, [333], 340, "kv", 1.0, "end"),
    ("g1_d64_r16_prefill_2tiles", 64, 16, 4, 4, 130, [400], 400, "kv", 1.0, "end"),
    ("g1_d128_r8_decode", 128, 8, 2, 2, 1, [129], 136, "kv", 1.0, "end"),
    ("d64_g4_r32_prefill", 64, 32, 8, 2, 33, [97], 104, "kv", 1.0, "end"),
    ("qv_prefill", 128, 16, 8, 2, 40, [256], 256, "v", 1.0, "end"),
    ("qv_decode", 128, 16, 8, 2, 1, [512, 300], 512, "v", 1.0, "end"),
    # The paper's QV setting over its rank range (value LR only).
    ("qv_r8_prefill", 128, 8, 8, 2, 45, [190], 192, "v", 1.0, "end"),
    ("qv_r32_decode", 128, 32, 8, 2, 1, [700, 129], 704, "v", 1.0, "end"),
    ("qv_r64_prefill", 128, 64, 8, 2, 33, [260], 264, "v", 1.0, "end"),
    ("qv_r64_decode", 128, 64, 8, 2, 1, [333], 336, "v", 1.0, "end"),
    ("qv_d64_r32_prefill", 64, 32, 4, 4, 70, [140], 144, "v", 1.0, "end"),
    ("k_only_prefill", 128, 16, 8, 2, 24, [128], 136, "k", 1.0, "end"),
    ("k_only_decode", 64, 8, 4, 2, 1, [90], 96, "k", 1.0, "end"),
    ("plain_prefill", 128, 16, 8, 2, 50, [300], 304, "none", 1.0, "end"),
    ("plain_decode", 128, 16, 8, 2, 1, [2000, 1], 2000, "none", 1.0, "end"),
    # Sharp data (O(1) outputs decided by a few planted keys at split and tile
    # boundaries) is covered by the planted-key set in test_gpu_sharp.py.
    ("mid_positions_prefill", 128, 16, 8, 2, 12, [300], 304, "kv", 1.0, "mid"),
    ("mid_positions_decode", 128, 16, 8, 2, 1, [300, 500], 512, "kv", 1.0, "mid"),
    ("many_requests_decode", 64, 16, 8, 8, 1, [64, 65, 63, 1, 17, 200, 31, 128], 256, "kv", 1.0, "end"),
    # Prefill calls too small to fill the chip split their KV tiles (16+
    # tiles of 64 keys): partials per split, then the merge.  Shorter
    # requests of a ragged batch leave whole splits empty, and mid positions
    # leave the last splits past every row's causal limit.
    ("split_prefill_ragged", 128, 16, 8, 2, 40, [1500, 300, 64], 1536, "kv", 1.0, "end"),
    ("split_r64_prefill", 128, 64, 10, 2, 20, [2000], 2048, "kv", 1.0, "end"),
    ("split_r32_prefill", 128, 32, 16, 2, 9, [1100, 1031], 1152, "kv", 1.0, "end"),
    ("split_d64_r8_prefill", 64, 8, 4, 4, 16, [1200], 1216, "kv", 1.0, "end"),
    ("split_qv_prefill", 128, 16, 8, 2, 24, [1300], 1344, "v", 1.0, "end"),
    ("split_k_only_d64_r32_prefill", 64, 32, 8, 2, 17, [1025], 1088, "k", 1.0, "end"),
    ("split_plain_prefill", 128, 16, 8, 2, 30, [1800], 1856, "none", 1.0, "end"),
    ("split_mid_positions_prefill", 128, 16, 8, 2, 12, [3000], 3008, "kv", 1.0, "mid"),
]


def _positions(kv_lens, n_tok, mode):
    pos = []
    for kl in kv_lens:
        end = kl if mode == "end" else max(n_tok, kl // 2)
        pos.append(list(range(end - n_tok, end)))
    return pos


def _case(cid, d, r, n_q, n_kv, n_tok, kv_lens, s_cap, lr, q_std, pos_mode, seed=0):
    cfg = mk_cfg(10 + len(cid), n_q, n_kv, d, r)
    return cfg, attention_case(cfg, batch=len(kv_lens), n_tok=n_tok, kv_len=kv_lens,
                               positions=_positions(kv_lens, n_tok, pos_mode), s_cap=s_cap,
                               seed_base=seed + 100 * len(cid), lr_k=lr in ("kv", "k"), lr_v=lr in ("kv", "v"),
                               q_std=q_std)


@pytest.mark.parametrize("case", ATTN_CASES, ids=[c[0] for c in ATTN_CASES])
def test_attention(case):
    print(f"attention {case[0]}", flush=True)
    cfg, c = _case(*case)
    O, lse = gpu_attention(to_dev(c), cfg.theta)
    Oref, lref = oracle_attention(c, cfg.theta)
    mx, mean = attn_errors(O, Oref)
    assert mx <= ATOL_MAX and mean <= ATOL_MEAN, (mx, mean)
    assert lse_error(lse, lref) <= LSE_ATOL


@pytest.mark.parametrize("cid", ["c1_prefill", "g4_r16_decode_ragged", "g5_r64_prefill", "g4_r16_decode_long",
                                 "split_prefill_ragged", "split_r64_prefill", "split_qv_prefill"])
def test_lr_sensitivity(cid):
    """The LR term's contribution, O - O(B=0), is reproduced (a kernel that drops
    or mis-rotates the LR term fails this even when O itself is small)."""
    case = next(c for c in ATTN_CASES if c[0] == cid)
    cfg, c = _case(*case)
    g = to_dev(c)
    O, _ = gpu_attention(g, cfg.theta)
    z = dict(g)
    for k in ("B_k", "B_v"):
        if z[k] is not None:
            z[k] = torch.zeros_like(z[k])
    O0, _ = gpu_attention(z, cfg.theta)
    Oref, _ = oracle_attention(c, cfg.theta)
    O0ref, _ = oracle_attention(c, cfg.theta, zero_b=True)
    dg, dr = f64(O) - f64(O0), Oref - O0ref
    rel = np.linalg.norm(dg - dr) / np.linalg.norm(dr)
    assert rel <= LR_SENS, rel


def test_absent_lr_equals_zero_up_projection():
    cfg, c = _case("qv_decode", 128, 16, 8, 2, 1, [512, 300], 512, "kv", 1.0, "end")
    g = to_dev(c)
    for n_tok in (1,):
        zk = dict(g, B_k=torch.zeros_like(g["B_k"]))
        nk = dict(g, L_k=None, B_k=None)
        Oz, lz = gpu_attention(zk, cfg.theta)
        On, ln = gpu_attention(nk, cfg.theta)
        assert torch.equal(Oz, On) and torch.equal(lz, ln)


def test_deterministic():
    for case in (ATTN_CASES[2], ATTN_CASES[4]):
        cfg, c = _case(*case)
        g = to_dev(c)
        O1, l1 = gpu_attention(g, cfg.theta)
        O2, l2 = gpu_attention(g, cfg.theta)
        assert torch.equal(O1, O2) and torch.equal(l1, l2)


def test_rows_without_visible_keys():
    """kv_len = 0 or a position before the first key: O = 0, lse = -inf."""
    cfg = mk_cfg(40, 8, 2, 128, 16)
    for n_tok in (1, 3):
        c = attention_case(cfg, batch=2, n_tok=n_tok, kv_len=[0, 50], positions=[[5] * n_tok, [-1] * n_tok],
                           s_cap=64, poison_tail=False)
        O, lse = gpu_attention(to_dev(c), cfg.theta)
        assert (f64(O) == 0).all()
        assert np.isneginf(f64(lse)).all()


def test_shared_buffers_across_requests():
    """Stride-0 base cache, LR plane and up-projection shared by every request."""
    cfg = mk_cfg(41, 8, 2, 128, 16)
    c = attention_case(cfg, batch=1, n_tok=1, kv_len=[400], positions=[[399]], s_cap=400)
    g = to_dev(c)
    B = 3
    Q = normal_bf16((B, 1, 8, 128), 1.0, 4242).cuda()
    pos = torch.tensor([[399], [250], [10]], dtype=torch.int32, device="cuda")
    kvl = torch.tensor([400, 251, 11], dtype=torch.int32, device="cuda")
    O, _ = prc.lr_shared_attention(Q, g["K_base"], g["V_base"], g["L_k"], g["L_v"], g["B_k"], g["B_v"],
                                   pos, kvl, rope_theta=cfg.theta)
    torch.cuda.synchronize()
    for b in range(B):
        n = int(kvl[b])
        Oref, _ = oracle.lr_shared_attention(f64(Q[b:b + 1]), f64(c["K_base"])[:, :n], f64(c["V_base"])[:, :n],
                                             f64(c["L_k"])[:, :n], f64(c["L_v"])[:, :n], f64(c["B_k"]),
                                             f64(c["B_v"]), pos[b:b + 1].cpu().numpy(), [n], cfg.theta)
        mx, mean = attn_errors(O[b:b + 1], Oref)
        assert mx <= ATOL_MAX and mean <= ATOL_MEAN


# Several agents decoding over one shared base cache (request stride 0), each
# with its own LR plane, up-projections, query and position: the shared-base
# decode kernel, which reads each base tile once for all of them.
# id, d, r, n_q, n_kv, kv_lens, positions (None: kv_len - 1), s_cap, lr
SHARED_BASE_CASES = [
    ("sb_d128_r16_kv", 128, 16, 16, 4, [300, 299, 150, 1, 77, 300, 256, 33], None, 304, "kv"),
    ("sb_d64_r8_kv_two_groups", 64, 8, 8, 4, [90, 13, 64, 65, 1, 200, 199, 31, 128, 100, 7], None, 200, "kv"),
    ("sb_d128_r64_kv", 128, 64, 8, 2, [400, 390, 17, 256, 399], None, 400, "kv"),
    ("sb_d128_r32_qv", 128, 32, 16, 2, [130, 64, 1, 129, 100, 33, 64, 65, 128], None, 136, "v"),
    ("sb_plain", 128, 16, 8, 2, [222, 100, 222, 5], None, 224, "none"),
    ("sb_mid_positions", 128, 16, 8, 2, [500, 500, 500], [[100], [499], [250]], 512, "kv"),
    ("sb_long_splits", 128, 16, 8, 2, [5000, 4001, 4999], None, 5008, "kv"),
]


@pytest.mark.parametrize("case", SHARED_BASE_CASES, ids=[c[0] for c in SHARED_BASE_CASES])
def test_shared_base_decode(case):
    cid, d, r, n_q, n_kv, kv_lens, pos, s_cap, lr = case
    print(f"shared-base decode {cid}", flush=True)
    B = len(kv_lens)
    pos = [[k - 1] for k in kv_lens] if pos is None else pos
    cfg = mk_cfg(60 + len(cid), n_q, n_kv, d, r)
    c = attention_case(cfg, batch=B, n_tok=1, kv_len=kv_lens, positions=pos, s_cap=s_cap, seed_base=7 * len(cid),
                       lr_k=lr in ("kv", "k"), lr_v=lr in ("kv", "v"), poison_tail=False)
    # One base cache for every request, valid up to the longest request; each
    # request's own LR rows past its length are poisoned.
    top = max(kv_lens)
    for name in ("K_base", "V_base"):
        c[name] = c[name][:1].clone()
        c[name][0, top:] = float("nan")
    for name in ("L_k", "L_v"):
        if c[name] is not None:
            for b in range(B):
                c[name][b, kv_lens[b]:] = float("nan")
    g = to_dev(c)
    O, lse = gpu_attention(g, cfg.theta)
    Oref, lref = oracle_attention(c, cfg.theta)
    mx, mean = attn_errors(O, Oref)
    assert mx <= ATOL_MAX and mean <= ATOL_MEAN, (mx, mean)
    assert lse_error(lse, lref) <= LSE_ATOL


def test_custom_softmax_scale():
    cfg, c = _case("plain_prefill", 128, 16, 8, 2, 9, [100], 104, "kv", 1.0, "end")
    O, _ = gpu_attention(to_dev(c), cfg.theta, softmax_scale=0.05)
    Q = f64(c["Q"])
    Ks, Vs = oracle.materialize_agent_kv(f64(c["K_base"]), f64(c["V_base"]), f64(c["L_k"]), f64(c["L_v"]),
                                         f64(c["B_k"]), f64(c["B_v"]), [100], cfg.theta)
    Oref, _ = oracle.attention(Q[0], Ks[0], Vs[0], c["positions"].numpy()[0], 100, scale=0.05)
    mx, mean = attn_errors(O[0], Oref)
    assert mx <= ATOL_MAX and mean <= ATOL_MEAN


# ---------------------------------------------------------------- materialise
@pytest.mark.parametrize("cid", ["c1_prefill", "g5_r64_decode", "qv_decode", "k_only_decode"])
def test_materialize(cid):
    case = next(c for c in ATTN_CASES if c[0] == cid)
    cfg, c = _case(*case)
    g = to_dev(c)
    Kf, Vf = prc.materialize_agent_kv(g["K_base"], g["V_base"], g["L_k"], g["L_v"], g["B_k"], g["B_v"],
                                      g["kv_len"], rope_theta=cfg.theta)
    torch.cuda.synchronize()
    Ks, Vs = oracle.materialize_agent_kv(f64(c["K_base"]), f64(c["V_base"]), f64(c["L_k"]), f64(c["L_v"]),
                                         f64(c["B_k"]), f64(c["B_v"]), c["kv_len"].numpy(),
                                         cfg.theta)
    for b, n in enumerate(c["kv_len"].tolist()):
        for got, ref in ((f64(Kf)[b, :n], Ks[b]), (f64(Vf)[b, :n], Vs[b])):
            # One bf16 rounding of the rebuilt value: |err| <= 2^-8 |x| (+ fp32 slack).
            assert (np.abs(got - ref) <= np.abs(ref) * 2.0 ** -8 + 1e-3).all()
    # Materialise-then-attend matches the oracle too, and the fused path.
    O_m, _ = prc.lr_shared_attention(g["Q"], Kf, Vf, None, None, None, None, g["positions"], g["kv_len"],
                                     rope_theta=cfg.theta)
    O_f, _ = gpu_attention(g, cfg.theta)
    Oref, _ = oracle_attention(c, cfg.theta)
    mx, mean = attn_errors(O_m, Oref)
    assert mx <= ATOL_MAX and mean <= ATOL_MEAN
    assert (f64(O_m) - f64(O_f)).__abs__().max() <= ATOL_MAX


# ------------------------------------------------- the tiny workload, end to end
def test_tiny_workload_full_chain():
    """Hidden states -> frozen projections (oracle) -> LR precompute (GPU) ->
    LR-shared attention (GPU) for every agent, against the all-fp64 chain:
    this is Eq. 1 checked end to end on the GPU."""
    cfg = CONFIGS[1]
    from workload import lora_case
    S = cfg.context + cfg.prefill_tokens
    lc = lora_case(cfg, S)
    X, N, r, d = f64(lc["X"]), cfg.n_agents, cfg.rank, cfg.head_dim
    t = np.arange(S)
    Kb = oracle.rope((X @ f64(lc["W_k"])).reshape(S, cfg.n_kv, d), t[:, None], cfg.theta)
    Vb = (X @ f64(lc["W_v"])).reshape(S, cfg.n_kv, d)
    Q_all = oracle.rope((X @ f64(lc["W_q"])).reshape(S, cfg.n_q, d), t[:, None], cfg.theta)
    bf = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(torch.bfloat16)
    Kb_t, Vb_t, Q_t = bf(Kb)[None], bf(Vb)[None], bf(Q_all)
    L = torch.zeros((2, N, S, r), dtype=torch.bfloat16, device="cuda")
    prc.precompute_lr_cache(lc["X"].cuda(), lc["A_stack"].cuda(), 2, N, r, L)
    L_or = oracle.precompute_lr_cache(X, f64(lc["A_stack"]), 2, N, r)
    for n_tok in (cfg.prefill_tokens, 1):
        q_t = Q_t[S - n_tok:][None]
        pos = torch.arange(S - n_tok, S, dtype=torch.int32)[None]
        kvl = torch.tensor([S], dtype=torch.int32)
        for a in range(N):
            O, _ = prc.lr_shared_attention(q_t.cuda(), Kb_t.cuda(), Vb_t.cuda(), L[0, a][None], L[1, a][None],
                                           lc["B_k"][a][None].cuda(), lc["B_v"][a][None].cuda(),
                                           pos.cuda(), kvl.cuda(), rope_theta=cfg.theta)
            torch.cuda.synchronize()
            Oref, _ = oracle.lr_shared_attention(f64(q_t), f64(Kb_t), f64(Vb_t), L_or[0, a][None], L_or[1, a][None],
                                                 f64(lc["B_k"][a][None]), f64(lc["B_v"][a][None]),
                                                 pos.numpy(), kvl.numpy(), cfg.theta)
            mx, mean = attn_errors(O, Oref)
            assert mx <= ATOL_MAX and mean <= ATOL_MEAN, (n_tok, a, mx, mean)


def test_multi_turn_stack_chain():
    """The 32-layer multi-turn schedule at small scale (2 layers, 3 turns of
    256 tokens, 32-token prefills, 3 decode steps): per turn, a segment
    precompute per layer, a prefill whose LR rows come from a 32-row
    precompute, and decode steps that each append one LR row (1-row
    precompute) before attending.  Every attention output is checked against
    the oracle run on its own fp64 LR rows of the same hidden states; the
    last turn's decode loop, captured in a HIP graph, is replayed three times
    with eager work in between and must equal the eager outputs bitwise."""
    n_layers, turns, turn, n_pre, n_dec = 2, 3, 256, 32, 3
    hid, n_q, n_kv, d, r, N, theta = 256, 8, 2, 128, 16, 3, 5e5
    S_cap = turns * turn + n_pre + n_dec
    seed = iter(range(9100, 9999))

    def rnd(shape, std=1.0):
        return normal_bf16(shape, std, next(seed))

    K = [rnd((1, S_cap, n_kv, d)) for _ in range(n_layers)]
    V = [rnd((1, S_cap, n_kv, d)) for _ in range(n_layers)]
    A = [rnd((hid, 2 * N * r), 1.0 / math.sqrt(hid)) for _ in range(n_layers)]
    Bk = [rnd((N, r, n_kv * d), math.sqrt(0.02)) for _ in range(n_layers)]
    Bv = [rnd((N, r, n_kv * d), math.sqrt(0.02)) for _ in range(n_layers)]
    X_seg = [rnd((turn, hid)) for _ in range(turns)]
    X_pre = [rnd((n_pre, hid)) for _ in range(turns)]
    X_dec = [rnd((n_dec, hid)) for _ in range(turns)]
    Q_pre = rnd((1, n_pre, n_q, d))
    Q_dec = rnd((n_dec, 1, n_q, d))
    g = {k: [t.cuda() for t in v] for k, v in dict(K=K, V=V, A=A, Bk=Bk, Bv=Bv).items()}
    Lp = [torch.zeros((2, N, S_cap, r), dtype=torch.bfloat16, device="cuda") for _ in range(n_layers)]
    L_or = [np.zeros((2, N, S_cap, r)) for _ in range(n_layers)]
    Xg = {k: [t.cuda() for t in v] for k, v in dict(seg=X_seg, pre=X_pre, dec=X_dec).items()}
    Qg_pre, Qg_dec = Q_pre.cuda(), Q_dec.cuda()

    def append(l, X, Xc, off):
        prc.precompute_lr_cache(Xc, g["A"][l], 2, N, r, Lp[l], tok_offset=off)
        L_or[l][:, :, off:off + X.shape[0]] = oracle.precompute_lr_cache(f64(X), f64(A[l]), 2, N, r)

    def attend(k, l, Qc, Qh, pos, kvl, O):
        s, a = turn * (k + 1) + n_pre + n_dec, (k + 1) % N
        prc.lr_shared_attention(Qc, g["K"][l][:, :s], g["V"][l][:, :s], Lp[l][0, a, :s][None],
                                Lp[l][1, a, :s][None], g["Bk"][l][a:a + 1], g["Bv"][l][a:a + 1],
                                pos.cuda(), kvl.cuda(), rope_theta=theta, O=O)
        ref, _ = oracle.lr_shared_attention(f64(Qh), f64(K[l][:, :s]), f64(V[l][:, :s]), L_or[l][0, a, :s][None],
                                            L_or[l][1, a, :s][None], f64(Bk[l][a:a + 1]),
                                            f64(Bv[l][a:a + 1]), pos.numpy(), kvl.numpy(), theta)
        return ref

    checks = []
    for k in range(turns):
        T = turn * (k + 1)
        for l in range(n_layers):
            append(l, X_seg[k], Xg["seg"][k], T - turn)
        for l in range(n_layers):
            append(l, X_pre[k], Xg["pre"][k], T)
            O = torch.empty((1, n_pre, n_q, d), dtype=torch.bfloat16, device="cuda")
            pos = torch.arange(T, T + n_pre, dtype=torch.int32)[None]
            ref = attend(k, l, Qg_pre, Q_pre, pos, torch.tensor([T + n_pre], dtype=torch.int32), O)
            checks.append((("prefill", k, l), O, ref))
        for j in range(n_dec):
            p = T + n_pre + j
            for l in range(n_layers):
                append(l, X_dec[k][j:j + 1], Xg["dec"][k][j:j + 1], p)
                O = torch.empty((1, 1, n_q, d), dtype=torch.bfloat16, device="cuda")
                ref = attend(k, l, Qg_dec[j:j + 1], Q_dec[j:j + 1], torch.tensor([[p]], dtype=torch.int32),
                             torch.tensor([p + 1], dtype=torch.int32), O)
                checks.append((("decode", k, j, l), O, ref))
    torch.cuda.synchronize()
    for what, O, ref in checks:
        mx, mean = attn_errors(O, ref)
        assert mx <= ATOL_MAX and mean <= ATOL_MEAN, (what, mx, mean)

    # The last turn's decode loop as a HIP graph: device-resident positions,
    # preallocated outputs and workspace, nothing allocated inside.
    k = turns - 1
    T = turn * turns
    s, a = T + n_pre + n_dec, turns % N
    pos_d = torch.tensor([[T + n_pre + j] for j in range(n_dec)], dtype=torch.int32, device="cuda")
    kvl_d = pos_d[:, 0] + 1
    O_all = torch.empty((n_dec, n_layers, 1, 1, n_q, d), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(1 << 20, dtype=torch.uint8, device="cuda")

    def loop():
        for j in range(n_dec):
            for l in range(n_layers):
                prc.precompute_lr_cache(Xg["dec"][k][j:j + 1], g["A"][l], 2, N, r, Lp[l], tok_offset=T + n_pre + j)
                prc.lr_shared_attention(Qg_dec[j:j + 1], g["K"][l][:, :s], g["V"][l][:, :s],
                                        Lp[l][0, a, :s][None], Lp[l][1, a, :s][None], g["Bk"][l][a:a + 1],
                                        g["Bv"][l][a:a + 1], pos_d[j:j + 1], kvl_d[j:j + 1], rope_theta=theta,
                                        O=O_all[j, l], workspace=ws)

    loop()
    torch.cuda.synchronize()
    eager = O_all.clone()
    for (what, O, _) in checks:
        if what[0] == "decode" and what[1] == k:
            assert torch.equal(O, eager[what[2], what[3]]), what
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        loop()
    for rep in range(3):
        O_all.zero_()
        # Eager work between replays: a prefill over the same caches.
        prc.lr_shared_attention(Qg_pre, g["K"][0][:, :s], g["V"][0][:, :s], Lp[0][0, a, :s][None],
                                Lp[0][1, a, :s][None], g["Bk"][0][a:a + 1], g["Bv"][0][a:a + 1],
                                torch.arange(T, T + n_pre, dtype=torch.int32, device="cuda")[None],
                                torch.tensor([T + n_pre], dtype=torch.int32, device="cuda"), rope_theta=theta)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(O_all, eager), rep


@pytest.mark.parametrize("rank", [16, 32, 64])
def test_split_prefill_without_lr_ignores_dims_rank(rank):
    """A plain call (no LR cache) whose dims still carry a built rank: the
    header says the rank is then ignored, so the split prefill's partials and
    their merge must agree on the layout whatever dims.rank says."""
    import ctypes
    from paper_2609_34054_amd.binding import lib, make_dims
    print(f"plain split prefill with dims.rank={rank}", flush=True)
    cfg, c = _case("split_plain_prefill", 128, 16, 8, 2, 30, [1800], 1856, "none", 1.0, "end")
    g = to_dev(c)
    dims = make_dims(g["Q"], g["K_base"], None, None, None, None, cfg.theta)
    dims.rank = rank
    need = lib().lr_shared_attention_workspace_size(ctypes.byref(dims))
    assert need > 0  # the call splits its KV tiles
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    O = torch.empty_like(g["Q"])
    lse = torch.empty(g["Q"].shape[:3], dtype=torch.float32, device="cuda")
    p = lambda t: ctypes.c_void_p(t.data_ptr())
    st = lib().lr_shared_attention(ctypes.byref(dims), p(g["Q"]), p(g["K_base"]), p(g["V_base"]), None, None,
                                   None, None, p(g["positions"]), p(g["kv_len"]), p(O), p(lse), p(ws), need,
                                   ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == 0, lib().prc_last_error()
    torch.cuda.synchronize()
    Oref, lref = oracle_attention(c, cfg.theta)
    mx, mean = attn_errors(O, Oref)
    assert mx <= ATOL_MAX and mean <= ATOL_MEAN, (mx, mean)
    assert lse_error(lse, lref) <= LSE_ATOL
