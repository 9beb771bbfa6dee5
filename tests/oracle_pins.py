"""Pins that tie the fp64 oracle to facts fixed by the paper or by mathematics.

Each ``pin_*`` takes an oracle module (the real one, or a copy with a planted
mistake) and raises ``AssertionError`` when the oracle contradicts the fact.
None of them re-types an oracle formula; each compares the oracle with an
independently written route to the same number:

* pin_merged_weights   Eq. 1 (Sec. 2.1) + App. D.2: base cache plus LR cache must
                       equal attention with the explicitly merged weights W + A B,
                       by brute force with a loop-based RoPE (2x2 rotation per pair).
* pin_plain_attention  B = 0 reduces to plain attention over the base cache (the
                       FullShared case, Sec. 2.2): torch's scaled_dot_product_attention
                       in float64 is the independent routine; an absent LR cache
                       equals B = 0; lse equals torch.logsumexp.
* pin_softmax_rows     softmax rows sum to one, masked entries are exactly zero.
* pin_rope             rotate-half RoPE: identity at position 0, norm preserving,
                       relative-position property, explicit 2x2 rotation matrices,
                       and hand-derived closed forms (omega_0 = 1, omega_{d/4} =
                       theta^(-1/2)).
* pin_value_assoc      App. D.2: P (V_base + L_v B_v) = P V_base + (P L_v) B_v.
* pin_closed_forms     one visible key gives its value; Q = 0 gives the mean of
                       the visible values; identical keys give uniform weights.
* pin_permutation      without LR and without a mask, key order is irrelevant.
* pin_split_merge      log-sum-exp merge of two disjoint key ranges equals the
                       whole range (the identity split-KV decoding relies on).
* pin_precompute       Sec. 3.1 precompute: each agent's block equals X A_a, by a
                       naive triple loop.
* pin_golden           hand-derived worked cases (tests/golden/worked_cases.json).
"""
from __future__ import annotations

import math

import numpy as np
import torch

RTOL_EXACT = 1e-10


def _rng(seed):
    return np.random.default_rng(seed)


# ---------------------------------------------------------------------------
# Independent helpers (written without the oracle's vectorised formulas)
# ---------------------------------------------------------------------------
def loop_rope(vec, pos, theta):
    """RoPE of one vector by explicit 2x2 rotations of the pairs (j, j + d/2)."""
    d = len(vec)
    out = np.array(vec, dtype=np.float64)
    for j in range(d // 2):
        phi = pos * math.pow(theta, -2.0 * j / d)
        rot = np.array([[math.cos(phi), -math.sin(phi)],
                        [math.sin(phi), math.cos(phi)]])
        out[[j, j + d // 2]] = rot @ np.array([vec[j], vec[j + d // 2]])
    return out


def loop_attention(Q, K, V, positions, group, scale):
    """Causal GQA attention by per-query loops (Q [n, n_q, d], K/V [S, n_kv, d])."""
    n_tok, n_q, d = Q.shape
    O = np.zeros((n_tok, n_q, V.shape[2]))
    for i in range(n_tok):
        for h in range(n_q):
            g = h // group
            vis = [t for t in range(K.shape[0]) if t <= positions[i]]
            sc = [float(np.dot(Q[i, h], K[t, g])) * scale for t in vis]
            mx = max(sc)
            w = [math.exp(s - mx) for s in sc]
            z = sum(w)
            O[i, h] = sum((wt / z) * V[t, g] for wt, t in zip(w, vis))
    return O


def _tiny(seed, d=8, n_q=4, n_kv=2, S=24, r=4, hidden=16, n_agents=3):
    g = _rng(seed)
    return dict(
        d=d, n_q=n_q, n_kv=n_kv, S=S, r=r, hidden=hidden, N=n_agents,
        X=g.standard_normal((S, hidden)),
        Wq=g.standard_normal((hidden, n_q * d)) / math.sqrt(hidden),
        Wk=g.standard_normal((hidden, n_kv * d)) / math.sqrt(hidden),
        Wv=g.standard_normal((hidden, n_kv * d)) / math.sqrt(hidden),
        Ak=g.standard_normal((n_agents, hidden, r)) / math.sqrt(hidden),
        Av=g.standard_normal((n_agents, hidden, r)) / math.sqrt(hidden),
        Bk=g.standard_normal((n_agents, r, n_kv * d)) * 0.5,
        Bv=g.standard_normal((n_agents, r, n_kv * d)) * 0.5,
    )


# ---------------------------------------------------------------------------
# Pins
# ---------------------------------------------------------------------------
def pin_merged_weights(orc, seed=1, d=8, theta=500.0, S=24, n_new=5, t0=0):
    """(a) Eq. 1: base cache + LR cache == attention with merged weights W + A B.

    With ``t0 > 0`` the trajectory is preceded by t0 all-zero hidden states, so
    its S tokens sit at absolute positions t0 .. t0 + S - 1 (a zero state has
    zero keys, values and LR rows, in both routes alike)."""
    c = _tiny(seed, d=d, S=S)
    n_q, n_kv, r, N = c["n_q"], c["n_kv"], c["r"], c["N"]
    X = np.concatenate([np.zeros((t0, c["hidden"])), c["X"]])
    n = t0 + S
    group = n_q // n_kv
    pos = np.arange(n - n_new, n)
    scale = 1.0 / math.sqrt(d)

    def keys(Wk):
        K = np.zeros((n, n_kv, d))
        for t in range(t0, n):
            K[t] = np.stack([loop_rope((X[t] @ Wk)[g * d:(g + 1) * d], t, theta) for g in range(n_kv)])
        return K

    # Oracle route: precompute every agent's LR caches from X (Sec. 3.1), base
    # caches from the frozen weights, then LR-shared attention.
    A_stack = np.concatenate([c["Ak"][a] for a in range(N)] + [c["Av"][a] for a in range(N)], axis=1)
    L = orc.precompute_lr_cache(X, A_stack, 2, N, r)
    Kb = keys(c["Wk"])
    Vb = (X @ c["Wv"]).reshape(n, n_kv, d)
    Q = np.stack([np.stack([loop_rope((X[p] @ c["Wq"])[h * d:(h + 1) * d], p, theta)
                            for h in range(n_q)]) for p in pos])
    for a in range(N):
        O, _ = orc.lr_shared_attention(Q[None], Kb[None], Vb[None], L[0, a][None], L[1, a][None],
                                       c["Bk"][a][None], c["Bv"][a][None], pos[None], [n], theta)
        # Merged route: the adapted projections of Eq. 1, written out.
        Wk_a = c["Wk"] + c["Ak"][a] @ c["Bk"][a]
        Wv_a = c["Wv"] + c["Av"][a] @ c["Bv"][a]
        Kf = keys(Wk_a)
        Vf = (X @ Wv_a).reshape(n, n_kv, d)
        ref = loop_attention(Q, Kf, Vf, pos, group, scale)
        err = np.abs(O[0] - ref).max()
        assert err <= RTOL_EXACT * max(1.0, np.abs(ref).max()), f"agent {a}: merged-weights mismatch {err}"


def pin_plain_attention(orc, seed=2, d=16, n_q=6, n_kv=2, S=40, n_tok=7, theta=1e4):
    """(b) B = 0 (and an absent LR cache) reduces to plain attention."""
    g = _rng(seed)
    r = 4
    Q = g.standard_normal((1, n_tok, n_q, d))
    Kb = g.standard_normal((1, S, n_kv, d))
    Vb = g.standard_normal((1, S, n_kv, d))
    Lk = g.standard_normal((1, S, r))
    Lv = g.standard_normal((1, S, r))
    Z = np.zeros((1, r, n_kv * d))
    pos = np.sort(g.choice(np.arange(3, S), size=n_tok, replace=False))[None]
    O0, lse0 = orc.lr_shared_attention(Q, Kb, Vb, Lk, Lv, Z, Z, pos, [S], theta)
    On, lsen = orc.lr_shared_attention(Q, Kb, Vb, None, None, None, None, pos, [S], theta)
    assert np.abs(O0 - On).max() <= RTOL_EXACT, "absent LR cache differs from B = 0"
    assert np.abs(lse0 - lsen).max() <= RTOL_EXACT
    group = n_q // n_kv
    q = torch.from_numpy(Q[0]).permute(1, 0, 2)                          # [n_q, n_tok, d]
    k = torch.from_numpy(Kb[0]).permute(1, 0, 2).repeat_interleave(group, 0)  # [n_q, S, d]
    v = torch.from_numpy(Vb[0]).permute(1, 0, 2).repeat_interleave(group, 0)
    mask = torch.from_numpy(np.arange(S)[None, :] <= pos[0][:, None])   # [n_tok, S]
    ref = torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=mask)
    ref = ref.permute(1, 0, 2).numpy()
    assert np.abs(O0[0] - ref).max() <= RTOL_EXACT, "B = 0 differs from scaled_dot_product_attention"
    sc = torch.matmul(q, k.transpose(1, 2)) / math.sqrt(d)
    sc = sc.masked_fill(~mask, float("-inf"))
    lse_ref = torch.logsumexp(sc, dim=-1).permute(1, 0).numpy()
    assert np.abs(lse0[0] - lse_ref).max() <= RTOL_EXACT, "lse differs from torch.logsumexp"


def pin_softmax_rows(orc, seed=3, d=16, n_q=4, n_kv=4, S=33, n_tok=9):
    """(c) Softmax rows sum to one; masked keys get exactly zero weight."""
    g = _rng(seed)
    Q = g.standard_normal((n_tok, n_q, d)) * 3
    K = g.standard_normal((S, n_kv, d))
    pos = np.arange(S - n_tok, S) - 4
    P, _ = orc.attention_probs(Q, K, pos, S)
    assert np.abs(P.sum(-1) - 1).max() <= 1e-12, "softmax rows do not sum to 1"
    assert (P >= 0).all()
    for i in range(n_tok):
        assert (P[i, :, pos[i] + 1:] == 0).all(), "masked key got weight"
        assert (P[i, :, : pos[i] + 1] > 0).all(), "visible key got no weight"


def pin_rope(orc, seed=4):
    g = _rng(seed)
    for d, theta in ((8, 1e4), (64, 1e4), (128, 5e5)):
        x = g.standard_normal(d)
        assert np.abs(orc.rope(x, 0, theta) - x).max() == 0, "rope at position 0 is not the identity"
        for t in (1, 17, 4099, 65535):
            y = orc.rope(x, t, theta)
            assert abs(np.linalg.norm(y) - np.linalg.norm(x)) <= 1e-12 * np.linalg.norm(x)
            assert np.abs(y - loop_rope(x, t, theta)).max() <= 1e-10, "rope differs from 2x2 rotations"
        q, k = g.standard_normal(d), g.standard_normal(d)
        for m, n in ((5, 2), (300, 297), (70000, 69997)):
            lhs = float(orc.rope(q, m, theta) @ orc.rope(k, n, theta))
            rhs = float(orc.rope(q, m - n, theta) @ k)
            assert abs(lhs - rhs) <= 1e-9, "rope scores are not relative-position only"
    # Hand-derived closed forms: omega_0 = 1 and omega_{d/4} = theta^(-1/2).
    d = 64
    e0 = np.zeros(d); e0[0] = 1.0
    y = orc.rope(e0, 2.5, 1e4)
    assert abs(y[0] - math.cos(2.5)) < 1e-15 and abs(y[d // 2] - math.sin(2.5)) < 1e-15
    e16 = np.zeros(d); e16[16] = 1.0
    y = orc.rope(e16, 100, 1e4)          # omega_16 = 1e4^(-1/2) = 0.01 -> angle 1 rad
    assert abs(y[16] - math.cos(1.0)) < 1e-12 and abs(y[48] - math.sin(1.0)) < 1e-12
    assert np.abs(np.delete(y, [16, 48])).max() == 0
    # Batched positions broadcast over leading axes.
    xs = g.standard_normal((5, 3, 8))
    ys = orc.rope(xs, np.arange(5)[:, None], 1e4)
    for t in range(5):
        for h in range(3):
            assert np.abs(ys[t, h] - loop_rope(xs[t, h], t, 1e4)).max() <= 1e-12


def pin_value_assoc(orc, seed=5, d=16, n_q=4, n_kv=2, S=30, n_tok=4, r=6, theta=1e4):
    """App. D.2: P (V_base + L_v B_v) = P V_base + (P L_v) B_v."""
    g = _rng(seed)
    Q = g.standard_normal((n_tok, n_q, d))
    Kb = g.standard_normal((S, n_kv, d))
    Vb = g.standard_normal((S, n_kv, d))
    Lv = g.standard_normal((S, r))
    Bv = g.standard_normal((r, n_kv * d))
    pos = np.arange(S - n_tok, S)
    O, _ = orc.lr_shared_attention(Q[None], Kb[None], Vb[None], None, Lv[None], None, Bv[None],
                                   pos[None], [S], theta)
    P, _ = orc.attention_probs(Q, Kb, pos, S)
    group = n_q // n_kv
    for i in range(n_tok):
        for h in range(n_q):
            gg = h // group
            ref = P[i, h] @ Vb[:, gg, :] + (P[i, h] @ Lv) @ Bv[:, gg * d:(gg + 1) * d]
            assert np.abs(O[0, i, h] - ref).max() <= RTOL_EXACT, "value associativity fails"


def pin_closed_forms(orc, seed=6, d=8, n_q=2, n_kv=1, S=12):
    g = _rng(seed)
    Q = g.standard_normal((3, n_q, d))
    Kb = g.standard_normal((S, n_kv, d))
    Vb = g.standard_normal((S, n_kv, d))
    # Query at position 0 sees only key 0.
    O, lse = orc.attention(Q, Kb, Vb, np.array([0, 0, 0]), S)
    assert np.abs(O - Vb[0, 0][None, None, :]).max() <= RTOL_EXACT, "single visible key"
    # Q = 0: uniform weights over the visible keys.
    pos = np.array([0, 4, S - 1])
    O, lse = orc.attention(np.zeros_like(Q), Kb, Vb, pos, S)
    for i, p in enumerate(pos):
        assert np.abs(O[i, 0] - Vb[: p + 1, 0].mean(0)).max() <= RTOL_EXACT, "mean of visible values"
        assert abs(lse[i, 0] - math.log(p + 1)) <= RTOL_EXACT
    # Identical keys: uniform weights whatever the query.
    Kc = np.repeat(Kb[:1], S, axis=0)
    P, _ = orc.attention_probs(Q, Kc, np.array([S - 1] * 3), S)
    assert np.abs(P - 1.0 / S).max() <= 1e-12


def pin_permutation(orc, seed=7, d=8, n_q=4, n_kv=2, S=20):
    g = _rng(seed)
    Q = g.standard_normal((3, n_q, d))
    Kb = g.standard_normal((S, n_kv, d))
    Vb = g.standard_normal((S, n_kv, d))
    pos = np.array([S - 1] * 3)
    O1, l1 = orc.attention(Q, Kb, Vb, pos, S)
    perm = g.permutation(S)
    O2, l2 = orc.attention(Q, Kb[perm], Vb[perm], pos, S)
    assert np.abs(O1 - O2).max() <= RTOL_EXACT and np.abs(l1 - l2).max() <= RTOL_EXACT


def pin_split_merge(orc, seed=8, d=8, n_q=4, n_kv=2, S=37, n_tok=5):
    """Attention over [0,S) equals the lse-merge of [0,S1) and [S1,S)."""
    g = _rng(seed)
    Q = g.standard_normal((n_tok, n_q, d)) * 2
    K = g.standard_normal((S, n_kv, d))
    V = g.standard_normal((S, n_kv, d))
    pos = np.array([S - 1, S - 3, 20, 25, S - 2])
    Of, lf = orc.attention(Q, K, V, pos, S)
    for S1 in (1, 13, 21):
        O1, l1 = orc.attention(Q, K[:S1], V[:S1], pos, S1)
        # Second range: keys S1..S-1 re-indexed from 0; a query sees key t iff
        # t + S1 <= pos.  Rows with no visible key have lse = -inf.
        rows_vis = pos >= S1
        O2 = np.zeros_like(Of)
        l2 = np.full(lf.shape, -np.inf)
        if rows_vis.any():
            o, l = orc.attention(Q[rows_vis], K[S1:], V[S1:], pos[rows_vis] - S1, S - S1)
            O2[rows_vis], l2[rows_vis] = o, l
        with np.errstate(invalid="ignore"):
            Om, lm = orc.merge_partials([(O1, l1), (O2, l2)])
        assert np.abs(Om - Of).max() <= RTOL_EXACT and np.abs(lm - lf).max() <= RTOL_EXACT


def pin_precompute(orc, seed=9, T=7, d_in=5, n_proj=2, N=3, r=2):
    g = _rng(seed)
    X = g.standard_normal((T, d_in))
    A = [[g.standard_normal((d_in, r)) for _ in range(N)] for _ in range(n_proj)]
    A_stack = np.concatenate([A[p][a] for p in range(n_proj) for a in range(N)], axis=1)
    L = orc.precompute_lr_cache(X, A_stack, n_proj, N, r)
    assert L.shape == (n_proj, N, T, r)
    for p in range(n_proj):
        for a in range(N):
            for t in range(T):
                for j in range(r):
                    ref = sum(X[t, k] * A[p][a][k, j] for k in range(d_in))
                    assert abs(L[p, a, t, j] - ref) <= 1e-12, "precompute block mismatch"


def pin_projection(orc, seed=10, T=5, d_in=6, n_kv=2, d=8, n_proj=2, N=2, r=2, theta=50.0, t0=3):
    """Base K/V of a segment by per-element sums and explicit pair rotations;
    the LR planes as in pin_precompute."""
    g = _rng(seed)
    X = g.standard_normal((T, d_in))
    W_k = g.standard_normal((d_in, n_kv * d))
    W_v = g.standard_normal((d_in, n_kv * d))
    A_stack = g.standard_normal((d_in, n_proj * N * r))
    pos = np.arange(t0, t0 + T)
    K, V, L = orc.project_kv_and_lr(X, W_k, W_v, A_stack, n_kv, n_proj, N, r, pos, theta)
    assert K.shape == (T, n_kv, d) and V.shape == (T, n_kv, d) and L.shape == (n_proj, N, T, r)
    for t in range(T):
        for h in range(n_kv):
            xk = [sum(X[t, k] * W_k[k, h * d + j] for k in range(d_in)) for j in range(d)]
            xv = [sum(X[t, k] * W_v[k, h * d + j] for k in range(d_in)) for j in range(d)]
            assert np.allclose(K[t, h], loop_rope(xk, int(pos[t]), theta), atol=1e-12), "key projection"
            assert np.allclose(V[t, h], xv, atol=1e-12), "value projection"
    for p in range(n_proj):
        for a in range(N):
            col = (p * N + a) * r
            for t in range(T):
                for j in range(r):
                    ref = sum(X[t, k] * A_stack[k, col + j] for k in range(d_in))
                    assert abs(L[p, a, t, j] - ref) <= 1e-12, "projection LR block"


def pin_golden(orc):
    """Hand-derived worked cases (tests/golden/worked_cases.json)."""
    import json
    import os
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "worked_cases.json")
    for c in json.load(open(path))["cases"]:
        if "Q" in c:
            Bk = np.array([c["B_k_unit"]]) * (math.sqrt(2.0) * math.log(3.0))
            O, lse = orc.lr_shared_attention(
                np.array(c["Q"])[None], np.array(c["K_base"])[None], np.array(c["V_base"])[None],
                np.array(c["L_k"])[None], np.array(c["L_v"])[None], Bk[None], np.array(c["B_v"])[None],
                np.array([c["positions"]]), [len(c["K_base"])], c["theta"])
            assert np.allclose(O[0], c["expected_O"], atol=1e-12), c["name"]
            assert np.allclose(lse[0], c["expected_lse"], atol=1e-12), c["name"]
        else:
            L = orc.precompute_lr_cache(np.array(c["X"]), np.array(c["A_stack"]), 1, 2, 1)
            assert np.array_equal(L, np.array(c["expected_L"])), c["name"]


ALL_PINS = [pin_golden, pin_merged_weights, pin_plain_attention, pin_softmax_rows, pin_rope,
            pin_value_assoc, pin_closed_forms, pin_permutation, pin_split_merge,
            pin_precompute, pin_projection]
