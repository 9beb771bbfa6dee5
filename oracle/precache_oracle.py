"""fp64 CPU oracle for the PreLRShared hot path of PReCache.

TEST INFRASTRUCTURE ONLY.  This module is what the GPU kernels are checked
against.  It is plain numpy in float64, slow on purpose, and follows the
paper's definitions step by step with no blocking, fusion or reordering:

* Eq. 1 (Sec. 2.1): an adapted projection splits into a base contribution
  ``X W0`` and an adapter contribution ``(X A_i) B_i``.
* Sec. 2.2: the base cache is ``X W0`` and agent i's LR cache is ``X A_i``
  (r numbers per token).
* Sec. 3.1: PreLRShared applies every agent's down-projection ``A_k`` to the
  hidden states of a newly processed segment (the LR-cache precompute) and the
  current agent attends over the shared base cache plus its own LR cache.
* App. D.2: the key-side adapter contribution is expanded from rank r before
  RoPE is applied; the value side is linear, so ``P (V_base + L_v B_v)``
  equals ``P V_base + (P L_v) B_v``.

Conventions where the paper is silent (each one is listed with its reason in
the design notes of this repository):

* RoPE is the rotate-half form: element j pairs with j + d/2, frequency
  ``omega_j = theta ** (-2 j / d)`` for j < d/2, angles in float64.
* K_base and Q arrive already rotated; only the LR key term is rotated here,
  each token at its own absolute position t (KV token t sits at position t).
* Query token i of request b may see key t iff ``t <= positions[b, i]`` and
  ``t < kv_len[b]``.
* q head h reads KV head ``h // (n_q / n_kv)`` (contiguous GQA groups).
* A_stack columns are projection-major, then agent: columns
  ``[(p*N + a)*r, (p*N + a + 1)*r)`` hold agent a's down-projection for
  projection p (p = 0 for k, p = 1 for v).
* B maps the r-wide LR vector to all KV heads: ``B [r, n_kv*d]``, head g uses
  columns ``[g*d, (g+1)*d)``.
* No LoRA scale alpha/r is applied (Eq. 1 has none); a caller folds it into B.
* The default softmax scale is ``1/sqrt(d)``.

Every function here is pinned by ``tests/test_oracle_pins.py`` against facts
that the paper or the mathematics fix (Eq. 1 by brute force with merged
weights, B = 0 against torch's scaled_dot_product_attention, RoPE closed forms
and invariants, softmax normalisation, value associativity, closed-form
attention cases, permutation and split invariance, the precompute against a
naive triple loop, the base projection against per-element sums and explicit
pair rotations).
"""
from __future__ import annotations

import numpy as np


def _f64(x):
    return None if x is None else np.asarray(x, dtype=np.float64)


# ----------------------------------------------------------------------------
# RoPE (the only rotation on the path: App. D.2 says the key LR term is
# expanded from rank r and then rotated)
# ----------------------------------------------------------------------------
def rope_frequencies(d: int, theta: float) -> np.ndarray:
    """Rotation frequencies omega_j = theta^(-2j/d), j = 0 .. d/2-1 (float64)."""
    if d % 2:
        raise ValueError("head dimension must be even for RoPE")
    j = np.arange(d // 2, dtype=np.float64)
    return np.power(np.float64(theta), -2.0 * j / d)


def rope(x, pos, theta: float) -> np.ndarray:
    """Rotate-half RoPE of ``x [..., d]`` at positions ``pos``.

    ``pos`` broadcasts against ``x.shape[:-1]``.  For j < d/2:
      out_j       = x_j cos(pos*omega_j) - x_{j+d/2} sin(pos*omega_j)
      out_{j+d/2} = x_{j+d/2} cos(pos*omega_j) + x_j sin(pos*omega_j)
    """
    x = _f64(x)
    d = x.shape[-1]
    omega = rope_frequencies(d, theta)
    ang = np.asarray(pos, dtype=np.float64)[..., None] * omega
    c, s = np.cos(ang), np.sin(ang)
    lo, hi = x[..., : d // 2], x[..., d // 2:]
    return np.concatenate([lo * c - hi * s, hi * c + lo * s], axis=-1)


# ----------------------------------------------------------------------------
# Kernel 1: LR-cache precompute (Sec. 3.1, Fig. 1 A1-A3)
# ----------------------------------------------------------------------------
def precompute_lr_cache(X, A_stack, n_proj: int, n_agents: int, rank: int) -> np.ndarray:
    """LR caches of every agent for one segment of hidden states.

    ``X [T, d_in]`` are the hidden states of the newly processed segment and
    ``A_stack [d_in, n_proj*n_agents*rank]`` holds every agent's LoRA
    down-projection side by side (projection-major, then agent).  Returns
    ``L [n_proj, n_agents, T, rank]`` with ``L[p, a] = X @ A_{p,a}``, i.e. the
    LR cache ``X A_k`` of Sec. 2.2 for every agent k at once (Sec. 3.1).
    """
    X, A_stack = _f64(X), _f64(A_stack)
    T, d_in = X.shape
    if A_stack.shape != (d_in, n_proj * n_agents * rank):
        raise ValueError(f"A_stack shape {A_stack.shape} does not match "
                         f"({d_in}, {n_proj * n_agents * rank})")
    L = np.empty((n_proj, n_agents, T, rank), dtype=np.float64)
    for p in range(n_proj):
        for a in range(n_agents):
            col = (p * n_agents + a) * rank
            L[p, a] = X @ A_stack[:, col: col + rank]
    return L


def project_kv_and_lr(X, W_k, W_v, A_stack, n_kv: int, n_proj: int, n_agents: int, rank: int,
                      positions, theta: float):
    """Base cache and every agent's LR cache of one segment of hidden states.

    ``X [T, d_in]``; ``W_k, W_v [d_in, n_kv*d]`` (the base key and value
    projections, paper orientation); ``A_stack`` as in ``precompute_lr_cache``;
    ``positions [T]`` the tokens' absolute positions.  Returns
    ``K_base [T, n_kv, d] = RoPE(X W_k)`` (Sec. 2.2 base cache ``X W0`` on the
    key side, rotated at each token's position as the keys of a RoPE model
    are), ``V_base [T, n_kv, d] = X W_v`` and the LR planes of
    ``precompute_lr_cache`` (Sec. 3.1).
    """
    X, W_k, W_v = _f64(X), _f64(W_k), _f64(W_v)
    T = X.shape[0]
    if W_k.shape != W_v.shape or W_k.shape[0] != X.shape[1] or W_k.shape[1] % n_kv:
        raise ValueError(f"W_k {W_k.shape} / W_v {W_v.shape} do not fit X {X.shape} and n_kv={n_kv}")
    d = W_k.shape[1] // n_kv
    K = (X @ W_k).reshape(T, n_kv, d)
    K = rope(K, np.asarray(positions, dtype=np.float64)[:, None], theta)
    V = (X @ W_v).reshape(T, n_kv, d)
    return K, V, precompute_lr_cache(X, A_stack, n_proj, n_agents, rank)


# ----------------------------------------------------------------------------
# Per-agent K/V as the method defines them (Eq. 1 + Sec. 2.2 + App. D.2)
# ----------------------------------------------------------------------------
def rebuild_kv(K_base, V_base, L_k, L_v, B_k, B_v, theta: float):
    """Agent's keys and values over one trajectory.

    ``K_base, V_base [S, n_kv, d]`` (K_base already rotated), ``L_k, L_v [S, r]``
    (agent's LR caches), ``B_k, B_v [r, n_kv*d]``.  A ``None`` LR cache means
    the projection is not adapted (the QV setting has ``L_k = None``).
      K[t] = K_base[t] + RoPE(L_k[t] B_k, t)
      V[t] = V_base[t] + L_v[t] B_v
    """
    K_base, V_base = _f64(K_base), _f64(V_base)
    S, n_kv, d = K_base.shape
    K = K_base.copy()
    V = V_base.copy()
    if (L_k is None) != (B_k is None) or (L_v is None) != (B_v is None):
        raise ValueError("an LR cache and its up-projection must be given together")
    t = np.arange(S, dtype=np.float64)
    if L_k is not None:
        E = (_f64(L_k)[:S] @ _f64(B_k)).reshape(S, n_kv, d)
        K = K + rope(E, t[:, None], theta)
    if L_v is not None:
        V = V + (_f64(L_v)[:S] @ _f64(B_v)).reshape(S, n_kv, d)
    return K, V


# ----------------------------------------------------------------------------
# Causal GQA softmax attention (the plain definition)
# ----------------------------------------------------------------------------
def attention_scores(Q, K, positions, kv_len: int, scale=None) -> np.ndarray:
    """Scaled scores ``[n_tok, n_q, kv_len]`` with masked entries at -inf.

    ``Q [n_tok, n_q, d]``, ``K [>=kv_len, n_kv, d]``; q head h reads KV head
    h // (n_q/n_kv); key t is visible to query i iff t <= positions[i].
    """
    Q, K = _f64(Q), _f64(K)
    n_tok, n_q, d = Q.shape
    n_kv = K.shape[1]
    if n_q % n_kv:
        raise ValueError("n_q must be a multiple of n_kv")
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    group = n_q // n_kv
    s = np.empty((n_tok, n_q, kv_len), dtype=np.float64)
    for h in range(n_q):
        g = h // group
        s[:, h, :] = (Q[:, h, :] @ K[:kv_len, g, :].T) * scale
    visible = np.arange(kv_len)[None, :] <= np.asarray(positions)[:, None]
    return np.where(visible[:, None, :], s, -np.inf)


def attention_probs(Q, K, positions, kv_len: int, scale=None):
    """Softmax probabilities ``[n_tok, n_q, kv_len]`` and log-sum-exp ``[n_tok, n_q]``."""
    s = attention_scores(Q, K, positions, kv_len, scale)
    m = s.max(axis=-1, keepdims=True)
    e = np.exp(s - m)
    z = e.sum(axis=-1, keepdims=True)
    return e / z, (m + np.log(z))[..., 0]


def attention(Q, K, V, positions, kv_len: int, scale=None):
    """``O [n_tok, n_q, d]`` and ``lse [n_tok, n_q]`` of causal GQA attention."""
    V = _f64(V)
    P, lse = attention_probs(Q, K, positions, kv_len, scale)
    n_tok, n_q, _ = P.shape
    n_kv = V.shape[1]
    group = n_q // n_kv
    O = np.empty((n_tok, n_q, V.shape[2]), dtype=np.float64)
    for h in range(n_q):
        O[:, h, :] = P[:, h, :] @ V[:kv_len, h // group, :]
    return O, lse


# ----------------------------------------------------------------------------
# Batched entry points, one per C-ABI call they check
# ----------------------------------------------------------------------------
def materialize_agent_kv(K_base, V_base, L_k, L_v, B_k, B_v, kv_len, theta: float):
    """The reference point: each request's full per-agent K/V written out.

    Shapes: ``K_base, V_base [B, S_cap, n_kv, d]``, ``L_k, L_v [B, S_cap, r]``
    (or None), ``B_k, B_v [B, r, n_kv*d]`` (or None), ``kv_len [B]``.
    Returns lists ``K[b], V[b]`` of shape ``[kv_len[b], n_kv, d]``.
    """
    Ks, Vs = [], []
    for b in range(len(kv_len)):
        n = int(kv_len[b])
        K, V = rebuild_kv(
            _f64(K_base)[b, :n], _f64(V_base)[b, :n],
            None if L_k is None else _f64(L_k)[b, :n],
            None if L_v is None else _f64(L_v)[b, :n],
            None if B_k is None else _f64(B_k)[b],
            None if B_v is None else _f64(B_v)[b], theta)
        Ks.append(K)
        Vs.append(V)
    return Ks, Vs


def lr_shared_attention(Q, K_base, V_base, L_k, L_v, B_k, B_v, positions, kv_len,
                        theta: float, scale=None):
    """Attention of each request's queries over base cache + its agent's LR cache.

    ``Q [B, n_tok, n_q, d]`` (already rotated), ``positions [B, n_tok]``; other
    shapes as in :func:`materialize_agent_kv`.  Returns ``O [B, n_tok, n_q, d]``
    and ``lse [B, n_tok, n_q]`` (natural log).  The result equals attention
    over the explicitly merged per-agent K/V (Eq. 1), which is what this
    function computes: rebuild the agent's K/V, then attend.
    """
    Q = _f64(Q)
    Bn, n_tok, n_q, d = Q.shape
    Ks, Vs = materialize_agent_kv(K_base, V_base, L_k, L_v, B_k, B_v, kv_len, theta)
    O = np.empty((Bn, n_tok, n_q, d), dtype=np.float64)
    lse = np.empty((Bn, n_tok, n_q), dtype=np.float64)
    for b in range(Bn):
        O[b], lse[b] = attention(Q[b], Ks[b], Vs[b], np.asarray(positions)[b],
                                 int(kv_len[b]), scale)
    return O, lse


def merge_partials(parts):
    """Combine attention results over disjoint key ranges.

    ``parts`` is a list of ``(O_s, lse_s)`` computed over disjoint key subsets;
    returns ``(O, lse)`` over their union:
      lse = log sum_s exp(lse_s),  O = sum_s exp(lse_s - lse) O_s.
    A part whose keys are all masked has ``lse_s = -inf`` and weight 0.
    """
    lses = np.stack([np.asarray(p[1], dtype=np.float64) for p in parts])
    m = lses.max(axis=0)
    w = np.exp(lses - m)
    z = w.sum(axis=0)
    O = sum(w[i][..., None] * np.asarray(p[0], dtype=np.float64)
            for i, p in enumerate(parts)) / z[..., None]
    return O, m + np.log(z)
