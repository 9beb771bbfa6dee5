"""Helpers for GPU parity tests: run the HIP path through the C ABI and the fp64
oracle on the same seeded inputs, and measure the differences."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import paper_2609_34054_amd as prc

# Tolerances fixed by the target: attention max abs 2e-2 and mean abs 2e-3
# (bf16 inputs, fp32 accumulation); precompute relative Frobenius 1e-2;
# the LR term's contribution must be reproduced to 5e-2 relative.
ATOL_MAX = 2e-2
ATOL_MEAN = 2e-3
PRE_REL = 1e-2
LR_SENS = 5e-2
LSE_ATOL = 2e-2


def f64(t):
    return None if t is None else t.detach().double().cpu().numpy()


def to_dev(case, dev="cuda"):
    return {k: (v.to(dev) if isinstance(v, torch.Tensor) else v) for k, v in case.items()}


def gpu_attention(g, theta, **kw):
    O, lse = prc.lr_shared_attention(g["Q"], g["K_base"], g["V_base"], g["L_k"], g["L_v"], g["B_k"],
                                     g["B_v"], g["positions"], g["kv_len"], rope_theta=theta,
                                     want_lse=True, **kw)
    torch.cuda.synchronize()
    return O, lse


def oracle_attention(c, theta, reqs=None, toks=None, zero_b=False):
    """Oracle on requests ``reqs`` (default all) and query tokens ``toks``."""
    B = c["Q"].shape[0]
    reqs = list(range(B)) if reqs is None else list(reqs)
    toks = slice(None) if toks is None else list(toks)

    def pick(name, per_req=True):
        t = c[name]
        if t is None:
            return None
        if t.shape[0] == 1 and B > 1:
            t = t.expand(B, *t.shape[1:])
        return t[reqs]

    Q = f64(pick("Q"))[:, toks]
    pos = c["positions"].numpy()[reqs][:, toks]
    Bk, Bv = f64(pick("B_k")), f64(pick("B_v"))
    if zero_b:
        Bk = None if Bk is None else np.zeros_like(Bk)
        Bv = None if Bv is None else np.zeros_like(Bv)
    return oracle.lr_shared_attention(Q, f64(pick("K_base")), f64(pick("V_base")), f64(pick("L_k")),
                                      f64(pick("L_v")), Bk, Bv, pos, c["kv_len"].numpy()[reqs], theta)


def attn_errors(O_gpu, O_ref):
    e = np.abs(f64(O_gpu) - O_ref)
    return float(e.max()), float(e.mean())


def lse_error(lse_gpu, lse_ref):
    g = f64(lse_gpu)
    both_inf = np.isneginf(g) & np.isneginf(lse_ref)
    d = np.where(both_inf, 0.0, np.abs(g - lse_ref))
    return float(np.nan_to_num(d, nan=np.inf).max())
