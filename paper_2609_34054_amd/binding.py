"""ctypes binding of libprecache.so (argument marshalling only).

Every step of the hot path runs in the library's HIP kernels.  These wrappers
take torch tensors for device memory and torch's current stream, derive the
sizes and strides the C ABI wants, and raise :class:`PrecacheError` on any
non-OK status.  There is no fallback: if the library is missing, the call
fails.
"""
from __future__ import annotations

import ctypes
import os

import torch

from .build import CHECKED_LIB_PATH, LIB_PATH

_LIBS: dict = {}
# The checked build (device-side kv_len/position checks, a stream wait per
# attention call) is selected with PRC_CHECKED=1 or use_checked_library().
_CHECKED = os.environ.get("PRC_CHECKED", "0") == "1"

STATUS_NAMES = {0: "PRC_OK", 1: "PRC_EINVAL", 2: "PRC_ESHAPE", 3: "PRC_EALIGN",
                4: "PRC_EUNSUPPORTED", 5: "PRC_EWORKSPACE", 6: "PRC_ELAUNCH", 7: "PRC_EDEVICE",
                8: "PRC_EDEVDATA"}

EXPORTS = ("precompute_lr_cache", "project_kv_and_lr_cache", "project_kv_and_lr_cache_paged",
           "lr_shared_attention", "lr_shared_attention_workspace_size", "lr_shared_attention_paged",
           "lr_shared_attention_paged_workspace_size", "lr_shared_attention_noalloc", "materialize_agent_kv",
           "prc_stream_read", "prc_last_error",
           "prc_status_string", "prc_version", "prc_device_checks")


class PrecacheError(RuntimeError):
    def __init__(self, func: str, status: int, message: str):
        self.status = status
        self.status_name = STATUS_NAMES.get(status, f"status {status}")
        super().__init__(f"{func}: {self.status_name}: {message}")


class LrsaDims(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("n_tok", ctypes.c_int32),
        ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("rank", ctypes.c_int32),
        ("s_cap", ctypes.c_int64),
        ("kv_req_stride", ctypes.c_int64),
        ("l_req_stride", ctypes.c_int64),
        ("b_req_stride", ctypes.c_int64),
        ("softmax_scale", ctypes.c_float),
        ("reserved0", ctypes.c_float),
        ("rope_theta", ctypes.c_double),
    ]


class LrsaPaging(ctypes.Structure):
    _fields_ = [
        ("kv_block_table", ctypes.c_void_p),
        ("lr_block_table", ctypes.c_void_p),
        ("block_size", ctypes.c_int32),
        ("max_blocks", ctypes.c_int32),
        ("n_kv_blocks", ctypes.c_int32),
        ("n_lr_blocks", ctypes.c_int32),
    ]


def use_checked_library(flag: bool = True) -> None:
    """Route every later call through libprecache_checked.so (or back)."""
    global _CHECKED
    _CHECKED = bool(flag)


def lib() -> ctypes.CDLL:
    """Load libprecache.so, or its checked twin (both built in-tree by
    ``build()``); raise if absent."""
    path = CHECKED_LIB_PATH if _CHECKED else LIB_PATH
    if path not in _LIBS:
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is not built: run __graft_entry__.build() "
                               "(python -m paper_2609_34054_amd.build)")
        L = ctypes.CDLL(path)
        vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
        L.precompute_lr_cache.argtypes = [vp, i64, i64, i64, vp, i32, i32, i32, vp, i64, i64, vp]
        L.precompute_lr_cache.restype = ctypes.c_int
        L.project_kv_and_lr_cache.argtypes = [vp, i64, i64, i64, vp, i32, i32, vp, i32, i32, i32, ctypes.c_double,
                                              vp, vp, vp, i64, i64, vp]
        L.project_kv_and_lr_cache.restype = ctypes.c_int
        L.project_kv_and_lr_cache_paged.argtypes = [vp, i64, i64, i64, vp, i32, i32, vp, i32, i32, i32,
                                                    ctypes.c_double, vp, vp, vp, vp, i32, i32, i32, i64, vp]
        L.project_kv_and_lr_cache_paged.restype = ctypes.c_int
        L.lr_shared_attention.argtypes = [ctypes.POINTER(LrsaDims), vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                          vp, vp, vp, ctypes.c_size_t, vp]
        L.lr_shared_attention.restype = ctypes.c_int
        L.lr_shared_attention_noalloc.argtypes = [ctypes.POINTER(LrsaDims), vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                                  vp, vp, vp]
        L.lr_shared_attention_noalloc.restype = ctypes.c_int
        L.lr_shared_attention_workspace_size.argtypes = [ctypes.POINTER(LrsaDims)]
        L.lr_shared_attention_workspace_size.restype = ctypes.c_size_t
        L.lr_shared_attention_paged.argtypes = [ctypes.POINTER(LrsaDims), ctypes.POINTER(LrsaPaging), vp, vp, vp,
                                                vp, vp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
        L.lr_shared_attention_paged.restype = ctypes.c_int
        L.lr_shared_attention_paged_workspace_size.argtypes = [ctypes.POINTER(LrsaDims)]
        L.lr_shared_attention_paged_workspace_size.restype = ctypes.c_size_t
        L.materialize_agent_kv.argtypes = [ctypes.POINTER(LrsaDims), vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.materialize_agent_kv.restype = ctypes.c_int
        L.prc_stream_read.argtypes = [vp, ctypes.c_size_t, vp, i32, vp]
        L.prc_stream_read.restype = ctypes.c_int
        L.prc_last_error.restype = ctypes.c_char_p
        L.prc_status_string.argtypes = [ctypes.c_int]
        L.prc_status_string.restype = ctypes.c_char_p
        L.prc_version.restype = ctypes.c_char_p
        L.prc_device_checks.restype = ctypes.c_int
        _LIBS[path] = L
    return _LIBS[path]


def _check(func: str, status: int) -> None:
    if status != 0:
        raise PrecacheError(func, status, lib().prc_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _bf16(name, t, ndim):
    if t is None:
        return
    if t.dtype != torch.bfloat16:
        raise TypeError(f"{name} must be bfloat16, got {t.dtype}")
    if t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims, got shape {tuple(t.shape)}")
    if t.stride(-1) != 1:
        raise ValueError(f"{name} must be contiguous in its last dimension")


def _req_stride(t, batch):
    """Elements between requests: 0 when one buffer serves every request."""
    if t is None or t.shape[0] == 1:
        return 0
    if t.shape[0] != batch:
        raise ValueError(f"leading dim {t.shape[0]} is neither 1 nor the batch {batch}")
    return t.stride(0)


def precompute_lr_cache(X, A_stack, n_proj: int, n_agents: int, rank: int, L_out, tok_offset: int = 0,
                        stream=None):
    """``L_out[p][a][tok_offset + t] = X[t] @ A_stack[:, (p*N+a)*r:(p*N+a+1)*r]`` (Sec. 3.1).

    ``X [T, d_in]`` bf16 (row stride may exceed d_in), ``A_stack [d_in, n_proj*N*r]``,
    ``L_out [n_proj, N, s_cap, r]`` bf16 contiguous.
    """
    _bf16("X", X, 2)
    _bf16("A_stack", A_stack, 2)
    _bf16("L_out", L_out, 4)
    if not A_stack.is_contiguous() or not L_out.is_contiguous():
        raise ValueError("A_stack and L_out must be contiguous")
    if tuple(A_stack.shape) != (X.shape[1], n_proj * n_agents * rank):
        raise ValueError(f"A_stack shape {tuple(A_stack.shape)} is not ({X.shape[1]}, {n_proj * n_agents * rank})")
    if tuple(L_out.shape[:2]) != (n_proj, n_agents) or L_out.shape[3] != rank:
        raise ValueError(f"L_out shape {tuple(L_out.shape)} does not match ({n_proj}, {n_agents}, s_cap, {rank})")
    T, d_in = X.shape
    st = lib().precompute_lr_cache(_ptr(X), T, d_in, X.stride(0), _ptr(A_stack), n_proj, n_agents, rank,
                                   _ptr(L_out), L_out.shape[2], tok_offset, _stream(stream))
    _check("precompute_lr_cache", st)
    return L_out


def project_kv_and_lr_cache(X, W, A_stack, n_kv_heads: int, head_dim: int, n_proj: int, n_agents: int,
                            rank: int, K_base, V_base, L_out, *, rope_theta: float, tok_offset: int = 0,
                            stream=None):
    """Base K/V (RoPE on keys) and every agent's LR rows of one segment in one GEMM
    over ``X`` (Sec. 2.2 base cache, Sec. 3.1 precompute).

    ``X [T, d_in]`` bf16; ``W [d_in, 2*n_kv*d]`` (``[W_k | W_v]``);
    ``A_stack [d_in, n_proj*N*r]``; ``K_base, V_base [s_cap, n_kv, d]`` and
    ``L_out [n_proj, N, s_cap, r]`` bf16 contiguous, rows ``tok_offset ..`` written.
    """
    _bf16("X", X, 2)
    _bf16("W", W, 2)
    _bf16("A_stack", A_stack, 2)
    _bf16("K_base", K_base, 3)
    _bf16("V_base", V_base, 3)
    _bf16("L_out", L_out, 4)
    for name, t in (("W", W), ("A_stack", A_stack), ("K_base", K_base), ("V_base", V_base),
                    ("L_out", L_out)):
        if t is not None and not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    s_cap = K_base.shape[0]
    if tuple(K_base.shape) != (s_cap, n_kv_heads, head_dim) or K_base.shape != V_base.shape:
        raise ValueError(f"K_base/V_base shapes {tuple(K_base.shape)}, {tuple(V_base.shape)} are not "
                         f"(s_cap, {n_kv_heads}, {head_dim})")
    if n_proj * n_agents and tuple(L_out.shape) != (n_proj, n_agents, s_cap, rank):
        raise ValueError(f"L_out shape {tuple(L_out.shape)} does not match ({n_proj}, {n_agents}, {s_cap}, {rank})")
    T, d_in = X.shape
    if tuple(W.shape) != (d_in, 2 * n_kv_heads * head_dim):
        raise ValueError(f"W shape {tuple(W.shape)} is not ({d_in}, {2 * n_kv_heads * head_dim})")
    st = lib().project_kv_and_lr_cache(_ptr(X), T, d_in, X.stride(0), _ptr(W), n_kv_heads, head_dim,
                                       _ptr(A_stack), n_proj, n_agents, rank, float(rope_theta), _ptr(K_base),
                                       _ptr(V_base), _ptr(L_out), s_cap, tok_offset, _stream(stream))
    _check("project_kv_and_lr_cache", st)
    return K_base, V_base, L_out


def project_kv_and_lr_cache_paged(X, W, A_stack, n_kv_heads: int, head_dim: int, n_proj: int,
                                  n_agents: int, rank: int, K_pool, V_pool, L_pool, block_table, *,
                                  rope_theta: float, tok_offset: int = 0, stream=None):
    """:func:`project_kv_and_lr_cache` writing into paged pools: token ``p`` goes to
    row ``p % blk`` of block ``block_table[p // blk]``.

    ``K_pool, V_pool [n_blocks, blk, n_kv, d]`` (None with ``n_kv_heads == 0``);
    ``L_pool [n_proj, N, n_blocks, blk, r]`` (None without LR planes);
    ``block_table [max_blocks]`` int32, contiguous.
    """
    _bf16("X", X, 2)
    _bf16("W", W, 2)
    _bf16("A_stack", A_stack, 2)
    _bf16("K_pool", K_pool, 4)
    _bf16("V_pool", V_pool, 4)
    _bf16("L_pool", L_pool, 5)
    for name, t in (("W", W), ("A_stack", A_stack), ("K_pool", K_pool), ("V_pool", V_pool),
                    ("L_pool", L_pool), ("block_table", block_table)):
        if t is not None and not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    if block_table.dtype != torch.int32 or block_table.dim() != 1:
        raise TypeError("block_table must be a 1-D int32 tensor")
    pool = K_pool if n_kv_heads else L_pool[0, 0]
    n_blocks, blk = pool.shape[0], pool.shape[1]
    if n_kv_heads and (tuple(K_pool.shape) != (n_blocks, blk, n_kv_heads, head_dim) or K_pool.shape != V_pool.shape):
        raise ValueError(f"K_pool/V_pool shapes {tuple(K_pool.shape)}, {tuple(V_pool.shape)} are not "
                         f"(n_blocks, blk, {n_kv_heads}, {head_dim})")
    if n_proj * n_agents and tuple(L_pool.shape) != (n_proj, n_agents, n_blocks, blk, rank):
        raise ValueError(f"L_pool shape {tuple(L_pool.shape)} does not match "
                         f"({n_proj}, {n_agents}, {n_blocks}, {blk}, {rank})")
    T, d_in = X.shape
    st = lib().project_kv_and_lr_cache_paged(_ptr(X), T, d_in, X.stride(0), _ptr(W), n_kv_heads, head_dim,
                                             _ptr(A_stack), n_proj, n_agents, rank, float(rope_theta),
                                             _ptr(K_pool), _ptr(V_pool), _ptr(L_pool), _ptr(block_table), blk,
                                             block_table.shape[0], n_blocks, tok_offset, _stream(stream))
    _check("project_kv_and_lr_cache_paged", st)
    return K_pool, V_pool, L_pool


def make_dims(Q, K_base, L_k, L_v, B_k, B_v, rope_theta: float, softmax_scale: float = 0.0,
              batch=None, n_q=None):
    """The lrsa_dims of a call, from tensor shapes (Q may be None for materialise)."""
    lr = L_k if L_k is not None else L_v
    bt = B_k if B_k is not None else B_v
    if Q is not None:
        batch, n_tok, n_q, d = Q.shape
    else:
        n_tok, d = 0, K_base.shape[3]
    s_cap, n_kv = K_base.shape[1], K_base.shape[2]
    if K_base.shape[3] != d:
        raise ValueError("head dims of Q and K_base differ")
    rank = lr.shape[-1] if lr is not None else 0
    if lr is not None and lr.shape[-2] != s_cap:
        raise ValueError(f"LR cache holds {lr.shape[-2]} rows, the base cache {s_cap}")
    if bt is not None and (bt.shape[-2] != rank or bt.shape[-1] != n_kv * d):
        raise ValueError(f"up-projection shape {tuple(bt.shape)} is not (.., {rank}, {n_kv * d})")
    return LrsaDims(batch=batch, n_tok=n_tok, n_q_heads=n_q, n_kv_heads=n_kv, head_dim=d, rank=rank,
                    s_cap=s_cap, kv_req_stride=_req_stride(K_base, batch),
                    l_req_stride=_req_stride(lr, batch), b_req_stride=_req_stride(bt, batch),
                    softmax_scale=softmax_scale, reserved0=0.0, rope_theta=rope_theta)


def workspace_size(dims: LrsaDims) -> int:
    return int(lib().lr_shared_attention_workspace_size(ctypes.byref(dims)))


def paged_workspace_size(dims: LrsaDims) -> int:
    return int(lib().lr_shared_attention_paged_workspace_size(ctypes.byref(dims)))


def lr_shared_attention(Q, K_base, V_base, L_k, L_v, B_k, B_v, positions, kv_len, *, rope_theta: float,
                        softmax_scale: float = 0.0, O=None, lse=None, want_lse: bool = False,
                        workspace=None, tile_cache: bool = True, stream=None):
    """Attention over the shared base cache plus one agent's LR cache (Sec. 3.1).

    Shapes: ``Q [B, n_tok, n_q, d]``; ``K_base, V_base [B|1, s_cap, n_kv, d]``;
    ``L_k, L_v [B|1, s_cap, r]`` or None; ``B_k, B_v [B|1, r, n_kv*d]`` or None
    (Eq. 1 orientation); ``positions [B, n_tok]`` and ``kv_len [B]`` int32.
    A workspace is allocated when none (or too small a one) is given; with
    ``tile_cache=False`` it is sized without the optional prefill tile cache
    (the size the paged query reports), so the call rebuilds every tile.
    Returns ``(O, lse)`` (``lse`` None unless requested).
    """
    for name, t, nd in (("Q", Q, 4), ("K_base", K_base, 4), ("V_base", V_base, 4), ("L_k", L_k, 3),
                        ("L_v", L_v, 3), ("B_k", B_k, 3), ("B_v", B_v, 3)):
        _bf16(name, t, nd)
    for name, t in (("Q", Q), ("K_base", K_base), ("V_base", V_base)):
        if not t[0].is_contiguous():
            raise ValueError(f"{name} must be contiguous within a request")
    if K_base.shape != V_base.shape or K_base.stride() != V_base.stride():
        raise ValueError("K_base and V_base must share shape and strides")
    if L_k is not None and L_v is not None and (L_k.shape != L_v.shape or L_k.stride() != L_v.stride()):
        raise ValueError("L_k and L_v must share shape and strides")
    if B_k is not None and B_v is not None and (B_k.shape != B_v.shape or B_k.stride() != B_v.stride()):
        raise ValueError("B_k and B_v must share shape and strides")
    dims = make_dims(Q, K_base, L_k, L_v, B_k, B_v, rope_theta, softmax_scale)
    if positions.dtype != torch.int32 or kv_len.dtype != torch.int32:
        raise TypeError("positions and kv_len must be int32")
    if tuple(positions.shape) != tuple(Q.shape[:2]) or not positions.is_contiguous():
        raise ValueError("positions must be a contiguous [B, n_tok] tensor")
    if tuple(kv_len.shape) != (Q.shape[0],):
        raise ValueError("kv_len must be a [B] tensor")
    if O is None:
        O = torch.empty_like(Q)
    if lse is None and want_lse:
        lse = torch.empty(Q.shape[:3], dtype=torch.float32, device=Q.device)
    need = workspace_size(dims) if tile_cache else paged_workspace_size(dims)
    if need and (workspace is None or workspace.numel() * workspace.element_size() < need):
        workspace = torch.empty(need, dtype=torch.uint8, device=Q.device)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    if not tile_cache:
        ws_bytes = min(ws_bytes, need)
        if ws_bytes == 0:
            workspace = None
    st = lib().lr_shared_attention(ctypes.byref(dims), _ptr(Q), _ptr(K_base), _ptr(V_base), _ptr(L_k),
                                   _ptr(L_v), _ptr(B_k), _ptr(B_v), _ptr(positions), _ptr(kv_len), _ptr(O),
                                   _ptr(lse), _ptr(workspace), ws_bytes, _stream(stream))
    _check("lr_shared_attention", st)
    return O, lse


def lr_shared_attention_noalloc(Q, K_base, V_base, L_k, L_v, B_k, B_v, positions, kv_len, *,
                                rope_theta: float, softmax_scale: float = 0.0, O, lse=None, stream=None):
    """:func:`lr_shared_attention` through the entry point that allocates nothing:
    the caller preallocates ``O`` (and ``lse``); split partials go to the
    library's static per-device workspace."""
    for name, t, nd in (("Q", Q, 4), ("K_base", K_base, 4), ("V_base", V_base, 4), ("L_k", L_k, 3),
                        ("L_v", L_v, 3), ("B_k", B_k, 3), ("B_v", B_v, 3), ("O", O, 4)):
        _bf16(name, t, nd)
    if K_base.shape != V_base.shape or K_base.stride() != V_base.stride():
        raise ValueError("K_base and V_base must share shape and strides")
    if tuple(O.shape) != tuple(Q.shape) or not O.is_contiguous():
        raise ValueError("O must be a contiguous tensor shaped like Q")
    if positions.dtype != torch.int32 or kv_len.dtype != torch.int32:
        raise TypeError("positions and kv_len must be int32")
    dims = make_dims(Q, K_base, L_k, L_v, B_k, B_v, rope_theta, softmax_scale)
    st = lib().lr_shared_attention_noalloc(ctypes.byref(dims), _ptr(Q), _ptr(K_base), _ptr(V_base), _ptr(L_k),
                                           _ptr(L_v), _ptr(B_k), _ptr(B_v), _ptr(positions), _ptr(kv_len),
                                           _ptr(O), _ptr(lse), _stream(stream))
    _check("lr_shared_attention_noalloc", st)
    return O, lse


def materialize_agent_kv(K_base, V_base, L_k, L_v, B_k, B_v, kv_len, *, rope_theta: float, K_full=None,
                         V_full=None, stream=None):
    """Write each request's full per-agent K/V (the materialise-then-attend reference point)."""
    for name, t, nd in (("K_base", K_base, 4), ("V_base", V_base, 4), ("L_k", L_k, 3), ("L_v", L_v, 3),
                        ("B_k", B_k, 3), ("B_v", B_v, 3)):
        _bf16(name, t, nd)
    batch = kv_len.shape[0]
    dims = make_dims(None, K_base, L_k, L_v, B_k, B_v, rope_theta, batch=batch, n_q=K_base.shape[2])
    shape = (batch,) + tuple(K_base.shape[1:])
    if K_full is None:
        K_full = torch.empty(shape, dtype=torch.bfloat16, device=K_base.device)
    if V_full is None:
        V_full = torch.empty(shape, dtype=torch.bfloat16, device=K_base.device)
    if tuple(K_full.shape) != shape or not K_full.is_contiguous() or not V_full.is_contiguous():
        raise ValueError("K_full/V_full must be contiguous [B, s_cap, n_kv, d]")
    st = lib().materialize_agent_kv(ctypes.byref(dims), _ptr(K_base), _ptr(V_base), _ptr(L_k), _ptr(L_v),
                                    _ptr(B_k), _ptr(B_v), _ptr(kv_len), _ptr(K_full), _ptr(V_full),
                                    _stream(stream))
    _check("materialize_agent_kv", st)
    return K_full, V_full


def _pool_stride(t, batch, ndim):
    """Elements between requests' pools: 0 for one pool (``ndim`` dims) shared by all."""
    if t is None or t.dim() == ndim:
        return 0
    if t.dim() != ndim + 1 or t.shape[0] not in (1, batch):
        raise ValueError(f"pool shape {tuple(t.shape)}: expected {ndim} dims, or {ndim + 1} with a leading 1 or {batch}")
    return 0 if t.shape[0] == 1 else t.stride(0)


def lr_shared_attention_paged(Q, K_pool, V_pool, L_k, L_v, B_k, B_v, positions, kv_len, kv_block_table, *,
                              rope_theta: float, lr_block_table=None, softmax_scale: float = 0.0, O=None,
                              lse=None, want_lse: bool = False, workspace=None, stream=None):
    """:func:`lr_shared_attention` over paged caches (block tables), e.g. one chunk
    of a chunked prefill over the tokens written so far.

    ``K_pool, V_pool [n_kv_blocks, blk, n_kv, d]`` (one pool) or
    ``[B, n_kv_blocks, blk, n_kv, d]`` (a pool per request); ``L_k, L_v
    [n_lr_blocks, blk, r]`` or ``[B, n_lr_blocks, blk, r]`` or None;
    ``B_k, B_v [B|1, r, n_kv*d]``; ``kv_block_table`` (and ``lr_block_table``,
    default: the same) ``[B, max_blocks]`` int32.
    """
    for name, t in (("K_pool", K_pool), ("V_pool", V_pool), ("L_k", L_k), ("L_v", L_v)):
        if t is not None:
            _bf16(name, t, t.dim())
            if not t.is_contiguous() and not t[0].is_contiguous():
                raise ValueError(f"{name} must be contiguous within a request")
    _bf16("Q", Q, 4)
    _bf16("B_k", B_k, 3)
    _bf16("B_v", B_v, 3)
    batch, n_tok, n_q, d = Q.shape
    if K_pool.shape != V_pool.shape or K_pool.stride() != V_pool.stride():
        raise ValueError("K_pool and V_pool must share shape and strides")
    if L_k is not None and L_v is not None and (L_k.shape != L_v.shape or L_k.stride() != L_v.stride()):
        raise ValueError("L_k and L_v must share shape and strides")
    if B_k is not None and B_v is not None and (B_k.shape != B_v.shape or B_k.stride() != B_v.stride()):
        raise ValueError("B_k and B_v must share shape and strides")
    n_kv_blocks, blk, n_kv, dk = K_pool.shape[-4:]
    if dk != d:
        raise ValueError("head dims of Q and K_pool differ")
    lr = L_k if L_k is not None else L_v
    bt = B_k if B_k is not None else B_v
    rank = lr.shape[-1] if lr is not None else 0
    n_lr_blocks = lr.shape[-3] if lr is not None else 0
    if lr is not None and lr.shape[-2] != blk:
        raise ValueError(f"LR pool blocks hold {lr.shape[-2]} tokens, base pool blocks {blk}")
    if bt is not None and (bt.shape[-2] != rank or bt.shape[-1] != n_kv * d):
        raise ValueError(f"up-projection shape {tuple(bt.shape)} is not (.., {rank}, {n_kv * d})")
    for name, t in (("kv_block_table", kv_block_table), ("lr_block_table", lr_block_table)):
        if t is None:
            continue
        if t.dtype != torch.int32 or t.dim() != 2 or t.shape[0] != batch or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous int32 [B, max_blocks] tensor")
    max_blocks = kv_block_table.shape[1]
    if lr_block_table is not None and lr_block_table.shape[1] != max_blocks:
        raise ValueError("the two block tables must have the same width")
    dims = LrsaDims(batch=batch, n_tok=n_tok, n_q_heads=n_q, n_kv_heads=n_kv, head_dim=d, rank=rank,
                    s_cap=max_blocks * blk, kv_req_stride=_pool_stride(K_pool, batch, 4),
                    l_req_stride=_pool_stride(lr, batch, 3), b_req_stride=_req_stride(bt, batch),
                    softmax_scale=softmax_scale, reserved0=0.0, rope_theta=rope_theta)
    paging = LrsaPaging(kv_block_table=kv_block_table.data_ptr(),
                        lr_block_table=None if lr_block_table is None else lr_block_table.data_ptr(),
                        block_size=blk, max_blocks=max_blocks, n_kv_blocks=n_kv_blocks, n_lr_blocks=n_lr_blocks)
    if positions.dtype != torch.int32 or kv_len.dtype != torch.int32:
        raise TypeError("positions and kv_len must be int32")
    if tuple(positions.shape) != (batch, n_tok) or not positions.is_contiguous():
        raise ValueError("positions must be a contiguous [B, n_tok] tensor")
    if tuple(kv_len.shape) != (batch,):
        raise ValueError("kv_len must be a [B] tensor")
    if O is None:
        O = torch.empty_like(Q)
    if lse is None and want_lse:
        lse = torch.empty(Q.shape[:3], dtype=torch.float32, device=Q.device)
    need = int(lib().lr_shared_attention_paged_workspace_size(ctypes.byref(dims)))
    if need and (workspace is None or workspace.numel() * workspace.element_size() < need):
        workspace = torch.empty(need, dtype=torch.uint8, device=Q.device)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = lib().lr_shared_attention_paged(ctypes.byref(dims), ctypes.byref(paging), _ptr(Q), _ptr(K_pool),
                                         _ptr(V_pool), _ptr(L_k), _ptr(L_v), _ptr(B_k), _ptr(B_v),
                                         _ptr(positions), _ptr(kv_len), _ptr(O), _ptr(lse), _ptr(workspace),
                                         ws_bytes, _stream(stream))
    _check("lr_shared_attention_paged", st)
    return O, lse


def stream_read(src, sink, grid: int, stream=None):
    """Measurement helper: stream all of ``src`` (a device tensor) through
    ``prc_stream_read``; ``sink`` is a uint32/int32 device tensor of ``grid``
    elements."""
    nbytes = src.numel() * src.element_size()
    if sink.numel() < grid or sink.element_size() != 4:
        raise ValueError("sink must hold grid 4-byte words")
    _check("prc_stream_read", lib().prc_stream_read(_ptr(src), nbytes, _ptr(sink), grid, _stream(stream)))
