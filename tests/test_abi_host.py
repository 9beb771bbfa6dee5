"""C-ABI checks that need no GPU: the library loads, exports every function
include/precache.h declares, and rejects bad arguments on the host before any
HIP call (so nothing here launches a kernel)."""
import ctypes
import os
import re

import pytest

import paper_2609_34054_amd as prc
from paper_2609_34054_amd.binding import LrsaDims

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "precache.h")

EINVAL, ESHAPE, EALIGN, EUNSUP, EWS = 1, 2, 3, 4, 5
A16 = 0x10000  # fake 16-byte-aligned addresses: never dereferenced on the host


def declared_functions():
    src = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    return sorted(set(re.findall(r"^(?:prc_status|size_t|const char\*|int)\s+(\w+)\s*\(", src, flags=re.M)))


def test_header_declares_the_boundary():
    assert declared_functions() == sorted(prc.EXPORTS)


def test_library_exports_every_declared_symbol():
    L = prc.lib()
    for name in declared_functions():
        assert hasattr(L, name), f"libprecache.so does not export {name}"
    out = os.popen(f"nm -D --defined-only {L._name}").read()
    exported = {ln.split()[-1] for ln in out.splitlines() if " T " in ln}
    assert exported == set(declared_functions()), exported ^ set(declared_functions())


def test_checked_build_exports_the_same_boundary():
    """libprecache_checked.so (device-side kv_len/position checks) exports
    exactly the release library's symbols and says which build it is."""
    from paper_2609_34054_amd.build import CHECKED_LIB_PATH
    C = ctypes.CDLL(CHECKED_LIB_PATH)
    out = os.popen(f"nm -D --defined-only {CHECKED_LIB_PATH}").read()
    exported = {ln.split()[-1] for ln in out.splitlines() if " T " in ln}
    assert exported == set(declared_functions())
    C.prc_status_string.restype = ctypes.c_char_p
    assert C.prc_device_checks() == 1 and prc.lib().prc_device_checks() == 0
    assert C.prc_status_string(8).decode() == "PRC_EDEVDATA"


def test_checked_library_is_selectable():
    from paper_2609_34054_amd.binding import use_checked_library
    try:
        use_checked_library(True)
        assert prc.lib().prc_device_checks() == 1
    finally:
        use_checked_library(False)
    assert prc.lib().prc_device_checks() == 0


def test_version_and_status_strings():
    L = prc.lib()
    assert L.prc_version().decode() == prc.__version__
    for code, name in prc.binding.STATUS_NAMES.items():
        assert L.prc_status_string(code).decode() == name


# ----------------------------------------------------------------- precompute
def _pc(X=A16, T=64, d_in=256, ld_x=256, A=A16, n_proj=2, N=3, r=8, L=A16, s_cap=128, off=0):
    return prc.lib().precompute_lr_cache(X, T, d_in, ld_x, A, n_proj, N, r, L, s_cap, off, None)


@pytest.mark.parametrize("kw,code", [
    (dict(T=-1), EINVAL),
    (dict(d_in=12, ld_x=16), EUNSUP),
    (dict(d_in=0), EUNSUP),
    (dict(ld_x=128), ESHAPE),
    (dict(ld_x=260), EALIGN),
    (dict(ld_x=1 << 24), EUNSUP),
    (dict(n_proj=0), EINVAL),
    (dict(N=0), EINVAL),
    (dict(r=12), EUNSUP),
    (dict(r=128), EUNSUP),
    (dict(s_cap=0), EINVAL),
    (dict(s_cap=1 << 31), EINVAL),
    (dict(off=100), ESHAPE),
    (dict(off=-1), ESHAPE),
    (dict(X=None), EINVAL),
    (dict(A=None), EINVAL),
    (dict(L=None), EINVAL),
    (dict(X=A16 + 8), EALIGN),
    (dict(L=A16 + 2), EALIGN),
])
def test_precompute_rejects(kw, code):
    assert _pc(**kw) == code
    assert prc.lib().prc_last_error().decode()


def test_precompute_empty_segment_is_a_noop():
    assert _pc(T=0, X=None, A=None, L=None) == 0


EDEVICE = 7


def test_valid_calls_need_a_gfx950_device():
    # Every argument check passes; the device check comes last, before any
    # launch, and this host has no GPU.
    assert _pc() == EDEVICE
    assert "device" in prc.lib().prc_last_error().decode()
    assert _pj() == EDEVICE
    d = _dims(n_tok=1)
    need = prc.lib().lr_shared_attention_workspace_size(ctypes.byref(d))
    assert _attn(d, ws=A16, ws_bytes=need) == EDEVICE
    assert _attn(_dims(n_tok=64, s_cap=256)) == EDEVICE
    assert _mat(_dims()) == EDEVICE


# -------------------------------------------------------- fused projection
def _pj(X=A16, T=64, d_in=256, ld_x=256, W=A16, n_kv=2, d=128, A=A16, n_proj=2, N=3, r=8, theta=1e4,
        K=A16, V=A16, L=A16, s_cap=128, off=0):
    return prc.lib().project_kv_and_lr_cache(X, T, d_in, ld_x, W, n_kv, d, A, n_proj, N, r, theta, K, V, L,
                                             s_cap, off, None)


@pytest.mark.parametrize("kw,code", [
    (dict(T=-1), EINVAL),
    (dict(d_in=12, ld_x=16), EUNSUP),
    (dict(ld_x=128), ESHAPE),
    (dict(ld_x=260), EALIGN),
    (dict(d=96), EUNSUP),
    (dict(d=32), EUNSUP),
    (dict(n_kv=0), EINVAL),
    (dict(n_kv=4096, d_in=65536, ld_x=65536), EUNSUP),
    (dict(N=-1), EINVAL),
    (dict(r=12), EUNSUP),
    (dict(theta=0.0), EINVAL),
    (dict(theta=-1.0), EINVAL),
    (dict(s_cap=0), EINVAL),
    (dict(s_cap=1 << 31), EINVAL),
    (dict(off=100), ESHAPE),
    (dict(W=None), EINVAL),
    (dict(K=None), EINVAL),
    (dict(V=None), EINVAL),
    (dict(L=None), EINVAL),
    (dict(W=A16 + 8), EALIGN),
    (dict(K=A16 + 2), EALIGN),
])
def test_projection_rejects(kw, code):
    assert _pj(**kw) == code
    assert prc.lib().prc_last_error().decode()


def test_projection_empty_segment_is_a_noop():
    assert _pj(T=0, X=None, W=None, A=None, K=None, V=None, L=None) == 0


def test_projection_without_lr_planes_needs_no_lr_buffers():
    # Rejected for a host-visible reason after the LR buffers were excused.
    assert _pj(N=0, A=None, L=None, off=100) == ESHAPE
    assert _pj(n_proj=0, A=None, L=None, r=12, K=None) == EINVAL


# ----------------------------------------------------- paged fused projection
def _pjp(X=A16, T=64, d_in=256, ld_x=256, W=A16, n_kv=2, d=128, A=A16, n_proj=2, N=3, r=8, theta=1e4,
         K=A16, V=A16, L=A16, tbl=A16, blk=128, max_blocks=4, n_blocks=16, off=0):
    return prc.lib().project_kv_and_lr_cache_paged(X, T, d_in, ld_x, W, n_kv, d, A, n_proj, N, r, theta, K, V,
                                                   L, tbl, blk, max_blocks, n_blocks, off, None)


@pytest.mark.parametrize("kw,code", [
    (dict(blk=0), EUNSUP),
    (dict(blk=96), EUNSUP),
    (dict(blk=-64), EUNSUP),
    (dict(max_blocks=0), EINVAL),
    (dict(n_blocks=0), EINVAL),
    (dict(max_blocks=1 << 25), EINVAL),   # max_blocks * blk reaches 2^31
    (dict(n_blocks=1 << 25), EINVAL),
    (dict(off=500), ESHAPE),              # 500 + 64 > 4 * 128
    (dict(tbl=None), EINVAL),
    (dict(tbl=A16 + 2), EALIGN),
    (dict(n_kv=-1), EINVAL),
    (dict(n_kv=0, N=0), EINVAL),          # nothing asked for
    (dict(d=96), EUNSUP),
    (dict(K=None), EINVAL),
    (dict(L=None), EINVAL),
    (dict(r=12), EUNSUP),
])
def test_paged_projection_rejects(kw, code):
    assert _pjp(**kw) == code
    assert prc.lib().prc_last_error().decode()


def test_paged_projection_lr_only_and_base_only_excuse_buffers():
    # LR planes alone: no weights, no base pools, head_dim and theta unused.
    # Each call stops at a host check placed after the excused buffers.
    assert _pjp(n_kv=0, W=None, K=None, V=None, d=0, theta=0.0, off=500) == ESHAPE
    assert _pjp(n_kv=0, W=None, K=None, V=None, d=0, theta=0.0, tbl=A16 + 2) == EALIGN
    assert _pjp(N=0, A=None, L=None, r=12, tbl=A16 + 2) == EALIGN
    assert _pjp(T=0, X=None, W=None, A=None, K=None, V=None, L=None, tbl=None) == 0


# ------------------------------------------------------------------ attention
def _dims(**kw):
    d = dict(batch=2, n_tok=4, n_q_heads=32, n_kv_heads=8, head_dim=128, rank=16, s_cap=1024,
             kv_req_stride=1024 * 8 * 128, l_req_stride=1024 * 16, b_req_stride=8 * 128 * 16,
             softmax_scale=0.0, reserved0=0.0, rope_theta=5e5)
    d.update(kw)
    return LrsaDims(**d)


def _attn(dims, Q=A16, K=A16, V=A16, Lk=A16, Lv=A16, Bk=A16, Bv=A16, pos=A16, kvl=A16, O=A16, lse=None,
          ws=None, ws_bytes=0):
    return prc.lib().lr_shared_attention(ctypes.byref(dims), Q, K, V, Lk, Lv, Bk, Bv, pos, kvl, O, lse, ws,
                                         ws_bytes, None)


@pytest.mark.parametrize("kw,code", [
    (dict(batch=-1), EINVAL),
    (dict(batch=70000), EINVAL),
    (dict(n_tok=-2), EINVAL),
    (dict(n_q_heads=30), ESHAPE),
    (dict(n_q_heads=0), EINVAL),
    (dict(n_q_heads=80, n_kv_heads=5), EUNSUP),
    (dict(head_dim=96), EUNSUP),
    (dict(head_dim=256), EUNSUP),
    (dict(rank=12), EUNSUP),
    (dict(s_cap=0), EINVAL),
    (dict(rope_theta=0.0), EINVAL),
    (dict(rope_theta=float("inf")), EINVAL),
    (dict(softmax_scale=float("nan")), EINVAL),
    (dict(reserved0=1.0), EINVAL),
    (dict(kv_req_stride=1000), ESHAPE),
    (dict(kv_req_stride=1024 * 8 * 128 + 4), EALIGN),
    (dict(l_req_stride=100), ESHAPE),
    (dict(b_req_stride=100), ESHAPE),
    (dict(l_req_stride=-8), EINVAL),
])
def test_attention_rejects_dims(kw, code):
    assert _attn(_dims(**kw)) == code


@pytest.mark.parametrize("kw,code", [
    (dict(Lk=None), EINVAL),          # L_k without B_k
    (dict(Bv=None), EINVAL),          # B_v without L_v
    (dict(Q=None), EINVAL),
    (dict(K=None), EINVAL),
    (dict(pos=None), EINVAL),
    (dict(kvl=None), EINVAL),
    (dict(O=None), EINVAL),
    (dict(Q=A16 + 4), EALIGN),
    (dict(V=A16 + 8), EALIGN),
    (dict(Bk=A16 + 2), EALIGN),
    (dict(O=A16 + 6), EALIGN),
    (dict(kvl=A16 + 2), EALIGN),
])
def test_attention_rejects_pointers(kw, code):
    assert _attn(_dims(), **kw) == code


def test_attention_empty_batch_is_a_noop():
    assert _attn(_dims(batch=0), Q=None, K=None, V=None, pos=None, kvl=None, O=None) == 0
    assert _attn(_dims(n_tok=0), Q=None, K=None, V=None, pos=None, kvl=None, O=None) == 0


def test_rank_ignored_without_lr_cache():
    # A plain call (no LR cache) never looks at rank, so an unbuilt rank is
    # fine there; it only fails once an LR cache is passed.  Workspace is the
    # first missing piece of this decode call, so the check stops there.
    d = _dims(n_tok=1, rank=0)
    assert _attn(d, Lk=None, Lv=None, Bk=None, Bv=None) == EWS
    assert _attn(d) == EUNSUP


def test_decode_workspace_query_and_check():
    L = prc.lib()
    d = _dims(n_tok=1)
    need = L.lr_shared_attention_workspace_size(ctypes.byref(d))
    assert need > 0
    # Prefill needs no split partials when one pass per KV head already fills
    # the chip (4096 queries, 8 KV heads) or the context is a handful of
    # tiles.  With an LR rank and 64 row tiles per KV head the query asks for
    # the optional tile cache instead: one flag per wave and tile, then 32 KB
    # of rebuilt K and V^T per tile (576 tiles x 8 KV heads).
    tiles = 36864 // 64
    cache = -(-(8 * tiles * 8 * 4) // 256) * 256 + 8 * tiles * 32768
    assert L.lr_shared_attention_workspace_size(ctypes.byref(_dims(n_tok=4096, batch=1, s_cap=36864))) == cache
    # Rank 8 takes it too (its L_v^T fragments stay outside the cached tile).
    assert L.lr_shared_attention_workspace_size(ctypes.byref(_dims(n_tok=4096, batch=1, s_cap=36864, rank=8))) == cache
    # No LR rank (plain attention), few row tiles, or paged caches: no cache.
    assert L.lr_shared_attention_workspace_size(ctypes.byref(_dims(n_tok=4096, batch=1, s_cap=36864, rank=0))) == 0
    assert L.lr_shared_attention_workspace_size(ctypes.byref(_dims(n_tok=8, s_cap=256))) == 0
    assert L.lr_shared_attention_paged_workspace_size(ctypes.byref(_dims(n_tok=4096, batch=1, s_cap=36864))) == 0
    assert _attn(d, ws=None) == EWS
    assert _attn(d, ws=A16, ws_bytes=need - 1) == EWS
    assert _attn(d, ws=A16 + 4, ws_bytes=need) == EALIGN
    # Workspace grows with the batch and shrinks to a single split for short
    # contexts.
    big = L.lr_shared_attention_workspace_size(ctypes.byref(_dims(n_tok=1, batch=16, s_cap=32768)))
    assert big >= 16 * 32 * (4 + 128 + 16) * 4


def test_split_prefill_workspace_query_and_check():
    # A small prefill over a long context splits its KV range: the call then
    # needs one fp32 partial (max, sum, d + r accumulators) per query row,
    # head and split, and refuses a missing or short workspace.
    L = prc.lib()
    d = _dims(n_tok=8, batch=2, s_cap=8192, kv_req_stride=8192 * 8 * 128, l_req_stride=8192 * 16)
    need = L.lr_shared_attention_workspace_size(ctypes.byref(d))
    rows = 2 * 8 * 32
    assert need > 0 and need % (rows * (4 + 128 + 16) * 4) == 0
    assert 2 <= need // (rows * (4 + 128 + 16) * 4) <= 8
    assert _attn(d, ws=None) == EWS
    assert _attn(d, ws=A16, ws_bytes=need - 1) == EWS
    assert _attn(d, ws=A16 + 4, ws_bytes=need) == EALIGN


# ------------------------------------------------------------ paged attention
def _paging(**kw):
    from paper_2609_34054_amd.binding import LrsaPaging
    p = dict(kv_block_table=A16, lr_block_table=None, block_size=128, max_blocks=8, n_kv_blocks=64,
             n_lr_blocks=16)
    p.update(kw)
    return LrsaPaging(**p)


def _pdims(**kw):
    d = dict(s_cap=1024, kv_req_stride=0, l_req_stride=16 * 128 * 16)
    d.update(kw)
    return _dims(**d)


def _pattn(dims, paging, Q=A16, K=A16, V=A16, Lk=A16, Lv=A16, Bk=A16, Bv=A16, pos=A16, kvl=A16, O=A16,
           lse=None, ws=None, ws_bytes=0):
    pg = None if paging is None else ctypes.byref(paging)
    return prc.lib().lr_shared_attention_paged(ctypes.byref(dims), pg, Q, K, V, Lk, Lv, Bk, Bv, pos, kvl, O,
                                               lse, ws, ws_bytes, None)


@pytest.mark.parametrize("dkw,pkw,code", [
    (dict(), dict(block_size=0), EUNSUP),
    (dict(), dict(block_size=100), EUNSUP),
    (dict(), dict(max_blocks=0), EINVAL),
    (dict(), dict(n_kv_blocks=0), EINVAL),
    (dict(), dict(n_lr_blocks=0), EINVAL),
    (dict(s_cap=2048), dict(), ESHAPE),                  # s_cap != max_blocks * block_size
    (dict(kv_req_stride=64 * 128 * 8 * 128 - 8), dict(), ESHAPE),  # < one request's pools
    (dict(l_req_stride=16 * 128 * 16 - 8), dict(), ESHAPE),
    (dict(), dict(kv_block_table=None), EINVAL),
    (dict(), dict(kv_block_table=A16 + 2), EALIGN),
    (dict(), dict(lr_block_table=A16 + 2), EALIGN),
    (dict(head_dim=96), dict(), EUNSUP),
])
def test_paged_attention_rejects(dkw, pkw, code):
    assert _pattn(_pdims(**dkw), _paging(**pkw)) == code
    assert prc.lib().prc_last_error().decode()


def test_paged_attention_needs_paging_and_lr_pools_only_with_lr():
    assert _pattn(_pdims(), None) == EINVAL
    # Without LR caches the LR pool size is never looked at.  The call then
    # stops at the first missing piece of a decode call, the workspace.
    d = _pdims(n_tok=1)
    assert _pattn(d, _paging(n_lr_blocks=0), Lk=None, Lv=None, Bk=None, Bv=None) == EWS
    assert _pattn(_pdims(batch=0), _paging(kv_block_table=None), Q=None, K=None, V=None, pos=None, kvl=None,
                  O=None) == 0


def test_paged_decode_workspace_is_the_per_request_plan():
    L = prc.lib()
    # One base pool shared by all requests (kv_req_stride 0): the contiguous
    # call would take the shared-base kernel; the paged one never does, and
    # sizes its workspace for the per-request split plan.
    d = _pdims(n_tok=1, batch=16, s_cap=32768)
    need = L.lr_shared_attention_paged_workspace_size(ctypes.byref(d))
    assert need > 0
    assert need == L.lr_shared_attention_workspace_size(ctypes.byref(_dims(n_tok=1, batch=16, s_cap=32768)))
    pg = _paging(max_blocks=256)
    assert _pattn(d, pg, ws=A16, ws_bytes=need - 1) == EWS
    assert _pattn(d, pg, ws=A16 + 4, ws_bytes=need) == EALIGN


# ---------------------------------------------------------------- materialise
def _mat(dims, K=A16, V=A16, Lk=A16, Lv=A16, Bk=A16, Bv=A16, kvl=A16, Kf=0x4000000, Vf=0x8000000):
    return prc.lib().materialize_agent_kv(ctypes.byref(dims), K, V, Lk, Lv, Bk, Bv, kvl, Kf, Vf, None)


def test_materialize_rejects():
    d = _dims()
    assert _mat(d, Kf=None) == EINVAL
    assert _mat(d, Vf=0x4000000 + 8) == EALIGN
    assert _mat(d, Kf=A16) == EINVAL          # output overlaps K_base
    assert _mat(d, Vf=0x4000000 + 16) == EINVAL  # K_full and V_full overlap
    # An output that starts inside an input's extent (K_base spans 2 requests
    # of 1024 x 8 x 128 elements from A16) overlaps it too.
    assert _mat(d, Kf=A16 + (1 << 20)) == EINVAL
    assert _mat(d, Kf=A16 + 2 * 1024 * 8 * 128 * 2 + (16 << 20)) == EDEVICE
    assert _mat(_dims(head_dim=80)) == EUNSUP
    assert _mat(_dims(batch=0), K=None, V=None, kvl=None) == 0


def test_python_wrappers_refuse_wrong_dtypes():
    import torch
    X = torch.zeros(4, 8, dtype=torch.float32)
    with pytest.raises(TypeError):
        prc.precompute_lr_cache(X, X, 1, 1, 8, torch.zeros(1, 1, 4, 8))


@pytest.mark.parametrize("n_tok,n_q,s_cap,splits", [
    (512, 32, 8704, 4),      # 64 units: one round of 4 splits beats two of 8
    (256, 32, 65920, 8),     # 32 units
    (2048, 40, 67584, 4),    # 320 units: 1280 workgroups, five full rounds
    (4096, 32, 36864, 1),    # 512 units: two full rounds already
    (16, 32, 256, 1),        # 4 tiles: too short to split
    (16128, 32, 65536, 1),   # 2016 units: 8 splits would gain 1.6%, below the 10% bar
    (4104, 32, 36864, 8),    # 520 units: a third round for 8 units; 8 splits gain 29%
])
def test_prefill_split_count(n_tok, n_q, s_cap, splits):
    """The prefill split count minimises ceil(units * ns / 256) / ns over
    ns in 1..8 (splits at least 8 tiles), smallest on ties, and splits only
    when that gains at least 10% over one pass; the workspace query reports
    one fp32 partial per row and split.  (The paged query: the same plan,
    without the optional tile cache that unsplit contiguous calls ask for.)"""
    d = _dims(batch=1, n_tok=n_tok, n_q_heads=n_q, n_kv_heads=8, s_cap=s_cap, kv_req_stride=0, l_req_stride=0,
              b_req_stride=0)
    need = prc.lib().lr_shared_attention_paged_workspace_size(ctypes.byref(d))
    assert need == (0 if splits == 1 else n_tok * n_q * splits * (4 + 128 + 16) * 4)


@pytest.mark.parametrize("batch,s_cap,splits", [
    (16, 32768, 32),   # two rounds of 512 workgroups, 32-tile splits
    (1, 36864, 231),   # two rounds would cut splits to 3 tiles: one round
    (1, 66048, 230),
    (1, 4480, 140),    # one 32-token tile per split
])
def test_decode_split_count(batch, s_cap, splits):
    d = _dims(batch=batch, n_tok=1, s_cap=s_cap, kv_req_stride=s_cap * 8 * 128, l_req_stride=s_cap * 16)
    need = prc.lib().lr_shared_attention_workspace_size(ctypes.byref(d))
    assert need == batch * 32 * splits * (4 + 128 + 16) * 4


def test_noalloc_checks_size_before_the_device():
    # The call with no workspace argument rejects a call whose split partials
    # exceed its static buffer on the host, before any device call.
    L = prc.lib()
    d = _dims(n_tok=1, batch=4096, kv_req_stride=0, l_req_stride=0, b_req_stride=0)
    assert L.lr_shared_attention_workspace_size(ctypes.byref(d)) > 32 << 20
    args = [ctypes.byref(d), A16, A16, A16, A16, A16, A16, A16, A16, A16, A16, None, None]
    assert L.lr_shared_attention_noalloc(*args) == EWS
    assert "static workspace" in L.prc_last_error().decode()
    # Argument checks come first, as for lr_shared_attention.
    bad = _dims(n_tok=1, head_dim=96)
    assert L.lr_shared_attention_noalloc(ctypes.byref(bad), *args[1:]) == EUNSUP
    ok = _dims(n_tok=1)
    assert L.lr_shared_attention_noalloc(ctypes.byref(ok), *args[1:]) == 7  # no gfx950 device here


def test_stream_read_helper_checks_arguments():
    L = prc.lib()
    assert L.prc_stream_read(None, 1 << 20, A16, 64, None) == EINVAL
    assert L.prc_stream_read(A16, 100, A16, 64, None) == EINVAL
    assert L.prc_stream_read(A16 + 8, 1 << 20, A16, 64, None) == EALIGN
    assert L.prc_stream_read(A16, 1 << 20, A16, 0, None) == EINVAL
    assert L.prc_stream_read(A16, 1 << 20, A16, 64, None) == 7  # no gfx950 device here
