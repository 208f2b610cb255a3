"""Host-side checks of the C-ABI library that need no GPU: it loads, exports every function
that include/tfm_layer.h declares, answers the size queries, and rejects invalid arguments with
the documented codes before launching anything."""

import ctypes
import os
import re

import numpy as np
import pytest

from paper_2606_03681_amd import tfm
from paper_2606_03681_amd import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    names = set()
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            text = open(os.path.join(ROOT, "include", fn)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names |= set(re.findall(r"\b(tfm_\w+)\s*\(", text))
    return names


def test_library_exports_every_declared_symbol():
    L = tfm.lib()
    declared = _declared_functions()
    assert declared >= set(tfm.EXPORTS)
    for name in declared:
        assert hasattr(L, name), name


def _dims(**kw):
    base = dict(B=2, R=64, C=8, E=64, heads=4, H=128, dtype="f32")
    base.update(kw)
    return tfm.make_dims(**base)


def test_param_count_matches_formula():
    for E, H in ((64, 128), (192, 384), (256, 768)):
        heads = E // 32
        d = _dims(E=E, H=H, heads=heads)
        assert tfm.param_count(d) == 8 * E * E + 8 * E + 2 * E * H + H + 7 * E
        assert tfm.param_count(d) == wl.param_count(E, H)
    assert tfm.param_count(_dims(E=192, H=384, heads=6)) == 445632


def test_prenorm_param_count_and_sizes():
    """The pre-norm block drops the three LayerNorm shifts; its packed count matches the
    workload generator's layout, and its saved state has room for x' and the norm outputs."""
    for E, H, heads in ((64, 192, 2), (192, 384, 6), (256, 768, 8)):
        d = _dims(E=E, H=H, heads=heads, dtype="bf16", block="pre", decay=0.95)
        assert tfm.param_count(d) == 8 * E * E + 8 * E + 2 * E * H + H + 4 * E
        assert tfm.param_count(d) == wl.param_count(E, H, "pre")
        post = _dims(E=E, H=H, heads=heads, dtype="bf16")
        assert tfm.param_count(post) - tfm.param_count(d) == 3 * E
        assert tfm.saved_bytes(d) > 0 and tfm.workspace_bytes(d) > 0


def test_sizes_positive_and_grow_with_batch():
    d1, d2 = _dims(), _dims(B=4)
    assert 0 < tfm.saved_bytes(d1) < tfm.saved_bytes(d2)
    assert 0 < tfm.workspace_bytes(d1) < tfm.workspace_bytes(d2)


@pytest.mark.parametrize("kw,code", [
    (dict(B=0), -1), (dict(R=0), -1), (dict(C=-1), -1), (dict(C=300), -1),
    (dict(E=48), -1), (dict(E=512), -1), (dict(H=100), -1), (dict(dtype=7), -1),
    (dict(heads=3), -2), (dict(E=128, heads=1), -2), (dict(E=256, heads=2), -2),
    (dict(block=2), -1), (dict(block="pre"), -1),                  # pre-norm needs bf16
    (dict(block="pre", dtype="bf16", E=96, heads=3), -1),          # ... and E in {64,...,256}
    (dict(block="pre", dtype="bf16", H=96), -1),                   # ... and H % E == 0
    (dict(block="pre", dtype="bf16", decay=float("nan")), -1),
    (dict(B=1, R=1 << 20, C=15, E=256, heads=4), -1),          # one dataset's Q|K|V > 4 GiB
    (dict(B=20, R=1 << 20, C=3), -1),                          # more than 2^26 cells
])
def test_invalid_dims_rejected(kw, code):
    d = _dims(**kw)
    assert tfm.param_count(d) == 0
    assert tfm.saved_bytes(d) == 0
    fake = 1 << 20
    rc = tfm.lib().tfm_layer_fwd(ctypes.byref(d), None, None, fake, fake, fake, fake, 1 << 40,
                                 fake, 1 << 40, None)
    assert rc == code
    assert tfm.last_error()


def _call_fwd(d, n_train, mask, ptr=1 << 20, sb=1 << 40, wb=1 << 40):
    nt = np.ascontiguousarray(n_train, dtype=np.int32)
    cm = np.ascontiguousarray(mask, dtype=np.uint8)
    return tfm.lib().tfm_layer_fwd(ctypes.byref(d), nt.ctypes.data, cm.ctypes.data, ptr, ptr,
                                   ptr, ptr, sb, ptr, wb, None)


def _call_bwd(d, n_train, mask, ptr=1 << 20, sb=1 << 40, wb=1 << 40):
    nt = np.ascontiguousarray(n_train, dtype=np.int32)
    cm = np.ascontiguousarray(mask, dtype=np.uint8)
    return tfm.lib().tfm_layer_bwd(ctypes.byref(d), nt.ctypes.data, cm.ctypes.data, ptr, ptr,
                                   ptr, sb, ptr, ptr, ptr, 0, ptr, wb, None)


@pytest.mark.parametrize("call", [_call_fwd, _call_bwd])
def test_bad_metadata_and_pointers_rejected_before_launch(call):
    d = _dims()
    mask = np.ones((2, 9), np.uint8)
    assert call(d, [0, 5], mask) == -3
    assert call(d, [5, 65], mask) == -3
    assert "n_train" in tfm.last_error()
    bad = mask.copy()
    bad[1, 8] = 0
    assert call(d, [5, 5], bad) == -4
    assert call(d, [5, 5], mask, ptr=0) == -5
    assert call(d, [5, 5], mask, ptr=(1 << 20) + 4) == -5
    assert call(d, [5, 5], mask, sb=16) == -7
    assert call(d, [5, 5], mask, wb=16) == -7
    rc = tfm.lib().tfm_layer_fwd(ctypes.byref(d), None, None, 1 << 20, 1 << 20, 1 << 20,
                                 1 << 20, 1 << 40, 1 << 20, 1 << 40, None)
    assert rc == -5


def _call_think(d, n_train, mask, T, ptr=1 << 20, wb=1 << 40, bwd=False):
    nt = np.ascontiguousarray(n_train, dtype=np.int32)
    cm = np.ascontiguousarray(mask, dtype=np.uint8)
    if bwd:
        return tfm.lib().tfm_thinking_rows_bwd(ctypes.byref(d), nt.ctypes.data, cm.ctypes.data,
                                               T, ptr, ptr, 0, ptr, wb, None)
    return tfm.lib().tfm_thinking_rows_fwd(ctypes.byref(d), nt.ctypes.data, cm.ctypes.data, T,
                                           ptr, ptr, ptr, wb, None)


@pytest.mark.parametrize("bwd", [False, True])
def test_thinking_rows_arguments_rejected_before_launch(bwd):
    d = _dims()
    mask = np.ones((2, 9), np.uint8)
    assert _call_think(d, [5, 5], mask, 0, bwd=bwd) == -1
    assert _call_think(d, [5, 3], mask, 4, bwd=bwd) == -1
    assert "thinking rows" in tfm.last_error()
    assert _call_think(d, [0, 5], mask, 1, bwd=bwd) == -3
    bad = mask.copy()
    bad[0, 8] = 0
    assert _call_think(d, [5, 5], bad, 1, bwd=bwd) == -4
    assert _call_think(d, [5, 5], mask, 1, ptr=0, bwd=bwd) == -5
    assert _call_think(d, [5, 5], mask, 1, ptr=(1 << 20) + 8, bwd=bwd) == -5
    assert _call_think(d, [5, 5], mask, 1, wb=16, bwd=bwd) == -7


def test_forward_only_sizes():
    d = _dims(dtype="bf16", E=192, heads=6, H=384, R=1024, C=100, B=16)
    wb = tfm.infer_workspace_bytes(d)
    assert 0 < wb < tfm.saved_bytes(d)
    cb = tfm.infer_cache_bytes(d)
    half = 16 * 101 * 1024 * 192 * 2
    assert cb == 2 * ((half + 255) // 256 * 256)
    assert tfm.infer_workspace_bytes(_dims(dtype="f32")) == 0
    assert "TFM_BF16" in tfm.last_error()
    pre = _dims(dtype="bf16", E=256, heads=4, H=768, block="pre")
    assert tfm.infer_workspace_bytes(pre) > tfm.infer_workspace_bytes(
        _dims(dtype="bf16", E=256, heads=4, H=768))


def _ctx(d, n_train, mask, ptr=1 << 20, cb=1 << 40, wb=1 << 40):
    nt = np.ascontiguousarray(n_train, dtype=np.int32)
    cm = np.ascontiguousarray(mask, dtype=np.uint8)
    return tfm.lib().tfm_layer_fwd_context(ctypes.byref(d), nt.ctypes.data, cm.ctypes.data, ptr,
                                           ptr, ptr, ptr, cb, ptr, wb, None)


def _qry(d, rc, n_train, mask, ptr=1 << 20, cb=1 << 40, wb=1 << 40):
    nt = np.ascontiguousarray(n_train, dtype=np.int32)
    cm = np.ascontiguousarray(mask, dtype=np.uint8)
    return tfm.lib().tfm_layer_fwd_query(ctypes.byref(d), rc, nt.ctypes.data, cm.ctypes.data,
                                         ptr, ptr, ptr, cb, ptr, ptr, wb, None)


def test_forward_only_arguments_rejected_before_launch():
    d = _dims(dtype="bf16")
    mask = np.ones((2, 9), np.uint8)
    assert _ctx(_dims(), [5, 5], mask) == -1              # fp32
    assert _ctx(d, [5, 65], mask) == -3
    assert _ctx(d, [5, 5], mask, ptr=0) == -5
    assert _ctx(d, [5, 5], mask, cb=16) == -7
    assert _ctx(d, [5, 5], mask, wb=16) == -7
    q = _dims(dtype="bf16", R=8)                          # 8 query rows
    assert _qry(q, 0, [5, 5], mask) == -1
    assert _qry(q, -3, [5, 5], mask) == -1
    assert _qry(q, 32, [5, 33], mask) == -3               # n_train beyond the context rows
    assert _qry(q, 32, [20, 32], mask, ptr=(1 << 20) + 2) == -5
    need = tfm.infer_cache_bytes(_dims(dtype="bf16", R=32))
    assert _qry(q, 32, [20, 32], mask, cb=need - 1) == -7
    assert "kv_cache" in tfm.last_error()
    bad = mask.copy()
    bad[1, 8] = 0
    assert _qry(q, 32, [20, 32], bad) == -4


# ---- the stack's two ends (include/tfm_ends.h) -------------------------------------------------

def _ends(**kw):
    base = dict(G=5, offsets=(0, 1, 3, 7, 12), F=8, T=0, Hd=96, K=10, decode_mean=1)
    base.update(kw)
    return tfm.make_ends(**base)


def test_ends_param_count_and_workspace():
    d = _dims(E=64)
    e = _ends()
    assert tfm.ends_param_count(d, e) == 64 * 5 + 3 * 64 + 96 * 64 + 96 + 10 * 96 + 10
    wb = tfm.ends_workspace_bytes(d, e)
    assert wb > 0
    # more rows, more decoder rows to hold
    assert tfm.ends_workspace_bytes(_dims(E=64, R=128), e) > wb
    # the decoder is sized for every row (the forward-only decoder takes tables without
    # labelled rows); thinking rows only shorten the encoders' row slabs
    assert tfm.ends_workspace_bytes(d, _ends(T=8)) <= wb


@pytest.mark.parametrize("kw", [dict(G=0, offsets=()), dict(K=65), dict(K=0), dict(T=64),
                                dict(T=-1), dict(Hd=0), dict(F=0), dict(decode_mean=2),
                                dict(G=1, offsets=(-1,)), dict(G=1, offsets=((1 << 20) + 1,))])
def test_ends_invalid_shape_rejected(kw):
    if kw.get("decode_mean") == 2:
        e = _ends()
        e.decode_mean = 2
    elif kw.get("G") == 0:
        e = _ends()
        e.G = 0
    else:
        e = _ends(**kw)
    assert tfm.ends_param_count(_dims(), e) == 0
    assert tfm.ends_workspace_bytes(_dims(), e) == 0
    assert tfm.last_error()


def _enc(d, e, n_train, n_feat, ptr=1 << 20, wb=1 << 40, bwd=False):
    nt = np.ascontiguousarray(n_train, dtype=np.int32)
    nf = np.ascontiguousarray(n_feat, dtype=np.int32)
    L = tfm.lib()
    if bwd:
        return L.tfm_encode_bwd(ctypes.byref(d), ctypes.byref(e), nt.ctypes.data, nf.ctypes.data,
                                ptr, ptr, ptr, ptr, 0, ptr, wb, None)
    return L.tfm_encode_fwd(ctypes.byref(d), ctypes.byref(e), nt.ctypes.data, nf.ctypes.data,
                            ptr, ptr, ptr, ptr, ptr, wb, None)


def _dec(d, e, n_train, n_feat, n_class, ptr=1 << 20, wb=1 << 40, logits=None):
    nt = np.ascontiguousarray(n_train, dtype=np.int32)
    nf = np.ascontiguousarray(n_feat, dtype=np.int32)
    nc = np.ascontiguousarray(n_class, dtype=np.int32)
    return tfm.lib().tfm_decode_loss(ctypes.byref(d), ctypes.byref(e), nt.ctypes.data,
                                     nf.ctypes.data, nc.ctypes.data, ptr, ptr, ptr, ptr, logits,
                                     ptr, ptr, 0, ptr, wb, None)


@pytest.mark.parametrize("bwd", [False, True])
def test_encoder_arguments_rejected_before_launch(bwd):
    d = _dims()                                   # B=2, R=64, C=8
    e = _ends(T=4)
    assert _enc(d, e, [4, 9], [8, 8], bwd=bwd) == -3      # no labelled data row
    assert "n_train" in tfm.last_error()
    assert _enc(d, e, [9, 65], [8, 8], bwd=bwd) == -3
    assert _enc(d, e, [9, 9], [0, 8], bwd=bwd) == -1
    assert _enc(d, e, [9, 9], [8, 9], bwd=bwd) == -1      # beyond C
    assert _enc(d, _ends(F=5), [9, 9], [6, 5], bwd=bwd) == -1   # beyond F
    assert "n_feat" in tfm.last_error()
    assert _enc(d, e, [9, 9], [8, 8], ptr=0, bwd=bwd) == -5
    assert _enc(d, e, [9, 9], [8, 8], ptr=(1 << 20) + 4, bwd=bwd) == -5
    assert _enc(d, e, [9, 9], [8, 8], wb=16, bwd=bwd) == -7
    assert _enc(_dims(C=0), e, [9, 9], [1, 1], bwd=bwd) == -1
    rc = tfm.lib().tfm_encode_fwd(ctypes.byref(d), ctypes.byref(e), None, None, 1 << 20,
                                  1 << 20, 1 << 20, 1 << 20, 1 << 20, 1 << 40, None)
    assert rc == -5


def test_decoder_arguments_rejected_before_launch():
    d = _dims()
    e = _ends()
    assert _dec(d, e, [9, 9], [8, 8], [2, 11]) == -1      # more classes than outputs
    assert "n_class" in tfm.last_error()
    assert _dec(d, e, [9, 9], [8, 8], [0, 2]) == -1
    assert _dec(d, e, [0, 9], [8, 8], [2, 2]) == -3
    assert _dec(d, e, [9, 9], [8, 8], [2, 2], ptr=0) == -5
    assert _dec(d, e, [9, 9], [8, 8], [2, 2], logits=(1 << 20) + 4) == -5
    assert _dec(d, e, [9, 9], [8, 8], [2, 2], wb=16) == -7
    nt = np.array([9, 9], np.int32)
    nf = np.array([8, 8], np.int32)
    rc = tfm.lib().tfm_decode_loss(ctypes.byref(d), ctypes.byref(e), nt.ctypes.data,
                                   nf.ctypes.data, None, 1 << 20, 1 << 20, 1 << 20, 1 << 20,
                                   None, 1 << 20, 1 << 20, 0, 1 << 20, 1 << 40, None)
    assert rc == -5


# ---- the optimiser step (include/tfm_optim.h) --------------------------------------------------

def _clip(nvec, counts, ptr=1 << 20, max_norm=1.0, wb=1 << 40, out=1 << 20):
    ptrs = (ctypes.c_void_p * max(nvec, 1))(*([ptr] * max(nvec, 1)))
    cnt = (ctypes.c_int64 * max(len(counts), 1))(*counts)
    return tfm.lib().tfm_clip_scale(nvec, ptrs, cnt, max_norm, out, None, 1 << 20, wb, None)


def test_clip_arguments_rejected_before_launch():
    assert _clip(0, [4]) == -1
    assert _clip(1, [-1]) == -1
    assert _clip(1, [8], ptr=0) == -5
    assert _clip(1, [8], ptr=(1 << 20) + 2) == -5
    assert _clip(1, [8], max_norm=0.0) == -1
    assert _clip(1, [8], max_norm=float("inf")) == -1
    assert _clip(1, [8], out=(1 << 20) + 4) == -5
    assert _clip(1, [8], wb=0) == -7
    assert tfm.clip_workspace_bytes([10, 5000]) == 256
    assert tfm.clip_workspace_bytes([4096 * 300]) == 300 * 4 + (256 - 300 * 4 % 256) % 256


def _sf(hp=None, t=1, segs=((0, 4),), ptr=1 << 20):
    hp = hp or tfm.tfm_sfadamw(1e-3, 0.9, 0.999, 1e-8, 0.0, 0)
    off = (ctypes.c_int64 * max(len(segs), 1))(*[o for o, _ in segs])
    ln = (ctypes.c_int64 * max(len(segs), 1))(*[n for _, n in segs])
    return tfm.lib().tfm_sfadamw_step(ctypes.byref(hp), t, len(segs), off, ln, ptr, ptr, ptr, ptr,
                                      None, None)


def test_sfadamw_arguments_rejected_before_launch():
    assert _sf(t=0) == -1
    assert _sf(segs=()) == -1
    assert _sf(segs=tuple((8 * k, 4) for k in range(65))) == -1
    assert _sf(segs=((0, 10), (8, 4))) == -1                 # overlap
    assert "overlap" in tfm.last_error()
    assert _sf(segs=((-1, 4),)) == -1
    assert _sf(hp=tfm.tfm_sfadamw(1e-3, 0.9, 1.0, 1e-8, 0.0, 0)) == -1
    assert _sf(hp=tfm.tfm_sfadamw(-1.0, 0.9, 0.9, 1e-8, 0.0, 0)) == -1
    assert _sf(hp=tfm.tfm_sfadamw(1e-3, 0.9, 0.9, 1e-8, 0.0, -2)) == -1
    assert _sf(ptr=0) == -5
    assert _sf(ptr=(1 << 20) + 2) == -5


def _mu(count=2, rows=8, cols=8, hp=None, ptr=1 << 20, wb=1 << 40):
    hp = hp or tfm.tfm_muon(0.02, 0.95, 0.0, 1, 5)
    arr = (ctypes.c_void_p * max(count, 1))(*([ptr] * max(count, 1)))
    return tfm.lib().tfm_muon_step(ctypes.byref(hp), count, rows, cols, arr, arr, arr, None,
                                   1 << 20, wb, None)


def test_muon_arguments_rejected_before_launch():
    assert _mu(count=0) == -1
    assert _mu(rows=0) == -1
    assert _mu(cols=8193) == -1
    assert _mu(hp=tfm.tfm_muon(0.02, 1.0, 0.0, 1, 5)) == -1
    assert _mu(hp=tfm.tfm_muon(0.02, 0.9, 0.0, 1, 0)) == -1
    assert _mu(hp=tfm.tfm_muon(0.02, 0.9, -0.1, 1, 5)) == -1
    assert _mu(ptr=0) == -5
    assert _mu(ptr=(1 << 20) + 2) == -5
    assert _mu(wb=16) == -7
    w1 = tfm.muon_workspace_bytes(8, 256, 256)
    assert w1 >= 8 * 256 * 256 * 4 * 4
    assert tfm.muon_workspace_bytes(16, 256, 256) > w1
    assert tfm.muon_workspace_bytes(1, 768, 256) == tfm.muon_workspace_bytes(1, 256, 768)
    assert tfm.muon_workspace_bytes(0, 8, 8) == 0


def test_noalloc_forward_limits_rejected_before_launch():
    """The allocation-free forward takes the bf16 matrix-core dims only, and rejects dims whose
    scratch (the plan and the bf16 weights) exceeds the library's fixed array, before any HIP
    call."""
    p = 1 << 20
    d = _dims()                                                   # float32: not supported
    rc = tfm.lib().tfm_layer_fwd_noalloc(ctypes.byref(d), None, None, p, p, p, p, 1 << 40, None)
    assert rc == -1 and "TFM_BF16" in tfm.last_error()
    # 10,000 datasets of 256 cells per row: ~61 MB of per-column plan alone
    d = _dims(B=10000, R=1, C=255, E=64, heads=2, H=128, dtype="bf16")
    rc = tfm.lib().tfm_layer_fwd_noalloc(ctypes.byref(d), None, None, p, p, p, p, 1 << 40, None)
    assert rc == -7 and "TFM_NOALLOC_SCRATCH_BYTES" in tfm.last_error()
    d = _dims(dtype="bf16")
    rc = tfm.lib().tfm_layer_fwd_noalloc(ctypes.byref(d), None, None, p, p, p, 0, 1 << 40, None)
    assert rc == -5
