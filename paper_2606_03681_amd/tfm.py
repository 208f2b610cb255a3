"""Thin ctypes binding of libtfmlayer.so (C ABI in include/tfm_layer.h, include/tfm_ends.h and
include/tfm_optim.h).

Argument marshalling only: every step of the layer runs in the library's HIP kernels.  torch
supplies device memory and the stream.  There is no fallback: if the library is missing, every
call raises.
"""

import ctypes
import os

import numpy as np

# TFM_LIB may name another build of the same library (the host-sanitizer build of build.py)
_LIB_PATH = os.environ.get("TFM_LIB") or \
    os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtfmlayer.so")
_lib = None

TFM_F32, TFM_BF16 = 0, 1
TFM_BLOCK_POSTNORM, TFM_BLOCK_PRENORM = 0, 1
ERRORS = {
    -1: "TFM_ERR_DIMS", -2: "TFM_ERR_HEAD_DIM", -3: "TFM_ERR_NTRAIN", -4: "TFM_ERR_MASK",
    -5: "TFM_ERR_POINTER", -6: "TFM_ERR_HIP", -7: "TFM_ERR_BUFFER",
}
EXPORTS = ("tfm_layer_param_count", "tfm_layer_saved_bytes", "tfm_layer_workspace_bytes",
           "tfm_layer_fwd", "tfm_layer_fwd_noalloc", "tfm_layer_bwd", "tfm_thinking_rows_fwd",
           "tfm_thinking_rows_bwd",
           "tfm_infer_workspace_bytes", "tfm_infer_cache_bytes", "tfm_layer_fwd_context",
           "tfm_layer_fwd_query", "tfm_last_error", "tfm_prof_enable", "tfm_prof_collect",
           "tfm_prof_step", "tfm_prof_item_bwd_fused_rows", "tfm_ends_param_count", "tfm_ends_workspace_bytes", "tfm_encode_fwd",
           "tfm_encode_bwd", "tfm_decode_fwd", "tfm_decode_loss", "tfm_clip_workspace_bytes",
           "tfm_clip_scale", "tfm_sfadamw_step", "tfm_muon_workspace_bytes", "tfm_muon_step")


class TfmError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{ERRORS.get(code, code)}: {msg}")
        self.code = code


class tfm_dims(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("B", "R", "C", "E", "heads", "H", "dtype",
                                               "block")] + [("decay", ctypes.c_float)]


def make_dims(B, R, C, E, heads, H, dtype, block="post", decay=1.0):
    dt = {"f32": TFM_F32, "bf16": TFM_BF16}.get(dtype, dtype)
    bk = {"post": TFM_BLOCK_POSTNORM, "pre": TFM_BLOCK_PRENORM}.get(block, block)
    return tfm_dims(int(B), int(R), int(C), int(E), int(heads), int(H), int(dt), int(bk),
                    float(decay))


class tfm_ends(ctypes.Structure):
    _fields_ = [("G", ctypes.c_int32), ("offsets", ctypes.c_int32 * 8)] + \
        [(n, ctypes.c_int32) for n in ("F", "T", "Hd", "K", "decode_mean")]


def make_ends(G, offsets, F, T, Hd, K, decode_mean):
    offs = list(offsets)
    if len(offs) != G or G > 8:
        raise ValueError(f"need G = {G} <= 8 offsets, got {offs}")
    arr = (ctypes.c_int32 * 8)(*(offs + [0] * (8 - len(offs))))
    return tfm_ends(int(G), arr, int(F), int(T), int(Hd), int(K), int(bool(decode_mean)))


class tfm_sfadamw(ctypes.Structure):
    _fields_ = [(n, ctypes.c_float) for n in ("lr", "beta1", "beta2", "eps", "weight_decay")] + \
        [("warmup", ctypes.c_int32)]


class tfm_muon(ctypes.Structure):
    _fields_ = [(n, ctypes.c_float) for n in ("lr", "momentum", "weight_decay")] + \
        [("nesterov", ctypes.c_int32), ("ns_steps", ctypes.c_int32)]


def lib():
    """Loads the library (once).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with "
                               "python paper_2606_03681_amd/build.py")
        L = ctypes.CDLL(_LIB_PATH)
        P = ctypes.POINTER
        vp, sz, i32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int
        for name in ("tfm_layer_param_count", "tfm_layer_saved_bytes",
                     "tfm_layer_workspace_bytes", "tfm_infer_workspace_bytes",
                     "tfm_infer_cache_bytes"):
            getattr(L, name).restype = sz
            getattr(L, name).argtypes = [P(tfm_dims)]
        L.tfm_last_error.restype = ctypes.c_char_p
        L.tfm_last_error.argtypes = []
        L.tfm_layer_fwd.restype = i32
        L.tfm_layer_fwd.argtypes = [P(tfm_dims), vp, vp, vp, vp, vp, vp, sz, vp, sz, vp]
        L.tfm_layer_fwd_noalloc.restype = i32
        L.tfm_layer_fwd_noalloc.argtypes = [P(tfm_dims), vp, vp, vp, vp, vp, vp, sz, vp]
        L.tfm_layer_bwd.restype = i32
        L.tfm_layer_bwd.argtypes = [P(tfm_dims), vp, vp, vp, vp, vp, sz, vp, vp, vp, i32, vp,
                                    sz, vp]
        L.tfm_thinking_rows_fwd.restype = i32
        L.tfm_thinking_rows_fwd.argtypes = [P(tfm_dims), vp, vp, i32, vp, vp, vp, sz, vp]
        L.tfm_thinking_rows_bwd.restype = i32
        L.tfm_thinking_rows_bwd.argtypes = [P(tfm_dims), vp, vp, i32, vp, vp, i32, vp, sz, vp]
        L.tfm_layer_fwd_context.restype = i32
        L.tfm_layer_fwd_context.argtypes = [P(tfm_dims), vp, vp, vp, vp, vp, vp, sz, vp, sz, vp]
        L.tfm_layer_fwd_query.restype = i32
        L.tfm_layer_fwd_query.argtypes = [P(tfm_dims), i32, vp, vp, vp, vp, vp, sz, vp, vp, sz,
                                          vp]
        E_ = P(tfm_ends)
        for name in ("tfm_ends_param_count", "tfm_ends_workspace_bytes"):
            getattr(L, name).restype = sz
            getattr(L, name).argtypes = [P(tfm_dims), E_]
        L.tfm_encode_fwd.restype = i32
        L.tfm_encode_fwd.argtypes = [P(tfm_dims), E_, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.tfm_encode_bwd.restype = i32
        L.tfm_encode_bwd.argtypes = [P(tfm_dims), E_, vp, vp, vp, vp, vp, vp, i32, vp, sz, vp]
        L.tfm_decode_fwd.restype = i32
        L.tfm_decode_fwd.argtypes = [P(tfm_dims), E_, vp, vp, vp, vp, vp, vp, sz, vp]
        L.tfm_decode_loss.restype = i32
        L.tfm_decode_loss.argtypes = [P(tfm_dims), E_, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                      i32, vp, sz, vp]
        i64, f32 = ctypes.c_int64, ctypes.c_float
        L.tfm_clip_workspace_bytes.restype = sz
        L.tfm_clip_workspace_bytes.argtypes = [i32, P(i64)]
        L.tfm_clip_scale.restype = i32
        L.tfm_clip_scale.argtypes = [i32, P(vp), P(i64), f32, vp, vp, vp, sz, vp]
        L.tfm_sfadamw_step.restype = i32
        L.tfm_sfadamw_step.argtypes = [P(tfm_sfadamw), i64, i32, P(i64), P(i64), vp, vp, vp, vp,
                                       vp, vp]
        L.tfm_muon_workspace_bytes.restype = sz
        L.tfm_muon_workspace_bytes.argtypes = [i32, i32, i32]
        L.tfm_muon_step.restype = i32
        L.tfm_muon_step.argtypes = [P(tfm_muon), i32, i32, i32, P(vp), P(vp), P(vp), vp, vp, sz,
                                    vp]
        L.tfm_prof_enable.restype = i32
        L.tfm_prof_enable.argtypes = [i32]
        L.tfm_prof_collect.restype = i32
        L.tfm_prof_collect.argtypes = []
        L.tfm_prof_step.restype = i32
        L.tfm_prof_step.argtypes = [i32, P(ctypes.c_char_p), P(ctypes.c_longlong),
                                    P(ctypes.c_double)]
        L.tfm_prof_item_bwd_fused_rows.restype = i32
        L.tfm_prof_item_bwd_fused_rows.argtypes = [i32]
        _lib = L
    return _lib


def last_error():
    return lib().tfm_last_error().decode()


def param_count(dims):
    return lib().tfm_layer_param_count(ctypes.byref(dims))


def saved_bytes(dims):
    return lib().tfm_layer_saved_bytes(ctypes.byref(dims))


def workspace_bytes(dims):
    return lib().tfm_layer_workspace_bytes(ctypes.byref(dims))


def infer_workspace_bytes(dims):
    return lib().tfm_infer_workspace_bytes(ctypes.byref(dims))


def infer_cache_bytes(dims):
    return lib().tfm_infer_cache_bytes(ctypes.byref(dims))


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _host(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data


def _check(rc):
    if rc != 0:
        raise TfmError(rc, last_error())


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return stream if isinstance(stream, int) else stream.cuda_stream


def layer_fwd(dims, n_train, cell_mask, X, params, Y, saved, workspace, stream=None):
    """tfm_layer_fwd.  n_train: host int32 [B]; cell_mask: host uint8 [B, C+1]; X, Y: device
    tensors [B, R, C+1, E] (float32 or bfloat16); params: device float32; saved, workspace:
    device byte tensors of saved_bytes(dims) / workspace_bytes(dims)."""
    nt, ntp = _host(n_train, np.int32)
    cm, cmp_ = _host(cell_mask, np.uint8)
    rc = lib().tfm_layer_fwd(ctypes.byref(dims), ntp, cmp_, _ptr(X), _ptr(params), _ptr(Y),
                             _ptr(saved), saved.numel() * saved.element_size(),
                             _ptr(workspace), workspace.numel() * workspace.element_size(),
                             _stream(stream))
    _check(rc)


def layer_fwd_noalloc(dims, n_train, cell_mask, X, params, Y, saved, stream=None):
    """tfm_layer_fwd_noalloc: tfm_layer_fwd with its scratch in the library's own device array
    (no workspace argument; calls on one GPU must not overlap)."""
    nt, ntp = _host(n_train, np.int32)
    cm, cmp_ = _host(cell_mask, np.uint8)
    rc = lib().tfm_layer_fwd_noalloc(ctypes.byref(dims), ntp, cmp_, _ptr(X), _ptr(params),
                                     _ptr(Y), _ptr(saved), saved.numel() * saved.element_size(),
                                     _stream(stream))
    _check(rc)


def layer_bwd(dims, n_train, cell_mask, X, params, saved, dY, dX, grads, accumulate, workspace,
              stream=None):
    """tfm_layer_bwd; grads: device float32 like params, overwritten or accumulated."""
    nt, ntp = _host(n_train, np.int32)
    cm, cmp_ = _host(cell_mask, np.uint8)
    rc = lib().tfm_layer_bwd(ctypes.byref(dims), ntp, cmp_, _ptr(X), _ptr(params), _ptr(saved),
                             saved.numel() * saved.element_size(), _ptr(dY), _ptr(dX),
                             _ptr(grads), int(bool(accumulate)), _ptr(workspace),
                             workspace.numel() * workspace.element_size(), _stream(stream))
    _check(rc)


def thinking_rows_fwd(dims, n_train, cell_mask, T, table, X, workspace, stream=None):
    """tfm_thinking_rows_fwd: writes table (device float32 [T, E]) into rows [0, T) of X
    (device [B, R, C+1, E]) at active columns, 0 at inactive ones."""
    nt, ntp = _host(n_train, np.int32)
    cm, cmp_ = _host(cell_mask, np.uint8)
    rc = lib().tfm_thinking_rows_fwd(ctypes.byref(dims), ntp, cmp_, int(T), _ptr(table), _ptr(X),
                                     _ptr(workspace),
                                     workspace.numel() * workspace.element_size(),
                                     _stream(stream))
    _check(rc)


def thinking_rows_bwd(dims, n_train, cell_mask, T, dX, dtable, accumulate, workspace,
                      stream=None):
    """tfm_thinking_rows_bwd: dtable (device float32 [T, E]) gets (or adds) the sum of dX rows
    [0, T) over datasets and active columns."""
    nt, ntp = _host(n_train, np.int32)
    cm, cmp_ = _host(cell_mask, np.uint8)
    rc = lib().tfm_thinking_rows_bwd(ctypes.byref(dims), ntp, cmp_, int(T), _ptr(dX),
                                     _ptr(dtable), int(bool(accumulate)), _ptr(workspace),
                                     workspace.numel() * workspace.element_size(),
                                     _stream(stream))
    _check(rc)


def _nbytes(t):
    return t.numel() * t.element_size()


def layer_fwd_context(dims, n_train, cell_mask, X, params, Y, kv_cache, workspace, stream=None):
    """tfm_layer_fwd_context: forward without saved state; the train rows' item-axis keys and
    values go to kv_cache (a device byte tensor of infer_cache_bytes(dims))."""
    nt, ntp = _host(n_train, np.int32)
    cm, cmp_ = _host(cell_mask, np.uint8)
    rc = lib().tfm_layer_fwd_context(ctypes.byref(dims), ntp, cmp_, _ptr(X), _ptr(params),
                                     _ptr(Y), _ptr(kv_cache), _nbytes(kv_cache), _ptr(workspace),
                                     _nbytes(workspace), _stream(stream))
    _check(rc)


def layer_fwd_query(dims, context_rows, n_train, cell_mask, X, params, kv_cache, Y, workspace,
                    stream=None):
    """tfm_layer_fwd_query: forward of unlabelled rows X [B, Rq, C+1, E] against the keys and
    values a context call with context_rows rows left in kv_cache."""
    nt, ntp = _host(n_train, np.int32)
    cm, cmp_ = _host(cell_mask, np.uint8)
    rc = lib().tfm_layer_fwd_query(ctypes.byref(dims), int(context_rows), ntp, cmp_, _ptr(X),
                                   _ptr(params), _ptr(kv_cache), _nbytes(kv_cache), _ptr(Y),
                                   _ptr(workspace), _nbytes(workspace), _stream(stream))
    _check(rc)


def ends_param_count(dims, ends):
    return lib().tfm_ends_param_count(ctypes.byref(dims), ctypes.byref(ends))


def ends_workspace_bytes(dims, ends):
    return lib().tfm_ends_workspace_bytes(ctypes.byref(dims), ctypes.byref(ends))


def encode_fwd(dims, ends, n_train, n_feat, x, labels, params, X, workspace, stream=None):
    """tfm_encode_fwd.  n_train, n_feat: host int32 [B]; x: device float32 [B, R-T, F];
    labels: device int32 [B, R-T]; params: device float32 packed ends vector; X: device
    [B, R, C+1, E] (rows [T, R) written)."""
    nt, ntp = _host(n_train, np.int32)
    nf, nfp = _host(n_feat, np.int32)
    rc = lib().tfm_encode_fwd(ctypes.byref(dims), ctypes.byref(ends), ntp, nfp, _ptr(x),
                              _ptr(labels), _ptr(params), _ptr(X), _ptr(workspace),
                              _nbytes(workspace), _stream(stream))
    _check(rc)


def encode_bwd(dims, ends, n_train, n_feat, x, labels, dX, grads, accumulate, workspace,
               stream=None):
    """tfm_encode_bwd: the encoder entries of grads from dX (device [B, R, C+1, E])."""
    nt, ntp = _host(n_train, np.int32)
    nf, nfp = _host(n_feat, np.int32)
    rc = lib().tfm_encode_bwd(ctypes.byref(dims), ctypes.byref(ends), ntp, nfp, _ptr(x),
                              _ptr(labels), _ptr(dX), _ptr(grads), int(bool(accumulate)),
                              _ptr(workspace), _nbytes(workspace), _stream(stream))
    _check(rc)


def decode_fwd(dims, ends, n_train, n_feat, Y, params, logits, workspace, stream=None):
    """tfm_decode_fwd: logits (device float32 [T_test, K]) of the unlabelled rows of Y."""
    nt, ntp = _host(n_train, np.int32)
    nf, nfp = _host(n_feat, np.int32)
    rc = lib().tfm_decode_fwd(ctypes.byref(dims), ctypes.byref(ends), ntp, nfp, _ptr(Y),
                              _ptr(params), _ptr(logits), _ptr(workspace), _nbytes(workspace),
                              _stream(stream))
    _check(rc)


def decode_loss(dims, ends, n_train, n_feat, n_class, labels, Y, params, loss, logits, dY, grads,
                accumulate, workspace, stream=None):
    """tfm_decode_loss: loss (device float32 [1]), logits (device float32 [T_test, K] or None),
    dY (device like Y) and the decoder entries of grads."""
    nt, ntp = _host(n_train, np.int32)
    nf, nfp = _host(n_feat, np.int32)
    nc, ncp = _host(n_class, np.int32)
    rc = lib().tfm_decode_loss(ctypes.byref(dims), ctypes.byref(ends), ntp, nfp, ncp,
                               _ptr(labels), _ptr(Y), _ptr(params), _ptr(loss), _ptr(logits),
                               _ptr(dY), _ptr(grads), int(bool(accumulate)), _ptr(workspace),
                               _nbytes(workspace), _stream(stream))
    _check(rc)


def _ptr_array(ptrs):
    return (ctypes.c_void_p * len(ptrs))(*[int(p) for p in ptrs])


def _i64_array(vals):
    return (ctypes.c_int64 * len(vals))(*[int(v) for v in vals])


def clip_workspace_bytes(counts):
    return lib().tfm_clip_workspace_bytes(len(counts), _i64_array(counts))


def clip_scale(grads, max_norm, scale, norm, workspace, stream=None):
    """tfm_clip_scale over device float32 tensors (or (pointer, count) pairs): writes the clip
    factor to scale[0] and the global norm to norm[0] (norm may be None)."""
    ptrs = [g[0] if isinstance(g, tuple) else g.data_ptr() for g in grads]
    counts = [g[1] if isinstance(g, tuple) else g.numel() for g in grads]
    rc = lib().tfm_clip_scale(len(ptrs), _ptr_array(ptrs), _i64_array(counts), float(max_norm),
                              _ptr(scale), _ptr(norm), _ptr(workspace), _nbytes(workspace),
                              _stream(stream))
    _check(rc)


def sfadamw_step(hp, t, segments, y, z, v, grad, grad_scale=None, stream=None):
    """tfm_sfadamw_step; segments: list of (offset, length) into the float32 vectors."""
    offs = [o for o, _ in segments]
    lens = [n for _, n in segments]
    rc = lib().tfm_sfadamw_step(ctypes.byref(hp), int(t), len(segments), _i64_array(offs),
                                _i64_array(lens), _ptr(y), _ptr(z), _ptr(v), _ptr(grad),
                                _ptr(grad_scale), _stream(stream))
    _check(rc)


def muon_workspace_bytes(count, rows, cols):
    return lib().tfm_muon_workspace_bytes(int(count), int(rows), int(cols))


def muon_step(hp, rows, cols, W, G, buf, grad_scale, workspace, stream=None):
    """tfm_muon_step on len(W) matrices of rows x cols; W, G, buf: lists of device pointers (or
    tensors) of the same length."""
    conv = [[p if isinstance(p, int) else p.data_ptr() for p in lst] for lst in (W, G, buf)]
    rc = lib().tfm_muon_step(ctypes.byref(hp), len(conv[0]), int(rows), int(cols),
                             _ptr_array(conv[0]), _ptr_array(conv[1]), _ptr_array(conv[2]),
                             _ptr(grad_scale), _ptr(workspace), _nbytes(workspace),
                             _stream(stream))
    _check(rc)


def prof_enable(on=True):
    """Turns per-step HIP-event timing of the library's launches on or off (tfm_prof.h)."""
    _check(lib().tfm_prof_enable(int(bool(on))))


def prof_item_bwd_fused_rows(head_dim):
    """Longest train prefix whose item-attention backward runs as the one-kernel step
    "item_attn_bwd" at this head dimension (0: never); see tfm_prof.h."""
    return int(lib().tfm_prof_item_bwd_fused_rows(int(head_dim)))


def prof_collect():
    """Waits for the recorded events; returns {step: (launches, total_ms)}."""
    n = lib().tfm_prof_collect()
    if n < 0:
        raise TfmError(n, "profiling events could not be read")
    out = {}
    for i in range(n):
        name = ctypes.c_char_p()
        cnt = ctypes.c_longlong()
        ms = ctypes.c_double()
        lib().tfm_prof_step(i, ctypes.byref(name), ctypes.byref(cnt), ctypes.byref(ms))
        out[name.value.decode()] = (cnt.value, ms.value)
    return out
