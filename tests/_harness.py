"""Shared helpers of the GPU parity tests: run a workload through the C-ABI library on the GPU
and through the float64 oracle on the CPU, and compare."""

import numpy as np

import oracle
from paper_2606_03681_amd import workloads as wl

TOL = {"f32": 1e-4, "bf16": 2e-2}


def nerr(a, b):
    """Normwise-max relative error max|a - b| / max|b|."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = np.abs(b).max()
    return float(np.abs(a - b).max() / (den if den > 0 else 1.0))


def _unpack(w):
    return oracle.unpack_prenorm_params if w.block == "pre" else oracle.unpack_params


def _param_names(w):
    return oracle.PRENORM_PARAM_ORDER if w.block == "pre" else oracle.PARAM_ORDER


def oracle_params(w):
    return [_unpack(w)(p, w.cfg["E"], w.cfg["H"]) for p in w.params64()]


def oracle_stack(w, X=None, dY=None):
    """Oracle forward + backward of the whole stack on the workload (post-norm blocks, or
    pre-norm blocks whose layer l scales its input by 0.95 ** l)."""
    X = w.X64() if X is None else X
    dY = w.dY64() if dY is None else dY
    Ps = oracle_params(w)
    if w.block == "pre":
        Y, caches = oracle.prenorm_stack_forward(X, Ps, w.n_train, w.cell_mask, w.cfg["heads"])
        dX, grads = oracle.prenorm_stack_backward(dY, caches)
        return Y, dX, [oracle.pack_prenorm_params(g) for g in grads]
    Y, caches = oracle.stack_forward(X, Ps, w.n_train, w.cell_mask, w.cfg["heads"])
    dX, grads = oracle.stack_backward(dY, caches)
    return Y, dX, [oracle.pack_params(g) for g in grads]


def storage_of(t, dtype):
    """device tensor -> host storage array (float32, or uint16 bfloat16 bits)."""
    import torch
    if dtype == "f32":
        return t.detach().cpu().numpy()
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def gpu_stack(w, X=None, dY=None, keep_acts=False, params=None, storage=False, first_layer=0):
    """GPU forward + backward of the whole stack (or of the given per-layer params).

    Returns float64 host arrays, or storage arrays (see storage_of) with storage=True."""
    import torch
    from paper_2606_03681_amd import tfm
    from paper_2606_03681_amd.stack import Stack, to_device

    dt = w.dtype
    conv = (lambda t: storage_of(t, dt)) if storage else \
        (lambda t: wl.storage_to_f64(storage_of(t, dt), dt))
    dims = tfm.make_dims(dtype=dt, block=w.block,
                         **{k: v for k, v in w.dims.items() if k != "dtype"})
    st = Stack(dims, w.n_train, w.cell_mask, w.params if params is None else params,
               first_layer=first_layer)
    Xd = to_device(w.X if X is None else X, dt)
    dYd = to_device(w.dY if dY is None else dY, dt)
    Y = st.forward(Xd)
    acts = [conv(a) for a in st.acts] if keep_acts else None
    Yh = conv(Y)
    dX = st.backward(dYd)
    torch.cuda.synchronize()
    out = dict(Y=Yh, dX=conv(dX), grads=[g.double().cpu().numpy() for g in st.grads],
               acts=acts)
    del st, Xd, dYd
    torch.cuda.empty_cache()
    return out


def compare_all(w, gpu, ref, tol=None):
    """Asserts parity of Y, dX and every parameter block of every layer; returns the worst
    error per tensor name."""
    tol = TOL[w.dtype] if tol is None else tol
    Y, dX, grads = ref
    errs = {"Y": nerr(gpu["Y"], Y), "dX": nerr(gpu["dX"], dX)}
    E, H = w.cfg["E"], w.cfg["H"]
    for l, (gg, gr) in enumerate(zip(gpu["grads"], grads)):
        pg = _unpack(w)(gg, E, H)
        pr = _unpack(w)(gr, E, H)
        for k in _param_names(w):
            errs[f"L{l}.{k}"] = nerr(pg[k], pr[k])
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, f"parity above {tol}: {bad}"
    return errs


def sample_rows(n, R, k_train=8, k_test=8, seed=0):
    rng = np.random.default_rng(seed)
    tr = np.sort(rng.choice(n, size=min(k_train, n), replace=False))
    te = np.sort(n + rng.choice(R - n, size=min(k_test, R - n), replace=False)) if R > n else \
        np.zeros(0, np.int64)
    return tr, te


def oracle_rows(Xb, mask_b, P, heads, n, rows_train, rows_test, dYq=None, block="post",
                decay=1.0):
    """Oracle on one dataset, outputs only at the sampled rows (train rows first).

    Xb: (R, S, E) float64 cell tensor of the dataset; returns Y at the sampled rows
    (len, S_b, E) and, if dYq (upstream gradient at the sampled rows) is given, dX on
    [train rows; sampled test rows] and the gradient dict."""
    act = np.flatnonzero(mask_b)
    keep = np.concatenate([np.arange(n), rows_test]).astype(np.int64)
    z = Xb[keep][:, act, :]
    q = np.concatenate([rows_train, np.arange(n, n + len(rows_test))]).astype(np.int64)
    if block == "pre":
        Y, c = oracle.prenorm_dataset_forward(z, P, heads, n, decay, query_rows=q)
    else:
        Y, c = oracle.dataset_forward(z, P, heads, n, query_rows=q)
    if dYq is None:
        return Y, None, None, act, keep
    if block == "pre":
        dz, g = oracle.prenorm_dataset_backward(dYq, c, P, heads)
    else:
        dz, g = oracle.dataset_backward(dYq, c, P, heads)
    return Y, dz, g, act, keep
