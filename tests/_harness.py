"""Shared helpers of the GPU parity tests: run a workload through the C-ABI library on the GPU
and through the float64 oracle on the CPU, and compare."""

import numpy as np

import oracle
from oracle import ends as oe
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


# ---- the stack's two ends and a whole training step ---------------------------------------

def ends_setup(name, T=None, G=None, mean=None, dtype=None, n_train=None):
    """A workload (its stack parameters and train prefixes, T thinking rows if given, at least
    one labelled data row per dataset) and the inputs of its two ends."""
    w = wl.make_workload(name, with_dY=False)
    cfg = dict(w.cfg)
    if T is not None:
        cfg["thinking"] = T
    if dtype is not None:
        cfg["dtype"] = dtype
    w.cfg = cfg
    T = cfg.get("thinking", 0)
    if n_train is not None:
        w.n_train = np.asarray(n_train, np.int32)
    w.n_train = np.maximum(w.n_train, T + 1).astype(np.int32)
    e = wl.make_ends_inputs(w, G=G, mean=mean)
    return w, e


def ends_dims(w):
    from paper_2606_03681_amd import tfm
    return tfm.make_dims(dtype=w.dtype, block=w.block,
                         **{k: v for k, v in w.dims.items() if k != "dtype"})


def ends_struct(e):
    from paper_2606_03681_amd import tfm
    return tfm.make_ends(e.G, e.offsets, e.F, e.T, e.Hd, e.K, e.mean)


def to_dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def ends_oracle_params(w, e):
    return oe.unpack_ends_params(e.params.astype(np.float64), w.cfg["E"], e.G, e.Hd, e.K)


def full_labels(w, e):
    """Labels aligned with the rows of the stack input (thinking rows get 0, never read)."""
    y = np.zeros((len(w.n_train), w.cfg["R"]))
    y[:, e.T:] = e.labels
    return y


def oracle_encode(w, e, b=None):
    sl = slice(None) if b is None else slice(b, b + 1)
    return oe.encode_forward(e.x[sl], e.labels[sl].astype(np.float64),
                             (w.n_train - e.T)[sl], e.n_feat[sl], w.cfg["C"], e.offsets,
                             ends_oracle_params(w, e))


def oracle_train_step(w, e):
    """The oracle's training step: encoders (and thinking rows), the stack, the decoder and loss,
    and the backward pass.  Returns (loss, packed block gradients, ends gradients, dtable)."""
    T, C = e.T, w.cfg["C"]
    P = ends_oracle_params(w, e)
    Xd, _, cache = oracle_encode(w, e)
    X = oracle.thinking_rows_forward(Xd, e.table.astype(np.float64), e.cell_mask) if T else Xd
    Ps = oracle_params(w)
    heads = w.cfg["heads"]
    if w.block == "pre":
        Y, caches = oracle.prenorm_stack_forward(X, Ps, w.n_train, e.cell_mask, heads)
    else:
        Y, caches = oracle.stack_forward(X, Ps, w.n_train, e.cell_mask, heads)
    mode = "mean" if e.mean else "target"
    loss, dY, dP, _ = oe.decode_loss(Y, full_labels(w, e), w.n_train, e.n_feat, e.n_class, C,
                                     P, mode)
    if w.block == "pre":
        dX, grads = oracle.prenorm_stack_backward(dY, caches)
        grads = [oracle.pack_prenorm_params(g) for g in grads]
    else:
        dX, grads = oracle.stack_backward(dY, caches)
        grads = [oracle.pack_params(g) for g in grads]
    dtable = None
    if T:
        dX, dtable = oracle.thinking_rows_backward(dX, e.cell_mask, T)
    dP.update(oe.encode_backward(dX, cache))
    return loss, grads, dP, dtable


def gpu_train_step(w, e):
    """The same step on the GPU (stack.TrainStep); returns the step object and the loss."""
    import torch
    from paper_2606_03681_amd.stack import TrainStep
    ts = TrainStep(ends_dims(w), ends_struct(e), w.n_train, e.n_feat, e.n_class, w.params,
                   e.params, e.table)
    loss = ts.run(to_dev(e.x), to_dev(e.labels))
    torch.cuda.synchronize()
    return ts, float(loss.item())
