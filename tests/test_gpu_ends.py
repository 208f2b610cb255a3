"""GPU parity of the stack's two ends (include/tfm_ends.h) against the float64 oracle of
oracle/ends.py: the encoders, the decoder with the loss, a whole training step through
encoders, stack and decoder on small shapes, and the ends of the full-size workloads in the
benchmark's launch configuration.  Tolerance: normwise-max relative error <= 1e-4 (float32
storage) and <= 2e-2 (bfloat16 storage) per tensor, and the same relative bound on the loss."""

import sys

import numpy as np
import pytest

import oracle
from oracle import ends as oe
from paper_2606_03681_amd import workloads as wl
from paper_2606_03681_amd.stack import to_device

from _harness import (TOL, nerr, ends_setup as _setup, ends_dims as _dims,
                      ends_struct as _ends, to_dev as _dev, ends_oracle_params as _oparams,
                      full_labels as _full_labels, oracle_encode as _oracle_encode,
                      oracle_train_step as _oracle_step, gpu_train_step as _gpu_step)

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    from paper_2606_03681_amd import tfm
    tfm.lib()


def _storage(t, dtype):
    import torch
    if dtype == "f32":
        return t.detach().cpu().numpy()
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def _ws(dims, en):
    import torch
    from paper_2606_03681_amd import tfm
    return torch.empty(tfm.ends_workspace_bytes(dims, en), dtype=torch.uint8, device="cuda")


def _elt(w):
    import torch
    return torch.float32 if w.dtype == "f32" else torch.bfloat16


ENC_CASES = [("ragged-small-f32", 0, 1), ("ragged-small-f32", 3, 5),
             ("ragged-small-bf16", 0, 3), ("prenorm-small-bf16", 7, 5), ("d64-f32", 2, 8)]


@pytest.mark.parametrize("name,T,G", ENC_CASES)
def test_encode_fwd_against_oracle(name, T, G):
    import torch
    from paper_2606_03681_amd import tfm
    w, e = _setup(name, T=T, G=G)
    dt, R, C = w.dtype, w.cfg["R"], w.cfg["C"]
    dims, en = _dims(w), _ends(e)
    X = torch.full((len(w.n_train), R, C + 1, w.cfg["E"]), 3.0, dtype=_elt(w), device="cuda")
    tfm.encode_fwd(dims, en, w.n_train, e.n_feat, _dev(e.x), _dev(e.labels), _dev(e.params), X,
                   _ws(dims, en))
    got = wl.storage_to_f64(_storage(X, dt), dt)
    ref, mask, _ = _oracle_encode(w, e)
    err = nerr(got[:, T:], ref)
    _say(f"[ends] encode_fwd {name} T={T} G={G}: err {err:.3g}")
    assert err <= TOL[dt]
    assert np.all(got[:, :T] == 3.0)                     # thinking rows untouched
    for b in range(len(w.n_train)):
        assert np.all(got[b, T:, ~mask[b].astype(bool)] == 0)
    assert np.array_equal(mask, e.cell_mask.astype(bool))


@pytest.mark.parametrize("name,T,G", ENC_CASES)
def test_encode_bwd_against_oracle(name, T, G):
    import torch
    from paper_2606_03681_amd import tfm
    w, e = _setup(name, T=T, G=G)
    dt, R, C, E = w.dtype, w.cfg["R"], w.cfg["C"], w.cfg["E"]
    dims, en = _dims(w), _ends(e)
    rng = np.random.default_rng(77)
    dX = wl.to_storage(rng.normal(size=(len(w.n_train), R, C + 1, E)), dt)
    grads = torch.full((len(e.params),), 7.0, device="cuda")
    ws = _ws(dims, en)
    args = (dims, en, w.n_train, e.n_feat, _dev(e.x), _dev(e.labels), _dev(dX))
    tfm.encode_bwd(*args, grads, False, ws)
    _, _, cache = _oracle_encode(w, e)
    ref = oe.encode_backward(wl.storage_to_f64(dX, dt)[:, T:], cache)
    g = grads.double().cpu().numpy()
    got = oe.unpack_ends_params(g, E, e.G, e.Hd, e.K)
    for k in ("W_fe", "b_fe", "W_te", "b_te"):
        err = nerr(got[k], ref[k])
        _say(f"[ends] encode_bwd {name} T={T} G={G} {k}: err {err:.3g}")
        assert err <= TOL[dt], k
    nenc = E * e.G + 3 * E
    assert np.all(g[nenc:] == 7.0)                       # decoder entries untouched
    tfm.encode_bwd(*args, grads, True, ws)
    torch.cuda.synchronize()
    assert np.array_equal(grads.double().cpu().numpy()[:nenc], 2 * g[:nenc])


DEC_CASES = [("ragged-small-f32", 0, False), ("ragged-small-f32", 3, True),
             ("ragged-small-bf16", 0, False), ("ragged-small-bf16", 0, True),
             ("prenorm-small-bf16", 5, True), ("d64-f32", 0, True)]


def _decode_gpu(w, e, Y, accumulate=False, logits=True):
    import torch
    from paper_2606_03681_amd import tfm
    dims, en = _dims(w), _ends(e)
    ntest = int((w.cfg["R"] - w.n_train).sum())
    loss = torch.full((4,), -1.0, device="cuda")
    lg = torch.empty((max(ntest, 1), e.K), device="cuda") if logits else None
    dY = torch.full(Y.shape, 5.0, dtype=Y.dtype, device="cuda")
    grads = torch.full((len(e.params),), 7.0, device="cuda")
    tfm.decode_loss(dims, en, w.n_train, e.n_feat, e.n_class, _dev(e.labels), Y, _dev(e.params),
                    loss, lg, dY, grads, accumulate, _ws(dims, en))
    torch.cuda.synchronize()
    return (float(loss[0].item()), None if lg is None else lg[:ntest].double().cpu().numpy(),
            dY, grads.double().cpu().numpy())


@pytest.mark.parametrize("name,T,mean", DEC_CASES)
def test_decode_loss_against_oracle(name, T, mean):
    w, e = _setup(name, T=T, mean=mean)
    if len(w.n_train) >= 3:
        # one dataset without unlabelled rows, one with a single class
        w.n_train[0] = w.cfg["R"]
        e.n_class[1] = 1
        e.labels[1] = 0
    dt, R, C, E = w.dtype, w.cfg["R"], w.cfg["C"], w.cfg["E"]
    Ys = wl.to_storage(np.random.default_rng(5).normal(size=(len(w.n_train), R, C + 1, E)), dt)
    loss, lg, dY, g = _decode_gpu(w, e, to_device(Ys, dt))
    P = _oparams(w, e)
    mode = "mean" if e.mean else "target"
    rl, rdY, rdP, rlg = oe.decode_loss(wl.storage_to_f64(Ys, dt), _full_labels(w, e), w.n_train,
                                       e.n_feat, e.n_class, C, P, mode)
    tol = TOL[dt]
    _say(f"[ends] decode {name} T={T} mean={mean}: loss {loss:.6g} vs {rl:.6g}")
    assert abs(loss - rl) <= tol * abs(rl)
    assert nerr(lg, rlg) <= tol
    assert nerr(wl.storage_to_f64(_storage(dY, dt), dt), rdY) <= tol
    got = oe.unpack_ends_params(g, E, e.G, e.Hd, e.K)
    for k in ("W_d1", "b_d1", "W_d2", "b_d2"):
        err = nerr(got[k], rdP[k])
        _say(f"[ends] decode {name} {k}: err {err:.3g}")
        assert err <= tol, k
    assert np.all(g[:E * e.G + 3 * E] == 7.0)            # encoder entries untouched


def test_decode_without_unlabelled_rows_gives_zeros():
    import torch
    w, e = _setup("ragged-small-f32", n_train=[200, 200, 200, 200])
    Y = torch.randn((4, 200, 21, 64), device="cuda")
    loss, _, dY, g = _decode_gpu(w, e, Y, logits=False)
    assert loss == 0.0
    assert torch.count_nonzero(dY).item() == 0
    E = 64
    assert np.all(g[E * e.G + 3 * E:] == 0) and np.all(g[:E * e.G + 3 * E] == 7.0)


def test_decode_fwd_matches_the_loss_call_logits():
    import torch
    from paper_2606_03681_amd import tfm
    w, e = _setup("ragged-small-bf16", mean=True)
    Ys = wl.to_storage(np.random.default_rng(9).normal(
        size=(len(w.n_train), w.cfg["R"], w.cfg["C"] + 1, w.cfg["E"])), "bf16")
    Y = to_device(Ys, "bf16")
    _, lg, _, _ = _decode_gpu(w, e, Y)
    dims, en = _dims(w), _ends(e)
    out = torch.empty((lg.shape[0], e.K), device="cuda")
    tfm.decode_fwd(dims, en, w.n_train, e.n_feat, Y, _dev(e.params), out, _ws(dims, en))
    torch.cuda.synchronize()
    assert np.array_equal(out.double().cpu().numpy(), lg)


def test_ends_bitwise_deterministic():
    w, e = _setup("ragged-small-bf16", mean=True)
    import torch
    Ys = wl.to_storage(np.random.default_rng(3).normal(
        size=(len(w.n_train), w.cfg["R"], w.cfg["C"] + 1, w.cfg["E"])), "bf16")
    a = _decode_gpu(w, e, to_device(Ys, "bf16"))
    b = _decode_gpu(w, e, to_device(Ys, "bf16"))
    assert a[0] == b[0] and np.array_equal(a[3], b[3])
    assert torch.equal(a[2], b[2])


# ---- a whole training step ---------------------------------------------------------------------

STEP_CASES = [("d64-f32", 0, None), ("ragged-small-f32", 2, None), ("d16-bf16", 0, None),
              ("prenorm-small-bf16", 4, None), ("prenorm-d64-bf16", 6, None)]


@pytest.mark.parametrize("name,T,G", STEP_CASES)
def test_training_step_against_oracle(name, T, G):
    w, e = _setup(name, T=T, G=G)
    dt = w.dtype
    tol = TOL[dt]
    ts, loss = _gpu_step(w, e)
    rl, rgrads, rdP, rdt = _oracle_step(w, e)
    _say(f"[step] {name} T={T}: loss {loss:.6g} vs {rl:.6g}")
    assert abs(loss - rl) <= tol * abs(rl)
    unpack = oracle.unpack_prenorm_params if w.block == "pre" else oracle.unpack_params
    names = oracle.PRENORM_PARAM_ORDER if w.block == "pre" else oracle.PARAM_ORDER
    E, H = w.cfg["E"], w.cfg["H"]
    worst = 0.0
    for l, (gg, gr) in enumerate(zip(ts.stack.grads, rgrads)):
        pg = unpack(gg.double().cpu().numpy(), E, H)
        pr = unpack(gr, E, H)
        for k in names:
            err = nerr(pg[k], pr[k])
            worst = max(worst, err)
            assert err <= tol, (l, k, err)
    got = oe.unpack_ends_params(ts.ends_grads.double().cpu().numpy(), E, e.G, e.Hd, e.K)
    for k in oe.ENDS_PARAM_ORDER:
        err = nerr(got[k], rdP[k])
        worst = max(worst, err)
        assert err <= tol, (k, err)
    if T:
        err = nerr(ts.table_grad.double().cpu().numpy(), rdt)
        worst = max(worst, err)
        assert err <= tol
    _say(f"[step] {name} T={T}: worst gradient error {worst:.3g}")


# ---- full-size workloads in the benchmark's launch configuration ------------------------------

@pytest.mark.parametrize("cfg", [2, "record9-bf16"])
def test_full_size_ends(cfg):
    """The whole step at full size; the encoders are checked against the oracle on the data the
    GPU step used (x, labels and the stack's dX as stored), the decoder on the stack output the
    GPU produced (as stored)."""
    w, e = _setup(cfg)
    dt, C, E, T = w.dtype, w.cfg["C"], w.cfg["E"], e.T
    tol = TOL[dt]
    _say(f"[ends-full] {w.cfg['name']}: GPU step")
    ts, loss = _gpu_step(w, e)
    P = _oparams(w, e)
    # encoder output, two datasets
    for b in (0, len(w.n_train) - 1):
        ref, _, _ = _oracle_encode(w, e, b)
        got = wl.storage_to_f64(_storage(ts.X[b, T:], dt), dt)
        err = nerr(got, ref[0])
        _say(f"[ends-full] encode_fwd dataset {b}: err {err:.3g}")
        assert err <= tol
    # decoder on the GPU's Y: per-dataset oracle calls combined with the global row weights
    ntest = w.cfg["R"] - w.n_train
    Ttot = float(ntest.sum())
    mode = "mean" if e.mean else "target"
    rl = 0.0
    rdP = {k: 0.0 for k in ("W_d1", "b_d1", "W_d2", "b_d2")}
    worst_dy = 0.0
    y = _full_labels(w, e)
    for b in range(len(w.n_train)):
        Yb = wl.storage_to_f64(_storage(ts.Y[b:b + 1], dt), dt)
        lb, dYb, dPb, _ = oe.decode_loss(Yb, y[b:b + 1], w.n_train[b:b + 1], e.n_feat[b:b + 1],
                                         e.n_class[b:b + 1], C, P, mode)
        s = ntest[b] / Ttot
        rl += lb * s
        for k in rdP:
            rdP[k] = rdP[k] + dPb[k] * s
        gdY = wl.storage_to_f64(_storage(ts.dY[b], dt), dt)
        worst_dy = max(worst_dy, nerr(gdY, dYb[0] * s))
    _say(f"[ends-full] loss {loss:.6g} vs {rl:.6g}; dY err {worst_dy:.3g}")
    assert abs(loss - rl) <= tol * abs(rl)
    assert worst_dy <= tol
    got = oe.unpack_ends_params(ts.ends_grads.double().cpu().numpy(), E, e.G, e.Hd, e.K)
    for k in rdP:
        err = nerr(got[k], rdP[k])
        _say(f"[ends-full] decoder {k}: err {err:.3g}")
        assert err <= tol, k
    # encoder gradients from the GPU's dX
    ref = {k: 0.0 for k in ("W_fe", "b_fe", "W_te", "b_te")}
    for b in range(len(w.n_train)):
        _, _, cache = _oracle_encode(w, e, b)
        dXb = wl.storage_to_f64(_storage(ts.dX[b:b + 1, T:], dt), dt)
        d = oe.encode_backward(dXb, cache)
        for k in ref:
            ref[k] = ref[k] + d[k]
    for k in ref:
        err = nerr(got[k], ref[k])
        _say(f"[ends-full] encoder {k}: err {err:.3g}")
        assert err <= tol, k


# ---- the optimiser step inside the training step -----------------------------------------------

OPT_CASES = [("d64-f32", 0), ("ragged-small-f32", 2), ("prenorm-small-bf16", 4)]


@pytest.mark.parametrize("name,T", OPT_CASES)
def test_training_step_optimizer_against_oracle(name, T):
    """Two training steps with the optimiser of Tab. 5 (baseline settings for the post-norm
    block, the record's Muon + schedule-free AdamW for the pre-norm one).  The oracle's clip,
    Muon and schedule-free AdamW, fed the gradients the GPU step produced, must give the same
    parameter changes: this checks which parameters go to which optimiser, the clip over every
    gradient, and the state carried from step to step."""
    import torch
    from oracle import optim
    from paper_2606_03681_amd.stack import (OPTIM_BASELINE, OPTIM_RECORD, Optimizer, TrainStep,
                                            muon_matrices)
    w, e = _setup(name, T=T)
    pre = w.block == "pre"
    st = OPTIM_RECORD if pre else OPTIM_BASELINE
    ts = TrainStep(_dims(w), _ends(e), w.n_train, e.n_feat, e.n_class, w.params, e.params,
                   e.table)
    opt = Optimizer(ts, st)
    x, lab = _dev(e.x), _dev(e.labels)
    E, H = w.cfg["E"], w.cfg["H"]
    mats = muon_matrices(E, H, w.block) if st["muon"] else []
    L = len(ts.stack.params)
    host = lambda: [v[0].double().cpu().numpy().copy() for v in opt.vectors]  # noqa: E731
    y0 = host()
    sf = [optim.ScheduleFreeAdamW(y[np.concatenate([np.arange(o, o + n) for o, n in v[4]])],
                                  st["lr"], weight_decay=st["adamw_wd"])
          for y, v in zip(y0, opt.vectors)]
    mbuf = {}
    for step in range(2):
        before = host()
        ts.run(x, lab)
        torch.cuda.synchronize()
        grads = [v[1].double().cpu().numpy().copy() for v in opt.vectors]
        opt.step()
        torch.cuda.synchronize()
        after = host()
        _, scale = optim.clip_scale(grads, st["clip"])
        for i, (v, b, a, g) in enumerate(zip(opt.vectors, before, after, grads)):
            ref = b.copy()
            idx = np.concatenate([np.arange(o, o + n) for o, n in v[4]])
            ref[idx] = sf[i].step(scale * g[idx])
            if i < L:
                for (o, r, c) in mats:
                    sl = slice(o, o + r * c)
                    Wn, mbuf[(i, o)] = optim.muon_step(
                        b[sl].reshape(1, r, c), scale * g[sl].reshape(1, r, c),
                        mbuf.get((i, o), np.zeros((1, r, c))), st["lr"] * st["muon_lr_ratio"],
                        st["muon_momentum"], st["muon_wd"])
                    ref[sl] = Wn.ravel()
            err = nerr(a - b, ref - b)
            # the float32 bar, plus the rounding of the stored float32 parameters: half an ulp
            # of the new value on the GPU, and the GPU's and the oracle's step-to-step drift
            # by as much again per step (a 1e-4 step on a value of 1 resolves to 6e-4)
            tol = 1e-4 + (step + 1) * 2 * 2.0 ** -24 * np.abs(b).max() / np.abs(ref - b).max()
            _say(f"[train] {name} step {step} vector {i}: update err {err:.3g} (bound {tol:.3g})")
            assert err <= tol, (step, i, err, tol)
            assert np.abs(a - b).max() > 0


# ---- evaluation: encoders, forward-only stack and decoder -------------------------------------

@pytest.mark.parametrize("name,T,chunk,n_train", [("d16-bf16", 0, 11, None),
                                                  ("prenorm-small-bf16", 4, 64,
                                                   [150, 120, 5, 199])])
def test_infer_model_matches_the_training_forward(name, T, chunk, n_train):
    """Logits of the forward-only path (context rows once, unlabelled rows in chunks) equal,
    bit for bit, the decoder applied to the training forward's output."""
    import torch
    from paper_2606_03681_amd import tfm
    from paper_2606_03681_amd.stack import InferModel, TrainStep
    w, e = _setup(name, T=T, n_train=n_train)
    dims, en = _dims(w), _ends(e)
    x, lab = _dev(e.x), _dev(e.labels)
    ts = TrainStep(dims, en, w.n_train, e.n_feat, e.n_class, w.params, e.params, e.table)
    ts.run(x, lab)
    ntest = int((w.cfg["R"] - w.n_train).sum())
    ref = torch.empty((ntest, e.K), device="cuda")
    tfm.decode_fwd(dims, en, w.n_train, e.n_feat, ts.Y, ts.ends_params, ref, ts.ends_ws)
    im = InferModel(dims, en, w.n_train, e.n_feat, w.params, e.params, e.table, chunk=chunk)
    got = im.predict(x, lab)
    torch.cuda.synchronize()
    _say(f"[infer-model] {name}: {ntest} rows, {len(im.spans)} query chunks")
    assert got.shape == ref.shape
    assert torch.equal(got, ref)


def test_ends_at_the_envelope_limits():
    """The largest group (8 shifts), the most decoder outputs (64 classes), 255 feature cells
    and a table whose feature count is 1; encoders and decoder against the oracle."""
    import torch
    from paper_2606_03681_amd import tfm
    rng = np.random.default_rng(31)
    B, R, C, E, Hd, K, G = 2, 24, 255, 64, 48, 64, 8
    offs = (0, 1, 3, 7, 12, 20, 30, 44)
    n_train = np.array([17, 3], np.int32)
    n_feat = np.array([255, 1], np.int32)
    n_class = np.array([64, 2], np.int32)
    x = rng.normal(size=(B, R, C)).astype(np.float32)
    lab = np.stack([rng.integers(0, n_class[b], R) for b in range(B)]).astype(np.int32)
    P = rng.normal(0, 0.3, oe.ends_param_count(E, G, Hd, K)).astype(np.float32)
    dims = tfm.make_dims(B, R, C, E, 2, 128, "f32")
    en = tfm.make_ends(G, offs, C, 0, Hd, K, 1)
    ws = torch.empty(tfm.ends_workspace_bytes(dims, en), dtype=torch.uint8, device="cuda")
    X = torch.empty((B, R, C + 1, E), device="cuda")
    tfm.encode_fwd(dims, en, n_train, n_feat, _dev(x), _dev(lab), _dev(P), X, ws)
    Po = oe.unpack_ends_params(P.astype(np.float64), E, G, Hd, K)
    Xr, mask, cache = oe.encode_forward(x, lab.astype(np.float64), n_train, n_feat, C, offs, Po)
    assert nerr(X.cpu().numpy(), Xr) <= TOL["f32"]
    Y = torch.randn((B, R, C + 1, E), device="cuda")
    loss = torch.empty(4, device="cuda")
    dY = torch.empty_like(Y)
    grads = torch.zeros(P.size, device="cuda")
    lg = torch.empty((int((R - n_train).sum()), K), device="cuda")
    tfm.decode_loss(dims, en, n_train, n_feat, n_class, _dev(lab), Y, _dev(P), loss, lg, dY,
                    grads, False, ws)
    dXs = torch.randn((B, R, C + 1, E), device="cuda")
    tfm.encode_bwd(dims, en, n_train, n_feat, _dev(x), _dev(lab), dXs, grads, False, ws)
    torch.cuda.synchronize()
    Yh = Y.double().cpu().numpy()
    rl, rdY, rdP, rlg = oe.decode_loss(Yh, lab.astype(np.float64), n_train, n_feat, n_class, C,
                                       Po, "mean")
    rdP.update(oe.encode_backward(dXs.double().cpu().numpy(), cache))
    assert abs(float(loss[0].item()) - rl) <= TOL["f32"] * abs(rl)
    assert nerr(lg.double().cpu().numpy(), rlg) <= TOL["f32"]
    assert nerr(dY.double().cpu().numpy(), rdY) <= TOL["f32"]
    got = oe.unpack_ends_params(grads.double().cpu().numpy(), E, G, Hd, K)
    for k in oe.ENDS_PARAM_ORDER:
        assert nerr(got[k], rdP[k]) <= TOL["f32"], k
