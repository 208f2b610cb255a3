"""GPU parity: the HIP path through the C ABI against the float64 oracle, element by element on
the same seeded inputs.  Tolerance: normwise-max relative error (max|gpu - ref| / max|ref| per
tensor) <= 1e-4 in float32 mode and <= 2e-2 in bfloat16 mode, on Y, dX and every parameter
gradient block of every layer.

Small shapes are compared in full.  The full-size workloads run in the benchmark's launch
configuration (whole batch, all layers) and are compared on sampled rows of sampled datasets,
layer by layer: the oracle evaluates a layer at a set of query rows from the train rows and
those rows only (exact by the isolation of test rows), and the backward check drives each layer
with an upstream gradient supported on those rows only."""

import sys

import numpy as np
import pytest

import oracle
from paper_2606_03681_amd import workloads as wl

from _harness import (TOL, compare_all, gpu_stack, nerr, oracle_params, oracle_rows,
                      oracle_stack, sample_rows)

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


@pytest.mark.parametrize("name", [0, "ragged-small-f32", "ragged-small-bf16", "d16-bf16",
                                  "d64-bf16", "d64-f32", "prenorm-small-bf16",
                                  "prenorm-d64-bf16", "wide-d32-bf16", "wide-d64-bf16",
                                  "wide-prenorm-d64-bf16", "mixed-prefix-bf16", "tiny-mlp-bf16"])
def test_parity_full(name):
    w = wl.make_workload(name)
    _say(f"[parity] {w.cfg['name']} seed={w.seed}")
    gpu = gpu_stack(w)
    errs = compare_all(w, gpu, oracle_stack(w))
    _say(f"[parity] {w.cfg['name']} worst={max(errs.values()):.3g}")


def test_parity_small_bf16_sampled_datasets():
    """cfg 1 (small bf16 layer): the whole batch on the GPU; the oracle on two datasets."""
    w = wl.make_workload(1)
    gpu = gpu_stack(w)
    sub = [0, 5]
    ws = wl.make_workload(1, datasets=sub)
    Y, dX, grads = oracle_stack(ws)
    tol = TOL["bf16"]
    assert nerr(gpu["Y"][sub], Y) <= tol
    assert nerr(gpu["dX"][sub], dX) <= tol
    # parameter gradients of the two datasets alone, through the library
    gsub = gpu_stack(ws)
    compare_all(ws, gsub, (Y, dX, grads))


def test_padding_is_inert_under_nan_poison():
    w = wl.make_workload("ragged-small-bf16")
    clean = gpu_stack(w, storage=True)
    X, dY = w.X.copy(), w.dY.copy()
    for b in range(X.shape[0]):
        off = w.cell_mask[b] == 0
        X[b][:, off] = 0x7FC0
        dY[b][:, off] = 0x7FC0
    pois = gpu_stack(w, X=X, dY=dY, storage=True)
    assert np.array_equal(pois["Y"], clean["Y"])
    assert np.array_equal(pois["dX"], clean["dX"])
    for a, b in zip(pois["grads"], clean["grads"]):
        assert np.array_equal(a, b)
    for b in range(X.shape[0]):
        off = w.cell_mask[b] == 0
        assert np.all(clean["Y"][b][:, off] == 0) and np.all(clean["dX"][b][:, off] == 0)


def test_bitwise_deterministic():
    w = wl.make_workload("ragged-small-bf16")
    a = gpu_stack(w, storage=True)
    b = gpu_stack(w, storage=True)
    assert np.array_equal(a["Y"], b["Y"]) and np.array_equal(a["dX"], b["dX"])
    for x, y in zip(a["grads"], b["grads"]):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("name", ["tiny-mlp-bf16", "ragged-small-f32", "prenorm-small-bf16",
                                  "mixed-prefix-bf16"])
def test_gradient_accumulation_is_exact(name):
    """A second backward with accumulate != 0 adds its gradients to the first call's: with a
    bitwise-reproducible backward the result is exactly twice the one-call gradients, on every
    reduction path (split-z sums, the folded LayerNorm affines, the LayerNorm column sums);
    dX is written, not accumulated."""
    import torch
    from paper_2606_03681_amd import tfm
    from paper_2606_03681_amd.stack import Stack, to_device
    w = wl.make_workload(name)
    dims = tfm.make_dims(dtype=w.dtype, block=w.block,
                         **{k: v for k, v in w.dims.items() if k != "dtype"})
    st = Stack(dims, w.n_train, w.cell_mask, w.params)
    st.forward(to_device(w.X, w.dtype))
    dY = to_device(w.dY, w.dtype)
    dx1 = st.backward(dY).clone()
    once = [g.clone() for g in st.grads]
    dx2 = st.backward(dY, accumulate=True)
    torch.cuda.synchronize()
    assert torch.equal(dx1, dx2)
    for g1, g2 in zip(once, st.grads):
        assert torch.equal(g2, 2 * g1)


def test_test_rows_do_not_change_train_outputs():
    """Changing every test row leaves the train rows' outputs bit-identical on the GPU."""
    w = wl.make_workload(1, datasets=[0, 1])
    a = gpu_stack(w, storage=True)
    X = w.X.copy()
    rng = np.random.default_rng(0)
    for b in range(2):
        n = w.n_train[b]
        X[b, n:] = wl.to_storage(rng.normal(0, 3, X[b, n:].shape), "bf16")
    c = gpu_stack(w, X=X, storage=True)
    for b in range(2):
        n = w.n_train[b]
        assert np.array_equal(a["Y"][b, :n], c["Y"][b, :n])


@pytest.mark.parametrize("cfg", [2, 3, 4, "record9-bf16"])
def test_full_size_sampled_rows(cfg):
    """Full-size workload in the benchmark's launch configuration, sampled rows per layer."""
    w = wl.make_workload(cfg)
    pre = w.block == "pre"
    dt, heads, R = w.dtype, w.cfg["heads"], w.cfg["R"]
    tol = TOL[dt]
    _say(f"[full] cfg{cfg} {w.cfg['name']}: GPU stack")
    run = gpu_stack(w, keep_acts=True, storage=True)
    Ps = oracle_params(w)
    order = np.argsort(w.n_train * w.cell_mask.sum(1), kind="stable")
    picks = [int(order[len(order) // 2])]
    inputs = [w.X] + run["acts"][:-1]
    for l in range(w.cfg["layers"]):
        for b in picks:
            n = int(w.n_train[b])
            tr, te = sample_rows(n, R, seed=100 * l + b)
            rows = np.concatenate([tr, te])
            Xb = wl.storage_to_f64(inputs[l][b], dt)
            Yq, _, _, act, keep = oracle_rows(Xb, w.cell_mask[b], Ps[l], heads, n, tr, te,
                                              block=w.block, decay=0.95 ** l)
            Yg = wl.storage_to_f64(run["acts"][l][b][rows][:, act], dt)
            e = nerr(Yg, Yq)
            _say(f"[full] cfg{cfg} layer {l} dataset {b} fwd err {e:.3g}")
            assert e <= tol
            # backward of this layer alone, upstream gradient only at the sampled rows
            dY = np.zeros_like(w.dY)
            dY[b][rows[:, None], act[None, :]] = w.dY[b][rows[:, None], act[None, :]]
            g = gpu_stack(w, X=inputs[l], dY=dY, params=[w.params[l]], storage=True,
                          first_layer=l)
            dYq = wl.storage_to_f64(dY[b][rows][:, act], dt)
            _, dz, gr, _, _ = oracle_rows(Xb, w.cell_mask[b], Ps[l], heads, n, tr, te, dYq,
                                          block=w.block, decay=0.95 ** l)
            dXg = wl.storage_to_f64(g["dX"], dt)
            e = nerr(dXg[b][keep][:, act], dz)
            _say(f"[full] cfg{cfg} layer {l} dataset {b} dX err {e:.3g}")
            assert e <= tol
            others = np.ones(dXg.shape[0], bool)
            others[b] = False
            assert np.all(dXg[others] == 0)
            rest = np.setdiff1d(np.arange(R), keep)
            assert np.all(dXg[b][rest] == 0)
            unpack = oracle.unpack_prenorm_params if pre else oracle.unpack_params
            names = oracle.PRENORM_PARAM_ORDER if pre else oracle.PARAM_ORDER
            pg = unpack(g["grads"][0], w.cfg["E"], w.cfg["H"])
            worst = max(nerr(pg[k], gr[k]) for k in names)
            _say(f"[full] cfg{cfg} layer {l} dataset {b} grads worst err {worst:.3g}")
            for k in names:
                assert nerr(pg[k], gr[k]) <= tol, k


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_thinking_rows_against_oracle(dtype):
    """Broadcast of the thinking-row table and its gradient, bit-exact for the broadcast (a copy
    with one rounding to the storage type) and within the float32 summation bound for dtable."""
    import torch
    from paper_2606_03681_amd import tfm
    from paper_2606_03681_amd.stack import to_device, to_host
    rng = np.random.default_rng(41)
    B, R, C, E, T = 3, 40, 13, 64, 5
    n_train = np.array([7, 5, 30], np.int32)
    mask = (rng.random((B, C + 1)) < 0.7).astype(np.uint8)
    mask[:, C] = 1
    dims = tfm.make_dims(B, R, C, E, 2, 128, dtype)
    ws = torch.empty(tfm.workspace_bytes(dims), dtype=torch.uint8, device="cuda")
    X = wl.to_storage(rng.normal(size=(B, R, C + 1, E)), dtype)
    table = rng.normal(size=(T, E)).astype(np.float32)
    Xd = to_device(X, dtype)
    tfm.thinking_rows_fwd(dims, n_train, mask, T, torch.from_numpy(table).cuda(), Xd, ws)
    got = to_host(Xd, dtype)
    ref = oracle.thinking_rows_forward(wl.storage_to_f64(X[:, T:], dtype),
                                       wl.storage_to_f64(wl.to_storage(table, dtype), dtype),
                                       mask)
    assert np.array_equal(got, ref)
    dX = wl.to_storage(rng.normal(size=(B, R, C + 1, E)), dtype)
    dt = torch.full((T, E), 7.0, device="cuda")
    tfm.thinking_rows_bwd(dims, n_train, mask, T, to_device(dX, dtype), dt, False, ws)
    _, dref = oracle.thinking_rows_backward(wl.storage_to_f64(dX, dtype), mask, T)
    n_terms = int(mask.sum())
    bound = n_terms * 2.0 ** -24 * np.abs(wl.storage_to_f64(dX, dtype)[:, :T]).sum(axis=(0, 2))
    assert np.all(np.abs(dt.cpu().numpy() - dref) <= bound + 1e-30)
    dt2 = dt.clone()
    tfm.thinking_rows_bwd(dims, n_train, mask, T, to_device(dX, dtype), dt2, True, ws)
    torch.cuda.synchronize()
    assert np.allclose(dt2.cpu().numpy(), 2 * dt.cpu().numpy(), rtol=1e-6, atol=0)
