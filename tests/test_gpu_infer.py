"""GPU parity of the forward-only calls (context and query) through the C ABI.

* A context call runs the layer exactly as the training forward does: the stack's outputs are
  bit-identical to those of tfm_layer_fwd.
* Query calls on chunks of unlabelled rows, against the key/value caches of the context rows,
  give those rows' outputs of the whole-table forward: bit-identical to the training forward on
  [context rows; query rows], and within the bf16 tolerance of the float64 oracle."""

import sys

import numpy as np
import pytest

import oracle
from paper_2606_03681_amd import workloads as wl

from _harness import TOL, nerr, oracle_params, storage_of

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


def _dims(w, R=None):
    from paper_2606_03681_amd import tfm
    kw = {k: v for k, v in w.dims.items() if k != "dtype"}
    if R is not None:
        kw["R"] = R
    return tfm.make_dims(dtype=w.dtype, block=w.block, **kw)


def _train_forward(w, X, n_train):
    import torch
    from paper_2606_03681_amd.stack import Stack, to_device
    st = Stack(_dims(w, X.shape[1]), n_train, w.cell_mask, w.params)
    Y = storage_of(st.forward(to_device(X, "bf16")), "bf16")
    torch.cuda.synchronize()
    return Y


def _oracle_forward(w, X, n_train):
    Ps = oracle_params(w)
    X64 = wl.storage_to_f64(X, "bf16")
    if w.block == "pre":
        Y, _ = oracle.prenorm_stack_forward(X64, Ps, n_train, w.cell_mask, w.cfg["heads"])
    else:
        Y, _ = oracle.stack_forward(X64, Ps, n_train, w.cell_mask, w.cfg["heads"])
    return Y


@pytest.mark.parametrize("name", ["ragged-small-bf16", "d16-bf16", "d64-bf16",
                                  "prenorm-small-bf16", "prenorm-d64-bf16", "wide-d32-bf16",
                                  "wide-prenorm-d64-bf16"])
def test_context_and_query_chunks(name):
    import torch
    from paper_2606_03681_amd.stack import InferStack, to_device
    w = wl.make_workload(name)
    R = w.cfg["R"]
    Rc = R - (R // 3 + 5)                       # context rows; the rest arrive as queries
    n_train = np.minimum(w.n_train, Rc).astype(np.int32)
    chunks = [(Rc, Rc + 37), (Rc + 37, R)]      # two ragged query chunks
    _say(f"[infer] {name} Rc={Rc} chunks={chunks}")
    full = _train_forward(w, w.X, n_train)
    inf = InferStack(_dims(w, Rc), n_train, w.cell_mask, w.params,
                     max_query_rows=max(b - a for a, b in chunks))
    Yc = storage_of(inf.context(to_device(np.ascontiguousarray(w.X[:, :Rc]), "bf16")), "bf16")
    parts = [Yc]
    for a, b in chunks:
        Xq = to_device(np.ascontiguousarray(w.X[:, a:b]), "bf16")
        parts.append(storage_of(inf.query(Xq), "bf16"))
    torch.cuda.synchronize()
    got = np.concatenate(parts, axis=1)
    # the training forward over the whole table, context and query rows alike
    assert np.array_equal(got, full)
    ref = _oracle_forward(w, w.X, n_train)
    e = nerr(wl.storage_to_f64(got, "bf16"), ref)
    _say(f"[infer] {name} err vs oracle {e:.3g}")
    assert e <= TOL["bf16"]


def test_context_on_whole_table_equals_training_forward():
    """cfg 1 (small bf16 layer) with its own n_train: the context call is the plain forward."""
    import torch
    from paper_2606_03681_amd.stack import InferStack, to_device
    w = wl.make_workload(1)
    full = _train_forward(w, w.X, w.n_train)
    inf = InferStack(_dims(w), w.n_train, w.cell_mask, w.params, max_query_rows=1)
    Y = storage_of(inf.context(to_device(w.X, "bf16")), "bf16")
    torch.cuda.synchronize()
    assert np.array_equal(Y, full)


def test_query_rows_independent_of_each_other():
    """A query row's output does not depend on the other rows of its chunk."""
    import torch
    from paper_2606_03681_amd.stack import InferStack, to_device
    w = wl.make_workload("prenorm-small-bf16")
    Rc = 120
    n_train = np.minimum(w.n_train, Rc).astype(np.int32)
    inf = InferStack(_dims(w, Rc), n_train, w.cell_mask, w.params, max_query_rows=64)
    inf.context(to_device(np.ascontiguousarray(w.X[:, :Rc]), "bf16"))
    a = storage_of(inf.query(to_device(np.ascontiguousarray(w.X[:, Rc:Rc + 64]), "bf16")),
                   "bf16")
    one = storage_of(inf.query(to_device(np.ascontiguousarray(w.X[:, Rc + 10:Rc + 11]),
                                         "bf16")), "bf16")
    torch.cuda.synchronize()
    assert np.array_equal(a[:, 10:11], one)


@pytest.mark.parametrize("cfg", [2, "record9-bf16"])
def test_full_size_forward_only_matches_training_forward(cfg):
    """The benchmark's forward-only configuration at full size (context = the longest train
    prefix, the remaining rows as query chunks of 128 and a ragged tail): bit-identical to the
    training forward, whose outputs the full-size sampled-row parity test checks against the
    oracle."""
    import torch
    from paper_2606_03681_amd.stack import InferStack, to_device
    w = wl.make_workload(cfg)
    R = w.cfg["R"]
    Rc = int(np.max(w.n_train))
    _say(f"[infer-full] {w.cfg['name']} Rc={Rc}")
    full = _train_forward(w, w.X, w.n_train)
    inf = InferStack(_dims(w, Rc), w.n_train, w.cell_mask, w.params, max_query_rows=128)
    got = [storage_of(inf.context(to_device(np.ascontiguousarray(w.X[:, :Rc]), "bf16")), "bf16")]
    for a in range(Rc, R, 128):
        b = min(a + 128, R) if a + 128 < R else R
        got.append(storage_of(inf.query(to_device(np.ascontiguousarray(w.X[:, a:b]), "bf16")),
                              "bf16"))
    torch.cuda.synchronize()
    got = np.concatenate(got, axis=1)
    for b in range(got.shape[0]):
        assert np.array_equal(got[b], full[b]), f"dataset {b}"
