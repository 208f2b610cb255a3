"""GPU parity at the full-size workloads with dense upstream gradients, against the float64 oracle.

The whole batch runs through the whole stack on the GPU in the benchmark's launch configuration
(every dataset, every layer, one forward and one backward per layer).  The oracle runs whole
datasets of that batch through the same stack, forward and backward, with the upstream gradient
of every row and every active cell:

* Y and dX of those datasets are compared with the whole-batch GPU run (the datasets of a batch
  are independent, so a dataset's outputs do not depend on which others share its launch);
* every parameter gradient is compared with a GPU run of those datasets alone (the whole-batch
  gradients sum over every dataset, which the oracle does not evaluate).

So the compounding of the bf16 roundings across the stacked layers, and the gradient sums over
every query row (the dK/dV and dQ accumulations of item attention over whole train prefixes,
6,144 keys in the many-rows workload) are compared at their real sizes.  Tolerance: the
normwise-max relative error per tensor, <= 2e-2 in bfloat16 mode, on Y, dX and every gradient
block of every layer.

The oracle evaluates the item-axis attention problems of a layer on several threads (an
execution setting of the oracle; the arithmetic of each problem is unchanged)."""

import os
import sys

import numpy as np
import pytest

from oracle import layer as oracle_layer
from paper_2606_03681_amd import workloads as wl

from _harness import TOL, compare_all, gpu_stack, nerr, oracle_stack

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
    oracle_layer.set_workers(min(os.cpu_count() or 1, 16))
    yield
    oracle_layer.set_workers(1)


def _picks(w, cfg):
    """Datasets checked against the oracle: for the ragged batch the smallest and the largest by
    n_train x active cells (the extremes of the train prefix and of the row width), otherwise
    two datasets of the batch."""
    if cfg == 4:
        size = w.n_train.astype(np.int64) * w.cell_mask.sum(1)
        return [int(np.argmin(size)), int(np.argmax(size))]
    if cfg == 3:
        return [1]
    return [0, len(w.n_train) - 1]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("cfg", [2, 3, 4])
def test_full_size_dense(cfg):
    w = wl.make_workload(cfg)
    sub = _picks(w, cfg)
    _say(f"[dense] cfg{cfg} {w.cfg['name']}: whole batch on the GPU "
         f"(B={len(w.n_train)}, layers={w.cfg['layers']})")
    gpu = gpu_stack(w)
    ws = wl.make_workload(cfg, datasets=sub)
    _say(f"[dense] cfg{cfg}: oracle on datasets {sub} (n_train={ws.n_train.tolist()}, "
         f"active cells per row={ws.cell_mask.sum(1).tolist()})")
    ref = oracle_stack(ws)
    Y, dX, _ = ref
    tol = TOL["bf16"]
    eY, edX = nerr(gpu["Y"][sub], Y), nerr(gpu["dX"][sub], dX)
    _say(f"[dense] cfg{cfg}: whole-batch Y err {eY:.3g}, dX err {edX:.3g}")
    assert eY <= tol and edX <= tol
    # padded cells of those datasets are exactly zero in the whole-batch run
    for i, b in enumerate(sub):
        off = ws.cell_mask[i] == 0
        assert np.all(gpu["Y"][b][:, off] == 0) and np.all(gpu["dX"][b][:, off] == 0)
    del gpu
    gsub = gpu_stack(ws)
    errs = compare_all(ws, gsub, ref)
    worst = max(errs, key=errs.get)
    _say(f"[dense] cfg{cfg}: datasets {sub} alone, worst {worst} {errs[worst]:.3g}")
