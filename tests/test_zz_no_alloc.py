"""The allocation-free forward (tfm_layer_fwd_noalloc) against tfm_layer_fwd, through the C ABI.

Two calls in a row share the library's scratch array, the second on a smaller input of other
dims.  Each must give Y bit for bit equal to the workspace entry point's, and a state that the
backward pass turns into the same dX and parameter gradients, bit for bit (the same kernels run
on the same inputs; only where the plan and the bfloat16 weights live differs)."""

import numpy as np
import pytest

from paper_2606_03681_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _same_call(name, datasets=None):
    import torch
    from paper_2606_03681_amd import tfm
    from paper_2606_03681_amd.stack import to_device
    w = wl.make_workload(name, datasets=datasets)
    dims = tfm.make_dims(dtype=w.dtype, block=w.block,
                         **{k: v for k, v in w.dims.items() if k != "dtype"})
    X = to_device(w.X, w.dtype)
    dY = to_device(w.dY, w.dtype)
    P = torch.from_numpy(np.ascontiguousarray(w.params[0])).cuda()
    sb, wb = tfm.saved_bytes(dims), tfm.workspace_bytes(dims)
    ws = torch.empty(wb, dtype=torch.uint8, device="cuda")
    Ya = torch.empty_like(X)
    Yb = torch.full_like(X, 3.0)          # garbage where the call must write zeros
    Sa = torch.zeros(sb, dtype=torch.uint8, device="cuda")
    Sb = torch.full((sb,), 0xAB, dtype=torch.uint8, device="cuda")
    tfm.layer_fwd(dims, w.n_train, w.cell_mask, X, P, Ya, Sa, ws)
    tfm.layer_fwd_noalloc(dims, w.n_train, w.cell_mask, X, P, Yb, Sb)
    torch.cuda.synchronize()
    assert torch.equal(Ya.view(torch.int16), Yb.view(torch.int16)), name
    out = []
    for S in (Sa, Sb):
        dX = torch.empty_like(X)
        g = torch.empty_like(P)
        tfm.layer_bwd(dims, w.n_train, w.cell_mask, X, P, S, dY, dX, g, False, ws)
        out.append((dX, g))
    torch.cuda.synchronize()
    assert torch.equal(out[0][0].view(torch.int16), out[1][0].view(torch.int16)), name
    assert torch.equal(out[0][1], out[1][1]), name


def test_noalloc_forward_two_calls():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    # first call: 5 datasets x 333 rows, E = 192 (6 heads of 32); second: a smaller input of
    # other dims (3 datasets x 130 rows, E = 64 with heads of 16), through the same scratch
    _same_call("ragged-small-bf16")
    _same_call("d16-bf16")
    # and the pre-norm block, again smaller than the first call
    _same_call("prenorm-small-bf16", datasets=[0, 3])
