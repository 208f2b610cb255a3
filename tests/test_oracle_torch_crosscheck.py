"""Cross-check of the float64 oracle against an independent construction of the same layer from
torch CPU float64 library routines (scaled_dot_product_attention with a boolean key mask,
layer_norm, linear, exact gelu) with gradients from autograd instead of the oracle's
hand-derived backward.  Padding is handled here by masks instead of by the oracle's slicing.
"""

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from paper_2606_03681_amd import workloads as wl


def _torch_layer(X, P, n_train, mask, heads):
    """X: (B, R, S, E) float64 tensor; P: dict of float64 tensors; mask: (B, S) bool tensor."""
    B, R, S, E = X.shape
    d = E // heads
    cell = mask[:, None, :, None].to(X.dtype)          # inactive cells forced to 0
    Z = X * cell
    # feature axis: sequences are the rows, length S; padded keys masked out
    qkv = F.linear(Z, P["Wqkv_f"], P["bqkv_f"]).reshape(B * R, S, 3, heads, d)
    q, k, v = (qkv[:, :, i].transpose(1, 2) for i in range(3))       # (B*R, h, S, d)
    kmask = mask[:, None, :].expand(B, R, S).reshape(B * R, 1, 1, S)
    o = F.scaled_dot_product_attention(q, k, v, attn_mask=kmask)
    o = o.transpose(1, 2).reshape(B, R, S, E)
    H1 = F.layer_norm(Z + F.linear(o, P["Wo_f"], P["bo_f"]), (E,), P["g1"], P["be1"], 1e-5)
    # item axis: sequences are the columns, length R; keys are rows t < n_train
    Zc = H1.permute(0, 2, 1, 3)                                       # (B, S, R, E)
    qkv = F.linear(Zc, P["Wqkv_i"], P["bqkv_i"]).reshape(B * S, R, 3, heads, d)
    q, k, v = (qkv[:, :, i].transpose(1, 2) for i in range(3))       # (B*S, h, R, d)
    t = torch.arange(R)
    tmask = (t[None, :] < n_train[:, None])                           # (B, R) keys
    tmask = tmask[:, None, :].expand(B, S, R).reshape(B * S, 1, 1, R)
    o = F.scaled_dot_product_attention(q, k, v, attn_mask=tmask)
    o = o.transpose(1, 2).reshape(B, S, R, E).permute(0, 2, 1, 3)
    H2 = F.layer_norm(H1 + F.linear(o, P["Wo_i"], P["bo_i"]), (E,), P["g2"], P["be2"], 1e-5)
    M = F.linear(F.gelu(F.linear(H2, P["W1"], P["b1"]), approximate="none"), P["W2"], P["b2"])
    Y = F.layer_norm(H2 + M, (E,), P["g3"], P["be3"], 1e-5)
    return Y * cell


def _nerr(a, b):
    return float(np.abs(a - b).max() / max(np.abs(b).max(), 1e-300))


@pytest.mark.parametrize("name", ["ragged-small-f32", "d16-bf16"])
def test_oracle_matches_torch_autograd(name):
    w = wl.make_workload(name)
    cfg = w.cfg
    E, H, heads = cfg["E"], cfg["H"], cfg["heads"]
    X = w.X64()
    dY = w.dY64()
    Ps = [oracle.unpack_params(p, E, H) for p in w.params64()]
    Y, caches = oracle.stack_forward(X, Ps, w.n_train, w.cell_mask, heads)
    dX, grads = oracle.stack_backward(dY, caches)

    Xt = torch.tensor(X, requires_grad=True)
    Pt = [{k: torch.tensor(v, requires_grad=True) for k, v in P.items()} for P in Ps]
    mask = torch.tensor(w.cell_mask.astype(bool))
    nt = torch.tensor(w.n_train.astype(np.int64))
    out = Xt
    for P in Pt:
        out = _torch_layer(out, P, nt, mask, heads)
    cell = mask[:, None, :, None].to(out.dtype)
    (out * torch.tensor(dY) * cell).sum().backward()

    assert _nerr(Y, out.detach().numpy()) < 1e-10
    assert _nerr(dX, (Xt.grad * cell).numpy()) < 1e-10
    for l in range(len(Ps)):
        for k in oracle.PARAM_ORDER:
            assert _nerr(grads[l][k], Pt[l][k].grad.numpy()) < 1e-10, (l, k)
