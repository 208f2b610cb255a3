"""Pins of the pre-norm (current best record) oracle against facts fixed by the mathematics:
finite differences of every gradient, the RMSNorm moments, the zero-weight block (identity times
the decay), test-row isolation, column equivariance, the thinking-row broadcast and its
gradient, and an independent rebuild from torch CPU float64 library routines with autograd."""

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle


def _micro(seed=11, n_train=(4, 3), R=6, S=4, E=8, heads=2, H=16, mask=None):
    rng = np.random.default_rng(seed)
    B = len(n_train)
    X = rng.normal(0, 1, (B, R, S, E))
    P = oracle.unpack_prenorm_params(rng.normal(0, 0.4, oracle.prenorm_param_count(E, H)), E, H)
    for g in ("g1", "g2", "g3"):
        P[g] = 1.0 + 0.3 * rng.normal(size=E)
    m = np.ones((B, S), bool) if mask is None else np.asarray(mask, bool)
    dY = rng.normal(0, 1, (B, R, S, E))
    return X, P, np.array(n_train), m, dY


def _loss(X, P, nt, m, dY, heads, decay):
    Y, _ = oracle.prenorm_layer_forward(X, P, nt, m, heads, decay)
    return float((Y * dY).sum())


def test_prenorm_finite_differences_every_parameter_and_input():
    mask = [[1, 1, 1, 1], [1, 1, 0, 1]]
    X, P, nt, m, dY = _micro(mask=mask)
    heads, decay = 2, 0.9025
    Y, cache = oracle.prenorm_layer_forward(X, P, nt, m, heads, decay)
    dX, grads = oracle.prenorm_layer_backward(dY, cache)
    h = 1e-6
    for name in oracle.PRENORM_PARAM_ORDER:
        arr = P[name]
        fd = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            old = arr[idx]
            arr[idx] = old + h
            lp = _loss(X, P, nt, m, dY, heads, decay)
            arr[idx] = old - h
            lm = _loss(X, P, nt, m, dY, heads, decay)
            arr[idx] = old
            fd[idx] = (lp - lm) / (2 * h)
        err = np.abs(fd - grads[name]).max() / max(np.abs(fd).max(), 1e-30)
        assert err < 1e-6, (name, err)
    fdx = np.zeros_like(X)
    for idx in np.ndindex(X.shape):
        old = X[idx]
        X[idx] = old + h
        lp = _loss(X, P, nt, m, dY, heads, decay)
        X[idx] = old - h
        lm = _loss(X, P, nt, m, dY, heads, decay)
        X[idx] = old
        fdx[idx] = (lp - lm) / (2 * h)
    assert np.abs(fdx - dX).max() / np.abs(fdx).max() < 1e-6
    assert np.all(dX[1, :, 2, :] == 0) and np.all(Y[1, :, 2, :] == 0)


def test_rmsnorm_moments_and_gradient():
    rng = np.random.default_rng(5)
    u = rng.normal(0, 3, (7, 16))
    y, uhat, rstd = oracle.rmsnorm(u, np.ones(16), eps=1e-6)
    ms = (u * u).mean(axis=1)
    assert np.allclose((y * y).mean(axis=1), ms / (ms + 1e-6), rtol=0, atol=1e-14)
    # scale invariance: RMS(a u) = RMS(u) up to eps
    y2, _, _ = oracle.rmsnorm(5.0 * u, np.ones(16), eps=0.0)
    y3, _, _ = oracle.rmsnorm(u, np.ones(16), eps=0.0)
    assert np.allclose(y2, y3, rtol=0, atol=1e-14)
    g = 1 + 0.2 * rng.normal(size=16)
    dy = rng.normal(size=u.shape)
    _, uh, rs = oracle.rmsnorm(u, g, eps=1e-6)
    du, dg = oracle.rmsnorm_backward(dy, uh, rs, g)
    h = 1e-6
    fd = np.zeros_like(u)
    for idx in np.ndindex(u.shape):
        up, um = u.copy(), u.copy()
        up[idx] += h
        um[idx] -= h
        fd[idx] = ((oracle.rmsnorm(up, g)[0] * dy).sum() - (oracle.rmsnorm(um, g)[0] * dy).sum()) / (2 * h)
    assert np.abs(fd - du).max() / np.abs(fd).max() < 1e-7
    assert np.allclose(dg, (dy * uh).sum(axis=0), rtol=1e-13)


def test_zero_weights_give_decayed_identity():
    """With every linear weight and bias 0 both attention outputs and the MLP output vanish, so
    the block returns its decayed input exactly and dX = decay * dY."""
    X, P, nt, m, dY = _micro()
    for k in P:
        if not k.startswith("g"):
            P[k][...] = 0.0
    Y, cache = oracle.prenorm_layer_forward(X, P, nt, m, 2, 0.95)
    assert np.array_equal(Y, 0.95 * X)
    dX, g = oracle.prenorm_layer_backward(dY, cache)
    assert np.allclose(dX, 0.95 * dY, rtol=1e-15, atol=0)
    assert np.allclose(g["b2"], dY.sum(axis=(0, 1, 2)), rtol=1e-13)


def test_prenorm_test_rows_isolated():
    X, P, nt, m, dY = _micro(n_train=(3, 3))
    Y, _ = oracle.prenorm_layer_forward(X, P, nt, m, 2, 1.0)
    X2 = X.copy()
    X2[:, 4] += 3.0                    # change one test row
    Y2, _ = oracle.prenorm_layer_forward(X2, P, nt, m, 2, 1.0)
    assert np.array_equal(Y[:, :4], Y2[:, :4]) and np.array_equal(Y[:, 5], Y2[:, 5])
    # a test row equals the block run on [train rows; that row]
    sub = X[:, [0, 1, 2, 5]]
    Ys, _ = oracle.prenorm_layer_forward(sub, P, nt, m, 2, 1.0)
    assert np.allclose(Ys[:, 3], Y[:, 5], rtol=0, atol=1e-13)


def test_prenorm_column_equivariance():
    X, P, nt, m, dY = _micro()
    perm = np.array([2, 0, 3, 1])
    Y, _ = oracle.prenorm_layer_forward(X, P, nt, m, 2, 0.95)
    Yp, _ = oracle.prenorm_layer_forward(X[:, :, perm], P, nt, m[:, perm], 2, 0.95)
    assert np.allclose(Yp, Y[:, :, perm], rtol=0, atol=1e-13)


def test_thinking_rows_broadcast_and_gradient():
    rng = np.random.default_rng(2)
    B, R, S, E, T = 2, 5, 4, 6, 3
    X = rng.normal(size=(B, R, S, E))
    table = rng.normal(size=(T, E))
    m = np.array([[1, 0, 1, 1], [1, 1, 1, 1]], bool)
    Z = oracle.thinking_rows_forward(X, table, m)
    assert Z.shape == (B, T + R, S, E)
    assert np.array_equal(Z[:, T:], X)
    for b in range(B):
        for c in range(S):
            want = table if m[b, c] else np.zeros_like(table)
            assert np.array_equal(Z[b, :T, c], want)
    dZ = rng.normal(size=Z.shape)
    dX, dt = oracle.thinking_rows_backward(dZ, m, T)
    assert np.array_equal(dX, dZ[:, T:])
    brute = np.zeros_like(table)
    for b in range(B):
        for c in range(S):
            if m[b, c]:
                brute += dZ[b, :T, c]
    assert np.allclose(dt, brute, rtol=1e-14)


def _torch_prenorm(X, P, n_train, mask, heads, decay, eps):
    B, R, S, E = X.shape
    d = E // heads
    cell = mask[:, None, :, None].to(X.dtype)
    x = decay * X * cell

    def attend(Z, W, b, Wo, bo, keymask, L):
        qkv = F.linear(Z, W, b).reshape(-1, L, 3, heads, d)
        q, k, v = (qkv[:, :, i].transpose(1, 2) for i in range(3))
        o = F.scaled_dot_product_attention(q, k, v, attn_mask=keymask)
        return F.linear(o.transpose(1, 2).reshape(-1, L, E), Wo, bo)

    r1 = F.rms_norm(x, (E,), P["g1"], eps)
    kmask = mask[:, None, :].expand(B, R, S).reshape(B * R, 1, 1, S)
    h1 = x + attend(r1.reshape(B * R, S, E), P["Wqkv_f"], P["bqkv_f"], P["Wo_f"], P["bo_f"],
                    kmask, S).reshape(B, R, S, E)
    r2 = F.rms_norm(h1, (E,), P["g2"], eps).permute(0, 2, 1, 3).reshape(B * S, R, E)
    t = torch.arange(R)
    tmask = (t[None, :] < n_train[:, None])[:, None, :].expand(B, S, R).reshape(B * S, 1, 1, R)
    a = attend(r2, P["Wqkv_i"], P["bqkv_i"], P["Wo_i"], P["bo_i"], tmask, R)
    h2 = h1 + a.reshape(B, S, R, E).permute(0, 2, 1, 3)
    r3 = F.rms_norm(h2, (E,), P["g3"], eps)
    y = h2 + F.linear(F.gelu(F.linear(r3, P["W1"], P["b1"]), approximate="none"), P["W2"],
                      P["b2"])
    return y * cell


def test_prenorm_matches_torch_autograd():
    X, P, nt, m, dY = _micro(mask=[[1, 1, 0, 1], [1, 1, 1, 1]], n_train=(4, 2), S=4)
    heads, decay = 2, 0.95
    Y, cache = oracle.prenorm_layer_forward(X, P, nt, m, heads, decay)
    dX, grads = oracle.prenorm_layer_backward(dY, cache)
    Xt = torch.tensor(X, requires_grad=True)
    Pt = {k: torch.tensor(v, requires_grad=True) for k, v in P.items()}
    Yt = _torch_prenorm(Xt, Pt, torch.tensor(nt), torch.tensor(m), heads, decay, oracle.RMS_EPS)
    (Yt * torch.tensor(dY * m[:, None, :, None])).sum().backward()
    assert np.abs(Yt.detach().numpy() - Y).max() <= 1e-10 * np.abs(Y).max()
    assert np.abs(Xt.grad.numpy() - dX).max() <= 1e-10 * np.abs(dX).max()
    for k in P:
        ref = Pt[k].grad.numpy()
        assert np.abs(ref - grads[k]).max() <= 1e-10 * max(np.abs(ref).max(), 1e-300), k


def test_prenorm_param_packing_roundtrip_and_count():
    E, H = 256, 768
    n = oracle.prenorm_param_count(E, H)
    assert n == 2 * (4 * E * E + 4 * E) + 2 * E * H + H + E + 3 * E == 921344
    flat = np.arange(n, dtype=np.float64)
    assert np.array_equal(oracle.pack_prenorm_params(oracle.unpack_prenorm_params(flat, E, H)), flat)
    with pytest.raises(ValueError):
        oracle.unpack_prenorm_params(flat[:-1], E, H)
