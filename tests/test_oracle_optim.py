"""Pins of the float64 optimiser oracle (oracle/optim.py) against facts independent of its own
formulas: the Newton-Schulz map against the SVD (it acts on the singular values alone), its
scale and transpose invariance, Muon's first-step and orientation closed forms, schedule-free
AdamW against its derived two-sequence (y, z) form, the averaging weights of its x sequence,
its reduction to bias-corrected RMSprop at b1 = 0 and Adam's sign-like first step, and the
clip factor against numpy's norm."""

import numpy as np
import pytest

from oracle import optim


def _phi(s, steps=5):
    a, b, c = optim.NS_COEFFS
    for _ in range(steps):
        s = a * s + b * s ** 3 + c * s ** 5
    return s


@pytest.mark.parametrize("shape", [(16, 16), (12, 20), (20, 12), (3, 40)])
def test_newton_schulz_acts_on_singular_values(shape):
    G = np.random.default_rng(1).normal(size=shape)
    U, S, Vt = np.linalg.svd(G, full_matrices=False)
    want = U @ np.diag(_phi(S / (np.linalg.norm(G) + optim.NS_EPS))) @ Vt
    assert np.allclose(optim.newton_schulz(G), want, rtol=1e-10, atol=1e-12)


def test_newton_schulz_scale_and_transpose_invariance():
    G = np.random.default_rng(2).normal(size=(10, 24))
    X = optim.newton_schulz(G)
    assert np.allclose(optim.newton_schulz(5.0 * G), X, rtol=1e-6, atol=1e-8)
    assert np.allclose(optim.newton_schulz(G.T), X.T, rtol=1e-12, atol=1e-14)
    # a well-conditioned input comes out near-orthogonal: singular values in [0.6, 1.25]
    Q, _ = np.linalg.qr(np.random.default_rng(3).normal(size=(24, 10)))
    s = np.linalg.svd(optim.newton_schulz(Q.T * np.linspace(1.0, 2.0, 10)[:, None]),
                      compute_uv=False)
    assert s.min() > 0.6 and s.max() < 1.25


def test_muon_first_step_is_the_orthogonalised_gradient():
    """buf = (1 - m) g and the Nesterov input (1 - m)(1 + m) g are multiples of g, and the map
    normalises its input, so the first step moves along NS(g) whatever the momentum."""
    rng = np.random.default_rng(4)
    W = rng.normal(size=(3, 8, 8))
    G = rng.normal(size=(3, 8, 8))
    lr, wd = 0.02, 0.1
    for m in (0.0, 0.5, 0.96):
        W1, buf = optim.muon_step(W, G, np.zeros_like(W), lr, m, wd)
        assert np.allclose(buf, (1 - m) * G)
        want = W * (1 - lr * wd) - lr * np.stack([optim.newton_schulz(g) for g in G])
        assert np.allclose(W1, want, rtol=1e-6, atol=1e-9)


def test_muon_second_step_uses_the_nesterov_look_ahead():
    rng = np.random.default_rng(5)
    W = rng.normal(size=(2, 6, 10))
    g1, g2 = rng.normal(size=(2, 2, 6, 10))
    m, lr = 0.9, 0.05
    W1, b1 = optim.muon_step(W, g1, np.zeros_like(W), lr, m, 0.0)
    W2, b2 = optim.muon_step(W1, g2, b1, lr, m, 0.0)
    buf = m * (1 - m) * g1 + (1 - m) * g2
    assert np.allclose(b2, buf)
    U = (1 - m) * g2 + m * buf
    assert np.allclose(W2, W1 - lr * np.stack([optim.newton_schulz(u) for u in U]))


def test_muon_tall_matrices_get_the_aspect_factor():
    rng = np.random.default_rng(6)
    for rows, cols in ((24, 6), (6, 24)):
        W = rng.normal(size=(1, rows, cols))
        G = rng.normal(size=(1, rows, cols))
        W1, _ = optim.muon_step(W, G, np.zeros_like(W), 0.1, 0.0, 0.0)
        k = max(1.0, rows / cols) ** 0.5
        assert np.allclose(W - W1, 0.1 * k * optim.newton_schulz(G[0])[None])


def _y_form(y0, grads, lr, b1, b2, eps, wd, warmup):
    """The schedule-free update rewritten on y and z alone (x = (y - (1 - b1) z) / b1 never
    stored): y <- y + c (z - y) + gamma (b1 (1 - c) - 1) u, z <- z - gamma u with
    u = g / (sqrt(v) + eps) + wd y."""
    y = y0.copy()
    z = y0.copy()
    v = np.zeros_like(y0)
    ssum = 0.0
    out = []
    for t, g in enumerate(grads, start=1):
        s = lr * (min(1.0, t / warmup) if warmup else 1.0)
        v = b2 * v + (1 - b2) * g * g
        gamma = s * np.sqrt(1 - b2 ** t)
        u = g / (np.sqrt(v) + eps) + wd * y
        ssum += gamma * gamma
        c = gamma * gamma / ssum
        y = y + c * (z - y) + gamma * (b1 * (1 - c) - 1) * u
        z = z - gamma * u
        out.append(y.copy())
    return out


@pytest.mark.parametrize("warmup,wd", [(0, 0.0), (4, 0.01)])
def test_schedule_free_matches_its_two_sequence_form(warmup, wd):
    rng = np.random.default_rng(7)
    y0 = rng.normal(size=50)
    grads = rng.normal(size=(10, 50))
    opt = optim.ScheduleFreeAdamW(y0, 1e-2, weight_decay=wd, warmup=warmup)
    ys = [opt.step(g) for g in grads]
    for a, b in zip(ys, _y_form(y0, grads, 1e-2, 0.9, 0.999, 1e-8, wd, warmup)):
        assert np.allclose(a, b, rtol=1e-12, atol=1e-14)


def test_schedule_free_x_is_the_weighted_average_of_z():
    rng = np.random.default_rng(8)
    opt = optim.ScheduleFreeAdamW(rng.normal(size=20), 3e-3, warmup=5)
    for g in rng.normal(size=(12, 20)):
        opt.step(g)
    w = np.array(opt.gamma_hist) ** 2
    avg = (w[:, None] * np.array(opt.z_hist[1:])).sum(axis=0) / w.sum()
    assert np.allclose(opt.x, avg, rtol=1e-12, atol=1e-15)


def test_schedule_free_averaging_weights_closed_form():
    """Without warm-up gamma_t^2 = lr^2 (1 - b2^t), so the averaging weights are
    c_{t+1} = (1 - b2^t) / (t - b2 (1 - b2^t) / (1 - b2)): 1, then 0.666556..., 0.499833...
    at b2 = 0.999 (not 1/t, which a schedule without the bias correction would give).  With
    b1 = 0, y is x, so x_{t+1} = (1 - c) x_t + c z_{t+1} can be checked step by step."""
    rng = np.random.default_rng(12)
    lr, b2 = 2e-2, 0.999
    opt = optim.ScheduleFreeAdamW(rng.normal(size=8), lr, beta1=0.0, beta2=b2)
    expected = [1.0, 0.6665555185, 0.4998333056]
    for t in range(1, 7):
        x_prev = opt.x.copy()
        opt.step(rng.normal(size=8))
        c = (1 - b2 ** t) / sum(1 - b2 ** i for i in range(1, t + 1))
        closed = (1 - b2 ** t) / (t - b2 * (1 - b2 ** t) / (1 - b2))
        assert abs(c - closed) < 1e-9
        if t <= 3:
            assert abs(c - expected[t - 1]) < 1e-9
        assert np.allclose(opt.x, (1 - c) * x_prev + c * opt.z, rtol=1e-13, atol=1e-15)


def test_schedule_free_without_momentum_is_bias_corrected_rmsprop():
    rng = np.random.default_rng(9)
    y0 = rng.normal(size=30)
    grads = rng.normal(size=(6, 30))
    opt = optim.ScheduleFreeAdamW(y0, 1e-2, beta1=0.0, weight_decay=0.05)
    y, v = y0.copy(), np.zeros(30)
    for t, g in enumerate(grads, start=1):
        v = 0.999 * v + 0.001 * g * g
        y = y - 1e-2 * np.sqrt(1 - 0.999 ** t) * (g / (np.sqrt(v) + 1e-8) + 0.05 * y)
        assert np.allclose(opt.step(g), y, rtol=1e-12, atol=1e-15)


def test_schedule_free_first_step_is_sign_like():
    """v_1 = (1 - b2) g^2 and the bias correction cancel it: with eps = 0 the first step moves
    z by exactly -lr sign(g), and since c_2 = 1 the next y is that z."""
    rng = np.random.default_rng(10)
    y0 = rng.normal(size=40)
    g = rng.normal(size=40)
    opt = optim.ScheduleFreeAdamW(y0, 0.25, eps=0.0)
    assert np.allclose(opt.step(g), y0 - 0.25 * np.sign(g), rtol=1e-13, atol=1e-13)


def test_clip_scale():
    rng = np.random.default_rng(11)
    gs = [rng.normal(size=s) for s in ((3, 4), (7,), (2, 2, 2))]
    norm = np.linalg.norm(np.concatenate([g.ravel() for g in gs]))
    n, s = optim.clip_scale(gs, 1e9)
    assert np.isclose(n, norm, rtol=1e-14) and s == 1.0
    n, s = optim.clip_scale(gs, 1.0)
    assert np.isclose(s * norm, 1.0, rtol=1e-5)
