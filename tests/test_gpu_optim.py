"""GPU parity of the optimiser step (include/tfm_optim.h) against the float64 oracle of
oracle/optim.py: the clip factor and global norm, schedule-free AdamW over segments of a vector
for several steps (the GPU runs the two-sequence form, the oracle the three-sequence form), and
Muon on batches of square, tall and wide matrices for several steps.  Tolerance: the float32
bar, normwise-max relative error <= 1e-4 per tensor (1e-5 for the norm)."""

import sys

import numpy as np
import pytest

from oracle import optim

from _harness import nerr

pytestmark = pytest.mark.gpu
TOL = 1e-4


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    from paper_2606_03681_amd import tfm
    tfm.lib()


def _dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def test_clip_scale_and_norm():
    import torch
    from paper_2606_03681_amd import tfm
    rng = np.random.default_rng(1)
    arrs = [rng.normal(size=n).astype(np.float32) for n in (1000, 5000, 1, 4097, 300000)]
    big = _dev(np.concatenate(arrs))
    # hand the arrays over as (pointer, count) pieces of one buffer: 4-byte aligned starts
    pieces, off = [], 0
    for a in arrs:
        pieces.append((big.data_ptr() + 4 * off, a.size))
        off += a.size
    counts = [n for _, n in pieces]
    ws = torch.empty(tfm.clip_workspace_bytes(counts), dtype=torch.uint8, device="cuda")
    for max_norm in (1e6, 2.0):
        out = torch.full((8,), -1.0, device="cuda")
        tfm.clip_scale(pieces, max_norm, out[0:], out[4:], ws)
        torch.cuda.synchronize()
        norm, scale = optim.clip_scale([a.astype(np.float64) for a in arrs], max_norm)
        gn, gs = float(out[4].item()), float(out[0].item())
        _say(f"[optim] clip max_norm={max_norm}: norm {gn:.8g} vs {norm:.8g}, scale {gs:.8g}")
        assert abs(gn - norm) <= 1e-5 * norm
        assert abs(gs - scale) <= 1e-5 * scale


@pytest.mark.parametrize("warmup,wd,b1", [(0, 0.0, 0.9), (3, 0.01, 0.9), (0, 0.05, 0.0)])
def test_sfadamw_against_three_sequence_oracle(warmup, wd, b1):
    import torch
    from paper_2606_03681_amd import tfm
    rng = np.random.default_rng(2)
    n = 10000
    segs = [(0, 100), (300, 4000), (5000, 1), (6000, 3999)]
    idx = np.concatenate([np.arange(o, o + k) for o, k in segs])
    y0 = rng.normal(size=n).astype(np.float32)
    lr = 1e-2
    hp = tfm.tfm_sfadamw(lr, b1, 0.999, 1e-8, wd, warmup)
    y, z, v = _dev(y0), _dev(y0), torch.zeros(n, device="cuda")
    gscale = torch.tensor([0.5], device="cuda")
    opt = optim.ScheduleFreeAdamW(y0[idx].astype(np.float64), lr, beta1=b1, weight_decay=wd,
                                  warmup=warmup)
    for t in range(1, 7):
        g = rng.normal(size=n).astype(np.float32)
        tfm.sfadamw_step(hp, t, segs, y, z, v, _dev(g), gscale)
        ref = opt.step(0.5 * g[idx].astype(np.float64))
        torch.cuda.synchronize()
        got = y.cpu().numpy().astype(np.float64)
        e = nerr(got[idx], ref)
        ez = nerr(z.cpu().numpy()[idx], opt.z)
        _say(f"[optim] sfadamw warmup={warmup} wd={wd} b1={b1} step {t}: y {e:.3g} z {ez:.3g}")
        assert e <= TOL and ez <= TOL
        rest = np.setdiff1d(np.arange(n), idx)
        assert np.array_equal(got[rest], y0[rest])
    # the step moved the parameters by more than the tolerance resolves
    assert nerr(y.cpu().numpy()[idx], y0[idx]) > 100 * TOL


MUON_CASES = [(3, 64, 64), (2, 96, 40), (2, 40, 96), (8, 256, 256), (1, 768, 256), (2, 17, 33)]


@pytest.mark.parametrize("count,rows,cols", MUON_CASES)
def test_muon_against_oracle(count, rows, cols):
    import torch
    from paper_2606_03681_amd import tfm
    rng = np.random.default_rng(rows * 1000 + cols)
    W0 = rng.normal(0, 0.05, size=(count, rows, cols)).astype(np.float32)
    # the matrices live back to back in one buffer, like Q, K and V of a packed projection
    Wd = _dev(W0.reshape(-1))
    bd = torch.zeros(count * rows * cols, device="cuda")
    nel = rows * cols
    lr, m, wd = 0.02, 0.96, 0.1
    hp = tfm.tfm_muon(lr, m, wd, 1, 5)
    ws = torch.empty(tfm.muon_workspace_bytes(count, rows, cols), dtype=torch.uint8,
                     device="cuda")
    gscale = torch.tensor([0.7], device="cuda")
    W, buf = W0.astype(np.float64), np.zeros((count, rows, cols))
    for step in range(3):
        G = rng.normal(size=(count, rows, cols)).astype(np.float32)
        Gd = _dev(G.reshape(-1))
        Wprev = Wd.cpu().numpy().reshape(count, rows, cols).astype(np.float64)
        tfm.muon_step(hp, rows, cols, [Wd.data_ptr() + 4 * i * nel for i in range(count)],
                      [Gd.data_ptr() + 4 * i * nel for i in range(count)],
                      [bd.data_ptr() + 4 * i * nel for i in range(count)], gscale, ws)
        W, buf = optim.muon_step(W, 0.7 * G.astype(np.float64), buf, lr, m, wd)
        torch.cuda.synchronize()
        gW = Wd.cpu().numpy().reshape(count, rows, cols).astype(np.float64)
        gb = bd.cpu().numpy().reshape(count, rows, cols).astype(np.float64)
        eW, eb = nerr(gW, W), nerr(gb, buf)
        # the orthogonalised update alone, from this step's change of the GPU's own weights
        k = lr * max(1.0, rows / cols) ** 0.5
        O_gpu = (Wprev * (1 - lr * wd) - gW) / k
        U = (1 - m) * 0.7 * G + m * gb
        O_ref = np.stack([optim.newton_schulz(u) for u in U])
        eO = nerr(O_gpu, O_ref)
        _say(f"[optim] muon {count}x{rows}x{cols} step {step}: W {eW:.3g} buf {eb:.3g} "
             f"update {eO:.3g}")
        assert eW <= TOL and eb <= TOL
        assert eO <= TOL  # the update itself, recovered through a float32 difference


@pytest.mark.parametrize("count,rows,cols", [(1, 1, 1), (3, 1, 40), (2, 40, 1), (1, 300, 7)])
def test_muon_degenerate_shapes(count, rows, cols):
    """1 x 1 matrices (the map drives a scalar toward sign), single rows and columns (the map
    normalises a vector), and a strongly tall matrix."""
    import torch
    from paper_2606_03681_amd import tfm
    rng = np.random.default_rng(count * 100 + rows + cols)
    W0 = rng.normal(0, 0.05, size=(count, rows, cols)).astype(np.float32)
    G = rng.normal(size=(count, rows, cols)).astype(np.float32)
    Wd, Gd = _dev(W0.reshape(-1)), _dev(G.reshape(-1))
    bd = torch.zeros(count * rows * cols, device="cuda")
    nel = rows * cols
    hp = tfm.tfm_muon(0.02, 0.95, 0.1, 1, 5)
    ws = torch.empty(tfm.muon_workspace_bytes(count, rows, cols), dtype=torch.uint8,
                     device="cuda")
    tfm.muon_step(hp, rows, cols, [Wd.data_ptr() + 4 * i * nel for i in range(count)],
                  [Gd.data_ptr() + 4 * i * nel for i in range(count)],
                  [bd.data_ptr() + 4 * i * nel for i in range(count)], None, ws)
    W, _ = optim.muon_step(W0.astype(np.float64), G.astype(np.float64),
                           np.zeros((count, rows, cols)), 0.02, 0.95, 0.1)
    torch.cuda.synchronize()
    got = Wd.cpu().numpy().reshape(count, rows, cols).astype(np.float64)
    e = nerr(got, W)
    _say(f"[optim] muon degenerate {count}x{rows}x{cols}: W {e:.3g}")
    assert e <= TOL


def test_sfadamw_long_warmup_schedule_scalars():
    """The step scalars come from a closed form of sum_{i<=t} s_i^2: check them deep into and
    past a long warm-up against the oracle run step by step."""
    import torch
    from paper_2606_03681_amd import tfm
    rng = np.random.default_rng(12)
    n = 64
    y0 = rng.normal(size=n).astype(np.float32)
    hp = tfm.tfm_sfadamw(3e-3, 0.9, 0.999, 1e-8, 0.01, 40)
    y, z, v = _dev(y0), _dev(y0), torch.zeros(n, device="cuda")
    opt = optim.ScheduleFreeAdamW(y0.astype(np.float64), 3e-3, weight_decay=0.01, warmup=40)
    for t in range(1, 61):
        g = rng.normal(size=n).astype(np.float32)
        tfm.sfadamw_step(hp, t, [(0, n)], y, z, v, _dev(g))
        ref = opt.step(g.astype(np.float64))
    torch.cuda.synchronize()
    e = nerr(y.cpu().numpy(), ref)
    _say(f"[optim] sfadamw 60 steps, warm-up 40: y {e:.3g}")
    assert e <= TOL
