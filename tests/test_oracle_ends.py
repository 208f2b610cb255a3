"""Pins of the float64 oracle of the stack's two ends (feature/target encoders, decoder and
cross-entropy loss) against facts fixed by the paper and by the mathematics: the co-occurrence
property of the (0, 1, 3) grouping that App. "Repeated Feature Grouping" states, the label-free
test rows of the target fill (Fig. 3 caption), closed forms of the loss, finite differences of
every gradient, and an independent construction from torch library routines with autograd."""

import itertools
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import ends


def _setup(seed=3, B=3, R=9, C=6, F_=6, E=8, G=3, Hd=12, K=5, n_train=(5, 3, 7),
           n_feat=(6, 2, 4), n_class=(5, 2, 3), offsets=(0, 1, 3)):
    rng = np.random.default_rng(seed)
    x = rng.normal(size=(B, R, F_))
    y = np.stack([rng.integers(0, n_class[b], R) for b in range(B)]).astype(np.float64)
    P = ends.unpack_ends_params(rng.normal(0, 0.5, ends.ends_param_count(E, G, Hd, K)),
                                E, G, Hd, K)
    return dict(x=x, y=y, n_train=np.array(n_train), n_feat=np.array(n_feat),
                n_class=np.array(n_class), C=C, offsets=offsets, P=P, E=E, G=G, Hd=Hd, K=K,
                rng=rng)


# ---------------------------------------------------------------------------------------------
# Repeated feature grouping
# ---------------------------------------------------------------------------------------------

@pytest.mark.parametrize("m", [7, 8, 11, 20, 100])
def test_grouping_013_pairs_cooccur_at_most_once(m):
    """For m >= 7 columns no two columns share more than one (0, 1, 3) group, every column is
    in exactly three groups and group j starts at column j."""
    idx = ends.group_columns(m, (0, 1, 3))
    assert idx.shape == (m, 3)
    assert np.array_equal(idx[:, 0], np.arange(m))
    assert np.array_equal(np.bincount(idx.ravel(), minlength=m), np.full(m, 3))
    seen = {}
    for j, g in enumerate(idx):
        assert len(set(g.tolist())) == 3
        for p in itertools.combinations(sorted(g.tolist()), 2):
            assert p not in seen, (p, seen.get(p), j)
            seen[p] = j
    assert len(seen) == 3 * m


def test_grouping_small_tables_wrap_and_repeat():
    """Below 7 columns the shifts wrap onto repeated columns: m = 2 gives (j, j+1, j+1)."""
    assert ends.group_columns(2, (0, 1, 3)).tolist() == [[0, 1, 1], [1, 0, 0]]
    assert ends.group_columns(1, (0, 1, 3)).tolist() == [[0, 0, 0]]
    assert ends.group_columns(5, (0, 1, 3))[4].tolist() == [4, 0, 2]


def test_group_size_one_is_a_per_feature_linear_map():
    s = _setup(G=1, offsets=(0,))
    X, mask, _ = ends.encode_forward(s["x"], s["y"], s["n_train"], s["n_feat"], s["C"],
                                     s["offsets"], s["P"])
    for b in range(3):
        m = s["n_feat"][b]
        want = s["x"][b, :, :m, None] * s["P"]["W_fe"][:, 0] + s["P"]["b_fe"]
        assert np.allclose(X[b, :, :m], want, rtol=1e-14, atol=1e-14)
        assert np.all(X[b, :, m:s["C"]] == 0)
        assert mask[b].tolist() == [True] * m + [False] * (s["C"] - m) + [True]


def test_encoder_uses_the_shifted_columns():
    """Cell j of a row equals the encoder applied to the values of columns (j+o) mod m: moving
    one column's value changes exactly the cells whose groups contain it."""
    s = _setup()
    b, r, col = 0, 2, 4
    X0, _, _ = ends.encode_forward(s["x"], s["y"], s["n_train"], s["n_feat"], s["C"],
                                   s["offsets"], s["P"])
    x = s["x"].copy()
    x[b, r, col] += 1.0
    X1, _, _ = ends.encode_forward(x, s["y"], s["n_train"], s["n_feat"], s["C"], s["offsets"],
                                   s["P"])
    m = s["n_feat"][b]
    changed = sorted(j for j in range(s["C"] + 1) if not np.array_equal(X0[b, r, j], X1[b, r, j]))
    assert changed == sorted({(col - o) % m for o in s["offsets"]})
    # the change in cell j is the encoder weight column of the shift that hits `col`
    for j in changed:
        k = [i for i, o in enumerate(s["offsets"]) if (j + o) % m == col]
        assert np.allclose(X1[b, r, j] - X0[b, r, j], s["P"]["W_fe"][:, k].sum(axis=1))
    diff = np.abs(X1 - X0).sum(axis=-1)
    diff[b, r] = 0
    assert np.all(diff == 0)


# ---------------------------------------------------------------------------------------------
# Target encoder and the train-mean fill
# ---------------------------------------------------------------------------------------------

def test_test_row_target_cells_ignore_test_labels_and_equal_train_mean_encoding():
    s = _setup()
    X0, _, _ = ends.encode_forward(s["x"], s["y"], s["n_train"], s["n_feat"], s["C"],
                                   s["offsets"], s["P"])
    y = s["y"].copy()
    for b in range(3):
        y[b, s["n_train"][b]:] = 1000.0 + b
    X1, _, _ = ends.encode_forward(s["x"], y, s["n_train"], s["n_feat"], s["C"], s["offsets"],
                                   s["P"])
    assert np.array_equal(X0, X1)
    C = s["C"]
    for b in range(3):
        n = s["n_train"][b]
        # an affine map commutes with the mean: the test rows carry the mean train encoding
        assert np.allclose(X0[b, n:, C], X0[b, :n, C].mean(axis=0), rtol=1e-13, atol=1e-13)
        assert np.allclose(X0[b, :n, C],
                           s["y"][b, :n, None] * s["P"]["W_te"] + s["P"]["b_te"])


def test_encoder_rejects_bad_counts():
    s = _setup()
    with pytest.raises(ValueError):
        ends.encode_forward(s["x"], s["y"], s["n_train"], np.array([7, 2, 4]), s["C"],
                            s["offsets"], s["P"])
    with pytest.raises(ValueError):
        ends.encode_forward(s["x"], s["y"], np.array([0, 3, 7]), s["n_feat"], s["C"],
                            s["offsets"], s["P"])


# ---------------------------------------------------------------------------------------------
# Decoder and loss: closed forms
# ---------------------------------------------------------------------------------------------

def _Y(s, seed=5):
    rng = np.random.default_rng(seed)
    return rng.normal(size=(len(s["n_train"]), s["x"].shape[1], s["C"] + 1, s["E"]))


@pytest.mark.parametrize("mode", ["target", "mean"])
def test_zero_output_layer_gives_log_class_count(mode):
    """Constant logits give a uniform softmax over each dataset's classes: the loss is the mean
    over test rows of log(n_class) and dY vanishes (the output layer's weight is zero)."""
    s = _setup()
    P = {k: v.copy() for k, v in s["P"].items()}
    P["W_d2"][:] = 0
    P["b_d2"][:] = 0.7
    Y = _Y(s)
    loss, dY, dP, _ = ends.decode_loss(Y, s["y"], s["n_train"], s["n_feat"], s["n_class"],
                                       s["C"], P, mode)
    R = Y.shape[1]
    cnt = R - s["n_train"]
    want = float((cnt * np.log(s["n_class"])).sum() / cnt.sum())
    assert math.isclose(loss, want, rel_tol=1e-14)
    assert np.all(dY == 0)
    assert np.all(dP["W_d1"] == 0) and np.all(dP["b_d1"] == 0)


def test_single_class_dataset_contributes_zero_loss_and_gradient():
    s = _setup(n_class=(1, 1, 1))
    Y = _Y(s)
    loss, dY, dP, _ = ends.decode_loss(Y, s["y"], s["n_train"], s["n_feat"], s["n_class"],
                                       s["C"], s["P"], "mean")
    assert loss == 0.0
    assert np.all(dY == 0)
    assert all(np.all(v == 0) for v in dP.values())


def test_masked_classes_are_inert_and_softmax_gradient_rows_sum_to_zero():
    s = _setup()
    Y = _Y(s)
    P = {k: v.copy() for k, v in s["P"].items()}
    loss0, dY0, dP0, logits = ends.decode_loss(Y, s["y"], s["n_train"], s["n_feat"],
                                               s["n_class"], s["C"], P, "target")
    kmax = int(s["n_class"].max())
    P["b_d2"][kmax:] += 50.0
    P["W_d2"][kmax:] *= -3.0
    loss1, dY1, dP1, _ = ends.decode_loss(Y, s["y"], s["n_train"], s["n_feat"], s["n_class"],
                                          s["C"], P, "target")
    assert loss0 == loss1 and np.array_equal(dY0, dY1)
    assert np.all(dP0["W_d2"][kmax:] == 0) and np.all(dP0["b_d2"][kmax:] == 0)
    # the logits' gradient (softmax - one-hot) sums to zero per row, so b_d2's gradient sums to 0
    assert abs(dP0["b_d2"].sum()) < 1e-15
    assert logits.shape == ((Y.shape[1] - s["n_train"]).sum(), s["K"])


def test_mean_decoder_ignores_padding_and_train_rows_and_is_cell_permutation_invariant():
    s = _setup()
    Y = _Y(s)
    args = (s["y"], s["n_train"], s["n_feat"], s["n_class"], s["C"], s["P"], "mean")
    loss, dY, _, lg = ends.decode_loss(Y, *args)
    Y2 = Y.copy()
    for b in range(3):
        m, n = s["n_feat"][b], s["n_train"][b]
        Y2[b, :, m:] = 99.0                  # padding cells and the target cell
        Y2[b, :n] = -7.0                     # train rows
        perm = np.random.default_rng(b).permutation(m)
        Y2[b, n:, :m] = Y[b, n:][:, perm]
    loss2, dY2, _, lg2 = ends.decode_loss(Y2, *args)
    assert np.allclose(lg, lg2, rtol=1e-13, atol=1e-13) and math.isclose(loss, loss2,
                                                                        rel_tol=1e-13)
    for b in range(3):
        m, n = s["n_feat"][b], s["n_train"][b]
        assert np.all(dY[b, :n] == 0) and np.all(dY[b, :, m:] == 0)
        # every feature cell of a test row gets the same share of the decoder input's gradient
        assert np.allclose(dY[b, n:, :m], dY[b, n:, :1])


def test_target_decoder_reads_only_the_target_cell_of_test_rows():
    s = _setup()
    Y = _Y(s)
    args = (s["y"], s["n_train"], s["n_feat"], s["n_class"], s["C"], s["P"], "target")
    loss, dY, _, _ = ends.decode_loss(Y, *args)
    Y2 = Y.copy()
    Y2[:, :, :s["C"]] = 5.0
    for b in range(3):
        Y2[b, :s["n_train"][b]] = 5.0
    assert ends.decode_loss(Y2, *args)[0] == loss
    assert np.all(dY[:, :, :s["C"]] == 0)


# ---------------------------------------------------------------------------------------------
# Finite differences
# ---------------------------------------------------------------------------------------------

def _fd(f, arr, h=1e-6):
    g = np.zeros_like(arr)
    for idx in np.ndindex(arr.shape):
        old = arr[idx]
        arr[idx] = old + h
        lp = f()
        arr[idx] = old - h
        lm = f()
        arr[idx] = old
        g[idx] = (lp - lm) / (2 * h)
    return g


@pytest.mark.parametrize("mode", ["target", "mean"])
def test_decoder_finite_differences(mode):
    s = _setup(B=2, R=6, n_train=(3, 4), n_feat=(6, 3), n_class=(5, 3))
    Y = _Y(s)
    P = s["P"]

    def f():
        return ends.decode_loss(Y, s["y"], s["n_train"], s["n_feat"], s["n_class"], s["C"], P,
                                mode)[0]

    _, dY, dP, _ = ends.decode_loss(Y, s["y"], s["n_train"], s["n_feat"], s["n_class"], s["C"],
                                    P, mode)
    for k in ("W_d1", "b_d1", "W_d2", "b_d2"):
        assert np.allclose(_fd(f, P[k]), dP[k], rtol=1e-6, atol=1e-8), k
    assert np.allclose(_fd(f, Y), dY, rtol=1e-6, atol=1e-8)


def test_encoder_finite_differences():
    s = _setup(B=2, R=6, n_train=(3, 4), n_feat=(6, 3), n_class=(5, 3))
    P = s["P"]
    dX = np.random.default_rng(9).normal(size=(2, 6, s["C"] + 1, s["E"]))

    def f():
        X, _, _ = ends.encode_forward(s["x"], s["y"], s["n_train"], s["n_feat"], s["C"],
                                      s["offsets"], P)
        return float((X * dX).sum())

    _, _, cache = ends.encode_forward(s["x"], s["y"], s["n_train"], s["n_feat"], s["C"],
                                      s["offsets"], P)
    d = ends.encode_backward(dX, cache)
    for k in ("W_fe", "b_fe", "W_te", "b_te"):
        assert np.allclose(_fd(f, P[k]), d[k], rtol=1e-7, atol=1e-8), k


def test_param_packing_roundtrip_and_count():
    E, G, Hd, K = 8, 5, 12, 10
    n = ends.ends_param_count(E, G, Hd, K)
    assert n == E * G + 3 * E + Hd * E + Hd + K * Hd + K
    v = np.arange(n, dtype=np.float64)
    assert np.array_equal(ends.pack_ends_params(ends.unpack_ends_params(v, E, G, Hd, K)), v)
    with pytest.raises(ValueError):
        ends.unpack_ends_params(np.zeros(n + 1), E, G, Hd, K)


# ---------------------------------------------------------------------------------------------
# Independent construction from torch library routines
# ---------------------------------------------------------------------------------------------

def _torch_ends(s, Y, mode):
    """Encoders by gather + F.linear, decoder by F.linear/F.gelu and F.cross_entropy with the
    absent classes masked to -inf; gradients from autograd."""
    P = {k: torch.tensor(v, requires_grad=True) for k, v in s["P"].items()}
    x = torch.tensor(s["x"])
    B, R = s["y"].shape
    C = s["C"]
    Xs = []
    for b in range(B):
        m, n = int(s["n_feat"][b]), int(s["n_train"][b])
        cols = (torch.arange(m)[:, None] + torch.tensor(s["offsets"])[None, :]) % m
        feat = F.linear(x[b][:, cols], P["W_fe"], P["b_fe"])                  # (R, m, E)
        yv = torch.tensor(s["y"][b])
        yv = torch.cat([yv[:n], yv[:n].mean().expand(R - n)])
        tgt = F.linear(yv[:, None], P["W_te"][:, None], P["b_te"])            # (R, E)
        pad = torch.zeros(R, C - m, s["E"], dtype=torch.float64)
        Xs.append(torch.cat([feat, pad, tgt[:, None]], dim=1))
    X = torch.stack(Xs)
    Yt = torch.tensor(Y, requires_grad=True)
    losses = []
    for b in range(B):
        m, n = int(s["n_feat"][b]), int(s["n_train"][b])
        z = Yt[b, n:, C] if mode == "target" else Yt[b, n:, :m].mean(dim=1)
        lg = F.linear(F.gelu(F.linear(z, P["W_d1"], P["b_d1"])), P["W_d2"], P["b_d2"])
        lg = lg.masked_fill(torch.arange(s["K"]) >= int(s["n_class"][b]), float("-inf"))
        lab = torch.tensor(s["y"][b, n:], dtype=torch.long)
        losses.append(F.cross_entropy(lg, lab, reduction="sum"))
    loss = torch.stack(losses).sum() / float((R - s["n_train"]).sum())
    dX = torch.tensor(np.random.default_rng(4).normal(size=X.shape))
    (loss + (X * dX).sum()).backward()
    return X.detach().numpy(), loss.item(), Yt.grad.numpy(), {k: v.grad.numpy()
                                                              for k, v in P.items()}, dX.numpy()


@pytest.mark.parametrize("mode", ["target", "mean"])
def test_ends_match_torch_autograd(mode):
    s = _setup(seed=8, B=3, R=10, C=7, F_=7, E=8, G=5, Hd=12, K=6, n_train=(6, 2, 9),
               n_feat=(7, 3, 5), n_class=(6, 2, 4), offsets=(0, 1, 3, 7, 12))
    Y = _Y(s, seed=12)
    Xt, losst, dYt, gt, dX = _torch_ends(s, Y, mode)
    X, _, cache = ends.encode_forward(s["x"], s["y"], s["n_train"], s["n_feat"], s["C"],
                                      s["offsets"], s["P"])
    assert np.allclose(X, Xt, rtol=1e-13, atol=1e-13)
    loss, dY, dP, _ = ends.decode_loss(Y, s["y"], s["n_train"], s["n_feat"], s["n_class"],
                                       s["C"], s["P"], mode)
    assert math.isclose(loss, losst, rel_tol=1e-13)
    assert np.allclose(dY, dYt, rtol=1e-12, atol=1e-14)
    dP.update(ends.encode_backward(dX, cache))
    for k in ends.ENDS_PARAM_ORDER:
        assert np.allclose(dP[k], gt[k], rtol=1e-12, atol=1e-13), k
