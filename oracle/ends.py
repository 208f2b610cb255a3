"""Float64 CPU oracle for the two ends of the stack: the feature and target encoders in front of
the first block, and the decoder with the cross-entropy loss behind the last one.

TEST INFRASTRUCTURE ONLY, like the rest of this package: only the test-suite, the smoke check
and the CPU-baseline leg of the benchmark may import it, and it imports nothing from the GPU
package.

What it computes (paper: "Speedrunning Tabular Foundation Model Pretraining"):

* Fig. 3 caption: the input features are encoded by a feature encoder, the labels by a target
  encoder whose test rows carry the mean over the train rows, the two streams are merged (the
  feature cells then the target cell of each row) and, after the stack, the test rows' outputs
  go to the decoder.
* App. "Repeated Feature Grouping": with m feature columns, cell j encodes the columns at
  positions (j + o) mod m for o in the group's offsets, (0, 1, 3) for groups of three; Tab. 5
  uses groups of five, whose offsets the paper does not give (the caller passes them).
* Fig. 4 caption and App. "Autoresearch": the current best record decodes the mean over the
  feature cells of each test row instead of its target cell.

Readings where the paper is silent (listed in the design doc as well):

* the feature encoder is one linear map from the G grouped values to E (weight [E][G] and a
  bias), shared by all cells; a table with m features has m feature cells, cells m .. C-1 are
  padding;
* the target encoder is a linear map from the label value (a float) to E; a test row's value
  is the mean of the train rows' labels, so its encoding is the mean of the train encodings;
* the decoder is Linear(E, Hd), exact-erf GELU, Linear(Hd, K); a dataset with k classes uses
  the first k logits (the rest are excluded from its softmax);
* the loss is the cross entropy of the test rows' labels, averaged over every test row of the
  batch.
"""

import numpy as np

from .layer import gelu, gelu_grad

# Packed parameter order of the two ends (row-major [out, in] weights).  This order is an
# interface shared with the C-ABI; it is written out here independently.
ENDS_PARAM_ORDER = ("W_fe", "b_fe", "W_te", "b_te", "W_d1", "b_d1", "W_d2", "b_d2")


def ends_param_shapes(E, G, Hd, K):
    return {"W_fe": (E, G), "b_fe": (E,), "W_te": (E,), "b_te": (E,),
            "W_d1": (Hd, E), "b_d1": (Hd,), "W_d2": (K, Hd), "b_d2": (K,)}


def ends_param_count(E, G, Hd, K):
    return sum(int(np.prod(s)) for s in ends_param_shapes(E, G, Hd, K).values())


def unpack_ends_params(flat, E, G, Hd, K):
    flat = np.asarray(flat, dtype=np.float64)
    shapes = ends_param_shapes(E, G, Hd, K)
    out, off = {}, 0
    for name in ENDS_PARAM_ORDER:
        n = int(np.prod(shapes[name]))
        out[name] = flat[off:off + n].reshape(shapes[name]).copy()
        off += n
    if off != flat.size:
        raise ValueError(f"packed ends vector has {flat.size} entries, expected {off}")
    return out


def pack_ends_params(p):
    return np.concatenate([np.asarray(p[k], dtype=np.float64).ravel() for k in ENDS_PARAM_ORDER])


def group_columns(m, offsets):
    """[m][G] column indices of the m groups: group j holds columns (j + o) mod m."""
    return np.array([[(j + o) % m for o in offsets] for j in range(m)], dtype=np.int64)


def encode_forward(x, y, n_train, n_feat, C, offsets, P):
    """x: [B][R][>= max n_feat] feature values, y: [B][R] labels.  Returns the stack input
    X [B][R][C+1][E], its cell mask [B][C+1] and the cache of the backward pass."""
    x = np.asarray(x, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    B, R = y.shape
    E = P["b_fe"].shape[0]
    X = np.zeros((B, R, C + 1, E))
    mask = np.zeros((B, C + 1), dtype=bool)
    groups, targets = [], []
    for b in range(B):
        m, n = int(n_feat[b]), int(n_train[b])
        if not (1 <= m <= C) or not (1 <= n <= R):
            raise ValueError("n_feat must lie in [1, C] and n_train in [1, R]")
        idx = group_columns(m, offsets)
        g = x[b][:, idx]                                  # [R][m][G]
        X[b, :, :m] = g @ P["W_fe"].T + P["b_fe"]
        t = y[b].copy()
        t[n:] = y[b, :n].mean()
        X[b, :, C] = t[:, None] * P["W_te"][None, :] + P["b_te"]
        mask[b, :m] = True
        mask[b, C] = True
        groups.append(g)
        targets.append(t)
    return X, mask, dict(groups=groups, targets=targets, n_feat=np.asarray(n_feat), C=C)


def encode_backward(dX, cache):
    """Parameter gradients of the encoders for the upstream gradient dX of the stack input."""
    dX = np.asarray(dX, dtype=np.float64)
    C = cache["C"]
    E = dX.shape[-1]
    G = cache["groups"][0].shape[-1]
    d = {"W_fe": np.zeros((E, G)), "b_fe": np.zeros(E), "W_te": np.zeros(E), "b_te": np.zeros(E)}
    for b, (g, t) in enumerate(zip(cache["groups"], cache["targets"])):
        m = int(cache["n_feat"][b])
        dc = dX[b, :, :m]                                 # [R][m][E]
        d["W_fe"] += np.einsum("rje,rjg->eg", dc, g)
        d["b_fe"] += dc.sum(axis=(0, 1))
        d["W_te"] += (dX[b, :, C] * t[:, None]).sum(axis=0)
        d["b_te"] += dX[b, :, C].sum(axis=0)
    return d


def decode_tokens(Y, n_train, n_feat, C, mode):
    """Decoder input of every test row, in (dataset, row) order: the target cell's output, or
    the mean of the feature cells' outputs."""
    Z = []
    for b in range(Y.shape[0]):
        n, m = int(n_train[b]), int(n_feat[b])
        if mode == "target":
            Z.append(Y[b, n:, C])
        else:
            Z.append(Y[b, n:, :m].mean(axis=1))
    return np.concatenate(Z, axis=0)


def decode_loss(Y, y, n_train, n_feat, n_class, C, P, mode):
    """Loss of the batch and its gradients: returns (loss, dY, dP, logits)."""
    Y = np.asarray(Y, dtype=np.float64)
    B, R = Y.shape[:2]
    K = P["b_d2"].shape[0]
    Z = decode_tokens(Y, n_train, n_feat, C, mode)       # [T][E]
    lab = np.concatenate([np.asarray(y[b][int(n_train[b]):]) for b in range(B)]).astype(np.int64)
    ncls = np.concatenate([np.full(R - int(n_train[b]), int(n_class[b])) for b in range(B)])
    T = Z.shape[0]
    h1 = Z @ P["W_d1"].T + P["b_d1"]
    a = gelu(h1)
    logits = a @ P["W_d2"].T + P["b_d2"]
    valid = np.arange(K)[None, :] < ncls[:, None]
    lg = np.where(valid, logits, -np.inf)
    mx = lg.max(axis=1, keepdims=True)
    e = np.where(valid, np.exp(lg - mx), 0.0)
    sm = e / e.sum(axis=1, keepdims=True)
    loss = float((-(np.log(sm[np.arange(T), lab]))).sum() / T)
    dlog = sm.copy()
    dlog[np.arange(T), lab] -= 1.0
    dlog /= T
    dP = {"W_d2": dlog.T @ a, "b_d2": dlog.sum(axis=0)}
    da = dlog @ P["W_d2"]
    dh1 = da * gelu_grad(h1)
    dP["W_d1"] = dh1.T @ Z
    dP["b_d1"] = dh1.sum(axis=0)
    dZ = dh1 @ P["W_d1"]
    dY = np.zeros_like(Y)
    row = 0
    for b in range(B):
        n, m = int(n_train[b]), int(n_feat[b])
        cnt = R - n
        if mode == "target":
            dY[b, n:, C] = dZ[row:row + cnt]
        else:
            dY[b, n:, :m] = dZ[row:row + cnt][:, None, :] / m
        row += cnt
    return loss, dY, dP, logits
