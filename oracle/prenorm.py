"""Float64 CPU oracle for the pre-norm block of the paper's current best record (forward and
backward).

TEST INFRASTRUCTURE ONLY, like the rest of this package: only the test-suite, the smoke check
and the CPU-baseline leg of the benchmark may import it, and it imports nothing from the GPU
package.

What it computes (paper: "Speedrunning Tabular Foundation Model Pretraining"):

* Sec. 5 "Residual Decay": the input of block i is multiplied by 0.95^i before the block
  (Tab. 5 "Residual decay 0.95"; Fig. 4 caption).
* Sec. 5 "SDPA, bf16, Learning Rate, Width" and the Fig. 4 caption: the norms move in front of
  the attention and MLP sub-layers (pre-norm).
* Sec. 5 "RMSNorm, Thinking Rows" and App. B.6: RMSNorm replaces all three LayerNorms.
* Tab. 5: embedding 256, 4 heads (head dim 64), MLP hidden 768.
* Thinking rows (App. B.6, Tab. 5): learnable E-vectors prepended along the row axis,
  broadcast over the columns and counted as train rows.  Inside a block they are ordinary train
  rows; `thinking_rows_forward/backward` give the broadcast and its gradient.

So, for one block with decay factor c (= 0.95^i) on the active cells of a dataset:

    x' = c x
    h1 = x' + A_f(RMS1(x'))            # feature-axis attention of Sec. 4.1, output projection
    h2 = h1 + A_i(RMS2(h1))            # item-axis attention over the train prefix
    y  = h2 + W2 GELU(W1 RMS3(h2) + b1) + b2

with RMS(u) = g * u / sqrt(mean(u^2) + eps).

Readings where the paper is silent (listed in the design doc as well): RMSNorm has a weight and no
bias, eps = 1e-6, mean over the E features; "lower precision" describes the paper's autocast
setting and is not a different function; every linear keeps its bias as in the baseline block;
the attention sub-layers are those of the baseline block unchanged.
"""

import numpy as np

from .layer import (_check, _feature_attention, _feature_attention_backward, _item_attention,
                    _item_attention_backward, gelu, gelu_grad, outer_sum)

RMS_EPS = 1e-6

# Packed parameter order of one pre-norm layer (row-major [out, in] weights).  This order is an
# interface shared with the C-ABI; it is written out here independently.
PRENORM_PARAM_ORDER = (
    "Wqkv_f", "bqkv_f", "Wo_f", "bo_f",
    "Wqkv_i", "bqkv_i", "Wo_i", "bo_i",
    "W1", "b1", "W2", "b2",
    "g1", "g2", "g3",
)


def prenorm_param_shapes(E, H):
    return {
        "Wqkv_f": (3 * E, E), "bqkv_f": (3 * E,), "Wo_f": (E, E), "bo_f": (E,),
        "Wqkv_i": (3 * E, E), "bqkv_i": (3 * E,), "Wo_i": (E, E), "bo_i": (E,),
        "W1": (H, E), "b1": (H,), "W2": (E, H), "b2": (E,),
        "g1": (E,), "g2": (E,), "g3": (E,),
    }


def prenorm_param_count(E, H):
    return sum(int(np.prod(s)) for s in prenorm_param_shapes(E, H).values())


def unpack_prenorm_params(flat, E, H):
    flat = np.asarray(flat, dtype=np.float64)
    shapes = prenorm_param_shapes(E, H)
    out, off = {}, 0
    for name in PRENORM_PARAM_ORDER:
        n = int(np.prod(shapes[name]))
        out[name] = flat[off:off + n].reshape(shapes[name]).copy()
        off += n
    if off != flat.size:
        raise ValueError(f"packed parameter vector has {flat.size} entries, expected {off}")
    return out


def pack_prenorm_params(p):
    return np.concatenate([np.asarray(p[name], dtype=np.float64).ravel()
                           for name in PRENORM_PARAM_ORDER])


def rmsnorm(u, g, eps=RMS_EPS):
    """RMSNorm over the last axis.  Returns (y, uhat, rstd) with uhat = u * rstd."""
    rstd = 1.0 / np.sqrt((u * u).mean(axis=-1, keepdims=True) + eps)
    uhat = u * rstd
    return g * uhat, uhat, rstd


def rmsnorm_backward(dy, uhat, rstd, g):
    """Gradient of RMSNorm: du = rstd (g dy - uhat mean(g dy uhat)); dg summed over all
    leading axes."""
    gd = g * dy
    du = rstd * (gd - uhat * (gd * uhat).mean(axis=-1, keepdims=True))
    lead = tuple(range(dy.ndim - 1))
    return du, (dy * uhat).sum(axis=lead)


def prenorm_dataset_forward(z0, P, heads, n_train, decay, eps=RMS_EPS, query_rows=None):
    """One pre-norm block for one dataset restricted to its active cells.  z0: (R, S_b, E).

    query_rows (optional): produce the output only at these rows (a row's output depends on its
    own cells and on the train rows only)."""
    R = z0.shape[0]
    qrows = np.arange(R) if query_rows is None else np.asarray(query_rows, dtype=np.int64)
    x = decay * z0
    r1, uh1, rs1 = rmsnorm(x, P["g1"], eps)
    a_f, cf = _feature_attention(r1, P, heads)
    h1 = x + a_f
    r2, uh2, rs2 = rmsnorm(h1, P["g2"], eps)
    a_i, ci = _item_attention(r2, P, heads, n_train, qrows)
    h2 = h1[qrows] + a_i
    r3, uh3, rs3 = rmsnorm(h2, P["g3"], eps)
    gpre = r3 @ P["W1"].T + P["b1"]
    u = gelu(gpre)
    y = h2 + u @ P["W2"].T + P["b2"]
    cache = {"r1": r1, "uh1": uh1, "rs1": rs1, "cf": cf, "r2": r2, "uh2": uh2, "rs2": rs2,
             "ci": ci, "r3": r3, "uh3": uh3, "rs3": rs3, "gpre": gpre, "u": u,
             "n_train": n_train, "qrows": qrows, "decay": decay, "R": R}
    return y, cache


def prenorm_dataset_backward(dy, cache, P, heads):
    """Hand-derived gradient of prenorm_dataset_forward (dy at the query rows).
    Returns (dz0, grads)."""
    g = {}
    qrows = cache["qrows"]
    # y = h2 + MLP(RMS3(h2))
    g["W2"] = outer_sum(dy, cache["u"])
    g["b2"] = dy.sum(axis=(0, 1))
    dgp = (dy @ P["W2"]) * gelu_grad(cache["gpre"])
    g["W1"] = outer_sum(dgp, cache["r3"])
    g["b1"] = dgp.sum(axis=(0, 1))
    dn3, g["g3"] = rmsnorm_backward(dgp @ P["W1"], cache["uh3"], cache["rs3"], P["g3"])
    dh2 = dy + dn3
    # h2 = h1[qrows] + A_i(RMS2(h1))
    dr2, gi = _item_attention_backward(dh2, cache["r2"], cache["ci"], P, heads,
                                       cache["n_train"], qrows)
    g.update(gi)
    dn2, g["g2"] = rmsnorm_backward(dr2, cache["uh2"], cache["rs2"], P["g2"])
    dh1 = dn2
    dh1[qrows] += dh2
    # h1 = x + A_f(RMS1(x))
    dr1, gf = _feature_attention_backward(dh1, cache["r1"], cache["cf"], P, heads)
    g.update(gf)
    dn1, g["g1"] = rmsnorm_backward(dr1, cache["uh1"], cache["rs1"], P["g1"])
    return cache["decay"] * (dh1 + dn1), g


def prenorm_layer_forward(X, params, n_train, cell_mask, heads, decay, eps=RMS_EPS):
    """Pre-norm block on the padded cell tensor X: (B, R, C+1, E); inactive cells are inert and
    their outputs are 0.  Returns (Y, cache)."""
    X = np.asarray(X, dtype=np.float64)
    n_train, cell_mask = _check(X, n_train, cell_mask, heads)
    Y = np.zeros_like(X)
    caches = []
    for b in range(X.shape[0]):
        act = np.flatnonzero(cell_mask[b])
        y, c = prenorm_dataset_forward(X[b][:, act, :], params, heads, int(n_train[b]), decay,
                                       eps)
        Y[b][:, act, :] = y
        caches.append((act, c))
    return Y, {"caches": caches, "shape": X.shape, "params": params, "heads": heads}


def prenorm_layer_backward(dY, cache):
    """Backward of prenorm_layer_forward.  dY at inactive cells is ignored."""
    dY = np.asarray(dY, dtype=np.float64)
    P, heads = cache["params"], cache["heads"]
    dX = np.zeros(cache["shape"])
    grads = {k: np.zeros_like(v) for k, v in P.items()}
    for b, (act, c) in enumerate(cache["caches"]):
        dz, g = prenorm_dataset_backward(dY[b][:, act, :], c, P, heads)
        dX[b][:, act, :] = dz
        for k in grads:
            grads[k] += g[k]
    return dX, grads


def prenorm_stack_forward(X, params_list, n_train, cell_mask, heads, decay_base=0.95,
                          eps=RMS_EPS):
    """Blocks applied in sequence; block i scales its input by decay_base ** i."""
    caches = []
    for i, P in enumerate(params_list):
        X, c = prenorm_layer_forward(X, P, n_train, cell_mask, heads, decay_base ** i, eps)
        caches.append(c)
    return X, caches


def prenorm_stack_backward(dY, caches):
    grads = [None] * len(caches)
    for i in range(len(caches) - 1, -1, -1):
        dY, grads[i] = prenorm_layer_backward(dY, caches[i])
    return dY, grads


def thinking_rows_forward(X, table, cell_mask):
    """Prepend the thinking-row table (T, E) to every active column of X (B, R, C+1, E):
    returns (B, T + R, C+1, E); inactive cells stay 0 in the new rows."""
    X = np.asarray(X, dtype=np.float64)
    B, R, S, E = X.shape
    T = table.shape[0]
    out = np.zeros((B, T + R, S, E))
    out[:, T:] = X
    m = np.asarray(cell_mask, dtype=bool)
    for b in range(B):
        out[b, :T][:, m[b], :] = table[:, None, :]
    return out


def thinking_rows_backward(dOut, cell_mask, T):
    """Gradient of thinking_rows_forward: (dX, dtable), dtable summed over every active cell of
    the T prepended rows."""
    m = np.asarray(cell_mask, dtype=bool)
    dtable = np.zeros((T, dOut.shape[-1]))
    for b in range(dOut.shape[0]):
        dtable += dOut[b, :T][:, m[b], :].sum(axis=1)
    return dOut[:, T:].copy(), dtable
