"""Float64 CPU oracle for the two-axis tabular transformer layer (forward and backward).

TEST INFRASTRUCTURE ONLY.  This module is the slow, obviously-correct reference that the GPU
path is checked against.  Only the test-suite, the smoke check and the CPU-baseline leg of the
benchmark may import it.  It imports nothing from the GPU package and the GPU package imports
nothing from it.

What it computes (paper: "Speedrunning Tabular Foundation Model Pretraining"):

* Section 4.1 (baseline) and the Fig. 3 caption: every block applies feature-axis attention,
  a norm, sample-axis (item-axis) attention, a norm, an MLP and a norm; the norms are post-norm
  LayerNorms.  Tab. 5 gives 6 heads, embedding 192 for the baseline.
* The item-axis attention lets every row attend only to the labelled (train) rows, which form a
  prefix of the rows of each dataset (the train/test split that the Fig. 3 caption describes,
  and that the thinking-row discussion in App. B.6 relies on when it counts prepended rows as
  part of the train portion).

Readings where the paper is silent (each is listed in the design doc as well):

* residual connection around each of the three sub-layers, followed by the norm (post-norm);
* two independent attention parameter sets (feature axis, item axis), each with a packed
  Q|K|V projection [3E, E] + bias and an output projection [E, E] + bias;
* every linear has a bias; LayerNorm is affine, eps = 1e-5, biased variance;
* GELU is the exact erf form, G * Phi(G);
* attention scale 1/sqrt(d), no dropout, no positional encoding;
* train rows attend to all train rows including themselves; a test row attends to the train
  rows only;
* feature-axis attention is full bidirectional attention among the active cells of a row
  (the target cell included); inactive (padded) cells are inert: they are neither keys nor
  queries, their outputs are 0 and they receive no gradient.

The arithmetic is plain numpy float64 with library matmuls; there is no blocking, fusion or
reordering beyond the definitions.  The softmax is recomputed from Q and K in the backward
pass exactly as in the forward pass.
"""

import math

import numpy as np
from scipy.special import erf

LN_EPS = 1e-5

# Packed parameter order of one layer (row-major [out, in] weights, nn.Linear convention).
# This order is an interface shared with the C-ABI; it is written out here independently.
PARAM_ORDER = (
    "Wqkv_f", "bqkv_f", "Wo_f", "bo_f",
    "Wqkv_i", "bqkv_i", "Wo_i", "bo_i",
    "W1", "b1", "W2", "b2",
    "g1", "be1", "g2", "be2", "g3", "be3",
)


def param_shapes(E, H):
    """Shapes of the per-layer parameters, in packed order."""
    return {
        "Wqkv_f": (3 * E, E), "bqkv_f": (3 * E,), "Wo_f": (E, E), "bo_f": (E,),
        "Wqkv_i": (3 * E, E), "bqkv_i": (3 * E,), "Wo_i": (E, E), "bo_i": (E,),
        "W1": (H, E), "b1": (H,), "W2": (E, H), "b2": (E,),
        "g1": (E,), "be1": (E,), "g2": (E,), "be2": (E,), "g3": (E,), "be3": (E,),
    }


def param_count(E, H):
    return sum(int(np.prod(s)) for s in param_shapes(E, H).values())


def unpack_params(flat, E, H):
    """Split a packed parameter vector into a dict of float64 arrays."""
    flat = np.asarray(flat, dtype=np.float64)
    shapes = param_shapes(E, H)
    out, off = {}, 0
    for name in PARAM_ORDER:
        n = int(np.prod(shapes[name]))
        out[name] = flat[off:off + n].reshape(shapes[name]).copy()
        off += n
    if off != flat.size:
        raise ValueError(f"packed parameter vector has {flat.size} entries, expected {off}")
    return out


def pack_params(p):
    return np.concatenate([np.asarray(p[name], dtype=np.float64).ravel() for name in PARAM_ORDER])


# ---------------------------------------------------------------------------------------------
# Elementary pieces
# ---------------------------------------------------------------------------------------------

def gelu(g):
    """Exact GELU: g * Phi(g) with Phi the standard normal CDF (erf form)."""
    return g * 0.5 * (1.0 + erf(g / math.sqrt(2.0)))


def gelu_grad(g):
    """d/dg [g Phi(g)] = Phi(g) + g phi(g)."""
    cdf = 0.5 * (1.0 + erf(g / math.sqrt(2.0)))
    pdf = np.exp(-0.5 * g * g) / math.sqrt(2.0 * math.pi)
    return cdf + g * pdf


def layernorm(u, gamma, beta, eps=LN_EPS):
    """LayerNorm over the last axis with the biased variance.  Returns (y, xhat, rstd)."""
    mu = u.mean(axis=-1, keepdims=True)
    var = ((u - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (u - mu) * rstd
    return gamma * xhat + beta, xhat, rstd


def layernorm_backward(dy, xhat, rstd, gamma):
    """Gradient of LayerNorm.  Returns (du, dgamma, dbeta); dgamma/dbeta summed over all
    leading axes."""
    g = dy * gamma
    du = rstd * (g - g.mean(axis=-1, keepdims=True)
                 - xhat * (g * xhat).mean(axis=-1, keepdims=True))
    lead = tuple(range(dy.ndim - 1))
    return du, (dy * xhat).sum(axis=lead), dy.sum(axis=lead)


def softmax(s):
    m = s.max(axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=-1, keepdims=True)


def attention_probs(q, k):
    """Scaled dot-product attention weights; q: (..., Lq, d), k: (..., Lk, d)."""
    d = q.shape[-1]
    return softmax((q @ np.swapaxes(k, -1, -2)) / math.sqrt(d))


def attention(q, k, v):
    """softmax(q k^T / sqrt(d)) v over the last two axes."""
    return attention_probs(q, k) @ v


def attention_backward(q, k, v, do):
    """Gradient of attention(q, k, v) given the output gradient do.  The probabilities are
    recomputed from q and k.  With D_r = <dO_r, O_r>:
        dV = P^T dO,  dP = dO V^T,  dS = P (dP - D),  dQ = tau dS K,  dK = tau dS^T Q."""
    tau = 1.0 / math.sqrt(q.shape[-1])
    p = attention_probs(q, k)
    o = p @ v
    dv = np.swapaxes(p, -1, -2) @ do
    dp = do @ np.swapaxes(v, -1, -2)
    dsum = (do * o).sum(axis=-1, keepdims=True)
    ds = p * (dp - dsum)
    dq = tau * (ds @ k)
    dk = tau * (np.swapaxes(ds, -1, -2) @ q)
    return dq, dk, dv


def outer_sum(dy, x):
    """Sum over all leading (cell) axes of the outer products dy_cell x_cell^T, i.e. the weight
    gradient of a linear layer: (..., N), (..., K) -> (N, K)."""
    return dy.reshape(-1, dy.shape[-1]).T @ x.reshape(-1, x.shape[-1])


def split_heads(x, heads):
    """(..., L, E) -> (..., heads, L, d); head j owns columns [j*d, (j+1)*d)."""
    *lead, L, E = x.shape
    d = E // heads
    x = x.reshape(*lead, L, heads, d)
    return np.moveaxis(x, -2, -3)


def merge_heads(x):
    """(..., heads, L, d) -> (..., L, heads*d)."""
    x = np.moveaxis(x, -3, -2)
    *lead, L, h, d = x.shape
    return x.reshape(*lead, L, h * d)


# ---------------------------------------------------------------------------------------------
# One dataset, active cells only
# ---------------------------------------------------------------------------------------------

def _feature_attention(z, P, heads, row_chunk=128):
    """Feature-axis self-attention: within each row, every active cell attends to every active
    cell.  z: (R, S, E).  Returns the sub-layer output (R, S, E) and the tensors its backward
    needs."""
    E = z.shape[-1]
    qkv = z @ P["Wqkv_f"].T + P["bqkv_f"]
    q, k, v = qkv[..., :E], qkv[..., E:2 * E], qkv[..., 2 * E:]
    o = np.empty_like(z)
    for r0 in range(0, z.shape[0], row_chunk):
        sl = slice(r0, r0 + row_chunk)
        o[sl] = merge_heads(attention(split_heads(q[sl], heads), split_heads(k[sl], heads),
                                      split_heads(v[sl], heads)))
    a = o @ P["Wo_f"].T + P["bo_f"]
    return a, {"q": q, "k": k, "v": v, "o": o}


def _feature_attention_backward(da, z, c, P, heads, row_chunk=128):
    E = z.shape[-1]
    g = {}
    g["Wo_f"] = outer_sum(da, c["o"])
    g["bo_f"] = da.sum(axis=(0, 1))
    do = da @ P["Wo_f"]
    dqkv = np.empty(z.shape[:-1] + (3 * E,))
    for r0 in range(0, z.shape[0], row_chunk):
        sl = slice(r0, r0 + row_chunk)
        dq, dk, dv = attention_backward(split_heads(c["q"][sl], heads),
                                        split_heads(c["k"][sl], heads),
                                        split_heads(c["v"][sl], heads),
                                        split_heads(do[sl], heads))
        dqkv[sl] = np.concatenate([merge_heads(dq), merge_heads(dk), merge_heads(dv)], axis=-1)
    g["Wqkv_f"] = outer_sum(dqkv, z)
    g["bqkv_f"] = dqkv.sum(axis=(0, 1))
    dz = dqkv @ P["Wqkv_f"]
    return dz, g


# Worker threads over the (column, head) problems of item-axis attention.  Execution only: each
# problem is computed by the same calls whatever the count (numpy releases the interpreter lock
# in its kernels, so the problems of large workloads run on several cores), and every problem
# writes its own slice of the result.
_WORKERS = 1


def set_workers(n):
    """Number of threads that evaluate item-axis attention problems (default 1)."""
    global _WORKERS
    _WORKERS = max(1, int(n))


def _each_problem(fn, S, heads):
    """fn(c, j) for every column c < S and head j < heads."""
    items = [(c, j) for c in range(S) for j in range(heads)]
    if _WORKERS <= 1 or len(items) <= 1:
        for c, j in items:
            fn(c, j)
        return
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(_WORKERS) as ex:
        for f in [ex.submit(fn, c, j) for c, j in items]:
            f.result()


def _item_attention(h, P, heads, n_train, qrows):
    """Item-axis attention down each column: every query row of a column attends to the rows
    t < n_train of the same column.  h: (R, S, E).  Keys and values are computed for the train
    rows only; queries for the rows listed in qrows (all rows in the plain layer).  Returns the
    sub-layer output at the query rows, (len(qrows), S, E)."""
    E = h.shape[-1]
    W, b = P["Wqkv_i"], P["bqkv_i"]
    zt = np.swapaxes(h, 0, 1)                                  # (S, R, E): one column per lead
    q = zt[:, qrows] @ W[:E].T + b[:E]                         # query rows
    k = zt[:, :n_train] @ W[E:2 * E].T + b[E:2 * E]            # train rows only
    v = zt[:, :n_train] @ W[2 * E:].T + b[2 * E:]
    qh, kh, vh = split_heads(q, heads), split_heads(k, heads), split_heads(v, heads)
    oh = np.empty_like(qh)                                     # (S, heads, len(qrows), d)

    def one(c, j):
        oh[c, j] = attention(qh[c, j], kh[c, j], vh[c, j])

    _each_problem(one, zt.shape[0], heads)
    o = np.swapaxes(merge_heads(oh), 0, 1)                     # (len(qrows), S, E)
    a = o @ P["Wo_i"].T + P["bo_i"]
    return a, {"q": q, "k": k, "v": v, "o": o}


def _item_attention_backward(da, h, c, P, heads, n_train, qrows):
    """Gradient of _item_attention; da: (len(qrows), S, E).  Returns dh for all R rows."""
    E = h.shape[-1]
    W = P["Wqkv_i"]
    g = {}
    g["Wo_i"] = outer_sum(da, c["o"])
    g["bo_i"] = da.sum(axis=(0, 1))
    dot = np.swapaxes(da @ P["Wo_i"], 0, 1)                    # (S, len(qrows), E)
    qh, kh, vh = split_heads(c["q"], heads), split_heads(c["k"], heads), split_heads(c["v"], heads)
    doh = split_heads(dot, heads)
    dqh, dkh, dvh = np.empty_like(qh), np.empty_like(kh), np.empty_like(vh)

    def one(cc, j):
        dqh[cc, j], dkh[cc, j], dvh[cc, j] = attention_backward(qh[cc, j], kh[cc, j], vh[cc, j],
                                                                doh[cc, j])

    _each_problem(one, dot.shape[0], heads)
    dq, dk, dv = merge_heads(dqh), merge_heads(dkh), merge_heads(dvh)
    zt = np.swapaxes(h, 0, 1)
    ztr = zt[:, :n_train]
    g["Wqkv_i"] = np.concatenate([
        outer_sum(dq, zt[:, qrows]),
        outer_sum(dk, ztr),
        outer_sum(dv, ztr)], axis=0)
    g["bqkv_i"] = np.concatenate([dq.sum(axis=(0, 1)), dk.sum(axis=(0, 1)), dv.sum(axis=(0, 1))])
    dzt = np.zeros_like(zt)
    dzt[:, qrows] += dq @ W[:E]
    dzt[:, :n_train] += dk @ W[E:2 * E] + dv @ W[2 * E:]
    return np.swapaxes(dzt, 0, 1), g


def dataset_forward(z0, P, heads, n_train, eps=LN_EPS, query_rows=None):
    """Layer forward for one dataset restricted to its active cells.  z0: (R, S_b, E).
    Returns (Y, cache).

    query_rows (optional): compute the output only at these rows.  A row's output depends on
    its own cells and on the train rows only, so this is the same arithmetic as the full layer
    restricted to those rows; Y then has shape (len(query_rows), S_b, E)."""
    R = z0.shape[0]
    qrows = np.arange(R) if query_rows is None else np.asarray(query_rows, dtype=np.int64)
    a_f, cf = _feature_attention(z0, P, heads)
    h1, xh1, rs1 = layernorm(z0 + a_f, P["g1"], P["be1"], eps)
    a_i, ci = _item_attention(h1, P, heads, n_train, qrows)
    h2, xh2, rs2 = layernorm(h1[qrows] + a_i, P["g2"], P["be2"], eps)
    gpre = h2 @ P["W1"].T + P["b1"]
    u = gelu(gpre)
    m = u @ P["W2"].T + P["b2"]
    y, xh3, rs3 = layernorm(h2 + m, P["g3"], P["be3"], eps)
    cache = {"z0": z0, "cf": cf, "h1": h1, "xh1": xh1, "rs1": rs1, "a_f": a_f,
             "ci": ci, "a_i": a_i, "h2": h2, "xh2": xh2, "rs2": rs2,
             "gpre": gpre, "u": u, "m": m, "xh3": xh3, "rs3": rs3, "n_train": n_train,
             "qrows": qrows}
    return y, cache


def dataset_backward(dy, cache, P, heads):
    """Hand-derived gradient of dataset_forward (dy at the query rows).  Returns (dz0, grads)."""
    g = {}
    qrows = cache["qrows"]
    du3, g["g3"], g["be3"] = layernorm_backward(dy, cache["xh3"], cache["rs3"], P["g3"])
    # MLP: M = GELU(H2 W1^T + b1) W2^T + b2
    g["W2"] = outer_sum(du3, cache["u"])
    g["b2"] = du3.sum(axis=(0, 1))
    dgp = (du3 @ P["W2"]) * gelu_grad(cache["gpre"])
    g["W1"] = outer_sum(dgp, cache["h2"])
    g["b1"] = dgp.sum(axis=(0, 1))
    dh2 = du3 + dgp @ P["W1"]
    du2, g["g2"], g["be2"] = layernorm_backward(dh2, cache["xh2"], cache["rs2"], P["g2"])
    dh1, gi = _item_attention_backward(du2, cache["h1"], cache["ci"], P, heads,
                                       cache["n_train"], qrows)
    g.update(gi)
    dh1[qrows] += du2
    du1, g["g1"], g["be1"] = layernorm_backward(dh1, cache["xh1"], cache["rs1"], P["g1"])
    dz_att, gf = _feature_attention_backward(du1, cache["z0"], cache["cf"], P, heads)
    g.update(gf)
    return du1 + dz_att, g


# ---------------------------------------------------------------------------------------------
# Batched layer over the padded [B, R, C+1, E] cell tensor
# ---------------------------------------------------------------------------------------------

def _check(X, n_train, cell_mask, heads):
    B, R, S, E = X.shape
    n_train = np.asarray(n_train)
    cell_mask = np.asarray(cell_mask).astype(bool)
    if E % heads:
        raise ValueError("E must be a multiple of heads")
    if n_train.shape != (B,) or cell_mask.shape != (B, S):
        raise ValueError("n_train must be [B] and cell_mask [B, C+1]")
    if np.any(n_train < 1) or np.any(n_train > R):
        raise ValueError("n_train must lie in [1, R]")
    if not np.all(cell_mask[:, S - 1]):
        raise ValueError("the target cell (index C) must be active")
    return n_train, cell_mask


def layer_forward(X, params, n_train, cell_mask, heads, eps=LN_EPS):
    """Forward of one layer on the padded cell tensor X: (B, R, C+1, E).

    params: dict of float64 arrays (see unpack_params).  n_train: (B,) ints in [1, R].
    cell_mask: (B, C+1) booleans, target cell C always active.  Inactive cells are inert and
    their outputs are 0.  Returns (Y, cache)."""
    X = np.asarray(X, dtype=np.float64)
    n_train, cell_mask = _check(X, n_train, cell_mask, heads)
    Y = np.zeros_like(X)
    caches = []
    for b in range(X.shape[0]):
        act = np.flatnonzero(cell_mask[b])
        y, c = dataset_forward(X[b][:, act, :], params, heads, int(n_train[b]), eps)
        Y[b][:, act, :] = y
        caches.append((act, c))
    return Y, {"caches": caches, "shape": X.shape, "params": params, "heads": heads}


def layer_backward(dY, cache):
    """Backward of layer_forward.  dY at inactive cells is ignored.  Returns (dX, grads) with
    grads a dict of float64 arrays summed over every active cell of every dataset."""
    dY = np.asarray(dY, dtype=np.float64)
    P, heads = cache["params"], cache["heads"]
    dX = np.zeros(cache["shape"])
    grads = {k: np.zeros_like(v) for k, v in P.items()}
    for b, (act, c) in enumerate(cache["caches"]):
        dz, g = dataset_backward(dY[b][:, act, :], c, P, heads)
        dX[b][:, act, :] = dz
        for k in grads:
            grads[k] += g[k]
    return dX, grads


def stack_forward(X, params_list, n_train, cell_mask, heads, eps=LN_EPS):
    """Layers applied in sequence, each with its own parameters."""
    caches = []
    for P in params_list:
        X, c = layer_forward(X, P, n_train, cell_mask, heads, eps)
        caches.append(c)
    return X, caches


def stack_backward(dY, caches):
    grads = [None] * len(caches)
    for i in range(len(caches) - 1, -1, -1):
        dY, grads[i] = layer_backward(dY, caches[i])
    return dY, grads

