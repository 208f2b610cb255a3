"""Seeded synthetic workloads for the two-axis layer, shared by the tests, the smoke check and
the benchmark.

This module draws inputs only.  It holds none of the layer's arithmetic: it produces the cell
tensor, the per-dataset train-prefix lengths, the active-cell masks, the packed per-layer
parameters and the upstream gradient, and it counts algorithmic work for reporting.

The shapes follow the workloads the paper trains and evaluates on (Sec. 4.1: a static dump of
synthetic classification datasets of 1,000 rows and up to 20 features; Sec. 3 / App. A: the
evaluation tables subsampled to at most 100 features and 1,000 rows).  Neither the prior dump
nor the evaluation tables are used; seeded synthetic tables of the same shapes stand in for
them.

Random streams: ``numpy.random.SeedSequence(seed)`` spawns one child stream for the metadata,
one per layer for the parameters, one per dataset for the cells and one per dataset for the
upstream gradient, so any subset of datasets can be regenerated exactly without drawing the
rest.  Values are drawn in float64 and rounded once to the storage type (float32, or bfloat16
by round-to-nearest-even from the float32 value); both the oracle and the GPU consume the
rounded values.
"""

from dataclasses import dataclass, field

import numpy as np

# ---------------------------------------------------------------------------------------------
# bfloat16 helpers (bit patterns held in numpy uint16 arrays)
# ---------------------------------------------------------------------------------------------


def f32_to_bf16_bits(x):
    """Round float32 values to bfloat16 (round to nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    nan = (u & 0x7FFFFFFF) > 0x7F800000
    r = ((u >> 16) & 1) + np.uint32(0x7FFF)
    out = ((u + r) >> 16).astype(np.uint16)
    out[nan] = ((u[nan] >> 16) | 0x40).astype(np.uint16)
    return out


def bf16_bits_to_f32(b):
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def to_storage(x64, dtype):
    """float64 -> storage array: float32 values, or bfloat16 bit patterns (uint16)."""
    x32 = np.asarray(x64, dtype=np.float64).astype(np.float32)
    return x32 if dtype == "f32" else f32_to_bf16_bits(x32)


def storage_to_f64(a, dtype):
    return (a if dtype == "f32" else bf16_bits_to_f32(a)).astype(np.float64)


# ---------------------------------------------------------------------------------------------
# Configurations
# ---------------------------------------------------------------------------------------------

CONFIGS = [
    # 0: tiny fp32 single layer; cells and weights N(0, 0.02^2), upstream grad N(0, 1)
    dict(name="tiny-fp32", dtype="f32", B=2, R=64, n_train=48, C=8, E=64, heads=4, H=128,
         layers=1, cells="small_normal", weights="small_normal"),
    # 1: small bf16 layer; features N(0,1) linearly embedded, target class in [0,10) embedded
    dict(name="small-bf16", dtype="bf16", B=8, R=512, n_train=384, C=32, E=192, heads=6,
         H=384, layers=1, cells="embedded", weights="xavier"),
    # 2: eval-scale bf16, 3 stacked layers
    dict(name="eval-scale-bf16", dtype="bf16", B=16, R=1024, n_train=768, C=100, E=192,
         heads=6, H=384, layers=3, cells="normal", weights="xavier"),
    # 3: many rows, long train prefix
    dict(name="many-rows-bf16", dtype="bf16", B=4, R=8192, n_train=6144, C=16, E=192,
         heads=6, H=384, layers=1, cells="normal", weights="xavier"),
    # 4: ragged batch: n_train ~ U{512..920}, active features ~ U{4..100} padded to 100 + 1
    dict(name="ragged-bf16", dtype="bf16", B=32, R=1024, n_train=(512, 920), C=100,
         active=(4, 100), E=192, heads=6, H=384, layers=3, cells="normal", weights="xavier"),
]

# Small shapes used only by tests: several tiles with ragged tails, non-prefix masks and the
# degenerate cases of the method (n_train = 1, n_train = R, a single active cell).
TEST_CONFIGS = {
    "micro": dict(name="micro", dtype="f32", B=2, R=6, n_train=4, C=3, E=8, heads=2, H=16,
                  layers=1, cells="normal", weights="xavier_bias"),
    "ragged-small-f32": dict(name="ragged-small-f32", dtype="f32", B=4, R=200,
                             n_train=(1, 200), C=20, active=(0, 20), mask="random", E=64,
                             heads=2, H=96, layers=2, cells="normal", weights="xavier_bias"),
    "ragged-small-bf16": dict(name="ragged-small-bf16", dtype="bf16", B=5, R=333,
                              n_train=(1, 333), C=24, active=(0, 24), mask="random", E=192,
                              heads=6, H=384, layers=2, cells="normal", weights="xavier_bias"),
    "d16-bf16": dict(name="d16-bf16", dtype="bf16", B=3, R=130, n_train=97, C=7, E=64,
                     heads=4, H=128, layers=1, cells="normal", weights="xavier_bias"),
    # head dim 64 (the current best record's width per head), post-norm, bf16 and fp32
    "d64-bf16": dict(name="d64-bf16", dtype="bf16", B=3, R=130, n_train=97, C=7, E=128,
                     heads=2, H=256, layers=1, cells="normal", weights="xavier_bias"),
    "d64-f32": dict(name="d64-f32", dtype="f32", B=2, R=40, n_train=30, C=5, E=64, heads=1,
                    H=64, layers=1, cells="normal", weights="xavier_bias"),
    # pre-norm block at d = 64 with rows of up to 41 active cells
    "prenorm-d64-bf16": dict(name="prenorm-d64-bf16", dtype="bf16", B=4, R=160,
                             n_train=(1, 160), C=40, active=(0, 40), mask="random", E=128,
                             heads=2, H=384, layers=2, cells="normal", weights="xavier_bias",
                             block="pre"),
    # pre-norm RMSNorm block with residual decay (the current best record's block), at d = 32
    "prenorm-small-bf16": dict(name="prenorm-small-bf16", dtype="bf16", B=4, R=200,
                               n_train=(1, 200), C=20, active=(0, 20), mask="random", E=64,
                               heads=2, H=192, layers=2, cells="normal", weights="xavier_bias",
                               block="pre"),
    # fewer active cells (2 x 9 x 3 = 54) than one tile of the fused MLP kernels (128 cells
    # forward, 192 backward): every workgroup of those kernels has clamped, masked cells
    "tiny-mlp-bf16": dict(name="tiny-mlp-bf16", dtype="bf16", B=2, R=9, n_train=5, C=2, E=192,
                          heads=6, H=384, layers=2, cells="normal", weights="xavier_bias"),
    # train prefixes on both sides of the one-kernel item-attention backward's limit (768
    # rows): its columns and those of the two-kernel form run in separate launches
    "mixed-prefix-bf16": dict(name="mixed-prefix-bf16", dtype="bf16", B=5, R=1000,
                              n_train=(600, 1000), C=6, active=(1, 6), mask="random", E=192,
                              heads=6, H=384, layers=1, cells="normal", weights="xavier_bias"),
    # rows wider than the matrix-core feature attention takes (more than 128 cells at d = 32,
    # more than 64 at d = 64): the bfloat16 feature attention runs on the vector kernels
    "wide-d32-bf16": dict(name="wide-d32-bf16", dtype="bf16", B=3, R=128, n_train=(1, 128),
                          C=150, active=(100, 150), mask="random", E=64, heads=2, H=128,
                          layers=1, cells="normal", weights="xavier_bias"),
    "wide-d64-bf16": dict(name="wide-d64-bf16", dtype="bf16", B=3, R=40, n_train=(1, 40),
                          C=90, active=(60, 90), mask="random", E=128, heads=2, H=256,
                          layers=1, cells="normal", weights="xavier_bias"),
    "wide-prenorm-d64-bf16": dict(name="wide-prenorm-d64-bf16", dtype="bf16", B=3, R=128,
                                  n_train=(1, 128), C=90, active=(60, 90), mask="random",
                                  E=128, heads=2, H=256, layers=2, cells="normal",
                                  weights="xavier_bias", block="pre"),
}


# Workloads of the widened scope (not parity configurations of the baseline block).
#   record9-bf16: the current best record's block (Tab. 5): pre-norm RMSNorm, residual decay,
#   E = 256 with 4 heads of 64, MLP 768, 5 blocks; 1000 data rows plus 24 thinking rows
#   prepended as train rows (750 labelled data rows); 20 features, the most the pretraining
#   prior draws (Sec. 4.1), and repeated grouping makes one group of 5 per feature column, so
#   20 feature cells plus the target cell per row.
EXTRA_CONFIGS = {
    "record9-bf16": dict(name="record9-bf16", dtype="bf16", B=16, R=1024, n_train=774, C=20,
                         E=256, heads=4, H=768, layers=5, cells="normal", weights="xavier",
                         block="pre", thinking=24),
}


def get_config(which):
    if isinstance(which, int):
        return dict(CONFIGS[which], index=which)
    if which in TEST_CONFIGS:
        return dict(TEST_CONFIGS[which], index=None)
    if which in EXTRA_CONFIGS:
        return dict(EXTRA_CONFIGS[which], index=None)
    for i, c in enumerate(CONFIGS):
        if c["name"] == which:
            return dict(c, index=i)
    raise KeyError(which)


def default_seed(cfg):
    idx = cfg.get("index")
    if idx is not None:
        return 1000 + idx
    return 5000 + sum(ord(ch) for ch in cfg["name"])


# ---------------------------------------------------------------------------------------------
# Parameter layout (packed order of the C-ABI; see include/tfm_layer.h)
# ---------------------------------------------------------------------------------------------

def param_layout(E, H, block="post"):
    """(name, shape, kind) in packed order; kind is 'w' (weight [out, in]), 'b' (bias),
    'g' (norm scale) or 'n' (norm shift).  The pre-norm block has RMSNorm weights only."""
    if block == "pre":
        return [
            ("Wqkv_f", (3 * E, E), "w"), ("bqkv_f", (3 * E,), "b"),
            ("Wo_f", (E, E), "w"), ("bo_f", (E,), "b"),
            ("Wqkv_i", (3 * E, E), "w"), ("bqkv_i", (3 * E,), "b"),
            ("Wo_i", (E, E), "w"), ("bo_i", (E,), "b"),
            ("W1", (H, E), "w"), ("b1", (H,), "b"),
            ("W2", (E, H), "w"), ("b2", (E,), "b"),
            ("g1", (E,), "g"), ("g2", (E,), "g"), ("g3", (E,), "g"),
        ]
    return [
        ("Wqkv_f", (3 * E, E), "w"), ("bqkv_f", (3 * E,), "b"),
        ("Wo_f", (E, E), "w"), ("bo_f", (E,), "b"),
        ("Wqkv_i", (3 * E, E), "w"), ("bqkv_i", (3 * E,), "b"),
        ("Wo_i", (E, E), "w"), ("bo_i", (E,), "b"),
        ("W1", (H, E), "w"), ("b1", (H,), "b"),
        ("W2", (E, H), "w"), ("b2", (E,), "b"),
        ("g1", (E,), "g"), ("be1", (E,), "n"),
        ("g2", (E,), "g"), ("be2", (E,), "n"),
        ("g3", (E,), "g"), ("be3", (E,), "n"),
    ]


def param_count(E, H, block="post"):
    return sum(int(np.prod(s)) for _, s, _ in param_layout(E, H, block))


def _draw_params(rng, E, H, style, block="post"):
    parts = []
    for _, shape, kind in param_layout(E, H, block):
        n = int(np.prod(shape))
        if style == "small_normal":
            v = rng.normal(0.0, 0.02, n)
            if kind == "g":
                v = 1.0 + v
        else:
            if kind == "w":
                fan_out, fan_in = shape
                a = np.sqrt(6.0 / (fan_in + fan_out))
                v = rng.uniform(-a, a, n)
            elif kind == "g":
                v = 1.0 + rng.normal(0.0, 0.02, n)
            else:
                # xavier_bias: larger biases and shifts so that they matter in tests
                v = rng.normal(0.0, 0.2 if style == "xavier_bias" else 0.02, n)
        parts.append(v)
    return np.concatenate(parts).astype(np.float32)


# ---------------------------------------------------------------------------------------------
# Workload
# ---------------------------------------------------------------------------------------------

@dataclass
class Workload:
    cfg: dict
    seed: int
    datasets: np.ndarray          # indices of the generated datasets within the full batch
    n_train: np.ndarray           # int32 [B']
    cell_mask: np.ndarray         # uint8 [B', C+1]
    X: np.ndarray                 # [B', R, C+1, E] float32, or uint16 bfloat16 bits
    params: list                  # per layer: float32 [param_count]
    dY: np.ndarray = field(default=None)

    @property
    def dtype(self):
        return self.cfg["dtype"]

    @property
    def block(self):
        return self.cfg.get("block", "post")

    @property
    def dims(self):
        c = self.cfg
        return dict(B=len(self.datasets), R=c["R"], C=c["C"], E=c["E"], heads=c["heads"],
                    H=c["H"], dtype=c["dtype"])

    def X64(self):
        return storage_to_f64(self.X, self.dtype)

    def dY64(self):
        return storage_to_f64(self.dY, self.dtype)

    def params64(self):
        return [p.astype(np.float64) for p in self.params]


def _metadata(cfg, rng):
    B, R, C = cfg["B"], cfg["R"], cfg["C"]
    S = C + 1
    nt = cfg["n_train"]
    if isinstance(nt, tuple):
        n_train = rng.integers(nt[0], nt[1] + 1, size=B)
    else:
        n_train = np.full(B, nt)
    mask = np.ones((B, S), dtype=np.uint8)
    if "active" in cfg:
        lo, hi = cfg["active"]
        counts = rng.integers(lo, hi + 1, size=B)
        mask[:] = 0
        mask[:, C] = 1
        for b in range(B):
            if cfg.get("mask") == "random":
                cols = rng.permutation(C)[:counts[b]]
            else:
                cols = np.arange(counts[b])
            mask[b, cols] = 1
    if cfg.get("mask") == "random" and B >= 3:
        # degenerate cases of the method: a dataset with a single labelled row, one with no
        # test row, and one whose only active cell is the target cell
        n_train[0] = 1
        n_train[1] = R
        mask[2, :C] = 0
    return n_train.astype(np.int32), mask


def _draw_cells(cfg, rng, n_train):
    R, C, E = cfg["R"], cfg["C"], cfg["E"]
    S = C + 1
    style = cfg["cells"]
    if style == "small_normal":
        return rng.normal(0.0, 0.02, (R, S, E))
    if style == "normal":
        return rng.normal(0.0, 1.0, (R, S, E))
    if style == "embedded":
        # feature cells: scalar x ~ N(0,1) embedded as x * w_x + b_x; target cell: class
        # y in [0, 10) embedded by a table T; test rows receive the mean of the train rows'
        # target embeddings (Fig. 3 caption)
        x = rng.normal(0.0, 1.0, (R, C))
        w_x = rng.normal(0.0, 1.0, E)
        b_x = rng.normal(0.0, 0.1, E)
        y = rng.integers(0, 10, R)
        T = rng.normal(0.0, 1.0, (10, E))
        cells = np.empty((R, S, E))
        cells[:, :C, :] = x[:, :, None] * w_x + b_x
        tgt = T[y]
        tgt[n_train:] = tgt[:n_train].mean(axis=0)
        cells[:, C, :] = tgt
        return cells
    raise ValueError(style)


def make_workload(which, seed=None, datasets=None, with_dY=True):
    """Generate the workload of a configuration (index into CONFIGS, or a TEST_CONFIGS name).

    datasets: optional list of dataset indices to generate (default: all B); the values of a
    dataset do not depend on which other datasets are generated."""
    cfg = get_config(which)
    seed = default_seed(cfg) if seed is None else seed
    B, L = cfg["B"], cfg["layers"]
    ss = np.random.SeedSequence(seed)
    kids = ss.spawn(1 + L + 2 * B)
    meta_rng = np.random.default_rng(kids[0])
    n_train_all, mask_all = _metadata(cfg, meta_rng)
    params = [_draw_params(np.random.default_rng(kids[1 + l]), cfg["E"], cfg["H"],
                           cfg["weights"], cfg.get("block", "post")) for l in range(L)]
    ds = np.arange(B) if datasets is None else np.asarray(datasets, dtype=np.int64)
    T = cfg.get("thinking", 0)
    # thinking rows: one table [T, E] broadcast into rows [0, T) of every active cell column
    table = meta_rng.normal(0.0, 1.0, (T, cfg["E"])) if T else None
    X = []
    dY = []
    for b in ds:
        x = _draw_cells(cfg, np.random.default_rng(kids[1 + L + b]), int(n_train_all[b]))
        if T:
            act = np.flatnonzero(mask_all[b])
            x[:T][:, act, :] = table[:, None, :]
        X.append(to_storage(x, cfg["dtype"]))
        if with_dY:
            g = np.random.default_rng(kids[1 + L + B + b]).normal(
                0.0, 1.0, (cfg["R"], cfg["C"] + 1, cfg["E"]))
            dY.append(to_storage(g, cfg["dtype"]))
    return Workload(cfg=cfg, seed=seed, datasets=ds, n_train=n_train_all[ds].copy(),
                    cell_mask=mask_all[ds].copy(), X=np.stack(X),
                    params=params, dY=np.stack(dY) if with_dY else None)


# ---------------------------------------------------------------------------------------------
# Work counts
# ---------------------------------------------------------------------------------------------

def forward_flops(R, E, H, n_train, active):
    """Algorithmic matmul flops (2 per multiply-add) of one layer forward for one dataset with
    `active` active cells per row: the linears over all active cells, item keys/values for the
    train rows only, feature attention (S x S per row), item attention over the train prefix."""
    S = active
    return (R * S * (12 * E * E + 4 * E * H) + n_train * S * 4 * E * E
            + R * S * S * 4 * E + S * R * n_train * 4 * E)


def work_counts(n_train, cell_mask, R, E, H, layers):
    """Active cell-layers and algorithmic flops of one stack fwd+bwd (bwd counted as 2x fwd)."""
    cells = 0
    flops = 0
    for b in range(len(n_train)):
        S = int(np.count_nonzero(cell_mask[b]))
        cells += R * S
        flops += forward_flops(R, E, H, int(n_train[b]), S)
    return dict(cell_layers=cells * layers, flops_fwd_bwd=3 * flops * layers,
                active_cells=cells)


# ---------------------------------------------------------------------------------------------
# Inputs of the stack's two ends (encoders, decoder, loss) for a full training step
# ---------------------------------------------------------------------------------------------

@dataclass
class EndsInputs:
    G: int                        # feature group size
    offsets: tuple                # group shifts
    F: int                        # columns per row of x
    T: int                        # thinking rows at the head of the stack input
    Hd: int                       # decoder hidden width
    K: int                        # decoder outputs
    mean: bool                    # decoder input: mean of the feature cells (else target cell)
    n_feat: np.ndarray            # int32 [B']
    n_class: np.ndarray           # int32 [B']
    cell_mask: np.ndarray         # uint8 [B', C+1]: feature cells [0, n_feat) and the target
    x: np.ndarray                 # float32 [B', R-T, F]
    labels: np.ndarray            # int32 [B', R-T]
    params: np.ndarray            # float32 packed ends vector
    table: np.ndarray = None      # float32 [T, E] thinking rows, or None


# Group shifts: (0, 1, 3) as the paper gives for groups of 3; for groups of 5 the paper gives
# none, and (0, 1, 3, 7, 12) keeps all pairwise differences distinct.
GROUP_SHIFTS = {1: (0,), 3: (0, 1, 3), 5: (0, 1, 3, 7, 12)}


def ends_param_layout(E, G, Hd, K):
    """(name, shape, fan_in, fan_out) in the packed order of the C-ABI (include/tfm_ends.h)."""
    return [("W_fe", (E, G), G, E), ("b_fe", (E,), 0, 0), ("W_te", (E,), 1, E),
            ("b_te", (E,), 0, 0), ("W_d1", (Hd, E), E, Hd), ("b_d1", (Hd,), 0, 0),
            ("W_d2", (K, Hd), Hd, K), ("b_d2", (K,), 0, 0)]


def _is_prefix_mask(mask_row):
    C = len(mask_row) - 1
    m = int(np.count_nonzero(mask_row[:C]))
    return m >= 1 and bool(np.all(mask_row[:m])) and mask_row[C] == 1


def make_ends_inputs(w, seed=None, G=None, mean=None, K=10, Hd=None, bias_scale=0.2,
                     n_class=None):
    """Draw the ends' inputs for workload w: feature values x ~ N(0, 1), labels uniform over each
    dataset's classes (2..K unless n_class is given), Xavier-uniform weights, N(0, bias_scale^2)
    biases, a N(0, 1) thinking-row table.  Defaults follow the block: the post-norm baseline
    encodes single features and decodes the target cell; the pre-norm record groups 5 features
    and decodes the feature mean (Tab. 5).  The feature count of a dataset is its workload's
    when the workload's mask is a prefix mask, else drawn from [1, C]."""
    cfg = w.cfg
    pre = cfg.get("block", "post") == "pre"
    G = (5 if pre else 1) if G is None else G
    mean = pre if mean is None else mean
    Hd = cfg["H"] if Hd is None else Hd
    T = cfg.get("thinking", 0)
    B_all, R, C, E = cfg["B"], cfg["R"], cfg["C"], cfg["E"]
    seed = (w.seed + 7919) if seed is None else seed
    kids = np.random.SeedSequence(seed).spawn(2 + B_all)
    meta = np.random.default_rng(kids[0])
    nc_all = (meta.integers(2, K + 1, size=B_all) if n_class is None
              else np.broadcast_to(np.asarray(n_class), (B_all,)).copy())
    nf_draw = meta.integers(1, C + 1, size=B_all)
    table = meta.normal(0.0, 1.0, (T, E)).astype(np.float32) if T else None
    prng = np.random.default_rng(kids[1])
    parts = []
    for _, shape, fi, fo in ends_param_layout(E, G, Hd, K):
        n = int(np.prod(shape))
        if fi:
            a = np.sqrt(6.0 / (fi + fo))
            parts.append(prng.uniform(-a, a, n))
        else:
            parts.append(prng.normal(0.0, bias_scale, n))
    params = np.concatenate(parts).astype(np.float32)
    ds = w.datasets
    B = len(ds)
    n_feat = np.empty(B, np.int32)
    mask = np.zeros((B, C + 1), np.uint8)
    xs, labs = [], []
    for i, b in enumerate(ds):
        m = (int(np.count_nonzero(w.cell_mask[i][:C])) if _is_prefix_mask(w.cell_mask[i])
             else int(nf_draw[b]))
        n_feat[i] = m
        mask[i, :m] = 1
        mask[i, C] = 1
        r = np.random.default_rng(kids[2 + b])
        xs.append(r.normal(0.0, 1.0, (R - T, C)).astype(np.float32))
        labs.append(r.integers(0, nc_all[b], R - T).astype(np.int32))
    return EndsInputs(G=G, offsets=GROUP_SHIFTS.get(G, tuple(range(G))), F=C, T=T, Hd=Hd, K=K,
                      mean=bool(mean), n_feat=n_feat, n_class=nc_all[ds].astype(np.int32),
                      cell_mask=mask, x=np.stack(xs), labels=np.stack(labs), params=params,
                      table=table)
