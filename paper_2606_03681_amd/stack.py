"""Device-side plumbing around the C ABI: buffers for a stack of layers and the call order of
their forward and backward passes (forward 0..L-1, backward L-1..0).  Allocation only; all
arithmetic is in the library."""

import numpy as np
import torch

from . import tfm
from . import workloads as wl
from .workloads import bf16_bits_to_f32


def to_device(a, dtype, device="cuda"):
    """numpy storage array (float32, or uint16 bfloat16 bits) -> device tensor."""
    if dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint16).view(np.int16))
    return t.to(device).view(torch.bfloat16)


def to_host(t, dtype):
    """device tensor -> numpy float64."""
    if dtype == "f32":
        return t.detach().float().cpu().numpy().astype(np.float64)
    bits = t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    return bf16_bits_to_f32(bits).astype(np.float64)


class Stack:
    """L layers with independent parameters over the same n_train / cell_mask.  For the pre-norm
    block, layer l multiplies its input by decay_base ** (first_layer + l)."""

    def __init__(self, dims, n_train, cell_mask, params, device="cuda", decay_base=0.95,
                 first_layer=0):
        self.dims = dims
        self.n_train = np.ascontiguousarray(n_train, dtype=np.int32)
        self.cell_mask = np.ascontiguousarray(cell_mask, dtype=np.uint8)
        self.device = device
        self.params = [p if isinstance(p, torch.Tensor) else
                       torch.from_numpy(np.ascontiguousarray(p, dtype=np.float32)).to(device)
                       for p in params]
        self.L = len(self.params)
        self.layer_dims = [dims] * self.L
        if dims.block == tfm.TFM_BLOCK_PRENORM:
            self.layer_dims = []
            for l in range(self.L):
                dl = tfm.tfm_dims.from_buffer_copy(dims)
                dl.decay = decay_base ** (first_layer + l)
                self.layer_dims.append(dl)
        self.elt = torch.float32 if dims.dtype == tfm.TFM_F32 else torch.bfloat16
        self.shape = (dims.B, dims.R, dims.C + 1, dims.E)
        sb, wb = tfm.saved_bytes(dims), tfm.workspace_bytes(dims)
        if sb == 0 or wb == 0:
            raise tfm.TfmError(-1, tfm.last_error())
        self.saved = [torch.empty(sb, dtype=torch.uint8, device=device) for _ in range(self.L)]
        self.workspace = torch.empty(wb, dtype=torch.uint8, device=device)
        self.acts = [torch.empty(self.shape, dtype=self.elt, device=device)
                     for _ in range(self.L)]
        self.grads = [torch.empty_like(p) for p in self.params]
        self.dxs = [torch.empty(self.shape, dtype=self.elt, device=device) for _ in range(2)]
        self.inputs = None

    def forward(self, X):
        """Runs every layer; returns the last layer's output (a buffer owned by the stack)."""
        self.inputs = [X] + self.acts[:-1]
        for l in range(self.L):
            tfm.layer_fwd(self.layer_dims[l], self.n_train, self.cell_mask, self.inputs[l],
                          self.params[l], self.acts[l], self.saved[l], self.workspace)
        return self.acts[-1]

    def backward(self, dY, accumulate=False):
        """Backward through every layer; returns dX of the first layer.  Parameter gradients
        land in self.grads."""
        g = dY
        for l in range(self.L - 1, -1, -1):
            out = self.dxs[l % 2]
            tfm.layer_bwd(self.layer_dims[l], self.n_train, self.cell_mask, self.inputs[l],
                          self.params[l], self.saved[l], g, out, self.grads[l], accumulate,
                          self.workspace)
            g = out
        return g


class InferStack:
    """Forward-only evaluation of L layers (no saved state): `context` runs the context rows
    (train rows first) through every layer once and keeps one key/value cache per layer;
    `query` then runs any number of chunks of unlabelled rows through every layer against
    those caches.  For the pre-norm block, layer l multiplies its input by
    decay_base ** (first_layer + l)."""

    def __init__(self, dims, n_train, cell_mask, params, max_query_rows, device="cuda",
                 decay_base=0.95, first_layer=0):
        self.n_train = np.ascontiguousarray(n_train, dtype=np.int32)
        self.cell_mask = np.ascontiguousarray(cell_mask, dtype=np.uint8)
        self.device = device
        self.params = [p if isinstance(p, torch.Tensor) else
                       torch.from_numpy(np.ascontiguousarray(p, dtype=np.float32)).to(device)
                       for p in params]
        self.L = len(self.params)
        self.Rc, self.Rq = dims.R, int(max_query_rows)
        self.ctx_dims = self._layer_dims(dims, dims.R, decay_base, first_layer)
        self.q_dims = None
        self.decay_base, self.first_layer, self.base = decay_base, first_layer, dims
        self.elt = torch.bfloat16
        wb = max(tfm.infer_workspace_bytes(self.ctx_dims[0]),
                 tfm.infer_workspace_bytes(self._copy(dims, self.Rq)))
        cb = tfm.infer_cache_bytes(self.ctx_dims[0])
        if wb == 0 or cb == 0:
            raise tfm.TfmError(-1, tfm.last_error())
        self.workspace = torch.empty(wb, dtype=torch.uint8, device=device)
        self.caches = [torch.empty(cb, dtype=torch.uint8, device=device) for _ in range(self.L)]
        S, E = dims.C + 1, dims.E
        self.ctx_out = [torch.empty((dims.B, self.Rc, S, E), dtype=self.elt, device=device)
                        for _ in range(min(self.L, 2))]
        self.q_flat = [torch.empty(dims.B * self.Rq * S * E, dtype=self.elt, device=device)
                       for _ in range(min(self.L, 2))]

    @staticmethod
    def _copy(dims, R):
        d = tfm.tfm_dims.from_buffer_copy(dims)
        d.R = int(R)
        return d

    def _layer_dims(self, dims, R, decay_base, first_layer):
        out = []
        for l in range(len(self.params)):
            d = self._copy(dims, R)
            if dims.block == tfm.TFM_BLOCK_PRENORM:
                d.decay = decay_base ** (first_layer + l)
            out.append(d)
        return out

    def context(self, X):
        """X: [B, Rc, C+1, E] bfloat16.  Returns the last layer's output (owned buffer)."""
        h = X
        for l in range(self.L):
            out = self.ctx_out[l % 2]
            tfm.layer_fwd_context(self.ctx_dims[l], self.n_train, self.cell_mask, h,
                                  self.params[l], out, self.caches[l], self.workspace)
            h = out
        return h

    def query(self, Xq):
        """Xq: [B, Rq', C+1, E] bfloat16 unlabelled rows (contiguous), Rq' <= max_query_rows.
        Returns the last layer's output for them (a view of an owned buffer)."""
        Rq = Xq.shape[1]
        if Rq > self.Rq:
            raise ValueError(f"{Rq} query rows exceed max_query_rows={self.Rq}")
        dims = self._layer_dims(self.base, Rq, self.decay_base, self.first_layer)
        h = Xq
        for l in range(self.L):
            B, _, S, E = Xq.shape
            out = self.q_flat[l % 2][:B * Rq * S * E].view(B, Rq, S, E)
            tfm.layer_fwd_query(dims[l], self.Rc, self.n_train, self.cell_mask, h,
                                self.params[l], self.caches[l], out, self.workspace)
            h = out
        return h


class TrainStep:
    """One training step through the whole model: the encoders build the stack input (and the
    thinking-row table fills its first T rows), the stack runs forward, the decoder computes the
    loss and the gradient of the stack output, the stack runs backward and the encoders (and the
    table) receive their gradients.  Allocation and call order only."""

    def __init__(self, dims, ends, n_train, n_feat, n_class, params, ends_params, table=None,
                 device="cuda", decay_base=0.95):
        self.dims, self.ends = dims, ends
        self.n_train = np.ascontiguousarray(n_train, dtype=np.int32)
        self.n_feat = np.ascontiguousarray(n_feat, dtype=np.int32)
        self.n_class = np.ascontiguousarray(n_class, dtype=np.int32)
        C = dims.C
        self.cell_mask = np.zeros((dims.B, C + 1), np.uint8)
        for b, m in enumerate(self.n_feat):
            self.cell_mask[b, :m] = 1
        self.cell_mask[:, C] = 1
        self.stack = Stack(dims, self.n_train, self.cell_mask, params, device=device,
                           decay_base=decay_base)
        self.ends_params = ends_params if isinstance(ends_params, torch.Tensor) else \
            torch.from_numpy(np.ascontiguousarray(ends_params, dtype=np.float32)).to(device)
        self.T = ends.T
        self.table = None
        if self.T:
            self.table = table if isinstance(table, torch.Tensor) else \
                torch.from_numpy(np.ascontiguousarray(table, dtype=np.float32)).to(device)
            self.table_grad = torch.empty_like(self.table)
        wb = tfm.ends_workspace_bytes(dims, ends)
        if wb == 0:
            raise tfm.TfmError(-1, tfm.last_error())
        self.ends_ws = torch.empty(wb, dtype=torch.uint8, device=device)
        self.X = torch.empty(self.stack.shape, dtype=self.stack.elt, device=device)
        self.dY = torch.empty(self.stack.shape, dtype=self.stack.elt, device=device)
        self.loss = torch.empty(4, dtype=torch.float32, device=device)
        self.ends_grads = torch.empty_like(self.ends_params)
        self.Y = self.dX = None

    def run(self, x, labels):
        """x: device float32 [B, R-T, F]; labels: device int32 [B, R-T].  Returns the loss as a
        device tensor of one element; gradients land in stack.grads, ends_grads, table_grad."""
        d, e = self.dims, self.ends
        if self.T:
            tfm.thinking_rows_fwd(d, self.n_train, self.cell_mask, self.T, self.table, self.X,
                                  self.stack.workspace)
        tfm.encode_fwd(d, e, self.n_train, self.n_feat, x, labels, self.ends_params, self.X,
                       self.ends_ws)
        self.Y = self.stack.forward(self.X)
        tfm.decode_loss(d, e, self.n_train, self.n_feat, self.n_class, labels, self.Y,
                        self.ends_params, self.loss, None, self.dY, self.ends_grads, False,
                        self.ends_ws)
        self.dX = self.stack.backward(self.dY)
        if self.T:
            tfm.thinking_rows_bwd(d, self.n_train, self.cell_mask, self.T, self.dX,
                                  self.table_grad, False, self.stack.workspace)
        tfm.encode_bwd(d, e, self.n_train, self.n_feat, x, labels, self.dX, self.ends_grads,
                       False, self.ends_ws)
        return self.loss[:1]


# Optimiser settings of Tab. 5 (baseline / current best record); b1, b2, eps and the absent
# warm-up are the schedule-free defaults.
OPTIM_BASELINE = dict(lr=1e-4, adamw_wd=0.0, clip=1.0, muon=False)
OPTIM_RECORD = dict(lr=1e-3, adamw_wd=0.01, clip=2.0, muon=True, muon_lr_ratio=0.1,
                    muon_momentum=0.96, muon_wd=0.1)


def muon_matrices(E, H, block):
    """(offset, rows, cols) of the hidden weight matrices in a packed layer vector that Muon
    updates: Q, K and V of each attention as three E x E matrices, both output projections, W1
    and W2."""
    out = []
    off = 0
    for name, shape, kind in wl.param_layout(E, H, block):
        n = int(np.prod(shape))
        if name in ("Wqkv_f", "Wqkv_i"):
            out += [(off + j * E * E, E, E) for j in range(3)]
        elif kind == "w":
            out.append((off, shape[0], shape[1]))
        off += n
    return out


def adamw_segments(total, matrices):
    """Segments of a packed vector of `total` floats not covered by the Muon matrices."""
    covered = sorted((o, o + r * c) for o, r, c in matrices)
    segs, pos = [], 0
    for a, b in covered:
        if a > pos:
            segs.append((pos, a - pos))
        pos = max(pos, b)
    if pos < total:
        segs.append((pos, total - pos))
    return segs


class Optimizer:
    """The optimiser step of a TrainStep: gradients clipped by their global norm, Muon on the
    blocks' hidden matrices (batched over all matrices of one shape), schedule-free AdamW on the
    rest (every parameter, for the baseline settings).  The model's parameters are the
    schedule-free y sequence; z starts as a copy of them."""

    def __init__(self, ts, settings, beta1=0.9, beta2=0.999, eps=1e-8, warmup=0):
        self.ts = ts
        self.s = dict(settings)
        dev = ts.ends_params.device
        E, H = ts.dims.E, ts.dims.H
        block = "pre" if ts.dims.block == tfm.TFM_BLOCK_PRENORM else "post"
        self.hp = tfm.tfm_sfadamw(self.s["lr"], beta1, beta2, eps, self.s["adamw_wd"], warmup)
        # (y, grad, z, v, segments) per parameter vector
        self.vectors = []
        mats = muon_matrices(E, H, block) if self.s["muon"] else []
        for p, g in zip(ts.stack.params, ts.stack.grads):
            self.vectors.append((p, g, p.clone(), torch.zeros_like(p),
                                 adamw_segments(p.numel(), mats)))
        extra = [(ts.ends_params, ts.ends_grads)]
        if ts.T:
            extra.append((ts.table.view(-1), ts.table_grad.view(-1)))
        for p, g in extra:
            self.vectors.append((p, g, p.clone(), torch.zeros_like(p), [(0, p.numel())]))
        self.muon = {}
        if mats:
            self.muon_hp = tfm.tfm_muon(self.s["lr"] * self.s["muon_lr_ratio"],
                                        self.s["muon_momentum"], self.s["muon_wd"], 1, 5)
            self.bufs = [torch.zeros_like(p) for p in ts.stack.params]
            for (o, r, c) in mats:
                grp = self.muon.setdefault((r, c), ([], [], []))
                for p, g, b in zip(ts.stack.params, ts.stack.grads, self.bufs):
                    grp[0].append(p.data_ptr() + 4 * o)
                    grp[1].append(g.data_ptr() + 4 * o)
                    grp[2].append(b.data_ptr() + 4 * o)
            wb = max(tfm.muon_workspace_bytes(len(v[0]), r, c) for (r, c), v in self.muon.items())
            self.muon_ws = torch.empty(wb, dtype=torch.uint8, device=dev)
        self.grads = [v[1] for v in self.vectors]
        self.clip_ws = torch.empty(tfm.clip_workspace_bytes([g.numel() for g in self.grads]),
                                   dtype=torch.uint8, device=dev)
        self.scale = torch.empty(4, dtype=torch.float32, device=dev)
        self.norm = torch.empty(4, dtype=torch.float32, device=dev)
        self.t = 0

    def step(self):
        self.t += 1
        tfm.clip_scale(self.grads, self.s["clip"], self.scale, self.norm, self.clip_ws)
        for (r, c), (W, G, B) in self.muon.items():
            tfm.muon_step(self.muon_hp, r, c, W, G, B, self.scale, self.muon_ws)
        for y, g, z, v, segs in self.vectors:
            if segs:
                tfm.sfadamw_step(self.hp, self.t, segs, y, z, v, g, self.scale)


class InferModel:
    """Evaluation of whole tables through the forward-only path: the encoders build the stack
    input of every row (the thinking-row table fills rows [0, T)), the context rows — rows
    [0, max n_train), which hold every labelled row — run through every layer once and leave
    key/value caches, the remaining rows run through every layer in chunks of unlabelled rows
    against those caches, and the decoder turns the outputs of each dataset's unlabelled rows
    into logits.  Allocation, call order and the row order of the result only."""

    def __init__(self, dims, ends, n_train, n_feat, params, ends_params, table=None,
                 chunk=256, device="cuda", decay_base=0.95):
        if dims.dtype != tfm.TFM_BF16:
            raise ValueError("the forward-only path runs in bfloat16")
        self.dims, self.ends = dims, ends
        self.n_train = np.ascontiguousarray(n_train, dtype=np.int32)
        self.n_feat = np.ascontiguousarray(n_feat, dtype=np.int32)
        B, R, C, E = dims.B, dims.R, dims.C, dims.E
        self.cell_mask = np.zeros((B, C + 1), np.uint8)
        for b, m in enumerate(self.n_feat):
            self.cell_mask[b, :m] = 1
        self.cell_mask[:, C] = 1
        self.Rc = int(self.n_train.max())
        self.chunk = max(1, int(chunk))
        self.spans = [(a, min(a + self.chunk, R)) for a in range(self.Rc, R, self.chunk)]
        dc = tfm.tfm_dims.from_buffer_copy(dims)
        dc.R = self.Rc
        self.ctx_dims = dc
        self.stack = InferStack(dc, self.n_train, self.cell_mask, params,
                                max_query_rows=self.chunk, device=device, decay_base=decay_base)
        self.ends_params = ends_params if isinstance(ends_params, torch.Tensor) else \
            torch.from_numpy(np.ascontiguousarray(ends_params, dtype=np.float32)).to(device)
        self.table = None
        if ends.T:
            self.table = table if isinstance(table, torch.Tensor) else \
                torch.from_numpy(np.ascontiguousarray(table, dtype=np.float32)).to(device)
        # the decoder calls see tables without thinking rows (T does not enter decoding)
        self.dec_ends = tfm.tfm_ends.from_buffer_copy(ends)
        self.dec_ends.T = 0
        wb = max(tfm.ends_workspace_bytes(dims, ends), tfm.ends_workspace_bytes(dims, self.dec_ends))
        self.ends_ws = torch.empty(wb, dtype=torch.uint8, device=device)
        self.X = torch.empty((B, R, C + 1, E), dtype=torch.bfloat16, device=device)
        self.xq = torch.empty(B * self.chunk * (C + 1) * E, dtype=torch.bfloat16, device=device)
        self.K = ends.K
        self.device = device

    def predict(self, x, labels):
        """x: device float32 [B, R-T, F]; labels: device int32 [B, R-T] (the labelled rows'
        entries are read).  Returns logits [T_test, K] of the unlabelled rows in (dataset, row)
        order, as tfm_decode_loss orders them."""
        d, e = self.dims, self.ends
        B, C, E = d.B, d.C, d.E
        if e.T:
            tfm.thinking_rows_fwd(d, self.n_train, self.cell_mask, e.T, self.table, self.X,
                                  self.stack.workspace)
        tfm.encode_fwd(d, e, self.n_train, self.n_feat, x, labels, self.ends_params, self.X,
                       self.ends_ws)
        Xc = self.X[:, :self.Rc].contiguous()
        parts = []  # (first row, per-dataset row counts, logits of the call)
        Yc = self.stack.context(Xc)
        nctx = self.Rc - self.n_train
        lg = torch.empty((max(int(nctx.sum()), 1), self.K), device=self.device)
        if nctx.sum() > 0:
            tfm.decode_fwd(self.ctx_dims, self.dec_ends, self.n_train, self.n_feat, Yc,
                           self.ends_params, lg, self.ends_ws)
        parts.append((nctx, lg))
        for a, b in self.spans:
            Rq = b - a
            xq = self.xq[:B * Rq * (C + 1) * E].view(B, Rq, C + 1, E)
            xq.copy_(self.X[:, a:b])
            Yq = self.stack.query(xq)
            dq = tfm.tfm_dims.from_buffer_copy(d)
            dq.R = Rq
            lq = torch.empty((B * Rq, self.K), device=self.device)
            tfm.decode_fwd(dq, self.dec_ends, np.zeros(B, np.int32), self.n_feat, Yq,
                           self.ends_params, lq, self.ends_ws)
            parts.append((np.full(B, Rq), lq))
        # (dataset, row) order: dataset b's rows come from the context call, then each chunk
        out = []
        offs = [np.concatenate([[0], np.cumsum(cnt)]) for cnt, _ in parts]
        for b in range(B):
            for (cnt, lgp), off in zip(parts, offs):
                if cnt[b]:
                    out.append(lgp[off[b]:off[b] + cnt[b]])
        return torch.cat(out) if out else torch.empty((0, self.K), device=self.device)
