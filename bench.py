"""Throughput of the two-axis layer stack (forward + backward) on one MI355X.

One step = forward of every layer of the stack, then backward of every layer, over one batch of
seeded synthetic tables already resident in HBM.  Prints one JSON line: ms_per_step is the median
of the timed steps (an event between consecutive steps, nothing else recorded), value the active
cell-layers per second at that median; the roofline object of the dominant kernel comes from a
separate pass with per-kernel events.

    python bench.py [--steps K] [--warmup W] [--config 2] [--no-cpu-baseline]
"""

import argparse
import hashlib
import json
import os
import platform
import subprocess
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2606_03681_amd import workloads as wl  # noqa: E402

METRIC = "two-axis layer fwd+bwd cells/sec (bf16) + % MFMA peak, 1x MI355X"
METRIC_INFER = "two-axis layer forward-only (context + query chunks) cells/sec (bf16), 1x MI355X"
METRIC_STEP = ("full training step (encoders, stack fwd+bwd, decoder and loss) cells/sec (bf16), "
               "1x MI355X")
PEAK_TFLOPS = {"mfma_bf16": 2516.6, "mfma_f32": 157.3, "alu_f32": 157.3}
HBM_PEAK_GBS = 8000.0


def step_flops(w, fused_rows=0):
    """Algorithmic matmul flops of one launch of each step (per layer), for the whole batch.
    fused_rows: the longest train prefix whose item-attention backward runs as the one-kernel
    step item_attn_bwd (tfm_prof_item_bwd_fused_rows); the columns of longer prefixes run as
    item_attn_dq and item_attn_dkdv, so each step is priced for the columns it runs."""
    R, E, H = w.cfg["R"], w.cfg["E"], w.cfg["H"]
    kv = fa = ia = ia_one = 0
    N = 0
    for b in range(len(w.n_train)):
        S = int(np.count_nonzero(w.cell_mask[b]))
        n = int(w.n_train[b])
        N += R * S
        kv += n * S * 4 * E * E
        fa += R * S * S * 4 * E
        ia += S * R * n * 4 * E
        if n <= fused_rows:
            ia_one += S * R * n * 4 * E
    f = {
        "feat_qkv": 6 * N * E * E, "feat_attn_fwd": fa, "feat_out": 2 * N * E * E,
        "item_qkv": 2 * N * E * E + kv, "item_attn_fwd": ia, "item_out": 2 * N * E * E,
        "mlp_up": 2 * N * E * H, "mlp_down": 2 * N * E * H,
        "feat_attn_bwd": 2 * fa, "item_attn_bwd": 2 * (ia_one if fused_rows else ia),
        # the two-kernel item-attention backward: dQ (dP and dQ products) and dK/dV (dV and dK
        # products), one forward's worth of products each over the columns it runs
        "item_attn_dq": ia - ia_one, "item_attn_dkdv": ia - ia_one,
        "mlp_down_dx": 2 * N * E * H, "mlp_up_dx": 2 * N * E * H,
        "item_out_dx": 2 * N * E * E, "item_qkv_dx": 2 * N * E * E + kv,
        "feat_out_dx": 2 * N * E * E, "feat_qkv_dx": 6 * N * E * E,
    }
    return f


def _sha(path):
    with open(os.path.join(ROOT, path), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def measured_traffic(step, workload):
    """HBM bytes per launch of `step` from the committed counter readings (profiles/traffic.json),
    or None when there are none for this workload or a source they were taken on has changed."""
    try:
        with open(os.path.join(ROOT, "profiles", "traffic.json")) as f:
            rec = json.load(f).get(step)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("workload") != workload:
        return None
    try:
        if any(_sha(p) != h for p, h in rec["sources"].items()):
            return None
    except OSError:
        return None
    return rec["bytes_per_launch"]


def git_rev():
    try:
        return subprocess.run(["git", "-C", ROOT, "rev-parse", "--short", "HEAD"],
                              capture_output=True, text=True, timeout=5).stdout.strip() or None
    except Exception:
        return None


# Query rows of the CPU-baseline sample: a dataset's rows up to this many (its outputs at those
# rows, keys and values over its whole train prefix), so that the oracle's run stays in the
# tens of seconds at the long-prefix workload.
CPU_SAMPLE_ROWS = 1024


def cpu_baseline(cfg_index, seed, forward_only=False):
    """The float64 oracle, untuned, on a bounded sample of the same workload: dataset 0 through
    one layer, forward and backward (or forward only), at the workload's per-dataset shape, its
    outputs taken at the first CPU_SAMPLE_ROWS rows (all rows of every workload but the
    many-rows one; a row's output needs the train prefix's keys and values, which are computed
    whole)."""
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        threads = os.cpu_count()
    w = wl.make_workload(cfg_index, seed=seed, datasets=[0])
    E, H, heads = w.cfg["E"], w.cfg["H"], w.cfg["heads"]
    R = w.cfg["R"]
    act = np.flatnonzero(w.cell_mask[0])
    z, dy = w.X64()[0][:, act], w.dY64()[0][:, act]
    n = int(w.n_train[0])
    q = np.arange(min(R, CPU_SAMPLE_ROWS))
    t0 = time.perf_counter()
    if w.block == "pre":
        P = oracle.unpack_prenorm_params(w.params64()[0], E, H)
        _, cache = oracle.prenorm_dataset_forward(z, P, heads, n, 1.0, query_rows=q)
        if not forward_only:
            oracle.prenorm_dataset_backward(dy[q], cache, P, heads)
    else:
        P = oracle.unpack_params(w.params64()[0], E, H)
        _, cache = oracle.dataset_forward(z, P, heads, n, query_rows=q)
        if not forward_only:
            oracle.dataset_backward(dy[q], cache, P, heads)
    dt = time.perf_counter() - t0
    cells = int(len(q) * len(act))
    kind = "fwd" if forward_only else "fwd+bwd"
    rows = f"all {R} rows" if len(q) == R else f"the first {len(q)} of its {R} rows"
    return {"value": cells / dt, "unit": "cells/s", "cores": int(threads), "kind": "oracle",
            "sample": f"dataset 0 of the workload, 1 layer {kind} at {rows} ({cells} active "
                      f"cells), {dt:.1f} s, host {platform.processor() or platform.machine()} "
                      f"({os.cpu_count()} logical CPUs)"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="2",
                    help="workload: an index of the baseline configurations, or a name")
    ap.add_argument("--seed", type=int, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true",
                    help="skip the per-step event timing (roofline of the dominant kernel)")
    ap.add_argument("--infer", action="store_true",
                    help="time the forward-only path instead: the context rows (the longest "
                         "train prefix) through every layer with key/value caches, then the "
                         "remaining rows as query chunks through every layer")
    ap.add_argument("--query-chunk", type=int, default=0,
                    help="rows per query chunk of --infer (0: all remaining rows at once)")
    ap.add_argument("--full-step", action="store_true",
                    help="time a whole training step instead: encoders (and thinking rows), the "
                         "stack forward and backward, the decoder with the loss, the encoders' "
                         "gradients and the optimiser step (clipping, Muon for the pre-norm "
                         "record's hidden matrices, schedule-free AdamW), from feature values "
                         "and labels in HBM")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run 5 device-to-device copies of MIB MiB (the known-size copy "
                         "that scales the FETCH_SIZE / WRITE_SIZE counters) and exit")
    args = ap.parse_args()
    if args.calibrate_copy:
        import torch
        n = args.calibrate_copy * (1 << 20) // 4
        a = torch.ones(n, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        for _ in range(5):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": n * 4, "copies": 5}))
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} (WORLD_SIZE={world}) is not "
              "supported: the datasets of a batch are independent, and sharding them across "
              "GPUs (one all-reduce of the parameter gradients per step) is not built.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_03681_amd import tfm
    from paper_2606_03681_amd.stack import Stack, to_device

    if str(args.config).isdigit():
        args.config = int(args.config)
    cfg = wl.get_config(args.config)
    seed = wl.default_seed(cfg) if args.seed is None else args.seed
    print(f"[bench] generating {cfg['name']} seed={seed}", file=sys.stderr, flush=True)
    w = wl.make_workload(args.config, seed=seed, with_dY=not args.full_step)
    ends_in = None
    if args.full_step:
        ends_in = wl.make_ends_inputs(w)
        w.cell_mask = ends_in.cell_mask
    counts = wl.work_counts(w.n_train, w.cell_mask, cfg["R"], cfg["E"], cfg["H"], cfg["layers"])
    dims = tfm.make_dims(dtype=w.dtype, block=w.block,
                         **{k: v for k, v in w.dims.items() if k != "dtype"})
    torch.cuda.set_device(0)
    if args.infer:
        from paper_2606_03681_amd.stack import InferStack
        R = cfg["R"]
        Rc = int(np.max(w.n_train))
        chunk = args.query_chunk if args.query_chunk > 0 else max(R - Rc, 1)
        spans = [(a, min(a + chunk, R)) for a in range(Rc, R, chunk)]
        dctx = tfm.make_dims(dtype=w.dtype, block=w.block,
                             **{k: (Rc if k == "R" else v) for k, v in w.dims.items()
                                if k != "dtype"})
        st = InferStack(dctx, w.n_train, w.cell_mask, w.params, max_query_rows=chunk)
        Xc = to_device(np.ascontiguousarray(w.X[:, :Rc]), w.dtype)
        Xq = [to_device(np.ascontiguousarray(w.X[:, a:b]), w.dtype) for a, b in spans]
        X = dY = None
        del w.X, w.dY

        def step():
            st.context(Xc)
            for x in Xq:
                st.query(x)
    elif args.full_step:
        from paper_2606_03681_amd.stack import (OPTIM_BASELINE, OPTIM_RECORD, Optimizer,
                                                TrainStep)
        e = ends_in
        ends = tfm.make_ends(e.G, e.offsets, e.F, e.T, e.Hd, e.K, e.mean)
        st = TrainStep(dims, ends, w.n_train, e.n_feat, e.n_class, w.params, e.params, e.table)
        opt = Optimizer(st, OPTIM_RECORD if w.block == "pre" else OPTIM_BASELINE)
        X = torch.from_numpy(e.x).cuda()
        dY = torch.from_numpy(e.labels).cuda()
        del w.X

        def step():
            st.run(X, dY)
            opt.step()
    else:
        st = Stack(dims, w.n_train, w.cell_mask, w.params)
        X = to_device(w.X, w.dtype)
        dY = to_device(w.dY, w.dtype)
        del w.X, w.dY

        def step():
            st.forward(X)
            st.backward(dY)

    print(f"[bench] warmup {args.warmup}", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    # Headline: K steps with one event between consecutive steps and nothing else recorded, so
    # the per-step times have no profiling work inside; ms_per_step is their median.
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    print(f"[bench] timing {args.steps} steps", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    evs[0].record(stream)
    for i in range(args.steps):
        step()
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per_step = [evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)]
    ev_ms = sum(per_step)
    ms_per_step = float(np.median(per_step))
    # Roofline of the dominant kernel: a separate pass of the same steps with per-kernel events
    # on the stream the kernels run on (tfm.prof_*), after the headline timing.
    prof = {}
    prof_steps = min(args.steps, 10)
    prof_ms = None
    if not args.no_profile:
        print(f"[bench] per-kernel timing pass, {prof_steps} steps", file=sys.stderr, flush=True)
        tfm.prof_enable(True)
        pe0, pe1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        pe0.record(stream)
        for _ in range(prof_steps):
            step()
        pe1.record(stream)
        torch.cuda.synchronize()
        prof_ms = pe0.elapsed_time(pe1)
        prof = tfm.prof_collect()
        tfm.prof_enable(False)
    value = counts["cell_layers"] / (ms_per_step / 1e3)
    step_total = counts["flops_fwd_bwd"] / 3 if args.infer else counts["flops_fwd_bwd"]
    tflops = step_total / (ms_per_step / 1e3) / 1e12
    peak = PEAK_TFLOPS["mfma_bf16"] if w.dtype == "bf16" else PEAK_TFLOPS["mfma_f32"]

    roof = None
    steps_out = {}
    if prof:
        mfma_path = w.dtype == "bf16"
        fl = step_flops(w, tfm.prof_item_bwd_fused_rows(cfg["E"] // cfg["heads"]) if mfma_path
                        else 0)
        for name, (n, ms) in sorted(prof.items(), key=lambda kv: -kv[1][1]):
            steps_out[name] = {"launches": n, "avg_ms": round(ms / n, 5),
                               "share": round(ms / (prof_ms or 1), 4)}
        # step names are "<step>/<unit>", unit in {mfma, valu, hbm}
        dom = max((k for k in prof if k.split("/")[0] in fl), key=lambda k: prof[k][1],
                  default=None)
        if dom is not None:
            n, ms = prof[dom]
            avg_s = ms / n / 1e3
            f = fl[dom.split("/")[0]]
            if args.infer:
                # the context and query launches of a step differ in size: their flops sum to
                # the whole-table figure of each layer, so use flops over time per step
                f = f * cfg["layers"] * prof_steps / n
            achieved = f / avg_s / 1e12
            mfma = dom.endswith("/mfma")
            pk = peak if mfma else PEAK_TFLOPS["alu_f32"]
            roof = {"kernel": dom, "bound": "mfma" if mfma else "alu",
                    "achieved": round(achieved, 3), "peak": pk, "unit": "TFLOP/s",
                    "frac": round(achieved / pk, 5),
                    "traffic": measured_traffic(dom.split("/")[0], cfg["name"]),
                    "flops_per_launch": f, "avg_launch_ms": round(ms / n, 5)}

    out = {
        "metric": METRIC_INFER if args.infer else (METRIC_STEP if args.full_step else METRIC),
        "value": round(value, 1),
        "unit": "cells/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "ms_per_step_mean": round(ev_ms / args.steps, 4),
        "ms_per_step_min": round(min(per_step), 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": cfg["name"], "B": cfg["B"], "R": cfg["R"],
                   "n_train": str(cfg["n_train"]), "C": cfg["C"], "E": cfg["E"],
                   "heads": cfg["heads"], "H": cfg["H"], "layers": cfg["layers"],
                   "block": cfg.get("block", "post"), "thinking_rows": cfg.get("thinking", 0),
                   "seed": seed, "active_cell_layers": counts["cell_layers"]},
        "mode": "forward-only" if args.infer else (
            "training step" if args.full_step else "forward+backward"),
        "tflops": round(tflops, 3), "mfma_peak_frac": round(tflops / peak, 5),
        "wall_ms_per_step": round(wall * 1e3 / args.steps, 4),
        "roofline": roof, "steps_profile": steps_out, "profile_steps": prof_steps if prof else 0,
        "profile_ms_per_step": round(prof_ms / prof_steps, 4) if prof_ms else None,
        "git": git_rev(),
        "gpu": torch.cuda.get_device_name(0),
    }
    if args.infer:
        out["config"].update(context_rows=Rc, query_chunks=[b - a for a, b in spans])
    if args.full_step:
        e = ends_in
        out["config"].update(group_size=e.G, group_shifts=list(e.offsets), decoder_hidden=e.Hd,
                             classes=e.K, decoder_input="feature mean" if e.mean else "target")
        out["loss"] = float(st.loss[0].item())
        out["ends_ms_per_step"] = round(sum(
            v["avg_ms"] * v["launches"] for k, v in steps_out.items()
            if k.startswith(("encode_", "dec_"))) / args.steps, 4) if steps_out else None
        out["optimizer_ms_per_step"] = round(sum(
            v["avg_ms"] * v["launches"] for k, v in steps_out.items()
            if k.startswith(("clip_", "sfadamw", "muon_"))) / args.steps, 4) if steps_out else None
        out["optimizer"] = "schedule-free AdamW + Muon" if w.block == "pre" else \
            "schedule-free AdamW"
    del st, X, dY
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline (oracle)", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(args.config, seed, forward_only=args.infer)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
