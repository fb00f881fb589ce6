"""Benchmark of the pooled embedding-bag hot path on one MI355X.

One step = one pass of the whole path over one batch: the forward pooled
lookup over every (bag, table) and, for the training configuration, the
sparse backward (key build, radix sort, segments, segmented reduce), queued
in that order on one stream.  (--overlap-index queues the backward's index
phase, which needs only the lookup ids, on a second stream beside the
forward instead; on MI355X that gains nothing, since the forward's
workgroups fill every CU and both are bound by the same per-CU memory
request rate.)  Inputs are seeded synthetic draws resident in HBM before
timing starts.  Prints one JSON line: whole-step lookups/s, the roofline of the
step's dominant kernel (and of the forward kernel) against HBM, per-phase
times, and the CPU oracle timed on a bounded sample of the same workload.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 5]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import workloads  # noqa: E402
from paper_2512_23236_amd import tbe  # noqa: E402

HBM_PEAK_GBS = 8000.0
DESCRIPTIONS = {
    1: "cfg1 forward: 1 fp32 table 10000x64, B=512, L~U{1..20}, uniform ids",
    2: "cfg2 forward: 26 fp16 tables (rows log-uniform 1e3..1e6) x128, B=2048, one-hot bags",
    3: "cfg3 forward: 100 fp16 tables (rows log-uniform 1e4..1e7, <=40 GB), dims {64,128,256}, "
       "B=16384, L=0 w.p. 0.02 else min(Poisson(30),200), Zipf(1.05) ids",
    4: "cfg4 forward: 40 bf16 tables 5e6x128 (51.2 GB), B=32768, L~Poisson(50), U(0,1) weights, Zipf(1.2) ids",
    5: "cfg5 training step on cfg3 shapes: forward + sparse backward (radix sort + segmented reduce) "
       "with grad_out N(0,1) fp32 [16384 x total_dim]",
}


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def forward_bytes(spec, offsets_host: np.ndarray, index_bytes: int = 8, out_bytes: int = 4) -> int:
    """Algorithmic bytes of one forward launch: each lookup reads its row
    (D_t * elem_size; for an 8-bit row-wise row its D_t codes and 8 bytes of
    scale and bias, not the padding) and its index (+ a 4-byte weight when
    weighted); each bag reads one offset and writes D_t outputs."""
    B = spec.B
    per_table_lookups = offsets_host[np.arange(1, spec.T + 1) * B] - offsets_host[np.arange(spec.T) * B]
    dims = spec.dims.astype(np.int64)
    read = dims + 8 if spec.dtype == "u8" else dims
    rows = int((per_table_lookups * read).sum()) * spec.elem_size
    n = int(offsets_host[-1])
    idx = index_bytes * n + (4 * n if spec.weighted else 0)
    bags = index_bytes * (spec.T * B + 1) + out_bytes * B * int(dims.sum())
    return rows + idx + bags


def compulsory_forward_bytes(spec, d, index_bytes: int = 8, out_bytes: int = 4) -> int:
    """Bytes one forward launch cannot avoid: every distinct row it looks up
    read once, every index (and weight) and offset read once, the output
    written once.  Under Zipf-skewed ids the per-lookup figure counts hot rows
    many times over; this one counts each once."""
    off = d["offsets"].cpu().numpy()
    B = spec.B
    rows = 0
    read = spec.dims.astype(np.int64) + 8 if spec.dtype == "u8" else spec.dims.astype(np.int64)
    for t in range(spec.T):
        s, e = int(off[t * B]), int(off[(t + 1) * B])
        if e > s:
            rows += int(torch.unique(d["indices"][s:e]).numel()) * int(read[t]) * spec.elem_size
    n = int(off[-1])
    return (rows + index_bytes * n + (4 * n if spec.weighted else 0) + index_bytes * (spec.T * B + 1)
            + out_bytes * B * spec.total_dim)


def host_info() -> dict:
    """CPU model, logical CPUs the process may use, and host RAM."""
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    ram = None
    try:
        for line in open("/proc/meminfo"):
            if line.startswith("MemTotal"):
                ram = int(line.split()[1]) * 1024
                break
    except OSError:
        pass
    return {"cpu_model": model, "cpus_available": len(os.sched_getaffinity(0)), "host_ram_bytes": ram}


def backward_bytes(spec, N: int, U: int, grad_floats: int, index_bytes: int = 8, grad_out_bytes: int = 4) -> int:
    """Compulsory bytes of one backward: indices and offsets read, the output
    gradient read once, int64 row ids, segment offsets and row offsets
    written, and the fp32 gradient rows written."""
    return (index_bytes * N + index_bytes * (spec.T * spec.B + 1) + grad_out_bytes * spec.B * spec.total_dim
            + 3 * 8 * (U + 1) + 4 * grad_floats)


def reduce_bytes(spec, N: int, grad_floats: int, carries_weight: bool, grad_out_bytes: int = 4) -> int:
    """Algorithmic bytes of one segmented-reduce launch: each sorted lookup's
    key and batch row (4 + 4 bytes, + 4 for its weight: the per-sample weight,
    or 1/L under mean pooling), the output gradient read once, and the fp32
    gradient rows written."""
    return ((8 + (4 if carries_weight else 0)) * N + grad_out_bytes * spec.B * spec.total_dim
            + 4 * grad_floats)


# Counter-derived HBM traffic per launch, with the hash of the kernel source it
# was measured on; a figure whose source has changed since is not reported.
KERNEL_SOURCES = {
    "forward_kernel": ["paper_2512_23236_amd/csrc/tbe_forward.hip", "paper_2512_23236_amd/csrc/tbe_internal.h"],
    "reduce_kernel": ["paper_2512_23236_amd/csrc/tbe_backward.hip", "paper_2512_23236_amd/csrc/tbe_internal.h"],
}


def source_hash(kernel: str) -> str:
    import hashlib
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_hit_rate(kernel: str, workload: str):
    """L2 (TCC) hit rate of the kernel from profiles/<kernel>_<workload>_tcc.md,
    if that file was written for the current kernel source."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_tcc.md")
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if ":" in line and line.startswith("- "):
            k, v = line[2:].split(":", 1)
            fields[k.strip()] = v.strip().strip("`")
    if fields.get("source_sha256") != source_hash(kernel):
        return None
    try:
        return float(fields["tcc_hit_rate"])
    except (KeyError, ValueError):
        return None


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch from profiles/<kernel>_<workload>_traffic.md
    (FETCH_SIZE and WRITE_SIZE, scaled by the copy-kernel calibration), if
    that file was written for the current kernel source."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.md")
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if ":" in line and line.startswith("- "):
            k, v = line[2:].split(":", 1)
            fields[k.strip()] = v.strip().strip("`")
    if fields.get("source_sha256") != source_hash(kernel):
        return None
    try:
        return int(fields["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_baseline(spec, d, target_s: float, pooling: str = "sum", training: bool = False):
    """The CPU oracle on a bounded sample: the first b_s bags of every table,
    their rows copied into compact host tables; b_s is sized so the oracle
    runs for roughly target_s seconds.  With training, the sample's backward
    (sort and segments, then the gradient rows against grad_out's first b_s
    rows) is timed with its forward, as the GPU step does both."""
    import oracle

    off = d["offsets"].cpu().numpy()
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))

    def sample(bs):
        tabs, idx_parts, lens, rows, w_parts = [], [], [], [], []
        for t in range(spec.T):
            s, e = int(off[t * spec.B]), int(off[t * spec.B + bs])
            idx = d["indices"][s:e].cpu().numpy().astype(np.int64)
            uniq, inv = np.unique(idx, return_inverse=True)
            R, E = int(spec.rows[t]), int(spec.row_elems[t])
            base = int(spec.table_offsets[t])
            full = d["tables"][base: base + R * E].view(R, E)
            sel = full[torch.as_tensor(uniq, device=full.device)].cpu() if len(uniq) else full[:1].cpu()
            tabs.append(sel.numpy() if spec.dtype in ("f32", "u8") else sel.view(torch.int16).numpy())
            rows.append(max(len(uniq), 1))
            idx_parts.append(inv.astype(np.int64))
            lens.append(np.diff(off[t * spec.B: t * spec.B + bs + 1]))
            if spec.weighted:
                w_parts.append(d["weights"][s:e].cpu().numpy())
        offsets = np.concatenate([[0], np.cumsum(np.concatenate(lens))]).astype(np.int64)
        indices = np.concatenate(idx_parts)
        w = np.concatenate(w_parts) if spec.weighted else None
        return tabs, rows, indices, offsets, w

    def run(bs):
        tabs, rows, indices, offsets, w = sample(bs)
        g = d["grad_out"][:bs].float().cpu().numpy() if training else None
        t0 = time.perf_counter()
        oracle.forward(rows, spec.dims, spec.dtype, tabs, indices, offsets, bs, w, pooling=pooling)
        if training:
            seg = oracle.backward_segments(rows, spec.dims, indices, offsets, bs)
            oracle.backward_rows(rows, spec.dims, offsets, bs, g, seg, w, pooling=pooling)
        return time.perf_counter() - t0, indices.size

    bs = max(1, min(spec.B, 64))
    dt, n = run(bs)
    while dt < target_s / 4 and bs < spec.B:
        bs = min(spec.B, int(bs * max(2.0, min(16.0, target_s / max(dt, 1e-3) * 0.8))))
        dt, n = run(bs)
    return {"value": n / dt, "unit": "lookups/s", "cores": threads, "kind": "oracle", **host_info(),
            "sample": (f"forward + backward (sort single-threaded; forward and gradient rows OpenMP) "
                       if training else "forward (OpenMP over bags) ")
                      + f"over the first {bs} bags of each of the {spec.T} tables ({n} lookups, {dt:.1f} s, "
                        f"binary64)"}


def weight_grad_bytes(spec, offsets_host: np.ndarray) -> int:
    """Algorithmic bytes of one per-sample-weight-gradient launch: each lookup
    reads its row (D_t * elem_size) and int64 index and writes one fp32; each
    bag reads its offset and its fp32 grad_out slice (4 * D_t) once."""
    B = spec.B
    per_table = offsets_host[np.arange(1, spec.T + 1) * B] - offsets_host[np.arange(spec.T) * B]
    dims = spec.dims.astype(np.int64)
    n = int(offsets_host[-1])
    return int((per_table * dims).sum()) * spec.elem_size + 12 * n + 8 * (spec.T * B + 1) + 4 * B * int(dims.sum())


def bench_weight_grad(args, spec, dev):
    spec = __import__("dataclasses").replace(spec, grad=True)
    log(f"[bench] weight_grad on {spec.name}: {spec.table_bytes / 1e9:.2f} GB of tables")
    d = workloads.gen_all(spec, dev)
    torch.cuda.synchronize()
    plan = tbe.Plan(spec.rows, spec.dims, spec.torch_dtype, spec.B, bounds_check=True, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    gw = torch.empty(d["N"], dtype=torch.float32, device=dev)
    for _ in range(args.warmup):
        tbe.weight_grad(plan, d["tables"], d["grad_out"], d["indices"], d["offsets"], out=gw, status=status)
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for e0, e1 in evs:
        e0.record()
        tbe.weight_grad(plan, d["tables"], d["grad_out"], d["indices"], d["offsets"], out=gw, status=status)
        e1.record()
    torch.cuda.synchronize()
    if int(status.item()) != 0:
        raise RuntimeError(f"device status {int(status.item())}")
    ms = float(np.mean([e0.elapsed_time(e1) for e0, e1 in evs]))
    nbytes = weight_grad_bytes(spec, d["offsets"].cpu().numpy())
    gbs = nbytes / (ms * 1e-3) / 1e9
    print(json.dumps({
        "metric": "per-sample-weight gradient: lookups/s and effective HBM GB/s", "op": "weight_grad",
        "value": d["N"] / (ms * 1e-3), "unit": "lookups/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "dtype": "f32",
        "data": "synthetic (seeded counter-based draws; no production data)",
        "config": {"workload": f"{DESCRIPTIONS[args.config]}; grad_out N(0,1) fp32", "lookups": d["N"]},
        "roofline": {"bound": "hbm", "kernel": "weight_grad_kernel", "achieved": gbs, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": gbs / HBM_PEAK_GBS, "traffic": None, "algorithmic_bytes": nbytes},
    }), flush=True)


def bench_optimizer(args, spec, dev):
    """The optimizer step alone on the sparse gradient of one backward of the
    training configuration (cfg5: 7 M unique rows of 64-256 columns)."""
    spec = __import__("dataclasses").replace(spec, grad=True)
    log(f"[bench] {args.op} on the sparse gradient of {spec.name}")
    d = workloads.gen_all(spec, dev)
    plan = tbe.Plan(spec.rows, spec.dims, spec.torch_dtype, spec.B, bounds_check=True, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    g = tbe.backward(plan, d["grad_out"], d["indices"], d["offsets"], d["weights"], status=status)
    torch.cuda.synchronize()
    U = g.num_unique()
    del d["grad_out"]
    kind = tbe.SGD if args.op == "sgd" else tbe.ROWWISE_ADAGRAD
    state = torch.zeros(int(spec.rows.sum()), dtype=torch.float32, device=dev) if kind else None
    tables = d["tables"]
    lr = 1e-3  # small: repeated steps keep the tables in range

    def once():
        tbe.apply_gradient(plan, tables, g, kind, lr, 1e-8, state=state, max_unique=U)

    for _ in range(args.warmup):
        once()
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for e0, e1 in evs:
        e0.record()
        once()
        e1.record()
    torch.cuda.synchronize()
    if int(status.item()) != 0:
        raise RuntimeError(f"device status {int(status.item())}")
    ms = float(np.mean([e0.elapsed_time(e1) for e0, e1 in evs]))
    floats = int(g.grad_row_offsets[U].item())
    # algorithmic bytes: each listed row's table elements read and written, its
    # fp32 gradient row read, its id and offset read (+ the state word read and written)
    nbytes = floats * (2 * spec.elem_size + 4) + 16 * U + (8 * U if kind else 0)
    gbs = nbytes / (ms * 1e-3) / 1e9
    print(json.dumps({
        "metric": f"sparse {args.op} step: rows/s and effective HBM GB/s", "op": args.op,
        "value": U / (ms * 1e-3), "unit": "rows/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms, "higher_is_better": True, "dtype": "f32",
        "data": "synthetic (seeded counter-based draws; no production data)",
        "config": {"workload": f"{args.op} on the sparse gradient of one {DESCRIPTIONS[args.config]}",
                   "unique_rows": U, "gradient_floats": floats},
        "roofline": {"bound": "hbm", "kernel": "apply_kernel", "achieved": gbs, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": gbs / HBM_PEAK_GBS, "traffic": None, "algorithmic_bytes": nbytes},
    }), flush=True)


def bench_step_apply(args, spec, dev):
    """The training step with the optimizer: forward, the backward's index
    phase, and the reduce phase with the SGD or row-wise Adagrad step made by
    the same kernels (tbe_backward_reduce_apply); beside it, timed in the same
    run, the two-pass form (tbe_backward, then tbe_apply_gradient)."""
    spec = __import__("dataclasses").replace(spec, grad=True)
    kind = tbe.SGD if args.op == "step_sgd" else tbe.ROWWISE_ADAGRAD
    log(f"[bench] {args.op} on {spec.name}")
    d = workloads.gen_all(spec, dev)
    N = d["N"]
    plan = tbe.Plan(spec.rows, spec.dims, spec.torch_dtype, spec.B, bounds_check=True, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    out = torch.empty((spec.B, plan.total_dim), dtype=torch.float32, device=dev)
    bounds = d["offsets"][:: spec.B].cpu().numpy().astype(np.int64)
    cap = int((np.diff(bounds) * spec.dims.astype(np.int64)).sum())
    grads = tbe.SparseGrad(torch.empty(cap, dtype=torch.float32, device=dev),
                           torch.empty(N, dtype=torch.int64, device=dev), torch.empty(N + 1, dtype=torch.int64, device=dev),
                           torch.empty(N + 1, dtype=torch.int64, device=dev), torch.zeros(1, dtype=torch.int64, device=dev))
    workspace = torch.empty(tbe.backward_workspace_bytes(plan, N), dtype=torch.uint8, device=dev)
    state = torch.zeros(int(spec.rows.sum()), dtype=torch.float32, device=dev) if kind else None
    tables = d["tables"]
    lr = 1e-3  # small: repeated steps keep the tables in range

    def fused():
        tbe.forward(plan, tables, d["indices"], d["offsets"], d["weights"], out=out, status=status)
        tbe.backward_index(plan, d["indices"], d["offsets"], d["weights"], workspace=workspace, status=status,
                           outputs=grads)
        tbe.backward_reduce_apply(plan, d["grad_out"], N, workspace, grads, tables, kind, lr, 1e-8, state=state,
                                  per_sample_weights=d["weights"], status=status)

    def two_pass():
        tbe.forward(plan, tables, d["indices"], d["offsets"], d["weights"], out=out, status=status)
        tbe.backward(plan, d["grad_out"], d["indices"], d["offsets"], d["weights"], workspace=workspace,
                     status=status, outputs=grads)
        tbe.apply_gradient(plan, tables, grads, kind, lr, 1e-8, state=state, max_unique=N)

    def timed(fn):
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            fn()
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) * 1e3 / args.steps

    ms_two = timed(two_pass)
    ms = timed(fused)
    if int(status.item()) != 0:
        raise RuntimeError(f"device status {int(status.item())}")
    print(json.dumps({
        "metric": f"training step with sparse {'SGD' if kind == tbe.SGD else 'row-wise Adagrad'}: lookups/s",
        "op": args.op, "value": N / (ms * 1e-3), "unit": "lookups/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "dtype": "f32",
        "data": "synthetic (seeded counter-based draws; no production data)",
        "config": {"workload": f"{DESCRIPTIONS[args.config]}; then the optimizer step on the listed rows",
                   "lookups": N},
        "two_pass_ms_per_step": ms_two, "saved_ms": ms_two - ms,
    }), flush=True)


def bench_map_ids(args, dev, n_unique=10000, batch=50000):
    d = workloads.gen_map_ids(n_unique, batch, device=dev)
    out = torch.empty_like(d["values"])
    for _ in range(args.warmup):
        tbe.map_ids(d["values"], d["mapping"], out=out)
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for e0, e1 in evs:
        e0.record()
        tbe.map_ids(d["values"], d["mapping"], out=out)
        e1.record()
    torch.cuda.synchronize()
    ms = float(np.mean([e0.elapsed_time(e1) for e0, e1 in evs]))
    # algorithmic bytes: each value read and its id written (int64), the mapping read once
    nbytes = 16 * batch + 8 * int(d["mapping"].numel())
    gbs = nbytes / (ms * 1e-3) / 1e9
    res = {
        "metric": "MapId preprocessing: values/s", "op": "map_ids", "value": batch / (ms * 1e-3),
        "unit": "values/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "dtype": "int64", "data": "synthetic (seeded counter-based draws)",
        "config": {"workload": f"MapId: {n_unique} known ids x {batch} values, 80% known"},
        "roofline": {"bound": "hbm", "kernel": "map_ids_kernel", "achieved": gbs, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": gbs / HBM_PEAK_GBS, "traffic": None, "algorithmic_bytes": nbytes},
        "context": "launch-bound at this size: the evaluation's shapes move under 1 MB",
    }
    if not args.no_cpu_baseline:
        import oracle
        v, m = d["values"].cpu().numpy(), d["mapping"].cpu().numpy()
        t0 = time.perf_counter()
        oracle.map_ids(v, m)
        dt = time.perf_counter() - t0
        res["cpu_baseline"] = {"value": batch / dt, "unit": "values/s",
                               "cores": int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1)),
                               "kind": "oracle", "sample": f"the whole workload ({batch} values, {dt:.2f} s)"}
    print(json.dumps(res), flush=True)


def variant_tag(args, spec) -> str:
    """Suffix naming the non-default options (traffic summaries are per variant)."""
    tag = ""
    if args.table_dtype and args.table_dtype != workloads.make_config(args.config, args.seed).dtype:
        tag += f"_{spec.dtype}"
    if args.pooling != "sum":
        tag += f"_{args.pooling}"
    if args.index_type != "i64":
        tag += f"_{args.index_type}"
    if args.out_dtype != "f32":
        tag += f"_out{args.out_dtype}"
    if args.train and not workloads.make_config(args.config, args.seed).grad:
        tag += "_train"
    return tag


def variant_text(args, spec) -> str:
    parts = []
    if args.table_dtype and args.table_dtype != workloads.make_config(args.config, args.seed).dtype:
        parts.append(f"tables redrawn as {spec.dtype}" + (" (8-bit row-wise: codes + fp32 scale/bias per row)"
                                                         if spec.dtype == "u8" else ""))
    if args.pooling != "sum":
        parts.append(f"{args.pooling} pooling")
    if args.index_type != "i64":
        parts.append("int32 indices and offsets")
    if args.out_dtype != "f32":
        parts.append(f"{args.out_dtype} output" + (" and grad_out" if spec.grad else ""))
    if args.train and not workloads.make_config(args.config, args.seed).grad:
        parts.append("training step (forward, backward" + (", per-sample weights' gradient)" if spec.weighted else ")")
                     + "; grad_out N(0,1)")
    return ("; " + ", ".join(parts)) if parts else ""


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=5)
    ap.add_argument("--seed", type=int, default=None)
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--flushed-steps", type=int, default=5,
                    help="extra steps, each after writing 1 GiB to evict L2 and the Infinity Cache, reported "
                         "as the secondary (cold-cache) timing; 0 skips them")
    ap.add_argument("--op", default="step", choices=["step", "weight_grad", "map_ids", "sgd", "adagrad", "step_sgd",
                                                     "step_adagrad"],
                    help="step: forward (+ backward for cfg5), the default; weight_grad: the per-sample-weight "
                         "gradient alone (use --config 4); map_ids: the MapId preprocessing step at the "
                         "evaluation's largest shape (10000 ids x 50000 values); sgd / adagrad: the optimizer "
                         "step alone, on the sparse gradient of one cfg5 backward; step_sgd / step_adagrad: the "
                         "training step with the optimizer made by the backward's reduce kernels, beside the "
                         "two-pass form")
    ap.add_argument("--graph", action="store_true",
                    help="also time the step captured in a HIP graph and replayed (reported under 'graph')")
    ap.add_argument("--overlap-index", action="store_true",
                    help="queue the backward's index phase on a second stream beside the forward")
    ap.add_argument("--train", action="store_true",
                    help="time the training step on any configuration: forward and backward, and with "
                         "per-sample weights also their gradient (cfg5 is a training step already)")
    ap.add_argument("--pooling", default="sum", choices=["sum", "mean"])
    ap.add_argument("--index-type", default="i64", choices=["i64", "i32"],
                    help="integer type of indices and offsets")
    ap.add_argument("--out-dtype", default="f32", choices=["f32", "f16", "bf16"],
                    help="element type of the forward output")
    ap.add_argument("--table-dtype", default=None, choices=["f32", "f16", "bf16", "u8"],
                    help="redraw the configuration's tables in this type (u8: 8-bit row-wise)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="only copy a device buffer of this size 3 times (calibrates the HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); the table-wise sharding over "
              "several GPUs exists as a design, not as code", file=sys.stderr)
        sys.exit(2)

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    if args.copy_probe_mib:
        n = args.copy_probe_mib << 20
        src = torch.ones(n // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": n, "copies": 3}), flush=True)
        return
    if args.op == "map_ids":
        return bench_map_ids(args, dev)
    spec = workloads.make_config(args.config, args.seed)
    if args.table_dtype:
        spec = __import__("dataclasses").replace(spec, dtype=args.table_dtype)
    if args.pooling == "mean" and spec.weighted:
        spec = __import__("dataclasses").replace(spec, weighted=False)  # mean pooling takes no weights
    if args.train:
        spec = __import__("dataclasses").replace(spec, grad=True)
    if args.op == "weight_grad":
        return bench_weight_grad(args, spec, dev)
    if args.op in ("sgd", "adagrad"):
        return bench_optimizer(args, spec, dev)
    if args.op in ("step_sgd", "step_adagrad"):
        return bench_step_apply(args, spec, dev)
    log(f"[bench] generating {spec.name}: {spec.table_bytes / 1e9:.2f} GB of tables")
    t0 = time.time()
    d = workloads.gen_all(spec, dev)
    index_dtype = torch.int32 if args.index_type == "i32" else torch.int64
    if args.index_type == "i32":
        d["indices"] = d["indices"].to(torch.int32)
        d["offsets"] = d["offsets"].to(torch.int32)
    out_dtype = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[args.out_dtype]
    torch.cuda.synchronize()
    log(f"[bench] inputs ready in {time.time() - t0:.1f} s, N = {d['N']}")
    plan = tbe.Plan(spec.rows, spec.dims, spec.torch_dtype, spec.B, bounds_check=True, device=dev,
                    pooling=args.pooling, index_dtype=index_dtype, out_dtype=out_dtype)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    out = torch.empty((spec.B, plan.total_dim), dtype=out_dtype, device=dev)
    if spec.grad and out_dtype != torch.float32:
        d["grad_out"] = d["grad_out"].to(out_dtype)  # the gradient of out has out's type
    training = spec.grad
    # with per-sample weights the training step also takes their gradient
    wgrad = training and spec.weighted
    gw = torch.empty(d["N"], dtype=torch.float32, device=dev) if wgrad else None
    grads = None
    side = torch.cuda.Stream(dev)  # the backward's index phase (default priority, like the main stream)
    if training:
        N = d["N"]
        bounds = d["offsets"][:: spec.B].cpu().numpy().astype(np.int64)
        cap = int((np.diff(bounds) * spec.dims.astype(np.int64)).sum())
        grads = tbe.SparseGrad(torch.empty(cap, dtype=torch.float32, device=dev),
                               torch.empty(N, dtype=torch.int64, device=dev),
                               torch.empty(N + 1, dtype=torch.int64, device=dev),
                               torch.empty(N + 1, dtype=torch.int64, device=dev),
                               torch.zeros(1, dtype=torch.int64, device=dev))
        workspace = torch.empty(tbe.backward_workspace_bytes(plan, N), dtype=torch.uint8, device=dev)
        log(f"[bench] backward workspace {workspace.numel() / 1e9:.2f} GB, grad_rows capacity {cap / 2.5e8:.2f} GB")

    def forward(ev=None):
        if ev is not None:
            ev[0].record()
        tbe.forward(plan, d["tables"], d["indices"], d["offsets"], d["weights"], out=out, status=status)
        if ev is not None:
            ev[1].record()

    def index_phase(ev=None):
        tbe.backward_index(plan, d["indices"], d["offsets"], d["weights"], workspace=workspace, status=status,
                           outputs=grads, events=ev)

    def reduce_phase(ev=None):
        tbe.backward_reduce(plan, d["grad_out"], d["N"], workspace, grads, per_sample_weights=d["weights"],
                            status=status, events=ev)

    def overlapped_step(ev=None):
        """The index phase on the side stream beside the forward, the reduce
        after both.  ev: forward (2), index phase (4) and reduce phase (3) events."""
        if not training:
            return forward(ev)
        main = torch.cuda.current_stream(dev)
        side.wait_stream(main)  # the previous step's reduce has read the workspace
        with torch.cuda.stream(side):
            index_phase(None if ev is None else ev[2:6])
        forward(ev)
        main.wait_stream(side)
        reduce_phase(None if ev is None else ev[6:9])
        if wgrad:
            weight_grad_phase(None if ev is None else ev[9:11])

    def weight_grad_phase(ev=None):
        if ev is not None:
            ev[0].record()
        tbe.weight_grad(plan, d["tables"], d["grad_out"], d["indices"], d["offsets"], out=gw, status=status)
        if ev is not None:
            ev[1].record()

    def serial_step(ev=None):
        """Forward, index phase, reduce phase (and the weights' gradient) in
        order on one stream."""
        forward(ev)
        if training:
            index_phase(None if ev is None else ev[2:6])
            reduce_phase(None if ev is None else ev[6:9])
        if wgrad:
            weight_grad_phase(None if ev is None else ev[9:11])

    step = overlapped_step if args.overlap_index else serial_step

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    if int(status.item()) != 0:
        raise RuntimeError(f"device status {int(status.item())}")

    nev = 2 + (7 if training else 0) + (2 if wgrad else 0)
    evs = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(nev)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1e3 / args.steps
    overlapped_fwd = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    sev = evs
    if args.overlap_index:
        # a serial pass as well: every part alone on one stream (kernel
        # durations for the rooflines)
        sev = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(nev)) for _ in range(args.steps)]
        for i in range(args.steps):
            serial_step(sev[i])
        torch.cuda.synchronize()
    fwd_ms = [e[0].elapsed_time(e[1]) for e in sev]
    fwd_avg = float(np.mean(fwd_ms))
    N = d["N"]
    off_host = d["offsets"].cpu().numpy().astype(np.int64)
    ib = 4 if args.index_type == "i32" else 8
    ob = 4 if args.out_dtype == "f32" else 2
    fbytes = forward_bytes(spec, off_host, ib, ob)
    cbytes = compulsory_forward_bytes(spec, d, ib, ob)
    achieved = fbytes / (fwd_avg * 1e-3) / 1e9

    res = {
        "metric": "pooled lookups/sec + effective HBM GB/s (fraction of 8 TB/s peak), fwd and bwd",
        "value": N / (ms_per_step * 1e-3),
        "unit": "lookups/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded counter-based draws; no production data)",
        "config": {"workload": DESCRIPTIONS[args.config] + variant_text(args, spec), "tables": spec.T,
                   "batch": spec.B, "table_dtype": spec.dtype, "lookups": N, "table_bytes": spec.table_bytes,
                   "total_dim": plan.total_dim, "seed": spec.seed, "training": training,
                   "pooling": args.pooling, "index_type": args.index_type, "out_dtype": args.out_dtype,
                   "schedule": ("forward, then the backward's index and reduce phases"
                                + (", then the per-sample weights' gradient" if wgrad else "") + ", on one stream"
                                if training and not args.overlap_index else
                                "backward index phase on a second stream beside the forward, then the reduce"
                                if training else "forward only")},
        "forward": {"ms": fwd_avg, "ms_p10": float(np.percentile(fwd_ms, 10)),
                    "ms_p90": float(np.percentile(fwd_ms, 90)), "lookups_per_s": N / (fwd_avg * 1e-3),
                    "algorithmic_bytes": fbytes, "effective_GBps": achieved,
                    "frac_of_hbm_peak": achieved / HBM_PEAK_GBS, "compulsory_bytes": cbytes,
                    "compulsory_GBps": cbytes / (fwd_avg * 1e-3) / 1e9,
                    "compulsory_frac_of_hbm_peak": cbytes / (fwd_avg * 1e-3) / 1e9 / HBM_PEAK_GBS,
                    "ms_in_timed_steps": overlapped_fwd},
    }
    workload = f"cfg{args.config}" + variant_tag(args, spec)

    def roof(kernel, ms, nbytes, extra=None):
        traffic = measured_traffic(kernel, workload)
        gbs = nbytes / (ms * 1e-3) / 1e9
        r = {"bound": "hbm", "kernel": kernel, "ms": ms, "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
             "frac": gbs / HBM_PEAK_GBS, "traffic": traffic, "algorithmic_bytes": nbytes,
             # the same time against the bytes the counters saw move beyond L2
             "traffic_GBps": None if traffic is None else traffic / (ms * 1e-3) / 1e9,
             "traffic_frac": None if traffic is None else traffic / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
             "l2_hit_rate": measured_hit_rate(kernel, workload)}
        r.update(extra or {})
        return r

    rf = {"forward_kernel": roof("forward_kernel", fwd_avg, fbytes,
                                 {"compulsory_bytes": cbytes,
                                  "compulsory_frac": cbytes / (fwd_avg * 1e-3) / 1e9 / HBM_PEAK_GBS})}
    if training:
        idx_ms = [e[2].elapsed_time(e[5]) for e in sev]
        red_ph = [e[6].elapsed_time(e[7]) for e in sev]
        comb_ph = [e[7].elapsed_time(e[8]) for e in sev]
        phase_ms = {"keys": [e[2].elapsed_time(e[3]) for e in sev], "sort": [e[3].elapsed_time(e[4]) for e in sev],
                    "segments": [e[4].elapsed_time(e[5]) for e in sev], "reduce": red_ph, "combine": comb_ph}
        bwd_ms = [a + b + c for a, b, c in zip(idx_ms, red_ph, comb_ph)]
        bwd_avg = float(np.mean(bwd_ms))
        U = grads.num_unique()
        gro_total = int(grads.grad_row_offsets[U].item())
        bbytes = backward_bytes(spec, N, U, gro_total, ib, ob)
        res["backward"] = {"ms": bwd_avg, "ms_p10": float(np.percentile(bwd_ms, 10)),
                           "ms_p90": float(np.percentile(bwd_ms, 90)), "lookups_per_s": N / (bwd_avg * 1e-3),
                           "unique_rows": U, "compulsory_bytes": bbytes,
                           "effective_GBps": bbytes / (bwd_avg * 1e-3) / 1e9,
                           "frac_of_hbm_peak": bbytes / (bwd_avg * 1e-3) / 1e9 / HBM_PEAK_GBS,
                           "phases_ms": {k: float(np.mean(v)) for k, v in phase_ms.items()},
                           "serial_step_ms": fwd_avg + bwd_avg}
        if wgrad:
            wg_ms = [e[9].elapsed_time(e[10]) for e in sev]
            res["weight_grad"] = {"ms": float(np.mean(wg_ms)), "lookups_per_s": N / (float(np.mean(wg_ms)) * 1e-3)}
            res["backward"]["serial_step_ms"] += res["weight_grad"]["ms"]
        red_ms = float(np.mean(red_ph))
        rbytes = reduce_bytes(spec, N, gro_total, spec.weighted or args.pooling == "mean", ob)
        rf["reduce_kernel"] = roof("reduce_kernel", red_ms, rbytes)
    # the roofline of the step's dominant kernel (the longest average launch)
    res["roofline"] = max(rf.values(), key=lambda r: r["ms"])
    res["roofline_forward"] = rf["forward_kernel"]
    if args.graph:
        # the same serial step captured once in a HIP graph and replayed (the
        # library queues only kernels, so a step is graph nodes end to end);
        # the saving is the host launch overhead between the step's kernels
        warm = torch.cuda.Stream(dev)
        warm.wait_stream(torch.cuda.current_stream(dev))
        with torch.cuda.stream(warm):
            serial_step()
        torch.cuda.current_stream(dev).wait_stream(warm)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            serial_step()
        graph.replay()
        torch.cuda.synchronize()
        g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        g0.record()
        for _ in range(args.steps):
            graph.replay()
        g1.record()
        torch.cuda.synchronize()
        res["graph"] = {"steps": args.steps, "step_ms": g0.elapsed_time(g1) / args.steps,
                        "eager_step_ms": ms_per_step}
        del graph
    if args.flushed_steps > 0:
        # secondary timing: every step starts with cold caches (1 GiB written
        # first, outside the timed events), parts serial
        junk = torch.empty(1 << 28, dtype=torch.float32, device=dev)
        fl = []
        for i in range(args.flushed_steps):
            junk.fill_(float(i))
            ev = tuple(torch.cuda.Event(enable_timing=True) for _ in range(nev))
            serial_step(ev)
            torch.cuda.synchronize()
            fl.append((ev[0].elapsed_time(ev[1]), ev[2].elapsed_time(ev[8]) if training else 0.0,
                       ev[9].elapsed_time(ev[10]) if wgrad else 0.0))
        del junk
        fw = [x[0] for x in fl]
        res["flushed"] = {"steps": args.flushed_steps, "forward_ms": float(np.median(fw)),
                          "forward_frac_of_hbm_peak": fbytes / (float(np.median(fw)) * 1e-3) / 1e9 / HBM_PEAK_GBS}
        if training:
            res["flushed"]["backward_ms"] = float(np.median([x[1] for x in fl]))
            res["flushed"]["serial_step_ms"] = float(np.median([x[0] + x[1] + x[2] for x in fl]))
        if wgrad:
            res["flushed"]["weight_grad_ms"] = float(np.median([x[2] for x in fl]))
    if int(status.item()) != 0:
        raise RuntimeError(f"device status {int(status.item())}")
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a sample")
        res["cpu_baseline"] = cpu_baseline(spec, d, args.cpu_seconds, args.pooling, training)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
