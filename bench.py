#!/usr/bin/env python3
"""Throughput of the dynamic-batching hot path on one MI355X.

Default workload (the configuration the headline metric is quoted on): 256 complete
balanced binary trees of 256 leaves (130,816 nodes, depth 9), binary Tree-LSTM with
hidden size 256 in fp32, leaf inputs of dimension 256; one step = forward + backward
(upstream gradient on the roots, weight gradients accumulated) through the C ABI.
Inputs are synthetic and seeded, and resident in HBM before the timed region.

Prints ONE JSON line: nodes/s over the timed steps, the roofline of the dominant
kernel (algorithmic FLOPs per launch / average launch time, live HIP events), the
schedule time, and the CPU oracle timed on a bounded sample on this host.

    python bench.py [--steps K] [--warmup W] [--config 1..5] [--no-cpu]
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAKS = {  # MI355X datasheet, dense
    "f32_mfma_tflops": 157.3,
    "bf16_mfma_tflops": 2500.0,
    "hbm_gbs": 8000.0,
}


def flops_by_kernel(w, sched_host, table_grad: bool) -> dict:
    """Algorithmic FLOPs of one forward + backward, by kernel class (2 FLOPs per multiply-add)."""
    from paper_1702_02181_amd import gen
    H = w.hidden
    dt = "bf16" if w.dtype == "bf16" else "f32"
    out = {}

    def add(k, v):
        out[k] = out.get(k, 0.0) + float(v)

    rows_of_op = {}
    for op_id, rows in zip(sched_host["group_op"], sched_host["group_rows"]):
        rows_of_op[int(op_id)] = rows_of_op.get(int(op_id), 0) + int(rows)
    for op_id, rows in rows_of_op.items():
        op = w.ops[op_id]
        if op.kind == gen.KIND_EMBED:
            continue
        G = gen.NUM_GATES[op.kind]
        ps = w.params[op.param_set]
        k_in = (ps.in_dim if op.has_input else 0) + op.arity * H
        name = gen.KIND_NAMES[op.kind]
        add(f"cell_fwd.{name}.{dt}", 2.0 * rows * k_in * G * H)
        if w.backward:
            add(f"bwd_dx.{dt}", 2.0 * rows * G * H * (op.arity * H + (ps.in_dim if (op.has_input and table_grad) else 0)))
            add(f"wgrad.{dt}", 2.0 * rows * k_in * G * H)
    return out


def cpu_baseline(w, budget_s: float):
    """The oracle as it stands, single thread, on whole graphs of the workload until ~budget_s."""
    from threadpoolctl import threadpool_limits

    from oracle import evaluate as EV
    from paper_1702_02181_amd import gen
    from tests._helpers import oracle_batch, oracle_params

    P = oracle_params(w)
    nodes = 0
    graphs = 0
    t0 = time.perf_counter()
    with threadpool_limits(limits=1):
        while graphs < w.num_graphs and (time.perf_counter() - t0) < budget_s:
            sub = gen.subset(w, [graphs])
            b = oracle_batch(sub)
            f = EV.forward(b, P, w.hidden, w.leaf_table)
            if w.backward:
                EV.backward(b, P, w.hidden, w.leaf_table, f, sub.dh_roots.astype("float64"), None,
                            want_table_grad=False)
            nodes += sub.num_nodes
            graphs += 1
    dt = time.perf_counter() - t0
    return {"value": nodes / dt, "unit": "graph nodes/s", "cores": 1, "kind": "oracle",
            "sample": f"{graphs} of {w.num_graphs} graphs ({nodes} nodes), fp64 "
                      f"{'forward+backward' if w.backward else 'forward'}, {dt:.1f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=2)
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--profile-only", action="store_true", help="skip the oracle leg and the schedule timing")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the dynamic-batching path here is a single-GPU build "
              "(graphs would shard across GPUs with one all-reduce of weight gradients; not built).",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_1702_02181_amd import fold as F
    from paper_1702_02181_amd import gen
    from paper_1702_02181_amd.runner import DeviceRun

    torch.cuda.set_device(0)
    # achievable peaks on this GPU (MFMA loop, stream copy), next to the datasheet figures
    probes = {}
    try:
        probes["mfma_f32_tflops"] = round(F.fold_probe_mfma(F.FOLD_F32), 1)
        probes["mfma_bf16_tflops"] = round(F.fold_probe_mfma(F.FOLD_BF16), 1)
        nbytes = 1 << 30
        src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        probes["copy_gbs"] = round(F.fold_probe_copy(dst, src, nbytes), 1)
        del src, dst
    except Exception as e:  # probes are diagnostics; the bench line does not depend on them
        probes["error"] = str(e)
    print(f"[bench] probes {probes}", file=sys.stderr, flush=True)
    print(f"[bench] generating config {args.config}", file=sys.stderr, flush=True)
    w = gen.make_config(args.config)
    table_grad = args.config in (3, 5)  # trainable embedding tables; config 2 / 4 leaf rows are data
    dev = DeviceRun(w)
    host = dev.sched.host_groups()
    N = w.num_nodes

    # schedule time: fold_schedule end to end (validate, depth, sort, emit, read-back)
    sched_ms = []
    if not args.profile_only:
        for _ in range(5):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            s = F.Schedule(dev.graph_ptr, dev.node_op, dev.child_ptr, dev.child_idx, dev.node_input, dev.ops,
                           dev.leaf_rows)
            torch.cuda.synchronize()
            sched_ms.append((time.perf_counter() - t0) * 1e3)
            del s
    schedule_ms = statistics.median(sched_ms) if sched_ms else None

    if w.backward:
        dev.alloc_grads(table_grad)
        dev.set_upstream(w.dh_roots)

    def step():
        if w.backward:
            dev.zero_grads()
        dev.forward()
        if w.backward:
            dev.backward()

    print(f"[bench] N={N} levels={dev.sched.num_levels} groups={len(host['group_op'])} warmup={args.warmup}",
          file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = e0.elapsed_time(e1) / args.steps
    print(f"[bench] timed {args.steps} steps: {ms_per_step:.3f} ms/step", file=sys.stderr, flush=True)

    # per-kernel durations over a second timed region (event pair around every launch)
    F.fold_profile_enable(True)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    stats = F.fold_profile_read()
    F.fold_profile_enable(False)
    flops = flops_by_kernel(w, host, table_grad)
    kernels = {}
    for name, (launches, total_ms, max_ms) in stats.items():
        per_step_ms = total_ms / args.steps
        kernels[name] = {"launches_per_step": launches / args.steps, "ms_per_step": round(per_step_ms, 4),
                         "avg_launch_us": round(1e3 * total_ms / max(launches, 1), 2)}
        if name in flops:
            kernels[name]["tflops"] = round(flops[name] / (per_step_ms * 1e-3) / 1e12, 2)
    mfma_kernels = [k for k in kernels if k in flops]
    dom = max(mfma_kernels, key=lambda k: kernels[k]["ms_per_step"]) if mfma_kernels else None
    roofline = None
    if dom:
        peak = PEAKS["bf16_mfma_tflops"] if dom.endswith("bf16") else PEAKS["f32_mfma_tflops"]
        launches = stats[dom][0] / args.steps
        avg_s = (stats[dom][1] / args.steps) / launches * 1e-3
        per_launch = flops[dom] / launches
        ach = per_launch / avg_s / 1e12
        roofline = {"bound": "mfma", "kernel": dom, "achieved": round(ach, 2), "peak": peak, "unit": "TFLOP/s",
                    "frac": round(ach / peak, 4), "traffic": None,
                    "flops_per_launch": per_launch, "avg_launch_us": round(avg_s * 1e6, 2)}
    total_flops = sum(flops.values())
    step_peak = PEAKS["bf16_mfma_tflops"] if w.dtype == "bf16" else PEAKS["f32_mfma_tflops"]

    cpu = None
    if not args.no_cpu and not args.profile_only:
        print(f"[bench] oracle on host cores (~{args.cpu_seconds:.0f} s)", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, args.cpu_seconds)

    value = N / (ms_per_step * 1e-3)
    out = {
        "metric": "graph nodes/sec (TreeLSTM fwd+bwd, 1 GPU)",
        "value": round(value, 1),
        "unit": "graph nodes/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if w.dtype == "f32" else "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "graphs": w.num_graphs, "nodes": N, "levels": dev.sched.num_levels,
                   "hidden": w.hidden, "pass": "forward+backward" if w.backward else "forward"},
        "schedule_ms": None if schedule_ms is None else round(schedule_ms, 3),
        "peaks": {"datasheet": PEAKS, "measured": probes},
        "roofline": roofline,
        "step_mfma_frac": round(total_flops / (ms_per_step * 1e-3) / 1e12 / step_peak, 4),
        "kernels": kernels,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
