#!/usr/bin/env python3
"""Throughput of the dynamic-batching hot path on one MI355X.

Default workload (the configuration the headline metric is quoted on): 256 complete
balanced binary trees of 256 leaves (130,816 nodes, depth 9), binary Tree-LSTM with
hidden size 256 in fp32, leaf inputs of dimension 256; one step = forward + backward
(upstream gradient on the roots, weight gradients accumulated) through the C ABI.
Inputs are synthetic and seeded, and resident in HBM before the timed region.

Prints ONE JSON line: nodes/s over the timed steps, the roofline of the dominant
kernel (algorithmic FLOPs per launch / average launch time, live HIP events), the
schedule time, and the CPU oracle timed on a bounded sample on this host.  A step is
one replay of the whole forward + backward recorded as a HIP graph (gradients zeroed
inside it); the same step issued call by call is timed beside it.

    python bench.py [--steps K] [--warmup W] [--config 1..5] [--no-cpu]
    python bench.py --traffic-from FETCH.csv WRITE.csv [--traffic-kernel CLASS]
        turns two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) of this bench into the
        HBM-traffic record that profiles/ keeps for the dominant kernel class
"""
from __future__ import annotations

import argparse
import collections
import csv
import glob
import hashlib
import json
import os
import re
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


# Sources whose code decides a kernel class's kernels: a traffic record is valid only while they are
# unchanged.
CLASS_SOURCES = {
    "cell_fwd": ("cells.hip", "dma.h", "mfma.h", "wide.h", "common.h", "internal.h"),
    "bwd_dx": ("cells.hip", "dma.h", "mfma.h", "wide.h", "common.h", "internal.h"),
    "wgrad": ("wgrad.hip", "dma.h", "mfma.h", "wide.h", "common.h", "internal.h"),
}
COPY_KERNEL = "k_probe_copy"
TRAFFIC_TAG = "traffic-record:"
KIND_IDS = {"embed": 0, "treernn": 1, "treelstm": 2, "lstm": 3, "proj": 4}
# template kind ids of a class's kernels: Tree-LSTM leaves run as their own kind (live gates only), the library's
# internal kind kTreeLstmLeaf = 8 (after the ABI's kinds 0-7)
KERNEL_KINDS = {"treelstm": (2, 8)}
CTYPE = {"f32": "float", "bf16": "unsigned short"}


def class_of(name: str) -> str:
    return name.split(".")[0]


def rocprof_role(kernel_class: str, name: str):
    """Role of a rocprofv3 kernel name in one launch of a library kernel class ("cell_fwd.treelstm.f32",
    "bwd_dx.bf16", "wgrad.f32"): "main" (exactly one dispatch per launch of the class), "extra" (the
    K-split epilogue or reduction that belongs to it) or None."""
    parts = kernel_class.split(".")
    cls, dt = parts[0], CTYPE[parts[-1]]
    if cls == "cell_fwd":
        kinds = "|".join(str(k) for k in KERNEL_KINDS.get(parts[1], (KIND_IDS[parts[1]],)))
        if re.search(rf"k_cell_fwd(_w)?<{dt}, ({kinds})[,>]", name):
            return "main"
        if re.search(rf"k_cell_epi<{dt}, ({kinds})>", name):
            return "extra"
    elif cls == "bwd_dx":
        if re.search(rf"k_bwd_dx(2|_w)<{dt}[,>]", name):
            return "main"
    elif cls == "wgrad":
        if re.search(r"k_wgrad_(f32|bf16)(_w)?\b|k_wgrad<", name):
            return "main"
    return None


def sources_sha256(cls: str) -> str:
    h = hashlib.sha256()
    for f in CLASS_SOURCES[cls]:
        with open(os.path.join(ROOT, "paper_1702_02181_amd", "csrc", f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()


def traffic_record(kernel: str, workload: str):
    """The HBM-traffic record of `kernel` on `workload` kept under profiles/, if the kernel's sources are
    unchanged since the counters were taken; else None."""
    want = sources_sha256(class_of(kernel))
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md"))):
        for line in open(path):
            if TRAFFIC_TAG not in line:
                continue
            rec = json.loads(line.split(TRAFFIC_TAG, 1)[1].strip().strip("`").strip())
            if rec.get("kernel") == kernel and rec.get("workload") == workload and rec.get("sources_sha256") == want:
                return rec
    return None


def traffic_from_counters(fetch_csv: str, write_csv: str, kernel: str, workload: str) -> dict:
    """HBM bytes per launch of a kernel class from a FETCH_SIZE run and a WRITE_SIZE run (rocprofv3 csv,
    KiB per dispatch), each scaled by what the same counter reads for the copy probe, which reads and
    writes PROBE_BYTES per dispatch.  Launches are counted by the class's main kernel."""
    cls = class_of(kernel)
    out = {"kernel": kernel, "workload": workload}
    for what, path in (("fetch", fetch_csv), ("write", write_csv)):
        copy, kib, launches = [], 0.0, 0
        for r in csv.DictReader(open(path)):
            name, v = r["Kernel_Name"], float(r["Counter_Value"])
            if COPY_KERNEL in name:
                copy.append(v)
            role = rocprof_role(kernel, name)
            if role:
                kib += v
                launches += role == "main"
        factor = (PROBE_BYTES / 1024.0) / statistics.median(copy)
        out[f"{what}_factor"] = round(factor, 4)
        out[f"{what}_launches"] = launches
        out[f"{what}_bytes_per_launch"] = round(kib * 1024.0 * factor / launches)
    out["bytes_per_launch"] = out["fetch_bytes_per_launch"] + out["write_bytes_per_launch"]
    out["sources_sha256"] = sources_sha256(cls)
    return out


PROBE_BYTES = 1 << 30


def live_gates(op) -> int:
    """Gate blocks an operation's cells compute: a Tree-LSTM leaf's forget gates multiply the zero state
    (no children), so they are dead arithmetic and neither computed nor counted."""
    from paper_1702_02181_amd import gen
    if op.kind == gen.KIND_TREELSTM and op.arity == 0:
        return 3
    return gen.NUM_GATES[op.kind]


def counters_table(mfma_csv: str, fetch_csv: str, write_csv: str, trace_csv: str, top: int = 14) -> str:
    """Per-kernel table from four rocprofv3 runs of the same bench command: a counter pass with MfmaUtil,
    GRBM_GUI_ACTIVE and the MFMA op counts, a FETCH_SIZE pass, a WRITE_SIZE pass (KiB per dispatch, each
    scaled by what it reads for the copy probe) and a kernel trace (durations).  MFMA utilisation is
    weighted by each dispatch's active cycles; GB/s = HBM bytes / summed duration."""
    def rows(path):
        return list(csv.DictReader(open(path)))
    mfma = collections.defaultdict(lambda: [0, 0.0, 0.0, 0.0])  # dispatches, cycles, util*cycles, mfma flops
    disp = collections.defaultdict(dict)
    for r in rows(mfma_csv):
        disp[(r["Dispatch_Id"], r["Kernel_Name"])][r["Counter_Name"]] = float(r["Counter_Value"])
    for (_, name), v in disp.items():
        m = mfma[name]
        g = v.get("GRBM_GUI_ACTIVE", 0.0)
        m[0] += 1
        m[1] += g
        m[2] += v.get("MfmaUtil", 0.0) * g
        m[3] += 512.0 * (v.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0) + v.get("SQ_INSTS_VALU_MFMA_MOPS_F32", 0.0))
    hbm = {}
    for what, path in (("fetch", fetch_csv), ("write", write_csv)):
        tot = collections.defaultdict(float)
        copy = []
        for r in rows(path):
            tot[r["Kernel_Name"]] += float(r["Counter_Value"])
            if COPY_KERNEL in r["Kernel_Name"]:
                copy.append(float(r["Counter_Value"]))
        factor = (PROBE_BYTES / 1024.0) / statistics.median(copy)
        hbm[what] = {k: v * 1024.0 * factor for k, v in tot.items()}
    dur = collections.defaultdict(float)
    for r in rows(trace_csv):
        dur[r["Kernel_Name"]] += (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9
    out = ["| kernel | dispatches | total ms | MFMA busy % | MFMA TFLOP/s executed | HBM read GB | HBM write GB | HBM GB/s |",
           "|---|---:|---:|---:|---:|---:|---:|---:|"]
    for name in sorted(dur, key=lambda k: -dur[k])[:top]:
        m = mfma.get(name, [0, 0.0, 0.0, 0.0])
        t = dur[name]
        rd, wr = hbm["fetch"].get(name, 0.0), hbm["write"].get(name, 0.0)
        short = re.sub(r"fold::\(anonymous namespace\)::", "", name)[:70]
        out.append(f"| `{short}` | {m[0]} | {t * 1e3:.1f} | {m[2] / max(m[1], 1.0):.1f} | {m[3] / t / 1e12:.0f} | "
                   f"{rd / 1e9:.1f} | {wr / 1e9:.1f} | {(rd + wr) / t / 1e9:.0f} |")
    return "\n".join(out)


def table_runs(w) -> dict:
    """Distinct leaf-table rows each operation with an input reads: the rows of its leaf-table gradient
    contraction (dz is summed over the op's nodes of one leaf-table row before it is contracted)."""
    import numpy as np
    node_op = np.asarray(w.node_op)
    node_input = np.asarray(w.node_input)
    return {o: int(np.unique(node_input[(node_op == o) & (node_input >= 0)]).size)
            for o, op in enumerate(w.ops) if op.has_input}


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
    runs = table_runs(w) if (w.backward and table_grad) else {}
    for op_id, rows in rows_of_op.items():
        op = w.ops[op_id]
        if op.kind == gen.KIND_EMBED or op.kind in gen.ATTN_KINDS:
            continue
        G = live_gates(op)
        ps = w.params[op.param_set]
        k_in = (ps.in_dim if op.has_input else 0) + op.arity * H
        name = gen.KIND_NAMES[op.kind]
        add(f"cell_fwd.{name}.{dt}", 2.0 * rows * k_in * G * H)
        if w.backward:
            if op.arity > 0:
                add(f"bwd_dx.{dt}", 2.0 * rows * G * H * op.arity * H)
            if op_id in runs:
                add(f"tgrad.{dt}", 2.0 * runs[op_id] * G * H * ps.in_dim)
            add(f"wgrad.{dt}", 2.0 * rows * k_in * G * H)
    return out


NARROW_S = 2e-6  # a level pass whose roofline time is below this is reported as time per pass


def attn_bytes(w, op, rows: int, kind: str) -> float:
    """Algorithmic HBM bytes of `rows` nodes of a feed-forward attention operation (Section 3.4), pass `kind`
    ("fwd", "bwd") or the scorer's weight gradient ("wgrad").  A node's state is its aggregate: acc (h, H values
    of the pool type) and (m, s) (8 bytes); its gradient is dh (fp32, H values) and ds (4 bytes).
      score  fwd: read the item h, write (h, e, 1)       bwd: read dh, ds, the item h; write the item's dh, de
      sum    fwd: read two aggregates, write one         bwd: read dh, ds, the children's (m, s); write both
                                                              children's (dh, ds)
      out    fwd: read one aggregate, write h            bwd: read dh, the child's acc and s; write its (dh, ds)
    plus the scorer vector once per pass; wgrad reads de and the item h per row and writes H + 1 floats."""
    from paper_1702_02181_amd import gen
    H = w.hidden
    bh = 2 if w.dtype == "bf16" else 4
    agg, grad = H * bh + 8, H * 4 + 4
    if kind == "wgrad":
        return float(rows * (4 + H * bh) + (H + 1) * 4)
    if op.kind == gen.KIND_ATTN_SCORE:
        per = (H * bh + agg) if kind == "fwd" else (grad + H * bh + grad)
        return float(rows * per + H * bh)
    if op.kind == gen.KIND_ATTN_SUM:
        return float(rows * ((2 * agg + agg) if kind == "fwd" else (grad + 16 + 2 * grad)))
    return float(rows * ((agg + H * bh) if kind == "fwd" else (H * 4 + agg + grad)))


def attn_kernel_bytes(w, host) -> dict:
    """Algorithmic HBM bytes of one step by attention kernel class ("attn_fwd.score", ...)."""
    from paper_1702_02181_amd import gen
    names = {gen.KIND_ATTN_SCORE: "score", gen.KIND_ATTN_SUM: "sum", gen.KIND_ATTN_OUT: "out"}
    out = {}
    for op_id, rows in zip(host["group_op"], host["group_rows"]):
        op = w.ops[int(op_id)]
        if op.kind not in names:
            continue
        for kind in ("fwd", "bwd") if w.backward else ("fwd",):
            k = f"attn_{kind}.{names[op.kind]}"
            out[k] = out.get(k, 0.0) + attn_bytes(w, op, int(rows), kind)
        if w.backward and op.kind == gen.KIND_ATTN_SCORE:
            out["attn_wgrad"] = out.get("attn_wgrad", 0.0) + attn_bytes(w, op, int(rows), "wgrad")
    return out


def pass_work(w, host, table_grad: bool) -> dict:
    """Algorithmic FLOPs and HBM bytes of every level pass of one step (weights counted once per pass).

    Keys: ("fwd", group), ("bwd", group) -- the cell's backward and dz . W^T of one (depth, op) group --
    ("wgrad", op), the deferred weight-gradient contraction of one operation over all its rows, and ("tgrad",
    op), its leaf-table gradient (dz summed per leaf-table row, then one contraction row per distinct row).
    Per node, with S = state bytes (h, plus fp32 c for cells that carry one) and S_g = its fp32
    gradient: forward reads the input row and the children's states and writes S; backward reads S_g
    and the children's states and writes the children's S_g (plus the leaf-table gradient row).
    Saved activations are implementation overhead, not counted."""
    from paper_1702_02181_amd import gen
    H = w.hidden
    bh = 2 if w.dtype == "bf16" else 4
    out = {}
    op_rows = {}
    for g, (op_id, rows) in enumerate(zip(host["group_op"], host["group_rows"])):
        op, rows = w.ops[int(op_id)], int(rows)
        op_rows[int(op_id)] = op_rows.get(int(op_id), 0) + rows
        if op.kind in gen.ATTN_KINDS:
            out[("fwd", g)] = (2.0 * rows * H if op.kind == gen.KIND_ATTN_SCORE else 0.0,
                               attn_bytes(w, op, rows, "fwd"))
            if w.backward:
                out[("bwd", g)] = (0.0, attn_bytes(w, op, rows, "bwd"))
            continue
        if op.kind == gen.KIND_EMBED:  # its leaf-table gradient is a ("tgrad", op) pass
            out[("fwd", g)] = (0.0, float(rows * 2 * H * bh))
            continue
        G = live_gates(op)
        din = w.params[op.param_set].in_dim if op.has_input else 0
        has_c = op.kind in (gen.KIND_TREELSTM, gen.KIND_LSTM, gen.KIND_PROJ)
        s_node = H * (bh + (4 if has_c else 0))
        sg_node = 4 * H * (2 if has_c else 1)
        k_in = din + op.arity * H
        out[("fwd", g)] = (2.0 * rows * k_in * G * H,
                           float(rows * (din * bh + op.arity * s_node + s_node) + k_in * G * H * bh + G * H * 4))
        if w.backward:
            k_dx = op.arity * H
            out[("bwd", g)] = (2.0 * rows * G * H * k_dx,
                               float(rows * (sg_node + op.arity * (s_node + sg_node)) + k_dx * G * H * bh))
    if w.backward and table_grad:
        runs = table_runs(w)
        for o, count in op_rows.items():
            op = w.ops[o]
            if o not in runs:
                continue
            if op.kind == gen.KIND_EMBED:  # every row's dh read once, each distinct leaf-table row read and written
                out[("tgrad", o)] = (0.0, float(count * 4 * H + runs[o] * H * 4 * 2))
                continue
            G, din = live_gates(op), w.params[op.param_set].in_dim
            # read every row's dz once, read and write each distinct leaf-table row, the weights once
            out[("tgrad", o)] = (2.0 * runs[o] * G * H * din,
                                 float(count * G * H * bh + runs[o] * din * 4 * 2 + din * G * H * bh))
    if w.backward:
        for o, count in op_rows.items():
            op = w.ops[o]
            if op.kind == gen.KIND_ATTN_SCORE:
                out[("wgrad", o)] = (2.0 * count * H, attn_bytes(w, op, count, "wgrad"))
            if op.kind == gen.KIND_EMBED or op.kind in gen.ATTN_KINDS:
                continue
            G = live_gates(op)
            k_in = (w.params[op.param_set].in_dim if op.has_input else 0) + op.arity * H
            out[("wgrad", o)] = (2.0 * count * k_in * G * H,
                                 float(count * (k_in + G * H) * bh + (k_in + 1) * G * H * 4))
    return out


def pass_of(name: str, group: int, op: int):
    """The level passes a profiled launch belongs to ([]: set-up, roots).  A level launch runs several
    consecutive groups of one level (tagged with its first group and op = -1 - span); its time is shared
    equally among them."""
    cls = class_of(name)
    groups = [group] if op >= -1 else list(range(group, group - 1 - op))
    if group >= 0 and cls in ("cell_fwd", "embed_fwd", "attn_fwd"):
        return [("fwd", g) for g in groups]
    if group >= 0 and cls in ("cell_bwd", "bwd_dx", "attn_bwd"):
        return [("bwd", g) for g in groups]
    if group < 0 and op >= 0 and cls in ("wgrad", "wgrad_reduce", "bias_partial", "bias_reduce", "attn_wgrad"):
        return [("wgrad", op)]
    if group < 0 and op >= 0 and cls in ("tgrad", "tgrad_sum", "tgrad_embed"):
        return [("tgrad", op)]
    return []


def level_classes(work: dict, launches: list, steps: int, peak_tflops: float, hbm_gbs: float) -> dict:
    """Roofline per class of level pass.  A pass is MFMA-bound ("wide") when its FLOPs at the matrix
    peak take at least as long as its bytes at the HBM peak, else "gather"-bound; a pass whose roofline
    time is under NARROW_S is "narrow" and reported as time per pass.  frac = sum of roofline times /
    sum of measured times over the class (time-weighted); also split by pass kind."""
    meas = {}
    other = 0.0
    for name, group, op, ms in launches:
        keys = pass_of(name, group, op)
        if not keys:
            other += ms
        for key in keys:
            meas[key] = meas.get(key, 0.0) + ms / steps / len(keys)
    cls = {c: {"passes": 0, "ms_per_step": 0.0, "roofline_ms": 0.0, "flops": 0.0, "bytes": 0.0, "by_pass": {}}
           for c in ("wide", "gather", "narrow")}
    for key, (F, B) in work.items():
        if key not in meas:
            continue
        t_m, t_h = F / (peak_tflops * 1e12), B / (hbm_gbs * 1e9)
        roof = max(t_m, t_h)
        c = "narrow" if roof < NARROW_S else ("wide" if t_m >= t_h else "gather")
        d = cls[c]
        d["passes"] += 1
        d["ms_per_step"] += meas[key]
        d["roofline_ms"] += roof * 1e3
        d["flops"] += F
        d["bytes"] += B
        bp = d["by_pass"].setdefault(key[0], [0, 0.0, 0.0])
        bp[0] += 1
        bp[1] += meas[key]
        bp[2] += roof * 1e3
    out = {}
    for c, d in cls.items():
        if d["passes"] == 0:
            continue
        t = d["ms_per_step"] * 1e-3
        e = {"passes": d["passes"], "ms_per_step": round(d["ms_per_step"], 4)}
        if c == "narrow":
            e["us_per_pass"] = round(d["ms_per_step"] * 1e3 / d["passes"], 2)
        else:
            e["bound"] = "mfma" if c == "wide" else "hbm"
            e["frac"] = round(d["roofline_ms"] / d["ms_per_step"], 4)
            if c == "wide":
                e["achieved_tflops"] = round(d["flops"] / t / 1e12, 1)
                e["peak_tflops"] = peak_tflops
            else:
                e["achieved_gbs"] = round(d["bytes"] / t / 1e9, 1)
                e["peak_gbs"] = hbm_gbs
            e["by_pass"] = {k: {"passes": v[0], "ms_per_step": round(v[1], 4), "frac": round(v[2] / v[1], 4)}
                            for k, v in sorted(d["by_pass"].items())}
        out[c] = e
    out["other_ms_per_step"] = round(other / steps, 4)
    return out


TABLE1_BATCHES = (1, 32, 64, 128, 256, 512, 1024)


def table1(batches, steps: int, warmup: int, dtype: str = "f32") -> dict:
    """The inference timing protocol of Section 2.1 (Table 1) on this GPU: batches of 127-node random trees
    (H = 1024, embedding-lookup leaves), forward only, timed as HIP-graph replays.  "manual" runs one batched
    group per tree node (one operation per node position) whose children are the consecutive rows of the child
    position's group, addressed as base + row with no gather index (the static graph's layout), "dynamic" one
    group per (depth, op) over trees of one shape, gathering children by index, "full" the same over trees of
    random shapes.  cost ratio = dynamic / manual time per batch;
    speedup ratio = manual time per tree at batch size 1 / full-dynamic time per tree."""
    import torch

    from paper_1702_02181_amd import gen
    from paper_1702_02181_amd.runner import DeviceRun
    stream = torch.cuda.current_stream()

    def timed(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    from paper_1702_02181_amd import fold as F
    rows = []
    for B in batches:
        row = {"batch": B}
        for mode in ("manual", "manual_level", "dynamic", "full"):
            # manual: one launch per node position, as a static graph runs; manual_level: the same schedule with
            # the independent node positions of a depth in shared launches (the library's default)
            w = gen.table1(B, "manual" if mode == "manual_level" else mode, dtype=dtype)
            prev = F.fold_level_launches(mode != "manual")
            dev = DeviceRun(w)
            graph = dev.make_graph(backward=False)
            F.fold_level_launches(prev)
            ms = timed(graph.launch)
            host = dev.sched.host_groups()
            slots = [(host[f"group_child_base{k}"][g] >= 0)
                     for g, op in enumerate(host["group_op"]) for k in range(w.ops[int(op)].arity)]
            row[mode] = {"batch_ms": round(ms, 4), "tree_ms": round(ms / B, 5),
                         "groups": len(host["group_op"]), "kernels": graph.num_nodes,
                         "gather_free_child_slots": f"{sum(slots)}/{len(slots)}"}
            del graph, dev
        row["cost_ratio"] = round(row["dynamic"]["batch_ms"] / row["manual"]["batch_ms"], 3)
        rows.append(row)
        print(f"[table1] batch {B}: manual {row['manual']['batch_ms']:.3f} ms (level launches "
              f"{row['manual_level']['batch_ms']:.3f} ms), dynamic {row['dynamic']['batch_ms']:.3f} ms, full "
              f"{row['full']['batch_ms']:.3f} ms", file=sys.stderr, flush=True)
    base = next((r["manual"]["tree_ms"] for r in rows if r["batch"] == 1), None)
    for r in rows:
        r["speedup_ratio"] = None if base is None else round(base / r["full"]["tree_ms"], 2)
    return {"table1": rows, "tree_nodes": 127, "hidden": 1024, "dtype": dtype, "pass": "forward",
            "steps": steps, "warmup": warmup}


def train_bench(config: int, steps: int, warmup: int, classes: int = 5, dropout: float = 0.0) -> dict:
    """Training steps of Section 3.5's setting on one workload: a class label on every node (uniform, seeded),
    forward, the per-node softmax cross-entropy head, backward from the head's gradients, Adam on every
    parameter tensor (weights, biases, the leaf table where it is trained, the classifier) and the in-place
    re-pack of the weights; the gradient pass (zero, forward, head, backward) is replayed as one recorded graph, Adam
    and the re-pack are issued call by call.  The batch is the same every step, so the mean loss falls.  With
    dropout > 0 every step first draws a fresh recurrent-dropout mask on the GPU (fold_dropout_mask)."""
    import numpy as np
    import torch

    from paper_1702_02181_amd import fold as F
    from paper_1702_02181_amd import gen
    from paper_1702_02181_amd.runner import TrainStep
    stream = torch.cuda.current_stream()
    w = gen.make_config(config)
    labels = np.random.default_rng(11).integers(0, classes, w.num_nodes).astype(np.int32)
    ts = TrainStep(w, labels, classes, train_table=config in (3, 5), dropout=dropout, dropout_seed=17)
    mean_loss = lambda: float(ts.node_loss[:w.num_nodes].sum().item() * ts.scale)
    ts.step()
    ts.capture_gradients()  # the gradient pass replays as one graph; Adam and the re-pack run call by call
    torch.cuda.synchronize()
    first = mean_loss()
    for _ in range(max(0, warmup - 1)):
        ts.step(graph=True)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        ts.step(graph=True)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    last = mean_loss()
    F.fold_profile_enable(True)
    for _ in range(steps):
        ts.step()
    torch.cuda.synchronize()
    stats = F.fold_profile_read()
    F.fold_profile_enable(False)
    kernels = {k: {"launches_per_step": n / steps, "ms_per_step": round(tot / steps, 4)}
               for k, (n, tot, _mx) in stats.items()}
    return {"metric": "training graph nodes/sec (Tree-LSTM, per-node softmax loss, Adam; 1 GPU)",
            "value": round(w.num_nodes / (ms * 1e-3), 1), "unit": "graph nodes/s", "n_gpus": 1, "steps": steps,
            "warmup": warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "dtype": w.dtype,
            "data": "synthetic", "config": {"workload": w.name, "nodes": w.num_nodes, "hidden": w.hidden,
                                            "classes": classes, "optimizer": "adam lr 1e-3 (0.9, 0.999, 1e-8)",
                                            "trained_leaf_table": config in (3, 5),
                                            "recurrent_dropout": dropout},
            "mean_loss": {"step_1": round(first, 5), f"step_{ts.t - steps}": round(last, 5)},
            "kernels": kernels}


def blocks_bench(steps: int, warmup: int, num_trees: int = 1024, hidden: int = 300, vocab: int = 20000) -> dict:
    """The combinator front end on sentiment-tree-shaped input: nested-tuple binary trees with U[5, 60] leaves
    (random splits, uniform tokens) compiled by the recursive Tree-LSTM block expression of Section 3.5, then the
    compiled batch's forward + backward step (HIP-graph replay).  Reports the host compile time beside the step."""
    import numpy as np
    import torch

    from paper_1702_02181_amd import blocks as B
    from paper_1702_02181_amd import gen
    from paper_1702_02181_amd.runner import DeviceRun
    rng = np.random.default_rng(17)

    def tree(n):
        if n == 1:
            return int(rng.integers(0, vocab))
        k = int(rng.integers(1, n))
        return (tree(k), tree(n - k))

    trees = [tree(int(n)) for n in rng.integers(5, 61, num_trees)]
    expr = B.ForwardDeclaration()
    word = B.AllOf(B.Scalar(), B.Zeros())
    pair = B.AllOf(B.Zeros(), B.Record([(0, expr()), (1, expr())]))
    expr.resolve_to(B.OneOf(lambda t: isinstance(t, tuple), {False: word, True: pair}) >> B.Op(gen.KIND_TREELSTM, 0))
    table = gen._finish_values(0.1 * rng.standard_normal((vocab, hidden)), "bf16")
    params = [gen.make_param_set(rng, gen.KIND_TREELSTM, hidden, 2, hidden, "bf16")]
    t0 = time.perf_counter()
    comp = B.Compiler(expr())
    w, _ = comp.build(trees, params, hidden, table, dtype="bf16", name="blocks_treelstm_h300_bf16")
    build_s = time.perf_counter() - t0
    dev = DeviceRun(w)
    dev.alloc_grads(True)
    dev.set_upstream(w.dh_roots)
    graph = dev.make_graph(backward=True, zero_grads=True)
    stream = torch.cuda.current_stream()
    for _ in range(warmup):
        graph.launch()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        graph.launch()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    return {"metric": "graph nodes/sec (Tree-LSTM fwd+bwd of a front-end-compiled batch, 1 GPU)",
            "value": round(w.num_nodes / (ms * 1e-3), 1), "unit": "graph nodes/s", "ms_per_step": round(ms, 4),
            "steps": steps, "warmup": warmup, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": w.name, "trees": num_trees, "nodes": w.num_nodes, "hidden": hidden,
                       "ops": len(comp.ops)},
            "host_compile_ms": round(build_s * 1e3, 1),
            "host_compile_nodes_per_s": round(w.num_nodes / build_s, 1)}


def attention_bench(steps: int, warmup: int) -> dict:
    """Feed-forward attention (Section 3.4, Appendix A) as a dynamic-batching workload: 1024 sequences of
    U{50..100} token rows, h_t = PROJ f(x_t), scored, merged by a balanced Reduce, attended, PROJ g on top;
    H = 256, bf16, forward + backward (the token rows are data: no leaf-table gradient).  The attention
    kernels are HBM-bound: each reports its algorithmic bytes per step over its measured time."""
    import torch

    from paper_1702_02181_amd import gen
    torch.cuda.set_device(0)
    print("[bench attention] generating", file=sys.stderr, flush=True)
    w = gen.attention()
    m = measure(w, steps, warmup, False, schedule_reps=3, tag=" attention")
    attn = {k: v for k, v in m["kernels"].items() if k.startswith("attn_")}
    by = sum(v.get("alg_bytes_per_step", 0) for v in attn.values())
    t = sum(v["ms_per_step"] for v in attn.values())
    return {"metric": "graph nodes/sec (feed-forward attention fwd+bwd, 1 GPU)", "value": m["value"],
            "unit": "graph nodes/s", "n_gpus": 1, "steps": steps, "warmup": warmup,
            "ms_per_step": m["ms_per_step"], "eager_ms_per_step": m["eager_ms_per_step"], "fwd_ms": m["fwd_ms"],
            "bwd_ms": m["bwd_ms"], "higher_is_better": True,
            "dtype": m["dtype"], "data": "synthetic", "config": m["config"], "schedule_ms": m["schedule_ms"],
            "attention_kernels": {"ms_per_step": round(t, 4), "alg_bytes_per_step": by,
                                  "gbs": round(by / (t * 1e-3) / 1e9, 1),
                                  "hbm_frac": round(by / (t * 1e-3) / 1e9 / PEAKS["hbm_gbs"], 4)},
            "roofline": m["roofline"], "level_classes": m["level_classes"], "kernels": m["kernels"]}


def _oracle_graph(w, g: int) -> int:
    """The oracle, as it stands, on graph g of the workload alone (fp64 forward, + backward if the workload
    has one); returns the graph's node count."""
    from oracle import evaluate as EV
    from paper_1702_02181_amd import gen
    from tests._helpers import oracle_batch, oracle_params
    sub = gen.subset(w, [g])
    b = oracle_batch(sub)
    P = oracle_params(sub)
    f = EV.forward(b, P, w.hidden, w.leaf_table)
    if w.backward:
        EV.backward(b, P, w.hidden, w.leaf_table, f, sub.dh_roots.astype("float64"), None, want_table_grad=False)
    return sub.num_nodes


def cpu_baseline(w, budget_s: float):
    """The oracle as it stands, single thread, on whole graphs of the workload until ~budget_s."""
    from threadpoolctl import threadpool_limits

    nodes = 0
    graphs = 0
    t0 = time.perf_counter()
    with threadpool_limits(limits=1):
        while graphs < w.num_graphs and (time.perf_counter() - t0) < budget_s:
            nodes += _oracle_graph(w, graphs)
            graphs += 1
    dt = time.perf_counter() - t0
    return {"value": nodes / dt, "unit": "graph nodes/s", "cores": 1, "kind": "oracle",
            "sample": f"graphs 0..{graphs - 1} of {w.num_graphs} ({nodes} nodes), fp64 "
                      f"{'forward+backward' if w.backward else 'forward'}, one thread, {dt:.1f} s"}


_POOL_W = None


def _pool_init(config: int):
    global _POOL_W
    from threadpoolctl import threadpool_limits
    from paper_1702_02181_amd import gen
    threadpool_limits(limits=1)
    _POOL_W = gen.make_config(config)


def _pool_ready(_):
    time.sleep(0.05)
    return os.getpid()


def _pool_graph(g: int) -> int:
    return _oracle_graph(_POOL_W, g)


def cpu_baseline_allcore(config: int, w, rate_1core: float, budget_s: float, max_workers: int = 16):
    """The same oracle over a process pool of single-threaded workers (graphs are independent), one worker
    per host core up to the machine's CPU share; graphs 0..K-1 with K sized from the one-core rate so that the
    timed map takes about budget_s.  Workers build the workload themselves before the timed region.  Runs
    before anything touches the GPU (workers are started by spawn from a process with no GPU state)."""
    import multiprocessing as mp
    workers = max(1, min(max_workers, os.cpu_count() or 1))
    per_graph = w.num_nodes / max(1, w.num_graphs)
    rounds = max(1, round(rate_1core * budget_s / per_graph))  # graphs per worker
    K = int(min(w.num_graphs, rounds * workers))
    ctx = mp.get_context("spawn")
    with ctx.Pool(workers, initializer=_pool_init, initargs=(config,)) as pool:
        pids = set(pool.map(_pool_ready, range(8 * workers), chunksize=1))
        t0 = time.perf_counter()
        nodes = sum(pool.map(_pool_graph, range(K), chunksize=1))
        dt = time.perf_counter() - t0
    return {"value": nodes / dt, "unit": "graph nodes/s", "cores": workers, "kind": "oracle",
            "host_cores": os.cpu_count(), "workers_started": len(pids),
            "sample": f"graphs 0..{K - 1} of {w.num_graphs} ({nodes} nodes), fp64 "
                      f"{'forward+backward' if w.backward else 'forward'}, {workers} single-threaded processes, "
                      f"{dt:.1f} s"}


def reference_schedule_ms(w) -> float:
    """The oracle's reference scheduler (validation, memoised depth recursion, stable sort, edge labels;
    Python) on the whole batch, in ms."""
    from tests import gpu_common as C
    t0 = time.perf_counter()
    C.oracle_schedule(w)
    return (time.perf_counter() - t0) * 1e3


def measure(w, steps: int, warmup: int, table_grad: bool, schedule_reps: int = 5, tag: str = "") -> dict:
    """One workload on the GPU: fold_schedule time, the step (forward + backward, or forward only) issued
    call by call and as a HIP-graph replay, per-launch HIP-event durations by kernel class, the roofline of
    the dominant kernel class and of every class of level pass."""
    import torch

    from paper_1702_02181_amd import fold as F
    from paper_1702_02181_amd.runner import DeviceRun

    dev = DeviceRun(w)
    host = dev.sched.host_groups()
    N = w.num_nodes
    sched_ms = []
    for _ in range(schedule_reps):
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

    print(f"[bench{tag}] {w.name}: N={N} levels={dev.sched.num_levels} groups={len(host['group_op'])} "
          f"warmup={warmup} steps={steps}", file=sys.stderr, flush=True)
    stream = torch.cuda.current_stream()

    def timed(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    # the step as issued call by call, then recorded once as a HIP graph and replayed
    eager_ms = timed(step)
    graph = dev.make_graph(backward=w.backward, zero_grads=True)
    graph_ms = timed(graph.launch)
    print(f"[bench{tag}] timed {steps} steps: graph {graph_ms:.3f} ms/step, eager {eager_ms:.3f} ms/step "
          f"({graph.num_nodes} graph nodes)", file=sys.stderr, flush=True)
    # the forward alone, recorded and replayed the same way; the backward is the rest of the step
    fwd_ms = graph_ms
    if w.backward:
        fgraph = dev.make_graph(backward=False)
        fwd_ms = timed(fgraph.launch)
        del fgraph

    # per-kernel durations over a second timed region (event pair around every launch, on the stream the
    # kernels run on)
    F.fold_profile_enable(True)
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    launch_times = F.fold_profile_read_launches()
    F.fold_profile_enable(False)
    stats = {}
    for name, _g, _o, ms in launch_times:
        n, tot, mx = stats.get(name, (0, 0.0, 0.0))
        stats[name] = (n + 1, tot + ms, max(mx, ms))
    flops = flops_by_kernel(w, host, table_grad)
    kernels = {}
    for name, (launches, total_ms, max_ms) in stats.items():
        per_step_ms = total_ms / steps
        kernels[name] = {"launches_per_step": launches / steps, "ms_per_step": round(per_step_ms, 4),
                         "avg_launch_us": round(1e3 * total_ms / max(launches, 1), 2)}
        if name in flops:
            kernels[name]["tflops"] = round(flops[name] / (per_step_ms * 1e-3) / 1e12, 2)
    mfma_kernels = [k for k in kernels if k in flops]
    dom = max(mfma_kernels, key=lambda k: kernels[k]["ms_per_step"]) if mfma_kernels else None
    roofline = None
    if dom:
        peak = PEAKS["bf16_mfma_tflops"] if dom.endswith("bf16") else PEAKS["f32_mfma_tflops"]
        launches = stats[dom][0] / steps
        avg_s = (stats[dom][1] / steps) / launches * 1e-3
        per_launch = flops[dom] / launches
        ach = per_launch / avg_s / 1e12
        rec = traffic_record(dom, w.name)
        roofline = {"bound": "mfma", "kernel": dom, "achieved": round(ach, 2), "peak": peak, "unit": "TFLOP/s",
                    "frac": round(ach / peak, 4), "traffic": None if rec is None else rec["bytes_per_launch"],
                    "traffic_unit": "bytes per launch (HBM read + write, rocprofv3 FETCH_SIZE / WRITE_SIZE "
                                    "scaled by the copy probe)",
                    "flops_per_launch": per_launch, "launches_per_step": launches,
                    "avg_launch_us": round(avg_s * 1e6, 2)}
        # algorithmic HBM bytes per launch of the class (the level passes it runs in, weights once per pass)
        kind = {"cell_fwd": "fwd", "bwd_dx": "bwd", "wgrad": "wgrad", "tgrad": "tgrad"}[class_of(dom)]
        alg = 0.0
        for (pk, key), (_fl, by) in pass_work(w, host, table_grad).items():
            if pk != kind:
                continue
            if kind == "fwd":
                from paper_1702_02181_amd import gen as _g
                if f"cell_fwd.{_g.KIND_NAMES[w.ops[int(host['group_op'][key])].kind]}." not in dom + ".":
                    continue
            alg += by
        roofline["algorithmic_bytes_per_launch"] = round(alg / launches)
        if rec is not None:
            roofline["traffic_vs_algorithmic"] = round(rec["bytes_per_launch"] / (alg / launches), 3)
    # attention kernels: algorithmic bytes over their measured time, against the HBM peak
    for name, by in attn_kernel_bytes(w, host).items():
        if name in kernels:
            gbs = by / (kernels[name]["ms_per_step"] * 1e-3) / 1e9
            kernels[name].update(alg_bytes_per_step=round(by), gbs=round(gbs, 1),
                                 hbm_frac=round(gbs / PEAKS["hbm_gbs"], 4))
    total_flops = sum(flops.values())
    step_peak = PEAKS["bf16_mfma_tflops"] if w.dtype == "bf16" else PEAKS["f32_mfma_tflops"]
    classes = level_classes(pass_work(w, host, table_grad), launch_times, steps, step_peak, PEAKS["hbm_gbs"])
    out = {
        "value": round(N / (graph_ms * 1e-3), 1),
        "ms_per_step": round(graph_ms, 4),
        "eager_ms_per_step": round(eager_ms, 4),
        "fwd_ms": round(fwd_ms, 4),
        "bwd_ms": round(graph_ms - fwd_ms, 4) if w.backward else None,
        "dtype": "f32" if w.dtype == "f32" else "bf16",
        "config": {"workload": w.name, "graphs": w.num_graphs, "nodes": N, "levels": dev.sched.num_levels,
                   "groups": len(host["group_op"]), "hidden": w.hidden,
                   "pass": "forward+backward" if w.backward else "forward",
                   "leaf_table_grad": bool(w.backward and table_grad)},
        "schedule_ms": None if schedule_ms is None else round(schedule_ms, 3),
        "graph_nodes": graph.num_nodes,
        "roofline": roofline,
        "step_mfma_frac": round(total_flops / (graph_ms * 1e-3) / 1e12 / step_peak, 4),
        "level_classes": classes,
        "kernels": kernels,
    }
    del graph, dev
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


# Plain library GEMMs (torch.matmul: hipBLASLt / rocBLAS) of the contraction shapes the workloads run, on random
# operands: what a dense vendor GEMM of the same size sustains on this GPU, without the gathers, the fused cells
# or the scatter-adds.  (M, N, K, dtype, label); K-major A for the weight-gradient shapes (X^T dz).
GEMM_SHAPES = [
    (32768, 1280, 512, "f32", "config 2 internal level (rows x 5H, K = 2H)", False),
    (65536, 768, 256, "f32", "config 2 leaf level (rows x 3H, K = in)", False),
    (32768, 512, 1280, "f32", "config 2 dz.W^T (rows x 2H, K = 5H)", False),
    (512, 1280, 65280, "f32", "config 2 weight gradient (2H x 5H, K = rows)", True),
    (131072, 5120, 2048, "bf16", "H = 1024 wide level (rows x 5H, K = 2H)", False),
    (131072, 2048, 5120, "bf16", "H = 1024 wide dz.W^T (rows x 2H, K = 5H)", False),
    (2048, 5120, 131072, "bf16", "H = 1024 weight gradient (2H x 5H, K = rows)", True),
    (2048, 5120, 2048, "bf16", "H = 1024 mid-size level (2,048 rows)", False),
    (8192, 8192, 8192, "bf16", "square 8192", False),
]


def gemm_ceiling(reps: int = 10) -> dict:
    import torch
    torch.cuda.set_device(0)
    rows = []
    for M, N, K, dt, label, kmajor in GEMM_SHAPES:
        dtype = torch.bfloat16 if dt == "bf16" else torch.float32
        g = torch.Generator(device="cuda").manual_seed(M + N + K)
        a = torch.rand((K, M) if kmajor else (M, K), device="cuda", dtype=dtype, generator=g) * 2 - 1
        b = torch.rand((K, N), device="cuda", dtype=dtype, generator=g) * 2 - 1
        A = a.t() if kmajor else a
        for _ in range(3):
            torch.matmul(A, b)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            torch.matmul(A, b)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        tf = 2.0 * M * N * K / (ms * 1e-3) / 1e12
        peak = PEAKS["bf16_mfma_tflops"] if dt == "bf16" else PEAKS["f32_mfma_tflops"]
        rows.append({"shape": label, "M": M, "N": N, "K": K, "dtype": dt, "ms": round(ms, 4),
                     "tflops": round(tf, 1), "frac_of_datasheet": round(tf / peak, 3)})
        del a, b
    return {"library_gemm": rows, "note": "torch.matmul on random operands in [-1, 1)"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=2)
    ap.add_argument("--cpu-seconds", type=float, default=8.0, help="time of each oracle leg (one core, all cores)")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--profile-only", action="store_true", help="skip the oracle legs and the other workloads")
    ap.add_argument("--extra-configs", default="3,5",
                    help="workloads measured after the headline one, reported under 'configs' ('' for none)")
    ap.add_argument("--traffic-from", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"))
    ap.add_argument("--traffic-kernel", default=None)
    ap.add_argument("--table1", action="store_true",
                    help="run the Table 1 protocol (manual / dynamic / full-dynamic batching) instead")
    ap.add_argument("--train", action="store_true",
                    help="time training steps (per-node softmax loss, Adam, re-pack) instead; default config 3")
    ap.add_argument("--dropout", type=float, default=0.0, help="recurrent dropout probability of --train")
    ap.add_argument("--attention", action="store_true",
                    help="time the feed-forward attention workload (1024 sequences of 50-100 items, H = 256, bf16)")
    ap.add_argument("--blocks", action="store_true",
                    help="compile sentiment-shaped trees with the combinator front end and time the compiled batch")
    ap.add_argument("--gemm-ceiling", action="store_true",
                    help="time plain library GEMMs (torch.matmul) of the workloads' contraction shapes instead")
    ap.add_argument("--counters-from", nargs=4, metavar=("MFMA_CSV", "FETCH_CSV", "WRITE_CSV", "TRACE_CSV"),
                    help="print the per-kernel MFMA utilisation / HBM bandwidth table of four rocprofv3 runs")
    args = ap.parse_args()
    if args.counters_from:
        print(counters_table(*args.counters_from))
        return
    if args.gemm_ceiling:
        print(json.dumps(gemm_ceiling()), flush=True)
        return
    if args.traffic_from:
        from paper_1702_02181_amd import gen as _gen
        w = _gen.make_config(args.config)
        rec = traffic_from_counters(args.traffic_from[0], args.traffic_from[1], args.traffic_kernel, w.name)
        print(TRAFFIC_TAG, json.dumps(rec))
        return
    if args.blocks:
        import torch
        torch.cuda.set_device(0)
        print(json.dumps(blocks_bench(args.steps, args.warmup)), flush=True)
        return
    if args.attention:
        print(json.dumps(attention_bench(args.steps, args.warmup)), flush=True)
        return
    if args.train:
        import torch
        torch.cuda.set_device(0)
        cfg = args.config if "--config" in sys.argv else 3
        print(json.dumps(train_bench(cfg, args.steps, args.warmup, dropout=args.dropout)), flush=True)
        return
    if args.table1:
        import torch
        torch.cuda.set_device(0)
        print(json.dumps(table1(TABLE1_BATCHES, args.steps, args.warmup)), flush=True)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the dynamic-batching path here is a single-GPU build "
              "(graphs would shard across GPUs with one all-reduce of weight gradients; not built).",
              file=sys.stderr)
        sys.exit(2)

    from paper_1702_02181_amd import gen

    print(f"[bench] generating config {args.config}", file=sys.stderr, flush=True)
    w = gen.make_config(args.config)
    table_grad = args.config in (3, 5)  # trainable embedding tables; config 2 / 4 leaf rows are data

    # host legs first, before anything touches the GPU: the oracle on one core and on a process pool, and
    # the oracle's reference scheduler on the whole batch
    cpu = None
    sched_ref_ms = None
    if not args.no_cpu and not args.profile_only:
        print(f"[bench] oracle on host cores ({args.cpu_seconds:.0f} s one core, then a process pool)",
              file=sys.stderr, flush=True)
        one = cpu_baseline(w, args.cpu_seconds)
        cpu = cpu_baseline_allcore(args.config, w, one["value"], args.cpu_seconds)
        cpu["single_core"] = one
        print(f"[bench] oracle: {one['value']:.0f} nodes/s on one core, {cpu['value']:.0f} on {cpu['cores']}",
              file=sys.stderr, flush=True)
        sched_ref_ms = reference_schedule_ms(w)
        print(f"[bench] reference scheduler: {sched_ref_ms:.0f} ms", file=sys.stderr, flush=True)

    import torch

    from paper_1702_02181_amd import fold as F

    torch.cuda.set_device(0)
    # achievable peaks on this GPU (MFMA loop, stream copy), next to the datasheet figures
    probes = {}
    try:
        # the copy probe doubles as the calibration kernel of the HBM byte counters (PROBE_BYTES a dispatch)
        probes["mfma_f32_tflops"] = round(F.fold_probe_mfma(F.FOLD_F32), 1)
        probes["mfma_bf16_tflops"] = round(F.fold_probe_mfma(F.FOLD_BF16), 1)
        # random operand bits: what the matrix cores sustain on the data the contractions multiply
        probes["mfma_f32_random_tflops"] = round(F.fold_probe_mfma_random(F.FOLD_F32), 1)
        probes["mfma_bf16_random_tflops"] = round(F.fold_probe_mfma_random(F.FOLD_BF16), 1)
        nbytes = PROBE_BYTES
        src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        probes["copy_gbs"] = round(F.fold_probe_copy(dst, src, nbytes), 1)
        del src, dst
    except Exception as e:  # probes are diagnostics; the bench line does not depend on them
        probes["error"] = str(e)
    print(f"[bench] probes {probes}", file=sys.stderr, flush=True)

    head = measure(w, args.steps, args.warmup, table_grad, schedule_reps=0 if args.profile_only else 5)
    del w
    extra = {}
    if not args.profile_only:
        for k in [int(x) for x in args.extra_configs.split(",") if x.strip()]:
            if k == args.config:
                continue
            print(f"[bench] generating config {k}", file=sys.stderr, flush=True)
            wk = gen.make_config(k)
            # config 5 steps take ~0.2 s: fewer steps keep the whole run within minutes
            steps_k = min(args.steps, 5) if wk.num_nodes > 1_000_000 else args.steps
            mk = measure(wk, steps_k, min(args.warmup, 2), k in (3, 5), schedule_reps=3, tag=f" cfg{k}")
            mk["steps"] = steps_k
            extra[wk.name] = mk
            del wk

    out = {
        "metric": "graph nodes/sec (TreeLSTM fwd+bwd, 1 GPU)",
        "value": head["value"],
        "unit": "graph nodes/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "eager_ms_per_step": head["eager_ms_per_step"],
        "fwd_ms": head["fwd_ms"],
        "bwd_ms": head["bwd_ms"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": head["dtype"],
        "data": "synthetic",
        "config": head["config"],
        "schedule_ms": head["schedule_ms"],
        "schedule_ms_oracle": None if sched_ref_ms is None else round(sched_ref_ms, 1),
        "graph_nodes": head["graph_nodes"],
        "peaks": {"datasheet": PEAKS, "measured": probes},
        "roofline": head["roofline"],
        "step_mfma_frac": head["step_mfma_frac"],
        "level_classes": head["level_classes"],
        "kernels": head["kernels"],
        "cpu_baseline": cpu,
        "configs": extra,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
