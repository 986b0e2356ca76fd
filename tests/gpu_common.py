"""Helpers of the GPU parity tests: run a workload through the C ABI and through the oracle,
and compare with the documented metric.  Tolerances (max relative error per row, see
oracle.compare): 1e-5 for fp32 workloads, 2e-2 for bf16 matrix-core workloads."""
from __future__ import annotations

import numpy as np

from oracle import compare, evaluate as EV, schedule as S
from tests._helpers import oracle_batch, oracle_params

TOL = {"f32": 1e-5, "bf16": 2e-2}

SCHED_KEYS = ("depth", "node_pos", "pos_node", "level_ptr", "group_level", "group_op", "group_row_begin",
              "group_rows", "group_idx_off", "child_pos", "input_idx", "root_pos")


def oracle_schedule(w):
    b = oracle_batch(w)
    return S.reference_schedule(b["node_op"], b["child_ptr"], b["child_idx"], b["node_input"], b["ops"])


def assert_schedule_equal(gpu: dict, ref: dict):
    assert gpu["num_levels"] == ref["num_levels"]
    for k in SCHED_KEYS:
        assert np.array_equal(np.asarray(gpu[k]), np.asarray(ref[k])), k
    host = gpu["host"]
    for k in ("level_ptr", "group_level", "group_op", "group_row_begin", "group_rows", "group_idx_off"):
        assert np.array_equal(host[k], ref[k]), "host " + k


def run_device(w, dh_nodes=None, table_grad=False, backward=None, u_mask=None):
    """u_mask: recurrent-dropout mask [N, H] in node order (placed into pool order here), or None."""
    import torch
    from paper_1702_02181_amd.runner import DeviceRun
    backward = w.backward if backward is None else backward
    dev = DeviceRun(w, with_backward=backward)
    mask = None
    if u_mask is not None:
        pool = np.zeros((dev.N, dev.ld), np.float32)
        pool[dev.sched_arrays()["node_pos"], :dev.H] = u_mask
        mask = torch.from_numpy(pool).cuda()
    dev.forward(mask)
    out = {}
    if backward:
        dev.alloc_grads(table_grad)
        dev.set_upstream(w.dh_roots, dh_nodes)
        # NaN-filled: the backward writes every row of dh_out / dc_out whole (a row it skipped stays NaN)
        dh_out = torch.full((dev.N, dev.ld), float("nan"), dtype=torch.float32, device="cuda")
        dc_out = torch.full_like(dh_out, float("nan"))
        dev.backward(dh_out, dc_out, mask)
        torch.cuda.synchronize()
        node_pos = dev.sched_arrays()["node_pos"]
        dhp, dcp = dh_out.cpu().numpy(), dc_out.cpu().numpy()
        assert np.isfinite(dhp).all() and np.isfinite(dcp).all(), "gradient rows left unwritten"
        assert not dhp[:, dev.H:].any() and not dcp[:, dev.H:].any(), "nonzero pad columns"
        out["dh"] = dhp[:, :dev.H][node_pos].astype(np.float64)
        out["dc"] = dcp[:, :dev.H][node_pos].astype(np.float64)
        out["grads"], out["d_table"] = dev.weight_grads()
    out["h"], out["c"] = dev.node_states()
    torch.cuda.synchronize()
    ld = dev.ld
    roots = dev.roots.float().cpu().numpy()[:dev.R, :dev.H].astype(np.float64)
    out["roots"] = roots
    out["sched"] = dev.sched_arrays()
    out["dev"] = dev
    return out


def run_oracle(w, dh_nodes=None, table_grad=False, backward=None, u_mask=None):
    backward = w.backward if backward is None else backward
    b, P = oracle_batch(w), oracle_params(w)
    f = EV.forward(b, P, w.hidden, w.leaf_table, u_mask)
    out = {"h": f["h"], "c": f["c"], "roots_nodes": EV.roots(b)}
    if backward:
        bw = EV.backward(b, P, w.hidden, w.leaf_table, f, w.dh_roots.astype(np.float64), dh_nodes,
                         want_table_grad=table_grad)
        out.update(dh=bw["dh"], dc=bw["dc"], grads=bw["grads"], d_table=bw["d_table"])
    return out


def compare_all(w, g, o, tol=None, check_backward=None, table_grad=False, whole_keys=()):
    """whole_keys: state tensors among h, c, dh, dc compared as one row (like the weight gradients)."""
    tol = TOL[w.dtype] if tol is None else tol
    errs = {}
    errs["h"] = compare.rel_err(g["h"], o["h"], whole="h" in whole_keys)
    errs["c"] = compare.rel_err(g["c"], o["c"], whole="c" in whole_keys)
    errs["roots"] = compare.rel_err(g["roots"], o["h"][o["roots_nodes"]])
    check_backward = w.backward if check_backward is None else check_backward
    if check_backward:
        errs["dh"] = compare.rel_err(g["dh"], o["dh"], whole="dh" in whole_keys)
        errs["dc"] = compare.rel_err(g["dc"], o["dc"], whole="dc" in whole_keys)
        for s, (gg, oo) in enumerate(zip(g["grads"], o["grads"])):
            for name in ("W_in", "W_rec", "bias"):
                if gg.get(name) is None or oo.get(name) is None:
                    continue
                errs[f"set{s}.{name}"] = compare.rel_err(gg[name], oo[name], whole=True)
        if table_grad:
            errs["d_table"] = compare.rel_err(g["d_table"], o["d_table"], whole=True)
    bad = {k: v for k, v in errs.items() if not (v <= tol)}
    assert not bad, f"over tolerance {tol}: {bad} (all: {errs})"
    return errs


def sampled_parity(w, sample, table_grad, u_mask=None, dh_nodes=None, exclude=(), raw=False, whole_keys=()):
    """Parity of a full-size batch on sampled graphs, for batches too large for the node-by-node oracle.

    Two properties that hold at any size carry it: batching invariance (a graph's states inside the batch
    equal those of the graph alone, so the sampled graphs' states are compared with the oracle on them
    alone) and linearity of the backward pass in the upstream gradient (with zero root and node gradients
    on every other graph, those graphs contribute exactly nothing: the full-batch weight gradients equal
    the oracle's on the sampled graphs alone, and every other node's gradient is exactly 0).
    u_mask, dh_nodes: [N, H] in node order (recurrent-dropout mask, per-node upstream gradient) or None;
    dh_nodes is zeroed outside the sampled graphs here.  exclude: gradient keys ("set<s>.<name>") left to the
    caller, who gets (errs, the device results, the oracle's on the sample, the sample's node rows) with raw."""
    from paper_1702_02181_amd import gen
    tol = TOL[w.dtype]
    rpg = gen.roots_per_graph(w.graph_ptr, w.child_idx)
    roff = np.concatenate([[0], np.cumsum(rpg)])
    dh = np.zeros_like(w.dh_roots)
    for g in sample:
        dh[roff[g]:roff[g + 1]] = w.dh_roots[roff[g]:roff[g + 1]]
    w.dh_roots = dh
    gp = w.graph_ptr
    rows = np.concatenate([np.arange(gp[g], gp[g + 1]) for g in sample])
    if dh_nodes is not None:
        keep = np.zeros((w.num_nodes, w.hidden), np.float32)
        keep[rows] = dh_nodes[rows]
        dh_nodes = keep
    g_out = run_device(w, dh_nodes=dh_nodes, table_grad=table_grad, u_mask=u_mask)
    sub = gen.subset(w, sample)
    o = run_oracle(sub, dh_nodes=None if dh_nodes is None else dh_nodes[rows].astype(np.float64),
                   table_grad=table_grad, u_mask=None if u_mask is None else u_mask[rows])
    errs = {k: compare.rel_err(g_out[k][rows], o[k], whole=k in whole_keys) for k in ("h", "c", "dh", "dc")}
    others = np.ones(w.num_nodes, bool)
    others[rows] = False
    assert np.all(g_out["dh"][others] == 0) and np.all(g_out["dc"][others] == 0)
    for s, (gg, oo) in enumerate(zip(g_out["grads"], o["grads"])):
        for name in ("W_in", "W_rec", "bias"):
            if gg.get(name) is None or oo.get(name) is None or f"set{s}.{name}" in exclude:
                continue
            errs[f"set{s}.{name}"] = compare.rel_err(gg[name], oo[name], whole=True)
    if table_grad:
        errs["d_table"] = compare.rel_err(g_out["d_table"], o["d_table"], whole=True)
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, (bad, errs)
    return (errs, g_out, o, rows) if raw else errs


def scorer_terms(w, o, pset):
    """sum_r |de_r| over the attention-scorer rows of parameter set pset, de_r = dh_r . h_child(r) + dc_r[1]
    (from the oracle's per-node gradients and states): the magnitude of the terms of the scorer's bias
    gradient, the scale of that sum's rounding error."""
    from paper_1702_02181_amd import gen
    tot = 0.0
    for v in range(w.num_nodes):
        op = w.ops[int(w.node_op[v])]
        if op.kind != gen.KIND_ATTN_SCORE or op.param_set != pset:
            continue
        c = int(w.child_idx[w.child_ptr[v]])
        hc = o["h"][c] if c >= 0 else np.zeros(w.hidden)
        tot += abs(float(np.dot(o["dh"][v], hc)) + float(o["dc"][v][1]))
    return tot
