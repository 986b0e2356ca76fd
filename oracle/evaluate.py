"""Forward and backward over whole batches, node by node (oracle; test infrastructure only).

The forward pass evaluates every graph of the batch on its own, each node by
memoised recursion (children first), in fp64 and without any batching --
which is what dynamic batching must reproduce, since batching only rewrites
the graph (Section 2).  The backward pass visits the nodes in reverse
topological order (the reverse of a depth-first post-order), applies the
hand-derived per-node gradients of ``cells`` and sums the contributions a
child receives from all of its parents.

Arrays in and out are in NODE order (row v = node v).  ``params`` is a list of
dicts with float64 ``W_in``, ``W_rec``, ``bias`` (None where absent); ``ops`` a
list of (kind, arity, has_input, param_set).
"""
from __future__ import annotations

import sys

import numpy as np

from . import cells


def _kids(batch, v):
    a, b = int(batch["child_ptr"][v]), int(batch["child_ptr"][v + 1])
    return [int(c) for c in batch["child_idx"][a:b]]


def _node_args(batch, params, H, table, v, h, c):
    """(kind, P, x, hs, cs) of node v given the states of its children."""
    kind, arity, has_input, pset = batch["ops"][int(batch["node_op"][v])]
    P = params[pset]
    x = table[int(batch["node_input"][v])] if has_input else None
    kids = _kids(batch, v)
    zero = np.zeros(H)
    hs = [h[k] if k >= 0 else zero for k in kids]
    cs = [c[k] if k >= 0 else zero for k in kids]
    while len(cs) < cells.SLOTS[kind]:          # a Tree-LSTM leaf: TreeLSTM(x, 0, 0)
        cs.append(zero)
    return kind, P, x, hs, cs


def forward(batch, params, H, table, u_mask=None):
    """Return dict(h [N,H], c [N,H], cache [N]) in node order.

    u_mask: [N, H] recurrent-dropout mask in node order (see cells.forward_node), or None; backward
    reads it back from the cache."""
    n = len(batch["node_op"])
    if n == 0:
        return dict(h=np.zeros((0, H)), c=np.zeros((0, H)), cache=[])
    table = np.asarray(table, dtype=np.float64)
    h = [None] * n
    c = [None] * n
    cache = [None] * n

    def evaluate(v):
        if h[v] is not None:
            return
        for k in _kids(batch, v):
            if k >= 0:
                evaluate(k)
        kind, P, x, hs, cs = _node_args(batch, params, H, table, v, h, c)
        m = None if u_mask is None else np.asarray(u_mask[v], dtype=np.float64)
        h[v], c[v], cache[v] = cells.forward_node(kind, P, H, x, hs, cs, m)

    old = sys.getrecursionlimit()
    sys.setrecursionlimit(max(old, 20000))
    try:
        gp = batch["graph_ptr"]
        for g in range(len(gp) - 1):
            for v in range(int(gp[g]), int(gp[g + 1])):
                evaluate(v)
    finally:
        sys.setrecursionlimit(old)
    return dict(h=np.stack(h), c=np.stack(c), cache=cache)


def roots(batch):
    """Nodes that are nobody's child, in ascending node id."""
    n = len(batch["node_op"])
    has_parent = np.zeros(n, dtype=bool)
    for k in batch["child_idx"]:
        if int(k) >= 0:
            has_parent[int(k)] = True
    return [v for v in range(n) if not has_parent[v]]


def postorder(batch):
    """Depth-first post-order of all nodes (children before parents)."""
    n = len(batch["node_op"])
    seen = [False] * n
    order = []
    for s in range(n):
        if seen[s]:
            continue
        seen[s] = True
        stack = [(s, iter(_kids(batch, s)))]
        while stack:
            v, it = stack[-1]
            nxt = None
            for k in it:
                if k >= 0 and not seen[k]:
                    nxt = k
                    break
            if nxt is None:
                order.append(v)
                stack.pop()
            else:
                seen[nxt] = True
                stack.append((nxt, iter(_kids(batch, nxt))))
    return order


def backward(batch, params, H, table, fwd, dh_roots, dh_nodes=None, want_table_grad=True):
    """Gradients of L = sum_r <dh_roots[r], h_root_r> (+ sum_v <dh_nodes[v], h_v>).

    Returns dict(dh [N,H], dc [N,H]: total upstream gradient of every node's
    outputs; grads: list per param set of dict(W_in, W_rec, bias) in the
    canonical layout; d_table [rows, in_dim] or None)."""
    n = len(batch["node_op"])
    table = np.asarray(table, dtype=np.float64)
    h, c, cache = fwd["h"], fwd["c"], fwd["cache"]
    dh = np.zeros((n, H))
    dc = np.zeros((n, H))
    for r, v in enumerate(roots(batch)):
        dh[v] += dh_roots[r]
    if dh_nodes is not None:
        dh += np.asarray(dh_nodes, dtype=np.float64)
    grads = []
    for P in params:
        grads.append({k: (np.zeros_like(P[k], dtype=np.float64) if P.get(k) is not None else None)
                      for k in ("W_in", "W_rec", "bias")})
    d_table = np.zeros_like(table) if want_table_grad else None
    for v in reversed(postorder(batch)):
        kind, P, x, hs, cs = _node_args(batch, params, H, table, v, h, c)
        dx, dhs, dcs, g = cells.backward_node(kind, P, H, x, hs, cs, cache[v], dh[v], dc[v])
        kids = _kids(batch, v)
        for j, k in enumerate(kids):
            if k < 0:
                continue
            if j < len(dhs):
                dh[k] += dhs[j]
            if j < len(dcs):
                dc[k] += dcs[j]
        pset = batch["ops"][int(batch["node_op"][v])][3]
        for name, val in g.items():
            grads[pset][name] += val
        if dx is not None and d_table is not None:
            d_table[int(batch["node_input"][v])] += dx
    return dict(dh=dh, dc=dc, grads=grads, d_table=d_table)
