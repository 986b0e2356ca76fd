"""Shared test helpers: small hand-built batches and the adapter from generated
workloads to the oracle's plain-dict inputs.  Holds none of the method's arithmetic."""
from __future__ import annotations

import numpy as np

from paper_1702_02181_amd import gen


def oracle_batch(w: gen.Workload) -> dict:
    return dict(graph_ptr=w.graph_ptr, node_op=w.node_op, child_ptr=w.child_ptr,
                child_idx=w.child_idx, node_input=w.node_input,
                ops=[(o.kind, o.arity, o.has_input, o.param_set) for o in w.ops])


def oracle_params(w: gen.Workload) -> list:
    out = []
    for p in w.params:
        out.append(dict(
            W_in=None if p.W_in is None else p.W_in.astype(np.float64),
            W_rec=None if p.W_rec is None else p.W_rec.astype(np.float64),
            bias=p.bias.astype(np.float64)))
    return out


def make_workload(graphs, ops, params, H, table, dtype="f32", dh_roots=None, seed=0, name="tiny"):
    """graphs: list of lists of (op, [local children or -1], input_row or -1).
    ops: list of gen.OpSpec; params: list of gen.ParamSet (float32 arrays).  For dtype "bf16" the weights
    and the leaf table are rounded to bf16 here (biases stay fp32), so the oracle sees exactly the values
    the GPU stores."""
    if dtype == "bf16":
        rb = lambda a: None if a is None else gen.round_bf16(a)
        params = [gen.ParamSet(p.kind, p.in_dim, p.arity, rb(p.W_in), rb(p.W_rec), p.bias) for p in params]
        table = gen.round_bf16(np.asarray(table, np.float32))
    arrs = []
    for g in graphs:
        b = gen._GraphBuilder()
        for (op, kids, inp) in g:
            b.add(op, kids, inp)
        arrs.append(b.arrays())
    csr = gen.assemble(arrs)
    r = gen.count_roots(csr["node_op"].shape[0], csr["child_idx"])
    if dh_roots is None:
        dh_roots = np.random.default_rng(seed).standard_normal((r, H)).astype(np.float32)
    return gen.Workload(name=name, dtype=dtype, hidden=H, ops=ops, params=params,
                        leaf_table=np.asarray(table, np.float32), dh_roots=dh_roots, **csr)


def random_params(rng, kind, in_dim, arity, H, scale=0.5):
    g = gen.NUM_GATES[kind]
    W_in = (scale * rng.standard_normal((in_dim, g * H))).astype(np.float32) if in_dim else None
    W_rec = (scale * rng.standard_normal((arity * H, g * H))).astype(np.float32) if arity else None
    b = (scale * rng.standard_normal(g * H)).astype(np.float32)
    return gen.ParamSet(kind, in_dim, arity, W_in, W_rec, b)


def random_tree(rng, leaves, vocab):
    """Local node list of one random-split binary tree (children before parents): op 0 = leaf with an
    input row, op 1 = internal node of arity 2."""
    nodes = []

    def build(n):
        if n == 1:
            nodes.append((0, [], int(rng.integers(vocab))))
            return len(nodes) - 1
        k = int(rng.integers(1, n))
        a, b = build(k), build(n - k)
        nodes.append((1, [a, b], -1))
        return len(nodes) - 1

    build(leaves)
    return nodes


def dropout_mask(rng, n, H, p):
    """Inverted-dropout mask [n, H]: 0 with probability p, else 1 / (1 - p)."""
    return np.where(rng.random((n, H)) < p, 0.0, 1.0 / (1.0 - p)).astype(np.float32)


def dropout_tree_case(dtype, H, trees, leaves, D_in=64, vocab=500, p=0.25, round_values=True):
    """Random Tree-LSTM trees (2..leaves leaves) with normal weights (scale 0.3 fp32, 0.2 bf16), a dropout
    mask and a per-node upstream gradient: (workload, mask, dh_nodes), all seeded by (H, trees).
    round_values=False keeps a bf16 workload's weights and table unrounded (a diagnostic only: the GPU
    would store their roundings)."""
    rng = np.random.default_rng(H + trees)
    prm = random_params(rng, gen.KIND_TREELSTM, D_in, 2, H, scale=0.3 if dtype == "f32" else 0.2)
    ops = [gen.OpSpec(gen.KIND_TREELSTM, 0, 1, 0), gen.OpSpec(gen.KIND_TREELSTM, 2, 0, 0)]
    table = rng.standard_normal((vocab, D_in)).astype(np.float32)
    graphs = [random_tree(rng, int(rng.integers(2, leaves + 1)), vocab) for _ in range(trees)]
    w = make_workload(graphs, ops, [prm], H, table, dtype=dtype if round_values else "f32", seed=7)
    w.dtype = dtype
    mask = dropout_mask(rng, w.num_nodes, H, p)
    dh_nodes = rng.standard_normal((w.num_nodes, H)).astype(np.float32)
    return w, mask, dh_nodes
