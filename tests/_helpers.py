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
    ops: list of gen.OpSpec; params: list of gen.ParamSet (float32 arrays)."""
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
