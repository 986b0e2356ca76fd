"""Typed computation graphs for the paper-form schedule (seeded generators and fixture loading; none of the
method's arithmetic).  A graph is (node_op, in_ptr, in_node, in_slot) with node_op[v] = -1 - t for a constant
of type t, and ops = [(in_types, out_types)]."""
from __future__ import annotations

import json
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def from_nodes(nodes):
    node_op = np.array([n["op"] for n in nodes], np.int32)
    in_ptr = np.zeros(len(nodes) + 1, np.int32)
    in_node, in_slot = [], []
    for v, n in enumerate(nodes):
        for (u, k) in n["inputs"]:
            in_node.append(u)
            in_slot.append(k)
        in_ptr[v + 1] = len(in_node)
    return node_op, in_ptr, np.array(in_node, np.int32), np.array(in_slot, np.int32)


def load_fixture(name):
    fx = json.load(open(os.path.join(GOLDEN, name)))
    ops = [(list(a), list(b)) for a, b in fx["ops"]]
    return fx, ops, from_nodes(fx["nodes"])


def random_ops(rng, num_types, num_ops, max_in=3, max_out=3):
    ops = []
    for _ in range(num_ops):
        nin = int(rng.integers(1, max_in + 1))
        nout = int(rng.integers(1, max_out + 1))
        ops.append(([int(t) for t in rng.integers(0, num_types, nin)],
                    [int(t) for t in rng.integers(0, num_types, nout)]))
    return ops


def random_typed_batch(rng, num_types, ops, n_graphs, max_nodes, const_frac=0.3):
    """Graphs as contiguous node ranges (graph_ptr); inside a graph, nodes read earlier nodes' outputs of the
    right type (constants are created on demand), then the node ids of each graph are shuffled."""
    node_op, ins = [], []
    graph_ptr = [0]
    for _ in range(n_graphs):
        base = len(node_op)
        local_op, local_in = [], []
        outs = {t: [] for t in range(num_types)}  # available (local node, slot) per type

        def const(t):
            local_op.append(-1 - t)
            local_in.append([])
            outs[t].append((len(local_op) - 1, 0))
            return outs[t][-1]

        n_target = int(rng.integers(1, max_nodes + 1))
        while len(local_op) < n_target:
            if rng.random() < const_frac:
                const(int(rng.integers(num_types)))
                continue
            o = int(rng.integers(len(ops)))
            srcs = []
            for t in ops[o][0]:
                if not outs[t] or rng.random() < 0.15:
                    srcs.append(const(t))
                else:
                    srcs.append(outs[t][int(rng.integers(len(outs[t])))])
            local_op.append(o)
            local_in.append(srcs)
            v = len(local_op) - 1
            for k, t in enumerate(ops[o][1]):
                outs[t].append((v, k))
        perm = rng.permutation(len(local_op))  # new id of local node i
        inv = np.argsort(perm)
        for new in range(len(local_op)):
            old = int(inv[new])
            node_op.append(local_op[old])
            ins.append([(base + int(perm[u]), k) for (u, k) in local_in[old]])
        graph_ptr.append(len(node_op))
    in_ptr = np.zeros(len(node_op) + 1, np.int32)
    in_node, in_slot = [], []
    for v, lst in enumerate(ins):
        for (u, k) in lst:
            in_node.append(u)
            in_slot.append(k)
        in_ptr[v + 1] = len(in_node)
    return (np.array(graph_ptr, np.int32), np.array(node_op, np.int32), in_ptr, np.array(in_node, np.int32),
            np.array(in_slot, np.int32))


def tree_lstm_paper_form(w):
    """A binary Tree-LSTM batch (leaves with a leaf-table row, internal nodes of arity 2) in the paper's typed
    form: type 0 = int word id (the leaf-table row, a constant), type 1 = float state; operations 0 = embed
    (int -> float), 1 = leaf Tree-LSTM (embedding -> h, c), 2 = internal Tree-LSTM (h_l, c_l, h_r, c_r -> h, c)
    -- as in Section 3.5, where a word is TreeLSTM(Embedding(word), 0, 0).  Returns (graph_ptr, node_op,
    in_ptr, in_node, in_slot), ops, num_types."""
    ops = [([0], [1]), ([1], [1, 1]), ([1, 1, 1, 1], [1, 1])]
    node_op, ins, graph_ptr = [], [], [0]
    cp, ci, ni = w.child_ptr, w.child_idx, w.node_input
    for g in range(w.num_graphs):
        a, b = int(w.graph_ptr[g]), int(w.graph_ptr[g + 1])
        local = {}
        order = []

        def add(op, inputs):
            node_op.append(op)
            ins.append(inputs)
            return len(node_op) - 1

        for v in range(a, b):  # generator graphs list children before parents
            kids = [int(c) for c in ci[cp[v]:cp[v + 1]]]
            if not kids:
                tok = add(-1, [])
                emb = add(0, [(tok, 0)])
                local[v] = add(1, [(emb, 0)])
            else:
                l, r = local[kids[0]], local[kids[1]]
                local[v] = add(2, [(l, 0), (l, 1), (r, 0), (r, 1)])
            order.append(v)
        graph_ptr.append(len(node_op))
    in_ptr = np.zeros(len(node_op) + 1, np.int32)
    in_node, in_slot = [], []
    for v, lst in enumerate(ins):
        for (u, k) in lst:
            in_node.append(u)
            in_slot.append(k)
        in_ptr[v + 1] = len(in_node)
    return ((np.array(graph_ptr, np.int32), np.array(node_op, np.int32), in_ptr, np.array(in_node, np.int32),
             np.array(in_slot, np.int32)), ops, 2)
