"""Pins of the oracle's validator and reference scheduler (CPU only).

Each check ties the oracle to something other than itself: the worked
example of Figure 1, brute-force definitions on tiny DAGs (depth by
fixed-point iteration, positions by counting), closed-form level widths of
balanced trees and caterpillars, and the structural invariants of Section 2's
scheduling steps."""
import json
import os

import numpy as np
import pytest

from oracle import schedule as S
from paper_1702_02181_amd import gen
from tests._helpers import make_workload, oracle_batch

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def sched_of(w):
    b = oracle_batch(w)
    return S.reference_schedule(b["node_op"], b["child_ptr"], b["child_idx"], b["node_input"], b["ops"])


def test_fig1_worked_example():
    fx = json.load(open(os.path.join(GOLDEN, "fig1_schedule.json")))
    ops = [tuple(o) for o in fx["ops"]]
    assert S.validate(fx["graph_ptr"], fx["node_op"], fx["child_ptr"], fx["child_idx"],
                      fx["node_input"], ops, 6) == S.E_OK
    s = S.reference_schedule(fx["node_op"], fx["child_ptr"], fx["child_idx"], fx["node_input"], ops)
    exp = fx["expected"]
    for k, v in exp.items():
        if k == "paper_labels_i":
            continue
        got = s[k]
        assert np.array_equal(np.asarray(got), np.asarray(v)), k
    # the paper's per-depth index i of every edge = position minus the start of its level
    labels = []
    for g in range(len(s["group_level"])):
        a = s["group_idx_off"][g]
        ar = ops[s["group_op"][g]][1]
        for r in range(s["group_rows"][g]):
            row = []
            for k in range(ar):
                p = s["child_pos"][a + r * ar + k]
                d = s["depth"][s["pos_node"][p]]
                row.append(int(p - s["level_ptr"][d - 1]))
            if row:
                labels.append(row)
    assert labels == exp["paper_labels_i"]


def random_dag(rng, n_graphs, max_nodes, num_ops=3, p_neg=0.1):
    """Random DAG batch: each node's children are earlier nodes of its own graph
    (then node ids are shuffled inside the graph)."""
    arities = [0, 1, 2]
    ops = [gen.OpSpec(gen.KIND_TREELSTM if a != 1 else gen.KIND_PROJ, a, 1 if a == 0 else 0, 0)
           for a in arities[:num_ops]]
    graphs = []
    for _ in range(n_graphs):
        n = int(rng.integers(1, max_nodes + 1))
        nodes = []
        for v in range(n):
            if v == 0:
                op = 0
            else:
                op = int(rng.integers(0, num_ops))
            ar = ops[op].arity
            kids = []
            for _k in range(ar):
                if rng.random() < p_neg:
                    kids.append(-1)
                else:
                    kids.append(int(rng.integers(0, v)))
            nodes.append((op, kids, 0 if ops[op].has_input else -1))
        perm = rng.permutation(n)
        inv = np.empty(n, int)
        inv[perm] = np.arange(n)
        shuffled = [None] * n
        for v, (op, kids, inp) in enumerate(nodes):
            shuffled[inv[v]] = (op, [int(inv[k]) if k >= 0 else -1 for k in kids], inp)
        graphs.append(shuffled)
    return make_workload(graphs, ops, [gen.ParamSet(gen.KIND_TREELSTM, 1, 2, None, None, np.zeros(5))],
                         1, np.zeros((1, 1)))


def brute_depth(w):
    """Fixed-point iteration of the depth rule (Bellman-Ford style), independent of recursion."""
    n = w.num_nodes
    d = np.zeros(n, np.int64)
    for _ in range(n + 1):
        new = np.ones(n, np.int64)
        for v in range(n):
            for j in range(w.child_ptr[v], w.child_ptr[v + 1]):
                c = w.child_idx[j]
                if c >= 0:
                    new[v] = max(new[v], d[c] + 1)
        if np.array_equal(new, d):
            break
        d = new
    return d


@pytest.mark.parametrize("seed", range(12))
def test_schedule_bruteforce_tiny_dags(seed):
    rng = np.random.default_rng(seed)
    w = random_dag(rng, n_graphs=int(rng.integers(1, 5)), max_nodes=9)
    b = oracle_batch(w)
    assert S.validate(b["graph_ptr"], b["node_op"], b["child_ptr"], b["child_idx"], b["node_input"],
                      b["ops"], 1) == S.E_OK
    s = sched_of(w)
    d = brute_depth(w)
    assert np.array_equal(s["depth"], d)
    n, K = w.num_nodes, w.num_ops
    key = (d - 1) * K + w.node_op
    # position of v = number of nodes whose (key, id) is smaller
    pos = np.array([sum(1 for u in range(n) if (key[u], u) < (key[v], v)) for v in range(n)])
    assert np.array_equal(s["node_pos"], pos)
    assert np.array_equal(s["pos_node"][pos], np.arange(n))
    # groups: the distinct keys present, ascending
    keys = sorted(set(key.tolist()))
    assert np.array_equal(s["group_level"], [k // K + 1 for k in keys])
    assert np.array_equal(s["group_op"], [k % K for k in keys])
    assert np.array_equal(s["group_rows"], [int((key == k).sum()) for k in keys])
    assert np.array_equal(s["group_row_begin"], [int((key < k).sum()) for k in keys])
    off = 0
    for gi, k in enumerate(keys):
        assert s["group_idx_off"][gi] == off
        members = sorted(v for v in range(n) if key[v] == k)
        ar = w.ops[k % K].arity
        for r, v in enumerate(members):
            for j in range(ar):
                c = w.child_idx[w.child_ptr[v] + j]
                assert s["child_pos"][off + r * ar + j] == (pos[c] if c >= 0 else -1)
        off += len(members) * ar
    assert s["num_levels"] == (int(d.max()) if n else 0)
    assert np.array_equal(s["level_ptr"], [int((d <= lv).sum()) for lv in range(s["num_levels"] + 1)])
    parents = np.zeros(n, int)
    for c in w.child_idx:
        if c >= 0:
            parents[c] += 1
    assert np.array_equal(s["root_pos"], pos[np.nonzero(parents == 0)[0]])
    assert np.array_equal(s["input_idx"], w.node_input[s["pos_node"]])


def check_invariants(w, s):
    n = w.num_nodes
    assert sorted(s["pos_node"].tolist()) == list(range(n))
    lvl = s["depth"]
    for v in range(n):
        ks = [c for c in w.child_idx[w.child_ptr[v]:w.child_ptr[v + 1]] if c >= 0]
        assert lvl[v] == 1 + max([lvl[c] for c in ks], default=0)
        for c in ks:
            assert lvl[c] < lvl[v]
    assert s["num_levels"] == lvl.max()
    keys = (s["group_level"] - 1) * w.num_ops + s["group_op"]
    assert np.all(np.diff(keys) > 0)
    assert s["group_rows"].sum() == n
    assert np.all(s["group_rows"] > 0)


@pytest.mark.parametrize("k,kw", [(1, {}), (2, dict(num_graphs=4, leaves=16, hidden=8)),
                                  (3, dict(num_graphs=6, hidden=8, emb_dim=8, vocab=50)),
                                  (4, dict(num_graphs=5, hidden=8, in_dim=4, max_chain=12)),
                                  (5, dict(num_graphs=4, hidden=8, vocab=50, spine_range=(5, 30),
                                           balanced_leaves=16))])
def test_schedule_invariants_on_workload_shapes(k, kw):
    w = gen.make_config(k, **kw)
    s = sched_of(w)
    check_invariants(w, s)


@pytest.mark.parametrize("B,k", [(1, 0), (1, 3), (3, 4), (5, 2)])
def test_balanced_tree_level_widths(B, k):
    """B complete trees with 2^k leaves: level l holds B * 2^(k+1-l) nodes; D = k + 1."""
    w = gen.config2(num_graphs=B, leaves=2 ** k, hidden=2)
    s = sched_of(w)
    assert s["num_levels"] == k + 1
    widths = np.diff(s["level_ptr"])
    assert np.array_equal(widths, [B * 2 ** (k + 1 - lv) for lv in range(1, k + 2)])


@pytest.mark.parametrize("spine", [1, 2, 7, 40])
def test_caterpillar_level_widths(spine):
    b = gen._GraphBuilder()
    gen.caterpillar(b, spine, 0, 1, range(spine + 1))
    csr = gen.assemble([b.arrays()])
    ops = [(gen.KIND_TREELSTM, 0, 1, 0), (gen.KIND_TREELSTM, 2, 0, 0)]
    s = S.reference_schedule(csr["node_op"], csr["child_ptr"], csr["child_idx"], csr["node_input"], ops)
    assert s["num_levels"] == spine + 1
    assert np.array_equal(np.diff(s["level_ptr"]), [spine + 1] + [1] * spine)


def test_single_graph_batches_within_the_graph():
    """Batch size 1 still batches per level: a 128-leaf balanced tree needs 8 steps, not 255."""
    w = gen.config2(num_graphs=1, leaves=128, hidden=2)
    s = sched_of(w)
    assert s["num_levels"] == 8 and len(s["group_level"]) == 8
    assert w.num_nodes == 255


def _val(w, num_inputs=None, ops=None):
    b = oracle_batch(w)
    return S.validate(b["graph_ptr"], b["node_op"], b["child_ptr"], b["child_idx"], b["node_input"],
                      ops if ops is not None else b["ops"],
                      num_inputs if num_inputs is not None else w.leaf_table.shape[0])


def test_validator_error_codes():
    w = gen.config1(num_graphs=3)
    assert _val(w) == S.E_OK
    # op out of range
    w2 = gen.subset(w, range(3)); w2.node_op = w2.node_op.copy(); w2.node_op[0] = 7
    assert _val(w2) == S.E_OP
    # arity mismatch: an internal node declared as embed (arity 0) but has 2 children
    w2 = gen.subset(w, range(3)); w2.node_op = w2.node_op.copy()
    v = int(np.nonzero(w2.node_op == 1)[0][0]); w2.node_op[v] = 0; w2.node_input = w2.node_input.copy(); w2.node_input[v] = 0
    assert _val(w2) == S.E_ARITY
    # child out of range, and child in another graph
    w2 = gen.subset(w, range(3)); w2.child_idx = w2.child_idx.copy(); w2.child_idx[0] = w2.num_nodes + 5
    assert _val(w2) == S.E_CHILD
    w2 = gen.subset(w, range(3)); w2.child_idx = w2.child_idx.copy()
    w2.child_idx[0] = w2.num_nodes - 1          # a node of the last graph
    assert _val(w2) == S.E_CHILD
    # input out of range, missing input, extra input
    w2 = gen.subset(w, range(3)); w2.node_input = w2.node_input.copy(); w2.node_input[0] = 100
    assert _val(w2) == S.E_INPUT
    w2 = gen.subset(w, range(3)); w2.node_input = w2.node_input.copy(); w2.node_input[0] = -1
    assert _val(w2) == S.E_INPUT
    w2 = gen.subset(w, range(3)); w2.node_input = w2.node_input.copy()
    w2.node_input[int(np.nonzero(w2.node_op == 1)[0][0])] = 3
    assert _val(w2) == S.E_INPUT
    # broken graph_ptr
    w2 = gen.subset(w, range(3)); w2.graph_ptr = w2.graph_ptr.copy(); w2.graph_ptr[-1] += 1
    assert _val(w2) == S.E_INVALID
    # cycle: make the first leaf's parent also a child of ... itself through a 2-cycle
    ops = [(gen.KIND_PROJ, 1, 0, 0)]
    gp, op, cp, ci, ni = [0, 2], [0, 0], [0, 1, 2], [1, 0], [-1, -1]
    assert S.validate(gp, op, cp, ci, ni, ops, 0) == S.E_CYCLE
    assert S.validate([0, 1], [0], [0, 1], [0], [-1], ops, 0) == S.E_CYCLE     # self loop
    assert S.validate([0, 1], [0], [0, 1], [-1], [-1], ops, 0) == S.E_OK      # -1 = zero state


def test_empty_batch():
    s = S.reference_schedule([], [0], [], [], [(0, 0, 1, 0)])
    assert s["num_levels"] == 0 and len(s["pos_node"]) == 0 and list(s["level_ptr"]) == [0]
