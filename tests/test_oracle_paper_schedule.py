"""Pins of the oracle's paper-form schedule (Section 2's five steps with typed states and pass-throughs).

  * Figure 1 worked out by hand: ((word_1, word_3), word_5) with an int word-id state and a float state
    (tests/golden/fig1_paper_schedule.json), and a hand-derived two-output operation whose outputs have
    different types (tests/golden/multi_output_paper_schedule.json): depths, state sizes, pass-throughs,
    batches, gather indices and every edge label;
  * random typed DAGs: running the schedule symbolically -- each depth's concatenations rebuilt from the
    batches in operation, output-slot and batch order, every gather resolved -- hands every operation node
    exactly the values its edges name and every pass-through the value it carries; the pass-through count
    equals a brute-force count; every label is inside its state; batch keys strictly increase;
  * malformed graphs are rejected."""
import numpy as np
import pytest

from oracle import paper_schedule as PS
from tests.typed_graphs import load_fixture, random_ops, random_typed_batch


@pytest.mark.parametrize("name", ["fig1_paper_schedule.json", "multi_output_paper_schedule.json"])
def test_hand_derived_fixture(name):
    fx, ops, g = load_fixture(name)
    r = PS.paper_schedule(*g, ops, fx["num_types"])
    e = fx["expected"]
    assert r["num_levels"] == e["num_levels"]
    assert r["depth"] == e["depth"]
    assert r["state_size"] == e["state_size"]
    assert [list(p) for p in r["passes"]] == e["passes"]
    assert [{k: b[k] for k in ("depth", "op", "rows", "gather_off")} for b in r["batches"]] == e["batches"]
    assert r["gather"] == e["gather"]
    assert sorted([v, j, *lab] for (v, j), lab in r["edge_label"].items()) == sorted(e["edge_labels"])


def symbolic_run(g, ops, T, r):
    """Execute the schedule on value identities; returns what every item received."""
    node_op, in_ptr, in_node, in_slot = g
    n, K = len(node_op), len(ops)
    D = r["num_levels"]
    state = [[[] for _ in range(T)] for _ in range(D + 1)]
    for v in range(n):
        if node_op[v] < 0:
            state[0][-1 - node_op[v]].append((v, 0))
    got = {}
    by_depth = {}
    for b in r["batches"]:
        by_depth.setdefault(b["depth"], []).append(b)
    for d in range(1, D + 1):
        for b in by_depth.get(d, []):
            o, rows, off = b["op"], b["rows"], b["gather_off"]
            in_types = ops[o][0] if o < K else [o - K]
            out_types = ops[o][1] if o < K else [o - K]
            for ri, item in enumerate(b["items"]):
                got[(item, d)] = [state[d - 1][t][r["gather"][off + j * rows + ri]] for j, t in enumerate(in_types)]
            # this batch's share of the depth-d concatenations: slot order, then batch order
            for k, t in enumerate(out_types):
                for item in b["items"]:
                    state[d][t].append((item[1], k) if item[0] == "node" else (item[1], item[2]))
    return got, state


@pytest.mark.parametrize("seed", range(12))
def test_random_typed_dags_run_as_the_original_graph(seed):
    rng = np.random.default_rng(300 + seed)
    T = int(rng.integers(1, 4))
    ops = random_ops(rng, T, int(rng.integers(1, 5)))
    gp, node_op, in_ptr, in_node, in_slot = random_typed_batch(rng, T, ops, int(rng.integers(1, 12)),
                                                               int(rng.integers(1, 40)))
    g = (node_op, in_ptr, in_node, in_slot)
    r = PS.paper_schedule(*g, ops, T)
    got, state = symbolic_run(g, ops, T, r)
    n = len(node_op)
    depth = r["depth"]
    for v in range(n):
        if node_op[v] >= 0:
            want = [(int(in_node[e]), int(in_slot[e])) for e in range(in_ptr[v], in_ptr[v + 1])]
            assert got[(("node", v), depth[v])] == want, v
    for (u, k, d) in r["passes"]:
        assert got[(("pass", u, k), d)] == [(u, k)]
    # every pass-through instance of a value carries that value (checked per depth from the states)
    for (u, k, d) in r["passes"]:
        assert (u, k) in state[d][PS.out_types(node_op, ops, u)[k]]
    assert [[len(s) for s in st] for st in state] == r["state_size"]
    # brute-force pass-through count: readers deeper than one level below the value
    last = {}
    for v in range(n):
        for e in range(in_ptr[v], in_ptr[v + 1]):
            key = (int(in_node[e]), int(in_slot[e]))
            last[key] = max(last.get(key, 0), depth[v])
    assert len(r["passes"]) == sum(max(0, L - depth[u] - 1) for (u, _k), L in last.items())
    keys = [(b["depth"], b["op"]) for b in r["batches"]]
    assert keys == sorted(set(keys)) and len(keys) == len(set(keys))
    assert r["num_levels"] == max([0] + depth)
    for (v, j), (d, t, i) in r["edge_label"].items():
        assert d == depth[v] - 1 and 0 <= i < r["state_size"][d][t]


def test_malformed_graphs_are_rejected():
    fx, ops, (node_op, in_ptr, in_node, in_slot) = load_fixture("fig1_paper_schedule.json")
    bad_type = in_slot.copy()
    with pytest.raises(ValueError):  # the cell's input from output 1 of an embed (it has one output)
        s = in_slot.copy()
        s[3] = 1
        PS.paper_schedule(node_op, in_ptr, in_node, s, ops, 2)
    with pytest.raises(ValueError):  # an embed reading a float (type mismatch)
        nn = in_node.copy()
        nn[0] = 3
        PS.paper_schedule(node_op, in_ptr, nn, in_slot, ops, 2)
    with pytest.raises(ValueError):  # a cycle
        nn = in_node.copy()
        nn[3] = 7
        PS.paper_schedule(node_op, in_ptr, nn, bad_type, ops, 2)
    with pytest.raises(ValueError):  # an operation out of range
        no = node_op.copy()
        no[3] = 5
        PS.paper_schedule(no, in_ptr, in_node, in_slot, ops, 2)
