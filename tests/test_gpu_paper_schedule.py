"""The paper-form schedule on the GPU (fold_schedule_typed) bit for bit against the oracle's five steps
(oracle.paper_schedule): Figure 1 and the two-output example worked out by hand, random typed DAG batches
(up to four types, multi-output operations, pass-throughs of constants and of operation outputs, shuffled
node ids), the sentiment-tree workload in typed form (int word ids, embed, leaf and internal Tree-LSTM with
two outputs each), and the error codes."""
import numpy as np
import pytest

from oracle import paper_schedule as PS
from paper_1702_02181_amd import gen
from tests.typed_graphs import load_fixture, random_ops, random_typed_batch, tree_lstm_paper_form

pytestmark = pytest.mark.gpu


def _gpu(gp, g, ops, T):
    import torch
    from paper_1702_02181_amd import fold as F
    i32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.int32)).cuda()
    s = F.TypedSchedule(i32(gp), i32(g[0]), i32(g[1]), i32(g[2]), i32(g[3]), ops, T)
    return s.arrays()


def _assert_equal(gs, r, g, T):
    node_op, in_ptr, in_node, in_slot = g
    D = r["num_levels"]
    assert gs["num_levels"] == D
    assert np.array_equal(gs["depth"], r["depth"])
    assert np.array_equal(gs["state_size"].reshape(D + 1, T), np.array(r["state_size"]).reshape(D + 1, T))
    assert np.array_equal(gs["host"]["state_size"], gs["state_size"])
    bt = r["batches"]
    for key, name in (("depth", "batch_depth"), ("op", "batch_op"), ("rows", "batch_rows"),
                      ("gather_off", "batch_gather_off")):
        want = np.array([b[key] for b in bt], np.int32)
        assert np.array_equal(gs[name], want), name
        assert np.array_equal(gs["host"][name], want), "host " + name
    assert np.array_equal(gs["gather"], np.array(r["gather"], np.int32))
    passes = np.array(r["passes"], np.int32).reshape(-1, 3)
    assert np.array_equal(gs["pass_node"], passes[:, 0])
    assert np.array_equal(gs["pass_slot"], passes[:, 1])
    assert np.array_equal(gs["pass_depth"], passes[:, 2])
    items = []
    pindex = {(u, k, d): p for p, (u, k, d) in enumerate(r["passes"])}
    for b in bt:
        for it in b["items"]:
            items.append(it[1] if it[0] == "node" else -1 - pindex[(it[1], it[2], b["depth"])])
    assert np.array_equal(gs["item_node"], np.array(items, np.int32))
    begins = np.cumsum([0] + [b["rows"] for b in bt])[:-1]
    assert np.array_equal(gs["batch_item_begin"], begins.astype(np.int32))
    want_edge = np.zeros(len(in_node), np.int32)
    for (v, j), (_d, _t, i) in r["edge_label"].items():
        want_edge[in_ptr[v] + j] = i
    assert np.array_equal(gs["edge_index"], want_edge)


@pytest.mark.parametrize("name", ["fig1_paper_schedule.json", "multi_output_paper_schedule.json"])
def test_hand_derived_fixtures(name):
    fx, ops, g = load_fixture(name)
    T = fx["num_types"]
    gs = _gpu(np.array([0, len(g[0])], np.int32), g, ops, T)
    r = PS.paper_schedule(*g, ops, T)
    _assert_equal(gs, r, g, T)
    assert list(gs["gather"]) == fx["expected"]["gather"]


@pytest.mark.parametrize("seed", range(10))
def test_random_typed_batches(seed):
    rng = np.random.default_rng(900 + seed)
    T = int(rng.integers(1, 5))
    ops = random_ops(rng, T, int(rng.integers(1, 7)))
    gp, *g = random_typed_batch(rng, T, ops, int(rng.integers(1, 60)), int(rng.integers(1, 80)))
    gs = _gpu(gp, g, ops, T)
    _assert_equal(gs, PS.paper_schedule(*g, ops, T), g, T)


def test_sentiment_trees_in_paper_form():
    w = gen.config3(num_graphs=300, hidden=8, vocab=100, emb_dim=8)
    (gp, *g), ops, T = tree_lstm_paper_form(w)
    gs = _gpu(gp, g, ops, T)
    r = PS.paper_schedule(*g, ops, T)
    _assert_equal(gs, r, g, T)
    assert r["passes"], "parse-shaped trees read shallow leaves from deep parents: pass-throughs exist"


def test_errors():
    from paper_1702_02181_amd import fold as F
    fx, ops, (node_op, in_ptr, in_node, in_slot) = load_fixture("fig1_paper_schedule.json")
    gp = np.array([0, len(node_op)], np.int32)

    def code(g, o=ops, T=2, graph_ptr=gp):
        with pytest.raises(F.FoldError) as e:
            _gpu(graph_ptr, g, o, T)
        return e.value.code

    s = in_slot.copy()
    s[3] = 1  # the cell reads output 1 of an embed, which has one output
    assert code((node_op, in_ptr, in_node, s)) == F.FOLD_E_INVALID
    n = in_node.copy()
    n[0] = 3  # an embed reads a float: wrong type
    assert code((node_op, in_ptr, n, in_slot)) == F.FOLD_E_INVALID
    n = in_node.copy()
    n[3] = 7  # a cycle through the two cells
    assert code((node_op, in_ptr, n, in_slot)) == F.FOLD_E_CYCLE
    o = node_op.copy()
    o[3] = 9
    assert code((o, in_ptr, in_node, in_slot)) == F.FOLD_E_OP
    o = node_op.copy()
    o[0] = -5  # a constant of type 4 with 2 types
    assert code((o, in_ptr, in_node, in_slot)) == F.FOLD_E_OP
    # two graphs with an edge across them
    assert code((node_op, in_ptr, in_node, in_slot), graph_ptr=np.array([0, 4, 8], np.int32)) == F.FOLD_E_CHILD
    assert code((node_op, in_ptr, in_node, in_slot), o=[([0], [1]), ([1, 1], [1])], T=0) == F.FOLD_E_INVALID
