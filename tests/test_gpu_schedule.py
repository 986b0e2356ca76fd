"""GPU scheduler parity: every schedule array bit-exact against the oracle's reference scheduler."""
import json
import os

import numpy as np
import pytest

from paper_1702_02181_amd import gen
from tests import gpu_common as C
from tests._helpers import make_workload
from tests.test_oracle_schedule import random_dag

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _gpu_sched(w):
    import torch
    from paper_1702_02181_amd import fold as F
    i32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.int32)).cuda()
    s = F.Schedule(i32(w.graph_ptr), i32(w.node_op), i32(w.child_ptr), i32(w.child_idx), i32(w.node_input),
                   [(o.kind, o.arity, o.has_input, o.param_set) for o in w.ops], w.leaf_table.shape[0])
    return s.arrays()


def test_fig1_on_gpu():
    fx = json.load(open(os.path.join(GOLDEN, "fig1_schedule.json")))
    ops = [gen.OpSpec(*o) for o in fx["ops"]]
    w = make_workload([[(0, [], 1), (0, [], 3), (1, [0, 1], -1), (0, [], 5), (1, [2, 3], -1)]], ops,
                      [gen.ParamSet(0, 2, 0, None, None, np.zeros(0)), gen.ParamSet(1, 0, 2, None, None, np.zeros(2))],
                      2, np.zeros((6, 2)))
    g = _gpu_sched(w)
    for k, v in fx["expected"].items():
        if k in ("paper_labels_i",):
            continue
        if k == "num_levels":
            assert g[k] == v
        else:
            assert np.array_equal(g[k], v), k


@pytest.mark.parametrize("seed", range(8))
def test_random_shuffled_dags(seed):
    rng = np.random.default_rng(100 + seed)
    w = random_dag(rng, n_graphs=int(rng.integers(1, 40)), max_nodes=int(rng.integers(2, 60)))
    C.assert_schedule_equal(_gpu_sched(w), C.oracle_schedule(w))


def test_large_graph_uses_global_scratch():
    """A graph too large for the depth kernel's LDS budget (one 1500-step chain plus a tree)."""
    b = gen._GraphBuilder()
    gen.caterpillar(b, 1500, 0, 1, range(1501))
    csr = gen.assemble([b.arrays()])
    w = gen.Workload("big", "f32", 2, ops=[gen.OpSpec(2, 0, 1, 0), gen.OpSpec(2, 2, 0, 0)], params=[],
                     leaf_table=np.zeros((1501, 2), np.float32), dh_roots=np.zeros((1, 2), np.float32), **csr)
    C.assert_schedule_equal(_gpu_sched(w), C.oracle_schedule(w))


def test_more_levels_than_the_first_read_back():
    """A 5,000-step caterpillar: 5,001 levels and groups, more than fold_schedule reads back with its error
    word (4,096), so it reads the rest of the level and group tables in a second copy."""
    b = gen._GraphBuilder()
    gen.caterpillar(b, 5000, 0, 1, range(5001))
    csr = gen.assemble([b.arrays()])
    w = gen.Workload("deep", "f32", 2, ops=[gen.OpSpec(2, 0, 1, 0), gen.OpSpec(2, 2, 0, 0)], params=[],
                     leaf_table=np.zeros((5001, 2), np.float32), dh_roots=np.zeros((1, 2), np.float32), **csr)
    ref = C.oracle_schedule(w)
    assert ref["num_levels"] == 5001 and len(ref["group_op"]) > 4096
    C.assert_schedule_equal(_gpu_sched(w), ref)


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_full_config_schedules(k):
    """All five workloads at full size, config 5's 2.0 M-node batch of 4,096 DAGs included."""
    w = gen.make_config(k)
    C.assert_schedule_equal(_gpu_sched(w), C.oracle_schedule(w))


def test_config5_shape_schedule_and_shuffled():
    w = gen.config5(num_graphs=256, hidden=8, vocab=100)
    C.assert_schedule_equal(_gpu_sched(w), C.oracle_schedule(w))
    ws = gen.shuffle_within_graphs(gen.config3(num_graphs=64, hidden=8, emb_dim=8, vocab=50), 7)
    C.assert_schedule_equal(_gpu_sched(ws), C.oracle_schedule(ws))


def _err(w):
    from paper_1702_02181_amd import fold as F
    with pytest.raises(F.FoldError) as e:
        _gpu_sched(w)
    return e.value.code


def test_error_codes():
    w = gen.config1(num_graphs=3)
    sub = lambda: gen.subset(w, range(3))
    x = sub(); x.node_op = x.node_op.copy(); x.node_op[0] = 7
    assert _err(x) == -2
    x = sub(); x.node_op = x.node_op.copy(); v = int(np.nonzero(x.node_op == 1)[0][0]); x.node_op[v] = 0
    x.node_input = x.node_input.copy(); x.node_input[v] = 0
    assert _err(x) == -3
    x = sub(); x.child_idx = x.child_idx.copy(); x.child_idx[0] = x.num_nodes + 5
    assert _err(x) == -4
    x = sub(); x.child_idx = x.child_idx.copy(); x.child_idx[0] = x.num_nodes - 1
    assert _err(x) == -4
    x = sub(); x.node_input = x.node_input.copy(); x.node_input[0] = 100
    assert _err(x) == -5
    x = sub(); x.node_input = x.node_input.copy(); x.node_input[0] = -1
    assert _err(x) == -5
    x = sub(); x.graph_ptr = x.graph_ptr.copy(); x.graph_ptr[1] = x.graph_ptr[2] + 1
    assert _err(x) == -1
    # a 2-cycle and a self loop
    cyc = gen.Workload("cyc", "f32", 2, graph_ptr=np.array([0, 2], np.int32), node_op=np.array([0, 0], np.int32),
                       child_ptr=np.array([0, 1, 2], np.int32), child_idx=np.array([1, 0], np.int32),
                       node_input=np.array([-1, -1], np.int32), ops=[gen.OpSpec(4, 1, 0, 0)], params=[],
                       leaf_table=np.zeros((1, 2), np.float32), dh_roots=np.zeros((0, 2), np.float32))
    assert _err(cyc) == -6
    # the library stays usable after errors
    C.assert_schedule_equal(_gpu_sched(w), C.oracle_schedule(w))


def test_empty_batch():
    w = gen.Workload("empty", "f32", 2, graph_ptr=np.array([0], np.int32), node_op=np.zeros(0, np.int32),
                     child_ptr=np.array([0], np.int32), child_idx=np.zeros(0, np.int32),
                     node_input=np.zeros(0, np.int32), ops=[gen.OpSpec(2, 0, 1, 0)], params=[],
                     leaf_table=np.zeros((1, 2), np.float32), dh_roots=np.zeros((0, 2), np.float32))
    g = _gpu_sched(w)
    assert g["num_levels"] == 0 and g["num_groups"] == 0 and g["num_roots"] == 0


def test_many_operations_one_group_per_tree_node():
    """Table 1's manual-batching emulation: every node position of a 127-node tree is an operation of its
    own, so the schedule has one group per tree node, bit-exact against the reference scheduler; 256
    operations are accepted and 257 rejected."""
    w = gen.table1(5, "manual", hidden=8, vocab=50)
    assert w.num_ops == 127
    g = _gpu_sched(w)
    C.assert_schedule_equal(g, C.oracle_schedule(w))
    assert g["num_groups"] == 127 and list(g["host"]["group_rows"]) == [5] * 127
    many = gen.subset(w, range(5))
    many.ops = list(w.ops) + [gen.OpSpec(gen.KIND_TREELSTM, 2, 0, 0)] * (256 - 127)
    C.assert_schedule_equal(_gpu_sched(many), C.oracle_schedule(many))
    many.ops = many.ops + [gen.OpSpec(gen.KIND_TREELSTM, 2, 0, 0)]
    assert _err(many) == -1


def _expected_child_bases(w, ref):
    """Per group and child slot: the first child row when the slot's children are consecutive pool rows with
    one parent edge each, else -1 (computed here from the reference schedule and the CSR)."""
    indeg = np.zeros(w.num_nodes, np.int64)
    kids = w.child_idx[w.child_idx >= 0]
    np.add.at(indeg, kids, 1)
    pos_node = np.asarray(ref["pos_node"])
    out = np.full((2, len(ref["group_op"])), -1, np.int64)
    cp = np.asarray(ref["child_pos"])
    for g, (op, rb, rows, off) in enumerate(zip(ref["group_op"], ref["group_row_begin"], ref["group_rows"],
                                                ref["group_idx_off"])):
        a = w.ops[int(op)].arity
        for k in range(min(a, 2)):
            c = cp[int(off) + np.arange(int(rows)) * a + k]
            if c[0] < 0 or not np.array_equal(c, c[0] + np.arange(int(rows))):
                continue
            if np.all(indeg[pos_node[c]] == 1):
                out[k, g] = c[0]
    return out


@pytest.mark.parametrize("case", ["manual", "dynamic", "full", "cfg2", "cfg4", "dag"])
def test_static_layout_child_bases(case):
    """The per-slot child bases the forward kernels use to skip child_pos: every slot of a manual-batching
    schedule (one operation per node position of identically shaped trees) has one; the gathered layouts
    have them only where their children happen to be consecutive single-parent rows."""
    if case in ("manual", "dynamic", "full"):
        w = gen.table1(8, case, hidden=8, vocab=50)
    elif case == "cfg2":
        w = gen.config2(num_graphs=3, leaves=16, hidden=8)
    elif case == "cfg4":
        w = gen.config4(num_graphs=5, max_chain=20, hidden=8, in_dim=8)
    else:
        w = random_dag(np.random.default_rng(5), n_graphs=20, max_nodes=40)
    g = _gpu_sched(w)
    ref = C.oracle_schedule(w)
    want = _expected_child_bases(w, ref)
    got = np.stack([g["host"]["group_child_base0"], g["host"]["group_child_base1"]])
    assert np.array_equal(got, want)
    assert np.array_equal(np.stack([g["group_child_base0"], g["group_child_base1"]]), want)
    if case == "manual":
        internal = [i for i, op in enumerate(ref["group_op"]) if w.ops[int(op)].arity == 2]
        assert internal and np.all(want[:, internal] >= 0)
