"""The seeded generators: reproducible, and shaped like the workloads they stand for."""
import numpy as np
import pytest

from paper_1702_02181_amd import gen


def _eq(a, b):
    for k in ("graph_ptr", "node_op", "child_ptr", "child_idx", "node_input"):
        assert np.array_equal(getattr(a, k), getattr(b, k)), k
    assert np.array_equal(a.leaf_table, b.leaf_table)
    assert np.array_equal(a.dh_roots, b.dh_roots)
    for p, q in zip(a.params, b.params):
        for n in ("W_in", "W_rec", "bias"):
            x, y = getattr(p, n), getattr(q, n)
            assert (x is None and y is None) or np.array_equal(x, y)


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_reproducible(k):
    _eq(gen.make_config(k), gen.make_config(k))


def test_config_shapes():
    w1 = gen.config1()
    assert w1.num_graphs == 8 and w1.hidden == 64 and w1.leaf_table.shape == (100, 64)
    leaves = np.diff(w1.graph_ptr) // 2 + 1          # binary tree: n = 2 L - 1
    assert np.all((leaves >= 2) & (leaves <= 16))
    w2 = gen.config2()
    assert w2.num_nodes == 130816 and w2.num_edges == 130560 and w2.leaf_table.shape == (65536, 256)
    w3 = gen.config3()
    nl = (np.diff(w3.graph_ptr) + 1) // 2
    assert w3.num_graphs == 1024 and nl.min() >= 5 and nl.max() <= 60
    assert np.all(gen.to_bf16_bits(w3.params[0].W_rec).view(np.uint16) is not None)
    assert np.array_equal(gen.round_bf16(w3.params[0].W_rec), w3.params[0].W_rec)
    w4 = gen.config4()
    assert w4.num_graphs == 512 and w4.dh_roots.shape == (512, 512)
    assert set(np.unique(w4.node_op)) == {0, 1, 2}


def test_bf16_rounding_ties_to_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 1.0 + 2 ** -9], np.float32)
    r = gen.round_bf16(x)
    assert r[0] == 1.0 and r[1] == 1.0 and r[2] == 1.0 + 4 * 2 ** -8 and r[3] == -2.5
    assert r[4] == 1.0


def test_config5_small_shape():
    w = gen.config5(num_graphs=8, hidden=4, vocab=50, spine_range=(20, 40), balanced_leaves=32)
    # every graph keeps one root; no node is orphaned by the sharing step
    assert np.all(gen.roots_per_graph(w.graph_ptr, w.child_idx) == 1)
    indeg = np.bincount(w.child_idx[w.child_idx >= 0], minlength=w.num_nodes)
    assert indeg.max() >= 2                     # some sub-expressions are shared


def test_table1_workloads():
    """Table 1 (Section 2.1): trees of 127 nodes (64 leaves) with embedding-lookup leaves; "dynamic" repeats one
    random shape, "full" draws a shape per tree, "manual" is the dynamic batch with one operation per node
    position.  The reference scheduler then gives one group per tree node for "manual" and one per (depth, op)
    otherwise, and the fp64 oracle computes identical states for "manual" and "dynamic"."""
    from oracle import evaluate as EV
    from oracle import schedule as OS
    from tests._helpers import oracle_batch, oracle_params
    B = 6
    d, m, f = (gen.table1(B, k, hidden=4, vocab=30) for k in ("dynamic", "manual", "full"))
    for w in (d, m, f):
        assert w.num_graphs == B and np.all(np.diff(w.graph_ptr) == 127) and not w.backward
    assert np.array_equal(d.child_idx, m.child_idx) and np.array_equal(d.node_input, m.node_input)
    assert np.all(d.child_idx.reshape(B, -1) - d.child_idx.reshape(B, -1)[0] == (np.arange(B) * 127)[:, None])
    assert not np.array_equal(f.child_idx, d.child_idx)
    assert m.num_ops == 127 and sorted(set(m.node_op.tolist())) == list(range(127))
    def sched(w):
        b = oracle_batch(w)
        return OS.reference_schedule(b["node_op"], b["child_ptr"], b["child_idx"], b["node_input"], b["ops"])
    sm = sched(m)
    assert len(sm["group_rows"]) == 127 and all(int(r) == B for r in sm["group_rows"])
    sd = sched(d)
    # one group per (depth, op): at most two per depth, every group a multiple of the batch
    assert sd["num_levels"] <= len(sd["group_rows"]) <= 2 * sd["num_levels"]
    assert all(int(r) % B == 0 for r in sd["group_rows"])
    hd = EV.forward(oracle_batch(d), oracle_params(d), d.hidden, d.leaf_table)["h"]
    hm = EV.forward(oracle_batch(m), oracle_params(m), m.hidden, m.leaf_table)["h"]
    assert np.array_equal(hd, hm)
