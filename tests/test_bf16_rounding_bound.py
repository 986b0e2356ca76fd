"""How far bf16 storage of h alone moves the states from the fp64 oracle (a CPU diagnostic beside the
oracle; it leaves the oracle unchanged).

The bf16 path stores every node's h in bf16 (round to nearest even) and its parents read that rounded
value; weights and leaf tables are bf16 values already (the oracle sees those exact values).  Emulating
only that rounding -- the oracle's own per-node cells in fp64, with h rounded to bf16 after every node --
gives the error that no kernel can avoid at a given workload, against the same metric and the 2e-2 bar:

  * random trees with N(0, 0.2^2) weights at H = 256 (K = 512 terms per gate; the z of a node amplifies
    its children's rounding, tree level after tree level) reach ~0.011 on h, under the bar.  Measured
    against an oracle that is given the weights and table UNROUNDED, the same emulation reaches ~0.028:
    that is the 0.028 the GPU once showed on this batch, when the test fed the oracle the fp32 values of
    weights the GPU stores in bf16 -- an input mismatch of the test, not a kernel defect;
  * the sentiment-tree workload (parse-shaped trees, H = 300, U(-0.1, 0.1) weights, a dropout mask)
    stays well under the bar, and its GPU parity test runs at that shape."""
import numpy as np

from oracle import cells, compare, evaluate as EV
from paper_1702_02181_amd import gen
from tests._helpers import dropout_mask, dropout_tree_case, oracle_batch, oracle_params


def _forward_bf16_h(w, u_mask):
    """h [N, H] of the batch with every node's h rounded to bf16 before its parents read it."""
    b, P = oracle_batch(w), oracle_params(w)
    H = w.hidden
    table = np.asarray(w.leaf_table, np.float64)
    n = w.num_nodes
    h = [None] * n
    c = [None] * n
    zero = np.zeros(H)
    order = []
    state = np.zeros(n, np.int8)
    for root in range(n):  # iterative post-order: children before parents
        if state[root]:
            continue
        stack = [(root, False)]
        while stack:
            v, done = stack.pop()
            if done:
                order.append(v)
                continue
            if state[v]:
                continue
            state[v] = 1
            stack.append((v, True))
            for k in w.child_idx[w.child_ptr[v]:w.child_ptr[v + 1]]:
                if k >= 0 and not state[k]:
                    stack.append((int(k), False))
    for v in order:
        kind, arity, has_input, pset = b["ops"][int(w.node_op[v])]
        kids = [int(k) for k in w.child_idx[w.child_ptr[v]:w.child_ptr[v + 1]]]
        hs = [h[k] if k >= 0 else zero for k in kids]
        cs = [c[k] if k >= 0 else zero for k in kids]
        while len(cs) < cells.SLOTS[kind]:
            cs.append(zero)
        x = table[int(w.node_input[v])] if has_input else None
        m = None if u_mask is None else np.asarray(u_mask[v], np.float64)
        hv, cv, _ = cells.forward_node(kind, P[pset], H, x, hs, cs, m)
        h[v] = gen.round_bf16(hv.astype(np.float32)).astype(np.float64)
        c[v] = cv
    return np.stack(h)


def _h_error(w, mask, ref_w=None):
    ref_w = w if ref_w is None else ref_w
    ref = EV.forward(oracle_batch(ref_w), oracle_params(ref_w), ref_w.hidden, ref_w.leaf_table, mask)["h"]
    return compare.rel_err(_forward_bf16_h(w, mask), ref)


def test_h_rounding_alone_stays_under_the_bar_on_random_trees():
    w, mask, _ = dropout_tree_case("bf16", 256, 400, 8)
    e = _h_error(w, mask)
    print("bf16 h rounding, random trees H=256 scale 0.2:", e)
    assert e < C_TOL


def test_unrounded_oracle_inputs_explain_the_former_excess():
    w, mask, _ = dropout_tree_case("bf16", 256, 400, 8)
    w_unrounded, mask_u, _ = dropout_tree_case("bf16", 256, 400, 8, round_values=False)
    assert np.array_equal(mask, mask_u)
    assert not np.array_equal(w.params[0].W_rec, w_unrounded.params[0].W_rec)
    e = _h_error(w, mask, ref_w=w_unrounded)
    print("bf16 h rounding against unrounded weights, random trees H=256 scale 0.2:", e)
    assert 0.02 < e < 0.04


def test_rounding_alone_stays_under_the_bar_on_sentiment_trees():
    w = gen.subset(gen.config3(num_graphs=96), list(range(96)))
    mask = dropout_mask(np.random.default_rng(3), w.num_nodes, w.hidden, 0.25)
    e = _h_error(w, mask)
    print("bf16 h rounding, sentiment trees H=300:", e)
    assert e < 0.5 * C_TOL


C_TOL = 2e-2
