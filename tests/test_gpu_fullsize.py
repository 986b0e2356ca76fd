"""Parity at the full workload sizes, in the launch configuration bench.py times.

The oracle cannot evaluate a whole 130 k - 2 M node batch node by node in test time,
so these tests sample graphs and rely on two properties that hold at any size:
  * batching invariance: a graph's states inside the full batch equal those of the
    graph evaluated alone (dynamic batching only rewrites the computation);
  * linearity of the backward pass in the upstream gradient: with the root
    gradients of every non-sampled graph set to zero, those graphs contribute exactly
    nothing, so the full-batch weight gradients equal the oracle's gradients of the
    sampled graphs alone, and every node outside them gets an exact zero gradient.
"""
import numpy as np
import pytest

from oracle import compare
from paper_1702_02181_amd import gen
from tests import gpu_common as C

pytestmark = pytest.mark.gpu


def _sampled_parity(w, sample, table_grad):
    return C.sampled_parity(w, sample, table_grad)


def test_config2_full_bench_workload():
    w = gen.config2()
    _sampled_parity(w, [0, 97, 255], table_grad=False)


def test_config3_full():
    w = gen.config3()
    _sampled_parity(w, [0, 511, 1023], table_grad=True)


def test_config4_full():
    w = gen.config4()
    # the longest chain and two others
    sizes = np.diff(w.graph_ptr)
    _sampled_parity(w, [int(np.argmax(sizes)), 1, 300], table_grad=False)


def test_config5_full():
    w = gen.config5()
    # one balanced tree with shared sub-expressions and the deepest caterpillar
    sizes = np.diff(w.graph_ptr)
    odd = np.arange(1, w.num_graphs, 2)
    deepest = int(odd[np.argmax(sizes[odd])])
    _sampled_parity(w, [0, deepest], table_grad=True)


def test_wide_kernels_bf16_h512_dag_with_node_gradients():
    """A batch that sends the wide kernels through the combinations the five workloads leave out:
    hidden 512 bf16 (two unit blocks per workgroup, 8 unit-block pairs: XCDs own column groups in the
    forward, row-shared order in dz . W^T with 4 column tiles), leaf levels of ~157 k rows (wide
    weight gradients of both ops, wide leaf-table gradient), caterpillar tails of a few hundred rows
    (K-split with atomic slices), shared sub-expressions, and an upstream gradient on every node of
    the sampled graphs.  Sampled parity as above (graph order, linearity)."""
    w = gen.config5(num_graphs=512, hidden=512, vocab=2000, spine_range=(200, 511))
    sizes = np.diff(w.graph_ptr)
    odd = np.arange(1, w.num_graphs, 2)
    sample = [2, int(odd[np.argmax(sizes[odd])])]
    rpg = gen.roots_per_graph(w.graph_ptr, w.child_idx)
    roff = np.concatenate([[0], np.cumsum(rpg)])
    dh = np.zeros_like(w.dh_roots)
    for g in sample:
        dh[roff[g]:roff[g + 1]] = w.dh_roots[roff[g]:roff[g + 1]]
    w.dh_roots = dh
    gp = w.graph_ptr
    rows = np.concatenate([np.arange(gp[g], gp[g + 1]) for g in sample])
    dh_nodes = np.zeros((w.num_nodes, w.hidden), np.float32)
    dh_nodes[rows] = np.random.default_rng(11).standard_normal((rows.shape[0], w.hidden)).astype(np.float32)
    g_out = C.run_device(w, dh_nodes=dh_nodes, table_grad=True)
    sub = gen.subset(w, sample)
    o = C.run_oracle(sub, dh_nodes=dh_nodes[rows].astype(np.float64), table_grad=True)
    tol = C.TOL[w.dtype]
    errs = {k: compare.rel_err(g_out[k][rows], o[k]) for k in ("h", "c", "dh", "dc")}
    mask = np.ones(w.num_nodes, bool)
    mask[rows] = False
    assert np.all(g_out["dh"][mask] == 0) and np.all(g_out["dc"][mask] == 0)
    for s, (gg, oo) in enumerate(zip(g_out["grads"], o["grads"])):
        for name in ("W_in", "W_rec", "bias"):
            if gg.get(name) is not None and oo.get(name) is not None:
                errs[f"set{s}.{name}"] = compare.rel_err(gg[name], oo[name], whole=True)
    errs["d_table"] = compare.rel_err(g_out["d_table"], o["d_table"], whole=True)
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, (bad, errs)


def test_wide_dx_two_k_slices_bf16():
    """dz . W^T of bf16 levels whose 256 x 256 tiles fill between half and all of the compute units runs as
    wide tiles with K in two slices added atomically into the children's dh.  H = 512 balanced-tree levels
    of 8-16 k rows have 128-255 such tiles.  Sampled parity as above."""
    from paper_1702_02181_amd.runner import DeviceRun
    w = gen.config5(num_graphs=256, hidden=512, vocab=2000, spine_range=(200, 511))
    dev = DeviceRun(w)
    host = dev.sched.host_groups()
    del dev
    nt = (2 * w.hidden + 255) // 256
    tiles = [((int(r) + 255) // 256) * nt for r, op in zip(host["group_rows"], host["group_op"])
             if w.ops[int(op)].arity == 2]
    assert any(128 <= t < 256 for t in tiles), tiles
    sizes = np.diff(w.graph_ptr)
    _sampled_parity(w, [0, 1 + 2 * int(np.argmax(sizes[1::2]))], table_grad=True)


def test_dx_256_row_tiles_two_k_slices_bf16():
    """bf16 dz . W^T levels with a long K (at least 64 stages of 64 bytes) whose 256-row tiles give between
    half and all of the compute units a tile run as 256 x 128 tiles with K in two slices, added atomically
    into the children's dh.  H = 512 (K = 2,560): levels of 3,841-8,191 rows; config 5's shape at 128 graphs
    has one in its balanced trees' third level (64 x 64 = 4,096 rows).  Sampled parity as above."""
    from paper_1702_02181_amd.runner import DeviceRun
    w = gen.config5(num_graphs=128, hidden=512, vocab=2000, spine_range=(200, 511))
    dev = DeviceRun(w)
    host = dev.sched.host_groups()
    del dev
    rows = [int(r) for r, op in zip(host["group_rows"], host["group_op"]) if w.ops[int(op)].arity == 2]
    nb = 2 * w.hidden // 128
    assert any(128 <= (r + 255) // 256 * nb < 256 and (r + 255) // 256 * 4 * 2 < 256 for r in rows), rows
    _sampled_parity(w, [0, 1, 64], table_grad=True)


def test_wide_weight_gradients_f32_ragged_tiles():
    """fp32 ops of at least 32 k rows whose 256 x 256 weight-gradient tiles fill the compute units take
    them.  H = 300 (padded to 320) leaves ragged tiles on every side: the leaves' 300-wide inputs (two
    weight-row tiles, the second partial) against 3 x 320 gate columns, and the children's rows 2 x 320
    (the second child's rows start inside the second weight-row tile) against 5 x 320 gate columns
    (partial last column tiles).  160 balanced trees: 40,960 leaves and 40,800 internal nodes, row counts
    that are no multiple of a stage.  Sampled parity as above, with the leaf-table gradient."""
    w = gen.config2(num_graphs=160, hidden=300)
    _sampled_parity(w, [0, 77, 159], table_grad=True)


def test_maximum_hidden_size():
    """H = 4096, the largest hidden size the library accepts (the backward stages a row's bf16 dz, G x 4096
    halves, in LDS): bf16 LSTM chains of 2 and 1 steps (64-wide inputs), forward and backward with an upstream
    gradient on every node and the leaf-table gradient, against the oracle.  (A Tree-LSTM at this size needs
    a 8192 x 20480 recurrent matrix, too slow for the fp64 oracle in test time.)"""
    from tests._helpers import make_workload
    rng = np.random.default_rng(4096)
    H = 4096
    ops = [gen.OpSpec(gen.KIND_LSTM, 1, 1, 0)]
    params = [gen.make_param_set(rng, gen.KIND_LSTM, 64, 1, H, "bf16")]
    table = gen._finish_values(0.5 * rng.standard_normal((5, 64)), "bf16")
    w = make_workload([[(0, [-1], 0), (0, [0], 1)], [(0, [-1], 2)]], ops, params, H, table, dtype="bf16", seed=2,
                      name="lstm_h4096")
    w.backward = True
    dh = rng.standard_normal((w.num_nodes, H))
    g = C.run_device(w, dh_nodes=dh, table_grad=True)
    o = C.run_oracle(w, dh_nodes=dh, table_grad=True)
    C.compare_all(w, g, o, table_grad=True)
