"""Feed-forward attention (Section 3.4, Appendix A) on the GPU, against the fp64 oracle.

The attention operations (scorer, pairwise merge of (m, s, acc) aggregates, output acc / s) run as dynamic-
batching operations of their own beside PROJ layers: the schedule bit for bit, the states (h = acc,
c = [m, s, 0..]), every node's dh / dc, the scorer's and the projections' weight gradients and the leaf-table
gradient within the tolerance of the parameters' type.  Cases: the generated attention model at small and full
size (sequences of 50-100 items, H = 256, bf16), merge trees of every shape, sequences of one item, empty sets
(zero-state children of merges, outputs and scorers), items shared by several merges or taken twice by one
(atomic adds into their gradients), upstream gradients on every node (the fixed-maximum reading at
intermediate merges) and ragged hidden sizes."""
import numpy as np
import pytest

from paper_1702_02181_amd import gen
from tests import gpu_common as C
from tests._helpers import make_workload

pytestmark = pytest.mark.gpu

EMB, PJ = gen.KIND_EMBED, gen.KIND_PROJ
SC, SM, OUT = gen.KIND_ATTN_SCORE, gen.KIND_ATTN_SUM, gen.KIND_ATTN_OUT


# The gradient of an attention node's c is one number, ds (column 1): at an output's child it is
# -(dh . acc) / s^2, a dot product that can cancel far below its terms, and the merges and scorers pass it on.
# Its error relative to its own value is not bounded by the arithmetic (an fp64 evaluation of the oracle with
# each node's h rounded to bf16, as the pools store it, moves such a row by 140 %), so dc is compared as one
# tensor, relative to its largest entry, like the weight gradients.
WHOLE = ("dc",)


def _check(w, dh_nodes=None, table_grad=True, tol=None):
    """compare_all (dc as one tensor), except the scorer's bias gradient: a sum of the rows' de whose exact
    value is 0 when only the roots carry a gradient (softmax does not change when every score shifts by one
    amount), so it is compared as |GPU - oracle| / sum_r |de_r|, the scale of a summation's rounding error."""
    g = C.run_device(w, dh_nodes=dh_nodes, table_grad=table_grad)
    C.assert_schedule_equal(g["sched"], C.oracle_schedule(w))
    o = C.run_oracle(w, dh_nodes=dh_nodes, table_grad=table_grad)
    tol = C.TOL[w.dtype] if tol is None else tol
    db = {}
    for s, p in enumerate(w.params):
        if p.kind == SC:
            db[s] = (float(g["grads"][s]["bias"][0]), float(o["grads"][s]["bias"][0]))
            g["grads"][s]["bias"] = None
    errs = C.compare_all(w, g, o, tol=tol, table_grad=table_grad, whole_keys=WHOLE)
    for s, (gd, od) in db.items():
        scale = C.scorer_terms(w, o, s)
        if dh_nodes is None:
            assert abs(od) <= 1e-12 * max(scale, 1e-300), (od, scale)  # shift invariance of the softmax
        errs[f"set{s}.bias"] = abs(gd - od) / max(scale, 1e-300)
        assert errs[f"set{s}.bias"] <= tol, (s, gd, od, scale)
    return errs


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("H", [256, 37])
def test_generated_attention_model(dtype, H):
    w = gen.attention(seed=3, num_graphs=24, length=(1, 40), hidden=H, dtype=dtype)
    errs = _check(w)
    assert errs["set2.W_rec"] >= 0  # the scorer's gradient is compared


def test_generated_attention_model_with_node_gradients():
    w = gen.attention(seed=4, num_graphs=16, length=(2, 30), hidden=130, dtype="f32")
    dh_nodes = np.random.default_rng(4).standard_normal((w.num_nodes, w.hidden)).astype(np.float32)
    _check(w, dh_nodes=dh_nodes)


def _hand_case(H, dtype, seed):
    """Merge trees of every shape with empty sets and shared items, without projections:
    op 0 lookup, 1 scorer, 2 merge, 3 output."""
    rng = np.random.default_rng(seed)
    V = 50
    table = rng.standard_normal((V, H)).astype(np.float32)
    ops = [gen.OpSpec(EMB, 0, 1, 0), gen.OpSpec(SC, 1, 0, 1), gen.OpSpec(SM, 2, 0, 2), gen.OpSpec(OUT, 1, 0, 3)]
    params = [gen.ParamSet(EMB, H, 0, None, None, np.zeros(0, np.float32)),
              gen.ParamSet(SC, 0, 1, None, rng.uniform(-0.5, 0.5, (H, 1)).astype(np.float32),
                           np.asarray([0.3], np.float32)),
              gen.ParamSet(SM, 0, 2, None, None, np.zeros(0, np.float32)),
              gen.ParamSet(OUT, 0, 1, None, None, np.zeros(0, np.float32))]
    graphs = []
    for T, shape in ((1, "balanced"), (2, "chain"), (7, "random"), (33, "balanced"), (20, "chain"), (16, "random")):
        nodes, items = [], []
        for _ in range(T):
            nodes.append((0, [], int(rng.integers(V))))
            nodes.append((1, [len(nodes) - 1], -1))
            items.append(len(nodes) - 1)
        cur = items

        def build(seq):
            if len(seq) == 1:
                return seq[0]
            m = len(seq) // 2 if shape == "balanced" else (len(seq) - 1 if shape == "chain" else
                                                           int(rng.integers(1, len(seq))))
            a, b = build(seq[:m]), build(seq[m:])
            nodes.append((2, [a, b], -1))
            return len(nodes) - 1
        top = build(cur)
        nodes.append((3, [top], -1))
        graphs.append(nodes)
    # empty sets: a merge with one or two zero-state children, an output over the zero state, a scorer of
    # the zero state, an output over the merge of two empty sets
    g = [(0, [], 3), (1, [0], -1), (2, [1, -1], -1), (2, [-1, 2], -1), (3, [3], -1), (3, [-1], -1),
         (1, [-1], -1), (2, [-1, -1], -1), (3, [7], -1), (2, [6, 2], -1), (3, [9], -1)]
    graphs.append(g)
    # shared items: an item in two merges, an item taken twice by one merge, a merge shared by two outputs
    g = [(0, [], 5), (1, [0], -1), (0, [], 6), (1, [2], -1), (2, [1, 3], -1), (2, [1, 1], -1),
         (2, [4, 5], -1), (3, [6], -1), (3, [6], -1), (3, [5], -1)]
    graphs.append(g)
    w = make_workload(graphs, ops, params, H, table, dtype=dtype, seed=seed, name=f"attn_hand_{seed}")
    w.backward = True
    return w


@pytest.mark.parametrize("dtype,H", [("f32", 64), ("f32", 2), ("f32", 97), ("bf16", 64), ("bf16", 300)])
def test_merge_shapes_empty_sets_and_shared_items(dtype, H):
    w = _hand_case(H, dtype, seed=H)
    dh_nodes = np.random.default_rng(H).standard_normal((w.num_nodes, H)).astype(np.float32)
    _check(w)
    _check(w, dh_nodes=dh_nodes)


def test_full_size_attention_workload_sampled():
    """The benchmark's attention workload (1024 sequences of 50-100 items, H = 256, bf16): the whole schedule bit
    for bit, and the states and gradients of sampled sequences inside the full batch (see sampled_parity)."""
    w = gen.attention()
    C.assert_schedule_equal(C.run_device(w, backward=False)["sched"], C.oracle_schedule(w))
    sample = [0, 1, 511, 1023]
    errs, g, o, rows = C.sampled_parity(w, sample, table_grad=True, exclude=("set2.bias",), raw=True,
                                        whole_keys=WHOLE)
    sub = gen.subset(w, sample)
    scale = C.scorer_terms(sub, o, 2)
    od, gd = float(o["grads"][2]["bias"][0]), float(g["grads"][2]["bias"][0])
    assert abs(od) <= 1e-12 * scale and abs(gd - od) <= C.TOL[w.dtype] * scale, (gd, od, scale)


def test_widest_hidden_size():
    """H = 4096 (the largest hidden size): every lane walks sixteen 256-column steps of a row.  fp32: in bf16 this
    batch's h is 4.1e-2 from the fp64 oracle, all of it from storing h in bf16 (an fp64 evaluation of the oracle
    with each node's h rounded to bf16 gives the same 4.1e-2 on a projection row whose 4,096 inputs carry that
    rounding).  The fp32 bar of 1e-5 is set for K <= 512 (configurations 1 and 2); the rounding of a sum of K
    fp32 products grows as sqrt(K), so for the projections' K = 4096 the bar is 1e-5 * sqrt(4096 / 512) = 2.8e-5."""
    w = gen.attention(seed=8, num_graphs=3, length=(1, 12), hidden=4096, dtype="f32")
    _check(w, tol=1e-5 * np.sqrt(4096 / 512))


def test_allocation_free_forward_with_attention():
    """fold_forward_noalloc runs the attention operations as fold_forward does: the same states bit for bit
    (the forward has no atomic additions), pad columns zero."""
    import torch
    from paper_1702_02181_amd import fold as F
    from paper_1702_02181_amd.runner import DeviceRun
    w = gen.attention(seed=9, num_graphs=20, length=(1, 40), hidden=96, dtype="bf16")
    dev = DeviceRun(w, with_backward=False)
    dev.forward()
    h2 = torch.full_like(dev.h_pool, float("nan"))
    c2 = torch.full_like(dev.c_pool, float("nan"))
    r2 = torch.full_like(dev.roots, float("nan"))
    F.fold_forward_noalloc(dev.sched.handle, dev.packed.handle, dev.table, dev.leaf_rows, h2, c2, r2)
    torch.cuda.synchronize()
    N, R = dev.N, dev.R
    assert torch.equal(h2[:N], dev.h_pool[:N]) and torch.equal(c2[:N], dev.c_pool[:N])
    assert torch.equal(r2[:R], dev.roots[:R])
    assert torch.all(h2[:N, dev.H:].float() == 0) and torch.all(c2[:N, dev.H:] == 0)
