"""Recurrent dropout through the C-ABI (fold_forward_dropout / fold_backward_dropout) against the oracle,
element by element: random binary trees of Tree-LSTM cells, and a mixed LSTM / Tree-LSTM / PROJ batch, with an
inverted-dropout mask (0 or 1/(1-p)) on the candidate update, fp32 and bf16 parameters."""
import numpy as np
import pytest

from paper_1702_02181_amd import gen
from tests._helpers import dropout_mask, dropout_tree_case, make_workload, random_params, random_tree
from tests.gpu_common import compare_all, run_device, run_oracle

pytestmark = pytest.mark.gpu
TL, LS, PJ = gen.KIND_TREELSTM, gen.KIND_LSTM, gen.KIND_PROJ


# Weights and leaf tables of the bf16 cases are bf16 values (make_workload rounds them), so the oracle sees
# exactly what the GPU stores.  bf16 pools still round every h to 8 bits of mantissa, an error that grows with
# depth against the fp64 oracle: on the H = 256 random trees (normal weights of scale 0.2, K = 512 terms per
# gate) that rounding alone reaches ~0.011 (CPU emulation, tests/test_bf16_rounding_bound.py).  fp32 at
# H = 256 uses trees of at most 16 leaves to stay within 1e-5.
@pytest.mark.parametrize("dtype,H,trees,leaves", [("f32", 48, 40, 20), ("bf16", 48, 120, 8),
                                                  ("f32", 256, 300, 16), ("bf16", 256, 400, 8)])
def test_dropout_random_trees(dtype, H, trees, leaves):
    w, mask, dh_nodes = dropout_tree_case(dtype, H, trees, leaves)
    g = run_device(w, dh_nodes, table_grad=True, backward=True, u_mask=mask)
    o = run_oracle(w, dh_nodes, table_grad=True, backward=True, u_mask=mask)
    print(dtype, H, w.num_nodes, compare_all(w, g, o, check_backward=True, table_grad=True), flush=True)
    # the mask changes the result: the same batch without it differs well beyond the tolerance
    assert np.abs(run_oracle(w, backward=False)["c"] - o["c"]).max() > 1e-2


def test_dropout_sentiment_trees_full_size_bf16():
    """Recurrent dropout at the sentiment-tree training shape: the whole config-3 batch (1,024 parse-shaped
    trees, 64 k nodes, H = 300 bf16, U(-0.1, 0.1) weights, Zipf tokens over the 20,000-row table), a mask
    with p = 0.25 on every node and an upstream gradient on every node of the sampled graphs.  Its leaf and
    first internal levels are wide enough for the wide forward kernel (its masked epilogue) and the wide
    backward kernels.  Sampled parity against the oracle (batching invariance, linearity)."""
    from tests.gpu_common import sampled_parity
    w = gen.config3()
    rng = np.random.default_rng(35)
    mask = dropout_mask(rng, w.num_nodes, w.hidden, 0.25)
    dh_nodes = rng.standard_normal((w.num_nodes, w.hidden)).astype(np.float32)
    sizes = np.diff(w.graph_ptr)
    sample = [0, int(np.argmax(sizes)), 700]
    print(sampled_parity(w, sample, table_grad=True, u_mask=mask, dh_nodes=dh_nodes), flush=True)


def test_dropout_mixed_lstm_treelstm_proj():
    H, D_in = 40, 24
    rng = np.random.default_rng(5)
    pl = random_params(rng, LS, D_in, 1, H)
    pt = random_params(rng, TL, 0, 2, H)
    pp = random_params(rng, PJ, 0, 1, H)
    ops = [gen.OpSpec(LS, 1, 1, 0), gen.OpSpec(TL, 2, 0, 1), gen.OpSpec(PJ, 1, 0, 2)]
    table = rng.standard_normal((30, D_in)).astype(np.float32)
    g = [(0, [-1], 0), (0, [0], 1), (0, [1], 2), (1, [0, 1], -1), (2, [3], -1), (1, [4, 2], -1)]
    graphs = [[(op, kids, (inp + k) % 30 if inp >= 0 else -1) for (op, kids, inp) in g] for k in range(50)]
    w = make_workload(graphs, ops, [pl, pt, pp], H, table, seed=9)
    mask = dropout_mask(rng, w.num_nodes, H, 0.4)
    dh_nodes = rng.standard_normal((w.num_nodes, H)).astype(np.float32)
    gd = run_device(w, dh_nodes, table_grad=True, backward=True, u_mask=mask)
    od = run_oracle(w, dh_nodes, table_grad=True, backward=True, u_mask=mask)
    compare_all(w, gd, od, check_backward=True, table_grad=True)


def test_dropout_null_mask_is_rejected():
    import torch
    from paper_1702_02181_amd import fold as F
    from paper_1702_02181_amd.runner import DeviceRun
    rng = np.random.default_rng(1)
    p = random_params(rng, TL, 8, 2, 8)
    w = make_workload([random_tree(rng, 3, 10)], [gen.OpSpec(TL, 0, 1, 0), gen.OpSpec(TL, 2, 0, 0)], [p], 8,
                      rng.standard_normal((10, 8)).astype(np.float32))
    dev = DeviceRun(w, with_backward=True)
    with pytest.raises(F.FoldError) as e:
        F.fold_forward_dropout(dev.sched.handle, dev.packed.handle, dev.table, dev.leaf_rows, dev.h_pool,
                               dev.c_pool, dev.roots, None, dev.ws, dev.ws_bytes, dev.stream)
    assert e.value.code == F.FOLD_E_INVALID
    torch.cuda.synchronize()
