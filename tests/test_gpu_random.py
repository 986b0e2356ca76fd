"""Random mixed-operation DAG batches with small and odd hidden sizes, against the fp64 oracle.

Every cell kind in one batch (embedding leaves, Tree-LSTM leaves and internal nodes, LSTM steps, projections,
TreeRNN nodes), children shared by several parents or taken twice by one, zero-state children (-1), an upstream
gradient on every node as well as on the roots, and the leaf-table gradient; fp32 and bf16 parameters.  The
hidden sizes (1, 7, 33, 65, 130) leave ragged tails in every tile and pad column of the pools."""
import numpy as np
import pytest

from paper_1702_02181_amd import gen
from tests import gpu_common as C
from tests._helpers import make_workload

pytestmark = pytest.mark.gpu

V = 37  # leaf-table rows


def _random_batch(seed: int, H: int, dtype: str, n_graphs: int = 6, max_nodes: int = 40):
    rng = np.random.default_rng(seed)
    ops = [gen.OpSpec(gen.KIND_EMBED, 0, 1, 0),      # 0 leaf: table row
           gen.OpSpec(gen.KIND_TREELSTM, 0, 1, 1),   # 1 leaf: Tree-LSTM on a table row
           gen.OpSpec(gen.KIND_TREELSTM, 2, 0, 1),   # 2 Tree-LSTM node (shares set 1 with the leaf)
           gen.OpSpec(gen.KIND_LSTM, 1, 1, 2),       # 3 LSTM step: one child and a table row
           gen.OpSpec(gen.KIND_PROJ, 1, 0, 3),       # 4 projection of one child
           gen.OpSpec(gen.KIND_TREERNN, 2, 0, 4)]    # 5 TreeRNN node
    # weights U(-0.1, 0.1) and table rows N(0, 0.1^2) as in the benchmark workloads (bf16-rounded for bf16):
    # much larger weights amplify the bf16 rounding of every h row level after level past the 2e-2 bar
    params = [gen.make_param_set(rng, gen.KIND_EMBED, H, 0, H, dtype),
              gen.make_param_set(rng, gen.KIND_TREELSTM, H, 2, H, dtype),
              gen.make_param_set(rng, gen.KIND_LSTM, H, 1, H, dtype),
              gen.make_param_set(rng, gen.KIND_PROJ, 0, 1, H, dtype),
              gen.make_param_set(rng, gen.KIND_TREERNN, 0, 2, H, dtype)]
    table = gen._finish_values(0.1 * rng.standard_normal((V, H)), dtype)
    arity = {0: 0, 1: 0, 2: 2, 3: 1, 4: 1, 5: 2}
    graphs = []
    for _ in range(n_graphs):
        n = int(rng.integers(1, max_nodes + 1))
        nodes = []
        for i in range(n):
            if i < 2 or rng.random() < 0.3:
                op = int(rng.integers(0, 2))
            else:
                op = int(rng.choice([2, 3, 4, 5]))
            kids = []
            for _ in range(arity[op]):
                # an earlier node of this graph (repeats make shared children), or the zero state
                kids.append(-1 if rng.random() < 0.1 else int(rng.integers(0, i)))
            inp = int(rng.integers(0, V)) if ops[op].has_input else -1
            nodes.append((op, kids, inp))
        # node order inside a graph is arbitrary: reverse half of the graphs
        if rng.random() < 0.5:
            perm = np.arange(n)[::-1]
            pos = {int(old): new for new, old in enumerate(perm)}
            nodes = [(op, [pos[k] if k >= 0 else -1 for k in kids], inp)
                     for (op, kids, inp) in (nodes[int(o)] for o in perm)]
        graphs.append(nodes)
    w = make_workload(graphs, ops, params, H, table, dtype=dtype, seed=seed, name=f"random_{seed}")
    w.backward = True
    return w


@pytest.mark.parametrize("seed,H,dtype", [(11, 1, "bf16"), (17, 1, "f32"), (12, 7, "f32"), (13, 33, "bf16"),
                                          (14, 65, "f32"), (15, 130, "f32"), (16, 130, "bf16")])
def test_random_mixed_dag_batches(seed, H, dtype):
    w = _random_batch(seed, H, dtype)
    dh = np.random.default_rng(seed + 100).standard_normal((w.num_nodes, H))
    g = C.run_device(w, dh_nodes=dh, table_grad=True)
    o = C.run_oracle(w, dh_nodes=dh, table_grad=True)
    C.compare_all(w, g, o, table_grad=True)
