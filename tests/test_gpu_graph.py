"""The whole step recorded as one HIP graph (fold_graph_create / fold_graph_launch), through the C ABI.

Each test replays the recorded step several times, with eager work and synchronisations in between
(the pools, gradients and outputs are overwritten with garbage before every replay), and checks every
replay against the eager calls and against the fp64 oracle."""
import numpy as np
import pytest

from oracle import compare
from paper_1702_02181_amd import fold as F
from paper_1702_02181_amd import gen
from tests import gpu_common as C

pytestmark = pytest.mark.gpu


def _snapshot(dev, dh_out, dc_out):
    import torch
    torch.cuda.synchronize()
    h, c = dev.node_states()
    out = {"h": h, "c": c, "roots": dev.roots.float().cpu().numpy()[:dev.R, :dev.H].astype(np.float64)}
    if dh_out is not None:
        node_pos = dev.sched_arrays()["node_pos"]
        out["dh"] = dh_out.cpu().numpy()[:, :dev.H][node_pos].astype(np.float64)
        out["dc"] = dc_out.cpu().numpy()[:, :dev.H][node_pos].astype(np.float64)
        out["grads"], out["d_table"] = dev.weight_grads()
    return out


def _scribble(dev, dh_out, dc_out):
    """Overwrite everything the step writes with finite garbage (eager torch work between replays)."""
    for t in (dev.h_pool, dev.c_pool, dev.roots):
        t.fill_(7.0)
    if dh_out is not None:
        dh_out.fill_(-3.0)
        dc_out.fill_(5.0)
        for s in dev.grad_tensors:
            for x in s:
                if x is not None:
                    x.fill_(11.0)
        if dev.d_table is not None:
            dev.d_table.fill_(13.0)


# Between two runs only the order of atomic scatter-adds differs (children with several parents, the
# leaf-table gradient).  In fp32 that moves results by a few ulps; with bf16 parameters dz is rounded to
# bf16, and an ulp-sized change can flip that rounding, one bf16 ulp (2^-8 relative) on one element.
RUN_TO_RUN = {"f32": 1e-6, "bf16": 1e-3}


@pytest.mark.parametrize("case", ["cfg2_fp32", "cfg4_mixed_bf16", "cfg5_dag_bf16", "cfg1_forward_only",
                                  "attention_bf16"])
def test_graph_replays_match_eager_and_oracle(case):
    import torch
    table_grad = True
    dh_nodes = None
    if case == "cfg2_fp32":
        w = gen.config2(num_graphs=3, leaves=40)
        dh_nodes = np.random.default_rng(3).standard_normal((w.num_nodes, w.hidden))
    elif case == "cfg4_mixed_bf16":
        w = gen.config4(num_graphs=8, max_chain=30, hidden=128, in_dim=64)
    elif case == "cfg5_dag_bf16":
        w = gen.config5(num_graphs=4, hidden=128, vocab=200, spine_range=(20, 60), balanced_leaves=32)
    elif case == "attention_bf16":
        w = gen.attention(seed=5, num_graphs=16, length=(1, 30), hidden=64, dtype="bf16")
    else:
        w = gen.config1()
        table_grad = False
    from paper_1702_02181_amd.runner import DeviceRun
    backward = w.backward
    dev = DeviceRun(w, with_backward=backward)
    dh_out = dc_out = None
    if backward:
        dev.alloc_grads(table_grad)
        dev.set_upstream(w.dh_roots, dh_nodes)
        dh_out = torch.zeros((dev.N, dev.ld), dtype=torch.float32, device="cuda")
        dc_out = torch.zeros_like(dh_out)
    # eager reference
    if backward:
        dev.zero_grads()
    dev.forward()
    if backward:
        dev.backward(dh_out, dc_out)
    eager = _snapshot(dev, dh_out, dc_out)

    o = C.run_oracle(w, dh_nodes=dh_nodes, table_grad=table_grad)
    graph = dev.make_graph(backward=backward, zero_grads=True, dh_out=dh_out, dc_out=dc_out)
    assert graph.num_nodes > 0
    for replay in range(3):
        _scribble(dev, dh_out, dc_out)
        torch.cuda.synchronize()
        graph.launch()
        got = _snapshot(dev, dh_out, dc_out)
        # the forward has no atomics: bit for bit the eager states
        for k in ("h", "c", "roots"):
            assert np.array_equal(got[k], eager[k]), (replay, k)
        if backward:
            # node gradients scatter-add with atomics where a child has several parents, and the
            # leaf-table gradient always does: equal up to the order of those additions
            tol = RUN_TO_RUN[w.dtype]
            for k in ("dh", "dc"):
                assert compare.rel_err(got[k], eager[k]) <= tol, (replay, k)
            for s, (gg, ee) in enumerate(zip(got["grads"], eager["grads"])):
                for name in ("W_in", "W_rec", "bias"):
                    if gg.get(name) is not None:
                        assert compare.rel_err(gg[name], ee[name], whole=True) <= tol, (replay, s, name)
            if table_grad:
                assert compare.rel_err(got["d_table"], eager["d_table"], whole=True) <= tol
        if case == "attention_bf16":
            # the scorer's bias gradient is exactly 0 against the oracle (softmax ignores a common shift of the
            # scores; compared against its terms in test_gpu_attention) and each attention node's dc is one
            # cancelling dot product (compared as one tensor there too)
            got["grads"][2]["bias"] = None
            C.compare_all(w, got, o, table_grad=table_grad, whole_keys=("dc",))
        else:
            C.compare_all(w, got, o, table_grad=table_grad)


def test_graph_accumulates_without_zero_flag():
    """Without FOLD_STEP_ZERO_GRADS two replays leave twice the gradients of one step."""
    import torch
    from paper_1702_02181_amd.runner import DeviceRun
    w = gen.config2(num_graphs=2, leaves=16)
    dev = DeviceRun(w)
    dev.alloc_grads(False)
    dev.set_upstream(w.dh_roots)
    g1 = dev.make_graph(zero_grads=True)
    g1.launch()
    one, _ = dev.weight_grads()
    g2 = dev.make_graph(zero_grads=False)
    g2.launch()
    two, _ = dev.weight_grads()
    torch.cuda.synchronize()
    for a, b in zip(one, two):
        for name in ("W_in", "W_rec", "bias"):
            if a.get(name) is not None:
                assert compare.rel_err(b[name], 2 * a[name], whole=True) <= 1e-6


def test_graph_argument_errors():
    import torch
    from paper_1702_02181_amd.runner import DeviceRun
    w = gen.config2(num_graphs=1, leaves=8)
    dev = DeviceRun(w)
    dev.alloc_grads(False)
    dev.set_upstream(w.dh_roots)
    b = F.fold_step_buffers()
    b.leaf_table, b.leaf_rows = F._ptr(dev.table), dev.leaf_rows
    b.h_pool, b.c_pool = F._ptr(dev.h_pool), F._ptr(dev.c_pool)
    b.ws, b.ws_bytes = F._ptr(dev.ws), dev.ws_bytes
    sh, ph = dev.sched.handle, dev.packed.handle
    with pytest.raises(F.FoldError) as e:
        F.fold_graph_create(sh, ph, b, 8)
    assert e.value.code == -1
    with pytest.raises(F.FoldError) as e:  # zeroing needs the backward
        F.fold_graph_create(sh, ph, b, F.FOLD_STEP_ZERO_GRADS)
    assert e.value.code == -1
    small = F.fold_step_buffers.from_buffer_copy(b)
    small.ws_bytes = 16
    with pytest.raises(F.FoldError) as e:
        F.fold_graph_create(sh, ph, small, F.FOLD_STEP_BACKWARD)
    assert e.value.code == -9
    nopool = F.fold_step_buffers.from_buffer_copy(b)
    nopool.h_pool = None
    with pytest.raises(F.FoldError) as e:
        F.fold_graph_create(sh, ph, nopool, 0)
    assert e.value.code == -1
    # a forward-only graph with a forward-sized workspace is fine
    fw = F.fold_step_buffers.from_buffer_copy(b)
    fw.ws_bytes = dev.fwd_bytes
    h = F.fold_graph_create(sh, ph, fw, 0)
    F.fold_graph_launch(h)
    torch.cuda.synchronize()
    F.fold_graph_free(h)


def test_profile_launch_records_carry_group_and_op():
    """Per-launch timing records name the (depth, op) group of every forward and backward cell launch in
    schedule order (backward level by level from the top), a level launch its span of groups, and the op of
    every weight-gradient launch."""
    import torch
    from paper_1702_02181_amd.runner import DeviceRun
    w = gen.config4(num_graphs=6)
    dev = DeviceRun(w)
    dev.alloc_grads(False)
    dev.set_upstream(w.dh_roots)
    host = dev.sched.host_groups()
    ng = len(host["group_op"])
    dev.forward()
    torch.cuda.synchronize()
    F.fold_profile_read_launches()  # drop anything recorded before
    F.fold_profile_enable(True)
    try:
        dev.zero_grads()
        dev.forward()
        dev.backward()
        torch.cuda.synchronize()
        recs = F.fold_profile_read_launches()
    finally:
        F.fold_profile_enable(False)
    assert F.fold_profile_read_launches() == []

    def groups_of(g, o):
        # a level launch (several groups of one level) is tagged with its first group and op = -1 - span
        return [g] if o >= -1 else list(range(g, g - 1 - o))

    def expanded(prefix):
        out = []
        for n, g, o, _ in recs:
            if n.startswith(prefix):
                assert o >= 0 or o <= -3, (n, g, o)  # an op id, or a level launch of two or more groups
                if o >= 0:
                    assert o == int(host["group_op"][g])
                out += groups_of(g, o)
        return out
    levels = host["group_level"]
    assert expanded("cell_fwd.") == list(range(ng))
    # backward: levels from the top, the groups of a level in order
    want = [g for lv in sorted(set(levels.tolist()), reverse=True) for g in range(ng) if levels[g] == lv]
    assert expanded("cell_bwd.") == want
    assert any(n.endswith(".level.bf16") or n == "cell_bwd.level" for n, _, _, _ in recs)  # config 4 merges
    for n, g, o, ms in recs:
        assert ms >= 0.0
        if n.startswith("bwd_dx."):
            assert 0 <= g < ng and (o == int(host["group_op"][g]) or (o <= -2 and g - 1 - o <= ng))
        if n.startswith("wgrad"):
            assert g == -1 and 0 <= o < len(w.ops)
        if n in ("bwd_init", "roots", "zero_grads"):
            assert g == -1 and o == -1
    assert {o for n, g, o, _ in recs if n.startswith("wgrad.")} == {int(x) for x in set(host["group_op"])}
