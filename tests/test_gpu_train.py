"""Parity of the training step around the path against the fp64 oracle (oracle.train, oracle.evaluate).

  * the per-node softmax cross-entropy head on seeded states written straight into a pool (every node
    labelled or not, hidden sizes 1 to 1000 with ragged tails, 2 to 32 classes up to H * C = 8000, fp32
    and bf16 pools, a batch with no label at all, a workspace full of NaN on entry): losses in node order,
    dh in pool order (pad columns zero), dW and db accumulated;
  * a whole training step: forward, head, backward with the head's dh on every node, against the oracle's
    forward, head and backward of the same seeded workload (all weight and leaf-table gradients, the
    classifier's gradients);
  * Adam against the oracle's update at steps 1 and 7 from seeded moments (vector and scalar paths, a
    ragged tail), the bf16 copy equal to the round-to-nearest-even of the fp32 result;
  * fold_pack_update: a forward after re-packing new weights in place equals, bit for bit, the forward of
    a handle packed from the new weights, also when replayed from a HIP graph recorded before the update;
  * two whole training steps (runner.TrainStep: forward, head, backward, Adam on every tensor, re-pack)
    against two steps of the oracle's chain and Adam; the gradient pass captured as a graph and replayed
    between eager steps gives the eager pass's gradients at every replay (up to fp32 atomic order);
  * argument errors of the three calls.
"""
import numpy as np
import pytest

from oracle import compare, evaluate as EV, train as OT
from paper_1702_02181_amd import fold as F
from paper_1702_02181_amd import gen
from tests import gpu_common as C
from tests._helpers import oracle_batch, oracle_params

pytestmark = pytest.mark.gpu


def _workload(H, dtype, seed):
    if dtype == "f32":
        return gen.config2(seed=seed, num_graphs=5, leaves=24, hidden=H)
    return gen.config3(seed=seed, num_graphs=24, hidden=H, vocab=300, emb_dim=H, leaf_range=(2, 40))


def _labels(rng, N, Cn, unlabelled=0.2):
    y = rng.integers(0, Cn, N).astype(np.int32)
    y[rng.random(N) < unlabelled] = -1
    return y


def _head_device(dev, h_pool, labels, W, b, scale):
    import torch
    Cn = W.shape[1]
    t = lambda a, dt=torch.float32: torch.from_numpy(np.ascontiguousarray(a)).to(dtype=dt, device="cuda")
    loss = torch.full((dev.N,), np.nan, dtype=torch.float32, device="cuda")
    dh = torch.full((dev.N, dev.ld), np.nan, dtype=torch.float32, device="cuda")
    dW = torch.zeros((dev.H, Cn), dtype=torch.float32, device="cuda")
    db = torch.zeros(Cn, dtype=torch.float32, device="cuda")
    nws = F.fold_loss_workspace_size(dev.packed.handle, Cn)
    ws = torch.full((nws // 4,), np.nan, dtype=torch.float32, device="cuda")
    F.fold_loss_softmax_ce(dev.sched.handle, dev.packed.handle, h_pool, t(labels, torch.int32), Cn,
                           t(W.astype(np.float32)), t(b.astype(np.float32)), scale, loss, dh, dW, db, ws, nws)
    torch.cuda.synchronize()
    return loss.cpu().numpy(), dh.cpu().numpy(), dW.cpu().numpy(), db.cpu().numpy()


@pytest.mark.parametrize("H,dtype,Cn,unlabelled", [(1, "f32", 2, 0.2), (33, "f32", 5, 0.2), (300, "bf16", 5, 0.2),
                                                    (130, "bf16", 3, 0.0), (250, "f32", 32, 0.3),
                                                    (1000, "f32", 8, 0.2), (65, "bf16", 10, 1.0)])
def test_loss_head_on_seeded_states(H, dtype, Cn, unlabelled):
    import torch
    from paper_1702_02181_amd.runner import DeviceRun, bf16_tensor
    w = _workload(H, dtype, seed=H + Cn)
    dev = DeviceRun(w, with_backward=False)
    rng = np.random.default_rng(1000 + H)
    N = w.num_nodes
    hp = (0.7 * rng.standard_normal((N, H))).astype(np.float32)
    if dtype == "bf16":
        hp = gen.round_bf16(hp)
    pool = np.zeros((N, dev.ld), np.float32)
    pool[:, :H] = hp
    h_pool = (bf16_tensor(pool) if dtype == "bf16" else torch.from_numpy(pool)).to("cuda")
    y = _labels(rng, N, Cn, unlabelled)
    y_dev = y.copy()
    if unlabelled not in (0.0, 1.0):  # labels outside [0, C) count as unlabelled
        off = np.nonzero(y < 0)[0]
        y_dev[off[::3]] = Cn
        y_dev[off[1::3]] = -7
    W = 0.3 * rng.standard_normal((H, Cn))
    b = 0.2 * rng.standard_normal(Cn)
    W, b = W.astype(np.float32).astype(np.float64), b.astype(np.float32).astype(np.float64)
    scale = 1.0 / max(1, int((y >= 0).sum()))
    loss, dh, dW, db = _head_device(dev, h_pool, y_dev, W, b, scale)
    node_pos = np.asarray(C.oracle_schedule(w)["node_pos"])
    o_loss, o_dh, o_dW, o_db = OT.softmax_ce(hp[node_pos].astype(np.float64), y, W, b, scale)
    assert np.all(dh[:, H:] == 0)
    errs = {"loss": compare.rel_err(loss, o_loss), "dh": compare.rel_err(dh[node_pos, :H], o_dh),
            "dW": compare.rel_err(dW, o_dW, whole=True), "db": compare.rel_err(db, o_db, whole=True)}
    if unlabelled == 1.0:
        assert np.all(loss == 0) and np.all(dh == 0) and np.all(dW == 0) and np.all(db == 0)
    assert all(v <= 1e-5 for v in errs.values()), errs


@pytest.mark.parametrize("H,dtype", [(33, "f32"), (64, "bf16")])
def test_training_step_gradients(H, dtype):
    """Forward, head on every node, backward: every gradient against the oracle's chain on the same
    seeded workload."""
    import torch
    from paper_1702_02181_amd.runner import DeviceRun
    w = _workload(H, dtype, seed=5 * H)
    table_grad = dtype == "bf16"
    Cn = 5
    rng = np.random.default_rng(77 + H)
    y = _labels(rng, w.num_nodes, Cn)
    W = (0.3 * rng.standard_normal((H, Cn))).astype(np.float32).astype(np.float64)
    b = (0.2 * rng.standard_normal(Cn)).astype(np.float32).astype(np.float64)
    scale = 1.0 / max(1, int((y >= 0).sum()))
    # device: forward, head (dh in pool order), backward from the head's dh alone
    dev = DeviceRun(w)
    dev.forward()
    _, dh_pool, dW, db = _head_device(dev, dev.h_pool, y, W, b, scale)
    dev.alloc_grads(table_grad)
    dev.set_upstream(np.zeros_like(w.dh_roots))
    dev.dh_nodes = torch.from_numpy(dh_pool).to("cuda")
    dev.backward()
    torch.cuda.synchronize()
    grads, d_table = dev.weight_grads()
    # oracle: the same chain in fp64
    ob, P = oracle_batch(w), oracle_params(w)
    f = EV.forward(ob, P, w.hidden, w.leaf_table)
    _, o_dh, o_dW, o_db = OT.softmax_ce(f["h"], y, W, b, scale)
    bw = EV.backward(ob, P, w.hidden, w.leaf_table, f, np.zeros_like(w.dh_roots, dtype=np.float64), o_dh,
                     want_table_grad=table_grad)
    tol = C.TOL[dtype]
    errs = {"dW_cls": compare.rel_err(dW, o_dW, whole=True), "db_cls": compare.rel_err(db, o_db, whole=True)}
    for s, (gg, oo) in enumerate(zip(grads, bw["grads"])):
        for name in ("W_in", "W_rec", "bias"):
            if gg.get(name) is not None and oo.get(name) is not None:
                errs[f"set{s}.{name}"] = compare.rel_err(gg[name], oo[name], whole=True)
    if table_grad:
        errs["d_table"] = compare.rel_err(d_table, bw["d_table"], whole=True)
    assert all(v <= tol for v in errs.values()), errs


@pytest.mark.parametrize("n,offset,step", [(4099, 0, 1), (4099, 0, 7), (1003, 1, 3)])
def test_adam_against_oracle(n, offset, step):
    import torch
    rng = np.random.default_rng(n + step)
    p0 = rng.standard_normal(n).astype(np.float32)
    g = (0.1 * rng.standard_normal(n)).astype(np.float32)
    m0 = np.zeros(n, np.float32) if step == 1 else (0.05 * rng.standard_normal(n)).astype(np.float32)
    v0 = np.zeros(n, np.float32) if step == 1 else (0.01 * rng.random(n)).astype(np.float32)
    dev = lambda a: torch.from_numpy(np.concatenate([np.zeros(offset, a.dtype), a])).to("cuda")
    P, G, M, V = dev(p0), dev(g), dev(m0), dev(v0)
    B = torch.zeros(n + offset, dtype=torch.int16, device="cuda")
    lr, b1, b2, eps = 1e-3, 0.9, 0.999, 1e-8
    F.fold_adam_step(n, P[offset:], B[offset:], G[offset:], M[offset:], V[offset:], lr, b1, b2, eps, step)
    torch.cuda.synchronize()
    p_o, m_o, v_o = OT.adam_step(p0, g, m0, v0, t=step, lr=lr, b1=b1, b2=b2, eps=eps)
    p_d = P.cpu().numpy()[offset:]
    np.testing.assert_allclose(p_d, p_o, rtol=1e-6, atol=1e-7)
    np.testing.assert_allclose(M.cpu().numpy()[offset:], m_o, rtol=1e-6, atol=1e-8)
    np.testing.assert_allclose(V.cpu().numpy()[offset:], v_o, rtol=1e-5, atol=1e-14)
    bits = B.cpu().numpy()[offset:].view(np.uint16)
    assert np.array_equal(bits, gen.to_bf16_bits(p_d))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_pack_update_equals_fresh_pack(dtype):
    import torch
    from paper_1702_02181_amd.runner import DeviceRun
    w = _workload(65, dtype, seed=3)
    dev = DeviceRun(w, with_backward=False)
    dev.forward()
    rng = np.random.default_rng(9)
    new_params = [gen.make_param_set(rng, p.kind, p.in_dim, p.arity, w.hidden, dtype) for p in w.params]
    w2 = gen.Workload(**{**w.__dict__, "params": new_params})
    fresh = DeviceRun(w2, with_backward=False)
    fresh.forward()
    sets = []
    for p in new_params:
        sets.append(dict(kind=p.kind, in_dim=p.in_dim, arity=p.arity,
                         W_in=None if p.W_in is None else dev._wt(p.W_in),
                         W_rec=None if p.W_rec is None else dev._wt(p.W_rec),
                         bias=None if p.kind == gen.KIND_EMBED else
                         torch.from_numpy(p.bias.astype(np.float32)).to("cuda")))
    dev.packed.update(sets)
    dev.forward()
    torch.cuda.synchronize()
    assert torch.equal(dev.h_pool, fresh.h_pool) and torch.equal(dev.c_pool, fresh.c_pool)
    o = C.run_oracle(w2, backward=False)
    assert compare.rel_err(dev.node_states()[0], o["h"]) <= C.TOL[dtype]


def test_argument_errors():
    import torch
    from paper_1702_02181_amd.runner import DeviceRun
    w = _workload(300, "bf16", seed=1)
    dev = DeviceRun(w, with_backward=False)
    z = torch.zeros(4 * dev.N * dev.ld + 64, dtype=torch.float32, device="cuda")
    y = torch.zeros(dev.N, dtype=torch.int32, device="cuda")
    nb = z.numel() * 4
    for Cn, code in ((9, F.FOLD_E_INVALID), (1, F.FOLD_E_INVALID), (32, F.FOLD_E_INVALID)):  # 300 * 32 > 8000
        with pytest.raises(F.FoldError) as e:
            F.fold_loss_softmax_ce(dev.sched.handle, dev.packed.handle, dev.h_pool, y, Cn, z, z, 1.0, z, z, z, z, z,
                                   nb)
        assert e.value.code == code
        with pytest.raises(F.FoldError) as e:
            F.fold_loss_workspace_size(dev.packed.handle, Cn)
        assert e.value.code == code
    with pytest.raises(F.FoldError) as e:
        F.fold_loss_softmax_ce(dev.sched.handle, dev.packed.handle, dev.h_pool, y, 5, z, z, float("nan"), z, z, z, z,
                               z, nb)
    assert e.value.code == F.FOLD_E_INVALID
    need = F.fold_loss_workspace_size(dev.packed.handle, 5)
    with pytest.raises(F.FoldError) as e:
        F.fold_loss_softmax_ce(dev.sched.handle, dev.packed.handle, dev.h_pool, y, 5, z, z, 1.0, z, z, z, z, z,
                               need - 4)
    assert e.value.code == F.FOLD_E_MISMATCH
    for args in ((16, z, None, z, z, z, 1e-3, 0.9, 0.999, 1e-8, 0), (16, z, None, z, z, z, 1e-3, 1.0, 0.999, 1e-8, 1),
                 (16, None, None, z, z, z, 1e-3, 0.9, 0.999, 1e-8, 1), (-1, z, None, z, z, z, 1e-3, 0.9, 0.999, 1e-8, 1)):
        with pytest.raises(F.FoldError) as e:
            F.fold_adam_step(*args)
        assert e.value.code == F.FOLD_E_INVALID
    other = _workload(64, "bf16", seed=1)
    od = DeviceRun(other, with_backward=False)
    with pytest.raises(F.FoldError) as e:
        dev.packed.update(od.set_tensors)
    assert e.value.code == F.FOLD_E_MISMATCH


def test_two_training_steps_match_oracle():
    """Every parameter tensor after two steps (weights, biases, the leaf table, the classifier), fp32."""
    from paper_1702_02181_amd.runner import TrainStep
    w = _workload(33, "f32", seed=21)
    # eps 1e-4: with the default 1e-8 an update lr g / (|g| + eps) of a gradient entry near 1e-8 would turn
    # fp32 rounding of g into changes of order lr
    H, Cn, lr, eps = w.hidden, 5, 1e-2, 1e-4
    y = _labels(np.random.default_rng(5), w.num_nodes, Cn)
    ts = TrainStep(w, y, Cn, train_table=True, seed=3, lr=lr, eps=eps)
    Wc, bc = ts.W_cls.cpu().numpy().astype(np.float64), np.zeros(Cn)
    P = oracle_params(w)
    table = w.leaf_table.astype(np.float64)
    ob = oracle_batch(w)
    keys = [(s, name) for s, pp in enumerate(P) for name in ("W_in", "W_rec", "bias") if pp.get(name) is not None]
    mom = {k: (0.0, 0.0) for k in keys + ["table", "Wc", "bc"]}
    for t in (1, 2):
        ts.step()
        f = EV.forward(ob, P, H, table)
        _, dh, dWc, dbc = OT.softmax_ce(f["h"], y, Wc, bc, ts.scale)
        bw = EV.backward(ob, P, H, table, f, np.zeros_like(w.dh_roots, dtype=np.float64), dh, want_table_grad=True)
        for s, name in keys:
            P[s][name], *mom[(s, name)] = OT.adam_step(P[s][name], bw["grads"][s][name], *mom[(s, name)], t=t, lr=lr, eps=eps)
        table, *mom["table"] = OT.adam_step(table, bw["d_table"], *mom["table"], t=t, lr=lr, eps=eps)
        Wc, *mom["Wc"] = OT.adam_step(Wc, dWc, *mom["Wc"], t=t, lr=lr, eps=eps)
        bc, *mom["bc"] = OT.adam_step(bc, dbc, *mom["bc"], t=t, lr=lr, eps=eps)
    want = [P[s][name] for s, name in keys] + [table, Wc, bc]
    got = [m.cpu().numpy() for m, _, _ in ts.tensors]
    assert len(got) == len(want)
    for k, (g, o) in enumerate(zip(got, want)):
        g = g.reshape(o.shape[0], -1)[:, :o.reshape(o.shape[0], -1).shape[1]].reshape(o.shape)  # table pad columns
        # an update moves a value by at most about 2 lr over two steps; fp32 gradients shift it by far less
        np.testing.assert_allclose(g, o, rtol=0, atol=lr * 1e-3, err_msg=f"tensor {k}")


def test_pack_update_seen_by_a_recorded_graph():
    """A step graph recorded before fold_pack_update reads the new weights on its next replay."""
    import torch
    from paper_1702_02181_amd.runner import DeviceRun
    w = _workload(64, "bf16", seed=4)
    dev = DeviceRun(w, with_backward=False)
    graph = dev.make_graph(backward=False)
    graph.launch()
    torch.cuda.synchronize()
    before = dev.h_pool.clone()
    rng = np.random.default_rng(12)
    new_params = [gen.make_param_set(rng, p.kind, p.in_dim, p.arity, w.hidden, "bf16") for p in w.params]
    fresh = DeviceRun(gen.Workload(**{**w.__dict__, "params": new_params}), with_backward=False)
    fresh.forward()
    sets = [dict(kind=p.kind, in_dim=p.in_dim, arity=p.arity,
                 W_in=None if p.W_in is None else dev._wt(p.W_in), W_rec=None if p.W_rec is None else dev._wt(p.W_rec),
                 bias=None if p.kind == gen.KIND_EMBED else torch.from_numpy(p.bias.astype(np.float32)).to("cuda"))
            for p in new_params]
    dev.packed.update(sets)
    for _ in range(2):
        graph.launch()
        torch.cuda.synchronize()
        assert torch.equal(dev.h_pool, fresh.h_pool) and torch.equal(dev.c_pool, fresh.c_pool)
    assert not torch.equal(before, dev.h_pool)


def test_captured_gradient_pass_replays_match_eager():
    """TrainStep's gradient pass (zero, forward, head, backward) recorded once as a graph: replayed several
    times, with eager Adam steps and re-packs between the replays, every replay's gradients equal those of the
    eager pass on the same weights up to the order of fp32 atomic additions (K-split slices of dz . W^T add into
    the children's dh in any order, so two eager passes differ in the last bits too): 1e-6 relative."""
    import torch
    from paper_1702_02181_amd.runner import TrainStep
    w = _workload(64, "bf16", seed=31)
    y = _labels(np.random.default_rng(6), w.num_nodes, 5)
    ts = TrainStep(w, y, 5, train_table=True, seed=2)
    ts.capture_gradients()
    grads = lambda: [g.clone() for _, _, g in ts.tensors] + [ts.node_loss.clone(), ts.dh_nodes.clone()]
    for it in range(3):
        ts.gradients()
        torch.cuda.synchronize()
        eager = grads()
        ts.graph.replay()
        torch.cuda.synchronize()
        replay = grads()
        for k, (a, b) in enumerate(zip(eager, replay)):
            err = compare.rel_err(b.cpu().numpy().reshape(a.shape[0], -1), a.cpu().numpy().reshape(a.shape[0], -1),
                                  whole=True)
            assert err <= 1e-6, (it, k, err)
        ts.step(graph=True)  # the weights move between the checks
        torch.cuda.synchronize()


@pytest.mark.parametrize("H,p,seed,step", [(1, 0.5, 0, 1), (7, 0.25, 12345, 2), (300, 0.25, (9 << 40) | 77, 3),
                                           (64, 0.0, 5, 1), (1024, 0.9, 3, (1 << 33) + 5), (130, 0.5, 1, 0)])
def test_dropout_mask_matches_oracle_bit_for_bit(H, p, seed, step):
    """fold_dropout_mask (Philox4x32-10 on the GPU) against the oracle's own Philox draw, every element: the
    counter layout (node, 4-unit block, step), the key (seed), the integer threshold and the scale, pool
    order with zero pad columns; node ids shuffled within graphs so that pool order differs from node order."""
    import torch
    from oracle import philox as PX
    from paper_1702_02181_amd.runner import DeviceRun
    w = gen.shuffle_within_graphs(gen.config3(seed=4, num_graphs=40, hidden=H, vocab=50, emb_dim=8), 3)
    dev = DeviceRun(w, with_backward=False)
    mask = torch.full((dev.N, dev.ld), float("nan"), dtype=torch.float32, device="cuda")
    F.fold_dropout_mask(dev.sched.handle, H, p, seed, step, mask)
    got = mask.cpu().numpy()
    assert np.all(got[:, H:] == 0)
    want = PX.dropout_mask(w.num_nodes, H, p, seed, step)
    node_pos = dev.sched_arrays()["node_pos"]
    assert np.array_equal(got[node_pos, :H], want)


def test_dropout_mask_argument_errors():
    import torch
    from paper_1702_02181_amd.runner import DeviceRun
    w = gen.config3(seed=4, num_graphs=3, hidden=8, vocab=20, emb_dim=8)
    dev = DeviceRun(w, with_backward=False)
    mask = torch.zeros((dev.N, dev.ld), dtype=torch.float32, device="cuda")
    for args in ((8, 1.0), (8, -0.1), (8, float("nan")), (0, 0.5), (4097, 0.5)):
        with pytest.raises(F.FoldError) as e:
            F.fold_dropout_mask(dev.sched.handle, args[0], args[1], 1, 1, mask)
        assert e.value.code == F.FOLD_E_INVALID
    with pytest.raises(F.FoldError) as e:
        F.fold_dropout_mask(dev.sched.handle, 8, 0.5, 1, 1, None)
    assert e.value.code == F.FOLD_E_INVALID
    torch.cuda.synchronize()


@pytest.mark.parametrize("graph", [False, True])
def test_training_steps_with_recurrent_dropout_match_oracle(graph):
    """Three TrainStep steps with recurrent dropout (p = 0.3, a fresh GPU-drawn mask every step; eagerly, and
    with the gradient pass replayed from a graph recorded once while the mask is redrawn outside it), fp32,
    against three oracle steps whose masks the oracle draws itself (same generator, counter and key): every
    parameter tensor after Adam."""
    dtype = "f32"
    from oracle import philox as PX
    from paper_1702_02181_amd.runner import TrainStep
    w = _workload(33, dtype, seed=23)
    H, Cn, lr, eps, p, dseed = w.hidden, 5, 1e-2, 1e-4, 0.3, 991
    y = _labels(np.random.default_rng(6), w.num_nodes, Cn)
    ts = TrainStep(w, y, Cn, train_table=True, seed=3, lr=lr, eps=eps, dropout=p, dropout_seed=dseed)
    if graph:
        ts.capture_gradients()
    Wc, bc = ts.W_cls.cpu().numpy().astype(np.float64), np.zeros(Cn)
    P = oracle_params(w)
    table = w.leaf_table.astype(np.float64)
    ob = oracle_batch(w)
    keys = [(s, name) for s, pp in enumerate(P) for name in ("W_in", "W_rec", "bias") if pp.get(name) is not None]
    mom = {k: (0.0, 0.0) for k in keys + ["table", "Wc", "bc"]}
    for t in (1, 2, 3):
        ts.step(graph=graph)
        m = PX.dropout_mask(w.num_nodes, H, p, dseed, t)
        f = EV.forward(ob, P, H, table, m)
        _, dh, dWc, dbc = OT.softmax_ce(f["h"], y, Wc, bc, ts.scale)
        bw = EV.backward(ob, P, H, table, f, np.zeros_like(w.dh_roots, dtype=np.float64), dh, want_table_grad=True)
        for s, name in keys:
            P[s][name], *mom[(s, name)] = OT.adam_step(P[s][name], bw["grads"][s][name], *mom[(s, name)], t=t, lr=lr,
                                                      eps=eps)
        table, *mom["table"] = OT.adam_step(table, bw["d_table"], *mom["table"], t=t, lr=lr, eps=eps)
        Wc, *mom["Wc"] = OT.adam_step(Wc, dWc, *mom["Wc"], t=t, lr=lr, eps=eps)
        bc, *mom["bc"] = OT.adam_step(bc, dbc, *mom["bc"], t=t, lr=lr, eps=eps)
    want = [P[s][name] for s, name in keys] + [table, Wc, bc]
    got = [mm.cpu().numpy() for mm, _, _ in ts.tensors]
    assert len(got) == len(want)
    # an update moves a value by at most about 2 lr a step; fp32 gradients shift it by far less
    atol = lr * 1e-3
    for k, (g, o) in enumerate(zip(got, want)):
        g = g.reshape(o.shape[0], -1)[:, :o.reshape(o.shape[0], -1).shape[1]].reshape(o.shape)
        np.testing.assert_allclose(g, o, rtol=0, atol=atol, err_msg=f"tensor {k}")
