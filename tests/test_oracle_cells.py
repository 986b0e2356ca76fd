"""Pins of the oracle's forward and backward (CPU only).

  * hand-expanded scalar formulas (H = 1, Python ``math``) on 1- to 3-node
    graphs of every operation, including a DAG whose root reads one leaf twice;
  * special cases that reduce to library routines: a Tree-LSTM chain whose
    other child is the zero state is exactly ``torch.nn.LSTMCell`` with zero
    input (on either side), a one-sided TreeRNN chain or a PROJ chain is
    ``torch.nn.RNNCell``, the LSTM op is ``torch.nn.LSTMCell`` -- forward and,
    through autograd, backward;
  * closed forms at depth with zero weights (balanced trees, caterpillars to
    depth 512);
  * central finite differences of every gradient on small trees and DAGs;
  * invariants: dead leaf forget-gate columns, linearity in the upstream
    gradient, fan-out sums, batching and graph-order invariance.
"""
import math

import numpy as np
import pytest
import torch

from oracle import evaluate as EV
from paper_1702_02181_amd import gen
from tests._helpers import make_workload, oracle_batch, oracle_params, random_params

EMB, RNN, TL, LS, PJ = gen.KIND_EMBED, gen.KIND_TREERNN, gen.KIND_TREELSTM, gen.KIND_LSTM, gen.KIND_PROJ


def run(w, dh_nodes=None, table_grad=True):
    b, P = oracle_batch(w), oracle_params(w)
    f = EV.forward(b, P, w.hidden, w.leaf_table)
    bw = EV.backward(b, P, w.hidden, w.leaf_table, f, w.dh_roots.astype(np.float64), dh_nodes,
                     want_table_grad=table_grad)
    return f, bw


def sig(x):
    return 1.0 / (1.0 + math.exp(-x))


# ---------------------------------------------------------------- hand-expanded, H = 1

def scalar_treelstm_params(rng):
    return random_params(rng, TL, 1, 2, 1)


def test_scalar_treelstm_leaf_and_three_node_tree():
    rng = np.random.default_rng(0)
    p = scalar_treelstm_params(rng)
    ops = [gen.OpSpec(TL, 0, 1, 0), gen.OpSpec(TL, 2, 0, 0)]
    table = np.array([[0.7], [-1.3]], np.float32)
    w = make_workload([[(0, [], 0), (0, [], 1), (1, [0, 1], -1)]], ops, [p], 1, table)
    f, _ = run(w)
    Wx, U, b = p.W_in.astype(float)[0], p.W_rec.astype(float), p.bias.astype(float)

    def leaf(x):
        z = [x * Wx[g] + b[g] for g in range(5)]
        i, o, u = sig(z[0]), sig(z[3]), math.tanh(z[4])
        c = i * u
        return o * math.tanh(c), c

    hl, cl = leaf(float(table[0, 0]))
    hr, cr = leaf(float(table[1, 0]))
    z = [hl * U[0, g] + hr * U[1, g] + b[g] for g in range(5)]
    i, fl, fr, o, u = sig(z[0]), sig(z[1]), sig(z[2]), sig(z[3]), math.tanh(z[4])
    c = i * u + fl * cl + fr * cr
    h = o * math.tanh(c)
    assert abs(f["h"][0, 0] - hl) < 1e-15 and abs(f["c"][1, 0] - cr) < 1e-15
    assert abs(f["c"][2, 0] - c) < 1e-15 and abs(f["h"][2, 0] - h) < 1e-15


def test_scalar_dag_root_reads_the_same_leaf_twice():
    rng = np.random.default_rng(1)
    p = scalar_treelstm_params(rng)
    ops = [gen.OpSpec(TL, 0, 1, 0), gen.OpSpec(TL, 2, 0, 0)]
    table = np.array([[0.4]], np.float32)
    g = np.array([[0.9]], np.float32)
    w = make_workload([[(0, [], 0), (1, [0, 0], -1)]], ops, [p], 1, table, dh_roots=g)
    f, bw = run(w)
    Wx, U, b = p.W_in.astype(float)[0], p.W_rec.astype(float), p.bias.astype(float)
    z = [float(table[0, 0]) * Wx[k] + b[k] for k in range(5)]
    i0, o0, u0 = sig(z[0]), sig(z[3]), math.tanh(z[4])
    c0 = i0 * u0
    h0 = o0 * math.tanh(c0)
    z = [h0 * (U[0, k] + U[1, k]) + b[k] for k in range(5)]
    i, fl, fr, o, u = sig(z[0]), sig(z[1]), sig(z[2]), sig(z[3]), math.tanh(z[4])
    c = i * u + (fl + fr) * c0
    h = o * math.tanh(c)
    assert abs(f["h"][1, 0] - h) < 1e-15
    # the shared leaf receives the sum of both slots' contributions
    gr = float(g[0, 0])
    tc = math.tanh(c)
    dct = gr * o * (1 - tc * tc)
    dz = [dct * u * i * (1 - i), dct * c0 * fl * (1 - fl), dct * c0 * fr * (1 - fr),
          gr * tc * o * (1 - o), dct * i * (1 - u * u)]
    dh_leaf = sum(dz[k] * (U[0, k] + U[1, k]) for k in range(5))
    dc_leaf = dct * (fl + fr)
    assert abs(bw["dh"][0, 0] - dh_leaf) < 1e-14
    assert abs(bw["dc"][0, 0] - dc_leaf) < 1e-14


def test_scalar_lstm_chain_proj_treernn_embed():
    rng = np.random.default_rng(2)
    pl = random_params(rng, LS, 1, 1, 1)
    pp = random_params(rng, PJ, 0, 1, 1)
    pr = random_params(rng, RNN, 0, 2, 1)
    pe = gen.ParamSet(EMB, 1, 0, None, None, np.zeros(0, np.float32))
    ops = [gen.OpSpec(LS, 1, 1, 0), gen.OpSpec(PJ, 1, 0, 1), gen.OpSpec(RNN, 2, 0, 2),
           gen.OpSpec(EMB, 0, 1, 3)]
    table = np.array([[0.5], [-0.8], [1.1]], np.float32)
    # graph: x0 -> lstm a ; x1 -> lstm b(a) ; proj(b) ; embed(x2) ; rnn(proj, embed)
    w = make_workload([[(0, [-1], 0), (0, [0], 1), (1, [1], -1), (3, [], 2), (2, [2, 3], -1)]],
                      ops, [pl, pp, pr, pe], 1, table)
    f, _ = run(w)
    Wx, U, b = pl.W_in.astype(float)[0], pl.W_rec.astype(float)[0], pl.bias.astype(float)

    def lstm(x, hp, cp):
        z = [x * Wx[k] + hp * U[k] + b[k] for k in range(4)]
        i, fg, o, u = sig(z[0]), sig(z[1]), sig(z[2]), math.tanh(z[3])
        c = i * u + fg * cp
        return o * math.tanh(c), c

    ha, ca = lstm(float(table[0, 0]), 0.0, 0.0)
    hb, cb = lstm(float(table[1, 0]), ha, ca)
    hp = math.tanh(hb * float(pp.W_rec[0, 0]) + float(pp.bias[0]))
    he = float(table[2, 0])
    hr = math.tanh(hp * float(pr.W_rec[0, 0]) + he * float(pr.W_rec[1, 0]) + float(pr.bias[0]))
    assert abs(f["h"][0, 0] - ha) < 1e-15 and abs(f["h"][1, 0] - hb) < 1e-15
    assert abs(f["h"][2, 0] - hp) < 1e-15 and f["c"][2, 0] == f["c"][1, 0]
    assert f["h"][3, 0] == he and f["c"][3, 0] == 0.0
    assert abs(f["h"][4, 0] - hr) < 1e-15


# ---------------------------------------------------------------- library reductions

def _chain(kind_leaf_op, n_int, side):
    """leaf, then n_int internal nodes each reading the previous one on ``side``."""
    nodes = [(0, [], 0)]
    for k in range(n_int):
        kids = [k, -1] if side == 0 else [-1, k]
        nodes.append((1, kids, -1))
    return nodes


def _blocks(M, H, order):
    """rows of a torch gate-stacked weight from our column blocks in ``order``."""
    return np.concatenate([M[:, g * H:(g + 1) * H].T for g in order], axis=0)


@pytest.mark.parametrize("side", [0, 1])
def test_treelstm_one_sided_chain_is_lstmcell(side):
    H, D_in, n_int = 4, 3, 6
    rng = np.random.default_rng(3 + side)
    p = random_params(rng, TL, D_in, 2, H)
    ops = [gen.OpSpec(TL, 0, 1, 0), gen.OpSpec(TL, 2, 0, 0)]
    table = rng.standard_normal((1, D_in)).astype(np.float32)
    w = make_workload([_chain(0, n_int, side)], ops, [p], H, table, seed=9)
    f, bw = run(w)
    fg = 1 + side                                  # the forget gate that sees the chain
    order = [0, fg, 4, 3]                          # torch gate order (i, f, g, o)
    Wx = torch.tensor(_blocks(p.W_in.astype(float), H, order), requires_grad=True)
    Uk = p.W_rec.astype(float)[side * H:(side + 1) * H]
    Uh = torch.tensor(_blocks(Uk, H, order), requires_grad=True)
    bb = torch.tensor(np.concatenate([p.bias.astype(float)[g * H:(g + 1) * H] for g in order]),
                      requires_grad=True)
    x = torch.tensor(table.astype(float))
    zero_in = torch.zeros(1, D_in, dtype=torch.float64)
    h = torch.zeros(1, H, dtype=torch.float64)
    c = torch.zeros(1, H, dtype=torch.float64)
    hs = []
    for t in range(n_int + 1):
        xin = x if t == 0 else zero_in
        gates = xin @ Wx.T + h @ Uh.T + bb
        i, fgt, g, o = gates.chunk(4, dim=1)
        c = torch.sigmoid(fgt) * c + torch.sigmoid(i) * torch.tanh(g)
        h = torch.sigmoid(o) * torch.tanh(c)
        hs.append(h)
    # same recurrence through the library cell, to pin our gate reading of LSTMCell
    cell = torch.nn.LSTMCell(D_in, H, dtype=torch.float64)
    with torch.no_grad():
        cell.weight_ih.copy_(Wx); cell.weight_hh.copy_(Uh); cell.bias_ih.copy_(bb); cell.bias_hh.zero_()
    hh = cc = torch.zeros(1, H, dtype=torch.float64)
    for t in range(n_int + 1):
        hh, cc = cell(x if t == 0 else zero_in, (hh, cc))
        assert torch.allclose(hh, hs[t], rtol=0, atol=1e-14)
    got = np.stack([f["h"][t] for t in range(n_int + 1)])
    ref = torch.cat(hs).detach().numpy()
    assert np.abs(got - ref).max() < 1e-14
    # backward: L = <g, h_root>
    g = torch.tensor(w.dh_roots.astype(float))
    (hs[-1] * g).sum().backward()
    gW = bw["grads"][0]
    ref_Wx = Wx.grad.numpy()
    ref_U = Uh.grad.numpy()
    ref_b = bb.grad.numpy()
    for j, gi in enumerate(order):
        assert np.abs(gW["W_in"][:, gi * H:(gi + 1) * H] - ref_Wx[j * H:(j + 1) * H].T).max() < 1e-13
        assert np.abs(gW["W_rec"][side * H:(side + 1) * H, gi * H:(gi + 1) * H]
                      - ref_U[j * H:(j + 1) * H].T).max() < 1e-13
        assert np.abs(gW["bias"][gi * H:(gi + 1) * H] - ref_b[j * H:(j + 1) * H]).max() < 1e-13
    other = 1 - side
    assert np.all(gW["W_rec"][other * H:(other + 1) * H] == 0)      # the zero child contributes nothing
    other_f = 1 + other
    assert np.all(gW["bias"][other_f * H:(other_f + 1) * H] == 0)   # its forget gate multiplies c = 0


def test_lstm_op_chain_is_lstmcell():
    H, D_in, n = 5, 3, 7
    rng = np.random.default_rng(5)
    p = random_params(rng, LS, D_in, 1, H)
    ops = [gen.OpSpec(LS, 1, 1, 0)]
    table = rng.standard_normal((n, D_in)).astype(np.float32)
    w = make_workload([[(0, [t - 1], t) for t in range(n)]], ops, [p], H, table, seed=4)
    f, bw = run(w)
    order = [0, 1, 3, 2]
    cell = torch.nn.LSTMCell(D_in, H, dtype=torch.float64)
    with torch.no_grad():
        cell.weight_ih.copy_(torch.tensor(_blocks(p.W_in.astype(float), H, order)))
        cell.weight_hh.copy_(torch.tensor(_blocks(p.W_rec.astype(float), H, order)))
        cell.bias_ih.copy_(torch.tensor(np.concatenate([p.bias.astype(float)[g * H:(g + 1) * H] for g in order])))
        cell.bias_hh.zero_()
    x = torch.tensor(table.astype(float))
    hh = cc = torch.zeros(1, H, dtype=torch.float64)
    for t in range(n):
        hh, cc = cell(x[t:t + 1], (hh, cc))
        assert np.abs(f["h"][t] - hh.detach().numpy()[0]).max() < 1e-14
        assert np.abs(f["c"][t] - cc.detach().numpy()[0]).max() < 1e-14
    (hh * torch.tensor(w.dh_roots.astype(float))).sum().backward()
    gW = bw["grads"][0]
    wih = cell.weight_ih.grad.numpy()
    whh = cell.weight_hh.grad.numpy()
    for j, gi in enumerate(order):
        assert np.abs(gW["W_in"][:, gi * H:(gi + 1) * H] - wih[j * H:(j + 1) * H].T).max() < 1e-13
        assert np.abs(gW["W_rec"][:, gi * H:(gi + 1) * H] - whh[j * H:(j + 1) * H].T).max() < 1e-13


@pytest.mark.parametrize("kind,side", [(RNN, 0), (RNN, 1), (PJ, 0)])
def test_treernn_and_proj_chains_are_rnncell(kind, side):
    H, n_int = 4, 5
    rng = np.random.default_rng(11 + side + kind)
    arity = 2 if kind == RNN else 1
    p = random_params(rng, kind, 0, arity, H)
    pe = gen.ParamSet(EMB, H, 0, None, None, np.zeros(0, np.float32))
    ops = [gen.OpSpec(EMB, 0, 1, 1), gen.OpSpec(kind, arity, 0, 0)]
    table = rng.standard_normal((1, H)).astype(np.float32)
    nodes = [(0, [], 0)]
    for k in range(n_int):
        kids = ([k, -1] if side == 0 else [-1, k]) if arity == 2 else [k]
        nodes.append((1, kids, -1))
    w = make_workload([nodes], ops, [p, pe], H, table, seed=2)
    f, bw = run(w)
    cell = torch.nn.RNNCell(1, H, nonlinearity="tanh", dtype=torch.float64)
    Wk = p.W_rec.astype(float)[side * H:(side + 1) * H]
    with torch.no_grad():
        cell.weight_hh.copy_(torch.tensor(Wk.T)); cell.bias_hh.copy_(torch.tensor(p.bias.astype(float)))
        cell.bias_ih.zero_()
    hh = torch.tensor(table.astype(float))
    assert np.abs(f["h"][0] - hh.numpy()[0]).max() == 0
    for t in range(1, n_int + 1):
        hh = cell(torch.zeros(1, 1, dtype=torch.float64), hh)
        assert np.abs(f["h"][t] - hh.detach().numpy()[0]).max() < 1e-14
    (hh * torch.tensor(w.dh_roots.astype(float))).sum().backward()
    gW = bw["grads"][0]["W_rec"][side * H:(side + 1) * H]
    assert np.abs(gW - cell.weight_hh.grad.numpy().T).max() < 1e-13
    assert np.abs(bw["grads"][0]["bias"] - cell.bias_hh.grad.numpy()).max() < 1e-13


# ---------------------------------------------------------------- closed forms at depth

def _zero_weight_treelstm(H, D_in, bu):
    bias = np.zeros(5 * H, np.float32)
    bias[4 * H:] = bu
    return gen.ParamSet(TL, D_in, 2, np.zeros((D_in, 5 * H), np.float32),
                        np.zeros((2 * H, 5 * H), np.float32), bias)


def test_zero_weight_balanced_tree_closed_form():
    """i = f_l = f_r = o = 1/2, u = tanh(b_u): a leaf has c = a = tanh(b_u)/2 and level l has
    c = l a, h = tanh(l a) / 2."""
    H, bu = 3, 0.37
    w = gen.config2(num_graphs=2, leaves=64, hidden=H)
    w.params = [_zero_weight_treelstm(H, H, bu)]
    b = oracle_batch(w)
    f = EV.forward(b, oracle_params(w), H, w.leaf_table)
    from oracle.schedule import depths
    d = np.asarray(depths(b["node_op"], b["child_ptr"], b["child_idx"]))
    a = 0.5 * math.tanh(np.float32(bu))
    assert np.abs(f["c"] - (d * a)[:, None]).max() < 1e-14
    assert np.abs(f["h"] - 0.5 * np.tanh(d * a)[:, None]).max() < 1e-14


def test_zero_weight_caterpillar_to_depth_512():
    """spine node k: c_k = a + (c_{k-1} + a)/2, tending to 3a; spine 511 gives depth 512."""
    H, bu, s = 2, -0.8, 511
    bld = gen._GraphBuilder()
    gen.caterpillar(bld, s, 0, 1, [0] * (s + 1))
    csr = gen.assemble([bld.arrays()])
    ops = [(TL, 0, 1, 0), (TL, 2, 0, 0)]
    P = [dict(W_in=np.zeros((1, 5 * H)), W_rec=np.zeros((2 * H, 5 * H)),
              bias=np.r_[np.zeros(4 * H), np.full(H, bu)])]
    b = dict(csr, ops=ops)
    f = EV.forward(b, P, H, np.zeros((1, 1)))
    a = 0.5 * math.tanh(bu)
    c = a                                  # bottom leaf
    spine_nodes = [v for v in range(len(csr["node_op"])) if csr["node_op"][v] == 1]
    for v in spine_nodes:
        c = a + 0.5 * (c + a)
        assert abs(f["c"][v, 0] - c) < 1e-13
        assert abs(f["h"][v, 0] - 0.5 * math.tanh(c)) < 1e-13
    assert abs(c - 3 * a) < 1e-12
    from oracle.schedule import depths
    assert max(depths(csr["node_op"], csr["child_ptr"], csr["child_idx"])) == 512


# ---------------------------------------------------------------- finite differences

def _loss(w, dh_nodes):
    b, P = oracle_batch(w), oracle_params(w)
    f = EV.forward(b, P, w.hidden, w.leaf_table.astype(np.float64))
    roots = EV.roots(b)
    L = sum(float(np.dot(w.dh_roots[r], f["h"][v])) for r, v in enumerate(roots))
    if dh_nodes is not None:
        L += float((dh_nodes * f["h"]).sum())
    return L


def _fd_check(w, dh_nodes, eps=1e-6, tol=1e-6):
    """Central differences in fp64 on every parameter and leaf-table entry."""
    _, bw = run(w, dh_nodes)
    # float64 copies so perturbations are exact
    w.leaf_table = w.leaf_table.astype(np.float64)
    for p in w.params:
        for name in ("W_in", "W_rec", "bias"):
            a = getattr(p, name)
            if a is not None:
                setattr(p, name, a.astype(np.float64))
    checked = 0
    for si, p in enumerate(w.params):
        for name in ("W_in", "W_rec", "bias"):
            arr = getattr(p, name)
            if arr is None or arr.size == 0:
                continue
            an = bw["grads"][si][name]
            for idx in np.ndindex(arr.shape):
                old = arr[idx]
                arr[idx] = old + eps; lp = _loss(w, dh_nodes)
                arr[idx] = old - eps; lm = _loss(w, dh_nodes)
                arr[idx] = old
                num = (lp - lm) / (2 * eps)
                assert abs(num - an[idx]) <= tol * max(1.0, abs(num)), (si, name, idx, num, an[idx])
                checked += 1
    tab = w.leaf_table
    for idx in np.ndindex(tab.shape):
        old = tab[idx]
        tab[idx] = old + eps; lp = _loss(w, dh_nodes)
        tab[idx] = old - eps; lm = _loss(w, dh_nodes)
        tab[idx] = old
        num = (lp - lm) / (2 * eps)
        assert abs(num - bw["d_table"][idx]) <= tol * max(1.0, abs(num)), ("table", idx)
        checked += 1
    return checked


def test_fd_treelstm_tree_and_dag():
    H, D_in = 2, 2
    rng = np.random.default_rng(21)
    p = random_params(rng, TL, D_in, 2, H)
    ops = [gen.OpSpec(TL, 0, 1, 0), gen.OpSpec(TL, 2, 0, 0)]
    table = rng.standard_normal((3, D_in)).astype(np.float32)
    g1 = [(0, [], 0), (0, [], 1), (1, [0, 1], -1), (0, [], 2), (1, [2, 3], -1)]
    g2 = [(0, [], 1), (1, [0, 0], -1), (1, [1, 0], -1), (1, [2, -1], -1)]     # shared leaf, fan-out 3
    w = make_workload([g1, g2], ops, [p], H, table, seed=3)
    dh_nodes = rng.standard_normal((w.num_nodes, H))
    assert _fd_check(w, dh_nodes) > 50


def test_fd_mixed_lstm_treelstm_proj():
    H, D_in = 2, 2
    rng = np.random.default_rng(22)
    pl = random_params(rng, LS, D_in, 1, H)
    pt = random_params(rng, TL, 0, 2, H)
    pp = random_params(rng, PJ, 0, 1, H)
    ops = [gen.OpSpec(LS, 1, 1, 0), gen.OpSpec(TL, 2, 0, 1), gen.OpSpec(PJ, 1, 0, 2)]
    table = rng.standard_normal((3, D_in)).astype(np.float32)
    g = [(0, [-1], 0), (0, [0], 1), (0, [1], 2), (1, [0, 1], -1), (2, [3], -1), (1, [4, 2], -1)]
    w = make_workload([g], ops, [pl, pt, pp], H, table, seed=5)
    assert _fd_check(w, rng.standard_normal((w.num_nodes, H))) > 40


def test_fd_treernn_embed():
    H = 2
    rng = np.random.default_rng(23)
    pr = random_params(rng, RNN, 0, 2, H)
    pe = gen.ParamSet(EMB, H, 0, None, None, np.zeros(0, np.float32))
    ops = [gen.OpSpec(EMB, 0, 1, 1), gen.OpSpec(RNN, 2, 0, 0)]
    table = rng.standard_normal((3, H)).astype(np.float32)
    g = [(0, [], 0), (0, [], 2), (1, [0, 1], -1), (0, [], 0), (1, [2, 3], -1)]
    w = make_workload([g], ops, [pr, pe], H, table, seed=6)
    assert _fd_check(w, rng.standard_normal((w.num_nodes, H))) > 10


# ---------------------------------------------------------------- invariants

def test_dead_leaf_forget_columns_and_linearity():
    w = gen.config3(num_graphs=3, hidden=4, emb_dim=3, vocab=30)
    _, bw = run(w)
    H = 4
    assert np.all(bw["grads"][0]["W_in"][:, H:3 * H] == 0)
    w2 = gen.subset(w, range(3))
    w2.dh_roots = 2.5 * w.dh_roots.astype(np.float64)
    _, bw2 = run(w2)
    for name in ("W_in", "W_rec", "bias"):
        assert np.abs(bw2["grads"][0][name] - 2.5 * bw["grads"][0][name]).max() < 1e-12


def test_batching_and_graph_order_invariance():
    w = gen.config4(num_graphs=4, hidden=3, in_dim=2, max_chain=6)
    f, bw = run(w)
    gp = w.graph_ptr
    for g in range(w.num_graphs):
        fg, _ = run(gen.subset(w, [g]))
        assert np.array_equal(fg["h"], f["h"][gp[g]:gp[g + 1]])
        assert np.array_equal(fg["c"], f["c"][gp[g]:gp[g + 1]])
    perm = [2, 0, 3, 1]
    wp = gen.subset(w, perm)
    fp, bwp = run(wp)
    off = 0
    for g in perm:
        n = gp[g + 1] - gp[g]
        assert np.array_equal(fp["h"][off:off + n], f["h"][gp[g]:gp[g + 1]])
        off += n
    for name in ("W_in", "W_rec", "bias"):
        a, b = bwp["grads"][0][name], bw["grads"][0][name]
        if a is not None:
            assert np.abs(a - b).max() < 1e-12
