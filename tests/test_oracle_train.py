"""Pins of the training-step oracle (per-node softmax cross entropy head and Adam; CPU only).

  * closed forms: zero weights give log C per labelled node and p - onehot = 1/C - onehot; two classes
    reduce to the logistic loss log(1 + e^(z_o - z_y)) with dz_y = -sigmoid(z_o - z_y) (Python ``math``);
  * a library routine: ``torch.nn.functional.cross_entropy`` (fp64, summed) through a linear layer and
    autograd gives the same loss and the same gradients of h, W and b;
  * central finite differences of the summed loss;
  * invariants: unlabelled nodes have no loss and no gradient and change nothing else, the bias gradient
    sums to zero over the classes, the gradients are linear in ``scale``;
  * Adam: with eps = 0 the first step moves every parameter by exactly lr * sign(g), a constant gradient
    keeps doing so at every step, and a random gradient sequence matches ``torch.optim.Adam`` (the
    bias-corrected form of Kingma and Ba's Algorithm 1) step by step; with eps > 0 one step matches
    torch's form with its eps scaled by 1 / sqrt(1 - b2^t).
"""
import math

import numpy as np
import pytest
import torch

from oracle import train as T


def _case(seed, N=9, H=7, C=5, unlabelled=2):
    rng = np.random.default_rng(seed)
    h = rng.standard_normal((N, H))
    W = 0.5 * rng.standard_normal((H, C))
    b = 0.3 * rng.standard_normal(C)
    y = rng.integers(0, C, N)
    y[rng.choice(N, unlabelled, replace=False)] = -1
    return h, y, W, b


def test_zero_weights_give_log_c():
    h, y, W, b = _case(1)
    C = W.shape[1]
    loss, dh, dW, db = T.softmax_ce(h, y, np.zeros_like(W), np.zeros_like(b), scale=1.0)
    live = y >= 0
    assert np.allclose(loss[live], math.log(C), rtol=0, atol=1e-15)
    assert np.all(loss[~live] == 0) and np.all(dh == 0)  # zero W: dh = dz W^T = 0
    expect_db = np.zeros(C)
    for v in np.nonzero(live)[0]:
        expect_db += 1.0 / C
        expect_db[y[v]] -= 1.0
    assert np.allclose(db, expect_db, atol=1e-14)


def test_two_classes_is_the_logistic_loss():
    h, y, W, b = _case(2, C=2, unlabelled=0)
    loss, dh, dW, db = T.softmax_ce(h, y, W, b, scale=1.0)
    for v in range(h.shape[0]):
        z = [sum(h[v, j] * W[j, c] for j in range(h.shape[1])) + b[c] for c in range(2)]
        t = z[1 - y[v]] - z[y[v]]
        assert loss[v] == pytest.approx(math.log1p(math.exp(t)), rel=1e-13, abs=1e-15)
        s = 1.0 / (1.0 + math.exp(-t))
        # dz_y = -sigmoid(t), dz_o = +sigmoid(t); dh = dz W^T
        for j in range(h.shape[1]):
            assert dh[v, j] == pytest.approx(-s * W[j, y[v]] + s * W[j, 1 - y[v]], rel=1e-12, abs=1e-14)


@pytest.mark.parametrize("scale", [1.0, 0.125])
def test_matches_torch_cross_entropy(scale):
    h, y, W, b = _case(3, N=11, H=6, C=4)
    loss, dh, dW, db = T.softmax_ce(h, y, W, b, scale=scale)
    th = torch.tensor(h, requires_grad=True)
    tW = torch.tensor(W, requires_grad=True)
    tb = torch.tensor(b, requires_grad=True)
    live = torch.tensor(y >= 0)
    z = th @ tW + tb
    per = torch.nn.functional.cross_entropy(z[live], torch.tensor(y)[live], reduction="none")
    (scale * per.sum()).backward()
    assert np.allclose(loss[y >= 0], per.detach().numpy(), rtol=1e-13, atol=1e-15)
    assert np.allclose(dh, th.grad.numpy(), rtol=1e-12, atol=1e-15)
    assert np.allclose(dW, tW.grad.numpy(), rtol=1e-12, atol=1e-15)
    assert np.allclose(db, tb.grad.numpy(), rtol=1e-12, atol=1e-15)


def test_finite_differences():
    h, y, W, b = _case(4, N=5, H=4, C=3, unlabelled=1)
    scale = 0.7
    _, dh, dW, db = T.softmax_ce(h, y, W, b, scale=scale)

    def objective(h_, W_, b_):
        return scale * T.softmax_ce(h_, y, W_, b_)[0].sum()

    eps = 1e-6
    for arr, grad, which in ((h, dh, 0), (W, dW, 1), (b, db, 2)):
        for idx in np.ndindex(arr.shape):
            args = [h.copy(), W.copy(), b.copy()]
            args[which][idx] += eps
            up = objective(*args)
            args[which][idx] -= 2 * eps
            dn = objective(*args)
            assert grad[idx] == pytest.approx((up - dn) / (2 * eps), rel=1e-6, abs=1e-8)


def test_unlabelled_nodes_change_nothing():
    h, y, W, b = _case(5, unlabelled=3)
    loss, dh, dW, db = T.softmax_ce(h, y, W, b, scale=1.0)
    live = y >= 0
    l2, dh2, dW2, db2 = T.softmax_ce(h[live], y[live], W, b, scale=1.0)
    assert np.allclose(loss[live], l2, rtol=1e-15, atol=0)
    assert np.all(dh[~live] == 0) and np.allclose(dh[live], dh2, rtol=1e-15, atol=0)
    assert np.allclose(dW, dW2, rtol=1e-13, atol=1e-15) and np.allclose(db, db2, rtol=1e-13, atol=1e-15)
    assert abs(db.sum()) < 1e-13  # each labelled row of dz sums to zero
    _, dh3, dW3, db3 = T.softmax_ce(h, y, W, b, scale=-2.5)
    assert np.allclose(dh3, -2.5 * dh) and np.allclose(dW3, -2.5 * dW) and np.allclose(db3, -2.5 * db)


def test_adam_first_step_is_lr_sign_g():
    rng = np.random.default_rng(6)
    p = rng.standard_normal(50)
    g = rng.standard_normal(50)
    p1, m1, v1 = T.adam_step(p, g, np.zeros(50), np.zeros(50), t=1, lr=0.01, eps=0.0)
    assert np.allclose(p1, p - 0.01 * np.sign(g), rtol=0, atol=1e-15)
    assert np.allclose(m1, 0.1 * g) and np.allclose(v1, 0.001 * g * g)


def test_adam_constant_gradient_steps_by_lr():
    rng = np.random.default_rng(7)
    p0 = rng.standard_normal(20)
    g = rng.standard_normal(20)
    p, m, v = p0.copy(), np.zeros(20), np.zeros(20)
    for t in range(1, 31):
        p, m, v = T.adam_step(p, g, m, v, t=t, lr=1e-3, eps=0.0)
        assert np.allclose(p, p0 - t * 1e-3 * np.sign(g), rtol=0, atol=1e-13)


def test_adam_matches_torch_optim():
    rng = np.random.default_rng(8)
    n, steps = 40, 12
    p0 = rng.standard_normal(n)
    grads = rng.standard_normal((steps, n))
    # eps = 0: the two forms are the same update
    tp = torch.tensor(p0.copy(), requires_grad=True)
    opt = torch.optim.Adam([tp], lr=3e-3, betas=(0.9, 0.999), eps=0.0)
    p, m, v = p0.copy(), np.zeros(n), np.zeros(n)
    for t in range(1, steps + 1):
        tp.grad = torch.tensor(grads[t - 1])
        opt.step()
        p, m, v = T.adam_step(p, grads[t - 1], m, v, t=t, lr=3e-3, eps=0.0)
        assert np.allclose(p, tp.detach().numpy(), rtol=1e-13, atol=1e-15)
    # eps > 0 at step t: TensorFlow's eps is torch's eps * sqrt(1 - b2^t) (torch adds it to sqrt(v_hat))
    for t in (1, 5):
        m0 = 0.1 * rng.standard_normal(n)
        v0 = 0.01 * rng.random(n)
        g = 1e-3 * rng.standard_normal(n)
        eps = 1e-4
        pt, _, _ = T.adam_step(p0, g, m0, v0, t=t, lr=1e-2, eps=eps)
        tp = torch.tensor(p0.copy(), requires_grad=True)
        opt = torch.optim.Adam([tp], lr=1e-2, betas=(0.9, 0.999), eps=eps / math.sqrt(1 - 0.999 ** t))
        # the optimizer state after step t - 1: moments m0, v0
        opt.state[tp] = {"step": torch.tensor(float(t - 1)), "exp_avg": torch.tensor(m0.copy()),
                         "exp_avg_sq": torch.tensor(v0.copy())}
        tp.grad = torch.tensor(g)
        opt.step()
        assert np.allclose(pt, tp.detach().numpy(), rtol=1e-12, atol=1e-15)
