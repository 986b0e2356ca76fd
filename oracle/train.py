"""The training step around the batched path, fp64 (test infrastructure only).

Section 3.5 trains the binary Tree-LSTM on sentiment trees in which every node carries a class label:
each node's state feeds a linear layer and a softmax, the loss is the cross entropy against the node's
label (a sparse softmax cross entropy, Section 3.3's pipeline example), and the parameters are updated by
TensorFlow's Adam optimizer (Section 3.3).

``softmax_ce``  per-node head over the nodes' states h [N, H]:
                    z = h W + b,  p = softmax(z),  loss_v = log sum_c exp(z_vc) - z_{v, y_v}
                the objective is  L = scale * sum over labelled nodes of loss_v  (label -1: no loss), and
                its gradients are  dz = scale (p - onehot(y)),  dh = dz W^T,  dW = h^T dz,  db = sum_v dz.
``adam_step``   one update of Kingma and Ba's Adam in the form TensorFlow's optimizer uses (the bias
                corrections folded into the step size):
                    m = b1 m + (1 - b1) g,   v = b2 v + (1 - b2) g^2,
                    lr_t = lr sqrt(1 - b2^t) / (1 - b1^t),   p = p - lr_t m / (sqrt(v) + eps)
                (with eps = 0 this is Algorithm 1 of Kingma and Ba exactly).

The product path never imports this module, and it imports nothing from the product package.
"""
from __future__ import annotations

import numpy as np


def softmax_ce(h: np.ndarray, labels: np.ndarray, W: np.ndarray, b: np.ndarray, scale: float = 1.0):
    """Per-node losses and the gradients of scale * (sum of the labelled nodes' losses).

    h [N, H], labels [N] int (-1: unlabelled), W [H, C], b [C].  Returns (loss [N], dh [N, H], dW [H, C],
    db [C]); unlabelled nodes have loss 0 and dh 0."""
    h = np.asarray(h, np.float64)
    W = np.asarray(W, np.float64)
    b = np.asarray(b, np.float64)
    labels = np.asarray(labels)
    N, C = h.shape[0], W.shape[1]
    z = h @ W + b
    zmax = z.max(axis=1, keepdims=True) if N else np.zeros((0, 1))
    lse = (zmax + np.log(np.exp(z - zmax).sum(axis=1, keepdims=True)))[:, 0]
    live = labels >= 0
    rows = np.arange(N)
    y = np.where(live, labels, 0)
    loss = np.where(live, lse - z[rows, y], 0.0)
    dz = np.exp(z - lse[:, None])
    dz[rows, y] -= 1.0
    dz *= scale * live[:, None]
    return loss, dz @ W.T, h.T @ dz, dz.sum(axis=0)


def adam_step(p, g, m, v, t: int, lr: float = 1e-3, b1: float = 0.9, b2: float = 0.999, eps: float = 1e-8):
    """Step t (1, 2, ...) of Adam on parameters p with gradient g and moments m, v.  Returns new (p, m, v)."""
    p, g, m, v = (np.asarray(a, np.float64) for a in (p, g, m, v))
    m = b1 * m + (1.0 - b1) * g
    v = b2 * v + (1.0 - b2) * g * g
    lr_t = lr * np.sqrt(1.0 - b2 ** t) / (1.0 - b1 ** t)
    return p - lr_t * m / (np.sqrt(v) + eps), m, v
