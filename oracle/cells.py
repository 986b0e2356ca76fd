"""Per-node operations of the oracle (fp64, unbatched; test infrastructure only).

Every function takes ONE node: its input row ``x`` (or None), the states of its
child slots ``hs``/``cs`` (zero vectors where the child is missing), and the
parameters of its operation family ``P`` = dict(W_in, W_rec, bias) as float64.
z is always

    z = x . W_in  +  sum_k h_k . W_rec[k H:(k+1) H]  +  bias

with the terms for an absent input or an absent child left out (they are zero).

Operations (the paper's experiments, Sections 2.1 and 3.3):

  EMBED     h = table[row]                             (embedding lookup)
  TREERNN   h = tanh(z),  z over [h_l; h_r]            (binary TreeRNN cell)
  TREELSTM  binary (N = 2) Tree-LSTM of Tai et al., eqs. 9-14 as the paper
            invokes them: gates (i | f_l | f_r | o | u),
              i, f_l, f_r, o = sigmoid(.),  u = tanh(.)
              c = i*u + f_l*c_l + f_r*c_r,  h = o*tanh(c)
            a leaf is TreeLSTM(Embedding(word), 0, 0), an internal node
            TreeLSTM(0, h_l, h_r) (the two equations of Section 3.5); the
            forget-gate biases are not tied.
  LSTM      one step of the chain that Fold(g, z = 0) builds: gates
            (i | f | o | u), c = i*u + f*c_p, h = o*tanh(c)
  PROJ      h = tanh(h_c . P + b), c = c_c (a unary projection)

The gradient functions are the chain rule written out by hand for each of
these; the tests pin them with central finite differences.
"""
from __future__ import annotations

import numpy as np

EMBED, TREERNN, TREELSTM, LSTM, PROJ = 0, 1, 2, 3, 4

# number of child slots and of gate blocks of each kind
SLOTS = {EMBED: 0, TREERNN: 2, TREELSTM: 2, LSTM: 1, PROJ: 1}
GATES = {EMBED: 0, TREERNN: 1, TREELSTM: 5, LSTM: 4, PROJ: 1}


def sigmoid(x):
    x = np.asarray(x, dtype=np.float64)
    out = np.empty_like(x)
    pos = x >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-x[pos]))
    ex = np.exp(x[~pos])
    out[~pos] = ex / (1.0 + ex)
    return out


def pre_activation(P, H, x, hs):
    """z = x W_in + sum_k h_k W_rec_k + b for the terms that are present."""
    z = np.array(P["bias"], dtype=np.float64, copy=True)
    if x is not None:
        z += x @ P["W_in"]
    for k, h in enumerate(hs):
        z += h @ P["W_rec"][k * H:(k + 1) * H]
    return z


def forward_node(kind, P, H, x, hs, cs, m=None):
    """Return (h, c, cache) of one node.

    m: the node's recurrent-dropout mask [H] or None. Section 3.5 trains with the recurrent dropout of
    Semeniuta et al.: the mask multiplies the candidate update u where it enters the memory cell,
    c = i*(m*u) + sum_k f_k*c_k, so the forget paths of the cell state are never dropped. The mask's values
    (0, or 1/(1-p) for inverted dropout) are drawn by the caller; the LSTM kinds use it, the others ignore it."""
    if kind == EMBED:
        return np.array(x, dtype=np.float64), np.zeros(H), {}
    z = pre_activation(P, H, x, hs)
    if kind in (TREERNN, PROJ):
        h = np.tanh(z)
        c = np.array(cs[0], dtype=np.float64) if kind == PROJ else np.zeros(H)
        return h, c, {"h": h}
    if kind == TREELSTM:
        i = sigmoid(z[0:H])
        fl = sigmoid(z[H:2 * H])
        fr = sigmoid(z[2 * H:3 * H])
        o = sigmoid(z[3 * H:4 * H])
        u = np.tanh(z[4 * H:5 * H])
        um = u if m is None else u * m
        cl, cr = cs
        c = i * um + fl * cl + fr * cr
        h = o * np.tanh(c)
        return h, c, {"i": i, "fl": fl, "fr": fr, "o": o, "u": u, "c": c, "m": m}
    if kind == LSTM:
        i = sigmoid(z[0:H])
        f = sigmoid(z[H:2 * H])
        o = sigmoid(z[2 * H:3 * H])
        u = np.tanh(z[3 * H:4 * H])
        um = u if m is None else u * m
        (cp,) = cs
        c = i * um + f * cp
        h = o * np.tanh(c)
        return h, c, {"i": i, "f": f, "o": o, "u": u, "c": c, "m": m}
    raise ValueError(f"unknown kind {kind}")


def backward_node(kind, P, H, x, hs, cs, cache, dh, dc):
    """Given dL/dh and dL/dc of the node's outputs, return
    (dx or None, [dh_k], [dc_k], {"W_in": .., "W_rec": .., "bias": ..})."""
    if kind == EMBED:
        return np.array(dh, dtype=np.float64), [], [], {}
    if kind in (TREERNN, PROJ):
        h = cache["h"]
        dz = dh * (1.0 - h * h)
        dcs = [np.array(dc, dtype=np.float64)] if kind == PROJ else [np.zeros(H) for _ in hs]
    elif kind == TREELSTM:
        i, fl, fr, o, u, c = (cache[k] for k in ("i", "fl", "fr", "o", "u", "c"))
        m = cache["m"] if cache["m"] is not None else 1.0
        cl, cr = cs
        tc = np.tanh(c)
        dct = dc + dh * o * (1.0 - tc * tc)
        dz = np.concatenate([
            dct * (m * u) * i * (1.0 - i),
            dct * cl * fl * (1.0 - fl),
            dct * cr * fr * (1.0 - fr),
            dh * tc * o * (1.0 - o),
            dct * i * m * (1.0 - u * u),
        ])
        dcs = [dct * fl, dct * fr]
    elif kind == LSTM:
        i, f, o, u, c = (cache[k] for k in ("i", "f", "o", "u", "c"))
        m = cache["m"] if cache["m"] is not None else 1.0
        (cp,) = cs
        tc = np.tanh(c)
        dct = dc + dh * o * (1.0 - tc * tc)
        dz = np.concatenate([
            dct * (m * u) * i * (1.0 - i),
            dct * cp * f * (1.0 - f),
            dh * tc * o * (1.0 - o),
            dct * i * m * (1.0 - u * u),
        ])
        dcs = [dct * f]
    else:
        raise ValueError(f"unknown kind {kind}")
    grads = {"bias": dz}
    dx = None
    if x is not None:
        dx = P["W_in"] @ dz
        grads["W_in"] = np.outer(x, dz)
    dhs = []
    if hs:
        Wr = P["W_rec"]
        gW = np.zeros_like(Wr, dtype=np.float64)
        for k, hk in enumerate(hs):
            dhs.append(Wr[k * H:(k + 1) * H] @ dz)
            gW[k * H:(k + 1) * H] = np.outer(hk, dz)
        grads["W_rec"] = gW
    return dx, dhs, dcs, grads
