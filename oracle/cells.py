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

Feed-forward attention (Section 3.4, Appendix A): e_t = a(h_t), alpha = softmax(e), c = sum_t alpha_t h_t,
with the scorer a(h) = w . h + b (W_rec = w as an [H, 1] matrix, bias = [b]).  The sums over t (the normaliser
and the weighted sum; Appendix A's two Sums) are carried together as the aggregate of a set of items,
    (m, s, acc) = (max_t e_t,  sum_t exp(e_t - m),  sum_t exp(e_t - m) h_t),
kept in the node's state as h = acc and c = [m, s, 0, ...] (H >= 2):
  ATTN_SCORE  one item from its child's h: (e, 1, h_child), e = w . h_child + b
  ATTN_SUM    the union of its two children's sets: m = max(m_1, m_2), x_k = exp(m_k - m),
              s = x_1 s_1 + x_2 s_2, acc = x_1 acc_1 + x_2 acc_2; a child with s = 0 (the zero state
              among them) is the empty set and takes no part, and the union of two empty sets is the
              zero state
  ATTN_OUT    c_att = acc / s as the node's h (c = 0); attention over the empty set is the zero vector
The aggregate's value does not depend on m (it scales s and acc alike and cancels in acc / s), so the
gradients hold m fixed: they are the exact derivatives of acc / s.

The gradient functions are the chain rule written out by hand for each of
these; the tests pin them with central finite differences.
"""
from __future__ import annotations

import numpy as np

EMBED, TREERNN, TREELSTM, LSTM, PROJ = 0, 1, 2, 3, 4
ATTN_SCORE, ATTN_SUM, ATTN_OUT = 5, 6, 7
ATTN = (ATTN_SCORE, ATTN_SUM, ATTN_OUT)

# number of child slots and of gate blocks of each kind
SLOTS = {EMBED: 0, TREERNN: 2, TREELSTM: 2, LSTM: 1, PROJ: 1, ATTN_SCORE: 1, ATTN_SUM: 2, ATTN_OUT: 1}
GATES = {EMBED: 0, TREERNN: 1, TREELSTM: 5, LSTM: 4, PROJ: 1}


def _attn_forward(kind, P, H, hs, cs):
    if kind == ATTN_SCORE:
        (hc,) = hs
        e = float(hc @ P["W_rec"][:, 0] + P["bias"][0])
        c = np.zeros(H)
        c[0], c[1] = e, 1.0
        return np.array(hc, dtype=np.float64), c, {"hc": np.array(hc, dtype=np.float64)}
    if kind == ATTN_SUM:
        live = [k for k in range(2) if cs[k][1] != 0.0]
        c = np.zeros(H)
        if not live:
            return np.zeros(H), c, {"x": [0.0, 0.0]}
        m = max(cs[k][0] for k in live)
        x = [np.exp(cs[k][0] - m) if k in live else 0.0 for k in range(2)]
        c[0] = m
        c[1] = sum(x[k] * cs[k][1] for k in range(2))
        acc = sum(x[k] * hs[k] for k in range(2))
        return acc, c, {"x": x}
    if kind == ATTN_OUT:
        (acc,), (cc,) = hs, cs
        s = float(cc[1])
        h = np.zeros(H) if s == 0.0 else np.asarray(acc, dtype=np.float64) / s
        return h, np.zeros(H), {"acc": np.array(acc, dtype=np.float64), "s": s}
    raise ValueError(kind)


def _attn_backward(kind, P, H, cache, dh, dc):
    """(dhs, dcs, grads) with m held fixed (see the module docstring)."""
    if kind == ATTN_SCORE:
        hc = cache["hc"]
        # acc = h_child exp(e - m), s = exp(e - m) at e = m: d/de acc = acc, d/de s = s = 1
        de = float(dh @ hc) + float(dc[1])
        w = P["W_rec"][:, 0]
        return [dh + de * w], [np.zeros(H)], {"W_rec": (de * hc)[:, None], "bias": np.array([de])}
    if kind == ATTN_SUM:
        x = cache["x"]
        dcs = []
        for k in range(2):
            d = np.zeros(H)
            d[1] = x[k] * dc[1]
            dcs.append(d)
        return [x[k] * dh for k in range(2)], dcs, {}
    if kind == ATTN_OUT:
        acc, s = cache["acc"], cache["s"]
        d = np.zeros(H)
        if s == 0.0:
            return [np.zeros(H)], [d], {}
        d[1] = -float(dh @ acc) / (s * s)
        return [dh / s], [d], {}
    raise ValueError(kind)


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
    if kind in ATTN:
        return _attn_forward(kind, P, H, hs, cs)
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
    if kind in ATTN:
        dhs, dcs, grads = _attn_backward(kind, P, H, cache, dh, dc)
        return None, dhs, dcs, grads
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
