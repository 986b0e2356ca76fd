"""Counter-based random numbers of the recurrent-dropout masks (oracle side; test infrastructure only).

The masks are the method's random draw (Section 3.5 trains the Tree-LSTM with recurrent dropout).  Both
the GPU library and this oracle draw them from one counter-based generator written from its published
definition, each side in its own code: Philox4x32-10 (Salmon, Moraes, Dror and Shaw, "Parallel random
numbers: as easy as 1, 2, 3", SC 2011).  A round maps the counter (c0, c1, c2, c3) under the key (k0, k1) to

    (hi(M1 c2) ^ c1 ^ k0,  lo(M1 c2),  hi(M0 c0) ^ c3 ^ k1,  lo(M0 c0))

with M0 = 0xD2511F53, M1 = 0xCD9E8D57 and hi/lo the halves of the 64-bit product; between rounds the key
advances by the Weyl constants (0x9E3779B9, 0xBB67AE85).  Ten rounds.

Mask of node v and hidden unit j (the dropout probability p in [0, 1), the 64-bit seed and step):
    counter = (v, j // 4, low 32 bits of step, high 32 bits of step),  key = (low, high 32 bits of seed),
    r = the (j mod 4)-th output word,
    m[v, j] = 0 if r < t else s,   t = min(floor(p 2^32), 2^32 - 1),  s = fp32(1 / (1 - p)) (inverted dropout).
The threshold decision is integer, so both sides draw the same mask bit for bit.

The product path never imports this module, and it imports nothing from the product package.
"""
from __future__ import annotations

import numpy as np

M0, M1 = 0xD2511F53, 0xCD9E8D57
W0, W1 = 0x9E3779B9, 0xBB67AE85
MASK32 = 0xFFFFFFFF


def philox4x32_10(counters, key):
    """counters: [n, 4] unsigned 32-bit words; key: (k0, k1).  Returns the [n, 4] output words (uint32)."""
    c = np.asarray(counters, dtype=np.uint64).reshape(-1, 4) & MASK32
    c0, c1, c2, c3 = (c[:, i].copy() for i in range(4))
    k0, k1 = int(key[0]) & MASK32, int(key[1]) & MASK32
    for r in range(10):
        if r > 0:
            k0 = (k0 + W0) & MASK32
            k1 = (k1 + W1) & MASK32
        p0 = c0 * np.uint64(M0)          # < 2^64: exact in uint64
        p1 = c2 * np.uint64(M1)
        hi0, lo0 = p0 >> np.uint64(32), p0 & np.uint64(MASK32)
        hi1, lo1 = p1 >> np.uint64(32), p1 & np.uint64(MASK32)
        c0, c1, c2, c3 = hi1 ^ c1 ^ np.uint64(k0), lo1, hi0 ^ c3 ^ np.uint64(k1), lo0
    return np.stack([c0, c1, c2, c3], axis=1).astype(np.uint32)


def dropout_threshold(p: float) -> int:
    if not (0.0 <= p < 1.0):
        raise ValueError("dropout probability must lie in [0, 1)")
    return int(min(np.floor(p * 4294967296.0), 4294967295.0))


def dropout_mask(num_nodes: int, H: int, p: float, seed: int, step: int) -> np.ndarray:
    """[num_nodes, H] float32 mask in NODE order (row v = node v): 0 or fp32(1 / (1 - p))."""
    t = dropout_threshold(p)
    s = np.float32(1.0 / (1.0 - p))
    blocks = (H + 3) // 4
    v = np.repeat(np.arange(num_nodes, dtype=np.uint64), blocks)
    jb = np.tile(np.arange(blocks, dtype=np.uint64), num_nodes)
    lo, hi = np.uint64(step & MASK32), np.uint64((step >> 32) & MASK32)
    ctr = np.stack([v, jb, np.full_like(v, lo), np.full_like(v, hi)], axis=1)
    r = philox4x32_10(ctr, (seed & MASK32, (seed >> 32) & MASK32)).reshape(num_nodes, blocks * 4)[:, :H]
    return np.where(r < np.uint32(t), np.float32(0.0), s).astype(np.float32)
