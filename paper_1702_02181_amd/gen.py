"""Seeded synthetic workloads for the dynamic-batching hot path.

This module decides *shapes and values* only: the topology of each input
graph (written as the CSR arrays the library takes), the op table, the
parameter tensors, the leaf table and the upstream gradients.  None of the
method's arithmetic lives here -- no depth, no sort, no cell -- so the CPU
oracle (test infrastructure) and the HIP path can both consume its output
without sharing any code.

The workloads stand in for the paper's two settings: the synthetic speed
benchmark of Section 2.1 (random binary trees, embedding-lookup leaves,
a Tree-LSTM variant at the non-terminals) and the sentiment experiment of
Section 3.5 (binarised parse trees whose leaves are word embeddings).  No
dataset is read; token frequencies follow a Zipf law as a stand-in for
natural-language text.

Graph conventions (the op table is "specified in advance and enumerated",
Section 2):
  * a batch is one disconnected DAG; ``graph_ptr[g]..graph_ptr[g+1]`` are the
    global node ids of graph ``g``;
  * node ``v`` runs op ``node_op[v]``; its children (inputs coming from other
    nodes) are ``child_idx[child_ptr[v]:child_ptr[v+1]]``, global ids, with
    ``-1`` standing for a zero state (the paper's ``Zeros`` block / the
    ``z = 0`` start of ``Fold``);
  * ``node_input[v]`` is the leaf-table row a node with an input reads, else
    ``-1``.

Parameter values for bf16 workloads are generated in fp32 and rounded to the
nearest bf16 (ties to even) here, so every consumer sees the same exact
values; they are kept as float32 arrays whose values are bf16-representable.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

# Operation kinds (mirrors the library's FOLD_* kind enumeration).
KIND_EMBED = 0
KIND_TREERNN = 1
KIND_TREELSTM = 2
KIND_LSTM = 3
KIND_PROJ = 4
KIND_ATTN_SCORE = 5
KIND_ATTN_SUM = 6
KIND_ATTN_OUT = 7
ATTN_KINDS = (KIND_ATTN_SCORE, KIND_ATTN_SUM, KIND_ATTN_OUT)

KIND_NAMES = {KIND_EMBED: "embed", KIND_TREERNN: "treernn", KIND_TREELSTM: "treelstm",
              KIND_LSTM: "lstm", KIND_PROJ: "proj", KIND_ATTN_SCORE: "attn_score",
              KIND_ATTN_SUM: "attn_sum", KIND_ATTN_OUT: "attn_out"}

# Gate blocks per kind: the width of z is NUM_GATES[kind] * hidden (the attention kinds have no z).
NUM_GATES = {KIND_EMBED: 0, KIND_TREERNN: 1, KIND_TREELSTM: 5, KIND_LSTM: 4, KIND_PROJ: 1,
             KIND_ATTN_SCORE: 0, KIND_ATTN_SUM: 0, KIND_ATTN_OUT: 0}
# Child slots of the attention kinds (their parameter sets' arity).
ATTN_SLOTS = {KIND_ATTN_SCORE: 1, KIND_ATTN_SUM: 2, KIND_ATTN_OUT: 1}


# --------------------------------------------------------------------------
# bf16 helpers (value preparation, not method arithmetic)
# --------------------------------------------------------------------------

def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round to nearest, ties to even); return raw bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    bias = ((u >> 16) & 1) + 0x7FFF
    return ((u + bias) >> 16).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """float32 array whose values are the bf16 roundings of ``x``."""
    return bf16_bits_to_f32(to_bf16_bits(x))


# --------------------------------------------------------------------------
# Containers
# --------------------------------------------------------------------------

@dataclass
class OpSpec:
    kind: int
    arity: int
    has_input: int
    param_set: int


@dataclass
class ParamSet:
    """Parameters of one operation family.

    ``W_in``  [in_dim, G*H]     applied to the leaf-table row (ops with input)
    ``W_rec`` [arity*H, G*H]    applied to the children's h, child k uses rows k*H..(k+1)*H
    ``bias``  [G*H]
    Gate blocks are in canonical order along the columns:
    Tree-LSTM (i | f_l | f_r | o | u), LSTM (i | f | o | u), TreeRNN / PROJ one block.
    The attention scorer (ATTN_SCORE) has W_rec [H, 1] (the vector w) and bias [1]; the ATTN_SUM and
    ATTN_OUT sets hold no values (W_rec None, bias empty).
    """
    kind: int
    in_dim: int
    arity: int
    W_in: Optional[np.ndarray]
    W_rec: Optional[np.ndarray]
    bias: np.ndarray


@dataclass
class Workload:
    name: str
    dtype: str            # "f32" or "bf16": weights, leaf table and h pool
    hidden: int
    graph_ptr: np.ndarray
    node_op: np.ndarray
    child_ptr: np.ndarray
    child_idx: np.ndarray
    node_input: np.ndarray
    ops: List[OpSpec]
    params: List[ParamSet]
    leaf_table: np.ndarray   # float32 [rows, in_dim]
    dh_roots: np.ndarray     # float32 [num_roots, H], upstream gradient on roots
    backward: bool = True
    meta: dict = field(default_factory=dict)

    @property
    def num_graphs(self) -> int:
        return int(self.graph_ptr.shape[0] - 1)

    @property
    def num_nodes(self) -> int:
        return int(self.node_op.shape[0])

    @property
    def num_edges(self) -> int:
        return int(self.child_idx.shape[0])

    @property
    def num_ops(self) -> int:
        return len(self.ops)


# --------------------------------------------------------------------------
# Graph assembly
# --------------------------------------------------------------------------

class _GraphBuilder:
    """Accumulates the nodes of one graph with local ids."""

    def __init__(self):
        self.op: List[int] = []
        self.kids: List[List[int]] = []
        self.inp: List[int] = []

    def add(self, op: int, kids: Sequence[int] = (), inp: int = -1) -> int:
        self.op.append(op)
        self.kids.append(list(kids))
        self.inp.append(inp)
        return len(self.op) - 1

    def arrays(self):
        op = np.asarray(self.op, dtype=np.int32)
        cnt = np.asarray([len(k) for k in self.kids], dtype=np.int32)
        flat = [c for k in self.kids for c in k]
        kids = np.asarray(flat, dtype=np.int64) if flat else np.zeros(0, np.int64)
        inp = np.asarray(self.inp, dtype=np.int64)
        return op, cnt, kids, inp


def assemble(graphs) -> dict:
    """Concatenate per-graph (op, child_count, child_local, input) arrays into one batch CSR."""
    ops, cnts, kids, inps, sizes = [], [], [], [], []
    off = 0
    for (op, cnt, kid, inp) in graphs:
        n = op.shape[0]
        ops.append(op)
        cnts.append(cnt)
        k = kid.copy()
        k[k >= 0] += off
        kids.append(k)
        inps.append(inp)
        sizes.append(n)
        off += n
    graph_ptr = np.zeros(len(graphs) + 1, dtype=np.int64)
    graph_ptr[1:] = np.cumsum(sizes)
    cnt = np.concatenate(cnts) if cnts else np.zeros(0, np.int32)
    child_ptr = np.zeros(cnt.shape[0] + 1, dtype=np.int64)
    child_ptr[1:] = np.cumsum(cnt)
    return dict(
        graph_ptr=graph_ptr.astype(np.int32),
        node_op=(np.concatenate(ops) if ops else np.zeros(0, np.int32)).astype(np.int32),
        child_ptr=child_ptr.astype(np.int32),
        child_idx=(np.concatenate(kids) if kids else np.zeros(0, np.int64)).astype(np.int32),
        node_input=(np.concatenate(inps) if inps else np.zeros(0, np.int64)).astype(np.int32),
    )


def count_roots(num_nodes: int, child_idx: np.ndarray) -> int:
    """Number of nodes that are nobody's child (used only to size upstream gradients)."""
    seen = np.zeros(num_nodes, dtype=bool)
    c = child_idx[child_idx >= 0]
    seen[c] = True
    return int(num_nodes - seen.sum())


def roots_per_graph(graph_ptr: np.ndarray, child_idx: np.ndarray) -> np.ndarray:
    n = int(graph_ptr[-1])
    seen = np.zeros(n, dtype=bool)
    seen[child_idx[child_idx >= 0]] = True
    is_root = ~seen
    cs = np.concatenate([[0], np.cumsum(is_root)])
    return (cs[graph_ptr[1:]] - cs[graph_ptr[:-1]]).astype(np.int64)


# --------------------------------------------------------------------------
# Tree shapes (all emitted in post-order, so children precede parents)
# --------------------------------------------------------------------------

def random_split_tree(b: _GraphBuilder, n_leaves: int, rng, leaf_op: int, node_op: int,
                      leaf_inputs) -> int:
    """Binary tree over ``n_leaves`` leaves: the left subtree gets k ~ U{1..n-1} leaves."""
    it = iter(leaf_inputs)

    def build(n):
        if n == 1:
            return b.add(leaf_op, (), int(next(it)))
        k = int(rng.integers(1, n))
        left = build(k)
        right = build(n - k)
        return b.add(node_op, (left, right))

    return build(n_leaves)


def balanced_tree(b: _GraphBuilder, n_leaves: int, leaf_op: int, node_op: int, leaf_inputs) -> int:
    """Complete binary tree (n_leaves a power of two for a perfectly balanced shape)."""
    it = iter(leaf_inputs)

    def build(n):
        if n == 1:
            return b.add(leaf_op, (), int(next(it)))
        half = n // 2
        left = build(half)
        right = build(n - half)
        return b.add(node_op, (left, right))

    return build(n_leaves)


def caterpillar(b: _GraphBuilder, spine: int, leaf_op: int, node_op: int, leaf_inputs) -> int:
    """Spine of ``spine`` internal nodes; each hangs one leaf, the bottom one two."""
    it = iter(leaf_inputs)
    cur = b.add(leaf_op, (), int(next(it)))
    for _ in range(spine):
        leaf = b.add(leaf_op, (), int(next(it)))
        cur = b.add(node_op, (cur, leaf))
    return cur


def share_subexpressions(op, cnt, kids, inp, frac, rng, leaf_op):
    """Turn a post-order binary tree into a DAG with shared sub-expressions.

    About ``frac`` of the non-root nodes become shared: for each chosen node v a
    fan-out f ~ U{2,3,4} is drawn and f-1 leaf-child slots of internal nodes that
    come later in post-order (hence are not descendants of v) are redirected to v;
    the leaves they displaced are deleted.  Acyclic by construction, no orphans.
    """
    n = op.shape[0]
    if n <= 2:
        return op, cnt, kids, inp
    ptr = np.zeros(n + 1, dtype=np.int64)
    ptr[1:] = np.cumsum(cnt)
    kids = kids.copy()
    is_leaf = cnt == 0
    # slot table: (parent, flat position) for every slot whose child is a leaf
    parent_of_slot = np.repeat(np.arange(n), cnt)
    slot_child = kids
    slot_ok = (slot_child >= 0) & is_leaf[np.maximum(slot_child, 0)]
    deleted = np.zeros(n, dtype=bool)
    shared = np.zeros(n, dtype=bool)
    target = int(round(frac * (n - 1)))
    made = 0
    attempts = 0
    while made < target and attempts < 8 * target + 16:
        attempts += 1
        v = int(rng.integers(0, n - 1))          # never the root (last in post-order)
        if deleted[v] or shared[v]:
            continue
        f = int(rng.integers(2, 5))
        cand = np.nonzero(slot_ok & (parent_of_slot > v) & (slot_child != v))[0]
        if cand.shape[0] == 0:
            continue
        take = min(f - 1, cand.shape[0])
        pick = rng.choice(cand, size=take, replace=False)
        for s in pick:
            leaf = int(slot_child[s])
            deleted[leaf] = True
            slot_child[s] = v
            slot_ok[s] = False
        # slots pointing at v or at a deleted leaf can no longer be redirected
        slot_ok &= ~(slot_child == v)
        shared[v] = True
        if is_leaf[v]:
            slot_ok &= slot_child != v
        made += 1
    keep = ~deleted
    new_id = np.full(n, -1, dtype=np.int64)
    new_id[keep] = np.arange(int(keep.sum()))
    kept_slots = keep[parent_of_slot]
    new_kids = slot_child[kept_slots]
    new_kids = np.where(new_kids >= 0, new_id[np.maximum(new_kids, 0)], -1)
    return op[keep], cnt[keep], new_kids, inp[keep]


def lstm_chain_reduce(b: _GraphBuilder, n: int, rng, row0: int, p_proj: float,
                      op_lstm: int, op_tree: int, op_proj: int) -> int:
    """LSTM chain over n token rows (Fold with z = 0), then a balanced Reduce over the
    chain states (the left half gets floor(n/2) items), with a PROJ node above each
    internal tree node with probability p_proj."""
    chain = []
    prev = -1
    for i in range(n):
        prev = b.add(op_lstm, (prev,), row0 + i)
        chain.append(prev)

    def reduce(items):
        if len(items) == 1:
            return items[0]
        m = len(items) // 2
        left = reduce(items[:m])
        right = reduce(items[m:])
        t = b.add(op_tree, (left, right))
        if rng.random() < p_proj:
            t = b.add(op_proj, (t,))
        return t

    return reduce(chain)


def attention_sequence(b: _GraphBuilder, n: int, row0: int, op_embed: int, op_f: int, op_score: int,
                       op_sum: int, op_out: int, op_g: int = -1) -> int:
    """Feed-forward attention over a sequence of n token rows (Section 3.4): h_t = f(x_t) for every
    element (an embedding lookup, then a PROJ layer f), one scorer node per element, the scored items
    summed by a balanced Reduce (the left half gets floor(n/2) items), the attention output c, and
    optionally a PROJ layer g on c."""
    items = []
    for i in range(n):
        x = b.add(op_embed, (), row0 + i)
        h = b.add(op_f, (x,))
        items.append(b.add(op_score, (h,)))

    def reduce(seq):
        if len(seq) == 1:
            return seq[0]
        m = len(seq) // 2
        left = reduce(seq[:m])
        right = reduce(seq[m:])
        return b.add(op_sum, (left, right))

    c = b.add(op_out, (reduce(items),))
    return b.add(op_g, (c,)) if op_g >= 0 else c


# --------------------------------------------------------------------------
# Value generators
# --------------------------------------------------------------------------

def zipf_tokens(rng, vocab: int, size: int, s: float = 1.0) -> np.ndarray:
    p = 1.0 / np.arange(1, vocab + 1, dtype=np.float64) ** s
    p /= p.sum()
    return rng.choice(vocab, size=size, p=p).astype(np.int64)


def _uniform(rng, shape, lo=-0.1, hi=0.1):
    return rng.uniform(lo, hi, size=shape).astype(np.float32)


def _finish_values(x: np.ndarray, dtype: str) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    return round_bf16(x) if dtype == "bf16" else x


def make_param_set(rng, kind: int, in_dim: int, arity: int, hidden: int, dtype: str) -> ParamSet:
    g = NUM_GATES[kind]
    if kind == KIND_EMBED:
        return ParamSet(kind, in_dim, 0, None, None, np.zeros(0, np.float32))
    if kind == KIND_ATTN_SCORE:
        return ParamSet(kind, 0, 1, None, _finish_values(_uniform(rng, (hidden, 1)), dtype), _uniform(rng, (1,)))
    if kind in (KIND_ATTN_SUM, KIND_ATTN_OUT):
        return ParamSet(kind, 0, ATTN_SLOTS[kind], None, None, np.zeros(0, np.float32))
    W_in = _finish_values(_uniform(rng, (in_dim, g * hidden)), dtype) if in_dim > 0 else None
    W_rec = _finish_values(_uniform(rng, (arity * hidden, g * hidden)), dtype) if arity > 0 else None
    bias = _uniform(rng, (g * hidden,))
    return ParamSet(kind, in_dim, arity, W_in, W_rec, bias)


def _finish(name, dtype, hidden, csr, ops, params, leaf_table, rng, backward, meta=None) -> Workload:
    r = count_roots(csr["node_op"].shape[0], csr["child_idx"])
    dh = rng.standard_normal((r, hidden)).astype(np.float32)
    return Workload(name=name, dtype=dtype, hidden=hidden, ops=ops, params=params,
                    leaf_table=np.ascontiguousarray(leaf_table, dtype=np.float32), dh_roots=dh,
                    backward=backward, meta=meta or {}, **csr)


# --------------------------------------------------------------------------
# The five benchmark configurations
# --------------------------------------------------------------------------

def config1(seed: int = 1, num_graphs: int = 8) -> Workload:
    """8 random-split binary trees, 2-16 leaves; TreeRNN h = tanh([h_l; h_r] W + b),
    H = 64, fp32; leaves embed tokens from a 100-row table ~ N(0, 0.1^2); forward only."""
    rng = np.random.default_rng(seed)
    H, vocab = 64, 100
    graphs = []
    for _ in range(num_graphs):
        nl = int(rng.integers(2, 17))
        toks = rng.integers(0, vocab, size=nl)
        b = _GraphBuilder()
        random_split_tree(b, nl, rng, 0, 1, toks)
        graphs.append(b.arrays())
    csr = assemble(graphs)
    ops = [OpSpec(KIND_EMBED, 0, 1, 0), OpSpec(KIND_TREERNN, 2, 0, 1)]
    E = (0.1 * rng.standard_normal((vocab, H))).astype(np.float32)
    params = [make_param_set(rng, KIND_EMBED, H, 0, H, "f32"),
              make_param_set(rng, KIND_TREERNN, 0, 2, H, "f32")]
    return _finish("cfg1_treernn_h64", "f32", H, csr, ops, params, E, rng, backward=False)


def config2(seed: int = 2, num_graphs: int = 256, leaves: int = 256, hidden: int = 256) -> Workload:
    """256 complete balanced binary trees of 256 leaves (511 nodes, depth 9); binary
    Tree-LSTM (5 gates), H = 256, fp32; one leaf-input row ~ N(0, 1) of dim 256 per leaf."""
    rng = np.random.default_rng(seed)
    H, D_in = hidden, hidden
    graphs = []
    row = 0
    for _ in range(num_graphs):
        b = _GraphBuilder()
        balanced_tree(b, leaves, 0, 1, range(row, row + leaves))
        row += leaves
        graphs.append(b.arrays())
    csr = assemble(graphs)
    ops = [OpSpec(KIND_TREELSTM, 0, 1, 0), OpSpec(KIND_TREELSTM, 2, 0, 0)]
    X = rng.standard_normal((row, D_in)).astype(np.float32)
    params = [make_param_set(rng, KIND_TREELSTM, D_in, 2, H, "f32")]
    return _finish("cfg2_treelstm_balanced_h256", "f32", H, csr, ops, params, X, rng, backward=True)


def config3(seed: int = 3, num_graphs: int = 1024, hidden: int = 300, vocab: int = 20000,
            emb_dim: int = 300, leaf_range=(5, 60), zipf: bool = True) -> Workload:
    """1024 parse-tree-shaped random-split trees with U[5,60] leaves; Zipf(1) tokens
    over a 20000 x 300 embedding table; binary Tree-LSTM H = 300; bf16 weights."""
    rng = np.random.default_rng(seed)
    H = hidden
    sizes = rng.integers(leaf_range[0], leaf_range[1] + 1, size=num_graphs)
    total = int(sizes.sum())
    toks = zipf_tokens(rng, vocab, total) if zipf else rng.integers(0, vocab, size=total)
    graphs = []
    off = 0
    for nl in sizes:
        b = _GraphBuilder()
        random_split_tree(b, int(nl), rng, 0, 1, toks[off:off + nl])
        off += int(nl)
        graphs.append(b.arrays())
    csr = assemble(graphs)
    ops = [OpSpec(KIND_TREELSTM, 0, 1, 0), OpSpec(KIND_TREELSTM, 2, 0, 0)]
    E = _finish_values(0.1 * rng.standard_normal((vocab, emb_dim)), "bf16")
    params = [make_param_set(rng, KIND_TREELSTM, emb_dim, 2, H, "bf16")]
    return _finish("cfg3_treelstm_parse_h300_bf16", "bf16", H, csr, ops, params, E, rng, backward=True)


def config4(seed: int = 4, num_graphs: int = 512, hidden: int = 512, in_dim: int = 128,
            max_chain: int = 100, p_proj: float = 0.2) -> Workload:
    """512 mixed-op graphs: an LSTM chain of n ~ U{1..100} steps over 128-dim token rows,
    a Reduce-shaped binary Tree-LSTM over the chain states, and a unary PROJ node above
    20% of the internal tree nodes.  Ops {LSTM, TREELSTM, PROJ}; H = 512; bf16."""
    rng = np.random.default_rng(seed)
    H = hidden
    graphs = []
    row = 0
    for _ in range(num_graphs):
        n = int(rng.integers(1, max_chain + 1))
        b = _GraphBuilder()
        lstm_chain_reduce(b, n, rng, row, p_proj, 0, 1, 2)
        row += n
        graphs.append(b.arrays())
    csr = assemble(graphs)
    ops = [OpSpec(KIND_LSTM, 1, 1, 0), OpSpec(KIND_TREELSTM, 2, 0, 1), OpSpec(KIND_PROJ, 1, 0, 2)]
    X = _finish_values(rng.standard_normal((row, in_dim)), "bf16")
    params = [make_param_set(rng, KIND_LSTM, in_dim, 1, H, "bf16"),
              make_param_set(rng, KIND_TREELSTM, 0, 2, H, "bf16"),
              make_param_set(rng, KIND_PROJ, 0, 1, H, "bf16")]
    return _finish("cfg4_mixed_lstm_treelstm_proj_h512_bf16", "bf16", H, csr, ops, params, X, rng,
                   backward=True)


def config5(seed: int = 5, num_graphs: int = 4096, hidden: int = 1024, vocab: int = 20000,
            spine_range=(200, 511), share_frac: float = 0.10, balanced_leaves: int = 256) -> Workload:
    """4096 graphs: even index a balanced 256-leaf tree, odd index a caterpillar with
    spine s ~ U{200..511} (depth <= 512); then ~10% of the non-root nodes of every graph
    become shared sub-expressions with fan-out 2-4.  Binary Tree-LSTM, H = 1024, bf16;
    Zipf(1) tokens over a 20000 x 1024 embedding table.  About 2.0 M nodes."""
    rng = np.random.default_rng(seed)
    H = hidden
    graphs = []
    for gi in range(num_graphs):
        b = _GraphBuilder()
        if gi % 2 == 0:
            nl = balanced_leaves
            balanced_tree(b, nl, 0, 1, zipf_tokens(rng, vocab, nl))
        else:
            s = int(rng.integers(spine_range[0], spine_range[1] + 1))
            caterpillar(b, s, 0, 1, zipf_tokens(rng, vocab, s + 1))
        op, cnt, kids, inp = b.arrays()
        graphs.append(share_subexpressions(op, cnt, kids, inp, share_frac, rng, 0))
    csr = assemble(graphs)
    ops = [OpSpec(KIND_TREELSTM, 0, 1, 0), OpSpec(KIND_TREELSTM, 2, 0, 0)]
    E = _finish_values(0.1 * rng.standard_normal((vocab, H)), "bf16")
    params = [make_param_set(rng, KIND_TREELSTM, H, 2, H, "bf16")]
    return _finish("cfg5_treelstm_dag_h1024_bf16", "bf16", H, csr, ops, params, E, rng, backward=True)


CONFIGS = {1: config1, 2: config2, 3: config3, 4: config4, 5: config5}


def table1(batch: int, mode: str, seed: int = 7, leaves: int = 64, hidden: int = 1024, vocab: int = 10000,
           dtype: str = "f32") -> Workload:
    """The inference timing benchmark of Section 2.1 (Table 1): `batch` random binary trees of `leaves` leaves
    (2 leaves - 1 nodes: 64 leaves = 127 nodes, the table's tree size of 128), leaves looked up in an embedding
    table, internal nodes a binary Tree-LSTM with state size `hidden`; forward only.
      "dynamic": every tree has the same random shape; two operations (leaf, internal node).
      "full":    every tree has a random shape of its own ("full dynamic").
      "manual":  the same shape as "dynamic", and every node position of the tree is an operation of its own,
                 all sharing one parameter set: the schedule then has one batched group per tree node, which is
                 what manual batching runs (one batched kernel per node of the tree's static graph), and each
                 group's children are the consecutive rows of the child position's group, which the scheduler
                 recognises as the static layout (children addressed by base + row, no gather index).
    Tokens ~ U{0..vocab-1}; table ~ N(0, 0.1^2); weights U(-0.1, 0.1)."""
    if mode not in ("dynamic", "full", "manual"):
        raise ValueError(mode)
    rng = np.random.default_rng(seed)
    H = hidden
    toks = rng.integers(0, vocab, size=(batch, leaves))
    shape_rng = np.random.default_rng(seed + 1)
    graphs = []
    base = None
    for t in range(batch):
        b = _GraphBuilder()
        # same shape: replay the same split choices for every tree
        r = shape_rng if mode == "full" else np.random.default_rng(seed + 1)
        random_split_tree(b, leaves, r, 0, 1, toks[t])
        op, cnt, kids, inp = b.arrays()
        if mode == "manual":
            if base is None:
                base = op.copy()
            op = np.arange(op.shape[0], dtype=np.int32)  # node position = operation id
        graphs.append((op, cnt, kids, inp))
    csr = assemble(graphs)
    if mode == "manual":
        ops = [OpSpec(KIND_TREELSTM, 0, 1, 0) if k == 0 else OpSpec(KIND_TREELSTM, 2, 0, 0) for k in base]
    else:
        ops = [OpSpec(KIND_TREELSTM, 0, 1, 0), OpSpec(KIND_TREELSTM, 2, 0, 0)]
    E = _finish_values(0.1 * rng.standard_normal((vocab, H)), dtype)
    params = [make_param_set(rng, KIND_TREELSTM, H, 2, H, dtype)]
    return _finish(f"table1_{mode}_b{batch}_n{2 * leaves - 1}_h{H}_{dtype}", dtype, H, csr, ops, params, E, rng,
                   backward=False)


def attention(seed: int = 6, num_graphs: int = 1024, length=(50, 100), hidden: int = 256,
              dtype: str = "bf16") -> Workload:
    """Feed-forward attention (Section 3.4, Appendix A): `num_graphs` sequences of T ~ U{length} elements,
    each element a row of a table of token vectors (N(0, 1) entries, one distinct row per element), the
    model of attention_sequence with a PROJ output layer g.  Ops: EMBED, PROJ f, ATTN_SCORE, ATTN_SUM,
    ATTN_OUT, PROJ g; weights U(-0.1, 0.1), the scorer's too (scores of standard deviation ~0.5, so that the
    attention weights of one sequence spread over a factor of ~3 between items one deviation apart); forward
    and backward."""
    rng = np.random.default_rng(seed)
    H = hidden
    graphs = []
    row = 0
    for _ in range(num_graphs):
        n = int(rng.integers(length[0], length[1] + 1))
        b = _GraphBuilder()
        attention_sequence(b, n, row, 0, 1, 2, 3, 4, 5)
        row += n
        graphs.append(b.arrays())
    csr = assemble(graphs)
    ops = [OpSpec(KIND_EMBED, 0, 1, 0), OpSpec(KIND_PROJ, 1, 0, 1), OpSpec(KIND_ATTN_SCORE, 1, 0, 2),
           OpSpec(KIND_ATTN_SUM, 2, 0, 3), OpSpec(KIND_ATTN_OUT, 1, 0, 4), OpSpec(KIND_PROJ, 1, 0, 5)]
    X = _finish_values(rng.standard_normal((row, H)), dtype)
    score = make_param_set(rng, KIND_ATTN_SCORE, 0, 1, H, dtype)
    params = [make_param_set(rng, KIND_EMBED, H, 0, H, dtype), make_param_set(rng, KIND_PROJ, 0, 1, H, dtype),
              score, make_param_set(rng, KIND_ATTN_SUM, 0, 2, H, dtype),
              make_param_set(rng, KIND_ATTN_OUT, 0, 1, H, dtype), make_param_set(rng, KIND_PROJ, 0, 1, H, dtype)]
    lo, hi = length
    return _finish(f"ffattn_b{num_graphs}_t{lo}-{hi}_h{H}_{dtype}", dtype, H, csr, ops, params, X, rng,
                   backward=True)


def make_config(k: int, **kw) -> Workload:
    return CONFIGS[k](**kw)


# --------------------------------------------------------------------------
# Sub-batches
# --------------------------------------------------------------------------

def subset(w: Workload, graph_ids: Sequence[int]) -> Workload:
    """The workload restricted to the listed graphs (in the listed order).

    The leaf table and parameters are shared unchanged; root gradients follow
    their graphs (roots are numbered in ascending node id, i.e. graph by graph)."""
    gp = w.graph_ptr.astype(np.int64)
    cp = w.child_ptr.astype(np.int64)
    rpg = roots_per_graph(w.graph_ptr, w.child_idx)
    roff = np.concatenate([[0], np.cumsum(rpg)])
    graphs = []
    dh = []
    for g in graph_ids:
        a, b_ = int(gp[g]), int(gp[g + 1])
        op = w.node_op[a:b_].copy()
        cnt = (cp[a + 1:b_ + 1] - cp[a:b_]).astype(np.int32)
        kids = w.child_idx[cp[a]:cp[b_]].astype(np.int64)
        kids = np.where(kids >= 0, kids - a, -1)
        inp = w.node_input[a:b_].astype(np.int64)
        graphs.append((op, cnt, kids, inp))
        dh.append(w.dh_roots[roff[g]:roff[g + 1]])
    csr = assemble(graphs)
    dh_roots = np.concatenate(dh, axis=0) if dh else np.zeros((0, w.hidden), np.float32)
    return Workload(name=w.name + f"_sub{len(graph_ids)}", dtype=w.dtype, hidden=w.hidden,
                    ops=w.ops, params=w.params, leaf_table=w.leaf_table, dh_roots=dh_roots,
                    backward=w.backward, meta=dict(w.meta, parent=w.name), **csr)


def shuffle_within_graphs(w: Workload, seed: int) -> Workload:
    """Same graphs, with the node ids inside every graph randomly permuted
    (node order within a graph is arbitrary, not necessarily topological)."""
    rng = np.random.default_rng(seed)
    gp = w.graph_ptr.astype(np.int64)
    cp = w.child_ptr.astype(np.int64)
    graphs = []
    for g in range(w.num_graphs):
        a, b_ = int(gp[g]), int(gp[g + 1])
        n = b_ - a
        perm = rng.permutation(n)            # new local id j holds old local id perm[j]
        inv = np.empty(n, np.int64)
        inv[perm] = np.arange(n)
        op = w.node_op[a:b_][perm]
        cnt = (cp[a + 1:b_ + 1] - cp[a:b_])[perm].astype(np.int32)
        kid_lists = []
        for j in range(n):
            v = a + perm[j]
            ks = w.child_idx[cp[v]:cp[v + 1]].astype(np.int64)
            kid_lists.append(np.where(ks >= 0, inv[np.maximum(ks - a, 0)], -1))
        kids = np.concatenate(kid_lists) if kid_lists else np.zeros(0, np.int64)
        inp = w.node_input[a:b_][perm].astype(np.int64)
        graphs.append((op, cnt, kids, inp))
    csr = assemble(graphs)
    # roots change ids but keep graph order; within a graph their relative order may change,
    # so draw fresh root gradients of the same shape.
    dh = np.random.default_rng(seed + 1).standard_normal(w.dh_roots.shape).astype(np.float32)
    return Workload(name=w.name + "_shuf", dtype=w.dtype, hidden=w.hidden, ops=w.ops,
                    params=w.params, leaf_table=w.leaf_table, dh_roots=dh, backward=w.backward,
                    meta=dict(w.meta), **csr)
