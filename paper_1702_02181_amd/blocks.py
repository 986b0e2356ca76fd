"""Combinator front end (Section 3 of the paper): blocks that turn Python inputs into the op table and CSR
graphs the library schedules, so a model over trees or sequences is written once as a block expression.

Types of the values that flow between blocks (Section 3.1, in the library's terms):
  * host objects (any Python value): what ``InputTransform`` and ``Record`` see;
  * ``Row(i)``: a row of the leaf table, the tensor an operation with an input reads (``Scalar`` makes one);
  * ``Node``: the state (h, c) of a node of the graph being built;
  * ``ZERO``: the zero state / absent input (``Zeros``);
  * tuples (``Record``, ``AllOf``) and lists (``Map``) of these.

Blocks (Section 3.2): ``b1 >> b2`` composition, ``InputTransform(fn)``, ``Scalar()``, ``Zeros()``, ``Map(b)``,
``Fold(g, z)`` (g(... g(g(z, x1), x2) ..., xn), a leftward chain), ``Reduce(g)`` (g over the two halves split at
floor(n / 2), a balanced tree), ``Record(fields)``, ``AllOf(*blocks)``, ``OneOf(key_fn, cases)``, ``Optional(b)``,
``ForwardDeclaration`` (recursion), and ``Op(kind, param_set)``, the library operation as a block (the paper's
``Function``).  An ``Op`` takes the pair (x, children): x a ``Row`` or ``ZERO``, children a ``Node``, ``ZERO`` or a
tuple of them; the pair decides the operation variant (a Tree-LSTM with an input and zero children is a leaf,
with no input and two children an internal node).

``Compiler(block, ...)`` enumerates every operation variant of the expression in advance (the op table, in the
order the expression lists them) and ``build(inputs)`` traces the block over each input into one graph of a
batch: a ``gen.Workload`` that ``runner.DeviceRun`` runs through the C ABI.  Nothing here computes a state: the
front end only records nodes, edges and leaf rows.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Any, Callable, Dict, List, Sequence, Tuple

import numpy as np

from . import gen


@dataclass(frozen=True)
class Row:
    index: int


@dataclass(frozen=True)
class Node:
    id: int  # local id in the graph being built


class _Zero:
    def __repr__(self):
        return "ZERO"


ZERO = _Zero()


class _Trace:
    """The graph being built for one input."""

    def __init__(self, compiler: "Compiler"):
        self.compiler = compiler
        self.b = gen._GraphBuilder()

    def add(self, op: int, kids: Sequence[int], inp: int) -> Node:
        return Node(self.b.add(op, kids, inp))


class Block:
    def __rshift__(self, other: "Block") -> "Block":
        return _Compose(self, other)

    def __call__(self, x, t: _Trace):
        raise NotImplementedError

    def children(self) -> List["Block"]:
        return []


class _Compose(Block):
    def __init__(self, a: Block, b: Block):
        self.a, self.b = a, b

    def __call__(self, x, t):
        return self.b(self.a(x, t), t)

    def children(self):
        return [self.a, self.b]


class InputTransform(Block):
    """Host object -> host object by a Python function (pre-processing)."""

    def __init__(self, fn: Callable[[Any], Any]):
        self.fn = fn

    def __call__(self, x, t):
        return self.fn(x)


class Scalar(Block):
    """A Python int -> the leaf-table row it names."""

    def __call__(self, x, t):
        return Row(int(x))


class Zeros(Block):
    """Anything -> the zero state."""

    def __call__(self, x, t):
        return ZERO


class Map(Block):
    def __init__(self, f: Block):
        self.f = f

    def __call__(self, xs, t):
        return [self.f(x, t) for x in xs]

    def children(self):
        return [self.f]


class Fold(Block):
    """g(... g(g(z, x1), x2) ..., xn); g receives the pair (state, x)."""

    def __init__(self, g: Block, z: Block = None):
        self.g, self.z = g, Zeros() if z is None else z

    def __call__(self, xs, t):
        s = self.z(None, t)
        for x in xs:
            s = self.g((s, x), t)
        return s

    def children(self):
        return [self.g, self.z]


class Reduce(Block):
    """g over a balanced binary tree: the first floor(n / 2) elements and the rest; g receives a pair."""

    def __init__(self, g: Block):
        self.g = g

    def __call__(self, xs, t):
        xs = list(xs)
        if not xs:
            return ZERO
        if len(xs) == 1:
            return xs[0]
        m = len(xs) // 2
        return self.g((self(xs[:m], t), self(xs[m:], t)), t)

    def children(self):
        return [self.g]


class Record(Block):
    """A dict (or sequence) -> the tuple of each field's block applied to that field, in the given order."""

    def __init__(self, fields):
        self.fields: List[Tuple[Any, Block]] = list(fields.items()) if isinstance(fields, dict) else list(fields)

    def __call__(self, x, t):
        return tuple(b(x[k], t) for k, b in self.fields)

    def children(self):
        return [b for _, b in self.fields]


class AllOf(Block):
    """The same input to every block; the tuple of their outputs."""

    def __init__(self, *blocks: Block):
        self.blocks = list(blocks)

    def __call__(self, x, t):
        return tuple(b(x, t) for b in self.blocks)

    def children(self):
        return list(self.blocks)


class OneOf(Block):
    """Dispatch on key_fn(input) to one of the case blocks (cases: dict or (key, block) pairs)."""

    def __init__(self, key_fn: Callable[[Any], Any], cases):
        self.key_fn = key_fn
        self.cases: Dict[Any, Block] = dict(cases)

    def __call__(self, x, t):
        return self.cases[self.key_fn(x)](x, t)

    def children(self):
        return list(self.cases.values())


class Optional(OneOf):
    """b if the input is not None, else the zero state."""

    def __init__(self, b: Block):
        super().__init__(lambda x: x is None, {False: b, True: Zeros()})


class ForwardDeclaration:
    """A name for a block defined later; calling it makes a reference, resolve_to binds every reference."""

    def __init__(self):
        self.target: Block = None

    def __call__(self) -> Block:
        return _Ref(self)

    def resolve_to(self, b: Block):
        self.target = b


class _Ref(Block):
    def __init__(self, decl: ForwardDeclaration):
        self.decl = decl

    def __call__(self, x, t):
        if self.decl.target is None:
            raise RuntimeError("ForwardDeclaration used before resolve_to")
        return self.decl.target(x, t)

    def children(self):
        return [self.decl.target] if self.decl.target is not None else []


# operation variants of each kind: (arity, has_input) in the order they enter the op table
_VARIANTS = {gen.KIND_EMBED: [(0, 1)], gen.KIND_TREELSTM: [(0, 1), (2, 0)], gen.KIND_LSTM: [(1, 1)],
             gen.KIND_TREERNN: [(2, 0)], gen.KIND_PROJ: [(1, 0)], gen.KIND_ATTN_SCORE: [(1, 0)],
             gen.KIND_ATTN_SUM: [(2, 0)], gen.KIND_ATTN_OUT: [(1, 0)]}


class Op(Block):
    """A library operation of the given kind on parameter set ``param_set``.  Arguments: EMBED a Row; PROJ,
    ATTN_SCORE and ATTN_OUT one state; TREERNN and ATTN_SUM a pair of states; LSTM Fold's (state, Row);
    TREELSTM (Row or ZERO, ZERO or a pair of states).  Feed-forward attention over a sequence (Section 3.4) is
    then Map(... >> Op(ATTN_SCORE)) >> Reduce(Op(ATTN_SUM)) >> Op(ATTN_OUT): the scored items, their softmax
    normaliser and weighted sum carried together through the merges (Appendix A's Sum, Broadcast and ZipWith
    in one aggregate)."""

    def __init__(self, kind: int, param_set: int):
        self.kind, self.param_set = kind, param_set

    def _split(self, x):
        """(input row or None, child node ids) of the block's argument."""
        if self.kind == gen.KIND_EMBED:
            return x, ()
        if self.kind == gen.KIND_LSTM:  # Fold's (state, x)
            s, r = x
            return r, (s,)
        if self.kind in (gen.KIND_PROJ, gen.KIND_ATTN_SCORE, gen.KIND_ATTN_OUT):
            return None, (x,)
        if self.kind in (gen.KIND_TREERNN, gen.KIND_ATTN_SUM):  # a pair (Reduce's)
            return None, tuple(x)
        r, kids = x  # Tree-LSTM: (x, children)
        kids = () if kids is ZERO else tuple(kids)
        return (None if r is ZERO else r), kids

    def __call__(self, x, t):
        r, kids = self._split(x)
        if r is not None and not isinstance(r, Row):
            raise TypeError(f"{type(self).__name__}: the input must be a Row, got {r!r}")
        arity, has_input = len(kids), int(r is not None)
        op = t.compiler.op_id(self, arity, has_input)
        ids = []
        for k in kids:
            if k is ZERO:
                ids.append(-1)
            elif isinstance(k, Node):
                ids.append(k.id)
            else:
                raise TypeError(f"child must be a Node or ZERO, got {k!r}")
        return t.add(op, ids, r.index if r is not None else -1)


class Compiler:
    """Enumerates the operations of a block expression and builds batches of graphs from Python inputs."""

    def __init__(self, root: Block):
        self.root = root
        self.ops: List[gen.OpSpec] = []
        self._ids: Dict[Tuple[int, int, int], int] = {}
        seen, stack = set(), [root]
        order = []
        while stack:  # every Op block of the expression, in depth-first order of the block tree
            b = stack.pop()
            if id(b) in seen:
                continue
            seen.add(id(b))
            if isinstance(b, Op):
                order.append(b)
            stack.extend(reversed(b.children()))
        for b in order:
            for arity, has_input in _VARIANTS[b.kind]:
                self._ids[(id(b), arity, has_input)] = len(self.ops)
                self.ops.append(gen.OpSpec(b.kind, arity, has_input, b.param_set))

    def op_id(self, b: Op, arity: int, has_input: int) -> int:
        key = (id(b), arity, has_input)
        if key not in self._ids:
            raise ValueError(f"operation kind {b.kind} has no variant with {arity} children and input={has_input}")
        return self._ids[key]

    def trace(self, x):
        """(graph arrays, output) of one input: the output is the block's value (Node ids local to the graph)."""
        t = _Trace(self)
        out = self.root(x, t)
        return t.b.arrays(), out

    def build(self, inputs, params, hidden: int, leaf_table: np.ndarray, dtype: str = "f32", seed: int = 0,
              name: str = "blocks") -> Tuple[gen.Workload, List[Any]]:
        """One graph per input.  Returns the workload and, per input, its output with Node ids made global."""
        graphs, outs, off = [], [], 0
        for x in inputs:
            arrs, out = self.trace(x)
            graphs.append(arrs)
            outs.append(_shift(out, off))
            off += arrs[0].shape[0]
        csr = gen.assemble(graphs)
        w = gen._finish(name, dtype, hidden, csr, list(self.ops), list(params), leaf_table,
                        np.random.default_rng(seed), backward=True)
        return w, outs


def _shift(v, off):
    if isinstance(v, Node):
        return Node(v.id + off)
    if isinstance(v, tuple):
        return tuple(_shift(u, off) for u in v)
    if isinstance(v, list):
        return [_shift(u, off) for u in v]
    return v
