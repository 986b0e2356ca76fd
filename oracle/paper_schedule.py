"""The paper's own form of the schedule (Section 2), written out step by step (oracle; test infrastructure
only).

Input: one disconnected DAG (a batch of graphs).  Source nodes are constants of a tensor type; every other
node invokes an operation enumerated in advance, whose inputs and outputs each have a fixed tensor type;
an edge connects output k of a node u to input j of a node v.

The five scheduling steps of Section 2, in order:
  1. depth: constants 0, an operation node 1 + the largest depth among the nodes it reads;
  2. pass-throughs: a value (u, k) read at depth d + 1 > depth(u) + 1 is carried by identity operations,
     one per intermediate depth, so that every node of depth d + 1 reads only results of depth d;
  3. batching: all nodes invoking the same operation at the same depth form one batch;
  4. concatenation: at each depth, the outputs of one tensor type are concatenated in the order the
     operations were enumerated;
  5. labels: every edge gets (d, t, i) -- the depth and type of the value it reads and its index into that
     concatenation; the schedule is the indices i grouped by depth and operation.

Readings where the paper is silent (the GPU scheduler makes the same choices):
  * pass-throughs are operations too, one per tensor type t, enumerated after the K user operations (op id
    K + t), with one input and one output of type t; one pass-through per value and depth, shared by all
    readers of that value (not one per edge);
  * inside a batch, nodes are in ascending node id; pass-through instances in ascending value order
    (node id, then output slot);
  * within one operation's share of a concatenation, its outputs of that type are in slot order, each
    taking the whole batch in batch order;
  * the depth-0 state of type t holds the constants of type t in ascending node id;
  * gather indices of a batch are stored input-slot-major: slot j of batch b, row r at off[b] + j * rows + r.

Node encoding: node_op[v] >= 0 is an operation id; node_op[v] = -1 - t marks a constant of type t (one
output, slot 0).  ops[o] = (in_types, out_types).

The product path never imports this module, and it imports nothing from the product package.
"""
from __future__ import annotations

from typing import Dict, List, Sequence, Tuple


def _inputs(in_ptr, in_node, in_slot, v):
    return [(int(in_node[e]), int(in_slot[e])) for e in range(int(in_ptr[v]), int(in_ptr[v + 1]))]


def out_types(node_op, ops, v) -> List[int]:
    o = int(node_op[v])
    return [-1 - o] if o < 0 else list(ops[o][1])


def validate(node_op, in_ptr, in_node, in_slot, ops, num_types) -> None:
    """Raises ValueError on a malformed typed graph (an operation or type out of range, a wrong input count,
    an edge from a missing output or of the wrong type, a constant with inputs, a cycle)."""
    n = len(node_op)
    if len(in_ptr) != n + 1 or in_ptr[0] != 0 or in_ptr[n] != len(in_node) or len(in_slot) != len(in_node):
        raise ValueError("malformed CSR")
    for v in range(n):
        o = int(node_op[v])
        ins = _inputs(in_ptr, in_node, in_slot, v)
        if o < 0:
            if -1 - o >= num_types:
                raise ValueError(f"node {v}: constant of an unknown type")
            if ins:
                raise ValueError(f"node {v}: a constant has inputs")
            continue
        if o >= len(ops):
            raise ValueError(f"node {v}: operation out of range")
        if len(ins) != len(ops[o][0]):
            raise ValueError(f"node {v}: {len(ins)} inputs for an operation of {len(ops[o][0])}")
        for j, (u, k) in enumerate(ins):
            if not 0 <= u < n:
                raise ValueError(f"node {v}: input {j} from a missing node")
            ot = out_types(node_op, ops, u)
            if not 0 <= k < len(ot):
                raise ValueError(f"node {v}: input {j} from a missing output")
            if ot[k] != ops[o][0][j]:
                raise ValueError(f"node {v}: input {j} has the wrong type")
    depths(node_op, in_ptr, in_node)


def depths(node_op, in_ptr, in_node) -> List[int]:
    """Step 1, by an explicit stack (long chains do not hit the interpreter's recursion limit)."""
    n = len(node_op)
    depth = [-1] * n
    state = [0] * n  # 0 new, 1 on the stack, 2 done
    for root in range(n):
        if state[root]:
            continue
        stack = [(root, 0)]
        state[root] = 1
        while stack:
            v, e = stack[-1]
            end = int(in_ptr[v + 1])
            e = max(e, int(in_ptr[v]))
            if e < end:
                stack[-1] = (v, e + 1)
                u = int(in_node[e])
                if state[u] == 1:
                    raise ValueError(f"cycle through node {u}")
                if state[u] == 0:
                    state[u] = 1
                    stack.append((u, 0))
                continue
            stack.pop()
            state[v] = 2
            if int(node_op[v]) < 0:
                depth[v] = 0
            else:
                depth[v] = 1 + max(depth[int(in_node[e])] for e in range(int(in_ptr[v]), end))
    return depth


def paper_schedule(node_op, in_ptr, in_node, in_slot, ops: Sequence[Tuple[Sequence[int], Sequence[int]]],
                   num_types: int) -> dict:
    validate(node_op, in_ptr, in_node, in_slot, ops, num_types)
    n, K, T = len(node_op), len(ops), num_types
    # step 1
    depth = depths(node_op, in_ptr, in_node)
    D = max([0] + depth)

    # step 2: the deepest reader of every value; pass-through instances (value, depth) in value order
    last: Dict[Tuple[int, int], int] = {}
    for v in range(n):
        for (u, k) in _inputs(in_ptr, in_node, in_slot, v):
            last[(u, k)] = max(last.get((u, k), 0), depth[v])
    values = [(u, k) for u in range(n) for k in range(len(out_types(node_op, ops, u)))]
    passes = [(u, k, d) for (u, k) in values for d in range(depth[u] + 1, last.get((u, k), 0))]

    # the items of steps 3-4: operation nodes and pass-through instances, each with its depth, operation,
    # inputs (value, depth it is read at) and output types
    items = []  # (depth, op, order key, inputs [(u, k)], output types, what)
    for v in range(n):
        o = int(node_op[v])
        if o >= 0:
            items.append((depth[v], o, (0, v, 0), _inputs(in_ptr, in_node, in_slot, v), list(ops[o][1]), ("node", v)))
    for (u, k, d) in passes:
        t = out_types(node_op, ops, u)[k]
        items.append((d, K + t, (1, u, k), [(u, k)], [t], ("pass", u, k)))
    # step 3: batches by (depth, op); nodes by id, pass-throughs by value
    items.sort(key=lambda it: (it[0], it[1], it[2]))
    batches = []  # (depth, op, [items])
    for it in items:
        if batches and batches[-1][0] == it[0] and batches[-1][1] == it[1]:
            batches[-1][2].append(it)
        else:
            batches.append((it[0], it[1], [it]))

    # step 4: concatenations per (depth, type); where = index of (value, depth) in concat(depth, its type)
    size = [[0] * T for _ in range(D + 1)]
    where: Dict[Tuple[int, int, int], int] = {}
    for v in range(n):  # depth 0: the constants of each type, ascending node id
        if int(node_op[v]) < 0:
            t = -1 - int(node_op[v])
            where[(v, 0, 0)] = size[0][t]
            size[0][t] += 1
    for (d, o, its) in batches:  # batches are already in (depth, enumeration order)
        for slot, t in enumerate(its[0][4]):
            for it in its:
                src = (it[5][1], 0) if it[5][0] == "node" else (it[5][1], it[5][2])
                key = (src[0], src[1] if it[5][0] == "pass" else slot, d)
                where[key] = size[d][t]
                size[d][t] += 1

    # step 5: labels; every read at depth d comes from depth d - 1 (the value itself or its pass-through)
    def label(u, k, d):
        src_d = d - 1
        t = out_types(node_op, ops, u)[k]
        return (src_d, t, where[(u, k, src_d if src_d > depth[u] else depth[u])])

    table = []
    gather: List[int] = []
    edge_label = {}
    for (d, o, its) in batches:
        off = len(gather)
        nin = len(its[0][3])
        for j in range(nin):
            for it in its:
                u, k = it[3][j]
                lab = label(u, k, d)
                gather.append(lab[2])
                if it[5][0] == "node":
                    edge_label[(it[5][1], j)] = lab
        table.append(dict(depth=d, op=o, rows=len(its), gather_off=off,
                          items=[it[5] for it in its]))
    return dict(num_levels=D, depth=depth, state_size=size, batches=table, gather=gather,
                passes=passes, edge_label=edge_label, num_types=T, num_ops=K)
