"""Reference validator and scheduler (oracle; test infrastructure only).

Follows the scheduling algorithm of Section 2 of the paper:
  1. depth: nodes with no dependencies (constants) get depth 0; a node whose
     dependencies have maximum depth d gets depth d + 1;
  2. pass-through identities so that depth d+1 reads only depth d -- here an
     identity on a pool that keeps every level, so nothing is emitted;
  3. batch all nodes running the same operation at the same depth;
  4. concatenate the outputs of one depth, in operation-enumeration order;
  5. label every edge with its index into the concatenated outputs; the
     schedule is those indices grouped by depth and operation.

Readings where the paper is silent:
  * the constants are the leaf-table rows and the ``-1`` zero states, which
    are not nodes, so an operation node with no node children has depth 1 and
    the number of batched steps equals the maximum depth;
  * inside one (depth, op) group, nodes keep ascending global node id;
  * groups within one depth follow ascending op id (enumeration order);
  * the edge label is a global position in one pool that holds every level
    (positions are in (depth, op, node id) order), which makes the
    pass-throughs unnecessary; the paper's per-depth index i equals
    ``pos - level_ptr[depth - 1]``;
  * roots are the nodes that are nobody's child, in ascending node id.
"""
from __future__ import annotations

import numpy as np

# Status codes (same numbering as the library's ABI).
E_OK = 0
E_INVALID = -1
E_OP = -2
E_ARITY = -3
E_CHILD = -4
E_INPUT = -5
E_CYCLE = -6


def _graph_of_nodes(graph_ptr, n):
    g_of = [-1] * n
    for g in range(len(graph_ptr) - 1):
        for v in range(int(graph_ptr[g]), int(graph_ptr[g + 1])):
            g_of[v] = g
    return g_of


def validate(graph_ptr, node_op, child_ptr, child_idx, node_input, ops, num_inputs) -> int:
    """Return E_OK or the first error found, checking structure, then each node in order.

    ``ops`` is a sequence of (kind, arity, has_input, param_set)."""
    graph_ptr = [int(x) for x in graph_ptr]
    child_ptr = [int(x) for x in child_ptr]
    n = len(node_op)
    e = len(child_idx)
    if len(graph_ptr) < 1 or graph_ptr[0] != 0 or graph_ptr[-1] != n:
        return E_INVALID
    if any(graph_ptr[i] > graph_ptr[i + 1] for i in range(len(graph_ptr) - 1)):
        return E_INVALID
    if len(child_ptr) != n + 1 or child_ptr[0] != 0 or child_ptr[-1] != e:
        return E_INVALID
    if any(child_ptr[i] > child_ptr[i + 1] for i in range(n)):
        return E_INVALID
    if len(node_input) != n:
        return E_INVALID
    g_of = _graph_of_nodes(graph_ptr, n)
    for v in range(n):
        op = int(node_op[v])
        if op < 0 or op >= len(ops):
            return E_OP
        kind, arity, has_input, _ = ops[op]
        if child_ptr[v + 1] - child_ptr[v] != arity:
            return E_ARITY
        for j in range(child_ptr[v], child_ptr[v + 1]):
            c = int(child_idx[j])
            if c == -1:
                continue
            if c < 0 or c >= n or g_of[c] != g_of[v]:
                return E_CHILD
        inp = int(node_input[v])
        if has_input:
            if inp < 0 or inp >= num_inputs:
                return E_INPUT
        elif inp != -1:
            return E_INPUT
    # cycles: depth-first search with three colours
    white, grey, black = 0, 1, 2
    colour = [white] * n
    for s in range(n):
        if colour[s] != white:
            continue
        stack = [(s, child_ptr[s])]
        colour[s] = grey
        while stack:
            v, j = stack[-1]
            if j < child_ptr[v + 1]:
                stack[-1] = (v, j + 1)
                c = int(child_idx[j])
                if c < 0:
                    continue
                if colour[c] == grey:
                    return E_CYCLE
                if colour[c] == white:
                    colour[c] = grey
                    stack.append((c, child_ptr[c]))
            else:
                colour[v] = black
                stack.pop()
    return E_OK


def children(child_ptr, child_idx, v):
    return [int(c) for c in child_idx[int(child_ptr[v]):int(child_ptr[v + 1])]]


def depths(node_op, child_ptr, child_idx):
    """depth(v) = 1 + max(depth of v's node children), a ``-1`` child being a depth-0
    constant and the max of nothing being 0.  Memoised; explicit stack instead of
    Python recursion so that long chains do not hit the interpreter's limit."""
    n = len(node_op)
    depth = [0] * n
    done = [False] * n
    for s in range(n):
        if done[s]:
            continue
        stack = [s]
        while stack:
            v = stack[-1]
            if done[v]:
                stack.pop()
                continue
            pending = [c for c in children(child_ptr, child_idx, v) if c >= 0 and not done[c]]
            if pending:
                stack.extend(pending)
                continue
            d = 0
            for c in children(child_ptr, child_idx, v):
                if c >= 0:
                    d = max(d, depth[c])
            depth[v] = 1 + d
            done[v] = True
            stack.pop()
    return depth


def reference_schedule(node_op, child_ptr, child_idx, node_input, ops) -> dict:
    """The schedule of a valid batch, by the plain definitions (see module docstring)."""
    n = len(node_op)
    num_ops = len(ops)
    depth = depths(node_op, child_ptr, child_idx)
    D = max(depth) if n else 0

    def key(v):
        return (depth[v] - 1) * num_ops + int(node_op[v])

    pos_node = sorted(range(n), key=lambda v: (key(v), v))
    node_pos = [0] * n
    for p, v in enumerate(pos_node):
        node_pos[v] = p
    # level_ptr[l] = number of nodes of depth <= l (first position of level l + 1)
    per_level = [0] * (D + 1)
    for v in range(n):
        per_level[depth[v]] += 1
    level_ptr = [0] * (D + 1)
    running = 0
    for lvl in range(D + 1):
        running += per_level[lvl]
        level_ptr[lvl] = running
    groups = []          # (level, op, row_begin, rows, idx_off)
    child_pos = []
    idx_off = 0
    p = 0
    while p < n:
        k = key(pos_node[p])
        q = p
        while q < n and key(pos_node[q]) == k:
            q += 1
        v0 = pos_node[p]
        op = int(node_op[v0])
        arity = ops[op][1]
        groups.append((depth[v0], op, p, q - p, idx_off))
        for r in range(p, q):
            for c in children(child_ptr, child_idx, pos_node[r]):
                child_pos.append(node_pos[c] if c >= 0 else -1)
        idx_off += (q - p) * arity
        p = q
    input_idx = [int(node_input[v]) for v in pos_node]
    has_parent = [False] * n
    for c in child_idx:
        if int(c) >= 0:
            has_parent[int(c)] = True
    root_pos = [node_pos[v] for v in range(n) if not has_parent[v]]
    a = np.asarray
    return dict(
        depth=a(depth, np.int32), num_levels=D,
        pos_node=a(pos_node, np.int32), node_pos=a(node_pos, np.int32),
        level_ptr=a(level_ptr, np.int32),
        group_level=a([g[0] for g in groups], np.int32), group_op=a([g[1] for g in groups], np.int32),
        group_row_begin=a([g[2] for g in groups], np.int32), group_rows=a([g[3] for g in groups], np.int32),
        group_idx_off=a([g[4] for g in groups], np.int32),
        child_pos=a(child_pos, np.int32), input_idx=a(input_idx, np.int32),
        root_pos=a(root_pos, np.int32),
    )
