"""Marshal a generated workload onto the GPU and drive the library through the binding.

Used by the tests, ``bench.py`` and the smoke check: it only moves arrays
between host and device and calls the C ABI; all arithmetic happens in the
HIP kernels."""
from __future__ import annotations

import numpy as np
import torch

from . import fold as F
from . import gen


def bf16_tensor(x: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(gen.to_bf16_bits(np.ascontiguousarray(x, np.float32)).view(np.int16)).view(torch.bfloat16)


def pad_cols(x: np.ndarray, ld: int) -> np.ndarray:
    x = np.asarray(x, np.float32)
    if x.shape[1] == ld:
        return np.ascontiguousarray(x)
    out = np.zeros((x.shape[0], ld), np.float32)
    out[:, :x.shape[1]] = x
    return out


class DeviceRun:
    def __init__(self, w: gen.Workload, device: str = "cuda", stream=None, with_backward=None):
        self.w = w
        self.device = device
        self.stream = stream
        H = w.hidden
        self.H = H
        self.ld = F.fold_row_ld(H)
        self.bf16 = w.dtype == "bf16"
        self.fdtype = F.FOLD_BF16 if self.bf16 else F.FOLD_F32
        self.tdtype = torch.bfloat16 if self.bf16 else torch.float32
        i32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.int32)).to(device)
        self.graph_ptr, self.node_op = i32(w.graph_ptr), i32(w.node_op)
        self.child_ptr, self.child_idx, self.node_input = i32(w.child_ptr), i32(w.child_idx), i32(w.node_input)
        self.ops = [(o.kind, o.arity, o.has_input, o.param_set) for o in w.ops]
        self.leaf_rows = int(w.leaf_table.shape[0])
        self.sched = F.Schedule(self.graph_ptr, self.node_op, self.child_ptr, self.child_idx, self.node_input,
                                self.ops, self.leaf_rows, stream)
        self.set_tensors = []
        for p in w.params:
            self.set_tensors.append(dict(
                kind=p.kind, in_dim=p.in_dim, arity=p.arity,
                W_in=None if p.W_in is None else self._wt(p.W_in),
                W_rec=None if p.W_rec is None else self._wt(p.W_rec),
                bias=(None if p.kind == gen.KIND_EMBED or p.bias is None or p.bias.size == 0
                      else torch.from_numpy(p.bias.astype(np.float32)).to(device))))
        self.packed = F.Packed(self.fdtype, H, self.set_tensors, stream)
        in_dim = int(w.leaf_table.shape[1])
        self.tld = F.fold_row_ld(in_dim)
        tab = pad_cols(w.leaf_table, self.tld)
        self.table = (bf16_tensor(tab) if self.bf16 else torch.from_numpy(tab)).to(device)
        N, R = w.num_nodes, self.sched.info.num_roots
        self.N, self.R = N, R
        self.h_pool = torch.zeros((max(N, 1), self.ld), dtype=self.tdtype, device=device)
        self.c_pool = torch.zeros((max(N, 1), self.ld), dtype=torch.float32, device=device)
        self.roots = torch.zeros((max(R, 1), self.ld), dtype=self.tdtype, device=device)
        self.fwd_bytes, self.bwd_bytes = F.fold_workspace_size(self.sched.handle, self.packed.handle)
        backward = w.backward if with_backward is None else with_backward
        self.ws_bytes = self.bwd_bytes if backward else self.fwd_bytes
        self.ws = torch.empty(max(self.ws_bytes, 1), dtype=torch.uint8, device=device)
        self.grads = None
        self.dh_roots = None
        self.dh_nodes = None

    def _wt(self, a):
        a = np.ascontiguousarray(a, np.float32)
        return (bf16_tensor(a) if self.bf16 else torch.from_numpy(a)).to(self.device)

    # ------------------------------------------------------------------ calls
    def forward(self, u_mask=None):
        """u_mask: recurrent-dropout mask [N, ld] fp32 in pool order (fold_forward_dropout), or None."""
        if u_mask is not None:
            F.fold_forward_dropout(self.sched.handle, self.packed.handle, self.table, self.leaf_rows, self.h_pool,
                                   self.c_pool, self.roots, u_mask, self.ws, self.ws_bytes, self.stream)
            return
        F.fold_forward(self.sched.handle, self.packed.handle, self.table, self.leaf_rows, self.h_pool,
                       self.c_pool, self.roots, self.ws, self.ws_bytes, self.stream)

    def alloc_grads(self, table_grad=True):
        sets = []
        for p in self.w.params:
            g = gen.NUM_GATES[p.kind] * self.H
            z = lambda *s: torch.zeros(s, dtype=torch.float32, device=self.device)
            if p.kind == gen.KIND_ATTN_SCORE:  # dw as [H, 1], db [1]
                sets.append((None, z(self.H, 1), z(1)))
                continue
            if p.kind == gen.KIND_EMBED or p.kind in gen.ATTN_KINDS:
                sets.append((None, None, None))
                continue
            sets.append((z(p.in_dim, g) if p.W_in is not None else None,
                         z(p.arity * self.H, g) if p.W_rec is not None else None, z(g)))
        self.grad_tensors = sets
        self.d_table = (torch.zeros((self.leaf_rows, self.tld), dtype=torch.float32, device=self.device)
                        if table_grad else None)
        self.grads = F.make_grads(sets, self.d_table)
        return sets

    def set_upstream(self, dh_roots: np.ndarray, dh_nodes_node_order: np.ndarray | None = None):
        self.dh_roots = torch.from_numpy(pad_cols(dh_roots, self.ld)).to(self.device) if self.R else None
        if dh_nodes_node_order is not None:
            node_pos = self.sched_arrays()["node_pos"]
            pool = np.zeros((self.N, self.ld), np.float32)
            pool[node_pos, :self.H] = dh_nodes_node_order
            self.dh_nodes = torch.from_numpy(pool).to(self.device)
        else:
            self.dh_nodes = None

    def zero_grads(self):
        for t in self.grad_tensors:
            for x in t:
                if x is not None:
                    x.zero_()
        if self.d_table is not None:
            self.d_table.zero_()

    def backward(self, dh_out=None, dc_out=None, u_mask=None):
        if u_mask is not None:
            F.fold_backward_dropout(self.sched.handle, self.packed.handle, self.table, self.leaf_rows, self.h_pool,
                                    self.c_pool, u_mask, self.dh_roots, self.dh_nodes, self.grads, dh_out, dc_out,
                                    self.ws, self.ws_bytes, self.stream)
            return
        F.fold_backward(self.sched.handle, self.packed.handle, self.table, self.leaf_rows, self.h_pool,
                        self.c_pool, self.dh_roots, self.dh_nodes, self.grads, dh_out, dc_out, self.ws,
                        self.ws_bytes, self.stream)

    def make_graph(self, backward=None, zero_grads=True, dh_out=None, dc_out=None):
        """Record one step (forward, then backward with the gradients zeroed first) as a HIP graph."""
        backward = self.w.backward if backward is None else backward
        return F.StepGraph(self.sched, self.packed, self.table, self.leaf_rows, self.h_pool, self.c_pool,
                           self.roots, self.ws, self.ws_bytes, backward=backward, dh_roots=self.dh_roots,
                           dh_nodes=self.dh_nodes, grads=self.grads if backward else None, dh_out=dh_out,
                           dc_out=dc_out, zero_grads=zero_grads and backward)

    # ------------------------------------------------------------------ results
    def sched_arrays(self):
        if not hasattr(self, "_sa"):
            self._sa = self.sched.arrays()
        return self._sa

    def node_states(self):
        """h, c in node order as float64 [N, H]."""
        torch.cuda.synchronize()
        node_pos = self.sched_arrays()["node_pos"]
        h = self.h_pool.float().cpu().numpy()[:self.N, :self.H].astype(np.float64)
        c = self.c_pool.cpu().numpy()[:self.N, :self.H].astype(np.float64)
        return h[node_pos], c[node_pos]

    def weight_grads(self):
        torch.cuda.synchronize()
        out = []
        for t in self.grad_tensors:
            out.append({k: (None if x is None else x.cpu().numpy().astype(np.float64))
                        for k, x in zip(("W_in", "W_rec", "bias"), t)})
        dt = None if self.d_table is None else self.d_table.cpu().numpy()[:, :self.w.leaf_table.shape[1]].astype(np.float64)
        return out, dt


class TrainStep:
    """One training step of a workload through the C ABI (Section 3.5's setting: a class label on every node,
    softmax cross entropy on every node's state, Adam): zero the gradients, fold_forward,
    fold_loss_softmax_ce, fold_backward from the head's dh alone, fold_adam_step on every parameter tensor
    (the weights of every set, the biases, the leaf table if trained, the classifier), fold_pack_update.

    fp32 master copies of the weights are kept here; for bf16 workloads Adam also writes the bf16 weights
    that fold_pack_update packs.  The loss is the mean over the labelled nodes (scale = 1 / their count).

    dropout > 0 trains with recurrent dropout (Section 3.5): every step first draws a fresh mask on the GPU
    (fold_dropout_mask with counter = (node, unit block, step number), key = dropout_seed) and runs
    fold_forward_dropout / fold_backward_dropout with it."""

    def __init__(self, w: gen.Workload, labels: np.ndarray, num_classes: int, train_table: bool, seed: int = 0,
                 lr: float = 1e-3, beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8,
                 dropout: float = 0.0, dropout_seed: int = 0):
        self.dev = dev = DeviceRun(w)
        self.dropout = float(dropout)
        self.dropout_seed = int(dropout_seed)
        self.u_mask = (torch.zeros((max(dev.N, 1), dev.ld), dtype=torch.float32, device=dev.device)
                       if self.dropout > 0 else None)
        self.C = num_classes
        self.hyper = (lr, beta1, beta2, eps)
        self.t = 0
        rng = np.random.default_rng(seed)
        cuda = lambda a, dt=torch.float32: torch.from_numpy(np.ascontiguousarray(a)).to(dtype=dt, device=dev.device)
        self.labels = cuda(labels, torch.int32)
        self.scale = 1.0 / max(1, int((labels >= 0).sum()))
        self.W_cls = cuda((0.1 * rng.standard_normal((w.hidden, num_classes))).astype(np.float32))
        self.b_cls = torch.zeros(num_classes, dtype=torch.float32, device=dev.device)
        self.dW_cls = torch.zeros_like(self.W_cls)
        self.db_cls = torch.zeros_like(self.b_cls)
        self.node_loss = torch.zeros(max(dev.N, 1), dtype=torch.float32, device=dev.device)
        self.dh_nodes = torch.zeros((max(dev.N, 1), dev.ld), dtype=torch.float32, device=dev.device)
        self.loss_ws_bytes = F.fold_loss_workspace_size(dev.packed.handle, num_classes)
        self.loss_ws = torch.empty(self.loss_ws_bytes, dtype=torch.uint8, device=dev.device)
        dev.alloc_grads(train_table)
        dev.set_upstream(np.zeros_like(w.dh_roots))
        dev.dh_nodes = self.dh_nodes
        # (fp32 master, bf16 copy or None, gradient) of every trained tensor
        self.tensors = []
        for p, st, gt in zip(w.params, dev.set_tensors, dev.grad_tensors):
            if p.kind == gen.KIND_EMBED:
                continue
            for name, g in zip(("W_in", "W_rec", "bias"), gt):
                if g is None:
                    continue
                cur = st[name]
                if cur.dtype == torch.float32:
                    self.tensors.append((cur, None, g))
                else:
                    self.tensors.append((cur.float(), cur, g))
        if train_table:
            self.tensors.append((dev.table.float(), dev.table if dev.bf16 else None, dev.d_table))
            if not dev.bf16:
                self.tensors[-1] = (dev.table, None, dev.d_table)
        self.tensors += [(self.W_cls, None, self.dW_cls), (self.b_cls, None, self.db_cls)]
        self.moments = [(torch.zeros_like(m), torch.zeros_like(m)) for m, _, _ in self.tensors]

    def draw_mask(self):
        """The recurrent-dropout mask of step self.t into self.u_mask (pool order)."""
        F.fold_dropout_mask(self.dev.sched.handle, self.dev.H, self.dropout, self.dropout_seed, self.t, self.u_mask,
                            self.dev.stream)

    def gradients(self):
        """Zero the gradients, forward, head, backward (kernel launches only: capturable as a graph).  With
        dropout they read the mask that step() draws first."""
        dev = self.dev
        dev.zero_grads()
        self.dW_cls.zero_()
        self.db_cls.zero_()
        dev.forward(self.u_mask)
        F.fold_loss_softmax_ce(dev.sched.handle, dev.packed.handle, dev.h_pool, self.labels, self.C, self.W_cls,
                               self.b_cls, self.scale, self.node_loss, self.dh_nodes, self.dW_cls, self.db_cls,
                               self.loss_ws, self.loss_ws_bytes, dev.stream)
        dev.backward(u_mask=self.u_mask)

    def capture_gradients(self):
        """Record gradients() once as a graph (torch.cuda.CUDAGraph over the library's launches on the capture
        stream); step(graph=True) then replays it.  Adam, the re-pack and the mask draw stay outside: the step
        count enters each of them."""
        self.graph = torch.cuda.CUDAGraph()
        torch.cuda.synchronize()
        with torch.cuda.graph(self.graph):
            self.gradients()
        torch.cuda.synchronize()

    def step(self, graph: bool = False):
        dev = self.dev
        self.t += 1
        if self.u_mask is not None:
            self.draw_mask()
        if graph:
            self.graph.replay()
        else:
            self.gradients()
        lr, b1, b2, eps = self.hyper
        for (master, low, grad), (m, v) in zip(self.tensors, self.moments):
            F.fold_adam_step(master.numel(), master, low, grad, m, v, lr, b1, b2, eps, self.t, dev.stream)
        dev.packed.update(dev.set_tensors, dev.stream)
