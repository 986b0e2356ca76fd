"""Thin Python binding of the C ABI in ``include/fold.h`` (ctypes).

Argument marshalling only: every step of the hot path runs in the HIP library.
PyTorch provides device memory (``tensor.data_ptr()``) and streams
(``torch.cuda.current_stream().cuda_stream``).  If ``libfold.so`` is missing the
binding raises -- there is no fallback.

The functions keep the ABI's names:
    fold_schedule, fold_sched_get_info, fold_sched_free,
    fold_pack_params, fold_packed_free, fold_workspace_size,
    fold_forward, fold_backward, fold_row_ld, fold_last_error,
    fold_graph_create, fold_graph_launch, fold_graph_num_nodes, fold_graph_free
``Schedule`` / ``Packed`` / ``StepGraph`` wrap them for tensors.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, byref, c_int32, c_int64, c_size_t, c_void_p

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfold.so")

FOLD_OK = 0
ERRORS = {-1: "FOLD_E_INVALID", -2: "FOLD_E_OP", -3: "FOLD_E_ARITY", -4: "FOLD_E_CHILD",
          -5: "FOLD_E_INPUT", -6: "FOLD_E_CYCLE", -7: "FOLD_E_NOMEM", -8: "FOLD_E_DEVICE",
          -9: "FOLD_E_MISMATCH"}
FOLD_E_INVALID, FOLD_E_OP, FOLD_E_ARITY, FOLD_E_CHILD, FOLD_E_INPUT, FOLD_E_CYCLE = -1, -2, -3, -4, -5, -6
FOLD_E_NOMEM, FOLD_E_DEVICE, FOLD_E_MISMATCH = -7, -8, -9
FOLD_EMBED, FOLD_TREERNN, FOLD_TREELSTM, FOLD_LSTM, FOLD_PROJ = 0, 1, 2, 3, 4
FOLD_ATTN_SCORE, FOLD_ATTN_SUM, FOLD_ATTN_OUT = 5, 6, 7
FOLD_F32, FOLD_BF16 = 0, 1
GATES = {FOLD_EMBED: 0, FOLD_TREERNN: 1, FOLD_TREELSTM: 5, FOLD_LSTM: 4, FOLD_PROJ: 1,
         FOLD_ATTN_SCORE: 0, FOLD_ATTN_SUM: 0, FOLD_ATTN_OUT: 0}


class fold_op(ctypes.Structure):
    _fields_ = [("kind", c_int32), ("arity", c_int32), ("has_input", c_int32), ("param_set", c_int32)]


class fold_batch(ctypes.Structure):
    _fields_ = [("num_graphs", c_int32), ("num_nodes", c_int32), ("num_edges", c_int32),
                ("num_ops", c_int32), ("num_inputs", c_int32),
                ("graph_ptr", c_void_p), ("node_op", c_void_p), ("child_ptr", c_void_p),
                ("child_idx", c_void_p), ("node_input", c_void_p), ("ops", POINTER(fold_op))]


_I32P = c_void_p


class fold_sched_info(ctypes.Structure):
    _fields_ = [("num_nodes", c_int32), ("num_edges", c_int32), ("num_graphs", c_int32),
                ("num_ops", c_int32), ("num_levels", c_int32), ("num_groups", c_int32),
                ("num_roots", c_int32), ("max_parents", c_int32),
                ("depth", _I32P), ("node_pos", _I32P), ("pos_node", _I32P), ("level_ptr", _I32P),
                ("group_level", _I32P), ("group_op", _I32P), ("group_row_begin", _I32P),
                ("group_rows", _I32P), ("group_idx_off", _I32P), ("child_pos", _I32P),
                ("input_idx", _I32P), ("root_pos", _I32P),
                ("h_level_ptr", POINTER(c_int32)), ("h_group_level", POINTER(c_int32)),
                ("h_group_op", POINTER(c_int32)), ("h_group_row_begin", POINTER(c_int32)),
                ("h_group_rows", POINTER(c_int32)), ("h_group_idx_off", POINTER(c_int32)),
                ("group_child_base0", _I32P), ("group_child_base1", _I32P),
                ("h_group_child_base0", POINTER(c_int32)), ("h_group_child_base1", POINTER(c_int32))]


class fold_typed_op(ctypes.Structure):
    _fields_ = [("num_inputs", c_int32), ("num_outputs", c_int32), ("in_type", POINTER(c_int32)),
                ("out_type", POINTER(c_int32))]


class fold_typed_batch(ctypes.Structure):
    _fields_ = [("num_graphs", c_int32), ("num_nodes", c_int32), ("num_edges", c_int32), ("num_ops", c_int32),
                ("num_types", c_int32), ("graph_ptr", c_void_p), ("node_op", c_void_p), ("in_ptr", c_void_p),
                ("in_node", c_void_p), ("in_slot", c_void_p), ("ops", POINTER(fold_typed_op))]


class fold_typed_sched_info(ctypes.Structure):
    _fields_ = [("num_levels", c_int32), ("num_batches", c_int32), ("num_passes", c_int32),
                ("num_items", c_int32), ("num_gather", c_int32), ("num_ops", c_int32), ("num_types", c_int32),
                ("depth", _I32P), ("batch_depth", _I32P), ("batch_op", _I32P), ("batch_rows", _I32P),
                ("batch_gather_off", _I32P), ("batch_item_begin", _I32P), ("item_node", _I32P),
                ("gather", _I32P), ("pass_node", _I32P), ("pass_slot", _I32P), ("pass_depth", _I32P),
                ("state_size", _I32P), ("edge_index", _I32P),
                ("h_batch_depth", POINTER(c_int32)), ("h_batch_op", POINTER(c_int32)),
                ("h_batch_rows", POINTER(c_int32)), ("h_batch_gather_off", POINTER(c_int32)),
                ("h_state_size", POINTER(c_int32))]


class fold_param_set(ctypes.Structure):
    _fields_ = [("kind", c_int32), ("in_dim", c_int32), ("arity", c_int32),
                ("W_in", c_void_p), ("W_rec", c_void_p), ("bias", c_void_p)]


class fold_params(ctypes.Structure):
    _fields_ = [("dtype", c_int32), ("hidden", c_int32), ("num_sets", c_int32),
                ("sets", POINTER(fold_param_set))]


class fold_param_grads(ctypes.Structure):
    _fields_ = [("dW_in", c_void_p), ("dW_rec", c_void_p), ("dbias", c_void_p)]


class fold_grads(ctypes.Structure):
    _fields_ = [("num_sets", c_int32), ("sets", POINTER(fold_param_grads)), ("d_leaf_table", c_void_p)]


class fold_step_buffers(ctypes.Structure):
    _fields_ = [("leaf_table", c_void_p), ("leaf_rows", c_int64), ("h_pool", c_void_p), ("c_pool", c_void_p),
                ("roots_out", c_void_p), ("dh_roots", c_void_p), ("dh_nodes", c_void_p),
                ("grads", POINTER(fold_grads)), ("dh_out", c_void_p), ("dc_out", c_void_p),
                ("ws", c_void_p), ("ws_bytes", c_size_t)]


FOLD_STEP_BACKWARD, FOLD_STEP_ZERO_GRADS = 1, 2


class fold_kernel_stat(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 48), ("launches", c_int64), ("total_ms", ctypes.c_double),
                ("max_ms", ctypes.c_double)]


class fold_launch_time(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 48), ("group", c_int32), ("op", c_int32), ("ms", ctypes.c_double)]


class FoldError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERRORS.get(code, code)}: {msg}")
        self.code = code


EXPORTS = ["fold_schedule", "fold_sched_get_info", "fold_sched_free", "fold_pack_params",
           "fold_packed_free", "fold_row_ld", "fold_workspace_size", "fold_forward",
           "fold_backward", "fold_last_error", "fold_profile_enable", "fold_profile_read",
           "fold_profile_read_launches",
           "fold_probe_mfma", "fold_probe_mfma_random", "fold_probe_copy", "fold_graph_create", "fold_graph_launch",
           "fold_graph_num_nodes", "fold_graph_free", "fold_pack_update", "fold_loss_softmax_ce",
           "fold_loss_workspace_size", "fold_adam_step", "fold_forward_dropout", "fold_backward_dropout",
           "fold_dropout_mask", "fold_forward_noalloc", "fold_schedule_typed", "fold_typed_sched_get_info",
           "fold_typed_sched_free", "fold_level_launches"]

_lib = None


def lib():
    """Load libfold.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_1702_02181_amd.build_lib.build()")
    # torch first: its HIP runtime (same soname) is then the one the library's calls reach.  Loaded the other
    # way round, the process would map two HIP runtimes and the library's would see no device.
    import torch  # noqa: F401
    L = ctypes.CDLL(LIB_PATH)
    L.fold_last_error.restype = ctypes.c_char_p
    L.fold_last_error.argtypes = []
    L.fold_row_ld.restype = c_int32
    L.fold_row_ld.argtypes = [c_int32]
    L.fold_schedule.restype = c_int32
    L.fold_schedule.argtypes = [POINTER(fold_batch), c_void_p, POINTER(c_void_p)]
    L.fold_sched_get_info.restype = c_int32
    L.fold_sched_get_info.argtypes = [c_void_p, POINTER(fold_sched_info)]
    L.fold_sched_free.restype = c_int32
    L.fold_sched_free.argtypes = [c_void_p]
    L.fold_pack_params.restype = c_int32
    L.fold_pack_params.argtypes = [POINTER(fold_params), c_void_p, POINTER(c_void_p)]
    L.fold_packed_free.restype = c_int32
    L.fold_packed_free.argtypes = [c_void_p]
    L.fold_workspace_size.restype = c_int32
    L.fold_workspace_size.argtypes = [c_void_p, c_void_p, POINTER(c_size_t), POINTER(c_size_t)]
    L.fold_forward.restype = c_int32
    L.fold_forward.argtypes = [c_void_p, c_void_p, c_void_p, c_int64, c_void_p, c_void_p, c_void_p,
                               c_void_p, c_size_t, c_void_p]
    L.fold_backward.restype = c_int32
    L.fold_backward.argtypes = [c_void_p, c_void_p, c_void_p, c_int64, c_void_p, c_void_p, c_void_p,
                                c_void_p, POINTER(fold_grads), c_void_p, c_void_p, c_void_p, c_size_t,
                                c_void_p]
    L.fold_forward_dropout.restype = c_int32
    L.fold_forward_dropout.argtypes = [c_void_p, c_void_p, c_void_p, c_int64, c_void_p, c_void_p, c_void_p,
                                       c_void_p, c_void_p, c_size_t, c_void_p]
    L.fold_backward_dropout.restype = c_int32
    L.fold_backward_dropout.argtypes = [c_void_p, c_void_p, c_void_p, c_int64, c_void_p, c_void_p, c_void_p,
                                        c_void_p, c_void_p, POINTER(fold_grads), c_void_p, c_void_p, c_void_p,
                                        c_size_t, c_void_p]
    L.fold_level_launches.restype = c_int32
    L.fold_level_launches.argtypes = [c_int32]
    L.fold_schedule_typed.restype = c_int32
    L.fold_schedule_typed.argtypes = [POINTER(fold_typed_batch), c_void_p, POINTER(c_void_p)]
    L.fold_typed_sched_get_info.restype = c_int32
    L.fold_typed_sched_get_info.argtypes = [c_void_p, POINTER(fold_typed_sched_info)]
    L.fold_typed_sched_free.restype = c_int32
    L.fold_typed_sched_free.argtypes = [c_void_p]
    L.fold_forward_noalloc.restype = c_int32
    L.fold_forward_noalloc.argtypes = [c_void_p, c_void_p, c_void_p, c_int64, c_void_p, c_void_p, c_void_p, c_void_p]
    L.fold_dropout_mask.restype = c_int32
    L.fold_dropout_mask.argtypes = [c_void_p, c_int32, ctypes.c_double, ctypes.c_uint64, ctypes.c_uint64, c_void_p,
                                    c_void_p]
    L.fold_graph_create.restype = c_int32
    L.fold_graph_create.argtypes = [c_void_p, c_void_p, POINTER(fold_step_buffers), c_int32, POINTER(c_void_p)]
    L.fold_graph_launch.restype = c_int32
    L.fold_graph_launch.argtypes = [c_void_p, c_void_p]
    L.fold_graph_num_nodes.restype = c_int32
    L.fold_graph_num_nodes.argtypes = [c_void_p, POINTER(c_int32)]
    L.fold_graph_free.restype = c_int32
    L.fold_graph_free.argtypes = [c_void_p]
    L.fold_profile_enable.restype = c_int32
    L.fold_profile_enable.argtypes = [c_int32]
    L.fold_profile_read.restype = c_int32
    L.fold_profile_read.argtypes = [POINTER(fold_kernel_stat), c_int32, POINTER(c_int32)]
    L.fold_profile_read_launches.restype = c_int32
    L.fold_profile_read_launches.argtypes = [POINTER(fold_launch_time), c_int32, POINTER(c_int32)]
    L.fold_probe_mfma.restype = c_int32
    L.fold_probe_mfma.argtypes = [c_int32, c_void_p, POINTER(ctypes.c_double)]
    L.fold_probe_mfma_random.restype = c_int32
    L.fold_probe_mfma_random.argtypes = [c_int32, c_void_p, POINTER(ctypes.c_double)]
    L.fold_probe_copy.restype = c_int32
    L.fold_probe_copy.argtypes = [c_void_p, c_void_p, c_size_t, c_void_p, POINTER(ctypes.c_double)]
    L.fold_pack_update.restype = c_int32
    L.fold_pack_update.argtypes = [c_void_p, POINTER(fold_params), c_void_p]
    L.fold_loss_softmax_ce.restype = c_int32
    L.fold_loss_softmax_ce.argtypes = [c_void_p, c_void_p, c_void_p, c_void_p, c_int32, c_void_p, c_void_p,
                                       ctypes.c_float, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_size_t,
                                       c_void_p]
    L.fold_loss_workspace_size.restype = c_int32
    L.fold_loss_workspace_size.argtypes = [c_void_p, c_int32, POINTER(c_size_t)]
    L.fold_adam_step.restype = c_int32
    L.fold_adam_step.argtypes = [c_int64, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, ctypes.c_double,
                                 ctypes.c_double, ctypes.c_double, ctypes.c_double, c_int32, c_void_p]
    _lib = L
    return L


def _check(rc: int):
    if rc != FOLD_OK:
        raise FoldError(rc, lib().fold_last_error().decode())


def fold_last_error() -> str:
    return lib().fold_last_error().decode()


def fold_profile_enable(on: bool):
    _check(lib().fold_profile_enable(1 if on else 0))


def fold_profile_read() -> dict:
    """{kernel class: (launches, total_ms, max_ms)}; waits for the recorded events and clears them."""
    cap = 128
    arr = (fold_kernel_stat * cap)()
    n = c_int32()
    _check(lib().fold_profile_read(arr, cap, byref(n)))
    return {arr[i].name.decode(): (int(arr[i].launches), float(arr[i].total_ms), float(arr[i].max_ms))
            for i in range(min(n.value, cap))}


def fold_profile_read_launches() -> list:
    """[(kernel class, group, op, ms)] in launch order; waits for the recorded events and clears them."""
    n = c_int32()
    _check(lib().fold_profile_read_launches(None, 0, byref(n)))  # count only
    cap = n.value
    arr = (fold_launch_time * max(cap, 1))()
    _check(lib().fold_profile_read_launches(arr, cap, byref(n)) if cap else 0)
    return [(arr[i].name.decode(), int(arr[i].group), int(arr[i].op), float(arr[i].ms))
            for i in range(min(n.value, cap))]


def fold_probe_mfma(dtype: int, stream=None) -> float:
    t = ctypes.c_double()
    _check(lib().fold_probe_mfma(int(dtype), _stream(stream), byref(t)))
    return float(t.value)


def fold_probe_mfma_random(dtype: int, stream=None) -> float:
    t = ctypes.c_double()
    _check(lib().fold_probe_mfma_random(int(dtype), _stream(stream), byref(t)))
    return float(t.value)


def fold_probe_copy(dst, src, nbytes: int, stream=None) -> float:
    g = ctypes.c_double()
    _check(lib().fold_probe_copy(_ptr(dst), _ptr(src), int(nbytes), _stream(stream), byref(g)))
    return float(g.value)


def fold_row_ld(width: int) -> int:
    return int(lib().fold_row_ld(int(width)))


def _ptr(t):
    return None if t is None else c_void_p(t.data_ptr())


def _stream(stream=None):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return c_void_p(s.cuda_stream)


# ----------------------------------------------------------------------------- raw calls

def fold_schedule(batch: fold_batch, stream=None) -> c_void_p:
    h = c_void_p()
    _check(lib().fold_schedule(byref(batch), _stream(stream), byref(h)))
    return h


def fold_sched_get_info(handle) -> fold_sched_info:
    info = fold_sched_info()
    _check(lib().fold_sched_get_info(handle, byref(info)))
    return info


def fold_sched_free(handle):
    _check(lib().fold_sched_free(handle))


def fold_pack_params(params: fold_params, stream=None) -> c_void_p:
    h = c_void_p()
    _check(lib().fold_pack_params(byref(params), _stream(stream), byref(h)))
    return h


def fold_pack_update(handle, params: fold_params, stream=None):
    _check(lib().fold_pack_update(handle, byref(params), _stream(stream)))


def fold_loss_workspace_size(packed, num_classes) -> int:
    n = c_size_t()
    _check(lib().fold_loss_workspace_size(packed, int(num_classes), byref(n)))
    return int(n.value)


def fold_loss_softmax_ce(sched, packed, h_pool, labels, num_classes, W_cls, b_cls, scale, node_loss, dh_nodes,
                         dW_cls, db_cls, ws, ws_bytes, stream=None):
    _check(lib().fold_loss_softmax_ce(sched, packed, _ptr(h_pool), _ptr(labels), int(num_classes), _ptr(W_cls),
                                      _ptr(b_cls), float(scale), _ptr(node_loss), _ptr(dh_nodes), _ptr(dW_cls),
                                      _ptr(db_cls), _ptr(ws), int(ws_bytes), _stream(stream)))


def fold_adam_step(n, param, param_bf16, grad, m, v, lr, beta1, beta2, eps, step, stream=None):
    _check(lib().fold_adam_step(int(n), _ptr(param), _ptr(param_bf16), _ptr(grad), _ptr(m), _ptr(v), float(lr),
                                float(beta1), float(beta2), float(eps), int(step), _stream(stream)))


def fold_level_launches(on) -> bool:
    """Turn level launches on or off for later calls; returns the previous setting."""
    return bool(lib().fold_level_launches(1 if on else 0))


def fold_forward_noalloc(sched, packed, table, table_rows, h_pool, c_pool, roots, stream=None):
    _check(lib().fold_forward_noalloc(sched, packed, _ptr(table), int(table_rows), _ptr(h_pool), _ptr(c_pool),
                                      _ptr(roots), _stream(stream)))


def fold_dropout_mask(sched, hidden, p, seed, step, mask, stream=None):
    _check(lib().fold_dropout_mask(sched, int(hidden), float(p), int(seed) & (2 ** 64 - 1), int(step) & (2 ** 64 - 1),
                                   _ptr(mask), _stream(stream)))


def fold_packed_free(handle):
    _check(lib().fold_packed_free(handle))


def fold_workspace_size(sched, packed):
    f, b = c_size_t(), c_size_t()
    _check(lib().fold_workspace_size(sched, packed, byref(f), byref(b)))
    return int(f.value), int(b.value)


def fold_forward(sched, packed, leaf_table, leaf_rows, h_pool, c_pool, roots_out, ws, ws_bytes, stream=None):
    _check(lib().fold_forward(sched, packed, _ptr(leaf_table), int(leaf_rows), _ptr(h_pool), _ptr(c_pool),
                              _ptr(roots_out), _ptr(ws), int(ws_bytes), _stream(stream)))


def fold_backward(sched, packed, leaf_table, leaf_rows, h_pool, c_pool, dh_roots, dh_nodes, grads,
                  dh_out, dc_out, ws, ws_bytes, stream=None):
    _check(lib().fold_backward(sched, packed, _ptr(leaf_table), int(leaf_rows), _ptr(h_pool), _ptr(c_pool),
                               _ptr(dh_roots), _ptr(dh_nodes), None if grads is None else byref(grads),
                               _ptr(dh_out), _ptr(dc_out), _ptr(ws), int(ws_bytes), _stream(stream)))


def fold_forward_dropout(sched, packed, leaf_table, leaf_rows, h_pool, c_pool, roots_out, u_mask, ws, ws_bytes,
                         stream=None):
    _check(lib().fold_forward_dropout(sched, packed, _ptr(leaf_table), int(leaf_rows), _ptr(h_pool), _ptr(c_pool),
                                      _ptr(roots_out), _ptr(u_mask), _ptr(ws), int(ws_bytes), _stream(stream)))


def fold_backward_dropout(sched, packed, leaf_table, leaf_rows, h_pool, c_pool, u_mask, dh_roots, dh_nodes, grads,
                          dh_out, dc_out, ws, ws_bytes, stream=None):
    _check(lib().fold_backward_dropout(sched, packed, _ptr(leaf_table), int(leaf_rows), _ptr(h_pool), _ptr(c_pool),
                                       _ptr(u_mask), _ptr(dh_roots), _ptr(dh_nodes),
                                       None if grads is None else byref(grads), _ptr(dh_out), _ptr(dc_out), _ptr(ws),
                                       int(ws_bytes), _stream(stream)))


def fold_graph_create(sched, packed, buffers: fold_step_buffers, flags: int) -> c_void_p:
    h = c_void_p()
    _check(lib().fold_graph_create(sched, packed, byref(buffers), int(flags), byref(h)))
    return h


def fold_graph_launch(graph, stream=None):
    _check(lib().fold_graph_launch(graph, _stream(stream)))


def fold_graph_num_nodes(graph) -> int:
    n = c_int32()
    _check(lib().fold_graph_num_nodes(graph, byref(n)))
    return int(n.value)


def fold_graph_free(graph):
    _check(lib().fold_graph_free(graph))


# ----------------------------------------------------------------------------- tensor wrappers

def _dev_copy_to_host(ptr: int, count: int) -> np.ndarray:
    """Copy `count` int32 from a library-owned device array to host (the schedule call has synchronised)."""
    out = np.empty(count, dtype=np.int32)
    if count:
        rc = _hip().hipMemcpy(c_void_p(out.ctypes.data), c_void_p(ptr), c_size_t(4 * count), 2)
        if rc != 0:
            raise RuntimeError(f"hipMemcpy failed ({rc})")
    return out


_hiplib = None


def _hip():
    global _hiplib
    if _hiplib is None:
        _hiplib = ctypes.CDLL("libamdhip64.so")
        _hiplib.hipMemcpy.restype = ctypes.c_int
        _hiplib.hipMemcpy.argtypes = [c_void_p, c_void_p, c_size_t, ctypes.c_int]
    return _hiplib


class Schedule:
    """fold_schedule over int32 CUDA tensors; frees the handle when collected."""

    def __init__(self, graph_ptr, node_op, child_ptr, child_idx, node_input, ops, num_inputs, stream=None):
        self._keep = (graph_ptr, node_op, child_ptr, child_idx, node_input)
        self._ops = (fold_op * len(ops))(*[fold_op(*o) for o in ops])
        b = fold_batch()
        b.num_graphs = graph_ptr.numel() - 1
        b.num_nodes = node_op.numel()
        b.num_edges = child_idx.numel()
        b.num_ops = len(ops)
        b.num_inputs = int(num_inputs)
        b.graph_ptr, b.node_op, b.child_ptr = _ptr(graph_ptr), _ptr(node_op), _ptr(child_ptr)
        b.child_idx = _ptr(child_idx) if child_idx.numel() else c_void_p(graph_ptr.data_ptr())
        b.node_input = _ptr(node_input)
        b.ops = self._ops
        self.batch = b
        self.handle = fold_schedule(b, stream)
        self.info = fold_sched_get_info(self.handle)

    def __del__(self):
        h = getattr(self, "handle", None)
        if h is not None and h.value:
            try:
                fold_sched_free(h)
            except Exception:
                pass
            self.handle = None

    @property
    def num_levels(self):
        return self.info.num_levels

    def host_groups(self) -> dict:
        i = self.info
        ng = i.num_groups

        def arr(p, n):
            return np.ctypeslib.as_array(p, shape=(n,)).copy() if n else np.zeros(0, np.int32)
        return dict(level_ptr=arr(i.h_level_ptr, i.num_levels + 1), group_level=arr(i.h_group_level, ng),
                    group_op=arr(i.h_group_op, ng), group_row_begin=arr(i.h_group_row_begin, ng),
                    group_rows=arr(i.h_group_rows, ng), group_idx_off=arr(i.h_group_idx_off, ng),
                    group_child_base0=arr(i.h_group_child_base0, ng),
                    group_child_base1=arr(i.h_group_child_base1, ng))

    def arrays(self) -> dict:
        """Every schedule array, copied to host numpy (device arrays and the host group table)."""
        i = self.info
        n, e, ng, D, R = i.num_nodes, i.num_edges, i.num_groups, i.num_levels, i.num_roots
        out = dict(num_levels=D, num_groups=ng, num_roots=R, max_parents=i.max_parents)
        for name, cnt in (("depth", n), ("node_pos", n), ("pos_node", n), ("level_ptr", D + 1),
                          ("group_level", ng), ("group_op", ng), ("group_row_begin", ng), ("group_rows", ng),
                          ("group_idx_off", ng), ("child_pos", e), ("input_idx", n), ("root_pos", R),
                          ("group_child_base0", ng), ("group_child_base1", ng)):
            p = getattr(i, name)
            out[name] = _dev_copy_to_host(p, cnt) if p else np.zeros(0, np.int32)
        out["host"] = self.host_groups()
        return out


class TypedSchedule:
    """fold_schedule_typed over CUDA int32 tensors (the paper's form: typed per-depth states, pass-throughs).
    ops: list of (in_types, out_types)."""

    def __init__(self, graph_ptr, node_op, in_ptr, in_node, in_slot, ops, num_types, stream=None):
        self._keep = [graph_ptr, node_op, in_ptr, in_node, in_slot]
        self._types = []
        arr = (fold_typed_op * len(ops))()
        for k, (ins, outs) in enumerate(ops):
            a = (c_int32 * max(1, len(ins)))(*ins)
            b = (c_int32 * max(1, len(outs)))(*outs)
            self._types += [a, b]
            arr[k] = fold_typed_op(len(ins), len(outs), a, b)
        self._ops = arr
        bt = fold_typed_batch(int(graph_ptr.numel()) - 1, int(node_op.numel()), int(in_node.numel()), len(ops),
                              int(num_types), _ptr(graph_ptr), _ptr(node_op), _ptr(in_ptr), _ptr(in_node),
                              _ptr(in_slot), arr)
        h = c_void_p()
        _check(lib().fold_schedule_typed(ctypes.byref(bt), _stream(stream), ctypes.byref(h)))
        self.handle = h
        self.info = fold_typed_sched_info()
        _check(lib().fold_typed_sched_get_info(h, ctypes.byref(self.info)))
        self.num_nodes, self.num_edges = int(node_op.numel()), int(in_node.numel())

    def __del__(self):
        if getattr(self, "handle", None) is not None and _lib is not None:
            _lib.fold_typed_sched_free(self.handle)
            self.handle = None

    def arrays(self) -> dict:
        i = self.info
        D, T, nb, P, M, G = i.num_levels, i.num_types, i.num_batches, i.num_passes, i.num_items, i.num_gather

        def dev(name, n):
            p = getattr(i, name)
            return _dev_copy_to_host(p, n) if (p and n) else np.zeros(0, np.int32)

        def host(p, n):
            return np.ctypeslib.as_array(p, shape=(n,)).copy() if n else np.zeros(0, np.int32)
        out = dict(num_levels=D, num_batches=nb, num_passes=P, num_items=M, num_gather=G)
        for name, n in (("depth", self.num_nodes), ("batch_depth", nb), ("batch_op", nb), ("batch_rows", nb),
                        ("batch_gather_off", nb), ("batch_item_begin", nb), ("item_node", M), ("gather", G),
                        ("pass_node", P), ("pass_slot", P), ("pass_depth", P), ("state_size", (D + 1) * T),
                        ("edge_index", self.num_edges)):
            out[name] = dev(name, n)
        out["host"] = dict(batch_depth=host(i.h_batch_depth, nb), batch_op=host(i.h_batch_op, nb),
                           batch_rows=host(i.h_batch_rows, nb), batch_gather_off=host(i.h_batch_gather_off, nb),
                           state_size=host(i.h_state_size, (D + 1) * T))
        return out


class Packed:
    """fold_pack_params over CUDA tensors (weights of the params' dtype, fp32 biases)."""

    def __init__(self, dtype: int, hidden: int, sets, stream=None):
        # sets: list of dict(kind, in_dim, arity, W_in, W_rec, bias) with tensors or None
        self._keep = sets
        arr = (fold_param_set * len(sets))()
        for k, s in enumerate(sets):
            arr[k] = fold_param_set(s["kind"], s["in_dim"], s["arity"], _ptr(s.get("W_in")),
                                    _ptr(s.get("W_rec")), _ptr(s.get("bias")))
        self._sets = arr
        p = fold_params(dtype, hidden, len(sets), arr)
        self.handle = fold_pack_params(p, stream)
        self.dtype, self.hidden, self.num_sets = dtype, hidden, len(sets)

    def update(self, sets, stream=None):
        """fold_pack_update: re-pack new values of the same parameters (same shapes) in place."""
        arr = (fold_param_set * len(sets))()
        for k, s in enumerate(sets):
            arr[k] = fold_param_set(s["kind"], s["in_dim"], s["arity"], _ptr(s.get("W_in")),
                                    _ptr(s.get("W_rec")), _ptr(s.get("bias")))
        fold_pack_update(self.handle, fold_params(self.dtype, self.hidden, len(sets), arr), stream)
        self._keep, self._sets = sets, arr

    def __del__(self):
        h = getattr(self, "handle", None)
        if h is not None and h.value:
            try:
                fold_packed_free(h)
            except Exception:
                pass
            self.handle = None


def make_grads(sets_tensors, d_leaf_table=None) -> fold_grads:
    """sets_tensors: list of (dW_in, dW_rec, dbias) fp32 CUDA tensors or None."""
    arr = (fold_param_grads * len(sets_tensors))()
    for k, (a, b, c) in enumerate(sets_tensors):
        arr[k] = fold_param_grads(_ptr(a), _ptr(b), _ptr(c))
    g = fold_grads(len(sets_tensors), arr, _ptr(d_leaf_table))
    g._keep = (arr, sets_tensors, d_leaf_table)
    return g


class StepGraph:
    """fold_graph_create over CUDA tensors: one recorded forward (+ backward) step.  Keeps every
    tensor it was built on alive; frees the graph when collected."""

    def __init__(self, sched, packed, leaf_table, leaf_rows, h_pool, c_pool, roots_out, ws, ws_bytes,
                 backward=False, dh_roots=None, dh_nodes=None, grads=None, dh_out=None, dc_out=None,
                 zero_grads=False):
        self._keep = (sched, packed, leaf_table, h_pool, c_pool, roots_out, ws, dh_roots, dh_nodes, grads,
                      dh_out, dc_out)
        b = fold_step_buffers()
        b.leaf_table, b.leaf_rows = _ptr(leaf_table), int(leaf_rows)
        b.h_pool, b.c_pool, b.roots_out = _ptr(h_pool), _ptr(c_pool), _ptr(roots_out)
        b.dh_roots, b.dh_nodes = _ptr(dh_roots), _ptr(dh_nodes)
        b.grads = None if grads is None else ctypes.pointer(grads)
        b.dh_out, b.dc_out = _ptr(dh_out), _ptr(dc_out)
        b.ws, b.ws_bytes = _ptr(ws), int(ws_bytes)
        flags = (FOLD_STEP_BACKWARD if backward else 0) | (FOLD_STEP_ZERO_GRADS if zero_grads else 0)
        self.handle = fold_graph_create(sched.handle, packed.handle, b, flags)
        self.num_nodes = fold_graph_num_nodes(self.handle)

    def launch(self, stream=None):
        fold_graph_launch(self.handle, stream)

    def __del__(self):
        h = getattr(self, "handle", None)
        if h is not None and h.value:
            try:
                fold_graph_free(h)
            except Exception:
                pass
            self.handle = None
