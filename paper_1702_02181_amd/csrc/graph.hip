// One whole step of the level loop recorded as a HIP graph.
//
// Dynamic batching runs one loop iteration per depth (Section 2), so a batch of depth D costs a few
// kernel launches per (depth, op) group in each direction; for deep batches of narrow levels the
// host-side launch cost and the gaps between dependent launches, not the work, set the step time.
// fold_graph_create records the launches of fold_forward (and of fold_backward, optionally preceded
// by zeroing the gradients) once, on a private stream in capture mode, and instantiates the graph;
// fold_graph_launch then submits the whole step with one call.  Nothing is allocated, copied or
// synchronised by a launch.  The recorded step holds only kernel nodes (the gradients are zeroed by a
// fill kernel, not a memset node).

#include <hip/hip_runtime.h>

#include <string>
#include <vector>

#include "common.h"
#include "internal.h"

namespace fold {

namespace {

int gfail(int code, const std::string& msg) {
  set_error(msg);
  return code;
}

// leaves capture mode on every path out of the recording
struct CaptureGuard {
  bool on = true;
  ~CaptureGuard() {
    if (on) set_capturing(false);
  }
};

}  // namespace

struct GraphStep {
  hipGraph_t graph = nullptr;
  hipGraphExec_t exec = nullptr;
  int device = 0;
  int nodes = 0;
};

}  // namespace fold

struct fold_graph {
  fold::GraphStep g;
};

using namespace fold;

namespace {

void graph_destroy(fold_graph* h) {
  if (!h) return;
  if (h->g.exec) (void)hipGraphExecDestroy(h->g.exec);
  if (h->g.graph) (void)hipGraphDestroy(h->g.graph);
  delete h;
}

// zero every gradient tensor the step accumulates into (canonical layouts, fp32)
void record_zero_grads(const Sched& s, const Packed& p, const fold_grads* g, int64_t leaf_rows, hipStream_t st) {
  if (!g) return;
  for (int i = 0; i < g->num_sets && i < (int)p.sets.size(); ++i) {
    const PackedSet& ps = p.sets[i];
    const fold_param_grads& pg = g->sets[i];
    const size_t cols = (size_t)ps.G * p.H;
    if (ps.kind == FOLD_EMBED || ps.kind == FOLD_ATTN_SUM || ps.kind == FOLD_ATTN_OUT) continue;
    if (ps.kind == FOLD_ATTN_SCORE) {  // dw [H], db [1]
      launch_zero_f32(pg.dW_rec, (size_t)p.H, st);
      launch_zero_f32(pg.dbias, 1, st);
      continue;
    }
    launch_zero_f32(pg.dW_in, (size_t)ps.in_dim * cols, st);
    launch_zero_f32(pg.dW_rec, (size_t)ps.arity * p.H * cols, st);
    launch_zero_f32(pg.dbias, cols, st);
  }
  const int tw = leaf_table_width(s, p);
  if (g->d_leaf_table && tw > 0) launch_zero_f32(g->d_leaf_table, (size_t)leaf_rows * row_ld(tw), st);
}

}  // namespace

extern "C" {

int32_t fold_graph_create(const fold_sched* sh, const fold_packed* ph, const fold_step_buffers* b, int32_t flags,
                          fold_graph** out) {
  try {
    clear_error();
    if (!out) return gfail(FOLD_E_INVALID, "fold_graph_create: out is NULL");
    *out = nullptr;
    if (!sh || !ph || !b) return gfail(FOLD_E_INVALID, "fold_graph_create: NULL argument");
    if (flags & ~(FOLD_STEP_BACKWARD | FOLD_STEP_ZERO_GRADS))
      return gfail(FOLD_E_INVALID, "fold_graph_create: unknown flag");
    const bool bwd = (flags & FOLD_STEP_BACKWARD) != 0;
    const bool zero = (flags & FOLD_STEP_ZERO_GRADS) != 0;
    if (zero && !bwd) return gfail(FOLD_E_INVALID, "fold_graph_create: FOLD_STEP_ZERO_GRADS needs FOLD_STEP_BACKWARD");
    const Sched& s = sh->s;
    const Packed& p = ph->p;
    int rc = check_forward_args(s, p, b->leaf_table, b->leaf_rows, b->h_pool, b->c_pool, "fold_graph_create");
    if (rc != FOLD_OK) return rc;
    const WsLayout L = workspace_layout(s, p);
    if (b->ws_bytes < (bwd ? L.bwd_bytes : L.fwd_bytes) || (bwd && !b->ws))
      return gfail(FOLD_E_MISMATCH, "fold_graph_create: workspace too small");
    if (bwd) {
      rc = check_grads(p, b->grads, "fold_graph_create");
      if (rc != FOLD_OK) return rc;
    }
    int dev = 0;
    FOLD_HIP_CHECK(hipGetDevice(&dev));
    if (dev != s.device || dev != p.device)
      return gfail(FOLD_E_MISMATCH, "fold_graph_create: schedule, parameters and current device differ");

    hipStream_t cs = nullptr;
    FOLD_HIP_CHECK(hipStreamCreateWithFlags(&cs, hipStreamNonBlocking));  // default priority
    auto h = new fold_graph();
    h->g.device = dev;
    hipError_t e = hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal);
    if (e != hipSuccess) {
      (void)hipStreamDestroy(cs);
      graph_destroy(h);
      return gfail(FOLD_E_DEVICE, std::string("fold_graph_create: hipStreamBeginCapture: ") + hipGetErrorString(e));
    }
    int32_t rec = FOLD_OK;
    {
      CaptureGuard guard;
      set_capturing(true);
      if (zero) record_zero_grads(s, p, b->grads, b->leaf_rows, cs);
      rec = forward_impl(s, p, b->leaf_table, b->leaf_rows, b->h_pool, b->c_pool, b->roots_out, b->ws,
                         b->ws_bytes, cs);
      if (rec == FOLD_OK && bwd)
        rec = backward_impl(s, p, b->leaf_table, b->leaf_rows, b->h_pool, b->c_pool, b->dh_roots, b->dh_nodes,
                            b->grads, b->dh_out, b->dc_out, b->ws, b->ws_bytes, cs);
    }
    hipGraph_t graph = nullptr;
    e = hipStreamEndCapture(cs, &graph);
    (void)hipStreamDestroy(cs);
    h->g.graph = graph;
    if (rec != FOLD_OK) {
      graph_destroy(h);
      return rec;
    }
    if (e != hipSuccess || !graph) {
      graph_destroy(h);
      return gfail(FOLD_E_DEVICE, std::string("fold_graph_create: capture failed: ") + hipGetErrorString(e));
    }
    size_t nn = 0;
    (void)hipGraphGetNodes(graph, nullptr, &nn);
    h->g.nodes = (int)nn;
    e = hipGraphInstantiate(&h->g.exec, graph, nullptr, nullptr, 0);
    if (e != hipSuccess) {
      graph_destroy(h);
      return gfail(FOLD_E_DEVICE, std::string("fold_graph_create: hipGraphInstantiate: ") + hipGetErrorString(e));
    }
    *out = h;
    return FOLD_OK;
  } catch (const std::exception& ex) {
    return gfail(FOLD_E_INVALID, std::string("internal error: ") + ex.what());
  } catch (...) {
    return gfail(FOLD_E_INVALID, "internal error");
  }
}

int32_t fold_graph_launch(const fold_graph* h, hipStream_t st) {
  try {
    clear_error();
    if (!h || !h->g.exec) return gfail(FOLD_E_INVALID, "fold_graph_launch: NULL graph");
    int dev = 0;
    FOLD_HIP_CHECK(hipGetDevice(&dev));
    if (dev != h->g.device) return gfail(FOLD_E_MISMATCH, "fold_graph_launch: graph belongs to another device");
    FOLD_HIP_CHECK(hipGraphLaunch(h->g.exec, st));
    return FOLD_OK;
  } catch (...) {
    return gfail(FOLD_E_INVALID, "internal error");
  }
}

int32_t fold_graph_num_nodes(const fold_graph* h, int32_t* nodes) {
  if (!h || !nodes) return gfail(FOLD_E_INVALID, "fold_graph_num_nodes: NULL argument");
  *nodes = h->g.nodes;
  return FOLD_OK;
}

int32_t fold_graph_free(fold_graph* h) {
  try {
    graph_destroy(h);
    return FOLD_OK;
  } catch (...) {
    return gfail(FOLD_E_INVALID, "internal error");
  }
}

}  // extern "C"
