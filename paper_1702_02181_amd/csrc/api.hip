// C ABI of the library: argument checking, handles, workspace layout and the level loops that drive
// the kernels.  Every entry point catches everything, so no C++ exception leaves the library.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <atomic>
#include <cstring>
#include <exception>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"
#include "internal.h"

namespace fold {

namespace {
thread_local std::string g_last_error;
}

void set_error(const std::string& msg) { g_last_error = msg; }
void clear_error() { g_last_error.clear(); }

// ---------------------------------------------------------------- kernel timing

namespace {
std::atomic<bool> g_prof_on{false};
std::mutex g_prof_mu;
struct ProfRec {
  std::string name;
  int group, op;
  hipEvent_t a, b;
};
thread_local int g_tag_group = -1, g_tag_op = -1;
std::vector<ProfRec> g_prof_recs;
std::vector<hipEvent_t> g_prof_free;

hipEvent_t prof_event() {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (!g_prof_free.empty()) {
    hipEvent_t e = g_prof_free.back();
    g_prof_free.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}
}  // namespace

namespace {
thread_local bool g_capturing = false;  // launches are being recorded into a graph: no event pairs
std::atomic<bool> g_level_launches{true};  // narrow groups of one level in one launch
}

void set_capturing(bool on) { g_capturing = on; }

void prof_tag(int group, int op) {
  g_tag_group = group;
  g_tag_op = op;
}

ProfScope::ProfScope(const char* name, hipStream_t st) : name_(name), st_(st) {
  if (!g_prof_on.load(std::memory_order_relaxed) || g_capturing) return;
  hipEvent_t a = prof_event(), b = prof_event();
  if (!a || !b) return;
  start_ = a;
  stop_ = b;
  (void)hipEventRecord(a, st);
}

ProfScope::~ProfScope() {
  if (!start_) return;
  (void)hipEventRecord(static_cast<hipEvent_t>(stop_), st_);
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof_recs.push_back(
      {name_, g_tag_group, g_tag_op, static_cast<hipEvent_t>(start_), static_cast<hipEvent_t>(stop_)});
}

namespace {

int fail(int code, const std::string& msg) {
  set_error(msg);
  return code;
}

bool valid_kind(int k) { return k >= FOLD_EMBED && k <= FOLD_ATTN_OUT; }

// a Tree-LSTM operation without children: its cells run on the live gates only
bool is_tree_lstm_leaf(const fold_op& op) { return op.kind == FOLD_TREELSTM && op.arity == 0; }

// child slots an operation family's recurrent weights cover
int slots_of(int kind) {
  switch (kind) {
    case FOLD_TREERNN: return 2;
    case FOLD_TREELSTM: return 2;
    case FOLD_LSTM: return 1;
    case FOLD_PROJ: return 1;
    case FOLD_ATTN_SCORE: return 1;
    case FOLD_ATTN_SUM: return 2;
    case FOLD_ATTN_OUT: return 1;
    default: return 0;
  }
}

int check_op_table(const fold_op* ops, int n) {
  for (int i = 0; i < n; ++i) {
    const fold_op& o = ops[i];
    if (!valid_kind(o.kind) || o.param_set < 0 || (o.has_input != 0 && o.has_input != 1) || o.arity < 0)
      return fail(FOLD_E_INVALID, "op " + std::to_string(i) + ": bad kind, param_set or has_input");
    bool ok = true;
    switch (o.kind) {
      case FOLD_EMBED: ok = o.arity == 0 && o.has_input == 1; break;
      case FOLD_TREERNN: ok = o.arity == 2; break;
      case FOLD_TREELSTM: ok = (o.arity == 2) || (o.arity == 0 && o.has_input == 1); break;
      case FOLD_LSTM: ok = o.arity == 1; break;
      case FOLD_PROJ: ok = o.arity == 1 && o.has_input == 0; break;
      case FOLD_ATTN_SCORE:
      case FOLD_ATTN_SUM:
      case FOLD_ATTN_OUT: ok = o.arity == slots_of(o.kind) && o.has_input == 0; break;
      default: ok = false;
    }
    if (!ok) return fail(FOLD_E_INVALID, "op " + std::to_string(i) + ": arity / has_input not valid for its kind");
  }
  return FOLD_OK;
}

// the single leaf-table width every op with an input reads (0 if none); -1 if they disagree
int table_width(const Sched& s, const Packed& p) {
  int w = 0;
  for (const fold_op& o : s.ops) {
    if (!o.has_input) continue;
    const int d = p.sets[o.param_set].in_dim;
    if (w == 0) w = d;
    else if (w != d) return -1;
  }
  return w;
}

int check_compat(const Sched& s, const Packed& p) {
  for (size_t i = 0; i < s.ops.size(); ++i) {
    const fold_op& o = s.ops[i];
    if (o.param_set >= (int)p.sets.size())
      return fail(FOLD_E_MISMATCH, "op " + std::to_string(i) + " names a missing parameter set");
    const PackedSet& ps = p.sets[o.param_set];
    if (ps.kind != o.kind) return fail(FOLD_E_MISMATCH, "op " + std::to_string(i) + ": parameter set of another kind");
    if (o.arity > ps.arity) return fail(FOLD_E_MISMATCH, "op " + std::to_string(i) + ": more children than W_rec covers");
    if (o.has_input && ps.in_dim <= 0) return fail(FOLD_E_MISMATCH, "op " + std::to_string(i) + ": reads an input but has no W_in");
    if (o.kind == FOLD_EMBED && ps.in_dim != p.H) return fail(FOLD_E_MISMATCH, "embedding width must equal hidden");
  }
  if (table_width(s, p) < 0) return fail(FOLD_E_MISMATCH, "ops with an input disagree on its width");
  return FOLD_OK;
}

}  // namespace

int check_forward_args(const Sched& s, const Packed& p, const void* table, int64_t table_rows,
                       const void* h_pool, const void* c_pool, const char* who) {
  int rc = check_compat(s, p);
  if (rc != FOLD_OK) return rc;
  const std::string w(who);
  if (s.N > 0 && (!h_pool || !c_pool)) return fail(FOLD_E_INVALID, w + ": NULL pool");
  if (table_width(s, p) > 0 && s.N > 0) {
    if (!table) return fail(FOLD_E_INVALID, w + ": leaf table is NULL");
    if (table_rows < s.num_inputs) return fail(FOLD_E_MISMATCH, w + ": leaf table has fewer rows than the batch names");
  }
  return FOLD_OK;
}

int check_grads(const Packed& p, const fold_grads* grads, const char* who) {
  const std::string w(who);
  if (grads && grads->num_sets != (int)p.sets.size())
    return fail(FOLD_E_MISMATCH, w + ": gradient sets differ from parameter sets");
  if (grads && grads->num_sets > 0 && !grads->sets) return fail(FOLD_E_INVALID, w + ": NULL gradient sets");
  return FOLD_OK;
}

int leaf_table_width(const Sched& s, const Packed& p) { return table_width(s, p); }

WsLayout workspace_layout(const Sched& s, const Packed& p) {
  WsLayout w;
  int gmax = 1;
  for (const fold_op& o : s.ops) gmax = std::max(gmax, gates_of(o.kind));
  // a row's saved activations, then its dz: fp32 with fp32 parameters; fp16 activations and bf16 dz (G * HP
  // halves) with bf16 parameters
  w.gstride = p.dtype == FOLD_BF16 ? gmax * p.HP / 2 : gmax * p.HP;
  const size_t N = (size_t)s.N;
  auto al = [](size_t x) { return (x + 255) / 256 * 256; };
  w.gates_off = 0;
  w.gates_bytes = al(N * w.gstride * sizeof(float));
  // the forward's launches and the partial sums each K-split group needs (a level launch's groups side by side)
  size_t zp = 0, run = 0;
  int nb = 0, in_batch = 0, prev_level = -1;
  w.batch.assign(s.num_groups, -1);
  w.zoff.assign(s.num_groups, 0);
  w.zneed.assign(s.num_groups, 0);
  for (int g = 0; g < s.num_groups; ++g) {
    const fold_op& op = s.ops[s.h_op[g]];
    const bool new_level = s.h_level[g] != prev_level;
    prev_level = s.h_level[g];
    if (new_level || in_batch == kMaxMerge) {
      if (in_batch > 0) ++nb;
      in_batch = 0;
      run = 0;
    }
    if (op.kind == FOLD_EMBED || is_attn(op.kind) || op.param_set >= (int)p.sets.size()) {
      if (in_batch > 0) ++nb;
      in_batch = 0;
      run = 0;
      continue;
    }
    const PackedSet& ps = p.sets[op.param_set];
    const FwdPlan pl = fwd_plan(s.h_rows[g], p.HP, op.has_input ? ps.INP : 0, op.arity,
                                p.dtype == FOLD_BF16 ? 2 : 4, true);
    const size_t need = pl.ksplit > 1 ? (size_t)pl.ksplit * s.h_rows[g] * ps.G * p.HP : 0;
    w.zneed[g] = need;
    if (pl.wide) {
      if (in_batch > 0) ++nb;
      in_batch = 0;
      run = 0;
      zp = std::max(zp, need);
      continue;
    }
    w.batch[g] = nb;
    w.zoff[g] = run;
    run += need;
    ++in_batch;
    zp = std::max(zp, run);
  }
  w.zpart_off = w.gates_bytes;
  w.zpart_bytes = al(zp * sizeof(float));
  w.dh_off = w.zpart_off + w.zpart_bytes;
  w.dc_off = w.dh_off + al(N * p.ld * sizeof(float));
  w.acc_bytes = w.dc_off + al(N * p.ld * sizeof(float)) - w.dh_off;
  size_t part = 0, bpart = 0;
  for (int o = 0; o < s.num_ops; ++o) {
    const fold_op& op = s.ops[o];
    if (op.kind == FOLD_EMBED || op.param_set >= (int)p.sets.size()) continue;
    const int count = s.h_op_row_ptr[o + 1] - s.h_op_row_ptr[o];
    if (is_attn(op.kind)) {  // the scorer's chunked partial sums
      if (op.kind == FOLD_ATTN_SCORE) part = std::max(part, (size_t)attn_wgrad_chunks(count) * (p.HP + kPadK));
      continue;
    }
    const PackedSet& ps = p.sets[op.param_set];
    const int Nw = ps.G * p.HP;
    size_t nb = (size_t)((count + 511) / 512);
    if (op.arity > 0) {
      WgradSplit sp = wgrad_split(count, op.arity * p.HP, Nw, p.dtype);
      part = std::max(part, (size_t)sp.nchunk * op.arity * p.HP * Nw);
      nb = std::max(nb, (size_t)sp.bparts);
    }
    if (op.has_input && ps.INP > 0) {
      WgradSplit sp = wgrad_split(count, ps.INP, Nw, p.dtype);
      part = std::max(part, (size_t)sp.nchunk * ps.INP * Nw);
      nb = std::max(nb, (size_t)sp.bparts);
      // the leaf-table gradient's dz sums (fp32, and their bf16 copy) use the same region before the op's
      // weight gradients: at most one row per distinct leaf-table row of the op, over its dz columns
      const bool leaf = is_tree_lstm_leaf(op);
      const size_t U = (size_t)std::min(count, std::max(s.num_inputs, 0));
      const size_t Kb = (size_t)(leaf ? gates_of(kTreeLstmLeaf) : ps.G) * p.HP;
      part = std::max(part, p.dtype == FOLD_BF16 ? U * Kb + (U * Kb + 1) / 2 : U * Kb);
    }
    bpart = std::max(bpart, nb * Nw);
  }
  w.part_off = w.dh_off + w.acc_bytes;
  w.part_bytes = al(part * sizeof(float));
  w.bpart_off = w.part_off + w.part_bytes;
  w.bpart_bytes = al(bpart * sizeof(float));
  w.fwd_bytes = w.gates_bytes + w.zpart_bytes;
  w.bwd_bytes = w.bpart_off + w.bpart_bytes;
  return w;
}

// Packing kernels of every set into the handle's buffers (allocated to the parameters' shapes).
static void pack_launch(const Packed& P, const fold_params* prm, hipStream_t st) {
  for (int i = 0; i < prm->num_sets; ++i) {
    const fold_param_set& s = prm->sets[i];
    const PackedSet& ps = P.sets[i];
    if (s.kind == FOLD_EMBED || s.kind == FOLD_ATTN_SUM || s.kind == FOLD_ATTN_OUT) continue;
    if (s.kind == FOLD_ATTN_SCORE) {
      launch_pack_score(P.dtype, P.H, P.HP, s.W_rec, s.bias, ps.Wf, ps.bias, st);
      continue;
    }
    const size_t nf = (size_t)ps.Nf * ps.Kf;
    const size_t nbr = (size_t)s.arity * P.HP * ps.G * P.HP;
    const size_t nbi = (size_t)ps.INP * ps.G * P.HP;
    const int G = ps.G, gid = gate_code_identity(G);
    launch_pack(P.dtype, 0, G, G, gid, P.H, P.HP, s.in_dim, ps.INP, s.arity, ps.Kf, s.W_in, s.W_rec, nullptr, ps.Wf,
                nf, st);
    if (nbr)
      launch_pack(P.dtype, 1, G, G, gid, P.H, P.HP, s.in_dim, ps.INP, s.arity, ps.Kf, s.W_in, s.W_rec, nullptr,
                  ps.Wb_rec, nbr, st);
    if (nbi)
      launch_pack(P.dtype, 2, G, G, gid, P.H, P.HP, s.in_dim, ps.INP, s.arity, ps.Kf, s.W_in, s.W_rec, nullptr,
                  ps.Wb_in, nbi, st);
    launch_pack(P.dtype, 3, G, G, gid, P.H, P.HP, s.in_dim, ps.INP, s.arity, ps.Kf, nullptr, nullptr, s.bias,
                ps.bias, (size_t)G * P.HP, st);
    if (s.kind == FOLD_TREELSTM) {
      const int GL = gates_of(kTreeLstmLeaf);
      const size_t nfl = (size_t)GL * P.HP * ps.INP, nbl = (size_t)ps.INP * GL * P.HP;
      if (nfl)
        launch_pack(P.dtype, 0, GL, G, kTreeLstmLeafGates, P.H, P.HP, s.in_dim, ps.INP, 0, ps.INP, s.W_in, nullptr,
                    nullptr, ps.Wf_leaf, nfl, st);
      if (nbl)
        launch_pack(P.dtype, 2, GL, G, kTreeLstmLeafGates, P.H, P.HP, s.in_dim, ps.INP, 0, ps.INP, s.W_in, nullptr,
                    nullptr, ps.Wb_in_leaf, nbl, st);
      launch_pack(P.dtype, 3, GL, G, kTreeLstmLeafGates, P.H, P.HP, s.in_dim, ps.INP, 0, ps.INP, nullptr, nullptr,
                  s.bias, ps.bias_leaf, (size_t)GL * P.HP, st);
    }
  }
}

int32_t pack_impl(const fold_params* prm, hipStream_t st, fold_packed** out) {
  auto* h = new fold_packed();
  Packed& P = h->p;
  P.dtype = prm->dtype;
  P.H = prm->hidden;
  P.HP = round_up(prm->hidden, kPadK);
  P.ld = row_ld(prm->hidden);
  (void)hipGetDevice(&P.device);
  const size_t es = prm->dtype == FOLD_BF16 ? 2 : 4;
  auto bail = [&](int code, const std::string& m) {
    packed_destroy_impl(h);
    return fail(code, m);
  };
  auto dalloc = [&](size_t bytes, void** ptr) -> bool {
    *ptr = nullptr;
    if (bytes == 0) return true;
    if (hipMalloc(ptr, bytes) != hipSuccess) return false;
    P.allocs.push_back(*ptr);
    return true;
  };
  for (int i = 0; i < prm->num_sets; ++i) {
    const fold_param_set& s = prm->sets[i];
    PackedSet ps;
    ps.kind = s.kind;
    ps.in_dim = s.in_dim;
    ps.arity = s.arity;
    ps.G = gates_of(s.kind);
    if (s.kind == FOLD_ATTN_SCORE) {  // the scorer vector (HP entries) and its bias (64 floats, [0] = b)
      if (!dalloc((size_t)P.HP * es, &ps.Wf) ||
          !dalloc((size_t)kPadK * sizeof(float), reinterpret_cast<void**>(&ps.bias)))
        return bail(FOLD_E_NOMEM, "fold_pack_params: out of device memory");
    } else if (s.kind != FOLD_EMBED && !is_attn(s.kind)) {
      ps.INP = (s.in_dim > 0) ? round_up(s.in_dim, kPadK) : 0;
      ps.Kf = ps.INP + s.arity * P.HP;
      ps.Nf = ps.G * P.HP;
      const size_t nf = (size_t)ps.Nf * ps.Kf;
      const size_t nbr = (size_t)s.arity * P.HP * ps.G * P.HP;
      const size_t nbi = (size_t)ps.INP * ps.G * P.HP;
      if (!dalloc(nf * es, &ps.Wf) || !dalloc(nbr * es, &ps.Wb_rec) || !dalloc(nbi * es, &ps.Wb_in) ||
          !dalloc((size_t)ps.G * P.HP * sizeof(float), reinterpret_cast<void**>(&ps.bias)))
        return bail(FOLD_E_NOMEM, "fold_pack_params: out of device memory");
      if (s.kind == FOLD_TREELSTM) {
        // leaf operations of this set: the live gates only, input segment only
        const int GL = gates_of(kTreeLstmLeaf);
        const size_t nfl = (size_t)GL * P.HP * ps.INP, nbl = (size_t)ps.INP * GL * P.HP;
        if (!dalloc(nfl * es, &ps.Wf_leaf) || !dalloc(nbl * es, &ps.Wb_in_leaf) ||
            !dalloc((size_t)GL * P.HP * sizeof(float), reinterpret_cast<void**>(&ps.bias_leaf)))
          return bail(FOLD_E_NOMEM, "fold_pack_params: out of device memory");
      }
    }
    P.sets.push_back(ps);
  }
  pack_launch(P, prm, st);
  // the zero row spans the widest K any kernel reads: G * HP (dz rows), INP, HP
  size_t zw = (size_t)P.HP;
  for (const PackedSet& ps : P.sets) zw = std::max(zw, (size_t)std::max(ps.G * P.HP, ps.INP));
  P.zero_bytes = zw * sizeof(float);
  if (!dalloc(P.zero_bytes, &P.zero)) return bail(FOLD_E_NOMEM, "fold_pack_params: out of device memory");
  if (hipMemsetAsync(P.zero, 0, P.zero_bytes, st) != hipSuccess)
    return bail(FOLD_E_DEVICE, "fold_pack_params: device error while packing");
  if (hipGetLastError() != hipSuccess || hipStreamSynchronize(st) != hipSuccess)
    return bail(FOLD_E_DEVICE, "fold_pack_params: device error while packing");
  *out = h;
  return FOLD_OK;
}

void packed_destroy_impl(fold_packed* h) {
  if (!h) return;
  for (void* q : h->p.allocs) (void)hipFree(q);
  delete h;
}

// clears the launch tag when a pass returns, whichever way it returns
struct TagScope {
  ~TagScope() { prof_tag(-1, -1); }
};

// arguments of an attention group's launches (the forward's; the backward adds its accumulators)
static AttnArgs attn_args(const Sched& s, const Packed& p, int g, void* h_pool, float* c_pool) {
  const fold_op& op = s.ops[s.h_op[g]];
  const PackedSet& ps = p.sets[op.param_set];
  AttnArgs a{};
  a.rows = s.h_rows[g];
  a.row_begin = s.h_row_begin[g];
  a.idx_off = s.h_idx_off[g];
  a.H = p.H;
  a.ld = p.ld;
  a.h_pool = h_pool;
  a.c_pool = c_pool;
  a.child_pos = s.child_pos;
  a.child_one = s.child_one;
  a.w = ps.Wf;
  a.bias = ps.bias;
  return a;
}

int32_t forward_impl(const Sched& s, const Packed& p, const void* table, int64_t table_rows, void* h_pool,
                     float* c_pool, void* roots_out, void* ws, size_t ws_bytes, hipStream_t st, const float* u_mask,
                     float* zpart_direct, size_t zcap) {
  const WsLayout L = workspace_layout(s, p);
  TagScope tags;
  float* gates = nullptr;
  float* zpart = nullptr;
  if (zpart_direct) {
    zpart = zpart_direct;
  } else if (ws) {
    if (ws_bytes < L.fwd_bytes) return fail(FOLD_E_MISMATCH, "fold_forward: workspace too small");
    gates = reinterpret_cast<float*>(static_cast<char*>(ws) + L.gates_off);
    zpart = reinterpret_cast<float*>(static_cast<char*>(ws) + L.zpart_off);
  }
  const int tw = table_width(s, p);
  const int tld = row_ld(tw);
  // Consecutive narrow groups of one level run as one launch (level launches); a wide group or an
  // embedding launches alone.  Merged launches are tagged with their first group and op = -1 - n.
  int pend_g0 = -1, pend_batch = -1;
  std::vector<int> pend_kind;
  std::vector<FwdArgs> pend_args;
  auto flush = [&]() {
    const int n = (int)pend_args.size();
    if (n == 1) {
      prof_tag(pend_g0, s.h_op[pend_g0]);
      launch_cell_fwd(p.dtype, pend_kind[0], pend_args[0], st);
    } else if (n > 1) {
      prof_tag(pend_g0, -1 - n);
      launch_level_fwd(p.dtype, pend_kind.data(), pend_args.data(), n, st);
    }
    pend_kind.clear();
    pend_args.clear();
    pend_g0 = -1;
  };
  for (int g = 0; g < s.num_groups; ++g) {
    const fold_op& op = s.ops[s.h_op[g]];
    const PackedSet& ps = p.sets[op.param_set];
    if (L.batch[g] != pend_batch) flush();
    pend_batch = L.batch[g];
    if (op.kind == FOLD_EMBED) {
      flush();
      prof_tag(g, s.h_op[g]);
      launch_embed_fwd(p.dtype, s.h_rows[g], s.h_row_begin[g], p.H, p.ld, tld, table, s.input_idx, h_pool, c_pool, st);
      continue;
    }
    if (is_attn(op.kind)) {
      flush();
      prof_tag(g, s.h_op[g]);
      launch_attn_fwd(p.dtype, op.kind, attn_args(s, p, g, h_pool, c_pool), st);
      continue;
    }
    FwdArgs a;
    a.rows = s.h_rows[g];
    a.row_begin = s.h_row_begin[g];
    a.idx_off = s.h_idx_off[g];
    a.arity = op.arity;
    a.has_input = op.has_input;
    a.H = p.H;
    a.HP = p.HP;
    a.ld = p.ld;
    a.in_dim = ps.in_dim;
    a.INP = ps.INP;
    a.tld = tld;
    a.Kf = ps.Kf;
    a.table = table;
    a.h_pool = h_pool;
    a.c_pool = c_pool;
    a.child_pos = s.child_pos;
    a.input_idx = s.input_idx;
    a.Wf = ps.Wf;
    a.bias = ps.bias;
    a.gates = gates;
    a.gstride = L.gstride;
    a.u_mask = u_mask;
    a.zero = p.zero;
    a.zpart = zpart;
    a.zcap = zpart_direct ? zcap : 0;
    a.cbase[0] = op.arity > 0 ? s.h_cbase0[g] : -1;
    a.cbase[1] = op.arity > 1 ? s.h_cbase1[g] : -1;
    int kind = op.kind;
    if (is_tree_lstm_leaf(op)) {  // live gates only, input segment only
      kind = kTreeLstmLeaf;
      a.Wf = ps.Wf_leaf;
      a.Kf = ps.INP;
      a.bias = ps.bias_leaf;
    }
    if (L.batch[g] < 0 || !g_level_launches.load(std::memory_order_relaxed)) {  // launched alone
      flush();
      prof_tag(g, s.h_op[g]);
      launch_cell_fwd(p.dtype, kind, a, st);
      continue;
    }
    // a level launch's groups run at once: each takes its own part of the partial sums
    if (zpart && !zpart_direct) {
      a.zpart = zpart + L.zoff[g];
    } else if (zpart_direct) {
      // the fixed scratch: parts in proportion to their needs when the level's needs exceed it
      size_t total = 0;
      for (int h = g; h >= 0 && L.batch[h] == L.batch[g]; --h) total = std::max(total, L.zoff[h] + L.zneed[h]);
      for (int h = g + 1; h < s.num_groups && L.batch[h] == L.batch[g]; ++h)
        total = std::max(total, L.zoff[h] + L.zneed[h]);
      if (total > zcap) {
        a.zpart = zpart + (size_t)((double)L.zoff[g] * zcap / total);
        a.zcap = (size_t)((double)L.zneed[g] * zcap / total);
        if (a.zcap == 0) a.zcap = 1;  // a nonzero cap: the split is clamped to what fits (none)
      } else {
        a.zpart = zpart + L.zoff[g];
        a.zcap = std::max<size_t>(L.zneed[g], 1);
      }
    }
    if (pend_args.empty()) pend_g0 = g;
    pend_kind.push_back(kind);
    pend_args.push_back(a);
  }
  flush();
  prof_tag(-1, -1);
  if (roots_out) launch_roots(p.dtype, s.R, p.ld, s.root_pos, h_pool, roots_out, st);
  (void)table_rows;
  if (hipGetLastError() != hipSuccess) return fail(FOLD_E_DEVICE, "fold_forward: kernel launch failed");
  return FOLD_OK;
}

int32_t backward_impl(const Sched& s, const Packed& p, const void* table, int64_t table_rows, const void* h_pool,
                      const float* c_pool, const float* dh_roots, const float* dh_nodes, const fold_grads* grads,
                      float* dh_out, float* dc_out, void* ws, size_t ws_bytes, hipStream_t st,
                      const float* u_mask) {
  const WsLayout L = workspace_layout(s, p);
  if (!ws || ws_bytes < L.bwd_bytes) return fail(FOLD_E_MISMATCH, "fold_backward: workspace too small");
  const auto misaligned = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15) != 0; };
  if (misaligned(dh_roots) || misaligned(dh_nodes) || misaligned(dh_out) || misaligned(dc_out) || misaligned(ws))
    return fail(FOLD_E_INVALID, "fold_backward: dh_roots, dh_nodes, dh_out, dc_out and ws must be 16-byte aligned");
  TagScope tags;
  char* wsb = static_cast<char*>(ws);
  float* gates = reinterpret_cast<float*>(wsb + L.gates_off);
  float* dh = dh_out ? dh_out : reinterpret_cast<float*>(wsb + L.dh_off);
  float* dc = dc_out ? dc_out : reinterpret_cast<float*>(wsb + L.dc_off);
  float* part = reinterpret_cast<float*>(wsb + L.part_off);
  float* bpart = reinterpret_cast<float*>(wsb + L.bpart_off);
  const int tw = table_width(s, p);
  const int tld = row_ld(tw);
  float* d_table = grads ? grads->d_leaf_table : nullptr;

  // Rows of nodes with one parent edge are not initialised: that parent's backward stores them whole (dh
  // rows only when no per-node upstream gradient has to be added to).
  const int dh_fresh = dh_nodes == nullptr;
  const int esize = p.dtype == FOLD_BF16 ? 2 : 4;
  launch_bwd_init(s.N, s.R, p.ld, dh_nodes, dh_roots, s.root_pos, s.pos_npar, dh, dc, st);
  // Level by level from the top.  The groups of a level are independent (their children are at lower
  // levels), so all their cell backwards run first and then all their dz . W^T; narrow ones of a level run
  // as level launches (tagged with the first group of the span and op = -1 - span).
  for (int g_hi = s.num_groups; g_hi > 0;) {
    int g_lo = g_hi - 1;
    while (g_lo > 0 && s.h_level[g_lo - 1] == s.h_level[g_hi - 1]) --g_lo;
    std::vector<int> ckind;
    std::vector<BwdCellArgs> cargs;
    std::vector<DxArgs> dargs;
    std::vector<int> dgroup;
    std::vector<AttnArgs> attn;
    std::vector<int> attn_kind, attn_group;
    for (int g = g_lo; g < g_hi; ++g) {
      const fold_op& op = s.ops[s.h_op[g]];
      const PackedSet& ps = p.sets[op.param_set];
      BwdCellArgs b;
      b.rows = s.h_rows[g];
      b.row_begin = s.h_row_begin[g];
      b.idx_off = s.h_idx_off[g];
      b.arity = op.arity;
      b.H = p.H;
      b.HP = p.HP;
      b.ld = p.ld;
      b.gstride = L.gstride;
      b.c_pool = c_pool;
      b.gates = gates;
      b.u_mask = u_mask;
      b.dh = dh;
      b.dc = dc;
      b.child_pos = s.child_pos;
      b.input_idx = s.input_idx;
      b.child_one = s.child_one;
      b.d_table = d_table;
      b.tld = tld;
      b.dz_bf16 = p.dtype == FOLD_BF16;
      if (is_attn(op.kind)) {  // adds into the children itself: no dz . W^T
        AttnArgs at = attn_args(s, p, g, const_cast<void*>(h_pool), const_cast<float*>(c_pool));
        at.dh = dh;
        at.dc = dc;
        at.gates = gates;
        at.gstride = L.gstride;
        at.dh_fresh = dh_fresh;
        attn.push_back(at);
        attn_kind.push_back(op.kind);
        attn_group.push_back(g);
        continue;
      }
      // an embedding has no children and no dz: its only gradient, the leaf table's, is added per op below
      if (op.kind == FOLD_EMBED) continue;
      const bool leaf = is_tree_lstm_leaf(op);
      const int Kb = (leaf ? gates_of(kTreeLstmLeaf) : ps.G) * p.HP;
      // a dz . W^T whose K slices add into the children atomically needs their dh rows zeroed first
      b.zero_child_dh = dh_fresh && op.arity > 0 && dx_plan(b.rows, op.arity * p.HP, Kb, esize, true).ksplit > 1;
      ckind.push_back(leaf ? kTreeLstmLeaf : op.kind);
      cargs.push_back(b);
      DxArgs d;
      d.rows = b.rows;
      d.row_begin = b.row_begin;
      d.idx_off = b.idx_off;
      d.arity = op.arity;
      d.H = p.H;
      d.HP = p.HP;
      d.ld = p.ld;
      d.gstride = L.gstride;
      d.Kb = Kb;
      d.dz = gates;
      d.dh = dh;
      d.child_pos = s.child_pos;
      d.d_table = d_table;
      d.input_idx = s.input_idx;
      d.in_dim = ps.in_dim;
      d.tld = tld;
      d.child_one = s.child_one;
      d.dh_fresh = dh_fresh;
      d.can_split = 1;
      d.zero = p.zero;
      if (op.arity > 0) {
        d.mode = 0;
        d.Nb = op.arity * p.HP;
        d.Wb = ps.Wb_rec;
        dargs.push_back(d);
        dgroup.push_back(g);
      }
    }
    for (size_t k = 0; k < attn.size(); ++k) {
      prof_tag(attn_group[k], s.h_op[attn_group[k]]);
      launch_attn_bwd(p.dtype, attn_kind[k], attn[k], st);
    }
    // cell backwards: the level's groups in chunks of at most kMaxMerge
    const int merge = g_level_launches.load(std::memory_order_relaxed) ? kMaxMerge : 1;
    for (int k0 = 0; k0 < (int)cargs.size(); k0 += merge) {
      const int n = std::min<int>(merge, (int)cargs.size() - k0);
      if (n == 1) {
        prof_tag(g_lo + k0, s.h_op[g_lo + k0]);
        launch_cell_bwd(ckind[k0], cargs[k0], st);
      } else {
        prof_tag(g_lo + k0, -1 - n);
        launch_level_cbwd(ckind.data() + k0, cargs.data() + k0, n, st);
      }
    }
    // dz . W^T: wide calls alone, narrow ones merged
    std::vector<DxArgs> nargs;
    std::vector<int> ngroup;
    for (size_t k = 0; k < dargs.size(); ++k) {
      if (bwd_dx_is_narrow(p.dtype, dargs[k])) {
        nargs.push_back(dargs[k]);
        ngroup.push_back(dgroup[k]);
      } else {
        prof_tag(dgroup[k], s.h_op[dgroup[k]]);
        launch_bwd_dx(p.dtype, dargs[k], st);
      }
    }
    for (int k0 = 0; k0 < (int)nargs.size(); k0 += merge) {
      const int n = std::min<int>(merge, (int)nargs.size() - k0);
      if (n == 1) {
        prof_tag(ngroup[k0], s.h_op[ngroup[k0]]);
        launch_bwd_dx(p.dtype, nargs[k0], st);
      } else {
        const int span = ngroup[k0 + n - 1] - ngroup[k0] + 1;
        prof_tag(ngroup[k0], -1 - span);
        launch_level_dx(p.dtype, nargs.data() + k0, n, st);
      }
    }
    g_hi = g_lo;
  }
  // weight gradients: one deferred contraction per (op, input segment)
  if (grads) {
    for (int o = 0; o < s.num_ops; ++o) {
      const fold_op& op = s.ops[o];
      prof_tag(-1, o);
      const int count = s.h_op_row_ptr[o + 1] - s.h_op_row_ptr[o];
      if (count <= 0) continue;
      if (op.kind == FOLD_EMBED) {  // the leaf-table gradient: dh summed over each leaf-table row's rows
        if (d_table)
          launch_tok_table(s.tok_rows, s.tok_seg, s.tok_start, s.tok_row, s.h_op_row_ptr[o], count, dh, p.ld, p.H,
                           d_table, tld, st);
        continue;
      }
      const PackedSet& ps = p.sets[op.param_set];
      const fold_param_grads& pg = grads->sets[op.param_set];
      if (is_attn(op.kind)) {
        if (op.kind == FOLD_ATTN_SCORE)
          launch_attn_wgrad(p.dtype, s.op_rows + s.h_op_row_ptr[o], s.op_cpos + 2 * (size_t)s.h_op_row_ptr[o], count,
                            p.H, p.HP, p.ld, h_pool, gates, L.gstride, part, pg.dW_rec, pg.dbias, st);
        continue;
      }
      // dz columns: the canonical gate blocks, or the live ones of a Tree-LSTM leaf (dead columns get +0)
      const bool leaf = is_tree_lstm_leaf(op);
      const int Gz = leaf ? gates_of(kTreeLstmLeaf) : ps.G;
      const int gcode = leaf ? kTreeLstmLeafGates : gate_code_identity(ps.G);
      const int Nw = Gz * p.HP;
      const int off = s.h_op_row_ptr[o];
      if (op.has_input && d_table && ps.INP > 0) {
        // leaf-table gradient: dz summed over the op's rows of each leaf-table row (in the weight-gradient
        // region, before this op's weight gradients use it), then one dz . W_in^T row per distinct leaf-table row
        const int u0 = s.h_tok_ptr[o], U = s.h_tok_ptr[o + 1] - u0;
        const bool bf = p.dtype == FOLD_BF16;
        float* zsum = part;
        uint16_t* zbf = reinterpret_cast<uint16_t*>(part + (size_t)U * Nw);
        launch_tok_sum(p.dtype, s.tok_rows, s.tok_seg, s.tok_start, off, count, u0, U, gates, L.gstride, Nw, zsum,
                       zbf, st);
        DxArgs d{};
        d.rows = U;
        d.H = p.H;
        d.HP = p.HP;
        d.ld = p.ld;
        d.gstride = bf ? Nw / 2 : Nw;
        d.Kb = Nw;
        d.Nb = ps.INP;
        d.dz = bf ? reinterpret_cast<const float*>(zbf) : zsum;
        d.Wb = leaf ? ps.Wb_in_leaf : ps.Wb_in;
        d.zero = p.zero;
        d.mode = 1;
        d.d_table = d_table;
        d.input_idx = s.tok_row + u0;
        d.in_dim = ps.in_dim;
        d.tld = tld;
        d.can_split = 1;
        launch_bwd_dx(p.dtype, d, st, bf ? "tgrad.bf16" : "tgrad.f32");
      }
      WgArgs w;
      w.op_rows = s.op_rows + off;
      w.op_cpos = s.op_cpos + 2 * (size_t)off;
      w.op_inp = s.op_inp + off;
      w.count = count;
      w.H = p.H;
      w.HP = p.HP;
      w.ld = p.ld;
      w.in_dim = ps.in_dim;
      w.tld = tld;
      w.gstride = L.gstride;
      w.Nw = Nw;
      w.dz = gates;
      w.partial = part;
      w.zero = p.zero;
      bool bias_done = false;
      auto run = [&](int seg, int Kw, const void* src, float* dW) {
        w.seg = seg;
        w.Kw = Kw;
        w.src = src;
        const WgradSplit sp = wgrad_split(count, Kw, Nw, p.dtype);
        w.chunk = sp.chunk;
        w.nchunk = sp.nchunk;
        w.wide = sp.wide;
        w.bpart = (pg.dbias && !bias_done) ? bpart : nullptr;
        launch_wgrad(p.dtype, w, st);
        launch_wgrad_reduce(part, sp.nchunk, Kw, Nw, seg, p.H, p.HP, ps.in_dim, ps.G, gcode, dW, st);
        if (w.bpart) {
          launch_bias_reduce(bpart, sp.bparts, Nw, p.H, p.HP, gcode, pg.dbias, st);
          bias_done = true;
        }
      };
      if (op.arity > 0 && pg.dW_rec) run(1, op.arity * p.HP, h_pool, pg.dW_rec);
      if (op.has_input && ps.INP > 0 && pg.dW_in) run(0, ps.INP, table, pg.dW_in);
      if (pg.dbias && !bias_done) {
        const int chunk = 512, nchunk = (count + chunk - 1) / chunk;
        launch_bias_partial(w.op_rows, count, chunk, nchunk, gates, L.gstride, Nw, p.dtype == FOLD_BF16, bpart, st);
        launch_bias_reduce(bpart, nchunk, Nw, p.H, p.HP, gcode, pg.dbias, st);
      }
    }
  }
  (void)table_rows;
  if (hipGetLastError() != hipSuccess) return fail(FOLD_E_DEVICE, "fold_backward: kernel launch failed");
  return FOLD_OK;
}

// ---------------------------------------------------------------- allocation-free inference
// fold_forward_noalloc keeps the K-split partial sums of narrow levels in this array instead of a caller
// workspace.  Host code never uses its name as an address (on the host it is only a stand-in symbol): the
// device address of each GPU's copy is looked up once per device with hipGetSymbolAddress and kept.
constexpr size_t kScratchBytes = size_t(16) << 20;  // 16 MiB per GPU, held until the process ends
static __device__ __align__(256) float scratch[kScratchBytes / sizeof(float)];

namespace {
std::mutex g_scratch_mu;
std::map<int, float*> g_scratch_ptr;  // device ordinal -> device address of that device's scratch
}  // namespace

// the current device's scratch address (looked up on its first use), or nullptr with the error set
float* scratch_address() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    set_error("fold_forward_noalloc: no current device");
    return nullptr;
  }
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  auto it = g_scratch_ptr.find(dev);
  if (it != g_scratch_ptr.end()) return it->second;
  float* ptr = nullptr;
  if (hipGetSymbolAddress((void**)&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) {
    set_error("fold_forward_noalloc: hipGetSymbolAddress of the scratch array failed");
    return nullptr;
  }
  g_scratch_ptr[dev] = ptr;
  return ptr;
}

}  // namespace fold

using namespace fold;

#define FOLD_GUARD_BEGIN try {
#define FOLD_GUARD_END                                                      \
  }                                                                         \
  catch (const std::exception& e) {                                         \
    return fail(FOLD_E_INVALID, std::string("internal error: ") + e.what()); \
  }                                                                         \
  catch (...) {                                                             \
    return fail(FOLD_E_INVALID, "internal error");                          \
  }

namespace {
// Takes every profiling record made so far, waits for its events, returns the durations (ms) and
// recycles the events.  Returns FOLD_E_DEVICE if an event could not be read (its duration is 0).
int32_t drain_prof(std::vector<fold::ProfRec>& recs, std::vector<float>& ms) {
  {
    std::lock_guard<std::mutex> lk(fold::g_prof_mu);
    recs.swap(fold::g_prof_recs);
  }
  int32_t rc = FOLD_OK;
  ms.assign(recs.size(), 0.f);
  for (size_t i = 0; i < recs.size(); ++i) {
    if (hipEventSynchronize(recs[i].b) != hipSuccess || hipEventElapsedTime(&ms[i], recs[i].a, recs[i].b) != hipSuccess)
      rc = FOLD_E_DEVICE;
  }
  std::lock_guard<std::mutex> lk(fold::g_prof_mu);
  for (auto& r : recs) {
    fold::g_prof_free.push_back(r.a);
    fold::g_prof_free.push_back(r.b);
  }
  return rc;
}
}  // namespace

extern "C" {

const char* fold_last_error(void) { return fold::g_last_error.c_str(); }

int32_t fold_probe_mfma(int32_t dtype, hipStream_t st, double* tflops) {
  FOLD_GUARD_BEGIN
  clear_error();
  if (!tflops || (dtype != FOLD_F32 && dtype != FOLD_BF16)) return fail(FOLD_E_INVALID, "fold_probe_mfma: bad argument");
  return probe_mfma(dtype, false, st, tflops);
  FOLD_GUARD_END
}

int32_t fold_probe_mfma_random(int32_t dtype, hipStream_t st, double* tflops) {
  FOLD_GUARD_BEGIN
  clear_error();
  if (!tflops || (dtype != FOLD_F32 && dtype != FOLD_BF16)) return fail(FOLD_E_INVALID, "fold_probe_mfma_random: bad argument");
  return probe_mfma(dtype, true, st, tflops);
  FOLD_GUARD_END
}

int32_t fold_probe_copy(void* dst, const void* src, size_t bytes, hipStream_t st, double* gbs) {
  FOLD_GUARD_BEGIN
  clear_error();
  if (!dst || !src || !gbs || bytes < 16 || (bytes % 16) != 0 || (reinterpret_cast<uintptr_t>(dst) % 16) != 0 ||
      (reinterpret_cast<uintptr_t>(src) % 16) != 0)
    return fail(FOLD_E_INVALID, "fold_probe_copy: NULL, unaligned or non-multiple-of-16 buffers");
  return probe_copy(dst, src, bytes, st, gbs);
  FOLD_GUARD_END
}

int32_t fold_level_launches(int32_t on) {
  return fold::g_level_launches.exchange(on != 0) ? 1 : 0;
}

int32_t fold_profile_enable(int32_t on) {
  fold::g_prof_on.store(on != 0);
  return FOLD_OK;
}

int32_t fold_profile_read(fold_kernel_stat* out, int32_t capacity, int32_t* count) {
  FOLD_GUARD_BEGIN
  if (!count || (capacity > 0 && !out)) return fail(FOLD_E_INVALID, "fold_profile_read: NULL argument");
  std::vector<fold::ProfRec> recs;
  std::vector<float> dur;
  const int32_t rc = drain_prof(recs, dur);
  std::map<std::string, fold_kernel_stat> agg;
  std::vector<std::string> order;
  for (size_t i = 0; i < recs.size(); ++i) {
    const auto& r = recs[i];
    const float ms = dur[i];
    auto it = agg.find(r.name);
    if (it == agg.end()) {
      fold_kernel_stat st{};
      std::strncpy(st.name, r.name.c_str(), sizeof(st.name) - 1);
      it = agg.emplace(r.name, st).first;
      order.push_back(r.name);
    }
    it->second.launches += 1;
    it->second.total_ms += ms;
    it->second.max_ms = std::max(it->second.max_ms, (double)ms);
  }
  int32_t n = 0;
  for (const auto& name : order) {
    if (n < capacity) out[n] = agg[name];
    ++n;
  }
  *count = n;
  if (rc != FOLD_OK) return fail(rc, "fold_profile_read: event query failed");
  return FOLD_OK;
  FOLD_GUARD_END
}

int32_t fold_profile_read_launches(fold_launch_time* out, int32_t capacity, int32_t* count) {
  FOLD_GUARD_BEGIN
  if (!count || (capacity > 0 && !out)) return fail(FOLD_E_INVALID, "fold_profile_read_launches: NULL argument");
  if (capacity == 0) {  // count only; the records stay
    std::lock_guard<std::mutex> lk(fold::g_prof_mu);
    *count = (int32_t)fold::g_prof_recs.size();
    return FOLD_OK;
  }
  std::vector<fold::ProfRec> recs;
  std::vector<float> dur;
  const int32_t rc = drain_prof(recs, dur);
  const int32_t n = (int32_t)recs.size();
  for (int32_t i = 0; i < n && i < capacity; ++i) {
    fold_launch_time t{};
    std::strncpy(t.name, recs[i].name.c_str(), sizeof(t.name) - 1);
    t.group = recs[i].group;
    t.op = recs[i].op;
    t.ms = dur[i];
    out[i] = t;
  }
  *count = n;
  if (rc != FOLD_OK) return fail(rc, "fold_profile_read_launches: event query failed");
  return FOLD_OK;
  FOLD_GUARD_END
}

int32_t fold_row_ld(int32_t width) { return width < 0 ? 0 : row_ld(width); }

int32_t fold_schedule(const fold_batch* b, hipStream_t st, fold_sched** out) {
  FOLD_GUARD_BEGIN
  clear_error();
  if (!out) return fail(FOLD_E_INVALID, "fold_schedule: out is NULL");
  *out = nullptr;
  if (!b) return fail(FOLD_E_INVALID, "fold_schedule: batch is NULL");
  if (b->num_graphs < 0 || b->num_nodes < 0 || b->num_edges < 0 || b->num_ops < 1 || b->num_inputs < 0)
    return fail(FOLD_E_INVALID, "fold_schedule: negative count or no operations");
  if (!b->ops || !b->graph_ptr || (b->num_nodes > 0 && (!b->node_op || !b->child_ptr || !b->node_input)) ||
      (b->num_edges > 0 && !b->child_idx) || !b->child_ptr)
    return fail(FOLD_E_INVALID, "fold_schedule: NULL array");
  int rc = check_op_table(b->ops, b->num_ops);
  if (rc != FOLD_OK) return rc;
  return schedule_impl(b, st, out);
  FOLD_GUARD_END
}

int32_t fold_sched_get_info(const fold_sched* h, fold_sched_info* o) {
  FOLD_GUARD_BEGIN
  if (!h || !o) return fail(FOLD_E_INVALID, "fold_sched_get_info: NULL argument");
  const Sched& s = h->s;
  o->num_nodes = s.N;
  o->num_edges = s.E;
  o->num_graphs = s.G;
  o->num_ops = s.num_ops;
  o->num_levels = s.D;
  o->num_groups = s.num_groups;
  o->num_roots = s.R;
  o->max_parents = s.max_parents;
  o->depth = s.depth;
  o->node_pos = s.node_pos;
  o->pos_node = s.pos_node;
  o->level_ptr = s.level_ptr;
  o->group_level = s.g_level;
  o->group_op = s.g_op;
  o->group_row_begin = s.g_row_begin;
  o->group_rows = s.g_rows;
  o->group_idx_off = s.g_idx_off;
  o->child_pos = s.child_pos;
  o->input_idx = s.input_idx;
  o->root_pos = s.root_pos;
  o->group_child_base0 = s.g_cbase0;
  o->group_child_base1 = s.g_cbase1;
  o->h_group_child_base0 = s.h_cbase0.data();
  o->h_group_child_base1 = s.h_cbase1.data();
  o->h_level_ptr = s.h_level_ptr.data();
  o->h_group_level = s.h_level.data();
  o->h_group_op = s.h_op.data();
  o->h_group_row_begin = s.h_row_begin.data();
  o->h_group_rows = s.h_rows.data();
  o->h_group_idx_off = s.h_idx_off.data();
  return FOLD_OK;
  FOLD_GUARD_END
}

int32_t fold_sched_free(fold_sched* h) {
  FOLD_GUARD_BEGIN
  sched_destroy_impl(h);
  return FOLD_OK;
  FOLD_GUARD_END
}

int32_t fold_schedule_typed(const fold_typed_batch* b, hipStream_t st, fold_typed_sched** out) {
  FOLD_GUARD_BEGIN
  clear_error();
  if (!out) return fail(FOLD_E_INVALID, "fold_schedule_typed: out is NULL");
  *out = nullptr;
  if (!b) return fail(FOLD_E_INVALID, "fold_schedule_typed: batch is NULL");
  if (b->num_graphs < 0 || b->num_nodes < 0 || b->num_edges < 0)
    return fail(FOLD_E_INVALID, "fold_schedule_typed: negative count");
  if (!b->ops || !b->graph_ptr || !b->in_ptr || (b->num_nodes > 0 && !b->node_op) ||
      (b->num_edges > 0 && (!b->in_node || !b->in_slot)))
    return fail(FOLD_E_INVALID, "fold_schedule_typed: NULL array");
  return schedule_typed_impl(b, st, out);
  FOLD_GUARD_END
}

int32_t fold_typed_sched_get_info(const fold_typed_sched* h, fold_typed_sched_info* o) {
  FOLD_GUARD_BEGIN
  if (!h || !o) return fail(FOLD_E_INVALID, "fold_typed_sched_get_info: NULL argument");
  const TypedSched& s = h->t;
  o->num_levels = s.D;
  o->num_batches = s.nb;
  o->num_passes = s.P;
  o->num_items = s.M;
  o->num_gather = s.ngather;
  o->num_ops = s.K;
  o->num_types = s.T;
  o->depth = s.depth;
  o->batch_depth = s.batch_depth;
  o->batch_op = s.batch_op;
  o->batch_rows = s.batch_rows;
  o->batch_gather_off = s.batch_goff;
  o->batch_item_begin = s.batch_begin;
  o->item_node = s.item_node;
  o->gather = s.gather;
  o->pass_node = s.pass_node;
  o->pass_slot = s.pass_slot;
  o->pass_depth = s.pass_depth;
  o->state_size = s.state_size;
  o->edge_index = s.edge_index;
  o->h_batch_depth = s.h_depth_b.data();
  o->h_batch_op = s.h_op_b.data();
  o->h_batch_rows = s.h_rows_b.data();
  o->h_batch_gather_off = s.h_goff_b.data();
  o->h_state_size = s.h_state_size.data();
  return FOLD_OK;
  FOLD_GUARD_END
}

int32_t fold_typed_sched_free(fold_typed_sched* h) {
  FOLD_GUARD_BEGIN
  typed_sched_destroy_impl(h);
  return FOLD_OK;
  FOLD_GUARD_END
}

static int check_params(const fold_params* prm, const char* who) {
  const std::string w = std::string(who) + ": ";
  if (!prm || !prm->sets || prm->num_sets < 1) return fail(FOLD_E_INVALID, w + "no parameter sets");
  if (prm->dtype != FOLD_F32 && prm->dtype != FOLD_BF16) return fail(FOLD_E_INVALID, w + "bad dtype");
  if (prm->hidden < 1 || prm->hidden > kMaxHidden)
    return fail(FOLD_E_INVALID, w + "hidden must be in 1.." + std::to_string(kMaxHidden));
  for (int i = 0; i < prm->num_sets; ++i) {
    const fold_param_set& s = prm->sets[i];
    const std::string at = w + "set " + std::to_string(i) + ": ";
    if (!valid_kind(s.kind)) return fail(FOLD_E_INVALID, at + "bad kind");
    if (s.in_dim < 0) return fail(FOLD_E_INVALID, at + "negative in_dim");
    if (s.kind == FOLD_EMBED) {
      if (s.in_dim != prm->hidden) return fail(FOLD_E_INVALID, at + "embedding width must equal hidden");
      continue;
    }
    if (is_attn(s.kind)) {
      if (s.in_dim != 0 || s.arity != slots_of(s.kind))
        return fail(FOLD_E_INVALID, at + "attention sets have in_dim 0 and the kind's child slots");
      if (prm->hidden < 2) return fail(FOLD_E_INVALID, at + "attention needs hidden >= 2 (c holds m and s)");
      if (s.kind == FOLD_ATTN_SCORE && (!s.W_rec || !s.bias))
        return fail(FOLD_E_INVALID, at + "the scorer needs W_rec (w) and bias (b)");
      continue;
    }
    if (s.arity != slots_of(s.kind)) return fail(FOLD_E_INVALID, at + "arity must be the kind's child slots");
    if (!s.bias) return fail(FOLD_E_INVALID, at + "bias is NULL");
    if (s.in_dim > 0 && !s.W_in) return fail(FOLD_E_INVALID, at + "W_in is NULL");
    if (!s.W_rec) return fail(FOLD_E_INVALID, at + "W_rec is NULL");
    // the packing kernels index every packed matrix with 32-bit arithmetic
    const long long HP = round_up(prm->hidden, kPadK), INP = round_up(s.in_dim, kPadK);
    if ((long long)gates_of(s.kind) * HP * (INP + s.arity * HP) >= (1LL << 32))
      return fail(FOLD_E_INVALID, at + "too large: a packed weight matrix would hold 2^32 entries or more");
  }
  return FOLD_OK;
}

int32_t fold_pack_params(const fold_params* prm, hipStream_t st, fold_packed** out) {
  FOLD_GUARD_BEGIN
  clear_error();
  if (!out) return fail(FOLD_E_INVALID, "fold_pack_params: out is NULL");
  *out = nullptr;
  const int rc = check_params(prm, "fold_pack_params");
  if (rc != FOLD_OK) return rc;
  return pack_impl(prm, st, out);
  FOLD_GUARD_END
}

int32_t fold_pack_update(fold_packed* h, const fold_params* prm, hipStream_t st) {
  FOLD_GUARD_BEGIN
  clear_error();
  if (!h) return fail(FOLD_E_INVALID, "fold_pack_update: NULL handle");
  const int rc = check_params(prm, "fold_pack_update");
  if (rc != FOLD_OK) return rc;
  const Packed& P = h->p;
  if (prm->dtype != P.dtype || prm->hidden != P.H || prm->num_sets != (int)P.sets.size())
    return fail(FOLD_E_MISMATCH, "fold_pack_update: dtype, hidden or number of sets differ from the handle's");
  for (int i = 0; i < prm->num_sets; ++i) {
    const fold_param_set& s = prm->sets[i];
    const PackedSet& ps = P.sets[i];
    if (s.kind != ps.kind || s.in_dim != ps.in_dim || (s.kind != FOLD_EMBED && s.arity != ps.arity))
      return fail(FOLD_E_MISMATCH, "fold_pack_update: set " + std::to_string(i) + " differs in kind, in_dim or arity");
  }
  int dev = -1;
  FOLD_HIP_CHECK(hipGetDevice(&dev));
  if (dev != P.device) return fail(FOLD_E_MISMATCH, "fold_pack_update: the handle belongs to another device");
  pack_launch(P, prm, st);
  FOLD_HIP_CHECK(hipGetLastError());
  return FOLD_OK;
  FOLD_GUARD_END
}

static int check_loss_classes(const Packed& p, int num_classes, const char* who) {
  if (!loss_classes_supported(num_classes))
    return fail(FOLD_E_INVALID, std::string(who) + ": num_classes must be 2..8, 10, 16 or 32");
  if ((long long)p.H * num_classes > kLossMaxHC)
    return fail(FOLD_E_INVALID, std::string(who) + ": hidden * num_classes must be at most " +
                                    std::to_string(kLossMaxHC));
  return FOLD_OK;
}

int32_t fold_loss_workspace_size(const fold_packed* ph, int32_t num_classes, size_t* bytes) {
  FOLD_GUARD_BEGIN
  clear_error();
  if (!ph || !bytes) return fail(FOLD_E_INVALID, "fold_loss_workspace_size: NULL argument");
  const int rc = check_loss_classes(ph->p, num_classes, "fold_loss_workspace_size");
  if (rc != FOLD_OK) return rc;
  *bytes = loss_workspace_bytes(ph->p.H, num_classes);
  return FOLD_OK;
  FOLD_GUARD_END
}

int32_t fold_loss_softmax_ce(const fold_sched* sh, const fold_packed* ph, const void* h_pool, const int32_t* labels,
                             int32_t num_classes, const float* W_cls, const float* b_cls, float scale,
                             float* node_loss, float* dh_nodes, float* dW_cls, float* db_cls, void* ws,
                             size_t ws_bytes, hipStream_t st) {
  FOLD_GUARD_BEGIN
  clear_error();
  if (!sh || !ph) return fail(FOLD_E_INVALID, "fold_loss_softmax_ce: NULL handle");
  const Sched& s = sh->s;
  const Packed& p = ph->p;
  int rc = check_compat(s, p);
  if (rc != FOLD_OK) return rc;
  rc = check_loss_classes(p, num_classes, "fold_loss_softmax_ce");
  if (rc != FOLD_OK) return rc;
  if (!std::isfinite(scale)) return fail(FOLD_E_INVALID, "fold_loss_softmax_ce: scale is not finite");
  if (s.N == 0) return FOLD_OK;
  if (!h_pool || !labels || !W_cls || !b_cls || !node_loss || !dh_nodes || !dW_cls || !db_cls || !ws)
    return fail(FOLD_E_INVALID, "fold_loss_softmax_ce: NULL buffer");
  if (ws_bytes < loss_workspace_bytes(p.H, num_classes))
    return fail(FOLD_E_MISMATCH, "fold_loss_softmax_ce: workspace smaller than fold_loss_workspace_size");
  launch_loss_ce(p.dtype, s.N, p.H, p.ld, num_classes, h_pool, s.pos_node, labels, W_cls, b_cls, scale, node_loss,
                 dh_nodes, dW_cls, db_cls, static_cast<float*>(ws), st);
  FOLD_HIP_CHECK(hipGetLastError());
  return FOLD_OK;
  FOLD_GUARD_END
}

int32_t fold_adam_step(int64_t n, float* param, uint16_t* param_bf16, const float* grad, float* m, float* v,
                       double lr, double beta1, double beta2, double eps, int32_t step, hipStream_t st) {
  FOLD_GUARD_BEGIN
  clear_error();
  if (n < 0) return fail(FOLD_E_INVALID, "fold_adam_step: negative count");
  if (step < 1) return fail(FOLD_E_INVALID, "fold_adam_step: step counts from 1");
  if (!(beta1 >= 0.0 && beta1 < 1.0) || !(beta2 >= 0.0 && beta2 < 1.0) || !(eps >= 0.0) || !std::isfinite(lr))
    return fail(FOLD_E_INVALID, "fold_adam_step: need 0 <= beta1, beta2 < 1, eps >= 0 and a finite lr");
  if (n == 0) return FOLD_OK;
  if (!param || !grad || !m || !v) return fail(FOLD_E_INVALID, "fold_adam_step: NULL buffer");
  // the bias corrections folded into the step size, in double
  const double lr_t = lr * std::sqrt(1.0 - std::pow(beta2, step)) / (1.0 - std::pow(beta1, step));
  launch_adam((size_t)n, param, param_bf16, grad, m, v, beta1, beta2, lr_t, eps, st);
  FOLD_HIP_CHECK(hipGetLastError());
  return FOLD_OK;
  FOLD_GUARD_END
}

int32_t fold_dropout_mask(const fold_sched* sh, int32_t hidden, double p, uint64_t seed, uint64_t step, float* mask,
                          hipStream_t st) {
  FOLD_GUARD_BEGIN
  clear_error();
  if (!sh) return fail(FOLD_E_INVALID, "fold_dropout_mask: NULL schedule");
  if (hidden < 1 || hidden > kMaxHidden) return fail(FOLD_E_INVALID, "fold_dropout_mask: hidden size out of range");
  if (!(p >= 0.0 && p < 1.0)) return fail(FOLD_E_INVALID, "fold_dropout_mask: need 0 <= p < 1");
  const Sched& s = sh->s;
  if (s.N == 0) return FOLD_OK;
  if (!mask) return fail(FOLD_E_INVALID, "fold_dropout_mask: NULL mask");
  if (reinterpret_cast<uintptr_t>(mask) & 15)
    return fail(FOLD_E_INVALID, "fold_dropout_mask: mask must be 16-byte aligned");
  // drop where the word is below floor(p 2^32); kept units carry 1 / (1 - p) (inverted dropout)
  const double t = std::min(std::floor(p * 4294967296.0), 4294967295.0);
  const float scale = (float)(1.0 / (1.0 - p));
  launch_dropout_mask(s.pos_node, s.N, hidden, row_ld(hidden), (unsigned)t, scale, (unsigned long long)seed,
                      (unsigned long long)step, mask, st);
  FOLD_HIP_CHECK(hipGetLastError());
  return FOLD_OK;
  FOLD_GUARD_END
}

int32_t fold_packed_free(fold_packed* h) {
  FOLD_GUARD_BEGIN
  packed_destroy_impl(h);
  return FOLD_OK;
  FOLD_GUARD_END
}

int32_t fold_workspace_size(const fold_sched* sh, const fold_packed* ph, size_t* fwd_bytes, size_t* bwd_bytes) {
  FOLD_GUARD_BEGIN
  if (!sh || !ph) return fail(FOLD_E_INVALID, "fold_workspace_size: NULL handle");
  int rc = check_compat(sh->s, ph->p);
  if (rc != FOLD_OK) return rc;
  WsLayout L = workspace_layout(sh->s, ph->p);
  if (fwd_bytes) *fwd_bytes = L.fwd_bytes;
  if (bwd_bytes) *bwd_bytes = L.bwd_bytes;
  return FOLD_OK;
  FOLD_GUARD_END
}

int32_t fold_forward(const fold_sched* sh, const fold_packed* ph, const void* table, int64_t table_rows,
                     void* h_pool, float* c_pool, void* roots_out, void* ws, size_t ws_bytes, hipStream_t st) {
  FOLD_GUARD_BEGIN
  clear_error();
  if (!sh || !ph) return fail(FOLD_E_INVALID, "fold_forward: NULL handle");
  const Sched& s = sh->s;
  const Packed& p = ph->p;
  int rc = check_forward_args(s, p, table, table_rows, h_pool, c_pool, "fold_forward");
  if (rc != FOLD_OK) return rc;
  return forward_impl(s, p, table, table_rows, h_pool, c_pool, roots_out, ws, ws_bytes, st);
  FOLD_GUARD_END
}

int32_t fold_forward_noalloc(const fold_sched* sh, const fold_packed* ph, const void* table, int64_t table_rows,
                             void* h_pool, float* c_pool, void* roots_out, hipStream_t st) {
  FOLD_GUARD_BEGIN
  clear_error();
  if (!sh || !ph) return fail(FOLD_E_INVALID, "fold_forward_noalloc: NULL handle");
  const Sched& s = sh->s;
  const Packed& p = ph->p;
  int rc = check_forward_args(s, p, table, table_rows, h_pool, c_pool, "fold_forward_noalloc");
  if (rc != FOLD_OK) return rc;
  int dev = 0;
  FOLD_HIP_CHECK(hipGetDevice(&dev));
  if (dev != s.device || dev != p.device)
    return fail(FOLD_E_MISMATCH, "fold_forward_noalloc: the schedule and parameters belong to another device "
                                 "than the current one");
  float* zp = scratch_address();
  if (!zp) return FOLD_E_DEVICE;
  return forward_impl(s, p, table, table_rows, h_pool, c_pool, roots_out, nullptr, 0, st, nullptr, zp,
                      kScratchBytes / sizeof(float));
  FOLD_GUARD_END
}

int32_t fold_backward(const fold_sched* sh, const fold_packed* ph, const void* table, int64_t table_rows,
                      const void* h_pool, const float* c_pool, const float* dh_roots, const float* dh_nodes,
                      const fold_grads* grads, float* dh_out, float* dc_out, void* ws, size_t ws_bytes,
                      hipStream_t st) {
  FOLD_GUARD_BEGIN
  clear_error();
  if (!sh || !ph) return fail(FOLD_E_INVALID, "fold_backward: NULL handle");
  const Sched& s = sh->s;
  const Packed& p = ph->p;
  int rc = check_forward_args(s, p, table, table_rows, h_pool, c_pool, "fold_backward");
  if (rc != FOLD_OK) return rc;
  rc = check_grads(p, grads, "fold_backward");
  if (rc != FOLD_OK) return rc;
  return backward_impl(s, p, table, table_rows, h_pool, c_pool, dh_roots, dh_nodes, grads, dh_out, dc_out, ws,
                       ws_bytes, st);
  FOLD_GUARD_END
}

int32_t fold_forward_dropout(const fold_sched* sh, const fold_packed* ph, const void* table, int64_t table_rows,
                             void* h_pool, float* c_pool, void* roots_out, const float* u_mask, void* ws,
                             size_t ws_bytes, hipStream_t st) {
  FOLD_GUARD_BEGIN
  clear_error();
  if (!sh || !ph) return fail(FOLD_E_INVALID, "fold_forward_dropout: NULL handle");
  if (!u_mask) return fail(FOLD_E_INVALID, "fold_forward_dropout: u_mask is NULL");
  const Sched& s = sh->s;
  const Packed& p = ph->p;
  int rc = check_forward_args(s, p, table, table_rows, h_pool, c_pool, "fold_forward_dropout");
  if (rc != FOLD_OK) return rc;
  return forward_impl(s, p, table, table_rows, h_pool, c_pool, roots_out, ws, ws_bytes, st, u_mask);
  FOLD_GUARD_END
}

int32_t fold_backward_dropout(const fold_sched* sh, const fold_packed* ph, const void* table, int64_t table_rows,
                              const void* h_pool, const float* c_pool, const float* u_mask, const float* dh_roots,
                              const float* dh_nodes, const fold_grads* grads, float* dh_out, float* dc_out, void* ws,
                              size_t ws_bytes, hipStream_t st) {
  FOLD_GUARD_BEGIN
  clear_error();
  if (!sh || !ph) return fail(FOLD_E_INVALID, "fold_backward_dropout: NULL handle");
  if (!u_mask) return fail(FOLD_E_INVALID, "fold_backward_dropout: u_mask is NULL");
  const Sched& s = sh->s;
  const Packed& p = ph->p;
  int rc = check_forward_args(s, p, table, table_rows, h_pool, c_pool, "fold_backward_dropout");
  if (rc != FOLD_OK) return rc;
  rc = check_grads(p, grads, "fold_backward_dropout");
  if (rc != FOLD_OK) return rc;
  return backward_impl(s, p, table, table_rows, h_pool, c_pool, dh_roots, dh_nodes, grads, dh_out, dc_out, ws,
                       ws_bytes, st, u_mask);
  FOLD_GUARD_END
}

}  // extern "C"
