// Host-side entry points between the library's translation units.
#pragma once

#include <algorithm>

#include "common.h"

namespace fold {

int32_t schedule_impl(const fold_batch* b, hipStream_t st, fold_sched** out);
void sched_destroy_impl(fold_sched* h);
int32_t schedule_typed_impl(const fold_typed_batch* b, hipStream_t st, fold_typed_sched** out);
void typed_sched_destroy_impl(fold_typed_sched* h);

int32_t pack_impl(const fold_params* p, hipStream_t st, fold_packed** out);
void packed_destroy_impl(fold_packed* h);

// Workspace layout shared by the forward and backward passes.
constexpr int kMaxMerge = 4;  // groups of one level in one launch

struct WsLayout {
  int gstride = 0;           // floats per pool row of saved gates / dz: Gmax * HP (fp32), Gmax * HP / 2 (bf16)
  size_t gates_off = 0, gates_bytes = 0;
  size_t zpart_off = 0, zpart_bytes = 0;  // K-split partial sums of narrow forward levels
  size_t dh_off = 0, dc_off = 0, acc_bytes = 0;
  size_t part_off = 0, part_bytes = 0;   // weight-gradient partial tiles
  size_t bpart_off = 0, bpart_bytes = 0; // bias partial sums
  size_t fwd_bytes = 0, bwd_bytes = 0;
  // The forward's launches: batch[g] = the level launch group g belongs to (consecutive narrow groups of one
  // level, at most kMaxMerge to a launch), or -1 for a group launched alone (an embedding, a wide group).
  // Groups of one level launch run at once, so each has its own part of the K-split partial sums: zoff[g]
  // (floats from the region's start) and zneed[g] (floats, 0 when it does not split).
  std::vector<int> batch;
  std::vector<size_t> zoff, zneed;
};
WsLayout workspace_layout(const Sched& s, const Packed& p);

// Weight-gradient work split: rows of one op reduced in `nchunk` chunks of `chunk` rows.
struct WgradSplit {
  int nchunk = 0, chunk = 0;
  int bparts = 0;     // rows of bias partial sums the launch writes
  bool wide = false;  // 256 x 256 tiles (bf16, many rows)
};
WgradSplit wgrad_split(int count, int Kw, int Nw, int dtype);

// Argument checks shared by fold_forward, fold_backward and fold_graph_create (set the error text).
int check_forward_args(const Sched& s, const Packed& p, const void* table, int64_t table_rows,
                       const void* h_pool, const void* c_pool, const char* who);
int check_grads(const Packed& p, const fold_grads* grads, const char* who);
int leaf_table_width(const Sched& s, const Packed& p);
// While set on this thread, kernel launchers record no profiling events (stream capture in progress).
void set_capturing(bool on);

// zpart_direct: K-split partial sums go there (at most zcap floats) and nothing is saved for the backward;
// ws is then ignored
int32_t forward_impl(const Sched& s, const Packed& p, const void* table, int64_t table_rows, void* h_pool,
                     float* c_pool, void* roots_out, void* ws, size_t ws_bytes, hipStream_t st,
                     const float* u_mask = nullptr, float* zpart_direct = nullptr, size_t zcap = 0);
int32_t backward_impl(const Sched& s, const Packed& p, const void* table, int64_t table_rows,
                      const void* h_pool, const float* c_pool, const float* dh_roots, const float* dh_nodes,
                      const fold_grads* grads, float* dh_out, float* dc_out, void* ws, size_t ws_bytes,
                      hipStream_t st, const float* u_mask = nullptr);

// ---- kernel launchers (cells.hip) ----
struct FwdArgs {
  int rows, row_begin, idx_off, arity, has_input;
  int H, HP, ld;
  int in_dim, INP, tld;
  int Kf;
  const void* table;
  void* h_pool;
  float* c_pool;
  const int* child_pos;
  const int* input_idx;
  const void* Wf;
  const float* bias;
  float* gates;
  int gstride;
  const void* zero;  // a zero row at least as wide as any K the kernels read (16-byte aligned)
  float* zpart;  // workspace for K-split partial sums, or NULL (no split)
  size_t zcap = 0;  // floats zpart holds (0: as many as the plan needs); a level whose split needs more
                    // splits into fewer slices
  int ksplit;    // set by the launcher
  int map;         // set by the launcher: workgroup order over the XCDs (kMapRows, kMapCols, kMapOwnCols)
  const float* u_mask = nullptr;  // recurrent dropout: [N, ld] fp32 multiplier of u in pool order, or NULL
  int cbase[2] = {-1, -1};  // child slot k's rows are cbase[k] + row (static-graph layout), or -1: child_pos
};
// pool row of child slot k of group row `row` (-1: the zero state)
__device__ __forceinline__ int fwd_child(const FwdArgs& a, int row, int k) {
  // a select, not a[k]: k may differ between lanes, and an index into a struct held in registers (the merged
  // level launches copy their group's arguments) would move the struct to scratch memory
  const int cb = k == 0 ? a.cbase[0] : a.cbase[1];
  return cb >= 0 ? cb + row : a.child_pos[a.idx_off + row * a.arity + k];
}
void launch_cell_fwd(int dtype, int kind, const FwdArgs& a, hipStream_t st);
// The narrow groups of one level (at most kMaxMerge, every one narrow by fwd_plan) as one launch, plus one for
// their K-split epilogues; kinds as for launch_cell_fwd.
void launch_level_fwd(int dtype, const int* kinds, const FwdArgs* args, int n, hipStream_t st);

// Tiling of one forward group.  Wide groups (at least one workgroup per compute unit) use the wide
// kernel: 256 rows x 2 unit blocks per workgroup of 8 waves.  Narrower groups use 128-row tiles of one
// unit block and, if still short of workgroups, split K (partial sums in the workspace, then an
// epilogue kernel).  (256-row narrow tiles, one workgroup per compute unit, measured slower on the
// 1,838-row levels of H = 1,024: 58 -> 68 us a level.)
struct FwdPlan {
  int ksplit = 1;
  bool wide = false;  // 256 rows x 2 unit blocks per workgroup of 8 waves
};
// alone: the group launches by itself (not in a level launch, whose groups' splits are cut together)
inline FwdPlan fwd_plan(int rows, int HP, int inp_used, int arity, int esize, bool can_split, bool alone = false) {
  const int BK = esize == 4 ? 32 : 64;
  const int nst = inp_used / BK + arity * (HP / BK);
  const long long ub = HP / 32;
  FwdPlan p;
  // wide tiles once they give every compute unit a workgroup (narrower levels: the K-split of
  // partial sums through the workspace costs more than a wide tile gains)
  p.wide = ((long long)(rows + 255) / 256) * (ub / 2) >= 256;
  if (p.wide) return p;
  const long long base = ((long long)(rows + 127) / 128) * ub;
  if (can_split && base < 192 && nst >= 4) {
    // aim at a workgroup per compute unit; a bf16 group alone with a short K (under 16 stages of 128 bytes) at
    // half of that: its slices are short, and the partial sums cost more than the extra workgroups gain
    // (config 3, H = 300: the forward 0.444 -> 0.423 ms a step; config 5's long K: no gain)
    const long long aim = alone && esize == 2 && nst < 16 ? 128 : 256;
    const long long want = (aim + base - 1) / base;
    p.ksplit = (int)std::min<long long>(want, nst / 2);
  }
  return p;
}

// dz . W^T tiling: wide groups use 256 x 256 tiles (8 waves); others 128 * mt rows x 128 columns.  In
// both, K may be cut into ksplit slices that add their partial products into the targets atomically.
struct DxPlan {
  int mt = 1, ksplit = 1;
  bool wide = false;  // 256 x 256 tiles per workgroup of 8 waves
};
// at most this many K slices: beyond it the atomic adds of the slices cost more than the shorter K loops
// save.  fp32: 8 (config 2's top levels of 256-4,096 rows at H = 256: 8 beats 4).  bf16: 4 (config 4's level
// launches of two or three groups of 50-500 rows at H = 512, up to 5.5 M atomic adds a level with 8 slices:
// 4 beats 2, 3, 6 and 8 -- 6.34 -> 5.97 ms a step; configs 3 and 5 unchanged)
constexpr int kDxMaxSplit = 8;
constexpr int kDxMaxSplitBf16 = 4;
// levels with fewer narrow tiles than this split K (measured: 256 beats 192, the same as 384 or 512)
constexpr int kDxSplitBelow = 256;
inline DxPlan dx_plan(int rows, int Nb, int Kb, int esize, bool can_split) {
  const int BK = esize == 4 ? 32 : 64;
  const int nst = Kb / BK;
  const long long nb = (Nb + 127) / 128;
  DxPlan p;
  // wide tiles once they give every compute unit a workgroup
  const long long wt = ((long long)(rows + 255) / 256) * ((Nb + 255) / 256);
  p.wide = wt >= 256;
  if (p.wide) return p;
  // bf16 levels whose wide tiles fill at least half the compute units, with a long K (at least 64
  // stages of 64 bytes): wide tiles with K cut in two (measured: faster than the narrow tiles there;
  // more slices, narrower levels or shorter K lose more to the atomic adds of the slices than the wide
  // tiles gain)
  if (can_split && esize == 2 && wt * 2 >= 256 && Kb * esize / 64 >= 64) {
    p.wide = true;
    p.ksplit = 2;
    return p;
  }
  // fp32: 128-row tiles, two workgroups per compute unit.  bf16: 256-row tiles on wide levels, and on levels
  // with a long K (at least 64 stages of 64 bytes) whose 256-row tiles give half the compute units a tile
  // (measured on the 1,024-4,095-row levels at H = 1,024: 78 -> 69 us a level; with the K of H = 300 the
  // 128-row tiles were faster)
  const long long t256 = ((long long)(rows + 255) / 256) * nb;
  p.mt = esize == 4 ? 1 : (t256 >= 256 || (t256 >= 128 && Kb * esize / 64 >= 64) ? 2 : 1);
  const long long base = ((long long)(rows + 128 * p.mt - 1) / (128 * p.mt)) * nb;
  if (can_split && base < kDxSplitBelow && nst >= 4) {
    // aim at a workgroup per compute unit; bf16 levels with a short K at half of that (config 3, H = 300: the
    // dz.W^T 0.509 -> 0.489 ms a step; with config 5's long K the halved grid was far slower)
    const long long aim = esize == 2 && Kb * esize / 64 < 64 ? 128 : 256;
    const long long want = (aim + base - 1) / base;
    p.ksplit = (int)std::min<long long>(std::min<long long>(want, nst / 2), esize == 2 ? kDxMaxSplitBf16 : kDxMaxSplit);
  }
  return p;
}
void launch_embed_fwd(int dtype, int rows, int row_begin, int H, int ld, int tld, const void* table,
                      const int* input_idx, void* h_pool, float* c_pool, hipStream_t st);
void launch_zero_f32(float* p, size_t n, hipStream_t st);
void launch_roots(int dtype, int R, int ld, const int* root_pos, const void* h_pool, void* roots_out,
                  hipStream_t st);

struct BwdCellArgs {
  int rows, row_begin, idx_off, arity;
  int H, HP, ld, gstride;
  const float* c_pool;
  float* gates;  // saved activations in, dz out
  float* dh;
  float* dc;
  const int* child_pos;
  const int* input_idx;
  // beside child_pos: the child has one parent edge.  Such a child's gradient rows start undefined (the
  // initialisation skips them) and this row's backward stores its dc row whole (pad columns and kinds without a
  // cell state included: zeros); a child with several parents gets fp32 atomic adds on zeroed rows.
  const int* child_one;
  float* d_table;
  int tld;
  int dz_bf16;  // write dz as bf16 (the operand type of bf16 parameters)
  const float* u_mask = nullptr;  // the forward's recurrent-dropout mask, or NULL
  // this group's dz . W^T adds K slices into its children's dh atomically: zero the dh rows of the children
  // with one parent edge first (their rows are not initialised)
  int zero_child_dh = 0;
};
void launch_cell_bwd(int kind, const BwdCellArgs& a, hipStream_t st);
void launch_level_cbwd(const int* kinds, const BwdCellArgs* args, int n, hipStream_t st);
// dh = dh_nodes on every row (if given); otherwise dh and dc rows are zeroed only where a node does not have
// exactly one parent edge (roots, shared children): every other row is stored whole by its parent's backward
void launch_bwd_init(int N, int R, int ld, const float* dh_nodes, const float* dh_roots, const int* root_pos,
                     const int* pos_npar, float* dh, float* dc, hipStream_t st);

struct DxArgs {
  int rows, row_begin, idx_off, arity;
  int H, HP, ld, gstride, Kb, Nb;
  const float* dz;
  const void* Wb;
  const void* zero;  // a zero row at least as wide as any K the kernels read
  int mode;  // 0: scatter into children's dh, 1: into leaf-table rows
  float* dh;
  const int* child_pos;
  float* d_table;
  const int* input_idx;
  int in_dim, tld;
  const int* child_one;  // beside child_pos: the child has one parent edge
  int dh_fresh;     // such children's dh rows are not initialised: stored whole (pad columns too), not added to
  int can_split;    // K may be split across workgroups (slices add into the targets atomically)
  int ksplit;       // set by the launcher
  int map;          // set by the launcher: workgroup order over the XCDs (kMapRows, kMapCols, kMapOwnCols)
};
// name: the profiling record's kernel class (NULL: bwd_dx.bf16 / bwd_dx.f32)
void launch_bwd_dx(int dtype, const DxArgs& a, hipStream_t st, const char* name = nullptr);
// dz summed over the rows of every run of equal (op, leaf-table row): entries i0 .. i0 + count - 1 of tok_rows
// (one op's), runs u0 .. u0 + U - 1, into zsum [U][Kb] fp32 (zeroed here), and for bf16 its bf16 copy zbf [U][Kb]
void launch_tok_sum(int dtype, const int* tok_rows, const int* tok_seg, const int* tok_start, int i0, int count,
                    int u0, int U, const float* dz, int gstride, int Kb, float* zsum, uint16_t* zbf, hipStream_t st);
// an embedding op's leaf-table gradient: its fp32 dh rows (stride ld) summed over the runs of entries i0 ..
// i0 + count - 1 and added into the runs' leaf-table rows (columns < H, stride tld)
void launch_tok_table(const int* tok_rows, const int* tok_seg, const int* tok_start, const int* tok_row, int i0,
                      int count, const float* dh, int ld, int H, float* d_table, int tld, hipStream_t st);
// true if launch_bwd_dx would run this call on narrow tiles (the ones a level launch can merge)
bool bwd_dx_is_narrow(int dtype, const DxArgs& a);
void launch_level_dx(int dtype, const DxArgs* args, int n, hipStream_t st);

// ---- feed-forward attention operations (attn.hip) ----
struct AttnArgs {
  int rows, row_begin, idx_off;
  int H, ld;
  void* h_pool;         // [N, ld] of the params' type: the forward writes the group's rows, the backward reads
  float* c_pool;        // [N, ld] (m, s) in columns 0 and 1
  const int* child_pos;
  const int* child_one;  // backward: the child has one parent edge (plain read-add-write)
  const void* w;        // scorer: w, HP entries of the params' type (zero padded)
  const float* bias;    // scorer: [0] = b
  float* dh;            // backward: per-node gradient accumulators [N, ld]
  float* dc;
  float* gates;         // backward: the scorer saves de at gates[p * gstride] (NULL: not saved)
  int gstride;
  int dh_fresh;         // backward: the dh rows of children with one parent edge start undefined (stored whole)
};
// rows of the scorer's weight gradient reduced by one workgroup (chunk order is fixed)
constexpr int kAttnWgradChunk = 128;
int attn_wgrad_chunks(int count);
void launch_attn_fwd(int dtype, int kind, const AttnArgs& a, hipStream_t st);
void launch_attn_bwd(int dtype, int kind, const AttnArgs& a, hipStream_t st);
// dw [H] += sum_r de_r h_c(r), db[0] += sum_r de_r over the op's rows; part holds chunks * (HP + 64) floats
void launch_attn_wgrad(int dtype, const int* op_rows, const int* op_cpos, int count, int H, int HP, int ld,
                       const void* h_pool, const float* gates, int gstride, float* part, float* dw, float* db,
                       hipStream_t st);
void launch_pack_score(int dtype, int H, int HP, const void* w, const float* b, void* wdst, float* bdst,
                       hipStream_t st);

// ---- weight gradients (wgrad.hip) ----
struct WgArgs {
  const int* op_rows;  // rows of this op (pool rows), count of them
  const int* op_cpos;  // [2 * count] children's pool rows per op row
  const int* op_inp;   // [count] leaf-table row per op row
  int count;
  int seg;  // 0: input rows from the leaf table, 1: children's h rows
  int H, HP, ld, in_dim, tld, gstride;
  int Kw, Nw;
  const void* src;
  const float* dz;
  int chunk, nchunk;
  int wide;        // 256 x 256 tiles (WgradSplit::wide)
  float* partial;  // [nchunk][Kw][Nw]
  float* bpart;    // [bparts][Nw] column sums of dz (see WgradSplit), or NULL
  const void* zero;  // a zero row at least 16 bytes past any column the kernels read
};
void launch_wgrad(int dtype, const WgArgs& a, hipStream_t st);
// Sum the partial tiles into the canonical dW ([rows][G * H]); partial column n is gate block n / HP of
// the dz layout, canonical gate gate_of_code(gcode, n / HP).
void launch_wgrad_reduce(const float* partial, int nchunk, int Kw, int Nw, int seg, int H, int HP, int in_dim,
                         int G, int gcode, float* dW, hipStream_t st);
void launch_bias_partial(const int* op_rows, int count, int chunk, int nchunk, const float* dz, int gstride,
                         int Nw, int bf, float* bpart, hipStream_t st);
void launch_bias_reduce(const float* bpart, int nchunk, int Nw, int H, int HP, int gcode, float* dbias,
                        hipStream_t st);

// ---- training step (train.hip) ----
bool loss_classes_supported(int C);
constexpr int kLossMaxHC = 8000;  // hidden * classes: W, the partial dW and db of a block within 64 KB of LDS
size_t loss_workspace_bytes(int H, int C);
void launch_loss_ce(int dtype, int N, int H, int ld, int C, const void* h_pool, const int* pos_node, const int* labels,
                    const float* W, const float* b, float scale, float* node_loss, float* dh, float* dW, float* db,
                    float* ws, hipStream_t st);
void launch_dropout_mask(const int* pos_node, int N, int H, int ld, unsigned thresh, float scale,
                         unsigned long long seed, unsigned long long step, float* mask, hipStream_t st);
void launch_adam(size_t n, float* p, uint16_t* p_bf16, const float* g, float* m, float* v, double b1, double b2,
                 double lr_t, double eps, hipStream_t st);

// ---- achievable-peak probes (diag.hip) ----
int32_t probe_mfma(int dtype, bool random_operands, hipStream_t st, double* tflops);
int32_t probe_copy(void* dst, const void* src, size_t bytes, hipStream_t st, double* gbs);

// ---- packing (pack.hip) ----
void launch_pack(int dtype, int mode, int G, int GC, int gcode, int H, int HP, int in_dim, int INP, int arity, int Kf,
                 const void* W_in, const void* W_rec, const float* bias, void* dst, size_t count,
                 hipStream_t st);

}  // namespace fold
