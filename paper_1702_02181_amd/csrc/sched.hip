// GPU scheduler for dynamic batching (Section 2 of the paper, the greedy
// scheduling algorithm), gfx950.
//
//   validate   CSR structure, op ids, arity, child range / same graph, inputs
//   depth      one workgroup per graph runs Kahn's algorithm bottom-up over the
//              graph's reverse edges in LDS: a node whose children are all done
//              gets depth 1 + max(child depths) (the zero state -1 and leaf-table
//              rows are depth-0 constants).  Unprocessed nodes mean a cycle.
//   sort       stable LSD radix sort (8-bit digits) of the node ids by the key
//              (depth - 1) * num_ops + op: ties stay in node-id order
//   emit       group table, level_ptr, child_pos (pool rows of every edge),
//              input_idx and root rows; the rows of every op in (op, row) order
//              for the deferred weight gradients (one more stable radix pass,
//              keyed by op)
// All results are integers and bit-exact by construction.  Everything runs on
// the stream without a host round trip until one read-back at the end: arrays
// are sized by N (levels and groups never outnumber nodes), the radix passes
// the actual depth needs are decided on the device, and every kernel after
// validation returns at once when the error word is set.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>

#include "common.h"
#include "internal.h"

namespace fold {

namespace {

constexpr unsigned long long kNoErr = ~0ull;
constexpr int kTooDeep = 0x7fffffff;  // error-word node of "depth * num_ops too large for the sort keys"
constexpr long long kMaxKeys = 1LL << 30;
constexpr int kBlock = 256;
constexpr int kMaxOps = 256;  // the op table travels as a kernel argument (2 KB)
constexpr int kDepthLdsInts = 8192;  // 32 KiB per workgroup; larger graphs use global scratch
constexpr int kScanItems = 8;        // items per thread in device-wide scans
constexpr int kScanTile = kBlock * kScanItems;
constexpr int kRadixItems = 8;
constexpr int kRadixTile = kBlock * kRadixItems;

struct OpTable {
  int n;
  int arity[kMaxOps];
  int has_input[kMaxOps];
};

// error word: ((node + 1) << 8) | (-code); structural errors use node + 1 = 0.  atomicMin keeps the
// lowest node with an error and, within it, the first check in the order op, arity, child, input.
__device__ __forceinline__ void report(unsigned long long* err, int node_plus_1, int code) {
  unsigned long long w = ((unsigned long long)(unsigned)node_plus_1 << 8) | (unsigned long long)(-code);
  atomicMin(err, w);
}

// ---------------------------------------------------------------- block scan helpers

// exclusive scan of one int per thread over a 256-thread block; returns the prefix, *total = sum
__device__ int block_exscan_256(int x, int* total) {
  __shared__ int wsum[kBlock / kWave];
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
  int v = x;
  for (int d = 1; d < kWave; d <<= 1) {
    int y = __shfl_up(v, d, kWave);
    if (lane >= d) v += y;
  }
  if (lane == kWave - 1) wsum[w] = v;
  __syncthreads();
  int pre = 0, tot = 0;
  for (int i = 0; i < kBlock / kWave; ++i) {
    int s = wsum[i];
    if (i < w) pre += s;
    tot += s;
  }
  __syncthreads();
  *total = tot;
  return pre + v - x;
}

// in-place exclusive scan of a[0..n) (generic pointer: LDS or global), a[n] = total
__device__ void block_exscan_array(int* a, int n) {
  const int t = threadIdx.x;
  const int chunk = (n + kBlock - 1) / kBlock;
  const int lo = min(n, t * chunk), hi = min(n, lo + chunk);
  int s = 0;
  for (int i = lo; i < hi; ++i) s += a[i];
  int tot;
  int pre = block_exscan_256(s, &tot);
  __syncthreads();
  for (int i = lo; i < hi; ++i) {
    int v = a[i];
    a[i] = pre;
    pre += v;
  }
  if (t == 0) a[n] = tot;
  __syncthreads();
}

// ---------------------------------------------------------------- validation

__global__ void k_check_struct(const int* gp, int G, const int* cp, int N, int E, unsigned long long* err) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i == 0) {
    if (gp[0] != 0 || gp[G] != N || cp[0] != 0 || cp[N] != E) report(err, 0, FOLD_E_INVALID);
  }
  if (i < G) {
    int a = gp[i], b = gp[i + 1];
    if (a < 0 || b > N || a > b) report(err, 0, FOLD_E_INVALID);
  }
  if (i < N) {
    int a = cp[i], b = cp[i + 1];
    if (a < 0 || b > E || a > b) report(err, 0, FOLD_E_INVALID);
  }
}

__global__ void k_node_graph(const int* gp, int* node_graph, const unsigned long long* err) {
  if (*err != kNoErr) return;
  const int g = blockIdx.x;
  for (int v = gp[g] + threadIdx.x; v < gp[g + 1]; v += blockDim.x) node_graph[v] = g;
}

__global__ void k_check_nodes(const int* node_op, const int* cp, const int* ci, const int* node_input,
                              const int* node_graph, int N, int num_inputs, OpTable ops,
                              unsigned long long* err) {
  if (*err != kNoErr) return;
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= N) return;
  const int op = node_op[v];
  if (op < 0 || op >= ops.n) { report(err, v + 1, FOLD_E_OP); return; }
  const int a = cp[v], b = cp[v + 1];
  if (b - a != ops.arity[op]) { report(err, v + 1, FOLD_E_ARITY); return; }
  const int gv = node_graph[v];
  for (int j = a; j < b; ++j) {
    int c = ci[j];
    if (c == -1) continue;
    if (c < 0 || c >= N || node_graph[c] != gv) { report(err, v + 1, FOLD_E_CHILD); return; }
  }
  const int inp = node_input[v];
  if (ops.has_input[op]) {
    if (inp < 0 || inp >= num_inputs) report(err, v + 1, FOLD_E_INPUT);
  } else if (inp != -1) {
    report(err, v + 1, FOLD_E_INPUT);
  }
}

// ---------------------------------------------------------------- depth (one workgroup per graph)

// meta[0] = max depth, meta[1] = max number of parents of a node
__global__ __launch_bounds__(kBlock) void k_depth(const int* gp, const int* cp, const int* ci, int* depth,
                                                  int* indeg, int* scratch, unsigned long long* err,
                                                  int* meta) {
  if (*err != kNoErr) return;
  extern __shared__ int lds[];
  __shared__ int qn[2];
  const int g = blockIdx.x, t = threadIdx.x;
  const int g0 = gp[g], n = gp[g + 1] - g0;
  if (n == 0) return;
  const int e0 = cp[g0], e = cp[g0 + n] - e0;
  const long long need = 6LL * n + 1 + e;
  int* base = (need <= kDepthLdsInts) ? lds : scratch + (6LL * g0 + g + e0);
  int* pend = base;         // [n] children not yet done
  int* dep = pend + n;      // [n]
  int* pptr = dep + n;      // [n+1] parent-list offsets (counts, then exclusive scan)
  int* pfill = pptr + n + 1;  // [n]
  int* q0 = pfill + n;      // [n]
  int* q1 = q0 + n;         // [n]
  int* plist = q1 + n;      // [e]

  for (int v = t; v < n; v += kBlock) { pptr[v] = 0; pfill[v] = 0; dep[v] = 0; }
  if (t == 0) { qn[0] = 0; qn[1] = 0; }
  __syncthreads();
  for (int v = t; v < n; v += kBlock) {
    int cnt = 0;
    for (int j = cp[g0 + v]; j < cp[g0 + v + 1]; ++j) {
      int c = ci[j];
      if (c >= 0) { ++cnt; atomicAdd(&pptr[c - g0], 1); }
    }
    pend[v] = cnt;
  }
  __syncthreads();
  block_exscan_array(pptr, n);
  for (int v = t; v < n; v += kBlock) {
    for (int j = cp[g0 + v]; j < cp[g0 + v + 1]; ++j) {
      int c = ci[j];
      if (c >= 0) {
        int s = atomicAdd(&pfill[c - g0], 1);
        plist[pptr[c - g0] + s] = v;
      }
    }
  }
  __syncthreads();
  int local_maxpar = 0;
  for (int v = t; v < n; v += kBlock) {
    indeg[g0 + v] = pfill[v];
    local_maxpar = max(local_maxpar, pfill[v]);
    if (pend[v] == 0) {
      dep[v] = 1;
      q0[atomicAdd(&qn[0], 1)] = v;
    }
  }
  __syncthreads();
  int processed = 0, cur = 0;
  while (true) {
    const int cnt = qn[cur];
    if (cnt == 0) break;
    processed += cnt;
    int* Q = cur ? q1 : q0;
    int* NQ = cur ? q0 : q1;
    for (int i = t; i < cnt; i += kBlock) {
      const int v = Q[i];
      const int dv = dep[v] + 1;
      for (int k = pptr[v]; k < pptr[v + 1]; ++k) {
        const int p = plist[k];
        atomicMax(&dep[p], dv);
        if (atomicSub(&pend[p], 1) == 1) NQ[atomicAdd(&qn[cur ^ 1], 1)] = p;
      }
    }
    __syncthreads();
    if (t == 0) qn[cur] = 0;
    __syncthreads();
    cur ^= 1;
  }
  if (processed < n) {
    if (t == 0) report(err, g0 + 1, FOLD_E_CYCLE);
    return;
  }
  int local_max = 0;
  for (int v = t; v < n; v += kBlock) {
    depth[g0 + v] = dep[v];
    local_max = max(local_max, dep[v]);
  }
  atomicMax(&meta[0], local_max);
  atomicMax(&meta[1], local_maxpar);
}

// ---------------------------------------------------------------- device-wide exclusive scan

__global__ void k_scan_reduce(const int* in, int n, int* partial) {
  const int b = blockIdx.x, t = threadIdx.x;
  const long long base = (long long)b * kScanTile + (long long)t * kScanItems;
  int s = 0;
  for (int i = 0; i < kScanItems; ++i) {
    long long j = base + i;
    if (j < n) s += in[j];
  }
  int tot;
  block_exscan_256(s, &tot);
  if (t == 0) partial[b] = tot;
}

// single block: exclusive scan of partial[0..nb) in place, *total = sum
__global__ void k_scan_partials(int* partial, int nb, int* total) {
  int carry = 0;
  for (int base = 0; base < nb; base += kBlock) {
    const int i = base + threadIdx.x;
    const int x = i < nb ? partial[i] : 0;
    int tot;
    const int pre = block_exscan_256(x, &tot);
    if (i < nb) partial[i] = carry + pre;
    carry += tot;
    __syncthreads();
  }
  if (threadIdx.x == 0) *total = carry;
}

__global__ void k_scan_down(const int* in, int n, const int* partial, int* out) {
  const int b = blockIdx.x, t = threadIdx.x;
  const long long base = (long long)b * kScanTile + (long long)t * kScanItems;
  int v[kScanItems];
  int s = 0;
  for (int i = 0; i < kScanItems; ++i) {
    long long j = base + i;
    v[i] = j < n ? in[j] : 0;
    s += v[i];
  }
  int tot;
  int pre = block_exscan_256(s, &tot) + partial[b];
  for (int i = 0; i < kScanItems; ++i) {
    long long j = base + i;
    if (j < n) out[j] = pre;
    pre += v[i];
  }
}

// exclusive scan in -> out (may alias), total -> *total (device); temp holds >= ceil(n / tile) ints
void scan_exclusive(const int* in, int* out, int n, int* total, int* temp, hipStream_t st) {
  const int nb = std::max(1, (n + kScanTile - 1) / kScanTile);
  hipLaunchKernelGGL(k_scan_reduce, dim3(nb), dim3(kBlock), 0, st, in, n, temp);
  hipLaunchKernelGGL(k_scan_partials, dim3(1), dim3(kBlock), 0, st, temp, nb, total);
  hipLaunchKernelGGL(k_scan_down, dim3(nb), dim3(kBlock), 0, st, in, n, temp, out);
}

// ---------------------------------------------------------------- stable LSD radix sort

__global__ void k_make_keys(const int* depth, const int* node_op, int N, int num_ops, unsigned* keys,
                            int* vals, const unsigned long long* err) {
  if (*err != kNoErr) return;
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= N) return;
  keys[v] = (unsigned)((depth[v] - 1) * num_ops + node_op[v]);
  vals[v] = v;
}

// number of 8-bit radix passes the keys (depth - 1) * num_ops + op need, from the depth found on the
// device: meta[0] = D, written to *passes (at least 1); a depth whose keys would pass kMaxKeys is an error
__global__ void k_sort_plan(const int* meta, int num_ops, unsigned long long* err, int* passes) {
  if (threadIdx.x != 0) return;
  const long long nk = (long long)meta[0] * num_ops;
  if (nk > kMaxKeys) {
    report(err, kTooDeep, FOLD_E_INVALID);
    *passes = 0;
    return;
  }
  unsigned long long mx = nk > 0 ? (unsigned long long)(nk - 1) : 0ull;
  int bits = 1;
  while (bits < 32 && (mx >> bits)) ++bits;
  *passes = (bits + 7) / 8;
}

// counts[d * B + b] = number of items of tile b whose digit is d.  Pass `pass` runs only below *passes
// (passes == nullptr: always) and when no error is set.
__global__ void k_radix_count(const unsigned* keys, int n, int shift, int* counts, int B, const unsigned long long* err,
                              const int* passes, int pass) {
  if (*err != kNoErr || (passes && pass >= *passes)) return;
  __shared__ int hist[256];
  const int b = blockIdx.x, t = threadIdx.x;
  hist[t] = 0;
  __syncthreads();
  const long long base = (long long)b * kRadixTile;
  for (int r = 0; r < kRadixItems; ++r) {
    long long i = base + (long long)r * kBlock + t;
    if (i < n) atomicAdd(&hist[(keys[i] >> shift) & 255u], 1);
  }
  __syncthreads();
  counts[t * B + b] = hist[t];
}

// Scatter in tile order.  Items of a round are ranked among equal digits by a wave-level match
// (one ballot per digit bit) plus the counts of earlier waves; rounds go in item order, so the
// scatter is stable.  A pass at or above *passes copies its tile unchanged (the keys are already
// sorted), so the host can launch the most passes N * num_ops could need and the result still ends in
// the output buffer of the last pass.
__global__ __launch_bounds__(kBlock) void k_radix_scatter(const unsigned* keys_in, const int* vals_in,
                                                          unsigned* keys_out, int* vals_out,
                                                          const int* offsets, int n, int shift, int B,
                                                          const unsigned long long* err, const int* passes,
                                                          int pass) {
  if (*err != kNoErr) return;
  __shared__ int base[256];
  __shared__ int wcnt[kBlock / kWave][256];
  const int b = blockIdx.x, t = threadIdx.x, lane = t & (kWave - 1), w = t / kWave;
  if (passes && pass >= *passes) {
    for (int r = 0; r < kRadixItems; ++r) {
      const long long i = (long long)b * kRadixTile + (long long)r * kBlock + t;
      if (i < n) {
        keys_out[i] = keys_in[i];
        vals_out[i] = vals_in[i];
      }
    }
    return;
  }
  base[t] = offsets[t * B + b];
  for (int i = 0; i < kBlock / kWave; ++i) wcnt[i][t] = 0;
  __syncthreads();
  const long long start = (long long)b * kRadixTile;
  const unsigned long long lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int r = 0; r < kRadixItems; ++r) {
    const long long i = start + (long long)r * kBlock + t;
    const bool valid = i < n;
    const unsigned k = valid ? keys_in[i] : 0u;
    const int d = valid ? (int)((k >> shift) & 255u) : 256;  // 256 marks padding
    unsigned long long m = ~0ull;
    for (int bit = 0; bit < 9; ++bit) {
      const int on = (d >> bit) & 1;
      const unsigned long long bal = __ballot(on);
      m &= on ? bal : ~bal;
    }
    const int lrank = __popcll(m & lt_mask);
    if (valid && lrank == 0) wcnt[w][d] = __popcll(m);
    __syncthreads();
    if (valid) {
      int pre = 0;
      for (int j = 0; j < w; ++j) pre += wcnt[j][d];
      const int pos = base[d] + pre + lrank;
      keys_out[pos] = k;
      vals_out[pos] = vals_in[i];
    }
    __syncthreads();
    int tot = 0;
    for (int j = 0; j < kBlock / kWave; ++j) { tot += wcnt[j][t]; wcnt[j][t] = 0; }
    base[t] += tot;
    __syncthreads();
  }
}

// ---------------------------------------------------------------- emission

__global__ void k_post_sort(const unsigned* keys, const int* vals, int N, int num_ops, int* pos_node,
                            int* node_pos, int* flag, int* level_ptr, const unsigned long long* err) {
  if (*err != kNoErr) return;
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= N) return;
  const int v = vals[p];
  pos_node[p] = v;
  node_pos[v] = p;
  const unsigned k = keys[p];
  const bool start = (p == 0) || (keys[p - 1] != k);
  flag[p] = start ? 1 : 0;
  const int lvl = (int)(k / (unsigned)num_ops) + 1;
  if (p == 0 || (int)(keys[p - 1] / (unsigned)num_ops) + 1 != lvl) level_ptr[lvl - 1] = p;
  if (p == N - 1) level_ptr[lvl] = N;
}

__global__ void k_group_starts(const unsigned* keys, const int* flag, const int* exs, int N, int num_ops,
                               int* gid, int* g_level, int* g_op, int* g_row_begin, const unsigned long long* err) {
  if (*err != kNoErr) return;
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= N) return;
  const int g = exs[p] + flag[p] - 1;
  gid[p] = g;
  if (flag[p]) {
    g_row_begin[g] = p;
    g_level[g] = (int)(keys[p] / (unsigned)num_ops) + 1;
    g_op[g] = (int)(keys[p] % (unsigned)num_ops);
  }
}

// ng = number of groups (device); rows and rows * arity of each group (g_edges has N entries)
__global__ void k_group_rows(const int* ng_ptr, int N, const int* g_row_begin, const int* g_op, OpTable ops,
                             int* g_rows, int* g_edges, const unsigned long long* err) {
  const int g = blockIdx.x * blockDim.x + threadIdx.x;
  if (*err != kNoErr || g >= N) return;
  const int ng = *ng_ptr;
  if (g >= ng) {
    g_edges[g] = 0;
    return;
  }
  const int end = (g + 1 < ng) ? g_row_begin[g + 1] : N;
  const int rows = end - g_row_begin[g];
  g_rows[g] = rows;
  g_edges[g] = rows * ops.arity[g_op[g]];
}

__global__ void k_emit(const int* pos_node, const int* node_pos, const int* gid, const int* g_row_begin,
                       const int* g_op, const int* g_idx_off, const int* cp, const int* ci,
                       const int* node_input, const int* indeg, int N, OpTable ops, int* child_pos,
                       int* child_one, int* input_idx, int* pos_npar, const unsigned long long* err) {
  if (*err != kNoErr) return;
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= N) return;
  const int v = pos_node[p];
  const int g = gid[p];
  const int a = ops.arity[g_op[g]];
  const int off = g_idx_off[g] + (p - g_row_begin[g]) * a;
  const int c0 = cp[v];
  for (int k = 0; k < a; ++k) {
    const int c = ci[c0 + k];
    child_pos[off + k] = c >= 0 ? node_pos[c] : -1;
    child_one[off + k] = c >= 0 && indeg[c] == 1 ? 1 : 0;
  }
  input_idx[p] = node_input[v];
  pos_npar[p] = indeg[v];
}

__global__ void k_root_flags(const int* indeg, int N, int* flag, const unsigned long long* err) {
  if (*err != kNoErr) return;
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v < N) flag[v] = indeg[v] == 0 ? 1 : 0;
}

__global__ void k_root_emit(const int* flag, const int* rank, const int* node_pos, int N, int* root_pos,
                            const unsigned long long* err) {
  if (*err != kNoErr) return;
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v < N && flag[v]) root_pos[rank[v]] = node_pos[v];
}

// error word "none", meta zero
__global__ void k_init_meta(void* em) {
  if (threadIdx.x == 0) *static_cast<unsigned long long*>(em) = kNoErr;
  int* meta = reinterpret_cast<int*>(static_cast<unsigned long long*>(em) + 1);
  if (threadIdx.x < 8) meta[threadIdx.x] = 0;
}

// keys of the second sort: the op of every pool row, with the row as its value; a stable sort by op
// lists every op's rows in (op, row) order
__global__ void k_op_keys(const int* gid, const int* g_op, int N, unsigned* keys, int* vals,
                          const unsigned long long* err) {
  if (*err != kNoErr) return;
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= N) return;
  keys[p] = (unsigned)g_op[gid[p]];
  vals[p] = p;
}

// for entry q of the (op, row) list: the row's children and leaf-table row
__global__ void k_op_rows(const int* op_rows, const int* gid, const int* g_row_begin, const int* g_op,
                          const int* g_idx_off, const int* child_pos, const int* input_idx, OpTable ops, int N,
                          int* op_cpos, int* op_inp, const unsigned long long* err) {
  if (*err != kNoErr) return;
  const int q = blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= N) return;
  const int p = op_rows[q];
  const int g = gid[p];
  const int r = p - g_row_begin[g];
  const int a = ops.arity[g_op[g]];
  op_cpos[2 * q] = a > 0 ? child_pos[g_idx_off[g] + r * a] : -1;
  op_cpos[2 * q + 1] = a > 1 ? child_pos[g_idx_off[g] + r * a + 1] : -1;
  op_inp[q] = input_idx[p];
}

// Static-graph layout of a group's child slot k: its children are the consecutive pool rows base .. base +
// rows - 1 and each has exactly one parent edge.  A batch of identically shaped graphs with one operation per
// node position (manual batching) has it on every slot; the kernels then address those children by
// base + row instead of loading child_pos.  First every group proposes its first child as the base ...
__global__ void k_cbase_init(const int* ng_ptr, int N, const int* g_op, const int* g_idx_off, const int* child_pos,
                             const int* child_one, OpTable ops, int* cb0, int* cb1, const unsigned long long* err) {
  if (*err != kNoErr) return;
  const int g = blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= N || g >= *ng_ptr) return;
  const int a = ops.arity[g_op[g]], off = g_idx_off[g];
  int b[2] = {-1, -1};
  for (int k = 0; k < a && k < 2; ++k) b[k] = child_one[off + k] ? child_pos[off + k] : -1;
  cb0[g] = b[0];
  cb1[g] = b[1];
}

// ... then every row withdraws it (-1) where its child is not base + r or has another parent edge
__global__ void k_cbase_check(int N, const int* gid, const int* g_row_begin, const int* g_op, const int* g_idx_off,
                              const int* child_pos, const int* child_one, OpTable ops, int* cb0, int* cb1,
                              const unsigned long long* err) {
  if (*err != kNoErr) return;
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= N) return;
  const int g = gid[p], r = p - g_row_begin[g], a = ops.arity[g_op[g]];
  for (int k = 0; k < a && k < 2; ++k) {
    int* cb = k == 0 ? cb0 : cb1;
    const int base = cb[g];
    if (base < 0) continue;
    const int e = g_idx_off[g] + r * a + k;
    if (child_pos[e] != base + r || !child_one[e]) cb[g] = -1;
  }
}

// The one read-back of a schedule: the error word and meta, then the first lcap + 1 entries of level_ptr
// and the first gcap groups of each group array, side by side.
constexpr int kHdr = 16;
constexpr int kGroupArrays = 7;
struct GroupArrays {
  const int* a[kGroupArrays];  // level, op, row_begin, rows, idx_off, child base of slot 0, of slot 1
};
__global__ void k_compact(const unsigned long long* err, const int* meta, const int* level_ptr, GroupArrays garr,
                          int lcap, int gcap, int* out) {
  const unsigned long long e = *err;
  if (threadIdx.x == 0) {
    out[0] = (int)(unsigned)(e & 0xffffffffull);
    out[1] = (int)(unsigned)(e >> 32);
    for (int i = 0; i < 8; ++i) out[2 + i] = meta[i];
  }
  if (e != kNoErr) return;
  const int nl = min(meta[0] + 1, lcap + 1), ng = min(meta[4], gcap);
  for (int i = threadIdx.x; i < nl; i += blockDim.x) out[kHdr + i] = level_ptr[i];
  int* go = out + kHdr + lcap + 1;
  for (int k = 0; k < kGroupArrays; ++k)
    for (int i = threadIdx.x; i < ng; i += blockDim.x) go[k * gcap + i] = garr.a[k][i];
}

inline dim3 grid_for(long long n) { return dim3((unsigned)std::max(1LL, (n + kBlock - 1) / kBlock)); }

// Stream-ordered temporaries of one phase: the sizes are declared first (reserve), then one allocation
// from the device's pool backs them all (commit); freed at scope exit.  One allocation per phase keeps
// the host cost of a schedule independent of how many temporaries it uses.
struct Temp {
  hipStream_t st;
  std::vector<void*> ptrs;
  std::vector<std::pair<void**, size_t>> want;
  size_t bytes = 0;
  explicit Temp(hipStream_t s) : st(s) {}
  ~Temp() {
    for (void* p : ptrs) (void)hipFreeAsync(p, st);
  }
  template <class T>
  void reserve(T** p, size_t count) {
    want.push_back({reinterpret_cast<void**>(p), bytes});
    bytes += (std::max<size_t>(count, 1) * sizeof(T) + 255) / 256 * 256;
  }
  hipError_t commit() {
    void* q = nullptr;
    hipError_t e = hipMallocAsync(&q, std::max<size_t>(bytes, 256), st);
    if (e != hipSuccess) return e;
    ptrs.push_back(q);
    for (auto& w : want) *w.first = static_cast<char*>(q) + w.second;
    want.clear();
    bytes = 0;
    return hipSuccess;
  }
};

int decode_error(unsigned long long w, std::string* msg) {
  const int code = -(int)(w & 0xffull);
  const long long node = (long long)(w >> 8) - 1;
  if ((long long)(w >> 8) == kTooDeep) {
    *msg = "fold_schedule: depth * num_ops exceeds 2^30 (the sort keys)";
    return code;
  }
  const char* what = "invalid batch";
  switch (code) {
    case FOLD_E_INVALID: what = "graph_ptr / child_ptr malformed"; break;
    case FOLD_E_OP: what = "node_op out of range"; break;
    case FOLD_E_ARITY: what = "child count differs from the operation's arity"; break;
    case FOLD_E_CHILD: what = "child out of range or in another graph"; break;
    case FOLD_E_INPUT: what = "node_input inconsistent with has_input or out of range"; break;
    case FOLD_E_CYCLE: what = "graph contains a cycle"; break;
    default: break;
  }
  *msg = std::string("fold_schedule: ") + what + (node >= 0 ? " (node " + std::to_string(node) + ")" : "");
  return code;
}

void init_pool_once(int device) {
  static bool done[64] = {false};
  if (device < 0 || device >= 64 || done[device]) return;
  hipMemPool_t pool;
  if (hipDeviceGetDefaultMemPool(&pool, device) == hipSuccess) {
    uint64_t thr = ~0ull;
    (void)hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &thr);
  }
  done[device] = true;
}

}  // namespace

void sched_destroy_impl(fold_sched* h);
static void sched_destroy(fold_sched* h) { sched_destroy_impl(h); }

int32_t schedule_impl(const fold_batch* b, hipStream_t st, fold_sched** out) {
  const int N = b->num_nodes, E = b->num_edges, G = b->num_graphs, K = b->num_ops;
  for (int i = 0; i < K; ++i)
    if (b->ops[i].arity > 2) {
      set_error("fold_schedule: operations take at most two children");
      return FOLD_E_INVALID;
    }
  if (K > kMaxOps) {
    set_error("fold_schedule: at most 256 operations are supported");
    return FOLD_E_INVALID;
  }
  OpTable ops{};
  ops.n = K;
  for (int i = 0; i < K; ++i) {
    ops.arity[i] = b->ops[i].arity;
    ops.has_input[i] = b->ops[i].has_input;
  }
  int device = 0;
  FOLD_HIP_CHECK(hipGetDevice(&device));
  init_pool_once(device);

  auto* h = new fold_sched();
  Sched& s = h->s;
  s.N = N; s.E = E; s.G = G; s.num_ops = K; s.device = device; s.num_inputs = b->num_inputs;
  s.ops.assign(b->ops, b->ops + K);
  auto fail = [&](int code) {
    sched_destroy(h);
    return code;
  };

  // persistent arrays sized by N and E; the level and group tables take N + 1 and 5 x N entries (there are
  // at most N levels and N groups), so nothing waits for the depth to be known on the host
  const size_t n1 = (size_t)N * 19 + 2 * (size_t)E + 16;
  if (hipMalloc(&s.blob, n1 * sizeof(int)) != hipSuccess) {
    set_error("fold_schedule: out of device memory");
    return fail(FOLD_E_NOMEM);
  }
  const size_t cap = std::max<size_t>(N, 1);
  int* q = static_cast<int*>(s.blob);
  s.depth = q; q += N;
  s.node_pos = q; q += N;
  s.pos_node = q; q += N;
  s.input_idx = q; q += N;
  s.root_pos = q; q += N;
  s.child_pos = q; q += E;
  s.child_one = q; q += E;
  s.pos_group = q; q += N;
  s.pos_npar = q; q += N;
  s.op_rows = q; q += N;
  s.op_cpos = q; q += 2 * (size_t)N;
  s.op_inp = q; q += N;
  s.level_ptr = q; q += cap + 1;
  s.g_level = q; q += cap;
  s.g_op = q; q += cap;
  s.g_row_begin = q; q += cap;
  s.g_rows = q; q += cap;
  s.g_idx_off = q; q += cap;
  s.g_cbase0 = q; q += cap;
  s.g_cbase1 = q; q += cap;

  // temporaries of the whole schedule, one pooled allocation
  Temp tmp(st);
  // err, then meta: [0] max depth, [1] max parents, [2] radix passes, [3] scratch total, [4] groups, [5] roots,
  // [6] scratch total
  struct ErrMeta {
    unsigned long long err;
    int meta[8];
  };
  ErrMeta* em = nullptr;
  int *node_graph = nullptr, *indeg = nullptr, *scratch = nullptr, *edges = nullptr, *stage = nullptr;
  unsigned *ka = nullptr, *kb = nullptr;
  int *va = nullptr, *vb = nullptr, *flag = nullptr, *exs = nullptr, *radix_counts = nullptr, *scan_tmp = nullptr;
  const long long scratch_ints = 6LL * N + G + E + 1;
  const int B = (N + kRadixTile - 1) / kRadixTile;
  const long long rc = 256LL * std::max(B, 1);
  const long long scan_tmp_n = std::max<long long>(rc, N) / kScanTile + 2;
  constexpr int kLcap = 4096, kGcap = 4096;  // levels and groups read back with the error word
  const size_t stage_n = kHdr + (kLcap + 1) + kGroupArrays * (size_t)kGcap;
  tmp.reserve(&em, 1);
  tmp.reserve(&stage, stage_n);
  if (N > 0) {
    tmp.reserve(&node_graph, N);
    tmp.reserve(&indeg, N);
    tmp.reserve(&scratch, (size_t)scratch_ints);
    tmp.reserve(&edges, N);
    tmp.reserve(&ka, N);
    tmp.reserve(&kb, N);
    tmp.reserve(&va, N);
    tmp.reserve(&vb, N);
    tmp.reserve(&flag, N);
    tmp.reserve(&exs, N);
    tmp.reserve(&radix_counts, rc);
    tmp.reserve(&scan_tmp, scan_tmp_n);
  }
  if (tmp.commit() != hipSuccess) {
    set_error("fold_schedule: out of device memory (temporaries)");
    return fail(FOLD_E_NOMEM);
  }
  unsigned long long* err = &em->err;
  int* meta = em->meta;
  hipLaunchKernelGGL(k_init_meta, dim3(1), dim3(64), 0, st, em);
  hipLaunchKernelGGL(k_check_struct, grid_for(std::max(G + 1, N + 1)), dim3(kBlock), 0, st, b->graph_ptr, G,
                     b->child_ptr, N, E, err);
  if (N > 0) {
    if (G > 0)
      hipLaunchKernelGGL(k_node_graph, dim3(G), dim3(kBlock), 0, st, b->graph_ptr, node_graph, err);
    hipLaunchKernelGGL(k_check_nodes, grid_for(N), dim3(kBlock), 0, st, b->node_op, b->child_ptr,
                       b->child_idx, b->node_input, node_graph, N, b->num_inputs, ops, err);
    if (G > 0)
      hipLaunchKernelGGL(k_depth, dim3(G), dim3(kBlock), kDepthLdsInts * sizeof(int), st, b->graph_ptr,
                         b->child_ptr, b->child_idx, s.depth, indeg, scratch, err, meta);

    // sort by (depth - 1) * num_ops + op: as many 8-bit passes as N * num_ops could need are launched; the
    // ones the actual depth does not need copy their tile
    hipLaunchKernelGGL(k_sort_plan, dim3(1), dim3(64), 0, st, meta, K, err, meta + 2);
    hipLaunchKernelGGL(k_make_keys, grid_for(N), dim3(kBlock), 0, st, s.depth, b->node_op, N, K, ka, va, err);
    const unsigned long long max_key = std::min<unsigned long long>((unsigned long long)N * K,
                                                                    (unsigned long long)kMaxKeys) - 1;
    int bits = 1;
    while (bits < 32 && (max_key >> bits)) ++bits;
    const int passes = (bits + 7) / 8;
    for (int ps = 0; ps < passes; ++ps) {
      const int shift = 8 * ps;
      hipLaunchKernelGGL(k_radix_count, dim3(B), dim3(kBlock), 0, st, ka, N, shift, radix_counts, B, err,
                         meta + 2, ps);
      scan_exclusive(radix_counts, radix_counts, (int)rc, meta + 3, scan_tmp, st);
      hipLaunchKernelGGL(k_radix_scatter, dim3(B), dim3(kBlock), 0, st, ka, va, kb, vb, radix_counts, N, shift, B,
                         err, meta + 2, ps);
      std::swap(ka, kb);
      std::swap(va, vb);
    }
    int* gid = s.pos_group;
    hipLaunchKernelGGL(k_post_sort, grid_for(N), dim3(kBlock), 0, st, ka, va, N, K, s.pos_node, s.node_pos,
                       flag, s.level_ptr, err);
    scan_exclusive(flag, exs, N, meta + 4, scan_tmp, st);
    hipLaunchKernelGGL(k_group_starts, grid_for(N), dim3(kBlock), 0, st, ka, flag, exs, N, K, gid, s.g_level,
                       s.g_op, s.g_row_begin, err);
    hipLaunchKernelGGL(k_group_rows, grid_for(N), dim3(kBlock), 0, st, meta + 4, N, s.g_row_begin, s.g_op, ops,
                       s.g_rows, edges, err);
    // idx_off = exclusive scan of rows * arity over the groups (entries past the group count are unused)
    scan_exclusive(edges, s.g_idx_off, N, meta + 6, scan_tmp, st);
    hipLaunchKernelGGL(k_emit, grid_for(N), dim3(kBlock), 0, st, s.pos_node, s.node_pos, gid, s.g_row_begin,
                       s.g_op, s.g_idx_off, b->child_ptr, b->child_idx, b->node_input, indeg, N, ops, s.child_pos,
                       s.child_one, s.input_idx, s.pos_npar, err);
    hipLaunchKernelGGL(k_root_flags, grid_for(N), dim3(kBlock), 0, st, indeg, N, flag, err);
    scan_exclusive(flag, exs, N, meta + 5, scan_tmp, st);
    hipLaunchKernelGGL(k_root_emit, grid_for(N), dim3(kBlock), 0, st, flag, exs, s.node_pos, N, s.root_pos, err);

    // rows of every op in (op, row) order: one stable pass keyed by op (at most 256 ops: one digit)
    hipLaunchKernelGGL(k_op_keys, grid_for(N), dim3(kBlock), 0, st, gid, s.g_op, N, kb, vb, err);
    hipLaunchKernelGGL(k_radix_count, dim3(B), dim3(kBlock), 0, st, kb, N, 0, radix_counts, B, err,
                       (const int*)nullptr, 0);
    scan_exclusive(radix_counts, radix_counts, (int)rc, meta + 3, scan_tmp, st);
    hipLaunchKernelGGL(k_radix_scatter, dim3(B), dim3(kBlock), 0, st, kb, vb, ka, s.op_rows, radix_counts, N, 0, B,
                       err, (const int*)nullptr, 0);
    hipLaunchKernelGGL(k_op_rows, grid_for(N), dim3(kBlock), 0, st, s.op_rows, gid, s.g_row_begin, s.g_op,
                       s.g_idx_off, s.child_pos, s.input_idx, ops, N, s.op_cpos, s.op_inp, err);
    hipLaunchKernelGGL(k_cbase_init, grid_for(N), dim3(kBlock), 0, st, meta + 4, N, s.g_op, s.g_idx_off,
                       s.child_pos, s.child_one, ops, s.g_cbase0, s.g_cbase1, err);
    hipLaunchKernelGGL(k_cbase_check, grid_for(N), dim3(kBlock), 0, st, N, gid, s.g_row_begin, s.g_op,
                       s.g_idx_off, s.child_pos, s.child_one, ops, s.g_cbase0, s.g_cbase1, err);
  }
  GroupArrays ga{{s.g_level, s.g_op, s.g_row_begin, s.g_rows, s.g_idx_off, s.g_cbase0, s.g_cbase1}};
  hipLaunchKernelGGL(k_compact, dim3(1), dim3(kBlock), 0, st, err, meta, s.level_ptr, ga, kLcap, kGcap, stage);
  if (hipGetLastError() != hipSuccess) {
    set_error("fold_schedule: kernel launch failed");
    return fail(FOLD_E_DEVICE);
  }
  // the one synchronisation: error word, meta, and the level / group tables up to kLcap / kGcap entries
  std::vector<int> hb(stage_n, 0);
  if (hipMemcpyAsync(hb.data(), stage, stage_n * sizeof(int), hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipStreamSynchronize(st) != hipSuccess) {
    set_error("fold_schedule: device error while scheduling");
    return fail(FOLD_E_DEVICE);
  }
  const unsigned long long ew = (unsigned long long)(unsigned)hb[0] | ((unsigned long long)(unsigned)hb[1] << 32);
  if (ew != kNoErr) {
    std::string msg;
    int code = decode_error(ew, &msg);
    set_error(msg);
    return fail(code);
  }
  const int* hm = hb.data() + 2;
  const int D = N > 0 ? hm[0] : 0;
  const int ng = N > 0 ? hm[4] : 0;
  s.D = D;
  s.max_parents = N > 0 ? hm[1] : 0;
  s.num_groups = ng;
  s.R = N > 0 ? hm[5] : 0;
  if (N == 0) {
    s.h_level_ptr.assign(1, 0);
  } else if (D + 1 <= kLcap + 1 && ng <= kGcap) {
    const int* hl = hb.data() + kHdr;
    s.h_level_ptr.assign(hl, hl + D + 1);
    const int* hg = hl + kLcap + 1;
    s.h_level.assign(hg, hg + ng);
    s.h_op.assign(hg + kGcap, hg + kGcap + ng);
    s.h_row_begin.assign(hg + 2 * kGcap, hg + 2 * kGcap + ng);
    s.h_rows.assign(hg + 3 * kGcap, hg + 3 * kGcap + ng);
    s.h_idx_off.assign(hg + 4 * kGcap, hg + 4 * kGcap + ng);
    s.h_cbase0.assign(hg + 5 * kGcap, hg + 5 * kGcap + ng);
    s.h_cbase1.assign(hg + 6 * kGcap, hg + 6 * kGcap + ng);
  } else {
    // more levels or groups than the first read-back holds: read the whole tables (a second synchronisation)
    s.h_level_ptr.resize(D + 1);
    std::vector<int>* dst[kGroupArrays] = {&s.h_level, &s.h_op, &s.h_row_begin, &s.h_rows, &s.h_idx_off,
                                           &s.h_cbase0, &s.h_cbase1};
    bool ok = hipMemcpyAsync(s.h_level_ptr.data(), s.level_ptr, (size_t)(D + 1) * sizeof(int),
                             hipMemcpyDeviceToHost, st) == hipSuccess;
    for (int k = 0; k < kGroupArrays; ++k) {
      dst[k]->resize(ng);
      ok = ok && hipMemcpyAsync(dst[k]->data(), ga.a[k], (size_t)ng * sizeof(int), hipMemcpyDeviceToHost, st) ==
                     hipSuccess;
    }
    if (!ok || hipStreamSynchronize(st) != hipSuccess) {
      set_error("fold_schedule: device error while reading the group table");
      return fail(FOLD_E_DEVICE);
    }
  }
  // ranges of op_rows per op
  s.h_op_row_ptr.assign(K + 1, 0);
  for (int g = 0; g < ng; ++g) s.h_op_row_ptr[s.h_op[g] + 1] += s.h_rows[g];
  for (int o = 0; o < K; ++o) s.h_op_row_ptr[o + 1] += s.h_op_row_ptr[o];
  *out = h;
  return FOLD_OK;
}

void sched_destroy_impl(fold_sched* h) {
  if (!h) return;
  if (h->s.blob) (void)hipFree(h->s.blob);
  delete h;
}

}  // namespace fold
