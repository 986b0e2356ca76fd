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

__global__ void k_zero_ints(int* p, int n) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) p[i] = 0;
}

__global__ void k_fill_ints(int* p, long long n, int v) {
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (long long)gridDim.x * blockDim.x)
    p[i] = v;
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

// The leaf-table gradient adds dz . W_in^T of every row into its leaf-table row; it is linear in dz, so the
// backward first sums dz over the rows of each (op, leaf-table row) and contracts once per distinct row.  Third
// sort: pool rows by (op, leaf-table row) -- stable passes over the leaf-table row (rows without one: 0), then
// one by op -- and the runs of equal keys in the result.
__global__ void k_tok_keys(const int* input_idx, int N, unsigned* keys, int* vals, const unsigned long long* err) {
  if (*err != kNoErr) return;
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= N) return;
  keys[p] = (unsigned)max(input_idx[p], 0);
  vals[p] = p;
}
__global__ void k_tok_opkeys(const int* vals, const int* gid, const int* g_op, int N, unsigned* keys,
                             const unsigned long long* err) {
  if (*err != kNoErr) return;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= N) return;
  keys[i] = (unsigned)g_op[gid[vals[i]]];
}
__global__ void k_tok_flags(const int* tok_rows, const int* gid, const int* g_op, const int* input_idx, int N,
                            int* flag, const unsigned long long* err) {
  if (*err != kNoErr) return;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= N) return;
  const int p = tok_rows[i];
  int f = 1;
  if (i > 0) {
    const int q = tok_rows[i - 1];
    f = g_op[gid[p]] != g_op[gid[q]] || input_idx[p] != input_idx[q];
  }
  flag[i] = f;
}
__global__ void k_tok_emit(const int* flag, const int* exs, const int* tok_rows, const int* gid, const int* g_op,
                           const int* input_idx, int N, int* tok_start, int* tok_row, int* tok_seg, int* op_runs,
                           const unsigned long long* err) {
  if (*err != kNoErr) return;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  bool f = false;
  int op = -1;
  if (i < N) {
    const int p = tok_rows[i];
    f = flag[i] != 0;
    const int u = exs[i] + (f ? 1 : 0) - 1;
    tok_seg[i] = u;
    if (f) {
      tok_start[u] = i;
      tok_row[u] = input_idx[p];
      op = g_op[gid[p]];
    }
    if (i == N - 1) tok_start[u + 1] = N;
  }
  // runs per operation, one atomic add per operation and wave: the list is sorted by operation, so a wave's
  // run starts belong to one or a few of them (one add per run start would serialise on the same counter
  // when every row is a run of its own)
  unsigned long long m = __ballot(f);
  while (m) {
    const int leader = __ffsll((long long)m) - 1;
    const int lop = __shfl(op, leader);
    const unsigned long long same = __ballot(f && op == lop);
    if ((int)(threadIdx.x & 63) == leader) atomicAdd(&op_runs[lop], __popcll(same));
    m &= ~same;
  }
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
                          int lcap, int gcap, const int* op_runs, int num_ops, int* out) {
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
  for (int o = threadIdx.x; o < num_ops; o += blockDim.x) go[kGroupArrays * gcap + o] = op_runs[o];
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
  const size_t n1 = (size_t)N * 23 + 2 * (size_t)E + 17;
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
  s.tok_rows = q; q += N;
  s.tok_seg = q; q += N;
  s.tok_start = q; q += N + 1;
  s.tok_row = q; q += N;
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
  const size_t stage_n = kHdr + (kLcap + 1) + kGroupArrays * (size_t)kGcap + kMaxOps;
  int* op_runs = nullptr;  // [kMaxOps] runs of equal (op, leaf-table row) per op
  tmp.reserve(&em, 1);
  tmp.reserve(&stage, stage_n);
  tmp.reserve(&op_runs, kMaxOps);
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
  hipLaunchKernelGGL(k_zero_ints, dim3(1), dim3(kBlock), 0, st, op_runs, kMaxOps);
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

    // rows in (op, leaf-table row) order and their runs (only if some op reads the leaf table)
    bool any_input = false;
    for (int i = 0; i < K; ++i) any_input = any_input || b->ops[i].has_input;
    if (any_input) {
      int ibits = 1;
      while (ibits < 31 && ((long long)std::max(b->num_inputs - 1, 0) >> ibits)) ++ibits;
      hipLaunchKernelGGL(k_tok_keys, grid_for(N), dim3(kBlock), 0, st, s.input_idx, N, ka, va, err);
      for (int ps = 0; ps < (ibits + 7) / 8; ++ps) {
        hipLaunchKernelGGL(k_radix_count, dim3(B), dim3(kBlock), 0, st, ka, N, 8 * ps, radix_counts, B, err,
                           (const int*)nullptr, 0);
        scan_exclusive(radix_counts, radix_counts, (int)rc, meta + 3, scan_tmp, st);
        hipLaunchKernelGGL(k_radix_scatter, dim3(B), dim3(kBlock), 0, st, ka, va, kb, vb, radix_counts, N, 8 * ps,
                           B, err, (const int*)nullptr, 0);
        std::swap(ka, kb);
        std::swap(va, vb);
      }
      hipLaunchKernelGGL(k_tok_opkeys, grid_for(N), dim3(kBlock), 0, st, va, gid, s.g_op, N, ka, err);
      hipLaunchKernelGGL(k_radix_count, dim3(B), dim3(kBlock), 0, st, ka, N, 0, radix_counts, B, err,
                         (const int*)nullptr, 0);
      scan_exclusive(radix_counts, radix_counts, (int)rc, meta + 3, scan_tmp, st);
      hipLaunchKernelGGL(k_radix_scatter, dim3(B), dim3(kBlock), 0, st, ka, va, kb, s.tok_rows, radix_counts, N, 0,
                         B, err, (const int*)nullptr, 0);
      hipLaunchKernelGGL(k_tok_flags, grid_for(N), dim3(kBlock), 0, st, s.tok_rows, gid, s.g_op, s.input_idx, N,
                         flag, err);
      scan_exclusive(flag, exs, N, meta + 7, scan_tmp, st);
      hipLaunchKernelGGL(k_tok_emit, grid_for(N), dim3(kBlock), 0, st, flag, exs, s.tok_rows, gid, s.g_op,
                         s.input_idx, N, s.tok_start, s.tok_row, s.tok_seg, op_runs, err);
    }
  }
  GroupArrays ga{{s.g_level, s.g_op, s.g_row_begin, s.g_rows, s.g_idx_off, s.g_cbase0, s.g_cbase1}};
  hipLaunchKernelGGL(k_compact, dim3(1), dim3(kBlock), 0, st, err, meta, s.level_ptr, ga, kLcap, kGcap, op_runs, K,
                     stage);
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
  // ranges of op_rows per op, and of the runs of equal (op, leaf-table row) per op
  s.h_op_row_ptr.assign(K + 1, 0);
  for (int g = 0; g < ng; ++g) s.h_op_row_ptr[s.h_op[g] + 1] += s.h_rows[g];
  for (int o = 0; o < K; ++o) s.h_op_row_ptr[o + 1] += s.h_op_row_ptr[o];
  s.h_tok_ptr.assign(K + 1, 0);
  const int* hr = hb.data() + kHdr + (kLcap + 1) + kGroupArrays * kGcap;
  for (int o = 0; o < K; ++o) s.h_tok_ptr[o + 1] = s.h_tok_ptr[o] + (N > 0 ? hr[o] : 0);
  *out = h;
  return FOLD_OK;
}

void sched_destroy_impl(fold_sched* h) {
  if (!h) return;
  if (h->s.blob) (void)hipFree(h->s.blob);
  delete h;
}

// ================================================================ the paper's form: typed states
// Section 2's five steps on a typed DAG (constants of a tensor type as sources, operations with typed inputs
// and outputs, edges from a specific output), with the pass-throughs and per-(depth, type) concatenations
// made explicit.  Phase 1 validates, takes depths (the per-graph depth kernel above, whose constants sit at
// 1: the paper's depth is one less), lists the values (node, output slot), finds each value's deepest
// reader and counts its pass-through instances; one read-back sizes phase 2.  Phase 2 emits the
// pass-through instances, sorts operation nodes and pass-throughs by (depth, operation) (stable: node ids,
// then value order), cuts the batches, lays out each depth's concatenation per type (operation order, then
// output slot, then batch order) and writes every gather index.

namespace {

constexpr int kMaxTypedOps = 64, kMaxTypes = 16, kMaxSlots = 8;

struct TypedOpTable {
  int K, T;
  unsigned char nin[kMaxTypedOps], nout[kMaxTypedOps];
  unsigned char in_type[kMaxTypedOps][kMaxSlots], out_type[kMaxTypedOps][kMaxSlots];
  unsigned char out_rank[kMaxTypedOps][kMaxSlots];  // rank of output k among the op's outputs of its type
  unsigned char nout_t[kMaxTypedOps][kMaxTypes];    // the op's outputs of type t
};

__device__ __forceinline__ int t_nout(const TypedOpTable& o, int op) { return op < 0 ? 1 : o.nout[op]; }

__global__ void k_typed_check(const int* node_op, const int* in_ptr, const int* in_node, const int* in_slot,
                              const int* node_graph, int N, TypedOpTable ops, unsigned long long* err) {
  if (*err != kNoErr) return;
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= N) return;
  const int op = node_op[v], a = in_ptr[v], b = in_ptr[v + 1];
  if (op < 0) {
    if (-1 - op >= ops.T) report(err, v + 1, FOLD_E_OP);
    else if (b != a) report(err, v + 1, FOLD_E_INVALID);
    return;
  }
  if (op >= ops.K) { report(err, v + 1, FOLD_E_OP); return; }
  if (b - a != ops.nin[op]) { report(err, v + 1, FOLD_E_INVALID); return; }
  for (int j = 0; j < b - a; ++j) {
    const int u = in_node[a + j], k = in_slot[a + j];
    if (u < 0 || u >= N) { report(err, v + 1, FOLD_E_INVALID); return; }
    if (node_graph[u] != node_graph[v]) { report(err, v + 1, FOLD_E_CHILD); return; }
    const int uop = node_op[u];
    if (uop >= ops.K || (uop < 0 && -1 - uop >= ops.T)) continue;  // that node reports its own error
    if (k < 0 || k >= t_nout(ops, uop)) { report(err, v + 1, FOLD_E_INVALID); return; }
    const int tu = uop < 0 ? -1 - uop : ops.out_type[uop][k];
    if (tu != ops.in_type[op][j]) { report(err, v + 1, FOLD_E_INVALID); return; }
  }
}

// paper depth (constants 0), the number of values of each node, the number of constants of each type
__global__ void k_typed_nodes(const int* kdepth, const int* node_op, int N, TypedOpTable ops, int* depth,
                              int* nout_v, int* meta, const unsigned long long* err) {
  if (*err != kNoErr) return;
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= N) return;
  const int op = node_op[v];
  depth[v] = kdepth[v] - 1;
  nout_v[v] = t_nout(ops, op);
  if (op < 0) atomicAdd(&meta[8 + (-1 - op)], 1);
}

// last[value] = the deepest depth that reads it (its own depth if nobody does)
__global__ void k_typed_last_init(const int* depth, const int* nout_v, const int* val_ptr, int N, int* last,
                                  const unsigned long long* err) {
  if (*err != kNoErr) return;
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= N) return;
  for (int k = 0; k < nout_v[v]; ++k) last[val_ptr[v] + k] = depth[v];
}

__global__ void k_typed_last(const int* depth, const int* in_ptr, const int* in_node, const int* in_slot,
                             const int* val_ptr, int N, int* last, const unsigned long long* err) {
  if (*err != kNoErr) return;
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= N) return;
  for (int e = in_ptr[v]; e < in_ptr[v + 1]; ++e) atomicMax(&last[val_ptr[in_node[e]] + in_slot[e]], depth[v]);
}

// pass-through instances of every value: one per depth strictly between its own and its deepest reader's
__global__ void k_typed_npass(const int* depth, const int* nout_v, const int* val_ptr, const int* last, int N,
                              int* npass, const unsigned long long* err) {
  if (*err != kNoErr) return;
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= N) return;
  for (int k = 0; k < nout_v[v]; ++k) {
    const int q = val_ptr[v] + k;
    npass[q] = max(0, last[q] - depth[v] - 1);
  }
}

__global__ void k_typed_pass_emit(const int* depth, const int* nout_v, const int* val_ptr, const int* npass,
                                  const int* pass_ptr, int N, int* pass_node, int* pass_slot, int* pass_depth) {
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= N) return;
  for (int k = 0; k < nout_v[v]; ++k) {
    const int q = val_ptr[v] + k, p0 = pass_ptr[q];
    for (int j = 0; j < npass[q]; ++j) {
      pass_node[p0 + j] = v;
      pass_slot[p0 + j] = k;
      pass_depth[p0 + j] = depth[v] + 1 + j;
    }
  }
}

// sort keys (depth - 1) * (K + T) + op of operation nodes and pass-throughs (op K + t); constants get `sent`,
// past every real key, and sort to the end
__global__ void k_typed_keys(const int* depth, const int* node_op, int N, const int* pass_node, const int* pass_slot,
                             const int* pass_depth, int P, TypedOpTable ops, unsigned sent, unsigned* keys,
                             int* vals) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  const int KT = ops.K + ops.T;
  if (i < N) {
    const int op = node_op[i];
    keys[i] = op < 0 ? sent : (unsigned)((depth[i] - 1) * KT + op);
    vals[i] = i;
  } else if (i < N + P) {
    const int p = i - N, u = pass_node[p], uop = node_op[u];
    const int t = uop < 0 ? -1 - uop : ops.out_type[uop][pass_slot[p]];
    keys[i] = (unsigned)((pass_depth[p] - 1) * KT + ops.K + t);
    vals[i] = i;
  }
}

__global__ void k_typed_items(const unsigned* keys, const int* vals, int M, int N, int* item_node, int* flag) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= M) return;
  const int x = vals[i];
  item_node[i] = x < N ? x : -1 - (x - N);
  flag[i] = (i == 0 || keys[i] != keys[i - 1]) ? 1 : 0;
}

__global__ void k_typed_batches(const unsigned* keys, const int* flag, const int* exs, int M, int KT, int* bidx,
                                int* b_begin, int* b_depth, int* b_op) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= M) return;
  const int b = exs[i] + flag[i] - 1;
  bidx[i] = b;
  if (flag[i]) {
    b_begin[b] = i;
    b_depth[b] = (int)(keys[i] / (unsigned)KT) + 1;
    b_op[b] = (int)(keys[i] % (unsigned)KT);
  }
}

// per batch (entries past the batch count get zeros): rows, gather entries, and per type t its outputs of
// type t (rows * the op's outputs of type t) at cnt[t * M + b]
__global__ void k_typed_batch_sizes(const int* nb_ptr, int M, const int* b_begin, const int* b_op, TypedOpTable ops,
                                    int* b_rows, int* gcount, int* cnt) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= M) return;
  const int nb = *nb_ptr;
  if (b >= nb) {
    gcount[b] = 0;
    for (int t = 0; t < ops.T; ++t) cnt[(size_t)t * M + b] = 0;
    return;
  }
  const int rows = (b + 1 < nb ? b_begin[b + 1] : M) - b_begin[b];
  const int op = b_op[b];
  b_rows[b] = rows;
  gcount[b] = rows * (op < ops.K ? ops.nin[op] : 1);
  for (int t = 0; t < ops.T; ++t)
    cnt[(size_t)t * M + b] = rows * (op < ops.K ? ops.nout_t[op][t] : (op - ops.K == t ? 1 : 0));
}

// first and last batch of every depth
__global__ void k_typed_depth_span(const int* nb_ptr, const int* b_depth, int* dfirst, int* dlast) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  const int nb = *nb_ptr;
  if (b >= nb) return;
  const int d = b_depth[b];
  if (b == 0 || b_depth[b - 1] != d) dfirst[d] = b;
  if (b == nb - 1 || b_depth[b + 1] != d) dlast[d] = b;
}

// state sizes: depth 0 from the constants per type (meta[8 + t]), deeper ones from the batch scans
__global__ void k_typed_state_size(int D, int M, int T, const int* dfirst, const int* dlast, const int* cnt,
                                   const int* cscan, const int* meta, int* size) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (D + 1) * T) return;
  const int d = i / T, t = i - d * T;
  if (d == 0) {
    size[i] = meta[8 + t];
    return;
  }
  const size_t o = (size_t)t * M;
  size[i] = cscan[o + dlast[d]] + cnt[o + dlast[d]] - cscan[o + dfirst[d]];
}

// concatenation index of every constant: its rank among the constants of its type (flag scan of type t)
__global__ void k_typed_const_flag(const int* node_op, int N, int t, int* flag) {
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v < N) flag[v] = node_op[v] == -1 - t ? 1 : 0;
}
__global__ void k_typed_const_idx(const int* flag, const int* exs, const int* val_ptr, int N, int* vidx) {
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v < N && flag[v]) vidx[val_ptr[v]] = exs[v];
}

// concatenation index of every item's outputs at the item's depth: vidx[value] for operation nodes,
// pidx[p] for pass-through instance p
__global__ void k_typed_out_idx(const int* item_node, const int* bidx, const int* b_begin, const int* b_depth,
                                const int* b_op, const int* b_rows, const int* dfirst, const int* cscan, int M,
                                const int* val_ptr, TypedOpTable ops, int* vidx, int* pidx) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= M) return;
  const int b = bidx[i], r = i - b_begin[b], op = b_op[b], rows = b_rows[b], f = dfirst[b_depth[b]];
  const int x = item_node[i];
  if (op < ops.K) {
    for (int k = 0; k < ops.nout[op]; ++k) {
      const size_t o = (size_t)ops.out_type[op][k] * M;
      vidx[val_ptr[x] + k] = cscan[o + b] - cscan[o + f] + ops.out_rank[op][k] * rows + r;
    }
  } else {
    const size_t o = (size_t)(op - ops.K) * M;
    pidx[-1 - x] = cscan[o + b] - cscan[o + f] + r;
  }
}

// the label index of value (u, k) read at depth d: the value itself if it was made at d - 1, else its
// pass-through instance at d - 1
__device__ __forceinline__ int typed_label(const int* depth, const int* val_ptr, const int* vidx, const int* pass_ptr,
                                           const int* pidx, int u, int k, int d) {
  const int du = depth[u], q = val_ptr[u] + k;
  return du == d - 1 ? vidx[q] : pidx[pass_ptr[q] + (d - 2 - du)];
}

__global__ void k_typed_gather(const int* item_node, const int* bidx, const int* b_begin, const int* b_depth,
                               const int* b_op, const int* b_rows, const int* b_goff, int M, const int* depth,
                               const int* in_ptr, const int* in_node, const int* in_slot, const int* val_ptr,
                               const int* vidx, const int* pass_ptr, const int* pidx, const int* pass_node,
                               const int* pass_slot, TypedOpTable ops, int* gather, int* edge_index) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= M) return;
  const int b = bidx[i], r = i - b_begin[b], d = b_depth[b], rows = b_rows[b];
  const int x = item_node[i];
  int* g = gather + b_goff[b] + r;
  if (b_op[b] < ops.K) {
    for (int e = in_ptr[x], j = 0; e < in_ptr[x + 1]; ++e, ++j) {
      const int lab = typed_label(depth, val_ptr, vidx, pass_ptr, pidx, in_node[e], in_slot[e], d);
      g[j * rows] = lab;
      edge_index[e] = lab;
    }
  } else {
    const int p = -1 - x;
    g[0] = typed_label(depth, val_ptr, vidx, pass_ptr, pidx, pass_node[p], pass_slot[p], d);
  }
}

__global__ void k_typed_compact(const unsigned long long* err, const int* meta, const int* b_depth, const int* b_op,
                                const int* b_rows, const int* b_goff, const int* size, int nb, int nsize, int cap,
                                int* out) {
  const unsigned long long e = *err;
  if (threadIdx.x == 0) {
    out[0] = (int)(unsigned)(e & 0xffffffffull);
    out[1] = (int)(unsigned)(e >> 32);
    for (int i = 0; i < 14; ++i) out[2 + i] = meta[i];
  }
  if (e != kNoErr) return;
  const int n = min(nb, cap), ns = min(nsize, cap);
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    out[kHdr + i] = b_depth[i];
    out[kHdr + cap + i] = b_op[i];
    out[kHdr + 2 * cap + i] = b_rows[i];
    out[kHdr + 3 * cap + i] = b_goff[i];
  }
  for (int i = threadIdx.x; i < ns; i += blockDim.x) out[kHdr + 4 * cap + i] = size[i];
}

}  // namespace

void typed_sched_destroy_impl(fold_typed_sched* h) {
  if (!h) return;
  if (h->t.blob) (void)hipFree(h->t.blob);
  delete h;
}

int32_t schedule_typed_impl(const fold_typed_batch* b, hipStream_t st, fold_typed_sched** out) {
  const int N = b->num_nodes, E = b->num_edges, G = b->num_graphs, K = b->num_ops, T = b->num_types;
  if (K < 1 || K > kMaxTypedOps || T < 1 || T > kMaxTypes) {
    set_error("fold_schedule_typed: need 1..64 operations and 1..16 types");
    return FOLD_E_INVALID;
  }
  TypedOpTable ops{};
  ops.K = K;
  ops.T = T;
  for (int o = 0; o < K; ++o) {
    const fold_typed_op& op = b->ops[o];
    if (op.num_inputs < 1 || op.num_inputs > kMaxSlots || op.num_outputs < 1 || op.num_outputs > kMaxSlots ||
        !op.in_type || !op.out_type) {
      set_error("fold_schedule_typed: operation " + std::to_string(o) + " needs 1..8 inputs and 1..8 outputs");
      return FOLD_E_INVALID;
    }
    ops.nin[o] = (unsigned char)op.num_inputs;
    ops.nout[o] = (unsigned char)op.num_outputs;
    for (int j = 0; j < op.num_inputs; ++j) {
      if (op.in_type[j] < 0 || op.in_type[j] >= T) {
        set_error("fold_schedule_typed: operation " + std::to_string(o) + " has an input type out of range");
        return FOLD_E_INVALID;
      }
      ops.in_type[o][j] = (unsigned char)op.in_type[j];
    }
    for (int k = 0; k < op.num_outputs; ++k) {
      const int t = op.out_type[k];
      if (t < 0 || t >= T) {
        set_error("fold_schedule_typed: operation " + std::to_string(o) + " has an output type out of range");
        return FOLD_E_INVALID;
      }
      ops.out_type[o][k] = (unsigned char)t;
      ops.out_rank[o][k] = ops.nout_t[o][t]++;
    }
  }
  int device = 0;
  FOLD_HIP_CHECK(hipGetDevice(&device));
  init_pool_once(device);
  auto* h = new fold_typed_sched();
  TypedSched& s = h->t;
  s.N = N; s.E = E; s.K = K; s.T = T;
  auto fail = [&](int code) {
    typed_sched_destroy_impl(h);
    return code;
  };
  auto device_error = [&](const char* what) {
    set_error(std::string("fold_schedule_typed: ") + what);
    return fail(FOLD_E_DEVICE);
  };

  // phase 1 temporaries (kept to the end): N-sized, and values (at most 8 per node)
  const long long Vmax = 8LL * std::max(N, 1);
  Temp tmp1(st);
  struct ErrMeta {
    unsigned long long err;
    int meta[8 + kMaxTypes];  // [0] max depth + 1, [1] max parents, [2] values, [3] pass-throughs,
                              // [4] batches, [5] gather entries, [6, 7] scratch totals, [8 + t] constants of type t
  };
  static_assert(offsetof(ErrMeta, meta) == sizeof(unsigned long long), "k_init_meta's layout");
  ErrMeta* em = nullptr;
  int *node_graph = nullptr, *indeg = nullptr, *scratch = nullptr, *kdepth = nullptr, *depth = nullptr,
      *nout_v = nullptr, *val_ptr = nullptr, *last = nullptr, *npass = nullptr, *pass_ptr = nullptr,
      *scan_tmp1 = nullptr;
  tmp1.reserve(&em, 1);
  tmp1.reserve(&node_graph, N);
  tmp1.reserve(&indeg, N);
  tmp1.reserve(&scratch, (size_t)(6LL * N + G + E + 1));
  tmp1.reserve(&kdepth, N);
  tmp1.reserve(&depth, N);
  tmp1.reserve(&nout_v, N);
  tmp1.reserve(&val_ptr, N);
  tmp1.reserve(&last, Vmax);
  tmp1.reserve(&npass, Vmax);
  tmp1.reserve(&pass_ptr, Vmax);
  tmp1.reserve(&scan_tmp1, (size_t)(Vmax / kScanTile + 2));
  if (tmp1.commit() != hipSuccess) {
    set_error("fold_schedule_typed: out of device memory (temporaries)");
    return fail(FOLD_E_NOMEM);
  }
  unsigned long long* err = &em->err;
  int* meta = em->meta;
  hipLaunchKernelGGL(k_init_meta, dim3(1), dim3(64), 0, st, em);
  hipLaunchKernelGGL(k_zero_ints, dim3(1), dim3(64), 0, st, meta + 8, kMaxTypes);
  // pass counts of values past the last one stay 0, so the scan over the largest possible value count
  // yields the exact total
  hipLaunchKernelGGL(k_fill_ints, grid_for(std::min<long long>(Vmax, 1 << 20)), dim3(kBlock), 0, st, npass, Vmax, 0);
  hipLaunchKernelGGL(k_check_struct, grid_for(std::max(G + 1, N + 1)), dim3(kBlock), 0, st, b->graph_ptr, G,
                     b->in_ptr, N, E, err);
  if (N > 0) {
    if (G > 0) hipLaunchKernelGGL(k_node_graph, dim3(G), dim3(kBlock), 0, st, b->graph_ptr, node_graph, err);
    hipLaunchKernelGGL(k_typed_check, grid_for(N), dim3(kBlock), 0, st, b->node_op, b->in_ptr, b->in_node,
                       b->in_slot, node_graph, N, ops, err);
    if (G > 0)
      hipLaunchKernelGGL(k_depth, dim3(G), dim3(kBlock), kDepthLdsInts * sizeof(int), st, b->graph_ptr, b->in_ptr,
                         b->in_node, kdepth, indeg, scratch, err, meta);
    hipLaunchKernelGGL(k_typed_nodes, grid_for(N), dim3(kBlock), 0, st, kdepth, b->node_op, N, ops, depth, nout_v,
                       meta, err);
    scan_exclusive(nout_v, val_ptr, N, meta + 2, scan_tmp1, st);
    hipLaunchKernelGGL(k_typed_last_init, grid_for(N), dim3(kBlock), 0, st, depth, nout_v, val_ptr, N, last, err);
    hipLaunchKernelGGL(k_typed_last, grid_for(N), dim3(kBlock), 0, st, depth, b->in_ptr, b->in_node, b->in_slot,
                       val_ptr, N, last, err);
    hipLaunchKernelGGL(k_typed_npass, grid_for(N), dim3(kBlock), 0, st, depth, nout_v, val_ptr, last, N, npass, err);
    scan_exclusive(npass, pass_ptr, (int)Vmax, meta + 3, scan_tmp1, st);
  }
  if (hipGetLastError() != hipSuccess) return device_error("kernel launch failed");
  // first synchronisation: the error word, the depth, and the sizes of phase 2
  ErrMeta hm{};
  if (hipMemcpyAsync(&hm, em, sizeof(hm), hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipStreamSynchronize(st) != hipSuccess)
    return device_error("device error while validating");
  if (hm.err != kNoErr) {
    std::string msg;
    int code = decode_error(hm.err, &msg);
    set_error("fold_schedule_typed" + msg.substr(msg.find(':')));
    return fail(code);
  }
  const int D = N > 0 ? hm.meta[0] - 1 : 0;
  const int V = N > 0 ? hm.meta[2] : 0;
  const int P = N > 0 ? hm.meta[3] : 0;
  if ((long long)(D + 1) * (K + T) > kMaxKeys) {
    set_error("fold_schedule_typed: depth * (operations + types) exceeds 2^30 (the sort keys)");
    return fail(FOLD_E_INVALID);
  }
  int nconst = 0;
  for (int t = 0; t < T; ++t) nconst += hm.meta[8 + t];
  const int M = N - nconst + P;  // items: operation nodes and pass-through instances
  s.D = D; s.P = P; s.M = M;
  const int ngather = E + P;
  s.ngather = ngather;

  // persistent arrays, now that P is known
  const size_t nsize = (size_t)(D + 1) * T;
  const size_t Mc = std::max(M, 1);
  const size_t n_int = (size_t)N + 6 * Mc + (size_t)std::max(ngather, 1) + 3 * (size_t)std::max(P, 1) + nsize +
                       (size_t)std::max(E, 1) + 16;
  if (hipMalloc(&s.blob, n_int * sizeof(int)) != hipSuccess) {
    set_error("fold_schedule_typed: out of device memory");
    return fail(FOLD_E_NOMEM);
  }
  int* q = static_cast<int*>(s.blob);
  s.depth = q; q += N;
  s.batch_depth = q; q += Mc;
  s.batch_op = q; q += Mc;
  s.batch_rows = q; q += Mc;
  s.batch_goff = q; q += Mc;
  s.batch_begin = q; q += Mc;
  s.item_node = q; q += Mc;
  s.gather = q; q += std::max(ngather, 1);
  s.pass_node = q; q += std::max(P, 1);
  s.pass_slot = q; q += std::max(P, 1);
  s.pass_depth = q; q += std::max(P, 1);
  s.state_size = q; q += nsize;
  s.edge_index = q; q += std::max(E, 1);
  if (N > 0 && hipMemcpyAsync(s.depth, depth, (size_t)N * sizeof(int), hipMemcpyDeviceToDevice, st) != hipSuccess)
    return device_error("copy of the depths failed");

  // phase 2
  const int NI = N + P;  // sort entries: every node (constants sort last) and every pass-through
  const int B = (NI + kRadixTile - 1) / kRadixTile;
  const long long rc = 256LL * std::max(B, 1);
  Temp tmp2(st);
  unsigned *ka = nullptr, *kb = nullptr;
  int *va = nullptr, *vb = nullptr, *flag = nullptr, *exs = nullptr, *radix_counts = nullptr, *scan_tmp = nullptr;
  int *bidx = nullptr, *gcount = nullptr, *cnt = nullptr, *cscan = nullptr, *dspan = nullptr, *vidx = nullptr,
      *pidx = nullptr, *stage = nullptr;
  constexpr int kCap = 4096;  // batches and state sizes read back with the final error word
  const size_t stage_n = kHdr + 5 * (size_t)kCap;
  const long long scan_n = std::max<long long>(std::max<long long>(rc, NI), (long long)T * Mc);
  tmp2.reserve(&stage, stage_n);
  tmp2.reserve(&ka, std::max(NI, 1));
  tmp2.reserve(&kb, std::max(NI, 1));
  tmp2.reserve(&va, std::max(NI, 1));
  tmp2.reserve(&vb, std::max(NI, 1));
  tmp2.reserve(&flag, std::max(NI, 1));
  tmp2.reserve(&exs, std::max(NI, 1));
  tmp2.reserve(&radix_counts, rc);
  tmp2.reserve(&scan_tmp, (size_t)(scan_n / kScanTile + 2));
  tmp2.reserve(&bidx, Mc);
  tmp2.reserve(&gcount, Mc);
  tmp2.reserve(&cnt, (size_t)T * Mc);
  tmp2.reserve(&cscan, (size_t)T * Mc);
  tmp2.reserve(&dspan, 2 * (size_t)(D + 1));
  tmp2.reserve(&vidx, std::max(V, 1));
  tmp2.reserve(&pidx, std::max(P, 1));
  if (tmp2.commit() != hipSuccess) {
    set_error("fold_schedule_typed: out of device memory (temporaries)");
    return fail(FOLD_E_NOMEM);
  }
  int* dfirst = dspan;
  int* dlast = dspan + (D + 1);
  const int KT = K + T;
  if (N > 0) {
    if (P > 0)
      hipLaunchKernelGGL(k_typed_pass_emit, grid_for(N), dim3(kBlock), 0, st, depth, nout_v, val_ptr, npass, pass_ptr,
                         N, s.pass_node, s.pass_slot, s.pass_depth);
    const unsigned sent = (unsigned)(D * KT);
    hipLaunchKernelGGL(k_typed_keys, grid_for(NI), dim3(kBlock), 0, st, depth, b->node_op, N, s.pass_node,
                       s.pass_slot, s.pass_depth, P, ops, sent, ka, va);
    int bits = 1;
    while (bits < 32 && ((unsigned long long)sent >> bits)) ++bits;
    const int passes = (bits + 7) / 8;
    for (int ps = 0; ps < passes; ++ps) {
      hipLaunchKernelGGL(k_radix_count, dim3(B), dim3(kBlock), 0, st, ka, NI, 8 * ps, radix_counts, B, err,
                         (const int*)nullptr, 0);
      scan_exclusive(radix_counts, radix_counts, (int)rc, meta + 6, scan_tmp, st);
      hipLaunchKernelGGL(k_radix_scatter, dim3(B), dim3(kBlock), 0, st, ka, va, kb, vb, radix_counts, NI, 8 * ps, B,
                         err, (const int*)nullptr, 0);
      std::swap(ka, kb);
      std::swap(va, vb);
    }
    if (M > 0) {
      hipLaunchKernelGGL(k_typed_items, grid_for(M), dim3(kBlock), 0, st, ka, va, M, N, s.item_node, flag);
      scan_exclusive(flag, exs, M, meta + 4, scan_tmp, st);
      hipLaunchKernelGGL(k_typed_batches, grid_for(M), dim3(kBlock), 0, st, ka, flag, exs, M, KT, bidx,
                         s.batch_begin, s.batch_depth, s.batch_op);
      hipLaunchKernelGGL(k_typed_batch_sizes, grid_for(M), dim3(kBlock), 0, st, meta + 4, M, s.batch_begin,
                         s.batch_op, ops, s.batch_rows, gcount, cnt);
      scan_exclusive(gcount, s.batch_goff, M, meta + 5, scan_tmp, st);
      for (int t = 0; t < T; ++t)
        scan_exclusive(cnt + (size_t)t * M, cscan + (size_t)t * M, M, meta + 7, scan_tmp, st);
      hipLaunchKernelGGL(k_typed_depth_span, grid_for(M), dim3(kBlock), 0, st, meta + 4, s.batch_depth, dfirst, dlast);
    }
    hipLaunchKernelGGL(k_typed_state_size, grid_for((long long)nsize), dim3(kBlock), 0, st, D, std::max(M, 1), T,
                       dfirst, dlast, cnt, cscan, meta, s.state_size);
    for (int t = 0; t < T; ++t) {
      hipLaunchKernelGGL(k_typed_const_flag, grid_for(N), dim3(kBlock), 0, st, b->node_op, N, t, flag);
      scan_exclusive(flag, exs, N, meta + 7, scan_tmp, st);
      hipLaunchKernelGGL(k_typed_const_idx, grid_for(N), dim3(kBlock), 0, st, flag, exs, val_ptr, N, vidx);
    }
    if (M > 0) {
      hipLaunchKernelGGL(k_typed_out_idx, grid_for(M), dim3(kBlock), 0, st, s.item_node, bidx, s.batch_begin,
                         s.batch_depth, s.batch_op, s.batch_rows, dfirst, cscan, M, val_ptr, ops, vidx, pidx);
      hipLaunchKernelGGL(k_typed_gather, grid_for(M), dim3(kBlock), 0, st, s.item_node, bidx, s.batch_begin,
                         s.batch_depth, s.batch_op, s.batch_rows, s.batch_goff, M, depth, b->in_ptr, b->in_node,
                         b->in_slot, val_ptr, vidx, pass_ptr, pidx, s.pass_node, s.pass_slot, ops, s.gather,
                         s.edge_index);
    }
  }
  // batches <= items; read back the batch table and the state sizes up to kCap entries each
  hipLaunchKernelGGL(k_typed_compact, dim3(1), dim3(kBlock), 0, st, err, meta, s.batch_depth, s.batch_op,
                     s.batch_rows, s.batch_goff, s.state_size, M, (int)nsize, kCap, stage);
  if (hipGetLastError() != hipSuccess) return device_error("kernel launch failed");
  std::vector<int> hb(stage_n, 0);
  if (hipMemcpyAsync(hb.data(), stage, stage_n * sizeof(int), hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipStreamSynchronize(st) != hipSuccess)
    return device_error("device error while scheduling");
  const int nb = M > 0 ? hb[2 + 4] : 0;
  s.nb = nb;
  if (nb <= kCap && (int)nsize <= kCap) {
    const int* hs = hb.data() + kHdr;
    s.h_depth_b.assign(hs, hs + nb);
    s.h_op_b.assign(hs + kCap, hs + kCap + nb);
    s.h_rows_b.assign(hs + 2 * kCap, hs + 2 * kCap + nb);
    s.h_goff_b.assign(hs + 3 * kCap, hs + 3 * kCap + nb);
    s.h_state_size.assign(hs + 4 * kCap, hs + 4 * kCap + nsize);
  } else {
    std::vector<int>* dst[4] = {&s.h_depth_b, &s.h_op_b, &s.h_rows_b, &s.h_goff_b};
    const int* src[4] = {s.batch_depth, s.batch_op, s.batch_rows, s.batch_goff};
    bool ok = true;
    for (int k = 0; k < 4; ++k) {
      dst[k]->resize(nb);
      ok = ok && hipMemcpyAsync(dst[k]->data(), src[k], (size_t)nb * sizeof(int), hipMemcpyDeviceToHost, st) ==
                     hipSuccess;
    }
    s.h_state_size.resize(nsize);
    ok = ok && hipMemcpyAsync(s.h_state_size.data(), s.state_size, nsize * sizeof(int), hipMemcpyDeviceToHost, st) ==
                   hipSuccess;
    if (!ok || hipStreamSynchronize(st) != hipSuccess) return device_error("device error while reading the batches");
  }
  *out = h;
  return FOLD_OK;
}

}  // namespace fold
