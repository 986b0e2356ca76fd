// Feed-forward attention operations (Section 3.4, Appendix A), gfx950.
//
// e_t = a(h_t) with a(h) = w . h + b, alpha = softmax(e), c = sum_t alpha_t h_t.  The two sums over t (the
// softmax normaliser and the weighted sum of the items) are carried together as the aggregate of a set of
// scored items, (m, s, acc) = (max e, sum exp(e - m), sum exp(e - m) h), which a node keeps as h = acc and
// c = [m, s, 0, ...].  Merging two aggregates is associative, so the sums run as a Reduce of pairwise merges
// that batch by depth like every other operation:
//   ATTN_SCORE  one item:            e = w . h_c + b;  h = h_c, c = [e, 1, 0..]
//   ATTN_SUM    union of two sets:   m = max(m_1, m_2), x_k = exp(m_k - m), s = x_1 s_1 + x_2 s_2,
//                                    acc = x_1 acc_1 + x_2 acc_2 (a child with s = 0 is the empty set)
//   ATTN_OUT    the attention output: h = acc / s (0 for the empty set), c = 0
// The value acc / s does not depend on m, so the gradients hold m fixed; they are the exact derivatives of
// acc / s with respect to the items and the scores.
//
// The operations are O(H) per node and HBM-bound: one wave per pool row (four rows per workgroup), each lane
// owning four consecutive columns of every 256 (16-byte fp32, 8-byte bf16 accesses); the dot products of the
// scorer and of the output's backward are wave sums of a fixed butterfly order.  The backward adds into the children's dh / dc directly (a plain
// read-add-write for a child with one parent edge, a hardware fp32 atomic otherwise), so no dz . W^T pass
// follows.  The scorer's weight gradient, dw = sum_r de_r h_c(r) and db = sum_r de_r, is reduced in fixed
// order (rows within a chunk, chunks within a quarter, quarters) from the de each row's backward saves.

#include <hip/hip_runtime.h>

#include <algorithm>

#include "common.h"
#include "internal.h"
#include "mfma.h"

namespace fold {

namespace {

constexpr int kRowsPerBlock = 4;  // one wave per row

// the dot products (scores, de, dh . acc) accumulate in fp64: their results can cancel far below their terms,
// and these kernels are bound by HBM, not by arithmetic
__device__ __forceinline__ double wave_total(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// four consecutive columns j .. j + 3 of a row (j a multiple of 4; rows are multiples of 64 wide)
__device__ __forceinline__ void ld4(const float* p, float (&v)[4]) {
  const float4 t = *reinterpret_cast<const float4*>(p);
  v[0] = t.x, v[1] = t.y, v[2] = t.z, v[3] = t.w;
}
__device__ __forceinline__ void ld4(const uint16_t* p, float (&v)[4]) {
  const uint2 t = *reinterpret_cast<const uint2*>(p);
  v[0] = bf2f(t.x & 0xffff), v[1] = bf2f(t.x >> 16), v[2] = bf2f(t.y & 0xffff), v[3] = bf2f(t.y >> 16);
}
__device__ __forceinline__ void st4(float* p, const float (&v)[4]) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ void st4(uint16_t* p, const float (&v)[4]) {
  *reinterpret_cast<uint2*>(p) = make_uint2(f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16),
                                            f2bf(v[2]) | ((uint32_t)f2bf(v[3]) << 16));
}
// columns j .. j + 3 of pool row `row` (zero for the zero state and past H)
template <typename T>
__device__ __forceinline__ void ld_h4(const T* h, int row, int ld, int H, int j, float (&v)[4]) {
  if (row >= 0) {
    ld4(h + (size_t)row * ld + j, v);
  } else {
    v[0] = v[1] = v[2] = v[3] = 0.f;
  }
#pragma unroll
  for (int e = 0; e < 4; ++e)
    if (j + e >= H) v[e] = 0.f;
}
// the c row of an attention node: (m, s) in columns 0 and 1, zeros after
__device__ __forceinline__ void put_ms(float* co, int ld, int lane, float m, float s) {
  for (int j = 4 * lane; j < ld; j += 4 * kWave) {
    const float v[4] = {j == 0 ? m : 0.f, j == 0 ? s : 0.f, 0.f, 0.f};
    st4(co + j, v);
  }
}

// A child's gradient row gets v at columns j .. j + 3: stored when the child has one parent edge and its row
// starts undefined (fresh), read-add-written when it has one parent edge, fp32 atomics on a zeroed row otherwise.
__device__ __forceinline__ void add4(float* dst, const float (&v)[4], bool single, bool fresh) {
  if (single && fresh) {
    st4(dst, v);
  } else if (single) {
    float o[4];
    ld4(dst, o);
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] += v[e];
    st4(dst, o);
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) unsafeAtomicAdd(dst + e, v[e]);
  }
}
// A child's dc row, whose only nonzero entry is column 1 (ds): a child with one parent edge gets the whole row
// stored (its row is never initialised), a shared child an atomic add of ds into its zeroed row.
__device__ __forceinline__ void ds_to(float* row, int ld, int lane, float ds, bool single) {
  if (single) {
    put_ms(row, ld, lane, 0.f, ds);
  } else if (lane == 0 && ds != 0.f) {
    unsafeAtomicAdd(row + 1, ds);
  }
}
// Lanes own four consecutive columns each, 256 columns a wave step.
template <typename T, int KIND>
__global__ __launch_bounds__(kRowsPerBlock* kWave) void k_attn_fwd(AttnArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const int row = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  if (row >= a.rows) return;
  const size_t p = (size_t)(a.row_begin + row);
  const T* hp = static_cast<const T*>(a.h_pool);
  T* ho = static_cast<T*>(a.h_pool) + p * a.ld;
  float* co = a.c_pool + p * a.ld;
  if constexpr (KIND == FOLD_ATTN_SCORE) {
    const int c0 = a.child_pos[a.idx_off + row];
    const T* w = static_cast<const T*>(a.w);
    double part = 0.0;
    for (int j = 4 * lane; j < a.ld; j += 4 * kWave) {
      float v[4], wv[4];
      ld_h4(hp, c0, a.ld, a.H, j, v);
      ld4(w + j, wv);  // zero past H
#pragma unroll
      for (int e = 0; e < 4; ++e) part += (double)v[e] * wv[e];
      st4(ho + j, v);
    }
    const float e = (float)(wave_total(part) + a.bias[0]);
    put_ms(co, a.ld, lane, e, 1.f);
  } else if constexpr (KIND == FOLD_ATTN_SUM) {
    const int c0 = a.child_pos[a.idx_off + 2 * row], c1 = a.child_pos[a.idx_off + 2 * row + 1];
    const float m0 = c0 >= 0 ? a.c_pool[(size_t)c0 * a.ld] : 0.f, s0 = c0 >= 0 ? a.c_pool[(size_t)c0 * a.ld + 1] : 0.f;
    const float m1 = c1 >= 0 ? a.c_pool[(size_t)c1 * a.ld] : 0.f, s1 = c1 >= 0 ? a.c_pool[(size_t)c1 * a.ld + 1] : 0.f;
    const bool l0 = s0 != 0.f, l1 = s1 != 0.f;
    const float m = l0 && l1 ? fmaxf(m0, m1) : (l0 ? m0 : m1);
    const float x0 = l0 ? fast_exp(m0 - m) : 0.f, x1 = l1 ? fast_exp(m1 - m) : 0.f;
    for (int j = 4 * lane; j < a.ld; j += 4 * kWave) {
      float v0[4], v1[4], v[4];
      ld_h4(hp, l0 ? c0 : -1, a.ld, a.H, j, v0);
      ld_h4(hp, l1 ? c1 : -1, a.ld, a.H, j, v1);
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = x0 * v0[e] + x1 * v1[e];
      st4(ho + j, v);
    }
    put_ms(co, a.ld, lane, l0 || l1 ? m : 0.f, x0 * s0 + x1 * s1);
  } else {  // FOLD_ATTN_OUT
    const int c0 = a.child_pos[a.idx_off + row];
    const float s = c0 >= 0 ? a.c_pool[(size_t)c0 * a.ld + 1] : 0.f;
    for (int j = 4 * lane; j < a.ld; j += 4 * kWave) {
      float v[4];
      ld_h4(hp, s != 0.f ? c0 : -1, a.ld, a.H, j, v);
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = s != 0.f ? v[e] / s : 0.f;
      st4(ho + j, v);
    }
    put_ms(co, a.ld, lane, 0.f, 0.f);
  }
}

template <typename T, int KIND>
__global__ __launch_bounds__(kRowsPerBlock* kWave) void k_attn_bwd(AttnArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const int row = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  if (row >= a.rows) return;
  const size_t p = (size_t)(a.row_begin + row);
  const T* hp = static_cast<const T*>(a.h_pool);
  const float* dh = a.dh + p * a.ld;
  if constexpr (KIND == FOLD_ATTN_SCORE) {
    // de = dh . h_c + dc[1] (d acc / de = acc = h_c and d s / de = s = 1 at e = m); dh_c += dh + de w
    const int c0 = a.child_pos[a.idx_off + row];
    const bool one = a.child_one[a.idx_off + row] != 0;
    const T* w = static_cast<const T*>(a.w);
    double part = 0.0;
    for (int j = 4 * lane; j < a.ld; j += 4 * kWave) {
      float g[4], v[4];
      ld4(dh + j, g);
      ld_h4(hp, c0, a.ld, a.H, j, v);
#pragma unroll
      for (int e = 0; e < 4; ++e) part += (double)g[e] * v[e];
    }
    const float de = (float)(wave_total(part) + a.dc[p * a.ld + 1]);
    if (lane == 0 && a.gates) a.gates[p * a.gstride] = de;
    if (c0 >= 0) {
      for (int j = 4 * lane; j < a.ld; j += 4 * kWave) {
        float g[4], wv[4];
        ld4(dh + j, g);
        ld4(w + j, wv);
#pragma unroll
        for (int e = 0; e < 4; ++e) g[e] = j + e < a.H ? g[e] + de * wv[e] : 0.f;
        add4(&a.dh[(size_t)c0 * a.ld + j], g, one, a.dh_fresh);
      }
      ds_to(a.dc + (size_t)c0 * a.ld, a.ld, lane, 0.f, one);  // an item passes no cell-state gradient down
    }
  } else if constexpr (KIND == FOLD_ATTN_SUM) {
    // with m fixed, acc and s are linear in the children's: dh_k += x_k dh, ds_k += x_k ds
    const float m = a.c_pool[p * a.ld];
    const float ds = a.dc[p * a.ld + 1];
    int ck[2];
    float xk[2];
    bool one[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      ck[k] = a.child_pos[a.idx_off + 2 * row + k];
      one[k] = a.child_one[a.idx_off + 2 * row + k] != 0;
      // an empty set (s = 0) takes no part: x_k = 0; else the forward's x_k, bit for bit
      xk[k] = ck[k] >= 0 && a.c_pool[(size_t)ck[k] * a.ld + 1] != 0.f ? fast_exp(a.c_pool[(size_t)ck[k] * a.ld] - m)
                                                                      : 0.f;
    }
    for (int j = 4 * lane; j < a.ld; j += 4 * kWave) {
      float g[4];
      ld4(dh + j, g);
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        // an empty set's gradient is zero: stored into a child's row that starts undefined, skipped otherwise
        if (ck[k] < 0 || (xk[k] == 0.f && !(one[k] && a.dh_fresh))) continue;
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = j + e < a.H ? xk[k] * g[e] : 0.f;
        add4(&a.dh[(size_t)ck[k] * a.ld + j], v, one[k], a.dh_fresh);
      }
    }
#pragma unroll
    for (int k = 0; k < 2; ++k)
      if (ck[k] >= 0) ds_to(a.dc + (size_t)ck[k] * a.ld, a.ld, lane, xk[k] * ds, one[k]);
  } else {  // FOLD_ATTN_OUT: h = acc / s -> dacc = dh / s, ds = -(dh . acc) / s^2
    const int c0 = a.child_pos[a.idx_off + row];
    if (c0 < 0) return;
    const float s = a.c_pool[(size_t)c0 * a.ld + 1];
    const bool one = a.child_one[a.idx_off + row] != 0;
    if (s == 0.f) {  // attention over the empty set: a zero gradient, stored into rows nobody else writes
      if (one) {
        const float z[4] = {0.f, 0.f, 0.f, 0.f};
        if (a.dh_fresh)
          for (int j = 4 * lane; j < a.ld; j += 4 * kWave) st4(&a.dh[(size_t)c0 * a.ld + j], z);
        put_ms(a.dc + (size_t)c0 * a.ld, a.ld, lane, 0.f, 0.f);
      }
      return;
    }
    double part = 0.0;
    for (int j = 4 * lane; j < a.ld; j += 4 * kWave) {
      float g[4], v[4];
      ld4(dh + j, g);
      ld_h4(hp, c0, a.ld, a.H, j, v);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        part += (double)g[e] * v[e];
        g[e] = j + e < a.H ? g[e] / s : 0.f;
      }
      add4(&a.dh[(size_t)c0 * a.ld + j], g, one, a.dh_fresh);
    }
    const double tot = wave_total(part);
    ds_to(a.dc + (size_t)c0 * a.ld, a.ld, lane, (float)(-tot / ((double)s * s)), one);
  }
}

// Partial sums of the scorer's gradient over chunks of kAttnWgradChunk op rows (workgroup x) and 256 columns
// (workgroup y): column j < H of chunk q is sum_r de_r h_c(r)[j]; column HP holds sum_r de_r (first column
// block).  The chunk's de and child rows are staged in LDS first; then each of the four waves sums a quarter of
// the rows in order, a lane over four consecutive columns (sixteen rows' loads in flight), and the waves' sums
// are added in wave order.
template <typename T>
__global__ __launch_bounds__(256) void k_attn_wgrad(const int* op_rows, const int* op_cpos, int count, int H,
                                                    int HP, int ld, const T* h_pool, const float* gates,
                                                    int gstride, float* part) {
  constexpr int kQ = kAttnWgradChunk / 4;  // rows per wave
  __shared__ float sde[kAttnWgradChunk];
  __shared__ int sch[kAttnWgradChunk];
  __shared__ float red[4][256];
  const int q0 = blockIdx.x * kAttnWgradChunk, n = min(count, q0 + kAttnWgradChunk) - q0;
  for (int t = threadIdx.x; t < n; t += blockDim.x) {
    sde[t] = gates[(size_t)op_rows[q0 + t] * gstride];
    sch[t] = op_cpos[2 * (size_t)(q0 + t)];
  }
  __syncthreads();
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x >> 6;
  const int jl = 4 * lane, j = blockIdx.y * 256 + jl;  // this lane's four columns (j < ld: rows are 64-wide)
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  const int t0 = w * kQ, t1 = min(n, t0 + kQ);
  if (j < H) {
    for (int t = t0; t < t1; t += 16) {
      float v[16][4];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int c = t + u < t1 ? sch[t + u] : -1;
        if (c >= 0)
          ld4(h_pool + (size_t)c * ld + j, v[u]);
        else
          v[u][0] = v[u][1] = v[u][2] = v[u][3] = 0.f;
      }
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const float d = t + u < t1 ? sde[t + u] : 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[e] += d * v[u][e];
      }
    }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) red[w][jl + e] = acc[e];
  __syncthreads();
  float* out = part + (size_t)blockIdx.x * (HP + kPadK);
  const int c = blockIdx.y * 256 + threadIdx.x;
  if (c < H) out[c] = ((red[0][threadIdx.x] + red[1][threadIdx.x]) + red[2][threadIdx.x]) + red[3][threadIdx.x];
  if (blockIdx.y == 0 && threadIdx.x == 0) {
    float bsum = 0.f;
    for (int t = 0; t < n; ++t) bsum += sde[t];
    out[HP] = bsum;
  }
}

// Sum of the chunks' partials, 64 columns (column H: the bias) per workgroup: the four waves sum a quarter
// of the chunks each, in chunk order, and their sums are added in wave order.
__global__ __launch_bounds__(256) void k_attn_wgrad_reduce(const float* part, int nchunk, int H, int HP, float* dw,
                                                           float* db) {
  __shared__ float red[4][kWave];
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x >> 6;
  const int jc = blockIdx.x * kWave + lane;  // 0 .. H (H: the bias)
  const bool live = jc <= H;
  const int col = jc < H ? jc : HP;
  const int per = (nchunk + 3) / 4, q0 = min(nchunk, w * per), q1 = min(nchunk, q0 + per);
  float acc = 0.f;
  if (live) {
    int q = q0;
    for (; q + 8 <= q1; q += 8) {
      float t[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) t[u] = part[(size_t)(q + u) * (HP + kPadK) + col];
#pragma unroll
      for (int u = 0; u < 8; ++u) acc += t[u];
    }
    for (; q < q1; ++q) acc += part[(size_t)q * (HP + kPadK) + col];
  }
  red[w][lane] = acc;
  __syncthreads();
  if (w != 0 || !live) return;
  const float tot = ((red[0][lane] + red[1][lane]) + red[2][lane]) + red[3][lane];
  if (jc < H) {
    if (dw) dw[jc] += tot;
  } else if (db) {
    db[0] += tot;
  }
}

// scorer vector (H entries of the params' type) -> HP entries, zero padded; bias [1] -> 64 floats
template <typename T>
__global__ void k_pack_score(int H, int HP, const T* w, const float* b, T* wdst, float* bdst) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j < HP) wdst[j] = j < H ? w[j] : from_f32<T>(0.f);
  if (j < kPadK) bdst[j] = j == 0 ? b[0] : 0.f;
}

template <typename T>
void attn_fwd_t(int kind, const AttnArgs& a, hipStream_t st) {
  const dim3 grid((unsigned)((a.rows + kRowsPerBlock - 1) / kRowsPerBlock)), block(kRowsPerBlock * kWave);
  switch (kind) {
    case FOLD_ATTN_SCORE: hipLaunchKernelGGL((k_attn_fwd<T, FOLD_ATTN_SCORE>), grid, block, 0, st, a); break;
    case FOLD_ATTN_SUM: hipLaunchKernelGGL((k_attn_fwd<T, FOLD_ATTN_SUM>), grid, block, 0, st, a); break;
    case FOLD_ATTN_OUT: hipLaunchKernelGGL((k_attn_fwd<T, FOLD_ATTN_OUT>), grid, block, 0, st, a); break;
    default: break;
  }
}

template <typename T>
void attn_bwd_t(int kind, const AttnArgs& a, hipStream_t st) {
  const dim3 grid((unsigned)((a.rows + kRowsPerBlock - 1) / kRowsPerBlock)), block(kRowsPerBlock * kWave);
  switch (kind) {
    case FOLD_ATTN_SCORE: hipLaunchKernelGGL((k_attn_bwd<T, FOLD_ATTN_SCORE>), grid, block, 0, st, a); break;
    case FOLD_ATTN_SUM: hipLaunchKernelGGL((k_attn_bwd<T, FOLD_ATTN_SUM>), grid, block, 0, st, a); break;
    case FOLD_ATTN_OUT: hipLaunchKernelGGL((k_attn_bwd<T, FOLD_ATTN_OUT>), grid, block, 0, st, a); break;
    default: break;
  }
}

const char* attn_name(int kind, bool fwd) {
  switch (kind) {
    case FOLD_ATTN_SCORE: return fwd ? "attn_fwd.score" : "attn_bwd.score";
    case FOLD_ATTN_SUM: return fwd ? "attn_fwd.sum" : "attn_bwd.sum";
    default: return fwd ? "attn_fwd.out" : "attn_bwd.out";
  }
}

}  // namespace

void launch_attn_fwd(int dtype, int kind, const AttnArgs& a, hipStream_t st) {
  if (a.rows <= 0) return;
  ProfScope prof(attn_name(kind, true), st);
  if (dtype == FOLD_BF16)
    attn_fwd_t<uint16_t>(kind, a, st);
  else
    attn_fwd_t<float>(kind, a, st);
}

void launch_attn_bwd(int dtype, int kind, const AttnArgs& a, hipStream_t st) {
  if (a.rows <= 0) return;
  ProfScope prof(attn_name(kind, false), st);
  if (dtype == FOLD_BF16)
    attn_bwd_t<uint16_t>(kind, a, st);
  else
    attn_bwd_t<float>(kind, a, st);
}

int attn_wgrad_chunks(int count) { return (count + kAttnWgradChunk - 1) / kAttnWgradChunk; }

void launch_attn_wgrad(int dtype, const int* op_rows, const int* op_cpos, int count, int H, int HP, int ld,
                       const void* h_pool, const float* gates, int gstride, float* part, float* dw, float* db,
                       hipStream_t st) {
  if (count <= 0 || (!dw && !db)) return;
  ProfScope prof("attn_wgrad", st);
  const int nchunk = attn_wgrad_chunks(count);
  const dim3 grid((unsigned)nchunk, (unsigned)((H + 255) / 256));
  if (dtype == FOLD_BF16)
    hipLaunchKernelGGL(k_attn_wgrad<uint16_t>, grid, dim3(256), 0, st, op_rows, op_cpos, count, H, HP, ld,
                       static_cast<const uint16_t*>(h_pool), gates, gstride, part);
  else
    hipLaunchKernelGGL(k_attn_wgrad<float>, grid, dim3(256), 0, st, op_rows, op_cpos, count, H, HP, ld,
                       static_cast<const float*>(h_pool), gates, gstride, part);
  hipLaunchKernelGGL(k_attn_wgrad_reduce, dim3((unsigned)((H + 1 + kWave - 1) / kWave)), dim3(256), 0, st, part,
                     nchunk, H, HP, dw, db);
}

void launch_pack_score(int dtype, int H, int HP, const void* w, const float* b, void* wdst, float* bdst,
                       hipStream_t st) {
  const unsigned blocks = (unsigned)((std::max(HP, kPadK) + 255) / 256);
  if (dtype == FOLD_BF16)
    hipLaunchKernelGGL(k_pack_score<uint16_t>, dim3(blocks), dim3(256), 0, st, H, HP,
                       static_cast<const uint16_t*>(w), b, static_cast<uint16_t*>(wdst), bdst);
  else
    hipLaunchKernelGGL(k_pack_score<float>, dim3(blocks), dim3(256), 0, st, H, HP, static_cast<const float*>(w), b,
                       static_cast<float*>(wdst), bdst);
}

}  // namespace fold
