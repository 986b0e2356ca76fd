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
// owning the row's columns lane, lane + 64, ...; the dot products of the scorer and of the output's backward
// are wave sums of a fixed butterfly order.  The backward adds into the children's dh / dc directly (a plain
// read-add-write for a child with one parent edge, a hardware fp32 atomic otherwise), so no dz . W^T pass
// follows.  The scorer's weight gradient, dw = sum_r de_r h_c(r) and db = sum_r de_r, is reduced in fixed
// chunk order from the de each row's backward saves.

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

template <typename T>
__device__ __forceinline__ float ld_h(const T* h, int row, int ld, int j) {
  return row >= 0 ? to_f32<T>(h[(size_t)row * ld + j]) : 0.f;
}

// dst += v (dst's old value read first) when it has a single writer, else a hardware fp32 atomic add
__device__ __forceinline__ void add_to(float* dst, float v, bool single) {
  if (single)
    *dst += v;
  else
    unsafeAtomicAdd(dst, v);
}

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
    for (int j = lane; j < a.ld; j += kWave) {
      const float v = j < a.H ? ld_h(hp, c0, a.ld, j) : 0.f;
      if (j < a.H) part += (double)v * to_f32<T>(w[j]);
      ho[j] = from_f32<T>(v);
    }
    const float e = (float)(wave_total(part) + a.bias[0]);
    for (int j = lane; j < a.ld; j += kWave) co[j] = j == 0 ? e : (j == 1 ? 1.f : 0.f);
  } else if constexpr (KIND == FOLD_ATTN_SUM) {
    const int c0 = a.child_pos[a.idx_off + 2 * row], c1 = a.child_pos[a.idx_off + 2 * row + 1];
    const float m0 = c0 >= 0 ? a.c_pool[(size_t)c0 * a.ld] : 0.f, s0 = c0 >= 0 ? a.c_pool[(size_t)c0 * a.ld + 1] : 0.f;
    const float m1 = c1 >= 0 ? a.c_pool[(size_t)c1 * a.ld] : 0.f, s1 = c1 >= 0 ? a.c_pool[(size_t)c1 * a.ld + 1] : 0.f;
    const bool l0 = s0 != 0.f, l1 = s1 != 0.f;
    const float m = l0 && l1 ? fmaxf(m0, m1) : (l0 ? m0 : m1);
    const float x0 = l0 ? fast_exp(m0 - m) : 0.f, x1 = l1 ? fast_exp(m1 - m) : 0.f;
    for (int j = lane; j < a.ld; j += kWave) {
      float v = 0.f;
      if (j < a.H) {
        if (l0) v += x0 * ld_h(hp, c0, a.ld, j);
        if (l1) v += x1 * ld_h(hp, c1, a.ld, j);
      }
      ho[j] = from_f32<T>(v);
    }
    const bool any = l0 || l1;
    const float s = x0 * s0 + x1 * s1;
    for (int j = lane; j < a.ld; j += kWave) co[j] = j == 0 ? (any ? m : 0.f) : (j == 1 ? s : 0.f);
  } else {  // FOLD_ATTN_OUT
    const int c0 = a.child_pos[a.idx_off + row];
    const float s = c0 >= 0 ? a.c_pool[(size_t)c0 * a.ld + 1] : 0.f;
    for (int j = lane; j < a.ld; j += kWave) {
      const float v = (j < a.H && s != 0.f) ? ld_h(hp, c0, a.ld, j) / s : 0.f;
      ho[j] = from_f32<T>(v);
      co[j] = 0.f;
    }
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
    for (int j = lane; j < a.H; j += kWave) part += (double)dh[j] * ld_h(hp, c0, a.ld, j);
    const float de = (float)(wave_total(part) + a.dc[p * a.ld + 1]);
    if (lane == 0 && a.gates) a.gates[p * a.gstride] = de;
    if (c0 >= 0)
      for (int j = lane; j < a.H; j += kWave)
        add_to(&a.dh[(size_t)c0 * a.ld + j], dh[j] + de * to_f32<T>(w[j]), one);
  } else if constexpr (KIND == FOLD_ATTN_SUM) {
    // with m fixed, acc and s are linear in the children's: dh_k += x_k dh, ds_k += x_k ds
    const float m = a.c_pool[p * a.ld];
    const float ds = a.dc[p * a.ld + 1];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int ck = a.child_pos[a.idx_off + 2 * row + k];
      if (ck < 0) continue;
      const float sk = a.c_pool[(size_t)ck * a.ld + 1];
      if (sk == 0.f) continue;  // an empty set: x_k = 0
      const float xk = fast_exp(a.c_pool[(size_t)ck * a.ld] - m);  // the forward's x_k, bit for bit
      const bool one = a.child_one[a.idx_off + 2 * row + k] != 0;
      for (int j = lane; j < a.H; j += kWave) add_to(&a.dh[(size_t)ck * a.ld + j], xk * dh[j], one);
      if (lane == 0) add_to(&a.dc[(size_t)ck * a.ld + 1], xk * ds, one);
    }
  } else {  // FOLD_ATTN_OUT: h = acc / s -> dacc = dh / s, ds = -(dh . acc) / s^2
    const int c0 = a.child_pos[a.idx_off + row];
    if (c0 < 0) return;
    const float s = a.c_pool[(size_t)c0 * a.ld + 1];
    if (s == 0.f) return;
    const bool one = a.child_one[a.idx_off + row] != 0;
    double part = 0.0;
    for (int j = lane; j < a.H; j += kWave) part += (double)dh[j] * ld_h(hp, c0, a.ld, j);
    const double tot = wave_total(part);
    for (int j = lane; j < a.H; j += kWave) add_to(&a.dh[(size_t)c0 * a.ld + j], dh[j] / s, one);
    if (lane == 0) add_to(&a.dc[(size_t)c0 * a.ld + 1], (float)(-tot / ((double)s * s)), one);
  }
}

// Partial sums of the scorer's gradient over chunks of the op's rows: column j < H of chunk q is
// sum_r de_r h_c(r)[j] over the chunk's rows in order, column H (stored at HP) is sum_r de_r.
template <typename T>
__global__ __launch_bounds__(256) void k_attn_wgrad(const int* op_rows, const int* op_cpos, int count, int chunk,
                                                    int H, int HP, int ld, const T* h_pool, const float* gates,
                                                    int gstride, float* part) {
  const int j = blockIdx.y * blockDim.x + threadIdx.x;
  if (j > H) return;
  const int q0 = blockIdx.x * chunk, q1 = min(count, q0 + chunk);
  float acc = 0.f;
  int q = q0;
  // eight rows' loads in flight, added in row order
  for (; q + 8 <= q1; q += 8) {
    float de[8], v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      de[u] = gates[(size_t)op_rows[q + u] * gstride];
      v[u] = j < H ? ld_h(h_pool, op_cpos[2 * (size_t)(q + u)], ld, j) : 1.f;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) acc += de[u] * v[u];
  }
  for (; q < q1; ++q) {
    const float de = gates[(size_t)op_rows[q] * gstride];
    acc += de * (j < H ? ld_h(h_pool, op_cpos[2 * (size_t)q], ld, j) : 1.f);
  }
  part[(size_t)blockIdx.x * (HP + kPadK) + (j < H ? j : HP)] = acc;
}

__global__ __launch_bounds__(256) void k_attn_wgrad_reduce(const float* part, int nchunk, int H, int HP, float* dw,
                                                           float* db) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j > H) return;
  const int col = j < H ? j : HP;
  float acc = 0.f;
  for (int q = 0; q < nchunk; ++q) acc += part[(size_t)q * (HP + kPadK) + col];
  if (j < H) {
    if (dw) dw[j] += acc;
  } else if (db) {
    db[0] += acc;
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
  const dim3 grid((unsigned)nchunk, (unsigned)((H + 1 + 255) / 256));
  if (dtype == FOLD_BF16)
    hipLaunchKernelGGL(k_attn_wgrad<uint16_t>, grid, dim3(256), 0, st, op_rows, op_cpos, count, kAttnWgradChunk, H,
                       HP, ld, static_cast<const uint16_t*>(h_pool), gates, gstride, part);
  else
    hipLaunchKernelGGL(k_attn_wgrad<float>, grid, dim3(256), 0, st, op_rows, op_cpos, count, kAttnWgradChunk, H, HP,
                       ld, static_cast<const float*>(h_pool), gates, gstride, part);
  hipLaunchKernelGGL(k_attn_wgrad_reduce, dim3((unsigned)((H + 1 + 255) / 256)), dim3(256), 0, st, part, nchunk, H,
                     HP, dw, db);
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
