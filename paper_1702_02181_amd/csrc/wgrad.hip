// Weight gradients, deferred to the end of the backward pass (gfx950).
//
// For an operation with rows R (every pool row running it, all levels together) the gradient of its
// weights is one contraction over those rows:
//     dW_rec += [h_c0 | h_c1 | ...]^T . dz      (children's h rows gathered by child_pos)
//     dW_in  += x^T . dz                        (leaf-table rows gathered by input_idx)
//     db     += sum_rows dz
// The rows are split into `nchunk` contiguous chunks; a workgroup reduces one chunk for one 64x64 tile
// of dW on the matrix cores and writes its partial tile (no atomics); a second kernel sums the
// partial tiles in chunk order and adds the result to the caller's canonical-layout gradient, so the
// result does not depend on scheduling.

#include <hip/hip_runtime.h>

#include <algorithm>

#include "common.h"
#include "internal.h"
#include "mfma.h"

namespace fold {

namespace {

constexpr int kThreads = 256;
constexpr int kTile = 64;

template <typename T>
__global__ __launch_bounds__(kThreads) void k_wgrad(WgArgs a) {
  using M = Mma<T>;
  constexpr int BK = M::BK, VEC = M::VEC, PITCH = BK + M::PAD;
  __shared__ __attribute__((aligned(16))) T As[kTile * PITCH];  // As[m][k] = X[row k][m]
  __shared__ __attribute__((aligned(16))) T Bs[kTile * PITCH];  // Bs[n][k] = dz[row k][n]
  __shared__ int prow[BK], srow[BK];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int chunk_id = blockIdx.x;
  const int m0 = blockIdx.y * kTile, n0 = blockIdx.z * kTile;
  const int k = a.seg ? m0 / a.HP : 0;
  const int jin0 = a.seg ? m0 - k * a.HP : m0;
  const int width = a.seg ? a.H : a.in_dim;
  const int sld = a.seg ? a.ld : a.tld;
  const T* src = static_cast<const T*>(a.src);
  const int lo = chunk_id * a.chunk, hi = min(a.count, lo + a.chunk);

  f32x16 acc;
  for (int r = 0; r < 16; ++r) acc[r] = 0.f;

  for (int r0 = lo; r0 < hi; r0 += BK) {
    if (tid < BK) {
      const int i = r0 + tid;
      int p = -1, s = -1;
      if (i < hi) {
        p = a.op_rows[i];
        if (a.seg) {
          const int g = a.pos_group[p];
          s = a.child_pos[a.g_idx_off[g] + (p - a.g_row_begin[g]) * a.arity + k];
        } else {
          s = a.input_idx[p];
        }
      }
      prow[tid] = p;
      srow[tid] = s;
    }
    __syncthreads();
    constexpr int AV = kTile / VEC;  // vectors per row of the X tile
    for (int i = tid; i < BK * AV; i += kThreads) {
      const int kk = i / AV, v = i - kk * AV;
      const int s = srow[kk];
      uint4 x = make_uint4(0u, 0u, 0u, 0u);
      if (s >= 0) x = load_row_vec<T>(src + (size_t)s * sld, jin0 + v * VEC, width);
      const T* e = reinterpret_cast<const T*>(&x);
#pragma unroll
      for (int q = 0; q < VEC; ++q) As[(v * VEC + q) * PITCH + kk] = e[q];
    }
    constexpr int BV = kTile / 4;  // float4 per row of the dz tile
    for (int i = tid; i < BK * BV; i += kThreads) {
      const int kk = i / BV, v = i - kk * BV;
      const int p = prow[kk];
      float4 f = make_float4(0.f, 0.f, 0.f, 0.f);
      if (p >= 0) f = *reinterpret_cast<const float4*>(a.dz + (size_t)p * a.gstride + n0 + v * 4);
      Bs[(v * 4 + 0) * PITCH + kk] = from_f32<T>(f.x);
      Bs[(v * 4 + 1) * PITCH + kk] = from_f32<T>(f.y);
      Bs[(v * 4 + 2) * PITCH + kk] = from_f32<T>(f.z);
      Bs[(v * 4 + 3) * PITCH + kk] = from_f32<T>(f.w);
    }
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < BK; ks += M::KSTEP) {
      const typename M::frag af = M::load(&As[(wm * 32 + (lane & 31)) * PITCH + ks + (lane >> 5) * M::KPL]);
      const typename M::frag bf = M::load(&Bs[(wn * 32 + (lane & 31)) * PITCH + ks + (lane >> 5) * M::KPL]);
      acc = M::mma(af, bf, acc);
    }
    __syncthreads();
  }
  float* out = a.partial + (size_t)chunk_id * a.Kw * a.Nw;
  const int n = n0 + wn * 32 + (lane & 31);
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int m = m0 + wm * 32 + acc_row(r, lane);
    out[(size_t)m * a.Nw + n] = acc[r];
  }
}

// dW[row, col] += sum over chunks of partial[chunk, m, n], (m, n) in the padded layout
__global__ void k_wgrad_reduce(const float* partial, int nchunk, int Kw, int Nw, int seg, int H, int HP,
                               int in_dim, int G, float* dW) {
  const size_t total = (size_t)Kw * Nw;
  for (size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (size_t)gridDim.x * blockDim.x) {
    const int m = (int)(idx / Nw), n = (int)(idx - (size_t)m * Nw);
    const int g = n / HP, j = n - g * HP;
    if (j >= H) continue;
    int row;
    if (seg) {
      const int k = m / HP, jin = m - k * HP;
      if (jin >= H) continue;
      row = k * H + jin;
    } else {
      if (m >= in_dim) continue;
      row = m;
    }
    float s = 0.f;
    for (int c = 0; c < nchunk; ++c) s += partial[(size_t)c * total + idx];
    dW[(size_t)row * G * H + g * H + j] += s;
  }
}

__global__ void k_bias_partial(const int* op_rows, int count, int chunk, const float* dz, int gstride, int Nw,
                               float* bpart) {
  const int c = blockIdx.x;
  const int n = blockIdx.y * blockDim.x + threadIdx.x;
  if (n >= Nw) return;
  const int lo = c * chunk, hi = min(count, lo + chunk);
  float s = 0.f;
  for (int i = lo; i < hi; ++i) s += dz[(size_t)op_rows[i] * gstride + n];
  bpart[(size_t)c * Nw + n] = s;
}

__global__ void k_bias_reduce(const float* bpart, int nchunk, int Nw, int H, int HP, float* dbias) {
  const int n = blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= Nw) return;
  const int g = n / HP, j = n - g * HP;
  if (j >= H) return;
  float s = 0.f;
  for (int c = 0; c < nchunk; ++c) s += bpart[(size_t)c * Nw + n];
  dbias[g * H + j] += s;
}

}  // namespace

WgradSplit wgrad_split(int count, int Kw, int Nw) {
  WgradSplit w;
  if (count <= 0 || Kw <= 0 || Nw <= 0) return w;
  const long long tiles = (long long)(Kw / kTile) * (Nw / kTile);
  long long want = (2048 + tiles - 1) / tiles;  // enough workgroups to fill the chip
  long long most = std::max(1, (count + 255) / 256);
  w.nchunk = (int)std::max(1LL, std::min(want, most));
  w.chunk = round_up((count + w.nchunk - 1) / w.nchunk, 64);
  w.nchunk = (count + w.chunk - 1) / w.chunk;
  return w;
}

void launch_wgrad(int dtype, const WgArgs& a, hipStream_t st) {
  if (a.count <= 0) return;
  ProfScope prof(dtype == FOLD_BF16 ? "wgrad.bf16" : "wgrad.f32", st);
  dim3 grid(a.nchunk, a.Kw / kTile, a.Nw / kTile);
  if (dtype == FOLD_BF16)
    hipLaunchKernelGGL(k_wgrad<uint16_t>, grid, dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL(k_wgrad<float>, grid, dim3(kThreads), 0, st, a);
}

void launch_wgrad_reduce(const float* partial, int nchunk, int Kw, int Nw, int seg, int H, int HP, int in_dim,
                         int G, float* dW, hipStream_t st) {
  ProfScope prof("wgrad_reduce", st);
  const size_t total = (size_t)Kw * Nw;
  const unsigned blocks = (unsigned)std::min<size_t>((total + 255) / 256, 65536);
  hipLaunchKernelGGL(k_wgrad_reduce, dim3(blocks), dim3(256), 0, st, partial, nchunk, Kw, Nw, seg, H, HP, in_dim,
                     G, dW);
}

void launch_bias_grad(const int* op_rows, int count, int chunk, int nchunk, const float* dz, int gstride, int Nw,
                      float* bpart, int G, int H, int HP, float* dbias, hipStream_t st) {
  if (count <= 0) return;
  ProfScope prof("bias_grad", st);
  hipLaunchKernelGGL(k_bias_partial, dim3(nchunk, (Nw + 255) / 256), dim3(256), 0, st, op_rows, count, chunk, dz,
                     gstride, Nw, bpart);
  hipLaunchKernelGGL(k_bias_reduce, dim3((Nw + 255) / 256), dim3(256), 0, st, bpart, nchunk, Nw, H, HP, dbias);
}

}  // namespace fold
