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

// Workgroup tile: 128 weight rows (m) x 256 gate columns (n); waves 2 x 2, each 64 x 128.
constexpr int kTM = 128, kTN = 256;

// Row indices of the pool rows a stage reduces over (pool row, child 0 / input row, child 1),
// loaded two stages ahead into one of three LDS slots.
template <int BK>
struct WgIndex {
  int (*slots)[3][BK];
  const int* op_rows;
  const int* op_cpos;
  const int* op_inp;
  int lo, hi, seg;
  int rp, r0, r1, ok;
  __device__ __forceinline__ void load(int c) {
    const int t = threadIdx.x % BK;  // every thread loads (no branch around the loads); BK of them store
    const int r = lo + c * BK + t;
    ok = r < hi;
    const int rc = ok ? r : lo;
    rp = op_rows[rc];
    if (seg) {
      r0 = op_cpos[2 * rc];
      r1 = op_cpos[2 * rc + 1];
    } else {
      r0 = op_inp[rc];
      r1 = -1;
    }
  }
  __device__ __forceinline__ void store(int c) {
    const int t = threadIdx.x;
    if (t < BK) {
      slots[c % 3][0][t] = ok ? rp : -1;
      slots[c % 3][1][t] = ok ? r0 : -1;
      slots[c % 3][2][t] = ok ? r1 : -1;
    }
  }
  __device__ __forceinline__ void prologue(int nst) {
    for (int c = 0; c < 2 && c < nst; ++c) {
      load(c);
      store(c);
    }
    __syncthreads();
  }
};

// X^T operand: gathered children's h rows (seg 1) or leaf-table rows (seg 0)
template <typename T, int BK, int VROW>
struct WgX {
  using raw = Raw4;
  const T* src;
  int sld, width, HP, Kw, m0, seg;
  int (*slots)[3][BK];
  __device__ __forceinline__ raw fetch(int c, int i) const {
    constexpr int VEC = Mma<T>::VEC;
    const int kk = i / VROW, v = i - kk * VROW;
    const int m = m0 + v * VEC;
    const int k = seg ? min(m / HP, 1) : 0;
    const int jin = seg ? m - k * HP : m;
    const int s = slots[c % 3][1 + k][kk];
    const int nv = (s >= 0 && m < Kw) ? min(max(width - jin, 0), VEC) : 0;
    const size_t off = nv > 0 ? (size_t)s * sld + jin : 0;
    return {*reinterpret_cast<const uint4*>(src + off), nv};
  }
  __device__ __forceinline__ uint4 put(const raw& r) const { return finish<T>(r); }
};

// dz^T operand; the fp32 values also feed the bias column sums
template <typename T, int BK, int VROW>
struct WgDz;

template <int BK, int VROW>
struct WgDz<float, BK, VROW> {
  using raw = Raw4;
  const float* dz;
  int gstride, Nw, n0;
  int (*slots)[3][BK];
  bool bias;
  float bsum[4];
  __device__ __forceinline__ raw fetch(int c, int i) const {
    const int kk = i / VROW, v = i - kk * VROW;
    const int p = slots[c % 3][0][kk];
    const int n = n0 + v * 4;
    const int ok = p >= 0 && n < Nw;
    return {*reinterpret_cast<const uint4*>(dz + (ok ? (size_t)p * gstride + n : 0)), ok ? 4 : 0};
  }
  __device__ __forceinline__ uint4 put(const raw& r) {
    const uint4 x = finish<float>(r);
    if (bias) {
      bsum[0] += __uint_as_float(x.x);
      bsum[1] += __uint_as_float(x.y);
      bsum[2] += __uint_as_float(x.z);
      bsum[3] += __uint_as_float(x.w);
    }
    return x;
  }
};

template <int BK, int VROW>
struct WgDz<uint16_t, BK, VROW> {
  using raw = Raw8;
  const float* dz;
  int gstride, Nw, n0;
  int (*slots)[3][BK];
  bool bias;
  float bsum[8];
  __device__ __forceinline__ raw fetch(int c, int i) const {
    const int kk = i / VROW, v = i - kk * VROW;
    const int p = slots[c % 3][0][kk];
    const int n = n0 + v * 8;
    const int ok = p >= 0 && n < Nw;
    const float* q = dz + (ok ? (size_t)p * gstride + n : 0);
    return {reinterpret_cast<const uint4*>(q)[0], reinterpret_cast<const uint4*>(q)[1], ok ? 8 : 0};
  }
  __device__ __forceinline__ uint4 put(const raw& r) {
    if (bias && r.nv > 0) {
      const uint32_t in[8] = {r.x0.x, r.x0.y, r.x0.z, r.x0.w, r.x1.x, r.x1.y, r.x1.z, r.x1.w};
#pragma unroll
      for (int q = 0; q < 8; ++q) bsum[q] += __uint_as_float(in[q]);
    }
    return finish_bf16(r);
  }
};

template <typename T>
__global__ __launch_bounds__(kThreads) void k_wgrad(WgArgs a) {
  using M = Mma<T>;
  constexpr int BK = M::BK, VEC = M::VEC;
  constexpr int LAY = sizeof(T) == 4 ? kKR : kRKT;
  using TA = Tile<T, kTM, LAY>;  // X^T: weight rows x pool rows
  using TB = Tile<T, kTN, LAY>;  // dz^T: gate columns x pool rows
  __shared__ __attribute__((aligned(16))) T As[TA::ELEMS];
  __shared__ __attribute__((aligned(16))) T Bs[TB::ELEMS];
  __shared__ int slots[3][3][BK];
  __shared__ float red[256 / TB::VROW][kTN];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  // all tiles of one row chunk read the same X and dz rows: keep them on one XCD
  const int NT = (a.Nw + kTN - 1) / kTN, MTm = (a.Kw + kTM - 1) / kTM;
  int tx, chunk_id;
  if (!xcd_tile(MTm * NT, a.nchunk, tx, chunk_id)) return;
  const int mt_ = tx % MTm;
  const int m0 = mt_ * kTM, n0 = (tx / MTm) * kTN;
  const int lo = chunk_id * a.chunk, hi = min(a.count, lo + a.chunk);
  const bool do_bias = a.bpart != nullptr && mt_ == 0;

  WgIndex<BK> ix{slots, a.op_rows, a.op_cpos, a.op_inp, lo, hi, a.seg, 0, 0, 0, 0};
  WgX<T, BK, TA::VROW> la{static_cast<const T*>(a.src), a.seg ? a.ld : a.tld, a.seg ? a.H : a.in_dim, a.HP,
                          a.Kw, m0, a.seg, slots};
  WgDz<T, BK, TB::VROW> lb{a.dz, a.gstride, a.Nw, n0, slots, do_bias, {}};
#pragma unroll
  for (int q = 0; q < VEC; ++q) lb.bsum[q] = 0.f;
  f32x16 acc[2][4];
  zero_acc(acc);
  const int nst = (hi - lo + BK - 1) / BK;
  mainloop<T, TA, TB, 2, 4>(nst, la, lb, ix, As, Bs, acc, wm * 64, wn * 128);

  float* out = a.partial + (size_t)chunk_id * a.Kw * a.Nw;
#pragma unroll
  for (int tm = 0; tm < 2; ++tm)
#pragma unroll
    for (int tn = 0; tn < 4; ++tn) {
      const int n = n0 + wn * 128 + tn * 32 + (lane & 31);
      if (n >= a.Nw) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + wm * 64 + tm * 32 + acc_row(r, lane);
        if (m < a.Kw) out[(size_t)m * a.Nw + n] = acc[tm][tn][r];
      }
    }
  if (do_bias) {
    // every thread's dz vectors share one column group (TB::VROW divides the block), so the column
    // sums finish with a fixed-order reduction over the threads of that group
    const int v = tid % TB::VROW, j = tid / TB::VROW;
#pragma unroll
    for (int q = 0; q < VEC; ++q) red[j][v * VEC + q] = lb.bsum[q];
    __syncthreads();
    for (int col = tid; col < kTN; col += kThreads) {
      float s = 0.f;
      for (int jj = 0; jj < 256 / TB::VROW; ++jj) s += red[jj][col];
      if (n0 + col < a.Nw) a.bpart[(size_t)chunk_id * a.Nw + n0 + col] = s;
    }
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
  const long long tiles = (long long)((Kw + kTM - 1) / kTM) * ((Nw + kTN - 1) / kTN);
  // enough workgroups to fill the chip, and chunks in multiples of the 8 XCDs (one XCD per chunk)
  const long long want = std::max(8LL, ((1024 + tiles - 1) / tiles + 7) / 8 * 8);
  const long long most = std::max(1, (count + 511) / 512);
  w.nchunk = (int)std::max(1LL, std::min(want, most));
  w.chunk = round_up((count + w.nchunk - 1) / w.nchunk, 64);
  w.nchunk = (count + w.chunk - 1) / w.chunk;
  return w;
}

void launch_wgrad(int dtype, const WgArgs& a, hipStream_t st) {
  if (a.count <= 0) return;
  ProfScope prof(dtype == FOLD_BF16 ? "wgrad.bf16" : "wgrad.f32", st);
  dim3 grid(xcd_grid(((a.Kw + kTM - 1) / kTM) * ((a.Nw + kTN - 1) / kTN), a.nchunk));
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

void launch_bias_partial(const int* op_rows, int count, int chunk, int nchunk, const float* dz, int gstride, int Nw,
                         float* bpart, hipStream_t st) {
  if (count <= 0) return;
  ProfScope prof("bias_partial", st);
  hipLaunchKernelGGL(k_bias_partial, dim3(nchunk, (Nw + 255) / 256), dim3(256), 0, st, op_rows, count, chunk, dz,
                     gstride, Nw, bpart);
}

void launch_bias_reduce(const float* bpart, int nchunk, int Nw, int H, int HP, float* dbias, hipStream_t st) {
  if (nchunk <= 0) return;
  ProfScope prof("bias_reduce", st);
  hipLaunchKernelGGL(k_bias_reduce, dim3((Nw + 255) / 256), dim3(256), 0, st, bpart, nchunk, Nw, H, HP, dbias);
}

}  // namespace fold
