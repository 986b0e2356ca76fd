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
#include "dma.h"
#include "mfma.h"

namespace fold {

namespace {

constexpr int kThreads = 256;

// Workgroup tile: 128 weight rows (m) x 256 gate columns (n); waves 2 x 2, each 64 x 128.
constexpr int kTM = 128, kTN = 256;
constexpr int kWgNW = 128;  // fp32 tile columns (two workgroups per compute unit)

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

// ---------------------------------------------------------------- fp32: direct loads into LDS
// A stage is 32 op rows.  X^T tile: the 32 rows x 128 weight rows (512 bytes a row), dz^T tile: the 32
// rows x NW gate columns.  Both are loaded straight into LDS, row-major in the op rows; a fragment read
// (one K value per lane and instruction) is then one dword per lane, 32 consecutive columns per half
// wave.  Odd rows have their 16-byte units permuted by ^ 8 so that the two half waves, which read
// rows 2 s and 2 s + 1, hit different halves of the 64 banks.
template <int NW>
struct WgDma {
  static constexpr int TM = 2, TN = NW / 64;      // wave tile 64 x NW / 2 (waves 2 x 2)
  static constexpr int ABYTES = 32 * kTM * 4, BBYTES = 32 * NW * 4;
  static constexpr int PA = ABYTES / 4096, PB = BBYTES / 4096;  // instructions per wave and stage
  static constexpr int BLANES = NW / 4;           // lanes per dz row in one instruction
};

template <int NW>
__global__ __launch_bounds__(kThreads) void k_wgrad_f32(WgArgs a) {
  using D = WgDma<NW>;
  constexpr int TM = D::TM, TN = D::TN, PA = D::PA, PB = D::PB;
  __shared__ __attribute__((aligned(16))) char A0[D::ABYTES], A1[D::ABYTES], B0[D::BBYTES], B1[D::BBYTES];
  const int tid = threadIdx.x, lane = tid & 63, wave = wave_id();
  const int wm = wave & 1, wn = wave >> 1, h = lane >> 5, l32 = lane & 31;
  // all tiles of one row chunk read the same X and dz rows: keep them on one XCD
  const int NT = (a.Nw + NW - 1) / NW, MTm = (a.Kw + kTM - 1) / kTM;
  int tx, chunk_id;
  if (!xcd_tile(MTm * NT, a.nchunk, tx, chunk_id)) return;
  const int mt_ = tx % MTm, nt = tx / MTm;
  const int m0 = mt_ * kTM, n0 = nt * NW;
  const int lo = chunk_id * a.chunk, hi = min(a.count, lo + a.chunk);
  const int nst = (hi - lo + 31) / 32;
  const char* zero = static_cast<const char*>(a.zero);
  const char* xbase = static_cast<const char*>(a.src);
  const size_t xstride = (size_t)(a.seg ? a.ld : a.tld) * 4, dstride = (size_t)a.gstride * 4;

  // per instruction: the op row inside the stage and the byte column this lane fetches
  int amr[PA], acol[PA], achild[PA], bmr[PB], bcol[PB];
  bool aok[PA], bok[PB];
#pragma unroll
  for (int i = 0; i < PA; ++i) {
    const int t = wave * PA + i;
    amr[i] = 2 * t + (lane >> 5);
    const int u = (lane & 31) ^ (8 * (lane >> 5));
    const int kw = m0 + 4 * u;
    const int k = a.seg ? min(kw / a.HP, 1) : 0;
    achild[i] = k;
    acol[i] = (a.seg ? kw - k * a.HP : kw) * 4;
    aok[i] = kw < a.Kw;
  }
#pragma unroll
  for (int i = 0; i < PB; ++i) {
    const int t = wave * PB + i;
    bmr[i] = t * (64 / D::BLANES) + lane / D::BLANES;
    const int u = (lane % D::BLANES) ^ (8 * (bmr[i] & 1));
    const int n = n0 + 4 * u;
    bcol[i] = n * 4;
    bok[i] = n < a.Nw;
  }
  // Row indices of a stage: X rows (children's or leaf-table rows) and dz rows, loaded from a clamped
  // (always valid) position; whether the row is real is kept apart and applied when the loads are
  // issued, so no branch waits on an index load.
  struct Idx {
    int a[PA], b[PB];
    bool va[PA], vb[PB];
  };
  auto load_idx = [&](int c, Idx& x) {
#pragma unroll
    for (int i = 0; i < PA; ++i) {
      const int r = lo + c * 32 + amr[i];
      const int rc = min(r, hi - 1);
      x.a[i] = a.seg ? a.op_cpos[2 * rc + achild[i]] : a.op_inp[rc];
      x.va[i] = r < hi && aok[i];
    }
#pragma unroll
    for (int i = 0; i < PB; ++i) {
      const int r = lo + c * 32 + bmr[i];
      x.b[i] = a.op_rows[min(r, hi - 1)];
      x.vb[i] = r < hi && bok[i];
    }
  };
  auto issue = [&](const Idx& x, char* Ad, char* Bd) {
#pragma unroll
    for (int i = 0; i < PA; ++i)
      dma16(x.va[i] && x.a[i] >= 0 ? xbase + (size_t)x.a[i] * xstride + acol[i] : zero, Ad + (wave * PA + i) * 1024);
#pragma unroll
    for (int i = 0; i < PB; ++i)
      dma16(x.vb[i] ? reinterpret_cast<const char*>(a.dz) + (size_t)x.b[i] * dstride + bcol[i] : zero,
            Bd + (wave * PB + i) * 1024);
  };
  // fragment byte offsets (row 2 s + h adds (2 s + h) * row bytes)
  int aoff[TM], boff[TN];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
    const int kw = wm * 64 + tm * 32 + l32;
    aoff[tm] = h * (kTM * 4) + ((kw >> 2) ^ (8 * h)) * 16 + (kw & 3) * 4;
  }
#pragma unroll
  for (int tn = 0; tn < TN; ++tn) {
    const int n = wn * (NW / 2) + tn * 32 + l32;
    boff[tn] = h * (NW * 4) + ((n >> 2) ^ (8 * h)) * 16 + (n & 3) * 4;
  }
  // bias column sums: thread tid sums column tid % NW over the stage rows r with r % MTm == mt_ and
  // (r / MTm) % (256 / NW) == tid / NW, so the chunk's rows are split over its MTm row tiles
  const bool do_bias = a.bpart != nullptr;
  const int bc = tid % NW, bg = tid / NW;
  const int bcoff = ((bc >> 2)) * 16 + (bc & 3) * 4;
  float bsum = 0.f;

  f32x16 acc[TM][TN];
  zero_acc(acc);
  auto stage = [&](const char* As, const char* Bs) {
#pragma unroll
    for (int s = 0; s < 16; ++s) {
      float av[TM], bv[TN];
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) av[tm] = *reinterpret_cast<const float*>(As + aoff[tm] + s * 2 * kTM * 4);
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) bv[tn] = *reinterpret_cast<const float*>(Bs + boff[tn] + s * 2 * NW * 4);
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[tm], bv[tn], acc[tm][tn], 0, 0, 0);
    }
    if (do_bias) {
      for (int r = mt_ + MTm * bg; r < 32; r += MTm * (256 / NW))
        bsum += *reinterpret_cast<const float*>(Bs + r * NW * 4 + (((bc >> 2) ^ (8 * (r & 1))) * 16) + (bc & 3) * 4);
    }
  };
  (void)bcoff;

  if (nst > 0) {
    Idx iC, iN;
    load_idx(0, iC);
    vm_wait();
    issue(iC, A0, B0);
    if (nst > 1) load_idx(1, iN);
    vm_wait();
    __syncthreads();
    int c = 0;
    for (; c + 2 <= nst; c += 2) {
      issue(iN, A1, B1);
      if (c + 2 < nst) load_idx(c + 2, iC);
      __builtin_amdgcn_sched_barrier(0);
      stage(A0, B0);
      vm_wait();
      __syncthreads();
      if (c + 2 < nst) {
        issue(iC, A0, B0);
        if (c + 3 < nst) load_idx(c + 3, iN);
      }
      __builtin_amdgcn_sched_barrier(0);
      stage(A1, B1);
      vm_wait();
      __syncthreads();
    }
    if (c < nst) stage(A0, B0);
  }

  float* out = a.partial + (size_t)chunk_id * a.Kw * a.Nw;
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const int n = n0 + wn * (NW / 2) + tn * 32 + l32;
      if (n >= a.Nw) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + wm * 64 + tm * 32 + acc_row(r, lane);
        if (m < a.Kw) out[(size_t)m * a.Nw + n] = acc[tm][tn][r];
      }
    }
  if (do_bias && n0 + bc < a.Nw)
    a.bpart[((size_t)(chunk_id * MTm + mt_) * (256 / NW) + bg) * a.Nw + n0 + bc] = bsum;
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

// db[col] += sum over partial rows, 64 columns per block: four thread groups sum interleaved partial
// rows, then the four sums are added in a fixed order (the result does not depend on scheduling)
__global__ void k_bias_reduce(const float* bpart, int nparts, int Nw, int H, int HP, float* dbias) {
  __shared__ float red[4][64];
  const int cg = threadIdx.x & 63, pg = threadIdx.x >> 6;
  const int n = blockIdx.x * 64 + cg;
  float s = 0.f;
  if (n < Nw)
    for (int c = pg; c < nparts; c += 4) s += bpart[(size_t)c * Nw + n];
  red[pg][cg] = s;
  __syncthreads();
  if (pg != 0 || n >= Nw) return;
  const int g = n / HP, j = n - g * HP;
  if (j >= H) return;
  dbias[g * H + j] += (red[0][cg] + red[1][cg]) + (red[2][cg] + red[3][cg]);
}

}  // namespace

WgradSplit wgrad_split(int count, int Kw, int Nw, int dtype) {
  WgradSplit w;
  if (count <= 0 || Kw <= 0 || Nw <= 0) return w;
  const int tn = dtype == FOLD_BF16 ? kTN : kWgNW;
  const long long tiles = (long long)((Kw + kTM - 1) / kTM) * ((Nw + tn - 1) / tn);
  // enough workgroups to fill the chip, and chunks in multiples of the 8 XCDs (one XCD per chunk)
  const long long want = std::max(8LL, ((1024 + tiles - 1) / tiles + 7) / 8 * 8);
  const long long most = std::max(1, (count + 511) / 512);
  w.nchunk = (int)std::max(1LL, std::min(want, most));
  w.chunk = round_up((count + w.nchunk - 1) / w.nchunk, 64);
  w.nchunk = (count + w.chunk - 1) / w.chunk;
  // bias partial rows: one per chunk (bf16), one per (chunk, weight-row tile, thread group) (fp32)
  w.bparts = dtype == FOLD_BF16 ? w.nchunk : w.nchunk * ((Kw + kTM - 1) / kTM) * (256 / kWgNW);
  return w;
}

void launch_wgrad(int dtype, const WgArgs& a, hipStream_t st) {
  if (a.count <= 0) return;
  ProfScope prof(dtype == FOLD_BF16 ? "wgrad.bf16" : "wgrad.f32", st);
  if (dtype == FOLD_BF16) {
    dim3 grid(xcd_grid(((a.Kw + kTM - 1) / kTM) * ((a.Nw + kTN - 1) / kTN), a.nchunk));
    hipLaunchKernelGGL(k_wgrad<uint16_t>, grid, dim3(kThreads), 0, st, a);
  } else {
    dim3 grid(xcd_grid(((a.Kw + kTM - 1) / kTM) * ((a.Nw + kWgNW - 1) / kWgNW), a.nchunk));
    hipLaunchKernelGGL(k_wgrad_f32<kWgNW>, grid, dim3(kThreads), 0, st, a);
  }
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
  hipLaunchKernelGGL(k_bias_reduce, dim3((Nw + 63) / 64), dim3(256), 0, st, bpart, nchunk, Nw, H, HP, dbias);
}

}  // namespace fold
