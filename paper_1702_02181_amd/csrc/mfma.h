// Matrix-core building blocks for gfx950: 32x32 MFMA tiles fed from LDS.
//
// One wave computes a 32 x 32 fp32 tile per instruction:
//   fp32 operands  v_mfma_f32_32x32x2_f32   (K = 2 per instruction, one element per lane)
//   bf16 operands  v_mfma_f32_32x32x16_bf16 (K = 16 per instruction, eight elements per lane)
// Operand fragments: lane l supplies row (l % 32) of A and column (l % 32) of B, for the
// K slice starting at (l / 32) * KPL.
// Result: lane l, register r holds C[8 * (r / 4) + 4 * (l / 32) + (r % 4)][l % 32].
#pragma once

#include "common.h"

namespace fold {

template <typename T>
struct Mma;

template <>
struct Mma<float> {
  static constexpr int BK = 32;    // K elements per LDS stage (128 bytes of a row)
  static constexpr int KSTEP = 2;  // K per instruction
  static constexpr int KPL = 1;    // K elements per lane per instruction
  static constexpr int VEC = 4;    // elements per 16-byte vector
  typedef float frag;
  __device__ static __forceinline__ frag load(const float* p) { return *p; }
  __device__ static __forceinline__ f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

template <>
struct Mma<uint16_t> {
  static constexpr int BK = 64;
  static constexpr int KSTEP = 16;
  static constexpr int KPL = 8;
  static constexpr int VEC = 8;
  typedef bf16x8 frag;
  __device__ static __forceinline__ frag load(const uint16_t* p) { return *reinterpret_cast<const bf16x8*>(p); }
  __device__ static __forceinline__ f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};

// Workgroups of a launch are handed to the 8 XCDs round-robin in launch order, and every XCD has its
// own L2.  A launch of X * round_up(Y, 8) workgroups is decoded so that all X workgroups of one y run
// on the same XCD and are dispatched back to back there: XCD k owns y in [k*Y8/8, (k+1)*Y8/8).  The
// operand those X workgroups share (a row tile's gathered rows, a weight slice, a row chunk) is then
// fetched into that XCD's L2 once.  Returns false for the padding workgroups (y >= Y), which exit.
// (L: the workgroup's index in its launch; a launch that runs several such grids back to back passes each
// workgroup's index within its own grid, which keeps the XCD assignment when every grid starts at a multiple
// of 8)
__device__ __forceinline__ bool xcd_tile_at(unsigned L, int X, int Y, int& x, int& y) {
  // unsigned arithmetic: the indices are never negative, and unsigned division is the cheaper sequence
  const unsigned per = ((unsigned)Y + 7u) >> 3, xcd = L & 7u, slot = L >> 3;
  x = (int)(slot % (unsigned)X);
  y = (int)(xcd * per + slot / (unsigned)X);
  return y < Y;
}
__device__ __forceinline__ bool xcd_tile(int X, int Y, int& x, int& y) { return xcd_tile_at(blockIdx.x, X, Y, x, y); }
inline int xcd_grid(int X, int Y) { return X * (((Y + 7) >> 3) << 3); }

// Wide launches over C column tiles (C a multiple of 8) and R row tiles, launched as C * R2 workgroups
// (R2 = R rounded up to even): the 8 XCDs form a 4 x 2 grid.  XCD k owns column tiles
// [(k & 3) C / 4, ((k & 3) + 1) C / 4) of the row tiles of parity k >> 2, so its weight slice stays in its
// L2 while the row tiles stream past, and two of its workgroups read each row tile (measured against one
// eighth of the columns over all row tiles: 1-3 % faster at H = 1,024).
__device__ __forceinline__ void xcd_cols(int C, int& col, int& row) {
  const int L = blockIdx.x, k = L & 7, per = C >> 2, slot = L >> 3;
  col = (k & 3) * per + slot % per;
  row = 2 * (slot / per) + (k >> 2);
}
inline int xcd_cols_grid(int C, int R) { return C * ((R + 1) / 2 * 2); }

// how a launch orders its workgroups over the XCDs
enum { kMapRows = 0, kMapCols = 1, kMapOwnCols = 2 };

// row of the 32x32 result tile held by register r of lane `lane`
__device__ __forceinline__ int acc_row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }

template <typename T>
__device__ __forceinline__ float to_f32(T x);
template <>
__device__ __forceinline__ float to_f32<float>(float x) { return x; }
template <>
__device__ __forceinline__ float to_f32<uint16_t>(uint16_t x) { return bf2f(x); }

template <typename T>
__device__ __forceinline__ T from_f32(float x);
template <>
__device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <>
__device__ __forceinline__ uint16_t from_f32<uint16_t>(float x) { return f2bf(x); }

// ---------------------------------------------------------------- LDS tiles

// Layouts of one LDS stage holding ROWS rows (M or N side of the output) by BK values of K:
//   kRK   [row][k], filled by 16-byte vectors that run along k          (both operands of the
//         forward cell and of dz . W^T: rows gathered from the pools, weights n-major)
//   kKR   [k][row], filled by vectors along rows; fp32 only (one K value per lane and
//         instruction, so the fragment read is one dword per lane)   (fp32 weight gradients)
//   kRKT  [row][k], filled by vectors along rows scattered element by element
//         (bf16 weight gradients, whose operands arrive row-major in K)
enum { kRK = 0, kKR = 1, kRKT = 2 };

template <typename T, int ROWS, int LAYOUT>
struct Tile {
  using M = Mma<T>;
  static constexpr int BK = M::BK, VEC = M::VEC;
  static constexpr int NVEC = ROWS * BK / VEC;
  static constexpr int PT = NVEC / 256;  // vectors per thread and stage
  static_assert(NVEC % 256 == 0, "tile must split evenly over 256 threads");
  static_assert(LAYOUT != kKR || sizeof(T) == 4, "k-major tiles are fp32 only");
  static constexpr int VROW = LAYOUT == kRK ? BK / VEC : ROWS / VEC;  // vectors per source line
  // fp32 [row][k]: rows of 34 dwords (8-byte aligned, written as two 8-byte halves); bf16 [row][k]:
  // rows of 72 halves (16-byte aligned).  k-major rows of ROWS + 32 dwords keep a fragment read
  // (32 consecutive rows at k, then at k + 1) on distinct banks.
  static constexpr int PITCH = LAYOUT == kKR ? ROWS + 32 : (sizeof(T) == 4 ? BK + 2 : BK + 8);
  static constexpr int ELEMS = LAYOUT == kKR ? BK * PITCH : ROWS * PITCH;

  __device__ static __forceinline__ void store(T* lds, int i, uint4 x) {
    const int a = i / VROW, b = i - a * VROW;
    if constexpr (LAYOUT == kRK) {
      T* d = lds + a * PITCH + b * VEC;
      if constexpr (sizeof(T) == 4) {
        reinterpret_cast<uint2*>(d)[0] = make_uint2(x.x, x.y);
        reinterpret_cast<uint2*>(d)[1] = make_uint2(x.z, x.w);
      } else {
        *reinterpret_cast<uint4*>(d) = x;
      }
    } else if constexpr (LAYOUT == kKR) {
      *reinterpret_cast<uint4*>(lds + a * PITCH + b * VEC) = x;
    } else {
      const T* e = reinterpret_cast<const T*>(&x);
#pragma unroll
      for (int q = 0; q < VEC; ++q) lds[(b * VEC + q) * PITCH + a] = e[q];
    }
  }

  __device__ static __forceinline__ typename M::frag frag(const T* lds, int row, int k) {
    if constexpr (LAYOUT == kKR)
      return lds[k * PITCH + row];
    else
      return M::load(lds + row * PITCH + k);
  }
};

// acc[TM][TN] += A(rows of this wave) . B(cols of this wave)^T over one LDS stage.
template <typename T, class TA, class TB, int TM, int TN>
__device__ __forceinline__ void mma_stage(const T* As, const T* Bs, f32x16 (&acc)[TM][TN], int arow0, int brow0,
                                          int lane) {
  using M = Mma<T>;
#pragma unroll
  for (int ks = 0; ks < M::BK; ks += M::KSTEP) {
    const int k = ks + (lane >> 5) * M::KPL;
    typename M::frag a[TM], b[TN];
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) a[tm] = TA::frag(As, arow0 + tm * 32 + (lane & 31), k);
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) b[tn] = TB::frag(Bs, brow0 + tn * 32 + (lane & 31), k);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm)
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) acc[tm][tn] = M::mma(a[tm], b[tn], acc[tm][tn]);
  }
}

// ---------------------------------------------------------------- prefetch registers
// Loads issued for the next stage must not be followed by branches that consume them, or the compiler
// waits for each load before the next one is issued.  So every fetch loads unconditionally from an
// address that is always valid (out-of-range rows and columns are clamped to a real element) and
// records how many of the fetched elements are real; masking and conversion happen when the registers
// are written to LDS, one stage later.
struct Raw4 {  // 16 bytes of operand data, nv leading elements valid
  uint4 x;
  int nv;
};
struct Raw8 {  // eight fp32 values that become eight bf16, nv leading elements valid
  uint4 x0, x1;
  int nv;
};

// zero the elements of a 16-byte vector of T from index nv on
template <typename T>
__device__ __forceinline__ uint4 mask_tail(uint4 v, int nv) {
  constexpr int VEC = 16 / sizeof(T);
  if (nv >= VEC) return v;
  uint32_t w[4] = {v.x, v.y, v.z, v.w};
  if constexpr (sizeof(T) == 4) {
#pragma unroll
    for (int e = 0; e < 4; ++e) w[e] = e < nv ? w[e] : 0u;
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t lo = (2 * e < nv) ? 0x0000ffffu : 0u, hi = (2 * e + 1 < nv) ? 0xffff0000u : 0u;
      w[e] &= lo | hi;
    }
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// an operand already in the LDS element type
template <typename T>
__device__ __forceinline__ uint4 finish(const Raw4& r) {
  return mask_tail<T>(r.x, r.nv);
}

// fp32 values rounded to bf16 (round to nearest even)
__device__ __forceinline__ uint4 finish_bf16(const Raw8& r) {
  const uint32_t in[8] = {r.x0.x, r.x0.y, r.x0.z, r.x0.w, r.x1.x, r.x1.y, r.x1.z, r.x1.w};
  uint32_t w[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float a = 2 * e < r.nv ? __uint_as_float(in[2 * e]) : 0.f;
    const float b = 2 * e + 1 < r.nv ? __uint_as_float(in[2 * e + 1]) : 0.f;
    w[e] = (uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16);
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// Row indices that a kernel reads from global memory before it can fetch a stage (the weight
// gradients' gathered rows) travel two stages ahead: loaded into registers at stage c, written to
// one of three LDS slots at the end of stage c, read by the fetch of stage c + 2 issued during
// stage c + 1.  Kernels without such indices use NoIndex.
struct NoIndex {
  __device__ void prologue(int) {}
  __device__ void load(int) {}
  __device__ void store(int) {}
};

// ---------------------------------------------------------------- the K loop

// K loop over `nchunks` LDS stages.  The global loads of stage c+1 are issued (into registers)
// right after stage c becomes visible in LDS, so their latency hides behind stage c's MFMAs.
// la / lb: fetch(c, i) -> raw registers of the i-th 16-byte vector of stage c; put(raw) -> uint4.
template <typename T, class TA, class TB, int TM, int TN, class LA, class LB, class IX>
__device__ __forceinline__ void mainloop(int nchunks, LA& la, LB& lb, IX& ix, T* As, T* Bs,
                                         f32x16 (&acc)[TM][TN], int arow0, int brow0) {
  const int tid = threadIdx.x, lane = tid & 63;
  ix.prologue(nchunks);
  typename LA::raw ra[TA::PT];
  typename LB::raw rb[TB::PT];
  if (nchunks > 0) {
#pragma unroll
    for (int i = 0; i < TA::PT; ++i) ra[i] = la.fetch(0, tid + i * 256);
#pragma unroll
    for (int i = 0; i < TB::PT; ++i) rb[i] = lb.fetch(0, tid + i * 256);
  }
  for (int c = 0; c < nchunks; ++c) {
    if (c + 2 < nchunks) ix.load(c + 2);
#pragma unroll
    for (int i = 0; i < TA::PT; ++i) TA::store(As, tid + i * 256, la.put(ra[i]));
#pragma unroll
    for (int i = 0; i < TB::PT; ++i) TB::store(Bs, tid + i * 256, lb.put(rb[i]));
    __syncthreads();
    if (c + 1 < nchunks) {
#pragma unroll
      for (int i = 0; i < TA::PT; ++i) ra[i] = la.fetch(c + 1, tid + i * 256);
#pragma unroll
      for (int i = 0; i < TB::PT; ++i) rb[i] = lb.fetch(c + 1, tid + i * 256);
    }
    mma_stage<T, TA, TB, TM, TN>(As, Bs, acc, arow0, brow0, lane);
    if (c + 2 < nchunks) ix.store(c + 2);
    __syncthreads();
  }
}

template <int TM, int TN>
__device__ __forceinline__ void zero_acc(f32x16 (&acc)[TM][TN]) {
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[tm][tn][r] = 0.f;
}

}  // namespace fold
