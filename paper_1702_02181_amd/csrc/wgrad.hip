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
#include "wide.h"

namespace fold {

namespace {

constexpr int kThreads = 256;

// Workgroup tile: 128 weight rows (m) x 256 gate columns (n); waves 2 x 2, each 64 x 128.
constexpr int kTM = 128;  // weight rows per tile
constexpr int kWgNW = 128;  // fp32 tile columns (two workgroups per compute unit)
constexpr int kWgWideF32Rows = 32768;  // fp32 ops with at least this many rows may use 256 x 256 tiles

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

// ---------------------------------------------------------------- bf16: direct loads + transposing reads
// A stage is 64 op rows.  X^T tile: 64 rows x 128 weight rows (256 bytes a row), dz^T tile: 64 rows x
// 128 gate columns of bf16 dz.  The bf16 MFMA operand is, per lane, eight consecutive op rows of one
// column; ds_read_b64_tr_b16 delivers them from the row-major tile: each group of 16 lanes addresses a
// block of 4 rows x 16 columns (lane i: row i / 4, columns 4 (i % 4) .. + 3) and lane i receives the 4
// values of column i.  Row m's 16-byte units are permuted by ^ 4 (m & 3), so the 4 rows of a block
// fall into different 64-byte bank ranges.
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4_t;
#define FOLD_LDS_AS __attribute__((address_space(3)))

__device__ __forceinline__ int wg16_off(int m, int col) {
  return m * 256 + (((col >> 3) ^ (4 * (m & 3))) << 4) + (col & 7) * 2;
}

__device__ __forceinline__ uint2 ld_tr16(const char* lds, int off) {
  const bf16x4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((FOLD_LDS_AS bf16x4_t*)(lds + off));
  return __builtin_bit_cast(uint2, v);
}

__global__ __launch_bounds__(kThreads) void k_wgrad_bf16(WgArgs a) {
  constexpr int NW = 128, TM = 2, TN = 2, BYTES = 64 * 256, PA = BYTES / 4096, PB = BYTES / 4096;
  __shared__ __attribute__((aligned(16))) char A0[BYTES], A1[BYTES], B0[BYTES], B1[BYTES];
  const int tid = threadIdx.x, lane = tid & 63, wave = wave_id();
  const int wm = wave & 1, wn = wave >> 1;
  const int NT = (a.Nw + NW - 1) / NW, MTm = (a.Kw + kTM - 1) / kTM;
  int tx, chunk_id;
  if (!xcd_tile(MTm * NT, a.nchunk, tx, chunk_id)) return;
  const int mt_ = tx % MTm, nt = tx / MTm;
  const int m0 = mt_ * kTM, n0 = nt * NW;
  const int lo = chunk_id * a.chunk, hi = min(a.count, lo + a.chunk);
  const int nst = (hi - lo + 63) / 64;
  const char* zero = static_cast<const char*>(a.zero);
  const char* xbase = static_cast<const char*>(a.src);
  const size_t xstride = (size_t)(a.seg ? a.ld : a.tld) * 2, dstride = (size_t)a.gstride * 4;

  // per instruction: the op row inside the stage (4 t + lane / 16) and this lane's byte column
  const int msub = lane >> 4, u = (lane & 15) ^ (4 * (msub & 3));
  const int kw = m0 + 8 * u, nw = n0 + 8 * u;
  const int achild = a.seg ? min(kw / a.HP, 1) : 0;
  const int acol = (a.seg ? kw - achild * a.HP : kw) * 2, bcol = nw * 2;
  const bool aok = kw < a.Kw, bok = nw < a.Nw;
  struct Idx {
    int a[PA], b[PB];
    bool va[PA], vb[PB];
  };
  auto load_idx = [&](int c, Idx& x) {
#pragma unroll
    for (int i = 0; i < PA; ++i) {
      const int r = lo + c * 64 + 4 * (wave * PA + i) + msub;
      const int rc = min(r, hi - 1);
      x.a[i] = a.seg ? a.op_cpos[2 * rc + achild] : a.op_inp[rc];
      x.va[i] = r < hi && aok;
      x.b[i] = a.op_rows[rc];
      x.vb[i] = r < hi && bok;
    }
  };
  auto issue = [&](const Idx& x, char* Ad, char* Bd) {
#pragma unroll
    for (int i = 0; i < PA; ++i)
      dma16(x.va[i] && x.a[i] >= 0 ? xbase + (size_t)x.a[i] * xstride + acol : zero, Ad + (wave * PA + i) * 1024);
#pragma unroll
    for (int i = 0; i < PB; ++i)
      dma16(x.vb[i] ? reinterpret_cast<const char*>(a.dz) + (size_t)x.b[i] * dstride + bcol : zero,
            Bd + (wave * PB + i) * 1024);
  };
  // transposing-read offsets: group g = lane / 16 serves rows (g & 1) * 16 .. + 15 of its 32-row
  // fragment and K half g >> 1; lane i of the group addresses row i / 4, columns 4 (i % 4) .. + 3
  const int g = lane >> 4, gi = lane & 15;
  int aoff[TM], boff[TN];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) aoff[tm] = wm * 64 + tm * 32 + 16 * (g & 1) + 4 * (gi & 3);
#pragma unroll
  for (int tn = 0; tn < TN; ++tn) boff[tn] = wn * 64 + tn * 32 + 16 * (g & 1) + 4 * (gi & 3);
  const int mrow = 8 * (g >> 1) + (gi >> 2);  // + 16 s + 4 j
  // bias column sums: thread tid sums column tid % 128 over the stage rows r with r % MTm == mt_ and
  // (r / MTm) % 2 == tid / 128
  const bool do_bias = a.bpart != nullptr;
  const int bc = tid & 127, bg = tid >> 7;
  float bsum = 0.f;

  f32x16 acc[TM][TN];
  zero_acc(acc);
  auto stage = [&](const char* As, const char* Bs) {
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      uint4 af[TM], bf[TN];
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) {
        const uint2 lo2 = ld_tr16(As, wg16_off(16 * s + mrow, aoff[tm]));
        const uint2 hi2 = ld_tr16(As, wg16_off(16 * s + mrow + 4, aoff[tm]));
        af[tm] = make_uint4(lo2.x, lo2.y, hi2.x, hi2.y);
      }
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        const uint2 lo2 = ld_tr16(Bs, wg16_off(16 * s + mrow, boff[tn]));
        const uint2 hi2 = ld_tr16(Bs, wg16_off(16 * s + mrow + 4, boff[tn]));
        bf[tn] = make_uint4(lo2.x, lo2.y, hi2.x, hi2.y);
      }
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
          acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, af[tm]),
                                                               __builtin_bit_cast(bf16x8, bf[tn]), acc[tm][tn], 0,
                                                               0, 0);
    }
    if (do_bias) {
      for (int r = mt_ + MTm * bg; r < 64; r += 2 * MTm)
        bsum += bf2f(*reinterpret_cast<const uint16_t*>(Bs + wg16_off(r, bc)));
    }
  };

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
      const int n = n0 + wn * 64 + tn * 32 + (lane & 31);
      if (n >= a.Nw) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + wm * 64 + tm * 32 + acc_row(r, lane);
        if (m < a.Kw) out[(size_t)m * a.Nw + n] = acc[tm][tn][r];
      }
    }
  if (do_bias && n0 + bc < a.Nw) a.bpart[((size_t)(chunk_id * MTm + mt_) * 2 + bg) * a.Nw + n0 + bc] = bsum;
}

// ---------------------------------------------------------------- bf16, wide: 256 x 256 tiles
// 8 waves, each 64 weight rows x 128 gate columns; a stage is 32 op rows (two MFMA K steps): X^T tile
// 32 x 256 weight rows and dz^T tile 32 x 256 columns, 512 bytes an op row, 128 FLOP per operand byte.
// Four stage slots keep three stages in flight (untracked direct loads, waves 0-3: 4 instructions of X
// and 4 of dz rows each, two op rows per instruction).  The op rows' indices (pool row of dz, children's
// or leaf-table row of X) reach LDS through an index ring three stages ahead of the data, loaded by
// wave 4 alone (two 4-byte-per-lane direct loads per stage), so every wait counts only its own loads.
// Row m's 16-byte units are permuted by ^ 4 (m & 3) for the transposing reads (as the 128-column
// kernel above).

// lane l of the wave copies 4 bytes from src to lds + 4 l
__device__ __forceinline__ void dma4_untracked(const void* src, void* lds) {
  const uint32_t base = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)lds);
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dword %1, off" ::"s"(base), "v"(src) : "memory", "m0");
}

__device__ __forceinline__ int wgw_off(int r, int col) {
  return r * 512 + (((col >> 3) ^ (4 * (r & 3))) << 4) + (col & 7) * 2;
}

__global__ __launch_bounds__(wide::kThreads) void k_wgrad_bf16_w(WgArgs a) {
  constexpr int TB = 256, TM = 2, TN = 4, NL = 8;
  constexpr int ABYTES = 32 * 512, SLOT = 2 * ABYTES;  // X^T then dz^T
  constexpr int NIDX = 8, IBYTES = 512;  // index ring: per stage [op_rows 32 | op_inp 32 | op_cpos 64] ints
  __shared__ __attribute__((aligned(16))) char ring[wide::kSlots * SLOT];
  __shared__ __attribute__((aligned(16))) int iring[NIDX][IBYTES / 4];
  const int tid = threadIdx.x, lane = tid & 63, wave = wave_id();
  const int wr = wave & 3, wc = wave >> 2;
  const int NT = (a.Nw + TB - 1) / TB, MTm = (a.Kw + TB - 1) / TB;
  int tx, chunk_id;
  if (!xcd_tile(MTm * NT, a.nchunk, tx, chunk_id)) return;
  const int mt_ = tx % MTm, nt = tx / MTm;
  const int m0 = mt_ * TB, n0 = nt * TB;
  const int lo = chunk_id * a.chunk, hi = min(a.count, lo + a.chunk);
  const int nst = (hi - lo + 31) / 32;
  const char* zero = static_cast<const char*>(a.zero);
  const char* xbase = static_cast<const char*>(a.src);
  const size_t xstride = (size_t)(a.seg ? a.ld : a.tld) * 2, dstride = (size_t)a.gstride * 4;

  // index loads (wave 4): stage c's indices into ring slot c % NIDX
  auto issue_idx = [&](int c) {
    const int q0 = lo + c * 32;
    int* slot = iring[c % NIDX];
    const int r = lane & 31;
    const int qa = min(q0 + r, hi - 1);
    dma4_untracked(lane < 32 ? a.op_rows + qa : a.op_inp + qa, slot);
    const int qc = min(2 * q0 + lane, 2 * hi - 1);
    dma4_untracked(a.op_cpos + qc, slot + 64);
  };
  // this lane's unit of an op row: weight-row column (A) and gate column (B) it fetches.  All but the
  // rows' indices is fixed for the workgroup; a stage's index reads are issued together, ahead of its
  // loads (each untracked load is a compiler barrier, so a read placed between two loads would wait alone)
  const int u = lane & 31;
  int sr[4], sxi[4];
  size_t sxcol[4], sdcol[4];
  bool sxok[4], sdok[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = 2 * (4 * wr + i) + (lane >> 5);  // op row within the stage
    const int gu = u ^ (4 * (r & 3));              // global 16-byte unit of the tile row
    const int m = m0 + 8 * gu;                     // X^T: weight rows m .. m + 7
    const int child = a.seg ? min(m / a.HP, 1) : 0;
    sr[i] = r;
    sxi[i] = a.seg ? 64 + 2 * r + child : 32 + r;
    sxcol[i] = (size_t)(a.seg ? m - child * a.HP : m) * 2;
    sxok[i] = m < a.Kw;
    const int n = n0 + 8 * gu;                     // dz^T: gate columns n .. n + 7
    sdcol[i] = (size_t)n * 2;
    sdok[i] = n < a.Nw;
  }
  auto issue = [&](int c, char* sl) {
    const int* ix = iring[c % NIDX];
    const int q0 = lo + c * 32;
    int xi[4], di[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      xi[i] = ix[sxi[i]];
      di[i] = ix[sr[i]];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const bool live = q0 + sr[i] < hi;
      const bool xa = live && sxok[i] && xi[i] >= 0;
      dma16_untracked(xa ? xbase + (size_t)xi[i] * xstride + sxcol[i] : zero, sl + (4 * wr + i) * 1024);
      const bool da = live && sdok[i];
      dma16_untracked(da ? reinterpret_cast<const char*>(a.dz) + (size_t)di[i] * dstride + sdcol[i] : zero,
                      sl + ABYTES + (4 * wr + i) * 1024);
    }
  };

  // transposing-read offsets (see k_wgrad_bf16): group g = lane / 16, lane gi of the group
  const int g = lane >> 4, gi = lane & 15;
  int aoff[TM], boff[TN];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) aoff[tm] = wr * 64 + tm * 32 + 16 * (g & 1) + 4 * (gi & 3);
#pragma unroll
  for (int tn = 0; tn < TN; ++tn) boff[tn] = wc * 128 + tn * 32 + 16 * (g & 1) + 4 * (gi & 3);
  const int mrow = 8 * (g >> 1) + (gi >> 2);
  // bias column sums (tiles of the first weight-row tile only): thread t sums column t % 256 over
  // the stage rows 16 (t / 256) .. + 15
  const bool do_bias = a.bpart != nullptr && mt_ == 0;
  const int bc = tid & 255, bg = tid >> 8;
  float bsum = 0.f;

  f32x16 acc[TM][TN];
  zero_acc(acc);
  const bool dloads = wave < 4, iloads = wave == 4;
  if (nst > 0) {
    if (iloads) {
      for (int c = 0; c < min(nst, 6); ++c) issue_idx(c);
      if (nst > 5) vm_wait_n<6>();  // indices of stages 0-2 landed, 3-5 in flight
      else if (nst > 4) vm_wait_n<4>();
      else if (nst > 3) vm_wait_n<2>();
      else vm_wait();
    }
    wg_barrier();
    if (dloads)
      for (int c = 0; c < min(nst, 3); ++c) issue(c, ring + c * SLOT);
    for (int c = 0; c < nst; ++c) {
      if (dloads) {
        if (c + 2 < nst) vm_wait_n<2 * NL>();
        else if (c + 1 < nst) vm_wait_n<NL>();
        else vm_wait();
      }
      if (iloads) {  // indices of stage c + 3 (issued at stage c - 3) landed; c + 4, c + 5 may be in flight
        const int later = min(2, max(0, nst - 1 - (c + 3)));
        if (later == 2) vm_wait_n<4>();
        else if (later == 1) vm_wait_n<2>();
        else vm_wait();
      }
      wg_barrier();
      if (dloads && c + 3 < nst) issue(c + 3, ring + ((c + 3) & 3) * SLOT);
      if (iloads && c + 6 < nst) issue_idx(c + 6);
      __builtin_amdgcn_sched_barrier(0);
      const char* As = ring + (c & 3) * SLOT;
      const char* Bs = As + ABYTES;
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        uint4 af[TM], bf[TN];
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) {
          const uint2 l2 = ld_tr16(As, wgw_off(16 * s + mrow, aoff[tm]));
          const uint2 h2 = ld_tr16(As, wgw_off(16 * s + mrow + 4, aoff[tm]));
          af[tm] = make_uint4(l2.x, l2.y, h2.x, h2.y);
        }
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) {
          const uint2 l2 = ld_tr16(Bs, wgw_off(16 * s + mrow, boff[tn]));
          const uint2 h2 = ld_tr16(Bs, wgw_off(16 * s + mrow + 4, boff[tn]));
          bf[tn] = make_uint4(l2.x, l2.y, h2.x, h2.y);
        }
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
#pragma unroll
          for (int tn = 0; tn < TN; ++tn)
            acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, af[tm]),
                                                                 __builtin_bit_cast(bf16x8, bf[tn]), acc[tm][tn],
                                                                 0, 0, 0);
      }
      if (do_bias) {
#pragma unroll
        for (int r = 0; r < 16; ++r) bsum += bf2f(*reinterpret_cast<const uint16_t*>(Bs + wgw_off(16 * bg + r, bc)));
      }
    }
  }

  float* out = a.partial + (size_t)chunk_id * a.Kw * a.Nw;
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const int n = n0 + wc * 128 + tn * 32 + (lane & 31);
      if (n >= a.Nw) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + wr * 64 + tm * 32 + acc_row(r, lane);
        if (m < a.Kw) out[(size_t)m * a.Nw + n] = acc[tm][tn][r];
      }
    }
  if (do_bias && n0 + bc < a.Nw) a.bpart[((size_t)chunk_id * 2 + bg) * a.Nw + n0 + bc] = bsum;
}

// ---------------------------------------------------------------- fp32, wide: 256 x 256 tiles
// Ops with many rows: 256 weight rows x 256 gate columns per workgroup of 8 waves (wave tile 64 x 128),
// twice the operand reuse of the 128 x 128 tiles above, so each matrix instruction needs half the
// L2 -> LDS feed.  A stage is 16 op rows: X^T (16 x 256) and dz^T (16 x 256), 16 KB each, row-major in the
// op rows, one op row (1 KB) per direct-load instruction; odd rows have their 16-byte units permuted by
// ^ 8 as in the 128-column kernel.  Four stage slots keep three stages in flight (waves 0-3 load, four
// op rows of X and four of dz each); the op rows' indices reach LDS through an index ring six stages
// ahead of the data, loaded by wave 4 alone (one 4-byte-per-lane direct load per stage), so every wait
// counts only its own loads.
__global__ __launch_bounds__(wide::kThreads) void k_wgrad_f32_w(WgArgs a) {
  constexpr int TB = 256, TM = 2, TN = 4, NL = 8, RS = 16;
  constexpr int ABYTES = RS * TB * 4, SLOT = 2 * ABYTES;  // X^T then dz^T
  constexpr int NIDX = 8;  // index ring: per stage [op_rows 16 | op_inp 16 | op_cpos 32] ints
  __shared__ __attribute__((aligned(16))) char ring[wide::kSlots * SLOT];
  __shared__ __attribute__((aligned(16))) int iring[NIDX][64];
  const int tid = threadIdx.x, lane = tid & 63, wave = wave_id();
  const int wr = wave & 3, wc = wave >> 2, h = lane >> 5, l32 = lane & 31;
  const int NT = (a.Nw + TB - 1) / TB, MTm = (a.Kw + TB - 1) / TB;
  int tx, chunk_id;
  if (!xcd_tile(MTm * NT, a.nchunk, tx, chunk_id)) return;
  const int mt_ = tx % MTm, nt = tx / MTm;
  const int m0 = mt_ * TB, n0 = nt * TB;
  const int lo = chunk_id * a.chunk, hi = min(a.count, lo + a.chunk);
  const int nst = (hi - lo + RS - 1) / RS;
  const char* zero = static_cast<const char*>(a.zero);
  const char* xbase = static_cast<const char*>(a.src);
  const char* dzbase = reinterpret_cast<const char*>(a.dz);
  const size_t xstride = (size_t)(a.seg ? a.ld : a.tld) * 4, dstride = (size_t)a.gstride * 4;

  // index loads (wave 4): stage c's indices into ring slot c % NIDX (rows past the chunk clamped to its
  // last row)
  auto issue_idx = [&](int c) {
    const int q0 = lo + c * RS;
    const int* src;
    if (lane < 32) {
      const int q = min(q0 + (lane & 15), hi - 1);
      src = lane < 16 ? a.op_rows + q : a.op_inp + q;
    } else {
      src = a.op_cpos + min(2 * q0 + (lane - 32), 2 * hi - 1);
    }
    dma4_untracked(src, iring[c % NIDX]);
  };
  // waves 0-3: op rows 4 wr .. 4 wr + 3 of stage c; lane l fetches global unit l ^ 8 (r & 1) of each row
  // (the wave's indices come in four 16-byte reads, all before the first load)
  auto issue = [&](int c, char* sl) {
    const int* ix = iring[c % NIDX];
    const int q0 = lo + c * RS;
    int rw[4], inp[4], cp[8];
    *reinterpret_cast<int4*>(rw) = *reinterpret_cast<const int4*>(ix + 4 * wr);
    *reinterpret_cast<int4*>(inp) = *reinterpret_cast<const int4*>(ix + 16 + 4 * wr);
    *reinterpret_cast<int4*>(cp) = *reinterpret_cast<const int4*>(ix + 32 + 8 * wr);
    *reinterpret_cast<int4*>(cp + 4) = *reinterpret_cast<const int4*>(ix + 36 + 8 * wr);
    const char* xs[4];
    const char* ds[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 4 * wr + i;
      const int gu = lane ^ (8 * (r & 1));
      const bool live = q0 + r < hi;
      // X^T: weight rows m0 + 4 gu .. + 3
      const int m = m0 + 4 * gu;
      const int child = a.seg ? min(m / a.HP, 1) : 0;
      const int xi = a.seg ? (child ? cp[2 * i + 1] : cp[2 * i]) : inp[i];
      const int col = a.seg ? m - child * a.HP : m;
      xs[i] = live && m < a.Kw && xi >= 0 ? xbase + (size_t)xi * xstride + (size_t)col * 4 : zero;
      // dz^T: gate columns n0 + 4 gu .. + 3
      const int n = n0 + 4 * gu;
      ds[i] = live && n < a.Nw ? dzbase + (size_t)rw[i] * dstride + (size_t)n * 4 : zero;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      dma16_untracked(xs[i], sl + (4 * wr + i) * 1024);
      dma16_untracked(ds[i], sl + ABYTES + (4 * wr + i) * 1024);
    }
  };
  // fragment byte offsets: K value h of step s is op row 2 s + h
  int aoff[TM], boff[TN];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
    const int kw = wr * 64 + tm * 32 + l32;
    aoff[tm] = h * 1024 + ((kw >> 2) ^ (8 * h)) * 16 + (kw & 3) * 4;
  }
#pragma unroll
  for (int tn = 0; tn < TN; ++tn) {
    const int n = wc * 128 + tn * 32 + l32;
    boff[tn] = h * 1024 + ((n >> 2) ^ (8 * h)) * 16 + (n & 3) * 4;
  }
  // bias column sums (tiles of the first weight-row tile only): thread t sums column t % 256 over the
  // stage rows 8 (t / 256) .. + 7
  const bool do_bias = a.bpart != nullptr && mt_ == 0;
  const int bc = tid & 255, bg = tid >> 8;
  float bsum = 0.f;

  f32x16 acc[TM][TN];
  zero_acc(acc);
  const bool dloads = wave < 4, iloads = wave == 4;
  if (nst > 0) {
    if (iloads) {
      for (int c = 0; c < min(nst, 6); ++c) issue_idx(c);
      if (nst > 5) vm_wait_n<3>();  // indices of stages 0-2 landed, 3-5 in flight
      else if (nst > 4) vm_wait_n<2>();
      else if (nst > 3) vm_wait_n<1>();
      else vm_wait();
    }
    wg_barrier();
    if (dloads)
      for (int c = 0; c < min(nst, 3); ++c) issue(c, ring + c * SLOT);
    for (int c = 0; c < nst; ++c) {
      if (dloads) {
        if (c + 2 < nst) vm_wait_n<2 * NL>();
        else if (c + 1 < nst) vm_wait_n<NL>();
        else vm_wait();
      }
      if (iloads) {  // indices of stage c + 3 (issued at stage c - 3) landed; c + 4, c + 5 may be in flight
        const int later = min(2, max(0, nst - 1 - (c + 3)));
        if (later == 2) vm_wait_n<2>();
        else if (later == 1) vm_wait_n<1>();
        else vm_wait();
      }
      // the previous stage's LDS reads (bias sums included) are done before its slot is refilled
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      wg_barrier();
      if (dloads && c + 3 < nst) issue(c + 3, ring + ((c + 3) & 3) * SLOT);
      if (iloads && c + 6 < nst) issue_idx(c + 6);
      __builtin_amdgcn_sched_barrier(0);
      const char* As = ring + (c & 3) * SLOT;
      const char* Bs = As + ABYTES;
#pragma unroll
      for (int s = 0; s < RS / 2; ++s) {
        float av[TM], bv[TN];
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) av[tm] = *reinterpret_cast<const float*>(As + aoff[tm] + s * 2048);
#pragma unroll
        for (int tn = 0; tn < TN; ++tn) bv[tn] = *reinterpret_cast<const float*>(Bs + boff[tn] + s * 2048);
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
#pragma unroll
          for (int tn = 0; tn < TN; ++tn)
            acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[tm], bv[tn], acc[tm][tn], 0, 0, 0);
      }
      if (do_bias) {
#pragma unroll
        for (int r = 8 * bg; r < 8 * bg + 8; ++r)
          bsum += *reinterpret_cast<const float*>(Bs + r * 1024 + (((bc >> 2) ^ (8 * (r & 1))) * 16) + (bc & 3) * 4);
      }
    }
  }

  float* out = a.partial + (size_t)chunk_id * a.Kw * a.Nw;
#pragma unroll
  for (int tm = 0; tm < TM; ++tm)
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const int n = n0 + wc * 128 + tn * 32 + l32;
      if (n >= a.Nw) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + wr * 64 + tm * 32 + acc_row(r, lane);
        if (m < a.Kw) out[(size_t)m * a.Nw + n] = acc[tm][tn][r];
      }
    }
  if (do_bias && n0 + bc < a.Nw) a.bpart[((size_t)chunk_id * 2 + bg) * a.Nw + n0 + bc] = bsum;
}

// dW[row, col] += sum over chunks of partial[chunk, m, n], (m, n) in the padded layout
__global__ void k_wgrad_reduce(const float* partial, int nchunk, int Kw, int Nw, int seg, int H, int HP,
                               int in_dim, int G, int gcode, float* dW) {
  const size_t total = (size_t)Kw * Nw;
  for (size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (size_t)gridDim.x * blockDim.x) {
    const int m = (int)(idx / Nw), n = (int)(idx - (size_t)m * Nw);
    const int gz = n / HP, j = n - gz * HP, g = gate_of_code(gcode, gz);
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
    // chunk order; the loads of eight chunks go out at once (absent chunks add an exact 0)
    constexpr int U = 8;
    float s = 0.f;
    for (int c0 = 0; c0 < nchunk; c0 += U) {
      float t[U];
#pragma unroll
      for (int u = 0; u < U; ++u) t[u] = c0 + u < nchunk ? partial[(size_t)(c0 + u) * total + idx] : 0.f;
#pragma unroll
      for (int u = 0; u < U; ++u) s += t[u];
    }
    dW[(size_t)row * G * H + g * H + j] += s;
  }
}

// column sums of dz (fp32, or bf16 at the start of each row) over one chunk of an op's rows
__global__ void k_bias_partial(const int* op_rows, int count, int chunk, const float* dz, int gstride, int Nw,
                               int bf, float* bpart) {
  const int c = blockIdx.x;
  const int n = blockIdx.y * blockDim.x + threadIdx.x;
  if (n >= Nw) return;
  const int lo = c * chunk, hi = min(count, lo + chunk);
  float s = 0.f;
  for (int i = lo; i < hi; ++i) {
    const float* row = dz + (size_t)op_rows[i] * gstride;
    s += bf ? bf2f(reinterpret_cast<const uint16_t*>(row)[n]) : row[n];
  }
  bpart[(size_t)c * Nw + n] = s;
}

// db[col] += sum over partial rows, 64 columns per block: four thread groups sum interleaved partial
// rows, then the four sums are added in a fixed order (the result does not depend on scheduling)
__global__ void k_bias_reduce(const float* bpart, int nparts, int Nw, int H, int HP, int gcode, float* dbias) {
  __shared__ float red[4][64];
  const int cg = threadIdx.x & 63, pg = threadIdx.x >> 6;
  const int n = blockIdx.x * 64 + cg;
  float s = 0.f;
  if (n < Nw) {
    constexpr int U = 8;  // partial rows pg, pg + 4, ... in order, eight loads in flight
    for (int c0 = pg; c0 < nparts; c0 += 4 * U) {
      float t[U];
#pragma unroll
      for (int u = 0; u < U; ++u) t[u] = c0 + 4 * u < nparts ? bpart[(size_t)(c0 + 4 * u) * Nw + n] : 0.f;
#pragma unroll
      for (int u = 0; u < U; ++u) s += t[u];
    }
  }
  red[pg][cg] = s;
  __syncthreads();
  if (pg != 0 || n >= Nw) return;
  const int gz = n / HP, j = n - gz * HP;
  if (j >= H) return;
  dbias[gate_of_code(gcode, gz) * H + j] += (red[0][cg] + red[1][cg]) + (red[2][cg] + red[3][cg]);
}

}  // namespace

// Chunks of an op's rows: a multiple of 8 (each XCD reduces whole chunks, all tiles of a chunk on one
// XCD) chosen so that an XCD's workgroups fill its resident slots in whole rounds (a launch of 2.2 rounds
// runs as 3), with chunks of at least min_rows and (if possible) at most max_rows rows.  Short chunks keep
// the workgroups that an XCD runs at once on the same rows, so the rows they share stay in its L2
// (measured on 1.25 M rows: 64 chunks of ~20 k rows cut the contraction from 44.6 to 42.2 ms against 8
// chunks; more chunks gain nothing and cost more in the partial-tile reduction).
static int wgrad_chunks(long long tiles, int count, int min_rows, int max_rows, int slots_per_xcd,
                        double* fill = nullptr) {
  const long long most8 = std::max(1, count / (8 * min_rows));  // chunks per XCD at most
  const long long least8 = std::min<long long>(most8, std::max<long long>(1, ((long long)count + 8LL * max_rows - 1) /
                                                                                 (8LL * max_rows)));
  int best = (int)least8;
  double best_eff = 0.0;
  for (int c8 = (int)least8; c8 <= std::max<long long>(least8, std::min<long long>(most8, 32)); ++c8) {
    const long long wg = tiles * c8;
    const double eff = (double)wg / (double)(((wg + slots_per_xcd - 1) / slots_per_xcd) * slots_per_xcd);
    if (eff > best_eff + 1e-9) {
      best = c8;
      best_eff = eff;
    }
    if (eff >= 0.9 && wg >= slots_per_xcd) break;
  }
  if (fill) *fill = best_eff;
  return 8 * best;
}

WgradSplit wgrad_split(int count, int Kw, int Nw, int dtype) {
  WgradSplit w;
  if (count <= 0 || Kw <= 0 || Nw <= 0) return w;
  // ops with many rows: 256 x 256 tiles (twice the operand reuse of 128 x 128), one workgroup per CU.
  // fp32 takes them only where their workgroups fill the compute units' slots (at least 90 %): on 65 k
  // rows, H = 256, the node weights' 10 tiles gain 5 % over 128 x 128, the leaf weights' 3 tiles (75 %
  // full) lose 11 %.  bf16 takes them from 16 k rows on where at least 70 % of the 256 x 256 tiles' area
  // is weight (H = 300: 74 %; the two ops of 32 k rows each, 0.27 -> 0.22 ms with their reductions)
  const long long wtiles = (long long)((Kw + 255) / 256) * ((Nw + 255) / 256);
  if (dtype == FOLD_BF16) {
    const double area = (double)Kw * Nw / ((double)wtiles * 65536.0);
    w.wide = count >= 65536 || (count >= 16384 && area >= 0.7);
  } else if (count >= kWgWideF32Rows) {
    double fill = 0.0;
    wgrad_chunks(wtiles, count, 1024, 20480, 32, &fill);
    w.wide = fill >= 0.9;
  }
  const long long tiles = w.wide ? wtiles : (long long)((Kw + kTM - 1) / kTM) * ((Nw + 127) / 128);
  w.nchunk = wgrad_chunks(tiles, count, w.wide ? 1024 : 512, w.wide ? 20480 : (1 << 30), w.wide ? 32 : 64);
  w.chunk = round_up((count + w.nchunk - 1) / w.nchunk, 64);
  w.nchunk = (count + w.chunk - 1) / w.chunk;
  // bias partial rows: one per (chunk, weight-row tile, thread group)
  w.bparts = w.wide ? w.nchunk * 2 : w.nchunk * ((Kw + kTM - 1) / kTM) * (dtype == FOLD_BF16 ? 2 : 256 / kWgNW);
  return w;
}

void launch_wgrad(int dtype, const WgArgs& a, hipStream_t st) {
  if (a.count <= 0) return;
  ProfScope prof(dtype == FOLD_BF16 ? "wgrad.bf16" : "wgrad.f32", st);
  if (a.wide) {
    dim3 grid(xcd_grid(((a.Kw + 255) / 256) * ((a.Nw + 255) / 256), a.nchunk));
    if (dtype == FOLD_BF16) hipLaunchKernelGGL(k_wgrad_bf16_w, grid, dim3(wide::kThreads), 0, st, a);
    else hipLaunchKernelGGL(k_wgrad_f32_w, grid, dim3(wide::kThreads), 0, st, a);
  } else if (dtype == FOLD_BF16) {
    dim3 grid(xcd_grid(((a.Kw + kTM - 1) / kTM) * ((a.Nw + 127) / 128), a.nchunk));
    hipLaunchKernelGGL(k_wgrad_bf16, grid, dim3(kThreads), 0, st, a);
  } else {
    dim3 grid(xcd_grid(((a.Kw + kTM - 1) / kTM) * ((a.Nw + kWgNW - 1) / kWgNW), a.nchunk));
    hipLaunchKernelGGL(k_wgrad_f32<kWgNW>, grid, dim3(kThreads), 0, st, a);
  }
}

void launch_wgrad_reduce(const float* partial, int nchunk, int Kw, int Nw, int seg, int H, int HP, int in_dim,
                         int G, int gcode, float* dW, hipStream_t st) {
  ProfScope prof("wgrad_reduce", st);
  const size_t total = (size_t)Kw * Nw;
  const unsigned blocks = (unsigned)std::min<size_t>((total + 255) / 256, 65536);
  hipLaunchKernelGGL(k_wgrad_reduce, dim3(blocks), dim3(256), 0, st, partial, nchunk, Kw, Nw, seg, H, HP, in_dim,
                     G, gcode, dW);
}

void launch_bias_partial(const int* op_rows, int count, int chunk, int nchunk, const float* dz, int gstride, int Nw,
                         int bf, float* bpart, hipStream_t st) {
  if (count <= 0) return;
  ProfScope prof("bias_partial", st);
  hipLaunchKernelGGL(k_bias_partial, dim3(nchunk, (Nw + 255) / 256), dim3(256), 0, st, op_rows, count, chunk, dz,
                     gstride, Nw, bf, bpart);
}

void launch_bias_reduce(const float* bpart, int nchunk, int Nw, int H, int HP, int gcode, float* dbias,
                        hipStream_t st) {
  if (nchunk <= 0) return;
  ProfScope prof("bias_reduce", st);
  hipLaunchKernelGGL(k_bias_reduce, dim3((Nw + 63) / 64), dim3(256), 0, st, bpart, nchunk, Nw, H, HP, gcode, dbias);
}

}  // namespace fold
