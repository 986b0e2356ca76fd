// Wide-level contraction tiles for gfx950: 256 rows per workgroup of 8 waves, 64-byte K stages.
//
// The L2 -> compute-unit fabric delivers about 13-17 TB/s to the whole chip (direct-to-LDS or into
// registers alike), so a bf16 contraction reaches a large share of the matrix-core peak only if every
// byte brought into LDS feeds enough multiply-adds.  A 256-row x 320-column tile (the 5 gate blocks of 64
// hidden units) does 146 FLOP per operand byte, twice the 128 x 160 tile.  Its operands take 36 KB per
// 64-byte stage; four stage slots (144 KB) keep three stages in flight, which is what the fabric needs
// to run near its bandwidth once every compute unit streams at once.
//
// Stage layout: row r of an operand tile holds 64 bytes of K, its four 16-byte units u at
// r * 64 + 16 (u ^ ((r >> 2) & 3)).  A 16-byte LDS read is served for 16 lanes at a time over 64 banks
// (16 groups of 16 bytes); 16 consecutive rows reading the same unit then fall in 16 distinct groups.
// One direct-load instruction fills 16 rows: lane l fetches unit (l & 3) ^ swz of row l >> 2.
#pragma once

#include "common.h"
#include "dma.h"
#include "mfma.h"

namespace fold {

namespace wide {

constexpr int kRows = 256;   // rows per workgroup tile
constexpr int kThreads = 512;
constexpr int kSlots = 4;    // stage slots in LDS; kSlots - 1 stages in flight

__device__ __forceinline__ int swz(int r) { return (r >> 2) & 3; }
// byte offset of row r, unit u in a stage tile
__device__ __forceinline__ int off(int r, int u) { return r * 64 + ((u ^ swz(r)) << 4); }
// row (within the 16 rows of one load instruction) and unit this lane fetches
__device__ __forceinline__ int lane_row(int lane) { return lane >> 2; }
__device__ __forceinline__ int lane_unit(int lane) { return (lane & 3) ^ swz(lane >> 2); }

// acc[TM][TN] += A . B^T over one 64-byte stage of K.  Lane half h takes units 2 h + q (q = 0, 1) for
// both operands, so the K order inside the stage is permuted identically on both sides.
template <typename T, int TM, int TN>
__device__ __forceinline__ void mma(const char* As, const char* Bs, f32x16 (&acc)[TM][TN], int arow0, int brow0,
                                    int lane) {
  const int h = lane >> 5, l32 = lane & 31;
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int u = 2 * h + q;
    uint4 a[TM], b[TN];
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) a[tm] = *reinterpret_cast<const uint4*>(As + off(arow0 + tm * 32 + l32, u));
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) b[tn] = *reinterpret_cast<const uint4*>(Bs + off(brow0 + tn * 32 + l32, u));
    if constexpr (sizeof(T) == 4) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) {
          const float av = __uint_as_float(e == 0 ? a[tm].x : e == 1 ? a[tm].y : e == 2 ? a[tm].z : a[tm].w);
#pragma unroll
          for (int tn = 0; tn < TN; ++tn) {
            const float bv = __uint_as_float(e == 0 ? b[tn].x : e == 1 ? b[tn].y : e == 2 ? b[tn].z : b[tn].w);
            acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, acc[tm][tn], 0, 0, 0);
          }
        }
      }
    } else {
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
          acc[tm][tn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a[tm]),
                                                               __builtin_bit_cast(bf16x8, b[tn]), acc[tm][tn], 0,
                                                               0, 0);
    }
  }
}

// K loop over nst stages through the kSlots-slot ring at `ring` (slot s at ring + s * SLOT, its A rows
// first, then its B rows at + BOFF).  issue(c, slot) starts the direct loads of stage c on the waves
// that load (NL instructions each, untracked by the compiler); the others issue none.  At stage c a
// loading wave waits until only the loads of the stages after c are outstanding, then one barrier
// publishes stage c to every wave and frees the slot that stage c + 3 overwrites (last read at stage
// c - 1).
template <typename T, int TM, int TN, int NL, int SLOT, int BOFF, class ISSUE>
__device__ __forceinline__ void loop(int nst, ISSUE& issue, bool loads, char* ring, f32x16 (&acc)[TM][TN],
                                     int arow0, int brow0, int lane) {
  static_assert(kSlots == 4, "the waits below assume three stages in flight");
#pragma unroll
  for (int c = 0; c < kSlots - 1; ++c)
    if (c < nst) issue(c, ring + c * SLOT);
  for (int c = 0; c < nst; ++c) {
    if (loads) {
      if (c + 2 < nst) vm_wait_n<2 * NL>();
      else if (c + 1 < nst) vm_wait_n<NL>();
      else vm_wait();
    }
    wg_barrier();
    if (c + 3 < nst) issue(c + 3, ring + ((c + 3) & 3) * SLOT);
    __builtin_amdgcn_sched_barrier(0);
    const char* s = ring + (c & 3) * SLOT;
    mma<T, TM, TN>(s, s + BOFF, acc, arow0, brow0, lane);
  }
}

}  // namespace wide

}  // namespace fold
