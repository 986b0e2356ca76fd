// Direct global -> LDS staging for the matrix-core kernels (gfx950).
//
// gfx950 can load 16 bytes per lane from global memory straight into LDS (global_load_lds_dwordx4):
// the data never passes through VGPRs, so a K loop needs no staging registers and no LDS store phase,
// and the loads of stage c + 1 run while the matrix cores work on stage c from the other LDS buffer.
// One wave instruction writes 1024 contiguous LDS bytes, lane l at byte 16 l; which global 16 bytes
// each lane fetches is free, and that choice is what lays the tile out in LDS.
#pragma once

#include "common.h"
#include "mfma.h"

namespace fold {

// lane l of the wave copies 16 bytes from src (its own address) to lds + 16 l (lds: one value per wave)
__device__ __forceinline__ void dma16(const void* src, void* lds) {
  __builtin_amdgcn_global_load_lds(src, lds, 16, 0, 0);
}

// The same load issued as inline assembly, which the compiler does not track.  Its own tracking of
// direct-to-LDS loads keeps only a few of them apart and otherwise waits for all of them before any LDS
// read, which would drain a pipeline that keeps two stages in flight.  A kernel using it waits for its
// loads explicitly (vm_wait / vm_wait_n) before the barrier that publishes them.
__device__ __forceinline__ void dma16_untracked(const void* src, void* lds) {
  const uint32_t base = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)lds);
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(base), "v"(src) : "memory", "m0");
}

// wait until this wave's global loads, direct-to-LDS ones included, have landed
__device__ __forceinline__ void vm_wait() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// wait until at most N of this wave's global loads are still outstanding (loads complete in order)
template <int N>
__device__ __forceinline__ void vm_wait_n() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Workgroup barrier without the release fence of __syncthreads(), which waits for every outstanding
// global load of the wave -- the stages still in flight included.  Callers wait for what must have
// landed (vm_wait_n) themselves; LDS reads of the previous stage are complete because the matrix
// instructions that consumed them were issued before the barrier.
__device__ __forceinline__ void wg_barrier() { asm volatile("s_barrier" ::: "memory"); }

__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// ---------------------------------------------------------------- row tiles
// A stage of a row operand: ROWS rows x 128 bytes of K (32 fp32 or 64 bf16 values).  Row r's 16-byte
// unit u sits in unit slot 8 r + (u ^ ((r >> 1) & 7)).  A 16-byte LDS read is served for 16 lanes at a
// time over 64 banks (16 groups of 16 bytes); sixteen consecutive rows reading the same unit land in
// slots whose (r & 1, u ^ ((r >> 1) & 7)) are all distinct, i.e. in 16 distinct bank groups.  Wave
// instruction t fills rows 8 t .. 8 t + 7: lane l fetches unit (l & 7) ^ swz(8 t + (l >> 3)) of row
// 8 t + (l >> 3).
__device__ __forceinline__ int swz(int r) { return (r >> 1) & 7; }
__device__ __forceinline__ int row_of_lane(int lane) { return lane >> 3; }
__device__ __forceinline__ int unit_of_lane(int lane, int t) { return (lane & 7) ^ swz(8 * t + (lane >> 3)); }

// byte offset of row r, unit u in a row tile
__device__ __forceinline__ int rt_off(int r, int u) { return (r * 8 + (u ^ swz(r))) * 16; }

// acc[TM][TN] += A . B^T over one 128-byte stage of K, A rows arow0 + 32 tm + (lane % 32), B rows
// brow0 + 32 tn + (lane % 32).  The K order inside the stage is permuted the same way for A and B:
// lane half h takes the units 4 h + q, q = 0..3, one 16-byte read each, which feed four fp32
// instructions (one K value each, K = 2 per instruction over the two halves) or one bf16 instruction
// (eight K values, K = 16 over the two halves).
template <typename T, int TM, int TN>
__device__ __forceinline__ void mma_rows(const char* As, const char* Bs, f32x16 (&acc)[TM][TN], int arow0,
                                         int brow0, int lane) {
  const int h = lane >> 5, l32 = lane & 31;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int u = 4 * h + q;
    uint4 a[TM], b[TN];
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) a[tm] = *reinterpret_cast<const uint4*>(As + rt_off(arow0 + tm * 32 + l32, u));
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) b[tn] = *reinterpret_cast<const uint4*>(Bs + rt_off(brow0 + tn * 32 + l32, u));
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

// Issue functor for operands whose rows do not change along K: every lane keeps one pointer per
// instruction (row and unit already applied) and a stage adds 128 bytes.
template <int PA, int PB>
struct FixedRowsIssue {
  const char* ap[PA];
  const char* bp[PB];
  int wave;
  __device__ __forceinline__ void operator()(int c, char* Ad, char* Bd) const {
    const int off = c * 128;
#pragma unroll
    for (int i = 0; i < PA; ++i) dma16(ap[i] + off, Ad + (wave * PA + i) * 1024);
#pragma unroll
    for (int i = 0; i < PB; ++i) dma16(bp[i] + off, Bd + (wave * PB + i) * 1024);
  }
};

// Double-buffered K loop over nst stages of row tiles.  issue(c, A, B) starts the direct loads of
// stage c into LDS buffers A and B; stage c + 1 is in flight while stage c is multiplied, and one
// barrier per stage both publishes the landed stage and frees the buffer the next loads overwrite.
// The loop is unrolled by two so that every LDS access names its buffer: the compiler then sees that
// the reads of one buffer do not depend on the loads in flight into the other and adds no wait.  A
// scheduling barrier after each issue keeps the loads ahead of the matrix instructions (left alone,
// the scheduler sinks them below the stage's MFMAs, which exposes their whole latency).
template <typename T, int TM, int TN, class ISSUE>
__device__ __forceinline__ void row_loop(int nst, ISSUE& issue, char* A0, char* A1, char* B0, char* B1,
                                         f32x16 (&acc)[TM][TN], int arow0, int brow0, int lane) {
  if (nst <= 0) return;
  issue(0, A0, B0);
  vm_wait();
  __syncthreads();
  int c = 0;
  for (; c + 2 <= nst; c += 2) {
    issue(c + 1, A1, B1);
    __builtin_amdgcn_sched_barrier(0);
    mma_rows<T, TM, TN>(A0, B0, acc, arow0, brow0, lane);
    vm_wait();
    __syncthreads();
    if (c + 2 < nst) issue(c + 2, A0, B0);
    __builtin_amdgcn_sched_barrier(0);
    mma_rows<T, TM, TN>(A1, B1, acc, arow0, brow0, lane);
    vm_wait();
    __syncthreads();
  }
  if (c < nst) mma_rows<T, TM, TN>(A0, B0, acc, arow0, brow0, lane);  // odd count: the last stage is in A0
}

}  // namespace fold
