// Matrix-core building blocks for gfx950: 32x32 MFMA tiles fed from LDS.
//
// One wave computes a 32 x 32 fp32 tile per instruction:
//   fp32 operands  v_mfma_f32_32x32x2_f32   (K = 2 per instruction, one element per lane)
//   bf16 operands  v_mfma_f32_32x32x16_bf16 (K = 16 per instruction, eight elements per lane)
// Operand fragments: lane l supplies row (l % 32) of A and column (l % 32) of B, for the
// K slice starting at (l / 32) * KPL.  Both A and B tiles live in LDS as [row][k] with k
// contiguous, so the two fragment loads are the same access pattern.
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
  static constexpr int PAD = 4;    // row padding in LDS (keeps 16-byte alignment)
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
  static constexpr int PAD = 8;
  typedef bf16x8 frag;
  __device__ static __forceinline__ frag load(const uint16_t* p) { return *reinterpret_cast<const bf16x8*>(p); }
  __device__ static __forceinline__ f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};

// row of the 32x32 result tile held by register r of lane `lane`
__device__ __forceinline__ int acc_row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }

// 16-byte load of elements [col, col + VEC) of a row; elements at or beyond `width` read as zero.
// The caller guarantees col + VEC <= the row's allocated stride.
template <typename T>
__device__ __forceinline__ uint4 load_row_vec(const T* row, int col, int width) {
  constexpr int VEC = 16 / sizeof(T);
  uint4 v = make_uint4(0u, 0u, 0u, 0u);
  if (col >= width) return v;
  v = *reinterpret_cast<const uint4*>(row + col);
  const int valid = width - col;
  if (valid < VEC) {
    uint32_t w[4] = {v.x, v.y, v.z, v.w};
    if (sizeof(T) == 4) {
      for (int e = 0; e < 4; ++e)
        if (e >= valid) w[e] = 0u;
    } else {
      for (int e = 0; e < 8; ++e)
        if (e >= valid) w[e >> 1] &= (e & 1) ? 0x0000ffffu : 0xffff0000u;
    }
    v = make_uint4(w[0], w[1], w[2], w[3]);
  }
  return v;
}

// 16 bytes of LDS operand from fp32 source values: 4 floats (T = float) or 8 floats rounded to bf16.
template <typename T>
__device__ __forceinline__ uint4 pack_from_f32(const float* src, int valid);

template <>
__device__ __forceinline__ uint4 pack_from_f32<float>(const float* src, int valid) {
  uint4 v = make_uint4(0u, 0u, 0u, 0u);
  if (valid >= 4) {
    float4 f = *reinterpret_cast<const float4*>(src);
    v = make_uint4(__float_as_uint(f.x), __float_as_uint(f.y), __float_as_uint(f.z), __float_as_uint(f.w));
  } else {
    uint32_t w[4] = {0u, 0u, 0u, 0u};
    for (int e = 0; e < valid; ++e) w[e] = __float_as_uint(src[e]);
    v = make_uint4(w[0], w[1], w[2], w[3]);
  }
  return v;
}

template <>
__device__ __forceinline__ uint4 pack_from_f32<uint16_t>(const float* src, int valid) {
  float f[8];
  if (valid >= 8) {
    float4 a = *reinterpret_cast<const float4*>(src);
    float4 b = *reinterpret_cast<const float4*>(src + 4);
    f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w; f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
  } else {
    for (int e = 0; e < 8; ++e) f[e] = e < valid ? src[e] : 0.f;
  }
  uint32_t w[4];
  for (int e = 0; e < 4; ++e) w[e] = (uint32_t)f2bf(f[2 * e]) | ((uint32_t)f2bf(f[2 * e + 1]) << 16);
  return make_uint4(w[0], w[1], w[2], w[3]);
}

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

}  // namespace fold
