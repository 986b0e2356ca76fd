// Achievable-peak probes (gfx950): an MFMA loop and a device-to-device stream copy, timed with HIP
// events, so that roofline fractions can be quoted against both the datasheet and what this GPU
// actually sustains.

#include <hip/hip_runtime.h>

#include "common.h"
#include "internal.h"

namespace fold {

namespace {

constexpr int kProbeWaves = 4;   // waves per workgroup
constexpr int kProbeAcc = 4;     // independent accumulators per wave

__global__ __launch_bounds__(256) void k_probe_mfma_f32(float* out, int iters) {
  f32x16 acc[kProbeAcc];
  for (int t = 0; t < kProbeAcc; ++t)
    for (int r = 0; r < 16; ++r) acc[t][r] = 0.f;
  const float a = 1e-3f * (float)(threadIdx.x & 63), b = 0.5f;
  for (int i = 0; i < iters; ++i)
#pragma unroll
    for (int t = 0; t < kProbeAcc; ++t) acc[t] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc[t], 0, 0, 0);
  float s = 0.f;
  for (int t = 0; t < kProbeAcc; ++t)
    for (int r = 0; r < 16; ++r) s += acc[t][r];
  out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

__global__ __launch_bounds__(256) void k_probe_mfma_bf16(float* out, int iters) {
  f32x16 acc[kProbeAcc];
  for (int t = 0; t < kProbeAcc; ++t)
    for (int r = 0; r < 16; ++r) acc[t][r] = 0.f;
  bf16x8 a, b;
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)(1e-3f * (float)(threadIdx.x & 63));
    b[e] = (__bf16)0.5f;
  }
  for (int i = 0; i < iters; ++i)
#pragma unroll
    for (int t = 0; t < kProbeAcc; ++t) acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[t], 0, 0, 0);
  float s = 0.f;
  for (int t = 0; t < kProbeAcc; ++t)
    for (int r = 0; r < 16; ++r) s += acc[t][r];
  out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

// The same loops with operands of random bits: every lane holds four different operand registers per side
// (uniform in [-1, 1)), cycled over the accumulators.  The matrix cores' power draw, and with it the clock the
// GPU holds, depends on the operand bits; random data is what the contractions multiply.
__device__ __forceinline__ float probe_rand(uint32_t& x) {
  x ^= x >> 15;
  x *= 2246822519u;
  x ^= x >> 13;
  x *= 3266489917u;
  x ^= x >> 16;
  return (float)(x & 0xffffu) * (1.f / 32768.f) - 1.f;
}

template <bool BF>
__global__ __launch_bounds__(256) void k_probe_mfma_rand(float* out, int iters) {
  f32x16 acc[kProbeAcc];
  for (int t = 0; t < kProbeAcc; ++t)
    for (int r = 0; r < 16; ++r) acc[t][r] = 0.f;
  uint32_t x = (blockIdx.x * 256u + threadIdx.x) * 2654435761u + 12345u;
  bf16x8 ab[4], bb[4];
  float af[4], bfl[4];
  for (int q = 0; q < 4; ++q) {
    af[q] = probe_rand(x);
    bfl[q] = probe_rand(x);
    for (int e = 0; e < 8; ++e) {
      ab[q][e] = (__bf16)probe_rand(x);
      bb[q][e] = (__bf16)probe_rand(x);
    }
  }
  for (int i = 0; i < iters; i += 4)
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int t = 0; t < kProbeAcc; ++t) {
        if constexpr (BF)
          acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ab[(t + u) & 3], bb[t & 3], acc[t], 0, 0, 0);
        else
          acc[t] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[(t + u) & 3], bfl[t & 3], acc[t], 0, 0, 0);
      }
  float s = 0.f;
  for (int t = 0; t < kProbeAcc; ++t)
    for (int r = 0; r < 16; ++r) s += acc[t][r];
  out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

__global__ void k_probe_copy(const uint4* __restrict__ src, uint4* __restrict__ dst, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}

}  // namespace

int32_t probe_mfma(int dtype, bool random_operands, hipStream_t st, double* tflops) {
  int dev = 0, cus = 0;
  FOLD_HIP_CHECK(hipGetDevice(&dev));
  FOLD_HIP_CHECK(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
  const int blocks = cus * 8;  // eight waves per SIMD
  float* out = nullptr;
  FOLD_HIP_CHECK(hipMalloc(&out, (size_t)blocks * 256 * sizeof(float)));
  hipEvent_t e0, e1;
  (void)hipEventCreate(&e0);
  (void)hipEventCreate(&e1);
  const int iters = dtype == FOLD_BF16 ? 20000 : 4000;  // multiples of 4 (the random loops' unrolling)
  auto launch = [&]() {
    if (random_operands) {
      if (dtype == FOLD_BF16)
        hipLaunchKernelGGL(k_probe_mfma_rand<true>, dim3(blocks), dim3(256), 0, st, out, iters);
      else
        hipLaunchKernelGGL(k_probe_mfma_rand<false>, dim3(blocks), dim3(256), 0, st, out, iters);
    } else if (dtype == FOLD_BF16) {
      hipLaunchKernelGGL(k_probe_mfma_bf16, dim3(blocks), dim3(256), 0, st, out, iters);
    } else {
      hipLaunchKernelGGL(k_probe_mfma_f32, dim3(blocks), dim3(256), 0, st, out, iters);
    }
  };
  launch();  // warm-up
  (void)hipEventRecord(e0, st);
  launch();
  (void)hipEventRecord(e1, st);
  hipError_t err = hipEventSynchronize(e1);
  float ms = 0.f;
  if (err == hipSuccess) err = hipEventElapsedTime(&ms, e0, e1);
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  (void)hipFree(out);
  if (err != hipSuccess) {
    set_error(std::string("fold_probe_mfma: ") + hipGetErrorString(err));
    return FOLD_E_DEVICE;
  }
  const double per = dtype == FOLD_BF16 ? 2.0 * 32 * 32 * 16 : 2.0 * 32 * 32 * 2;
  const double flops = per * kProbeAcc * (double)iters * blocks * kProbeWaves;
  *tflops = flops / (ms * 1e-3) / 1e12;
  return FOLD_OK;
}

int32_t probe_copy(void* dst, const void* src, size_t bytes, hipStream_t st, double* gbs) {
  const size_t n = bytes / 16;
  int dev = 0, cus = 0;
  FOLD_HIP_CHECK(hipGetDevice(&dev));
  FOLD_HIP_CHECK(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
  const unsigned blocks = (unsigned)std::min<size_t>((n + 255) / 256, (size_t)cus * 16);
  hipEvent_t e0, e1;
  (void)hipEventCreate(&e0);
  (void)hipEventCreate(&e1);
  ProfScope prof("probe_copy", st);
  hipLaunchKernelGGL(k_probe_copy, dim3(blocks), dim3(256), 0, st, static_cast<const uint4*>(src),
                     static_cast<uint4*>(dst), n);
  (void)hipEventRecord(e0, st);
  for (int r = 0; r < 5; ++r)
    hipLaunchKernelGGL(k_probe_copy, dim3(blocks), dim3(256), 0, st, static_cast<const uint4*>(src),
                       static_cast<uint4*>(dst), n);
  (void)hipEventRecord(e1, st);
  hipError_t err = hipEventSynchronize(e1);
  float ms = 0.f;
  if (err == hipSuccess) err = hipEventElapsedTime(&ms, e0, e1);
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  if (err != hipSuccess) {
    set_error(std::string("fold_probe_copy: ") + hipGetErrorString(err));
    return FOLD_E_DEVICE;
  }
  *gbs = 5.0 * 2.0 * (double)(n * 16) / (ms * 1e-3) / 1e9;
  return FOLD_OK;
}

}  // namespace fold
