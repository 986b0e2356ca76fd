// Parameter packing (gfx950): canonical row-major weights -> the layouts the matrix-core kernels read.
//
//   mode 0  forward   Wf[n'][k'], n-major.  n' walks hidden units in blocks of 32 with the G gate
//                     blocks of one unit block adjacent (n' = ub*G*32 + g*32 + u), so one workgroup's
//                     B tile holds every gate of its 32 units.  k' runs over the input segment
//                     (padded to a multiple of 64) and then one segment of HP per child slot.
//   mode 1  backward  Wb_rec[c*HP + jin][g*HP + j] = W_rec[c*H + jin][g*H + j]  (n-major for dz . W^T)
//   mode 2  backward  Wb_in[jin][g*HP + j]          = W_in[jin][g*H + j]
//   mode 3  bias      b[g*HP + j]                   = bias[g*H + j]
// The gate blocks packed are the canonical gates named by a gate code (gate_of_code): all G of them, or a
// subset in a compact order (the live gates of Tree-LSTM leaves); the canonical matrices have GC gate
// blocks.  Padding entries are zero.

#include <hip/hip_runtime.h>

#include <algorithm>

#include "common.h"
#include "internal.h"
#include "mfma.h"

namespace fold {

namespace {

template <typename T>
__global__ void k_pack(int mode, int G, int GC, int gcode, int H, int HP, int in_dim, int INP, int arity, int Kf,
                       const T* W_in, const T* W_rec, T* dst, size_t count) {
  for (size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x; idx < count;
       idx += (size_t)gridDim.x * blockDim.x) {
    float v = 0.f;
    const int GH = GC * H;
    const unsigned i32 = (unsigned)idx;  // packed matrices have fewer than 2^32 entries: 32-bit divisions
    if (mode == 0) {
      const int np = (int)(i32 / (unsigned)Kf), kp = (int)(i32 - (unsigned)np * (unsigned)Kf);
      const int ub = np / (G * 32), rem = np - ub * G * 32, j = ub * 32 + (rem & 31);
      const int g = gate_of_code(gcode, rem / 32);
      if (j < H) {
        if (kp < INP) {
          if (kp < in_dim) v = to_f32<T>(W_in[(size_t)kp * GH + g * H + j]);
        } else {
          const int kk = kp - INP, c = kk / HP, jin = kk - c * HP;
          if (jin < H && c < arity) v = to_f32<T>(W_rec[(size_t)(c * H + jin) * GH + g * H + j]);
        }
      }
    } else {
      const int KB = G * HP;
      const int n = (int)(i32 / (unsigned)KB), kk = (int)(i32 - (unsigned)n * (unsigned)KB);
      const int gc = kk / HP, j = kk - gc * HP, g = gate_of_code(gcode, gc);
      if (j < H) {
        if (mode == 1) {
          const int c = n / HP, jin = n - c * HP;
          if (jin < H) v = to_f32<T>(W_rec[(size_t)(c * H + jin) * GH + g * H + j]);
        } else {
          if (n < in_dim) v = to_f32<T>(W_in[(size_t)n * GH + g * H + j]);
        }
      }
    }
    dst[idx] = from_f32<T>(v);
  }
}

__global__ void k_pack_bias(int G, int gcode, int H, int HP, const float* bias, float* dst) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= G * HP) return;
  const int gc = idx / HP, j = idx - gc * HP;
  dst[idx] = j < H ? bias[gate_of_code(gcode, gc) * H + j] : 0.f;
}

}  // namespace

void launch_pack(int dtype, int mode, int G, int GC, int gcode, int H, int HP, int in_dim, int INP, int arity, int Kf,
                 const void* W_in, const void* W_rec, const float* bias, void* dst, size_t count, hipStream_t st) {
  if (count == 0) return;
  if (mode == 3) {
    hipLaunchKernelGGL(k_pack_bias, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, st, G, gcode, H, HP, bias,
                       static_cast<float*>(dst));
    return;
  }
  const unsigned blocks = (unsigned)std::min<size_t>((count + 255) / 256, 65536);
  if (dtype == FOLD_BF16)
    hipLaunchKernelGGL(k_pack<uint16_t>, dim3(blocks), dim3(256), 0, st, mode, G, GC, gcode, H, HP, in_dim, INP,
                       arity, Kf, static_cast<const uint16_t*>(W_in), static_cast<const uint16_t*>(W_rec),
                       static_cast<uint16_t*>(dst), count);
  else
    hipLaunchKernelGGL(k_pack<float>, dim3(blocks), dim3(256), 0, st, mode, G, GC, gcode, H, HP, in_dim, INP, arity,
                       Kf, static_cast<const float*>(W_in), static_cast<const float*>(W_rec),
                       static_cast<float*>(dst), count);
}

}  // namespace fold
