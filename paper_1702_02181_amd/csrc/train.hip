// The training step around the batched path (gfx950): the per-node softmax cross-entropy head and the
// Adam update.
//
// Section 3.5 trains the binary Tree-LSTM on trees in which every node carries a class label: a linear
// layer and a softmax on every node's state, the cross entropy against the node's label, the sum over the
// nodes as the loss (Section 3.3 attaches a sparse softmax cross entropy to the model's output), and
// TensorFlow's Adam optimizer (Section 3.3).
//
// k_loss_ce   one wave per 1-2 pool rows at a time (grid-stride; at most 768 blocks of 4 waves; the rows'
//             states all loaded before their first use, the next rows' positions and labels meanwhile): the C
//             logits z = h W + b as C dot products over each row's H values (W held in LDS), softmax and loss
//             in fp32 on every lane, dz = scale (p - onehot(y)), then dh = dz W^T written over the whole
//             padded row (zeros past H, and the whole row for an unlabelled node); h^T dz and sum dz are
//             summed over the wave's rows in registers (H <= 512, C <= 8; otherwise per row group into LDS),
//             then over the block's waves in LDS, and the block writes its sums to its row of the workspace.
//             HBM-bound: it reads each h row once (up to 512 columns kept in registers for the second pass)
//             and writes each dh row once.
// k_loss_reduce  dW, db += the blocks' partial sums in a fixed order (no atomics: every address would take
//             one from each block, one after another).  Inside a block the four waves' sums meet in LDS by
//             atomic adds in whatever order the waves arrive, so dW and db are reproducible up to the order
//             of those fp32 additions, not bit for bit.
// k_adam      elementwise, four values per thread: m, v and the fp32 parameters updated in place, plus an
//             optional bf16 copy of the parameters (the operand type of bf16 models).
// k_dropout_mask  the recurrent-dropout mask of a step (Section 3.5 trains with recurrent dropout), drawn
//             from the counter-based generator Philox4x32-10 (Salmon, Moraes, Dror and Shaw, SC 2011): one
//             generator call per (node, block of 4 hidden units), its four 32-bit words deciding the four
//             units; written in pool order as one 16-byte store per call.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "common.h"
#include "internal.h"

namespace fold {

namespace {

constexpr int kLossThreads = 256;  // 4 waves share one LDS copy of W and of the partial dW
constexpr int kLossBlocks = 768;   // three blocks of 4 waves per compute unit (the registers' occupancy): one round

template <typename T>
__device__ __forceinline__ float load_h(const T* p);
template <>
__device__ __forceinline__ float load_h<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float load_h<uint16_t>(const uint16_t* p) { return bf2f(*p); }

// Sum over the 64 lanes of a wave with DPP moves (no LDS traffic): pairs, quads, half rows and rows of 16
// lanes, then rows 0+1 and 2+3 by row broadcasts of lane 15 and lane 31; the total ends in lane 63 and is
// read back as a wave-uniform value.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_moved(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, ROW_MASK, 0xf,
                                                               false));
}
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_moved<0xb1, 0xf>(v);   // quad_perm [1, 0, 3, 2]
  v += dpp_moved<0x4e, 0xf>(v);   // quad_perm [2, 3, 0, 1]
  v += dpp_moved<0x141, 0xf>(v);  // row_half_mirror
  v += dpp_moved<0x140, 0xf>(v);  // row_mirror: every lane of a row holds the row's sum
  v += dpp_moved<0x142, 0xa>(v);  // row_bcast:15 into rows 1 and 3
  v += dpp_moved<0x143, 0xc>(v);  // row_bcast:31 into rows 2 and 3: lane 63 holds the total
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}

// Rows a wave takes at a time (their index, label and state loads all go out before the first use).
template <int C>
constexpr int loss_rows() { return C <= 8 ? 2 : 1; }

template <typename T, int C>
__global__ __launch_bounds__(kLossThreads) void k_loss_ce(int N, int H, int ld, const T* h_pool, const int* pos_node,
                                                          const int* labels, const float* W, const float* b,
                                                          float scale, float* node_loss, float* dh,
                                                          float* partial) {
  constexpr int R = loss_rows<C>(), U = 8;  // U: 64-column slices of a row loaded at once
  extern __shared__ float lds[];
  float* sW = lds;           // [H][C]
  float* sdW = lds + H * C;  // [H][C]
  __shared__ float sdb[C];
  const int tid = threadIdx.x, lane = tid & 63;
  for (int i = tid; i < H * C; i += kLossThreads) {
    sW[i] = W[i];
    sdW[i] = 0.f;
  }
  if (tid < C) sdb[tid] = 0.f;
  __syncthreads();
  float bias[C];
#pragma unroll
  for (int c = 0; c < C; ++c) bias[c] = b[c];
  const int step = gridDim.x * (kLossThreads / 64) * R;
  // dW and db of the wave's rows: in registers (columns lane + 64 u) when the row fits one set of slices and
  // C <= 8, else added per row group into the block's LDS sums
  constexpr bool kRegAcc = C <= 8;
  const bool reg = H <= 64 * U;
  float wacc[kRegAcc ? U : 1][kRegAcc ? C : 1], bacc[C];
#pragma unroll
  for (int u = 0; u < (kRegAcc ? U : 1); ++u)
#pragma unroll
    for (int c = 0; c < (kRegAcc ? C : 1); ++c) wacc[u][c] = 0.f;
#pragma unroll
  for (int c = 0; c < C; ++c) bacc[c] = 0.f;
  // Every load below is unconditional, from a clamped (valid) address, and masked afterwards: a load under
  // a branch would be waited for inside the branch, one after another.  The next rows' positions and
  // labels are loaded while the current rows are processed.
  auto fetch_labels = [&](int q0, int (&node)[R], int (&y)[R]) {
#pragma unroll
    for (int k = 0; k < R; ++k) node[k] = pos_node[min(q0 + k, N - 1)];
#pragma unroll
    for (int k = 0; k < R; ++k) {
      const int lab = labels[node[k]];
      y[k] = q0 + k < N && lab >= 0 && lab < C ? lab : -1;  // labels outside [0, C) count as unlabelled
      node[k] = q0 + k < N ? node[k] : -1;
    }
  };
  int p0 = (blockIdx.x * (kLossThreads / 64) + (tid >> 6)) * R;
  int nnode[R], ny[R];
  fetch_labels(min(p0, N - 1), nnode, ny);
  for (; p0 < N; p0 += step) {
    int node[R], y[R];
#pragma unroll
    for (int k = 0; k < R; ++k) {
      node[k] = nnode[k];
      y[k] = ny[k];
    }
    auto load_row = [&](int k, int j) {
      const float v = load_h<T>(h_pool + (size_t)min(p0 + k, N - 1) * ld + (j < H ? j : 0));
      return y[k] >= 0 && j < H ? v : 0.f;
    };
    // the first 64 U columns stay in registers for the second pass
    float h0[R][U];
#pragma unroll
    for (int k = 0; k < R; ++k)
#pragma unroll
      for (int u = 0; u < U; ++u) h0[k][u] = load_row(k, 64 * u + lane);
    if (p0 + step < N) fetch_labels(p0 + step, nnode, ny);
    // logits of the R rows (unlabelled rows read nothing and get zero logits)
    float z[R][C];
#pragma unroll
    for (int k = 0; k < R; ++k)
#pragma unroll
      for (int c = 0; c < C; ++c) z[k][c] = 0.f;
    for (int j0 = 0; j0 < H; j0 += 64 * U) {
      float hv[R][U];
#pragma unroll
      for (int k = 0; k < R; ++k)
#pragma unroll
        for (int u = 0; u < U; ++u) hv[k][u] = j0 == 0 ? h0[k][u] : load_row(k, j0 + 64 * u + lane);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int j = j0 + 64 * u + lane;
        if (j < H)
#pragma unroll
          for (int c = 0; c < C; ++c) {
            const float wv = sW[j * C + c];
#pragma unroll
            for (int k = 0; k < R; ++k) z[k][c] += hv[k][u] * wv;
          }
      }
    }
    // softmax without the cancellations of 1 - p_y and lse - z_y when the label's class dominates:
    // with m = max z (first at class a) and S = sum over c != a of e^(z_c - m), lse = m + log1p(S) and
    // loss = (m - z_y) + log1p(S); dz_c = scale p_c for c != y and dz_y = -scale (sum over c != y of p_c)
    float d[R][C];
#pragma unroll
    for (int k = 0; k < R; ++k) {
#pragma unroll
      for (int c = 0; c < C; ++c) {
        z[k][c] = wave_sum(z[k][c]) + bias[c];
      }
      int a = 0;
      float zmax = z[k][0];
#pragma unroll
      for (int c = 1; c < C; ++c)
        if (z[k][c] > zmax) {
          zmax = z[k][c];
          a = c;
        }
      float e[C], S = 0.f;
#pragma unroll
      for (int c = 0; c < C; ++c) {
        e[c] = expf(z[k][c] - zmax);
        S += c == a ? 0.f : e[c];
      }
      const float inv = 1.f / (1.f + S);
      float zy = 0.f, rest = 0.f;
#pragma unroll
      for (int c = 0; c < C; ++c) {
        zy = c == y[k] ? z[k][c] : zy;
        d[k][c] = y[k] >= 0 ? scale * (e[c] * inv) : 0.f;
        rest += c == y[k] ? 0.f : d[k][c];
      }
#pragma unroll
      for (int c = 0; c < C; ++c) d[k][c] = c == y[k] ? -rest : d[k][c];
      if (lane == 0 && node[k] >= 0) node_loss[node[k]] = y[k] >= 0 ? (zmax - zy) + log1pf(S) : 0.f;
    }
    // dh = dz W^T over the whole padded row; h^T dz and sum dz of the R rows into the block's LDS sums
    for (int j0 = 0; j0 < ld; j0 += 64 * U) {
      float hv[R][U];
#pragma unroll
      for (int k = 0; k < R; ++k)
#pragma unroll
        for (int u = 0; u < U; ++u) hv[k][u] = j0 == 0 ? h0[k][u] : load_row(k, j0 + 64 * u + lane);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int j = j0 + 64 * u + lane;
        if (j >= ld) continue;
        float g[R];
#pragma unroll
        for (int k = 0; k < R; ++k) g[k] = 0.f;
        if (j < H) {
#pragma unroll
          for (int c = 0; c < C; ++c) {
            const float wv = sW[j * C + c];
            float acc = 0.f;
#pragma unroll
            for (int k = 0; k < R; ++k) {
              g[k] += d[k][c] * wv;
              acc += hv[k][u] * d[k][c];
            }
            if constexpr (kRegAcc) {
              if (reg) wacc[u][c] += acc;
              else atomicAdd(&sdW[j * C + c], acc);
            } else {
              atomicAdd(&sdW[j * C + c], acc);
            }
          }
        }
#pragma unroll
        for (int k = 0; k < R; ++k)
          if (p0 + k < N) dh[(size_t)(p0 + k) * ld + j] = g[k];
      }
    }
#pragma unroll
    for (int c = 0; c < C; ++c)
#pragma unroll
      for (int k = 0; k < R; ++k) bacc[c] += d[k][c];
  }
  // the wave's sums into the block's: one LDS atomic per entry and wave
  if constexpr (kRegAcc) {
    if (reg)
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int j = 64 * u + lane;
        if (j < H)
#pragma unroll
          for (int c = 0; c < C; ++c) atomicAdd(&sdW[j * C + c], wacc[u][c]);
      }
  }
  if (lane < C) {
    float dl = 0.f;
#pragma unroll
    for (int c = 0; c < C; ++c) dl = c == lane ? bacc[c] : dl;
    atomicAdd(&sdb[lane], dl);
  }
  __syncthreads();
  // the block's partial sums: [H * C dW | C db] at block row blockIdx.x of the workspace
  float* part = partial + (size_t)blockIdx.x * (H * C + C);
  for (int i = tid; i < H * C; i += kLossThreads) part[i] = sdW[i];
  if (tid < C) part[H * C + tid] = sdb[tid];
}

// dW (entries 0 .. H C - 1) and db (the next C) += the blocks' partial sums.  A block of 1,024 threads
// takes 64 entries: its 16 thread groups sum every 16th partial row (eight loads in flight), then the 16
// group sums are added in group order, so the result does not depend on scheduling.
constexpr int kReduceGroups = 16;
__global__ __launch_bounds__(64 * kReduceGroups) void k_loss_reduce(const float* partial, int nblocks, int HC, int C,
                                                                    float* dW, float* db) {
  __shared__ float red[kReduceGroups][64];
  const int e = threadIdx.x & 63, grp = threadIdx.x >> 6;
  const int i = blockIdx.x * 64 + e;
  const int stride = HC + C;
  float s = 0.f;
  if (i < stride) {
    constexpr int U = 8;  // absent rows add an exact 0
    for (int b0 = grp; b0 < nblocks; b0 += kReduceGroups * U) {
      float t[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int b = b0 + kReduceGroups * u;
        t[u] = b < nblocks ? partial[(size_t)b * stride + i] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < U; ++u) s += t[u];
    }
  }
  red[grp][e] = s;
  __syncthreads();
  if (grp != 0 || i >= stride) return;
  float tot = 0.f;
#pragma unroll
  for (int g = 0; g < kReduceGroups; ++g) tot += red[g][e];
  if (i < HC) dW[i] += tot;
  else db[i - HC] += tot;
}

template <typename T>
void launch_loss_c(int C, dim3 grid, size_t lds, hipStream_t st, int N, int H, int ld, const T* h, const int* pos_node,
                   const int* labels, const float* W, const float* b, float scale, float* loss, float* dh,
                   float* partial) {
#define FOLD_LOSS_CASE(CC)                                                                                      \
  case CC:                                                                                                      \
    hipLaunchKernelGGL((k_loss_ce<T, CC>), grid, dim3(kLossThreads), lds, st, N, H, ld, h, pos_node, labels, W, b, \
                       scale, loss, dh, partial);                                                               \
    break;
  switch (C) {
    FOLD_LOSS_CASE(2)
    FOLD_LOSS_CASE(3)
    FOLD_LOSS_CASE(4)
    FOLD_LOSS_CASE(5)
    FOLD_LOSS_CASE(6)
    FOLD_LOSS_CASE(7)
    FOLD_LOSS_CASE(8)
    FOLD_LOSS_CASE(10)
    FOLD_LOSS_CASE(16)
    FOLD_LOSS_CASE(32)
    default: break;
  }
#undef FOLD_LOSS_CASE
}

__global__ void k_adam(size_t n, float* p, uint16_t* p_bf16, const float* g, float* m, float* v, float b1, float c1,
                       float b2, float c2, float lr_t, float eps) {
  const size_t stride = (size_t)gridDim.x * blockDim.x * 4;
  for (size_t i = ((size_t)blockIdx.x * blockDim.x + threadIdx.x) * 4; i < n; i += stride) {
    const int cnt = (int)std::min<size_t>(4, n - i);
    if (cnt == 4 && (((uintptr_t)(p + i) | (uintptr_t)(g + i) | (uintptr_t)(m + i) | (uintptr_t)(v + i)) & 15) == 0) {
      float4 pv = *reinterpret_cast<const float4*>(p + i), gv = *reinterpret_cast<const float4*>(g + i);
      float4 mv = *reinterpret_cast<const float4*>(m + i), vv = *reinterpret_cast<const float4*>(v + i);
      float* pa = &pv.x;
      float* ga = &gv.x;
      float* ma = &mv.x;
      float* va = &vv.x;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        ma[k] = b1 * ma[k] + c1 * ga[k];
        va[k] = b2 * va[k] + c2 * ga[k] * ga[k];
        pa[k] -= lr_t * ma[k] / (sqrtf(va[k]) + eps);
      }
      *reinterpret_cast<float4*>(p + i) = pv;
      *reinterpret_cast<float4*>(m + i) = mv;
      *reinterpret_cast<float4*>(v + i) = vv;
      if (p_bf16)
        for (int k = 0; k < 4; ++k) p_bf16[i + k] = f2bf(pa[k]);
    } else {
      for (int k = 0; k < cnt; ++k) {
        const float gk = g[i + k];
        const float mk = b1 * m[i + k] + c1 * gk;
        const float vk = b2 * v[i + k] + c2 * gk * gk;
        const float pk = p[i + k] - lr_t * mk / (sqrtf(vk) + eps);
        m[i + k] = mk;
        v[i + k] = vk;
        p[i + k] = pk;
        if (p_bf16) p_bf16[i + k] = f2bf(pk);
      }
    }
  }
}

// Philox4x32-10: ten rounds of (c0, c1, c2, c3) -> (hi(M1 c2) ^ c1 ^ k0, lo(M1 c2), hi(M0 c0) ^ c3 ^ k1,
// lo(M0 c0)), the key advancing by the Weyl constants between rounds.
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, unsigned k0, unsigned k1) {
  constexpr unsigned M0 = 0xD2511F53u, M1 = 0xCD9E8D57u, W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += W0;
      k1 += W1;
    }
    const unsigned hi0 = __umulhi(M0, c.x), lo0 = M0 * c.x;
    const unsigned hi1 = __umulhi(M1, c.z), lo1 = M1 * c.z;
    c = make_uint4(hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0);
  }
  return c;
}

// mask[q][4 b .. 4 b + 3] of pool row q (node v = pos_node[q]) from the call on counter (v, b, step_lo,
// step_hi) under the key (seed_lo, seed_hi): 0 where the word is below thresh, else scale; pad units
// (>= H) are 0.  One thread per (row, 4-unit block); blocks4 = ld / 4.
__global__ __launch_bounds__(256) void k_dropout_mask(const int* pos_node, long long total, int blocks4, int H,
                                                      unsigned thresh, float scale, unsigned k0, unsigned k1,
                                                      unsigned s0, unsigned s1, float* mask) {
  const long long t = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= total) return;
  const long long q = t / blocks4;
  const int b = (int)(t - q * blocks4);
  const unsigned v = (unsigned)pos_node[q];
  const uint4 r = philox4x32_10(make_uint4(v, (unsigned)b, s0, s1), k0, k1);
  const unsigned w[4] = {r.x, r.y, r.z, r.w};
  float out[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) out[i] = (4 * b + i < H && w[i] >= thresh) ? scale : 0.f;
  *reinterpret_cast<float4*>(mask + (size_t)t * 4) = make_float4(out[0], out[1], out[2], out[3]);
}

}  // namespace

void launch_dropout_mask(const int* pos_node, int N, int H, int ld, unsigned thresh, float scale,
                         unsigned long long seed, unsigned long long step, float* mask, hipStream_t st) {
  if (N <= 0) return;
  ProfScope prof("dropout_mask", st);
  const int blocks4 = ld / 4;
  const long long total = (long long)N * blocks4;
  const unsigned grid = (unsigned)((total + 255) / 256);
  hipLaunchKernelGGL(k_dropout_mask, dim3(grid), dim3(256), 0, st, pos_node, total, blocks4, H, thresh, scale,
                     (unsigned)(seed & 0xffffffffu), (unsigned)(seed >> 32), (unsigned)(step & 0xffffffffu),
                     (unsigned)(step >> 32), mask);
}

bool loss_classes_supported(int C) {
  return C == 2 || C == 3 || C == 4 || C == 5 || C == 6 || C == 7 || C == 8 || C == 10 || C == 16 || C == 32;
}

size_t loss_workspace_bytes(int H, int C) { return (size_t)kLossBlocks * (H * C + C) * sizeof(float); }

void launch_loss_ce(int dtype, int N, int H, int ld, int C, const void* h_pool, const int* pos_node, const int* labels,
                    const float* W, const float* b, float scale, float* node_loss, float* dh, float* dW, float* db,
                    float* ws, hipStream_t st) {
  if (N <= 0) return;
  ProfScope prof("loss_ce", st);
  const unsigned blocks = (unsigned)std::min<long long>(((long long)N + 4LL * 2 - 1) / (4LL * 2), kLossBlocks);
  const size_t lds = (size_t)2 * H * C * sizeof(float);
  if (dtype == FOLD_BF16)
    launch_loss_c<uint16_t>(C, dim3(blocks), lds, st, N, H, ld, static_cast<const uint16_t*>(h_pool), pos_node,
                            labels, W, b, scale, node_loss, dh, ws);
  else
    launch_loss_c<float>(C, dim3(blocks), lds, st, N, H, ld, static_cast<const float*>(h_pool), pos_node, labels, W,
                         b, scale, node_loss, dh, ws);
  const int total = H * C + C;
  hipLaunchKernelGGL(k_loss_reduce, dim3((total + 63) / 64), dim3(64 * kReduceGroups), 0, st, ws, (int)blocks, H * C,
                     C, dW, db);
}

void launch_adam(size_t n, float* p, uint16_t* p_bf16, const float* g, float* m, float* v, double b1, double b2,
                 double lr_t, double eps, hipStream_t st) {
  if (n == 0) return;
  ProfScope prof("adam", st);
  const unsigned blocks = (unsigned)std::min<size_t>((n + 1023) / 1024, 4096);
  hipLaunchKernelGGL(k_adam, dim3(blocks), dim3(256), 0, st, n, p, p_bf16, g, m, v, (float)b1, (float)(1.0 - b1),
                     (float)b2, (float)(1.0 - b2), (float)lr_t, (float)eps);
}

}  // namespace fold
