// Batched cells of one (depth, op) group, gfx950.
//
// Forward (Section 2: gather -> operation -> concat, one launch per group):
//   a workgroup owns BM pool rows of the group and one block of 32 hidden units.  It gathers the
//   rows' inputs -- leaf-table rows by input_idx and the children's h rows by child_pos -- into LDS,
//   contracts them with the packed weights on the matrix cores (all G gate blocks of its 32 units,
//   so every lane ends up holding i, f, o, u, ... of the same (row, unit)), applies the cell in
//   registers and writes h, c (and the activations the backward needs) straight into the pools.
// Backward:
//   k_cell_bwd  elementwise dz of every row from the saved activations; dc of the children
//               scatter-added; EMBED rows scatter dh into the leaf-table gradient
//   k_bwd_dx    dz . W^T on the matrix cores, scatter-added into the children's dh; for the leaf-table
//               gradient, after k_tok_sum has summed dz over the rows of every (op, leaf-table row), once per
//               distinct leaf-table row
// Cells (gate blocks in column order):
//   TREELSTM (i|f_l|f_r|o|u): c = i*u + f_l*c_l + f_r*c_r, h = o*tanh(c)   (Tai et al. N-ary, N = 2)
//   LSTM     (i|f|o|u):       c = i*u + f*c_p,             h = o*tanh(c)
//   TREERNN / PROJ:           h = tanh(z); PROJ passes the child's c through
//   Tree-LSTM leaf (i|o|u):   c = i*u, h = o*tanh(c)  (the forget gates of a leaf multiply the zero
//                             state: they are neither computed nor saved nor differentiated)

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

inline unsigned cdiv(long long a, long long b) { return (unsigned)((a + b - 1) / b); }

// Old values of the read-add-write targets among the 16 rows of one 32 x 32 result block that a lane holds
// (column jin of pool rows t[r] where one[r]; 0 elsewhere).  Such targets have a single parent edge, so they
// are distinct rows: all 16 loads are issued before any store, instead of each waiting behind the previous
// row's store.
__device__ __forceinline__ void read_targets16(const float* dh, int ld, int jin, const int (&t)[16],
                                               const bool (&one)[16], float (&old)[16]) {
#pragma unroll
  for (int r = 0; r < 16; ++r) old[r] = one[r] ? dh[(size_t)t[r] * ld + jin] : 0.f;
}

template <int KIND>
struct Gates {
  static constexpr int G = KIND == FOLD_TREELSTM ? 5 : (KIND == FOLD_LSTM ? 4 : (KIND == kTreeLstmLeaf ? 3 : 1));
};

// ---------------------------------------------------------------- forward

// Direct loads of one forward stage (128 bytes of K) for one wave: the gathered A rows of its share of
// the row tile (leaf-table rows by input_idx for the input segment, the children's h rows by child_pos
// after it; absent rows read the zero row) and its share of the weight slice's rows.
template <typename T, int BM, int PA, int PB>
struct FwdIssue {
  const FwdArgs& a;
  const int (*srow)[BM];
  int wskip;  // weight columns before the first segment read: the set's input block when this op
              // reads no input
  int c0, inp, wave, lr;
  int cur_seg = -1;
  const char* wp[PB];  // this lane's weight row per instruction (first stage), unit included
  const char* rp[PA];  // this lane's A row per instruction in the current segment, unit included
  __device__ __forceinline__ void reload(int seg) {
    constexpr int es = sizeof(T);
    const bool is_in = a.has_input && seg == 0;
    const char* base = static_cast<const char*>(is_in ? a.table : a.h_pool);
    const size_t stride = (size_t)(is_in ? a.tld : a.ld) * es;
#pragma unroll
    for (int i = 0; i < PA; ++i) {
      const int sr = srow[seg][8 * (wave * PA + i) + lr];
      const int lu16 = unit_of_lane(threadIdx.x & 63, wave * PA + i) * 16;
      rp[i] = (sr >= 0 ? base + (size_t)sr * stride : static_cast<const char*>(a.zero)) + lu16;
    }
    cur_seg = seg;
  }
  __device__ __forceinline__ void operator()(int c, char* Ad, char* Bd) {
    constexpr int es = sizeof(T), BK = 128 / es;
    const int kabs = (c0 + c) * BK;
    int seg, kc;
    if (kabs < inp) {
      seg = 0;
      kc = kabs;
    } else {
      const int k = (kabs - inp) / a.HP;
      seg = a.has_input + k;
      kc = kabs - inp - k * a.HP;
    }
    if (seg != cur_seg) reload(seg);
#pragma unroll
    for (int i = 0; i < PA; ++i) dma16(rp[i] + kc * es, Ad + (wave * PA + i) * 1024);
#pragma unroll
    for (int i = 0; i < PB; ++i) dma16(wp[i] + (kabs + wskip) * es, Bd + (wave * PB + i) * 1024);
  }
};

// children whose cell state a cell reads
template <int KIND>
struct CKids {
  static constexpr int N = KIND == FOLD_TREELSTM ? 2 : ((KIND == FOLD_LSTM || KIND == FOLD_PROJ) ? 1 : 0);
};

// Saved activation g of hidden unit j in a row's part of the workspace: fp32 with fp32 parameters; fp16 with
// bf16 parameters (the backward then overwrites each with its bf16 dz in place).  fp16 keeps 11 significant
// bits where bf16 keeps 8: the backward multiplies dc by the forget gates level after level, and over
// 512-level chains bf16 gates would add ~1e-2 to dc's relative error, fp16 gates ~1e-3.
template <typename T>
struct SavedGates {
  float* f;
  uint16_t* h;
  __device__ __forceinline__ SavedGates(float* row, int j) {
    f = row ? row + j : nullptr;
    h = row ? reinterpret_cast<uint16_t*>(row) + j : nullptr;
  }
  __device__ __forceinline__ explicit operator bool() const { return f != nullptr; }
  __device__ __forceinline__ void put(int off, float v) const {
    if constexpr (sizeof(T) == 4)
      f[off] = v;
    else
      h[off] = __builtin_bit_cast(uint16_t, (_Float16)v);
  }
};

// The cell on one (row, unit) given z (bias included) and the children's c (0 for the zero state):
// writes h, c and the saved activations.
template <typename T, int KIND>
__device__ __forceinline__ void cell_out(const FwdArgs& a, int row, int j, const float* z, float cl, float cr) {
  const size_t p = (size_t)(a.row_begin + row);
  float h, c;
  const SavedGates<T> gs(a.gates ? a.gates + p * a.gstride : nullptr, j);
  if constexpr (KIND == FOLD_TREELSTM) {
    const float i_ = sigmoidf_(z[0]), fl = sigmoidf_(z[1]), fr = sigmoidf_(z[2]), o = sigmoidf_(z[3]);
    const float u = tanhf_(z[4]);
    const float um = a.u_mask ? u * a.u_mask[p * a.ld + j] : u;
    c = i_ * um + fl * cl + fr * cr;
    h = o * tanhf_(c);
    if (gs) {
      gs.put(0, i_);
      gs.put(a.HP, fl);
      gs.put(2 * a.HP, fr);
      gs.put(3 * a.HP, o);
      gs.put(4 * a.HP, u);
    }
  } else if constexpr (KIND == kTreeLstmLeaf) {
    const float i_ = sigmoidf_(z[0]), o = sigmoidf_(z[1]), u = tanhf_(z[2]);
    (void)cl;
    (void)cr;
    c = i_ * (a.u_mask ? u * a.u_mask[p * a.ld + j] : u);
    h = o * tanhf_(c);
    if (gs) {
      gs.put(0, i_);
      gs.put(a.HP, o);
      gs.put(2 * a.HP, u);
    }
  } else if constexpr (KIND == FOLD_LSTM) {
    const float i_ = sigmoidf_(z[0]), f = sigmoidf_(z[1]), o = sigmoidf_(z[2]);
    const float u = tanhf_(z[3]);
    const float um = a.u_mask ? u * a.u_mask[p * a.ld + j] : u;
    c = i_ * um + f * cl;
    h = o * tanhf_(c);
    if (gs) {
      gs.put(0, i_);
      gs.put(a.HP, f);
      gs.put(2 * a.HP, o);
      gs.put(3 * a.HP, u);
    }
  } else {
    h = tanhf_(z[0]);
    c = 0.f;
    if constexpr (KIND == FOLD_PROJ) c = cl;
    (void)cr;
    if (gs) gs.put(0, h);
  }
  static_cast<T*>(a.h_pool)[p * a.ld + j] = from_f32<T>(h);
  a.c_pool[p * a.ld + j] = c;
}

// pad columns of the pools (H <= j < ld) are written as zero
template <typename T>
__device__ __forceinline__ void pad_out(const FwdArgs& a, int row, int j) {
  const size_t p = (size_t)(a.row_begin + row);
  static_cast<T*>(a.h_pool)[p * a.ld + j] = from_f32<T>(0.f);
  a.c_pool[p * a.ld + j] = 0.f;
}

// SPLIT: the K loop is cut into gridDim.z slices; each workgroup writes its partial z (no bias) to
// a.zpart[slice][row][g * HP + j] and k_cell_epi finishes the cell.  Used for narrow levels, whose
// few row tiles would otherwise leave most compute units idle for a whole K loop.
// The body of the narrow forward for workgroup L of its grid.  LDS comes in as separate arrays (two stages of A,
// BM rows, and of B, G gate blocks of 32 units, 128 bytes of K each; the source row of every tile row per input
// segment, -1: zero row): as distinct objects the compiler sees that the loads in flight into one stage buffer
// do not touch the other, and adds no wait between them.
template <typename T, int KIND, int MT, bool SPLIT>
__device__ __forceinline__ void cell_fwd_body(const FwdArgs a, unsigned L, char* A0, char* A1, char* B0, char* B1,
                                              int (*srow)[4 * 32 * MT]) {
  constexpr int G = Gates<KIND>::G;
  constexpr int BM = 4 * 32 * MT;  // four waves stacked along the rows
  constexpr int BN = G * 32;       // G gate blocks of 32 units
  constexpr int PA = BM / 32, PB = BN / 32;  // direct-load instructions per wave and stage
  constexpr int BK = 128 / sizeof(T);

  const int tid = threadIdx.x, lane = tid & 63, wave = wave_id();
  // co-locate on one XCD the workgroups that share the larger operand: the gathered rows of a row tile
  // or the weight slice of a unit block
  const int R = (a.rows + BM - 1) / BM, UB = a.HP / 32;
  int tx, ty, ub, rt, kz;
  if (a.map == kMapRows) {
    if (!xcd_tile_at(L, UB * a.ksplit, R, tx, ty)) return;
    rt = ty;
    ub = tx % UB;
    kz = tx / UB;
  } else {
    if (!xcd_tile_at(L, R * a.ksplit, UB, tx, ty)) return;
    ub = ty;
    rt = tx % R;
    kz = tx / R;
  }
  const int m0 = rt * BM;  // ub: hidden units ub*32 .. ub*32+31

  const int nseg = a.has_input + a.arity;
  for (int seg = 0; seg < nseg; ++seg) {
    const bool is_in = a.has_input && seg == 0;
    const int k = seg - a.has_input;
    for (int r = tid; r < BM; r += kThreads) {
      const int row = m0 + r;
      int sr = -1;
      if (row < a.rows) sr = is_in ? a.input_idx[a.row_begin + row] : fwd_child(a, row, k);
      srow[seg][r] = sr;
    }
  }
  __syncthreads();

  const int inp = a.has_input ? a.INP : 0;
  const int nst = (inp + a.arity * a.HP) / BK;
  int c0 = 0, c1 = nst;
  if constexpr (SPLIT) {
    const int per = (nst + a.ksplit - 1) / a.ksplit;
    c0 = min(nst, kz * per);
    c1 = min(nst, c0 + per);
  }
  const int lr = row_of_lane(lane);
  FwdIssue<T, BM, PA, PB> issue{a, srow, a.has_input ? 0 : a.INP, c0, inp, wave, lr};
#pragma unroll
  for (int i = 0; i < PB; ++i)
    issue.wp[i] = static_cast<const char*>(a.Wf) + ((size_t)ub * BN + 8 * (wave * PB + i) + lr) * a.Kf * sizeof(T) +
                  unit_of_lane(lane, wave * PB + i) * 16;
  f32x16 acc[MT][G];
  zero_acc(acc);
  row_loop<T, MT, G>(c1 - c0, issue, A0, A1, B0, B1, acc, wave * 32 * MT, 0, lane);

  const int j = ub * 32 + (lane & 31);
  if constexpr (SPLIT) {
    const int zs = G * a.HP;
    float* zp = a.zpart + (size_t)kz * a.rows * zs + j;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wave * 32 * MT + mt * 32 + acc_row(r, lane);
        if (row >= a.rows) continue;
#pragma unroll
        for (int g = 0; g < G; ++g) zp[(size_t)row * zs + g * a.HP] = acc[mt][g][r];
      }
    return;
  }
  // epilogue: the cell, in registers.  The children's c of every row this lane finishes is loaded
  // first, all at once (pool rows from the LDS row table; absent children and rows past the end read
  // the zero row), so the loads overlap instead of each waiting its turn.
  constexpr int NK = CKids<KIND>::N;
  float bz[G];
#pragma unroll
  for (int g = 0; g < G; ++g) bz[g] = a.bias[g * a.HP + j];
  float cc[MT][16][NK > 0 ? NK : 1];
  if constexpr (NK > 0) {
    const float* zf = static_cast<const float*>(a.zero) + j;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rl = wave * 32 * MT + mt * 32 + acc_row(r, lane);
#pragma unroll
        for (int k = 0; k < NK; ++k) {
          const int p = k < a.arity ? srow[a.has_input + k][rl] : -1;
          cc[mt][r][k] = *(p >= 0 ? a.c_pool + (size_t)p * a.ld + j : zf);
        }
      }
  }
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int rl = wave * 32 * MT + mt * 32 + acc_row(r, lane), row = m0 + rl;
      if (row >= a.rows) continue;
      if (j >= a.H) {
        if (j < a.ld) pad_out<T>(a, row, j);
        continue;
      }
      float z[G];
#pragma unroll
      for (int g = 0; g < G; ++g) z[g] = acc[mt][g][r] + bz[g];
      const float cl = NK > 0 ? cc[mt][r][0] : 0.f, cr = NK > 1 ? cc[mt][r][NK > 1 ? 1 : 0] : 0.f;
      cell_out<T, KIND>(a, row, j, z, cl, cr);
    }
  }
}

template <typename T, int KIND, int MT, bool SPLIT>
__global__ __launch_bounds__(kThreads) void k_cell_fwd(FwdArgs a) {
  constexpr int BM = 4 * 32 * MT, BN = Gates<KIND>::G * 32;
  __shared__ __attribute__((aligned(16))) char A0[BM * 128], A1[BM * 128], B0[BN * 128], B1[BN * 128];
  __shared__ int srow[3][BM];
  cell_fwd_body<T, KIND, MT, SPLIT>(a, blockIdx.x, A0, A1, B0, B1, srow);
}

// ---------------------------------------------------------------- forward, wide levels
// 256 rows x 2 unit blocks (all G gate blocks of 64 hidden units) per workgroup of 8 waves, each wave
// 64 rows x the G gate blocks of one unit block; 64-byte K stages, three in flight (see wide.h).  Waves
// 0-3 issue the loads of a stage: 4 instructions of gathered A rows (64 tile rows) and G of weight rows
// (16 G of the 64 G rows in the tile) each.

template <typename T, int G>
struct WideFwdIssue {
  const FwdArgs& a;
  const int (*srow)[wide::kRows];
  int wskip, inp, wave, cur_seg = -1;
  const char* wp[G];  // this lane's weight row per instruction, unit included (K offset 0)
  const char* rp[4];  // this lane's A row per instruction in the current segment, unit included
  __device__ __forceinline__ void reload(int seg) {
    constexpr int es = sizeof(T);
    const bool is_in = a.has_input && seg == 0;
    const char* base = static_cast<const char*>(is_in ? a.table : a.h_pool);
    const size_t stride = (size_t)(is_in ? a.tld : a.ld) * es;
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int sr = srow[seg][64 * wave + 16 * i + wide::lane_row(lane)];
      rp[i] = (sr >= 0 ? base + (size_t)sr * stride : static_cast<const char*>(a.zero)) + wide::lane_unit(lane) * 16;
    }
    cur_seg = seg;
  }
  __device__ __forceinline__ void operator()(int c, char* slot) {
    constexpr int es = sizeof(T), BK = 64 / es, BOFF = wide::kRows * 64;
    const int kabs = c * BK;
    int seg, kc;
    if (kabs < inp) {
      seg = 0;
      kc = kabs;
    } else {
      const int k = (kabs - inp) / a.HP;
      seg = a.has_input + k;
      kc = kabs - inp - k * a.HP;
    }
    if (seg != cur_seg) reload(seg);
#pragma unroll
    for (int i = 0; i < 4; ++i) dma16_untracked(rp[i] + kc * es, slot + (4 * wave + i) * 1024);
#pragma unroll
    for (int i = 0; i < G; ++i) dma16_untracked(wp[i] + (kabs + wskip) * es, slot + BOFF + (G * wave + i) * 1024);
  }
};

// workgroup -> (row tile, column group) for the wide kernels: kMapOwnCols (column groups a multiple of
// 8: each XCD keeps its own groups) or kMapRows (the column groups of a row tile on one XCD)
__device__ __forceinline__ bool wide_tile(int map, int R, int NC, int& rt, int& nc) {
  if (map == kMapOwnCols) {
    xcd_cols(NC, nc, rt);
    return rt < R;
  }
  return xcd_tile(NC, R, nc, rt);
}

template <typename T, int KIND>
__global__ __launch_bounds__(wide::kThreads) void k_cell_fwd_w(FwdArgs a) {
  constexpr int G = Gates<KIND>::G;
  constexpr int BM = wide::kRows, BN = 2 * G * 32;
  constexpr int BOFF = BM * 64, SLOT = (BM + BN) * 64;
  constexpr int MT = 2;  // 32-row blocks per wave
  __shared__ __attribute__((aligned(16))) char ring[wide::kSlots * SLOT];
  __shared__ int srow[3][BM];  // source row of every tile row, per input segment (-1: zero row)

  const int tid = threadIdx.x, lane = tid & 63, wave = wave_id();
  const int wr = wave & 3, wc = wave >> 2;
  const int R = (a.rows + BM - 1) / BM, NU = a.HP / 64;  // row tiles, unit-block pairs
  int rt, up;
  if (!wide_tile(a.map, R, NU, rt, up)) return;
  const int m0 = rt * BM;
  const int nseg = a.has_input + a.arity;
  for (int i = tid; i < nseg * BM; i += wide::kThreads) {
    const int seg = i / BM, r = i - seg * BM, row = m0 + r;
    const bool is_in = a.has_input && seg == 0;
    int sr = -1;
    if (row < a.rows)
      sr = is_in ? a.input_idx[a.row_begin + row] : fwd_child(a, row, seg - a.has_input);
    srow[seg][r] = sr;
  }
  __syncthreads();

  constexpr int BK = 64 / sizeof(T);
  const int inp = a.has_input ? a.INP : 0;
  const int nst = (inp + a.arity * a.HP) / BK;
  const bool loads = wave < 4;
  WideFwdIssue<T, G> issue{a, srow, a.has_input ? 0 : a.INP, inp, wr};
#pragma unroll
  for (int i = 0; i < G; ++i)
    issue.wp[i] = static_cast<const char*>(a.Wf) +
                  ((size_t)up * BN + 16 * (G * wr + i) + wide::lane_row(lane)) * a.Kf * sizeof(T) +
                  wide::lane_unit(lane) * 16;
  f32x16 acc[MT][G];
  zero_acc(acc);
  struct Gate {
    WideFwdIssue<T, G>& is;
    bool on;
    __device__ __forceinline__ void operator()(int c, char* slot) {
      if (on) is(c, slot);
    }
  } gate{issue, loads};
  wide::loop<T, MT, G, 4 + G, SLOT, BOFF>(nst, gate, loads, ring, acc, wr * 64, wc * G * 32, lane);

  const int j = (2 * up + wc) * 32 + (lane & 31);
  // epilogue: the cell in registers, one 32-row block at a time (children's c loaded for the block first)
  constexpr int NK = CKids<KIND>::N;
  float bz[G];
#pragma unroll
  for (int g = 0; g < G; ++g) bz[g] = a.bias[g * a.HP + j];
  const float* zf = static_cast<const float*>(a.zero) + j;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    float cc[16][NK > 0 ? NK : 1];
    if constexpr (NK > 0) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rl = wr * 64 + mt * 32 + acc_row(r, lane);
#pragma unroll
        for (int k = 0; k < NK; ++k) {
          const int p = k < a.arity ? srow[a.has_input + k][rl] : -1;
          cc[r][k] = *(p >= 0 ? a.c_pool + (size_t)p * a.ld + j : zf);
        }
      }
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int rl = wr * 64 + mt * 32 + acc_row(r, lane), row = m0 + rl;
      if (row >= a.rows) continue;
      if (j >= a.H) {
        if (j < a.ld) pad_out<T>(a, row, j);
        continue;
      }
      float z[G];
#pragma unroll
      for (int g = 0; g < G; ++g) z[g] = acc[mt][g][r] + bz[g];
      const float cl = NK > 0 ? cc[r][0] : 0.f, cr = NK > 1 ? cc[r][NK > 1 ? 1 : 0] : 0.f;
      cell_out<T, KIND>(a, row, j, z, cl, cr);
    }
  }
}

// finish a K-split level: sum the slices' partial z, add the bias, apply the cell
template <typename T, int KIND>
__device__ __forceinline__ void cell_epi_body(const FwdArgs a, int row, int nsplit) {
  constexpr int G = Gates<KIND>::G;
  const int zs = G * a.HP;
  const int p0 = a.arity >= 1 ? fwd_child(a, row, 0) : -1;
  const int p1 = a.arity >= 2 ? fwd_child(a, row, 1) : -1;
  const float* zf = static_cast<const float*>(a.zero);
  const float* c0r = p0 >= 0 ? a.c_pool + (size_t)p0 * a.ld : zf;
  const float* c1r = p1 >= 0 ? a.c_pool + (size_t)p1 * a.ld : zf;
  for (int j = threadIdx.x; j < a.HP; j += blockDim.x) {
    if (j >= a.H) {
      if (j < a.ld) pad_out<T>(a, row, j);
      continue;
    }
    // the slices are added in slice order; their loads go out eight slices (of every gate) at a time
    // rather than one after another (absent slices add an exact 0)
    constexpr int U = 8;
    float z[G];
#pragma unroll
    for (int g = 0; g < G; ++g) z[g] = a.bias[g * a.HP + j];
    const float* zp = a.zpart + (size_t)row * zs + j;
    const size_t slice = (size_t)a.rows * zs;
    for (int s0 = 0; s0 < nsplit; s0 += U) {
      float t[G][U];
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int g = 0; g < G; ++g) t[g][u] = s0 + u < nsplit ? zp[(size_t)(s0 + u) * slice + g * a.HP] : 0.f;
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int g = 0; g < G; ++g) z[g] += t[g][u];
    }
    cell_out<T, KIND>(a, row, j, z, c0r[j], c1r[j]);
  }
}

template <typename T, int KIND>
__global__ void k_cell_epi(FwdArgs a, int nsplit) {
  cell_epi_body<T, KIND>(a, blockIdx.x, nsplit);
}

template <typename T>
__global__ __launch_bounds__(256) void k_embed_fwd(int rows, int row_begin, int H, int ld, int tld, const T* table,
                                                   const int* input_idx, T* h_pool, float* c_pool) {
  // one wave per row, four rows a workgroup; a lane copies four consecutive elements (rows are whole 64-element
  // segments, 16-byte aligned)
  const int lane = threadIdx.x & 63, row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const size_t p = (size_t)(row_begin + row);
  const T* src = table + (size_t)input_idx[p] * tld;
  for (int j = 4 * lane; j < ld; j += 256) {
    if constexpr (sizeof(T) == 4) {
      float4 v = *reinterpret_cast<const float4*>(src + j);
      if (j + 4 > H) {
        v.x = j < H ? v.x : 0.f, v.y = j + 1 < H ? v.y : 0.f, v.z = j + 2 < H ? v.z : 0.f, v.w = 0.f;
      }
      *reinterpret_cast<float4*>(h_pool + p * ld + j) = v;
    } else {
      uint2 v = *reinterpret_cast<const uint2*>(src + j);
      if (j + 4 > H) {
        const uint32_t m0 = j < H ? (j + 1 < H ? 0xffffffffu : 0xffffu) : 0u;
        const uint32_t m1 = j + 2 < H ? (j + 3 < H ? 0xffffffffu : 0xffffu) : 0u;
        v.x &= m0, v.y &= m1;
      }
      *reinterpret_cast<uint2*>(h_pool + p * ld + j) = v;
    }
    *reinterpret_cast<float4*>(c_pool + p * ld + j) = make_float4(0.f, 0.f, 0.f, 0.f);
  }
}

// plain fill kernel (used where a memset node would be recorded into a graph)
__global__ void k_zero_f32(float* p, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0.f;
}

template <typename T>
__global__ void k_roots(int ld, const int* root_pos, const T* h_pool, T* out) {
  const int r = blockIdx.x;
  const size_t p = (size_t)root_pos[r];
  for (int j = threadIdx.x; j < ld; j += blockDim.x) out[(size_t)r * ld + j] = h_pool[p * ld + j];
}

// ---------------------------------------------------------------- backward, elementwise

// Rows of nodes with exactly one parent edge are stored whole by that parent's backward; every other row (roots,
// children of several parents) starts at zero.  A wave reads the parent counts of 64 consecutive rows at once and
// zeroes, all lanes together, only the rows that need it (a tree batch: its roots alone).
__global__ __launch_bounds__(256) void k_bwd_init(int N, int ld, const int* npar, float* dh, float* dc) {
  const int lane = threadIdx.x & (kWave - 1);
  const int p0 = (blockIdx.x * 4 + (threadIdx.x >> 6)) * kWave;
  if (p0 >= N) return;
  unsigned long long m = __ballot(p0 + lane < N && npar[p0 + lane] != 1);  // the same in every lane
  const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
  while (m) {
    const int l = __ffsll((unsigned long long)m) - 1;
    m &= m - 1;
    const size_t o = (size_t)(p0 + l) * ld;
    for (int j = 4 * lane; j < ld; j += 4 * kWave) {
      *reinterpret_cast<float4*>(dh + o + j) = z;
      *reinterpret_cast<float4*>(dc + o + j) = z;
    }
  }
}

// With per-node upstream gradients every dh row starts as that gradient; dc rows as above.
__global__ void k_bwd_init_nodes(int N, int ld, const float* dh_nodes, const int* npar, float* dh, float* dc) {
  for (int p = blockIdx.x; p < N; p += gridDim.x) {
    const bool init = npar[p] != 1;
    const size_t o = (size_t)p * ld;
    for (int j = 4 * threadIdx.x; j < ld; j += 4 * blockDim.x) {
      *reinterpret_cast<float4*>(dh + o + j) = *reinterpret_cast<const float4*>(dh_nodes + o + j);
      if (init) *reinterpret_cast<float4*>(dc + o + j) = make_float4(0.f, 0.f, 0.f, 0.f);
    }
  }
}

// roots are distinct rows, so adding their upstream gradient needs no atomics
__global__ void k_bwd_roots(int ld, const float* dh_roots, const int* root_pos, float* dh) {
  const int r = blockIdx.x;
  const size_t p = (size_t)root_pos[r];
  for (int j = threadIdx.x; j < ld; j += blockDim.x) dh[p * ld + j] += dh_roots[(size_t)r * ld + j];
}

// dz of one row from its saved activations, written over them in place (each thread rewrites only the
// elements it read): fp32 dz over fp32 activations (fp32 parameters), or bf16 dz over fp16 activations
// (bf16 parameters: the G*HP halves at the row's start, the matrix-core operand of dz . W^T and of the
// weight gradients).  A thread takes two adjacent columns (j even; rows are whole 64-column segments), so every
// access is a 4-byte (fp16 / bf16 pair) or 8-byte (fp32 pair) one; columns past H give zeros.
template <int KIND, bool BF>
__device__ __forceinline__ void cell_bwd_body(const BwdCellArgs a, int row) {
  static_assert(KIND != FOLD_EMBED, "an embedding has no cell backward (its leaf-table gradient runs per op)");
  constexpr int G = Gates<KIND>::G;
  constexpr int NK = KIND == FOLD_TREELSTM || KIND == FOLD_TREERNN ? 2
                     : (KIND == FOLD_LSTM || KIND == FOLD_PROJ ? 1 : 0);  // child slots
  const size_t p = (size_t)(a.row_begin + row);
  float* gb = a.gates + p * a.gstride;
  uint16_t* gh = reinterpret_cast<uint16_t*>(gb);
  int ck[2] = {-1, -1};
  bool sk[2] = {false, false};
#pragma unroll
  for (int k = 0; k < NK; ++k)
    if (k < a.arity) {
      ck[k] = a.child_pos[a.idx_off + row * a.arity + k];
      sk[k] = a.child_one[a.idx_off + row * a.arity + k] != 0;
    }
  auto ld2 = [](const float* q, float (&v)[2]) {
    const float2 t = *reinterpret_cast<const float2*>(q);
    v[0] = t.x, v[1] = t.y;
  };
  const float* own = a.c_pool + p * a.ld;
  for (int j = 2 * threadIdx.x; j < a.HP; j += 2 * blockDim.x) {
    const bool live[2] = {j < a.H, j + 1 < a.H};
    float g[G][2];
#pragma unroll
    for (int q = 0; q < G; ++q) {
      if constexpr (BF) {
        const uint32_t t = *reinterpret_cast<const uint32_t*>(gh + q * a.HP + j);
        g[q][0] = (float)__builtin_bit_cast(_Float16, (uint16_t)(t & 0xffff));
        g[q][1] = (float)__builtin_bit_cast(_Float16, (uint16_t)(t >> 16));
      } else {
        ld2(gb + q * a.HP + j, g[q]);
      }
    }
    float dh[2], dz[G][2], dck[2][2] = {{0.f, 0.f}, {0.f, 0.f}};  // dc passed to child slot k
    ld2(a.dh + p * a.ld + j, dh);
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      if constexpr (KIND == FOLD_TREELSTM || KIND == kTreeLstmLeaf || KIND == FOLD_LSTM) {
        const float dc = a.dc[p * a.ld + j + e];
        const float m = a.u_mask ? a.u_mask[p * a.ld + j + e] : 1.f;
        const float tc = tanhf_(own[j + e]);
        // gate order: Tree-LSTM i f_l f_r o u; leaf i o u; LSTM i f o u
        constexpr int GO = KIND == FOLD_TREELSTM ? 3 : (KIND == kTreeLstmLeaf ? 1 : 2);
        const float i_ = g[0][e], o = g[GO][e], u = g[G - 1][e];
        const float dct = dc + dh[e] * o * (1.f - tc * tc);
        dz[0][e] = dct * (m * u) * i_ * (1.f - i_);
        dz[GO][e] = dh[e] * tc * o * (1.f - o);
        dz[G - 1][e] = dct * i_ * m * (1.f - u * u);
#pragma unroll
        for (int k = 0; k < NK; ++k) {  // the forget gates: f_l, f_r (Tree-LSTM) or f (LSTM), gates 1 .. NK
          const float f = g[1 + k][e];
          const float cc = ck[k] >= 0 ? a.c_pool[(size_t)ck[k] * a.ld + j + e] : 0.f;
          dz[1 + k][e] = dct * cc * f * (1.f - f);
          dck[k][e] = dct * f;
        }
      } else {  // TreeRNN, PROJ: h = tanh(z)
        const float h = g[0][e];
        dz[0][e] = dh[e] * (1.f - h * h);
        if constexpr (KIND == FOLD_PROJ) dck[0][e] = a.dc[p * a.ld + j + e];  // c = c_child
      }
      if (!live[e]) {  // pad columns: zero dz and zero gradients for the children
#pragma unroll
        for (int q = 0; q < G; ++q) dz[q][e] = 0.f;
        dck[0][e] = dck[1][e] = 0.f;
      }
    }
#pragma unroll
    for (int q = 0; q < G; ++q) {
      if constexpr (BF)
        *reinterpret_cast<uint32_t*>(gh + q * a.HP + j) = (uint32_t)f2bf(dz[q][0]) | ((uint32_t)f2bf(dz[q][1]) << 16);
      else
        *reinterpret_cast<float2*>(gb + q * a.HP + j) = make_float2(dz[q][0], dz[q][1]);
    }
    // a child's gradients: its dc stored whole by its only parent (a TreeRNN passes zeros), added atomically into
    // a zeroed row otherwise; with K-split dz . W^T slices its dh row is zeroed here first
#pragma unroll
    for (int k = 0; k < NK; ++k) {
      if (ck[k] < 0) continue;
      float* dcr = a.dc + (size_t)ck[k] * a.ld + j;
      if (sk[k]) {
        *reinterpret_cast<float2*>(dcr) = make_float2(dck[k][0], dck[k][1]);
        if (a.zero_child_dh) *reinterpret_cast<float2*>(a.dh + (size_t)ck[k] * a.ld + j) = make_float2(0.f, 0.f);
      } else if (KIND != FOLD_TREERNN) {
#pragma unroll
        for (int e = 0; e < 2; ++e)
          if (live[e]) unsafeAtomicAdd(dcr + e, dck[k][e]);
      }
    }
  }
}

template <int KIND, bool BF>
__global__ void k_cell_bwd(BwdCellArgs a) {
  cell_bwd_body<KIND, BF>(a, blockIdx.x);
}

// ---------------------------------------------------------------- backward, dz . W^T


// dz . W^T for one tile of 128 * MT rows x 128 columns of the children's (or the input's) gradient:
// dz rows (fp32, or bf16 at the start of each row for bf16 parameters) and the packed W^T rows are
// loaded straight into LDS.
// The body of the narrow dz . W^T for workgroup L of its grid; LDS as separate arrays (see cell_fwd_body):
// tgt = per tile row child k's pool row (mode 0) or the leaf-table row (mode 1), sgl = the child has one parent
// edge (its row stored whole when it starts undefined, else read-add-written; not atomic)
template <typename T, int MT, bool SPLIT>
__device__ __forceinline__ void bwd_dx2_body(const DxArgs a, unsigned L, char* A0, char* A1, char* B0, char* B1,
                                             int (*tgt)[4 * 32 * MT], char (*sgl)[4 * 32 * MT]) {
  constexpr int TN = 4;
  constexpr int BM = 4 * 32 * MT, BN = 32 * TN;  // four waves of 32*MT rows x 128 columns
  constexpr int PA = BM / 32, PB = BN / 32;
  const int lane = threadIdx.x & 63, wave = wave_id();
  // co-locate the workgroups that share the larger operand (a row tile's dz rows or a column tile's
  // weight slice) on one XCD
  const int R = (a.rows + BM - 1) / BM, NT = (a.Nb + BN - 1) / BN;
  int tx, ty, nt, rt, kz;
  if (a.map == kMapRows) {
    if (!xcd_tile_at(L, NT * a.ksplit, R, tx, ty)) return;
    rt = ty;
    nt = tx % NT;
    kz = tx / NT;
  } else {
    if (!xcd_tile_at(L, R * a.ksplit, NT, tx, ty)) return;
    nt = ty;
    rt = tx % R;
    kz = tx / R;
  }
  const int m0 = rt * BM, n0 = nt * BN;
  {
    // scatter targets of the tile's rows, published by the K loop's first barrier
    for (int i = threadIdx.x; i < 2 * BM; i += kThreads) {
      const int k = i / BM, rl = i - k * BM, row = m0 + rl;
      int t = -1;
      char one = 0;
      if (row < a.rows) {
        if (a.mode == 0) {
          if (k < a.arity) {
            t = a.child_pos[a.idx_off + row * a.arity + k];
            one = a.child_one[a.idx_off + row * a.arity + k] != 0;
          }
        } else if (k == 0) {
          t = a.input_idx[a.row_begin + row];
        }
      }
      tgt[k][rl] = t;
      sgl[k][rl] = one;
    }
  }
  const int nst = a.Kb * (int)sizeof(T) / 128, per = (nst + a.ksplit - 1) / a.ksplit;
  const int c0 = min(nst, kz * per), c1 = min(nst, c0 + per);
  // an empty trailing K slice adds nothing (and its epilogue would read the target table unpublished)
  if (c1 <= c0) return;
  const int lr = row_of_lane(lane);
  const char* zero = static_cast<const char*>(a.zero);
  FixedRowsIssue<PA, PB> issue;
  issue.wave = wave;
#pragma unroll
  for (int i = 0; i < PA; ++i) {
    const int row = m0 + 8 * (wave * PA + i) + lr;
    const int lu16 = unit_of_lane(lane, wave * PA + i) * 16;
    issue.ap[i] = (row < a.rows ? reinterpret_cast<const char*>(a.dz + (size_t)(a.row_begin + row) * a.gstride) +
                                      c0 * 128
                                : zero) + lu16;
  }
  const char* wb = static_cast<const char*>(a.Wb);
#pragma unroll
  for (int i = 0; i < PB; ++i) {
    const int n = n0 + 8 * (wave * PB + i) + lr;
    const int lu16 = unit_of_lane(lane, wave * PB + i) * 16;
    issue.bp[i] = (n < a.Nb ? wb + (size_t)n * a.Kb * sizeof(T) + c0 * 128 : zero) + lu16;
  }
  f32x16 acc[MT][TN];
  zero_acc(acc);
  row_loop<T, MT, TN>(c1 - c0, issue, A0, A1, B0, B1, acc, wave * 32 * MT, 0, lane);
#pragma unroll
  for (int tm = 0; tm < MT; ++tm) {
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const int n = n0 + tn * 32 + (lane & 31);
      if (n >= a.Nb) continue;
      const int k = a.mode == 0 ? n / a.HP : 0, jin = a.mode == 0 ? n - k * a.HP : n;
      // pad columns (their products are 0) are stored only into rows that start undefined
      const bool pad = jin >= (a.mode == 0 ? a.H : a.in_dim);
      if (pad && !(a.mode == 0 && a.dh_fresh && !SPLIT)) continue;
      // K slices of one element add into it concurrently: atomics whenever K is split
      int tr[16];
      bool one[16], rd[16];
      float old[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rl = wave * 32 * MT + tm * 32 + acc_row(r, lane), row = m0 + rl;
        tr[r] = row < a.rows ? tgt[k][rl] : -1;
        one[r] = !SPLIT && a.mode == 0 && tr[r] >= 0 && sgl[k][rl];
        rd[r] = one[r] && !a.dh_fresh;
      }
      read_targets16(a.dh, a.ld, jin, tr, rd, old);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int t = tr[r];
        if (t < 0 || (pad && !one[r])) continue;
        if (a.mode == 0) {
          float* dst = &a.dh[(size_t)t * a.ld + jin];
          if (one[r]) *dst = old[r] + acc[tm][tn][r];  // old = 0 for a row that starts undefined
          else unsafeAtomicAdd(dst, acc[tm][tn][r]);
        } else {
          unsafeAtomicAdd(&a.d_table[(size_t)t * a.tld + jin], acc[tm][tn][r]);
        }
      }
    }
  }
}

template <typename T, int MT, bool SPLIT>
__global__ __launch_bounds__(kThreads) void k_bwd_dx2(DxArgs a) {
  constexpr int BM = 4 * 32 * MT, BN = 128;
  __shared__ __attribute__((aligned(16))) char A0[BM * 128], A1[BM * 128], B0[BN * 128], B1[BN * 128];
  __shared__ int tgt[2][BM];
  __shared__ char sgl[2][BM];
  bwd_dx2_body<T, MT, SPLIT>(a, blockIdx.x, A0, A1, B0, B1, tgt, sgl);
}

// dz . W^T on wide levels: 256 rows x 256 columns per workgroup of 8 waves (each 64 x 128), 64-byte K
// stages, three in flight (see wide.h).  Waves 0-3 issue the loads: 4 instructions of dz rows and 4 of
// W^T rows each.  With gridDim.y = ksplit > 1 workgroup (x, y) takes the y-th slice of the K stages and
// adds its partial product into the targets atomically (mid-size levels, too few tiles to fill the GPU).
template <typename T>
__global__ __launch_bounds__(wide::kThreads) void k_bwd_dx_w(DxArgs a) {
  constexpr int BM = wide::kRows, BN = 256, TM = 2, TN = 4, NL = 8;
  constexpr int BOFF = BM * 64, SLOT = (BM + BN) * 64;
  __shared__ __attribute__((aligned(16))) char ring[wide::kSlots * SLOT];
  __shared__ int tgt[2][BM];   // per tile row: child k's pool row (mode 0) or the leaf-table row (mode 1)
  __shared__ char sgl[2][BM];  // the child has one parent edge: stored (or read-add-written), not atomic
  const int tid = threadIdx.x, lane = tid & 63, wave = wave_id();
  const int wr = wave & 3, wc = wave >> 2;
  const int R = (a.rows + BM - 1) / BM, NT = (a.Nb + BN - 1) / BN;
  int nt, rt;
  if (!wide_tile(a.map, R, NT, rt, nt)) return;
  const int m0 = rt * BM, n0 = nt * BN;
  for (int i = tid; i < 2 * BM; i += wide::kThreads) {
    const int k = i / BM, rl = i - k * BM, row = m0 + rl;
    int t = -1;
    char one = 0;
    if (row < a.rows) {
      if (a.mode == 0) {
        if (k < a.arity) {
          t = a.child_pos[a.idx_off + row * a.arity + k];
          one = a.child_one[a.idx_off + row * a.arity + k] != 0;
        }
      } else if (k == 0) {
        t = a.input_idx[a.row_begin + row];
      }
    }
    tgt[k][rl] = t;
    sgl[k][rl] = one;
  }
  // published by the K loop's first barrier

  const int nst_all = a.Kb * (int)sizeof(T) / 64, per = (nst_all + a.ksplit - 1) / a.ksplit;
  const int c0 = min(nst_all, (int)blockIdx.y * per), nst = min(nst_all, c0 + per) - c0;
  if (nst <= 0) return;  // an empty K slice adds nothing (its epilogue would read the tables unpublished)
  const bool split = a.ksplit > 1;
  const bool loads = wave < 4;
  const char* zero = static_cast<const char*>(a.zero);
  const char* wb = static_cast<const char*>(a.Wb);
  struct Issue {
    const char* ap[4];
    const char* bp[4];
    bool on;
    __device__ __forceinline__ void operator()(int c, char* slot) const {
      if (!on) return;
      const int w = wave_id(), off = c * 64;
#pragma unroll
      for (int i = 0; i < 4; ++i) dma16_untracked(ap[i] + off, slot + (4 * w + i) * 1024);
#pragma unroll
      for (int i = 0; i < 4; ++i) dma16_untracked(bp[i] + off, slot + BOFF + (4 * w + i) * 1024);
    }
  } issue;
  issue.on = loads;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int lu16 = wide::lane_unit(lane) * 16;
    const int row = m0 + 64 * wr + 16 * i + wide::lane_row(lane);
    issue.ap[i] = (row < a.rows ? reinterpret_cast<const char*>(a.dz + (size_t)(a.row_begin + row) * a.gstride) +
                                      c0 * 64
                                : zero) + lu16;
    const int n = n0 + 64 * wr + 16 * i + wide::lane_row(lane);
    issue.bp[i] = (n < a.Nb ? wb + (size_t)n * a.Kb * sizeof(T) + c0 * 64 : zero) + lu16;
  }
  f32x16 acc[TM][TN];
  zero_acc(acc);
  wide::loop<T, TM, TN, NL, SLOT, BOFF>(nst, issue, loads, ring, acc, wr * 64, wc * 128, lane);
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) {
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const int n = n0 + wc * 128 + tn * 32 + (lane & 31);
      if (n >= a.Nb) continue;
      const int k = a.mode == 0 ? n / a.HP : 0, jin = a.mode == 0 ? n - k * a.HP : n;
      // pad columns (their products are 0) are stored only into rows that start undefined
      const bool pad = jin >= (a.mode == 0 ? a.H : a.in_dim);
      if (pad && !(a.mode == 0 && a.dh_fresh && !split)) continue;
      int tr[16];
      bool one[16], rd[16];
      float old[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rl = wr * 64 + tm * 32 + acc_row(r, lane), row = m0 + rl;
        tr[r] = row < a.rows ? tgt[k][rl] : -1;
        one[r] = !split && a.mode == 0 && tr[r] >= 0 && sgl[k][rl];
        rd[r] = one[r] && !a.dh_fresh;
      }
      read_targets16(a.dh, a.ld, jin, tr, rd, old);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int t = tr[r];
        if (t < 0 || (pad && !one[r])) continue;
        if (a.mode == 0) {
          float* dst = &a.dh[(size_t)t * a.ld + jin];
          if (one[r]) *dst = old[r] + acc[tm][tn][r];  // old = 0 for a row that starts undefined
          else unsafeAtomicAdd(dst, acc[tm][tn][r]);
        } else {
          unsafeAtomicAdd(&a.d_table[(size_t)t * a.tld + jin], acc[tm][tn][r]);
        }
      }
    }
  }
}


// ---------------------------------------------------------------- several groups of one level, one launch
// The groups of one depth are independent (each reads only rows of lower depths), so the narrow groups of a
// level can run as one launch: its grid is the groups' grids back to back (each a multiple of 8 workgroups,
// which keeps every group's XCD order) and each workgroup runs the body of its group's kernel variant.  On
// levels of several operations this replaces one dependent launch per group by one per level.

template <typename FA>
struct Merged {
  int n;
  int begin[kMaxMerge + 1];  // first workgroup (or row) of each part; begin[n] = total
  int variant[kMaxMerge];
  FA a[kMaxMerge];
};

__device__ __forceinline__ int merged_part(const int* begin, int n, int bid) {
  int i = 0;
  while (i + 1 < n && bid >= begin[i + 1]) ++i;
  return i;
}

// variant = 2 * kind + (K split); the LDS arrays are sized for the widest tile (5 gate blocks)
template <typename T>
__global__ __launch_bounds__(kThreads) void k_level_fwd(Merged<FwdArgs> m) {
  constexpr int BM = 128, BN = 5 * 32;
  __shared__ __attribute__((aligned(16))) char A0[BM * 128], A1[BM * 128], B0[BN * 128], B1[BN * 128];
  __shared__ int srow[3][BM];
  const int i = merged_part(m.begin, m.n, blockIdx.x);
  const unsigned bid = blockIdx.x - (unsigned)m.begin[i];
  const FwdArgs a = m.a[i];  // by value: the bodies then read it as values, not through a pointer
  switch (m.variant[i]) {
#define FOLD_V(K)                                                                      \
  case 2 * K: cell_fwd_body<T, K, 1, false>(a, bid, A0, A1, B0, B1, srow); break;     \
  case 2 * K + 1: cell_fwd_body<T, K, 1, true>(a, bid, A0, A1, B0, B1, srow); break;
    FOLD_V(FOLD_TREERNN)
    FOLD_V(FOLD_TREELSTM)
    FOLD_V(FOLD_LSTM)
    FOLD_V(FOLD_PROJ)
    FOLD_V(kTreeLstmLeaf)
#undef FOLD_V
    default: break;
  }
}

// K-split epilogues of a level: one workgroup per row, parts in rows; variant = kind
template <typename T>
__global__ void k_level_epi(Merged<FwdArgs> m) {
  const int i = merged_part(m.begin, m.n, blockIdx.x);
  const int row = blockIdx.x - m.begin[i];
  const FwdArgs a = m.a[i];
  switch (m.variant[i]) {
    case FOLD_TREERNN: cell_epi_body<T, FOLD_TREERNN>(a, row, a.ksplit); break;
    case FOLD_TREELSTM: cell_epi_body<T, FOLD_TREELSTM>(a, row, a.ksplit); break;
    case FOLD_LSTM: cell_epi_body<T, FOLD_LSTM>(a, row, a.ksplit); break;
    case FOLD_PROJ: cell_epi_body<T, FOLD_PROJ>(a, row, a.ksplit); break;
    case kTreeLstmLeaf: cell_epi_body<T, kTreeLstmLeaf>(a, row, a.ksplit); break;
    default: break;
  }
}

// cell backward of a level: one workgroup per row; variant = kind (the embedding writes no dz)
template <bool BF>
__global__ void k_level_cbwd(Merged<BwdCellArgs> m) {
  const int i = merged_part(m.begin, m.n, blockIdx.x);
  const int row = blockIdx.x - m.begin[i];
  const BwdCellArgs a = m.a[i];
  switch (m.variant[i]) {
    case FOLD_TREERNN: cell_bwd_body<FOLD_TREERNN, BF>(a, row); break;
    case FOLD_TREELSTM: cell_bwd_body<FOLD_TREELSTM, BF>(a, row); break;
    case FOLD_LSTM: cell_bwd_body<FOLD_LSTM, BF>(a, row); break;
    case FOLD_PROJ: cell_bwd_body<FOLD_PROJ, BF>(a, row); break;
    case kTreeLstmLeaf: cell_bwd_body<kTreeLstmLeaf, BF>(a, row); break;
    default: break;
  }
}

// dz . W^T of a level; variant = 2 * mt + (K split), mt <= MTMAX (the LDS is sized for MTMAX)
template <typename T, int MTMAX>
__global__ __launch_bounds__(kThreads) void k_level_dx(Merged<DxArgs> m) {
  constexpr int BM = 4 * 32 * MTMAX, BN = 128;
  __shared__ __attribute__((aligned(16))) char A0[BM * 128], A1[BM * 128], B0[BN * 128], B1[BN * 128];
  __shared__ int tgt[2][BM];
  __shared__ char sgl[2][BM];
  const int i = merged_part(m.begin, m.n, blockIdx.x);
  const unsigned bid = blockIdx.x - (unsigned)m.begin[i];
  const DxArgs a = m.a[i];
  // a part with mt = 1 uses the first 128 rows of every row array (same strides for A and B)
  switch (m.variant[i]) {
    case 2:
      bwd_dx2_body<T, 1, false>(a, bid, A0, A1, B0, B1, reinterpret_cast<int(*)[128]>(&tgt[0][0]),
                                reinterpret_cast<char(*)[128]>(&sgl[0][0]));
      break;
    case 3:
      bwd_dx2_body<T, 1, true>(a, bid, A0, A1, B0, B1, reinterpret_cast<int(*)[128]>(&tgt[0][0]),
                               reinterpret_cast<char(*)[128]>(&sgl[0][0]));
      break;
    case 4:
      if constexpr (MTMAX >= 2)
        bwd_dx2_body<T, 2, false>(a, bid, A0, A1, B0, B1, reinterpret_cast<int(*)[4 * 32 * 2]>(&tgt[0][0]),
                                  reinterpret_cast<char(*)[4 * 32 * 2]>(&sgl[0][0]));
      break;
    case 5:
      if constexpr (MTMAX >= 2)
        bwd_dx2_body<T, 2, true>(a, bid, A0, A1, B0, B1, reinterpret_cast<int(*)[4 * 32 * 2]>(&tgt[0][0]),
                                 reinterpret_cast<char(*)[4 * 32 * 2]>(&sgl[0][0]));
      break;
    default: break;
  }
}

template <typename T, int KIND>
void cell_fwd_kind(const FwdArgs& a0, hipStream_t st) {
  const FwdPlan pl = fwd_plan(a0.rows, a0.HP, a0.has_input ? a0.INP : 0, a0.arity, sizeof(T), a0.zpart != nullptr,
                              true);
  FwdArgs a = a0;
  if (pl.wide) {
    const int R = (int)cdiv(a.rows, wide::kRows), NU = a.HP / 64;
    a.ksplit = 1;
    a.map = NU % 8 == 0 ? kMapOwnCols : kMapRows;
    dim3 grid(a.map == kMapOwnCols ? xcd_cols_grid(NU, R) : xcd_grid(NU, R));
    hipLaunchKernelGGL((k_cell_fwd_w<T, KIND>), grid, dim3(wide::kThreads), 0, st, a);
    return;
  }
  a.ksplit = pl.ksplit;
  const int G = Gates<KIND>::G;
  if (a.ksplit > 1 && a.zcap > 0) {  // partial sums capped: as many slices as fit (none if fewer than two)
    const size_t fit = a.zcap / ((size_t)a.rows * G * a.HP);
    a.ksplit = (int)std::min<size_t>((size_t)a.ksplit, fit);
    if (a.ksplit < 2) a.ksplit = 1;
  }
  const int R = (int)cdiv(a.rows, 128), UB = a.HP / 32;  // 128-row tiles of one unit block
  a.map = a.rows >= G * a.HP ? kMapRows : kMapCols;  // gathered rows outweigh the weights: share row tiles
  dim3 grid(a.map == kMapRows ? xcd_grid(UB * a.ksplit, R) : xcd_grid(R * a.ksplit, UB));
  if (a.ksplit > 1) {
    hipLaunchKernelGGL((k_cell_fwd<T, KIND, 1, true>), grid, dim3(kThreads), 0, st, a);
    hipLaunchKernelGGL((k_cell_epi<T, KIND>), dim3(a.rows), dim3(std::min(a.HP, 1024)), 0, st, a, a.ksplit);
  } else {
    hipLaunchKernelGGL((k_cell_fwd<T, KIND, 1, false>), grid, dim3(kThreads), 0, st, a);
  }
}

template <typename T>
void cell_fwd_t(int kind, const FwdArgs& a, hipStream_t st) {
  switch (kind) {
    case FOLD_TREELSTM: cell_fwd_kind<T, FOLD_TREELSTM>(a, st); break;
    case kTreeLstmLeaf: cell_fwd_kind<T, kTreeLstmLeaf>(a, st); break;
    case FOLD_LSTM: cell_fwd_kind<T, FOLD_LSTM>(a, st); break;
    case FOLD_TREERNN: cell_fwd_kind<T, FOLD_TREERNN>(a, st); break;
    case FOLD_PROJ: cell_fwd_kind<T, FOLD_PROJ>(a, st); break;
    default: break;
  }
}

// ---------------------------------------------------------------- leaf-table gradient
// The leaf-table gradient of an op is sum over its rows of dz . W_in^T, added into each row's leaf-table row.
// It is linear in dz, so dz is first summed over the rows of every run of equal (op, leaf-table row), and the
// contraction then runs once per distinct leaf-table row (no two of its rows share a target).

constexpr int kTokRows = 256;  // at most this many entries of the (op, leaf-table row) list per workgroup

// A workgroup per `per` (at most kTokRows) consecutive entries of the op's list, a thread per four consecutive
// columns.  TABLE = false: dz (fp32, or bf16 at the start of each row) summed into zsum[run - u0][Kb]; a run that
// lies inside the workgroup's entries is stored, the first and the last run, which may cross its ends, are added
// atomically into the zeroed sums.  TABLE = true (an embedding op): its fp32 dh rows summed and added straight
// into the leaf-table gradient's row of the run (columns < ncols, row stride tld): read-add-written inside the
// workgroup's entries (each row once per op), atomically for the crossing runs.  Eight rows' loads go out before
// they are added.
template <bool BF, bool TABLE>
__global__ __launch_bounds__(256) void k_tok_sum(const int* tok_rows, const int* tok_seg, const int* tok_start,
                                                 const int* tok_row, int i0, int count, int per, int u0,
                                                 const float* dz, int gstride, int Kb, int ncols, int tld,
                                                 float* out) {
  __shared__ int srow[kTokRows], sseg[kTokRows], strow[kTokRows];
  const int b0 = i0 + blockIdx.x * per, b1 = min(i0 + count, b0 + per), n = b1 - b0;
  for (int t = threadIdx.x; t < n; t += blockDim.x) {
    srow[t] = tok_rows[b0 + t];
    sseg[t] = tok_seg[b0 + t];
  }
  __syncthreads();
  const int ufirst = sseg[0], ulast = sseg[n - 1];
  if constexpr (TABLE) {  // leaf-table rows of the workgroup's runs (at most one per entry)
    for (int t = threadIdx.x; t <= ulast - ufirst; t += blockDim.x) strow[t] = tok_row[ufirst + t];
    __syncthreads();
  }
  const bool first_out = tok_start[ufirst] < b0, last_out = tok_start[ulast + 1] > b1;
  auto load = [&](int t, int j, float (&v)[4]) {
    const float* row = dz + (size_t)srow[t] * gstride;
    if constexpr (BF) {
      const uint2 x = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint16_t*>(row) + j);
      v[0] = bf2f(x.x & 0xffff), v[1] = bf2f(x.x >> 16), v[2] = bf2f(x.y & 0xffff), v[3] = bf2f(x.y >> 16);
    } else {
      const float4 x = *reinterpret_cast<const float4*>(row + j);
      v[0] = x.x, v[1] = x.y, v[2] = x.z, v[3] = x.w;
    }
  };
  auto flush = [&](int u, int j, const float (&acc)[4]) {
    const bool crossing = (u == ufirst && first_out) || (u == ulast && last_out);
    if constexpr (TABLE) {
      float* dst = out + (size_t)strow[u - ufirst] * tld + j;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (j + e >= ncols) break;
        if (crossing)
          atomicAdd(dst + e, acc[e]);
        else
          dst[e] += acc[e];
      }
    } else {
      float* dst = out + (size_t)(u - u0) * Kb + j;
      if (crossing) {
#pragma unroll
        for (int e = 0; e < 4; ++e) atomicAdd(dst + e, acc[e]);
      } else {
        *reinterpret_cast<float4*>(dst) = make_float4(acc[0], acc[1], acc[2], acc[3]);
      }
    }
  };
  const int cols = TABLE ? ncols : Kb;
  for (int j = 4 * threadIdx.x; j < cols; j += 4 * blockDim.x) {
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    int u = ufirst;
    auto add = [&](int t, const float (&v)[4]) {
      if (sseg[t] != u) {
        flush(u, j, acc);
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[e] = 0.f;
        u = sseg[t];
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[e] += v[e];
    };
    int t = 0;
    for (; t + 8 <= n; t += 8) {
      float v[8][4];
#pragma unroll
      for (int e = 0; e < 8; ++e) load(t + e, j, v[e]);
#pragma unroll
      for (int e = 0; e < 8; ++e) add(t + e, v[e]);
    }
    for (; t < n; ++t) {
      float v[4];
      load(t, j, v);
      add(t, v);
    }
    flush(u, j, acc);
  }
}

__global__ void k_tok_cast(const float* in, size_t n, uint16_t* out) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    out[i] = f2bf(in[i]);
}

}  // namespace

const char* kind_name(int kind, int dtype) {
  static const char* n32[] = {"cell_fwd.embed.f32", "cell_fwd.treernn.f32", "cell_fwd.treelstm.f32",
                              "cell_fwd.lstm.f32", "cell_fwd.proj.f32"};
  static const char* n16[] = {"cell_fwd.embed.bf16", "cell_fwd.treernn.bf16", "cell_fwd.treelstm.bf16",
                              "cell_fwd.lstm.bf16", "cell_fwd.proj.bf16"};
  if (kind == kTreeLstmLeaf) kind = FOLD_TREELSTM;  // one class per operation family
  if (kind < 0 || kind > 4) return "cell_fwd";
  return dtype == FOLD_BF16 ? n16[kind] : n32[kind];
}

void launch_cell_fwd(int dtype, int kind, const FwdArgs& a, hipStream_t st) {
  if (a.rows <= 0) return;
  ProfScope prof(kind_name(kind, dtype), st);
  if (dtype == FOLD_BF16)
    cell_fwd_t<uint16_t>(kind, a, st);
  else
    cell_fwd_t<float>(kind, a, st);
}

void launch_embed_fwd(int dtype, int rows, int row_begin, int H, int ld, int tld, const void* table,
                      const int* input_idx, void* h_pool, float* c_pool, hipStream_t st) {
  if (rows <= 0) return;
  ProfScope prof("embed_fwd", st);
  if (dtype == FOLD_BF16)
    hipLaunchKernelGGL(k_embed_fwd<uint16_t>, dim3(cdiv(rows, 4)), dim3(256), 0, st, rows, row_begin, H, ld, tld,
                       static_cast<const uint16_t*>(table), input_idx, static_cast<uint16_t*>(h_pool), c_pool);
  else
    hipLaunchKernelGGL(k_embed_fwd<float>, dim3(cdiv(rows, 4)), dim3(256), 0, st, rows, row_begin, H, ld, tld,
                       static_cast<const float*>(table), input_idx, static_cast<float*>(h_pool), c_pool);
}

void launch_zero_f32(float* p, size_t n, hipStream_t st) {
  if (!p || n == 0) return;
  ProfScope prof("zero_grads", st);
  const unsigned blocks = (unsigned)std::min<size_t>((n + 255) / 256, 8192);
  hipLaunchKernelGGL(k_zero_f32, dim3(blocks), dim3(256), 0, st, p, n);
}

void launch_roots(int dtype, int R, int ld, const int* root_pos, const void* h_pool, void* out, hipStream_t st) {
  if (R <= 0) return;
  ProfScope prof("roots", st);
  if (dtype == FOLD_BF16)
    hipLaunchKernelGGL(k_roots<uint16_t>, dim3(R), dim3(256), 0, st, ld, root_pos,
                       static_cast<const uint16_t*>(h_pool), static_cast<uint16_t*>(out));
  else
    hipLaunchKernelGGL(k_roots<float>, dim3(R), dim3(256), 0, st, ld, root_pos, static_cast<const float*>(h_pool),
                       static_cast<float*>(out));
}

void launch_bwd_init(int N, int R, int ld, const float* dh_nodes, const float* dh_roots, const int* root_pos,
                     const int* pos_npar, float* dh, float* dc, hipStream_t st) {
  if (N <= 0) return;
  ProfScope prof("bwd_init", st);
  if (dh_nodes)
    hipLaunchKernelGGL(k_bwd_init_nodes, dim3((unsigned)std::min(N, 65536)), dim3(256), 0, st, N, ld, dh_nodes,
                       pos_npar, dh, dc);
  else
    hipLaunchKernelGGL(k_bwd_init, dim3(cdiv(N, 256)), dim3(256), 0, st, N, ld, pos_npar, dh, dc);
  if (dh_roots && R > 0) hipLaunchKernelGGL(k_bwd_roots, dim3(R), dim3(256), 0, st, ld, dh_roots, root_pos, dh);
}

void launch_cell_bwd(int kind, const BwdCellArgs& a, hipStream_t st) {
  if (a.rows <= 0) return;
  static const char* names[] = {"cell_bwd.embed", "cell_bwd.treernn", "cell_bwd.treelstm", "cell_bwd.lstm",
                                "cell_bwd.proj"};
  const int nk = kind == kTreeLstmLeaf ? FOLD_TREELSTM : kind;  // one class per operation family
  ProfScope prof(nk >= 0 && nk <= FOLD_PROJ ? names[nk] : "cell_bwd", st);
  // one thread per two hidden units (up to 1024 threads): every load of a row is in flight at once
  dim3 grid(a.rows), block(std::min(std::max(a.HP / 2, kWave), 1024));
#define FOLD_CB(K_)                                                                          \
  if (a.dz_bf16) hipLaunchKernelGGL((k_cell_bwd<K_, true>), grid, block, 0, st, a);          \
  else hipLaunchKernelGGL((k_cell_bwd<K_, false>), grid, block, 0, st, a);
  switch (kind) {
    case FOLD_TREERNN: FOLD_CB(FOLD_TREERNN) break;
    case FOLD_TREELSTM: FOLD_CB(FOLD_TREELSTM) break;
    case kTreeLstmLeaf: FOLD_CB(kTreeLstmLeaf) break;
    case FOLD_LSTM: FOLD_CB(FOLD_LSTM) break;
    case FOLD_PROJ: FOLD_CB(FOLD_PROJ) break;
    default: break;
  }
#undef FOLD_CB
}

// entries of the (op, leaf-table row) list per summing workgroup: enough workgroups to fill the GPU a few times
// over (short runs that cross a workgroup's ends cost atomic adds, so no fewer than 32 entries)
static int tok_per(int count) { return std::max(32, std::min(kTokRows, count / 1024 / 8 * 8)); }

void launch_tok_sum(int dtype, const int* tok_rows, const int* tok_seg, const int* tok_start, int i0, int count,
                    int u0, int U, const float* dz, int gstride, int Kb, float* zsum, uint16_t* zbf, hipStream_t st) {
  if (count <= 0 || U <= 0) return;
  ProfScope prof("tgrad_sum", st);
  const size_t n = (size_t)U * Kb;
  hipLaunchKernelGGL(k_zero_f32, dim3((unsigned)std::min<size_t>((n + 255) / 256, 8192)), dim3(256), 0, st, zsum, n);
  const int per = tok_per(count);
  const dim3 grid(cdiv(count, per));
  if (dtype == FOLD_BF16) {
    hipLaunchKernelGGL((k_tok_sum<true, false>), grid, dim3(256), 0, st, tok_rows, tok_seg, tok_start, nullptr, i0,
                       count, per, u0, dz, gstride, Kb, 0, 0, zsum);
    hipLaunchKernelGGL(k_tok_cast, dim3((unsigned)std::min<size_t>((n + 255) / 256, 8192)), dim3(256), 0, st, zsum,
                       n, zbf);
  } else {
    hipLaunchKernelGGL((k_tok_sum<false, false>), grid, dim3(256), 0, st, tok_rows, tok_seg, tok_start, nullptr, i0,
                       count, per, u0, dz, gstride, Kb, 0, 0, zsum);
  }
}

void launch_tok_table(const int* tok_rows, const int* tok_seg, const int* tok_start, const int* tok_row, int i0,
                      int count, const float* dh, int ld, int H, float* d_table, int tld, hipStream_t st) {
  if (count <= 0) return;
  ProfScope prof("tgrad_embed", st);
  const int per = tok_per(count);
  hipLaunchKernelGGL((k_tok_sum<false, true>), dim3(cdiv(count, per)), dim3(256), 0, st, tok_rows, tok_seg, tok_start,
                     tok_row, i0, count, per, 0, dh, ld, 0, H, tld, d_table);
}

void launch_bwd_dx(int dtype, const DxArgs& a0, hipStream_t st, const char* name) {
  if (a0.rows <= 0 || a0.Nb <= 0) return;
  DxArgs a = a0;
  ProfScope prof(name ? name : dtype == FOLD_BF16 ? "bwd_dx.bf16" : "bwd_dx.f32", st);
  const DxPlan pl = dx_plan(a.rows, a.Nb, a.Kb, dtype == FOLD_BF16 ? 2 : 4, a.can_split != 0);
  if (pl.wide) {
    const int R = (int)cdiv(a.rows, wide::kRows), NT = (int)cdiv(a.Nb, 256);
    a.ksplit = pl.ksplit;
    a.map = NT % 8 == 0 ? kMapOwnCols : kMapRows;
    // K slices along y: gridDim.x is a multiple of 8, so every slice of a tile runs on the tile's XCD
    dim3 grid(a.map == kMapOwnCols ? xcd_cols_grid(NT, R) : xcd_grid(NT, R), pl.ksplit);
    if (dtype == FOLD_BF16)
      hipLaunchKernelGGL(k_bwd_dx_w<uint16_t>, grid, dim3(wide::kThreads), 0, st, a);
    else
      hipLaunchKernelGGL(k_bwd_dx_w<float>, grid, dim3(wide::kThreads), 0, st, a);
    return;
  }
  const int MT = pl.mt;
  a.ksplit = pl.ksplit;
  const int R = (int)cdiv(a.rows, 128 * MT), NT = (int)cdiv(a.Nb, 128);
  a.map = a.rows >= a.Nb ? kMapRows : kMapCols;
  dim3 grid(a.map == kMapRows ? xcd_grid(NT * pl.ksplit, R) : xcd_grid(R * pl.ksplit, NT));
#define FOLD_DX(T_, MT_, S_) hipLaunchKernelGGL((k_bwd_dx2<T_, MT_, S_>), grid, dim3(kThreads), 0, st, a)
  const bool split = pl.ksplit > 1;
  if (dtype == FOLD_BF16) {
    if (MT == 2) { if (split) FOLD_DX(uint16_t, 2, true); else FOLD_DX(uint16_t, 2, false); }
    else { if (split) FOLD_DX(uint16_t, 1, true); else FOLD_DX(uint16_t, 1, false); }
  } else {
    if (MT == 2) { if (split) FOLD_DX(float, 2, true); else FOLD_DX(float, 2, false); }
    else { if (split) FOLD_DX(float, 1, true); else FOLD_DX(float, 1, false); }
  }
#undef FOLD_DX
}

// ---------------------------------------------------------------- level launches (host)

constexpr long long kLevelFwdWorkgroups = 256;  // the K-split forward of a level launch aims at this grid

void launch_level_fwd(int dtype, const int* kinds, const FwdArgs* args, int n, hipStream_t st) {
  Merged<FwdArgs> m{};
  Merged<FwdArgs> e{};  // the K-split parts' epilogues
  m.n = 0;
  e.n = 0;
  int total = 0, erows = 0, hp = 0;
  const int esize = dtype == FOLD_BF16 ? 2 : 4;
  // Each group's plan aims at one workgroup per compute unit; together they would give a level two or three.
  // The K splits are cut in proportion so that the level's grid stays near one workgroup per compute unit:
  // fewer, longer slices write and re-read fewer partial sums (config 4, two or three groups a level: the
  // forward 3.04 -> 2.76 ms a step; a cap of 512 workgroups gave 2.93, 384 2.83, 192 2.87, 128 3.00).
  long long planned = 0;
  for (int k = 0; k < n; ++k) {
    const FwdArgs& a = args[k];
    if (a.rows <= 0) continue;
    const FwdPlan pl = fwd_plan(a.rows, a.HP, a.has_input ? a.INP : 0, a.arity, esize, a.zpart != nullptr);
    planned += (long long)cdiv(a.rows, 128) * (a.HP / 32) * pl.ksplit;
  }
  for (int k = 0; k < n; ++k) {
    FwdArgs a = args[k];
    if (a.rows <= 0) continue;
    const FwdPlan pl = fwd_plan(a.rows, a.HP, a.has_input ? a.INP : 0, a.arity, esize, a.zpart != nullptr);
    const int G = gates_of(kinds[k]);
    a.ksplit = pl.ksplit;
    if (planned > kLevelFwdWorkgroups && a.ksplit > 1)
      a.ksplit = std::max<int>(1, (int)(a.ksplit * kLevelFwdWorkgroups / planned));
    if (a.ksplit > 1 && a.zcap > 0) {
      const size_t fit = a.zcap / ((size_t)a.rows * G * a.HP);
      a.ksplit = (int)std::min<size_t>((size_t)a.ksplit, fit);
      if (a.ksplit < 2) a.ksplit = 1;
    }
    const int R = (int)cdiv(a.rows, 128), UB = a.HP / 32;
    a.map = a.rows >= G * a.HP ? kMapRows : kMapCols;
    const int grid = a.map == kMapRows ? xcd_grid(UB * a.ksplit, R) : xcd_grid(R * a.ksplit, UB);
    m.begin[m.n] = total;
    m.variant[m.n] = 2 * kinds[k] + (a.ksplit > 1 ? 1 : 0);
    m.a[m.n++] = a;
    total += grid;
    if (a.ksplit > 1) {
      e.begin[e.n] = erows;
      e.variant[e.n] = kinds[k];
      e.a[e.n++] = a;
      erows += a.rows;
    }
    hp = a.HP;
  }
  if (m.n == 0) return;
  m.begin[m.n] = total;
  e.begin[e.n] = erows;
  ProfScope prof(dtype == FOLD_BF16 ? "cell_fwd.level.bf16" : "cell_fwd.level.f32", st);
  if (dtype == FOLD_BF16) {
    hipLaunchKernelGGL(k_level_fwd<uint16_t>, dim3(total), dim3(kThreads), 0, st, m);
    if (e.n) hipLaunchKernelGGL(k_level_epi<uint16_t>, dim3(erows), dim3(std::min(hp, 1024)), 0, st, e);
  } else {
    hipLaunchKernelGGL(k_level_fwd<float>, dim3(total), dim3(kThreads), 0, st, m);
    if (e.n) hipLaunchKernelGGL(k_level_epi<float>, dim3(erows), dim3(std::min(hp, 1024)), 0, st, e);
  }
}

void launch_level_cbwd(const int* kinds, const BwdCellArgs* args, int n, hipStream_t st) {
  Merged<BwdCellArgs> m{};
  m.n = 0;
  int total = 0, hp = 0;
  bool bf = false;
  for (int k = 0; k < n; ++k) {
    if (args[k].rows <= 0) continue;
    m.begin[m.n] = total;
    m.variant[m.n] = kinds[k];
    m.a[m.n++] = args[k];
    total += args[k].rows;
    hp = args[k].HP;
    if (kinds[k] != FOLD_EMBED && args[k].dz_bf16) bf = true;
  }
  if (m.n == 0) return;
  m.begin[m.n] = total;
  ProfScope prof("cell_bwd.level", st);
  if (bf)
    hipLaunchKernelGGL(k_level_cbwd<true>, dim3(total), dim3(std::min(std::max(hp / 2, kWave), 1024)), 0, st, m);
  else
    hipLaunchKernelGGL(k_level_cbwd<false>, dim3(total), dim3(std::min(std::max(hp / 2, kWave), 1024)), 0, st, m);
}

bool bwd_dx_is_narrow(int dtype, const DxArgs& a) {
  if (a.rows <= 0 || a.Nb <= 0) return false;
  return !dx_plan(a.rows, a.Nb, a.Kb, dtype == FOLD_BF16 ? 2 : 4, a.can_split != 0).wide;
}

void launch_level_dx(int dtype, const DxArgs* args, int n, hipStream_t st) {
  Merged<DxArgs> m{};
  m.n = 0;
  int total = 0, mtmax = 1;
  for (int k = 0; k < n; ++k) {
    DxArgs a = args[k];
    if (a.rows <= 0 || a.Nb <= 0) continue;
    const DxPlan pl = dx_plan(a.rows, a.Nb, a.Kb, dtype == FOLD_BF16 ? 2 : 4, a.can_split != 0);
    a.ksplit = pl.ksplit;
    const int R = (int)cdiv(a.rows, 128 * pl.mt), NT = (int)cdiv(a.Nb, 128);
    a.map = a.rows >= a.Nb ? kMapRows : kMapCols;
    const int grid = a.map == kMapRows ? xcd_grid(NT * pl.ksplit, R) : xcd_grid(R * pl.ksplit, NT);
    m.begin[m.n] = total;
    m.variant[m.n] = 2 * pl.mt + (pl.ksplit > 1 ? 1 : 0);
    m.a[m.n++] = a;
    total += grid;
    mtmax = std::max(mtmax, pl.mt);
  }
  if (m.n == 0) return;
  m.begin[m.n] = total;
  ProfScope prof(dtype == FOLD_BF16 ? "bwd_dx.level.bf16" : "bwd_dx.level.f32", st);
#define FOLD_LDX(T_, M_) hipLaunchKernelGGL((k_level_dx<T_, M_>), dim3(total), dim3(kThreads), 0, st, m)
  if (dtype == FOLD_BF16) {
    if (mtmax == 2) FOLD_LDX(uint16_t, 2); else FOLD_LDX(uint16_t, 1);
  } else {
    if (mtmax == 2) FOLD_LDX(float, 2); else FOLD_LDX(float, 1);
  }
#undef FOLD_LDX
}

}  // namespace fold
