// Internal definitions shared by the library's HIP sources (gfx950 / CDNA4 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "fold.h"

namespace fold {

// ---------------------------------------------------------------- constants

constexpr int kWave = 64;          // CDNA wavefront
constexpr int kUnit = 32;          // hidden units per MFMA output tile column block
constexpr int kPadK = 64;          // every K segment (input width, hidden) is padded to this
constexpr int kMaxGates = 5;
constexpr int kMaxHidden = 4096;   // the backward stages one row's bf16 dz (G * HP halves) in LDS

inline int round_up(int x, int m) { return (x + m - 1) / m * m; }
inline int64_t round_up64(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// Internal cell kind of a Tree-LSTM operation without children (a leaf: arity 0).  Its child cell states
// are the zero state, so the forget gates multiply zero and cannot change c, h or any gradient; the leaf
// kernels compute, save and differentiate only the live gates (i | o | u), in that compact order.
constexpr int kTreeLstmLeaf = 8;

// the feed-forward attention operations: elementwise kernels of their own, no matrix-core contraction
inline bool is_attn(int kind) { return kind >= FOLD_ATTN_SCORE && kind <= FOLD_ATTN_OUT; }

inline int gates_of(int kind) {
  switch (kind) {
    case FOLD_TREERNN: return 1;
    case FOLD_TREELSTM: return 5;
    case FOLD_LSTM: return 4;
    case FOLD_PROJ: return 1;
    case kTreeLstmLeaf: return 3;
    default: return 0;
  }
}

// Gate map of a compact gate layout: canonical gate index of compact gate g in bits [3g, 3g + 3).
inline int gate_code_identity(int G) {
  int c = 0;
  for (int g = 0; g < G; ++g) c |= g << (3 * g);
  return c;
}
constexpr int kTreeLstmLeafGates = 0 | (3 << 3) | (4 << 6);  // i, o, u of (i | f_l | f_r | o | u)
__host__ __device__ inline int gate_of_code(int code, int g) { return (code >> (3 * g)) & 7; }

// Row stride of every row the kernels read (pools, leaf table, gradients): whole K segments, so a stage
// of 128 bytes never runs past a row and the pad columns (zero) meet zero weights.
inline int row_ld(int width) { return round_up(width < 1 ? 1 : width, kPadK); }

// ---------------------------------------------------------------- error state

void set_error(const std::string& msg);
void clear_error();

#define FOLD_HIP_CHECK(expr)                                                        \
  do {                                                                              \
    hipError_t e_ = (expr);                                                         \
    if (e_ != hipSuccess) {                                                         \
      ::fold::set_error(std::string(#expr) + ": " + hipGetErrorString(e_));         \
      return FOLD_E_DEVICE;                                                         \
    }                                                                               \
  } while (0)

// ---------------------------------------------------------------- kernel timing

// Schedule group and op that the launches issued next on this thread belong to (-1: none); kept
// with every profiling record.
void prof_tag(int group, int op);

// Records a HIP event pair around the launches made while it is alive, if profiling is on.
class ProfScope {
 public:
  ProfScope(const char* name, hipStream_t st);
  ~ProfScope();
  ProfScope(const ProfScope&) = delete;
  ProfScope& operator=(const ProfScope&) = delete;

 private:
  const char* name_;
  hipStream_t st_;
  void* start_ = nullptr;
  void* stop_ = nullptr;
};

// ---------------------------------------------------------------- handles

struct Sched {
  int N = 0, E = 0, G = 0, num_ops = 0, D = 0, num_groups = 0, R = 0, max_parents = 0, num_inputs = 0;
  int device = 0;
  std::vector<fold_op> ops;
  // one device allocation holds every int array below (the level and group tables included)
  void* blob = nullptr;
  int32_t *depth = nullptr, *node_pos = nullptr, *pos_node = nullptr, *level_ptr = nullptr;
  int32_t *g_level = nullptr, *g_op = nullptr, *g_row_begin = nullptr, *g_rows = nullptr,
          *g_idx_off = nullptr;
  int32_t *child_pos = nullptr, *input_idx = nullptr, *root_pos = nullptr;
  int32_t *pos_group = nullptr;   // [N] group of every pool row
  int32_t *pos_npar = nullptr;    // [N] number of parent edges of every pool row
  int32_t *child_one = nullptr;   // [E] beside child_pos: 1 if that child has exactly one parent edge
  int32_t *op_rows = nullptr;     // [N] pool rows sorted by (op, row)
  int32_t *op_cpos = nullptr;     // [2N] child pool rows of op_rows[q] at 2q + k (-1 past the arity)
  int32_t *op_inp = nullptr;      // [N] leaf-table row of op_rows[q], or -1
  // pool rows sorted by (op, leaf-table row), and the runs of equal (op, leaf-table row) in that list: run u is
  // tok_rows[tok_start[u] .. tok_start[u + 1]), of leaf-table row tok_row[u]; tok_seg[i] = the run of entry i
  int32_t *tok_rows = nullptr, *tok_seg = nullptr, *tok_start = nullptr, *tok_row = nullptr;
  // [num_groups] per child slot k: first pool row of the slot's children when they are the consecutive
  // rows base .. base + rows - 1, each with one parent edge (a static-graph layout), else -1
  int32_t *g_cbase0 = nullptr, *g_cbase1 = nullptr;
  std::vector<int32_t> h_level_ptr, h_level, h_op, h_row_begin, h_rows, h_idx_off, h_cbase0, h_cbase1;
  std::vector<int32_t> h_op_row_ptr;  // [num_ops + 1] ranges of op_rows (and of tok_rows)
  std::vector<int32_t> h_tok_ptr;     // [num_ops + 1] ranges of the runs of each op
};

// The paper's own form of a schedule (typed per-depth states, pass-through operations), fold_schedule_typed.
struct TypedSched {
  int N = 0, E = 0, K = 0, T = 0, D = 0, nb = 0, P = 0, M = 0, ngather = 0;
  void* blob = nullptr;  // every device array below
  int32_t *depth = nullptr, *batch_depth = nullptr, *batch_op = nullptr, *batch_rows = nullptr,
          *batch_goff = nullptr, *batch_begin = nullptr, *item_node = nullptr, *gather = nullptr,
          *pass_node = nullptr, *pass_slot = nullptr, *pass_depth = nullptr, *state_size = nullptr,
          *edge_index = nullptr;
  std::vector<int32_t> h_depth_b, h_op_b, h_rows_b, h_goff_b, h_state_size;
};

// Packed weights of one parameter set.
struct PackedSet {
  int kind = 0, in_dim = 0, arity = 0, G = 0;
  int INP = 0;        // input segment width padded to kPadK (0 if no W_in)
  int Kf = 0;         // forward K = INP + arity * HP
  int Nf = 0;         // forward N = G * HP (gate blocks interleaved per kUnit units)
  // forward weights, n-major [Nf][Kf] (element type of the params)
  void* Wf = nullptr;
  // backward, n-major, K = G * HP in canonical gate-block order:
  void* Wb_rec = nullptr;  // [arity * HP][G * HP]
  void* Wb_in = nullptr;   // [INP][G * HP]
  float* bias = nullptr;   // [G * HP] fp32, zero padded
  // Tree-LSTM sets: the same three for leaf operations, over the live gates (i | o | u) only
  void* Wf_leaf = nullptr;     // [3 * HP interleaved per kUnit units][INP]
  void* Wb_in_leaf = nullptr;  // [INP][3 * HP]
  float* bias_leaf = nullptr;  // [3 * HP]
};

struct Packed {
  int dtype = 0, H = 0, HP = 0, ld = 0;
  int device = 0;
  void* zero = nullptr;  // zero_bytes of zeros: the row every absent operand row (child slot -1, tile
  size_t zero_bytes = 0; // rows past the end) is loaded from
  std::vector<PackedSet> sets;
  std::vector<void*> allocs;
};

}  // namespace fold

struct fold_sched { fold::Sched s; };
struct fold_typed_sched { fold::TypedSched t; };
struct fold_packed { fold::Packed p; };

// ---------------------------------------------------------------- device helpers
namespace fold {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

// fp32 -> bf16, round to nearest even (NaN kept quiet)
__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Gate nonlinearities on the hardware exp2 / reciprocal units (v_exp_f32, v_rcp_f32, about one ulp
// each): sigma(x) = 1 / (1 + e^-x); for x -> -inf, e^-x overflows to +inf and the reciprocal gives 0.
// tanh(x) = 2 sigma(2x) - 1 (absolute error a few 1e-7) for |x| >= 1/8; below, where that difference would lose
// the relative accuracy, the odd Taylor series x - x^3/3 + 2x^5/15 - 17x^7/315 (truncation < 2e-10 relative).
__device__ __forceinline__ float fast_exp(float x) { return __builtin_amdgcn_exp2f(x * 1.4426950408889634f); }
__device__ __forceinline__ float sigmoidf_(float x) { return __builtin_amdgcn_rcpf(1.f + fast_exp(-x)); }
__device__ __forceinline__ float tanhf_(float x) {
  const float x2 = x * x;
  const float series = x * (1.f + x2 * (-1.f / 3.f + x2 * (2.f / 15.f + x2 * (-17.f / 315.f))));
  return fabsf(x) < 0.125f ? series : 2.f * sigmoidf_(2.f * x) - 1.f;
}

}  // namespace fold
