/*
 * fold.h -- C ABI of the MI355X dynamic-batching library.
 *
 * Dynamic batching (Looks et al., "Deep Learning with Dynamic Computation
 * Graphs", Section 2) evaluates a batch of computation graphs of different
 * shapes and sizes by
 *   1. giving every node a depth (constants have depth 0; a node whose inputs
 *      have maximum depth d has depth d + 1),
 *   2. batching together all nodes that run the same operation at the same
 *      depth,
 *   3. gathering each batch's inputs by index from the concatenated outputs of
 *      earlier depths, running the operation once per (depth, operation), and
 *      concatenating the outputs back,
 * and back-propagates through the same gathers and concatenations.  This
 * library exposes that hot path as three calls:
 *
 *   fold_schedule   CSR graphs -> per-level, per-operation gather indices
 *   fold_forward    schedule + parameters + leaf rows -> every node's state
 *                   and the roots' outputs
 *   fold_backward   reverse-level pass: gradients scatter-added into child
 *                   states, weight gradients accumulated
 *
 * Conventions shared by every entry point
 *   - Every call returns FOLD_OK (0) or a negative FOLD_E_* code; the
 *     matching text is available from fold_last_error() on the calling
 *     thread.  No C++ exception crosses this boundary.
 *   - "device" pointers are HIP device allocations on the current device;
 *     "host" pointers are ordinary host memory.  The caller owns every
 *     buffer it passes in; the library owns the fold_sched / fold_packed
 *     handles it returns and everything they point to.
 *   - All work is enqueued on the given stream.  fold_schedule and
 *     fold_pack_params synchronise that stream (they read back sizes);
 *     fold_forward and fold_backward never synchronise and never allocate.
 *   - Node states live in one pool in SCHEDULE order: row p of a pool holds
 *     node pos_node[p].  Every row-major float/bf16 matrix the library reads
 *     or writes has a row stride of fold_row_ld(width) elements (width
 *     rounded up to 64); columns beyond the width are written as zero
 *     (pools) and must hold zeros in inputs (the leaf table): the kernels
 *     load whole 128-byte row segments and meet those columns with zero
 *     weights, so any finite value there is harmless and NaN / Inf is not.
 *   - Handles are immutable after creation (fold_pack_update aside, which
 *     rewrites a packed handle's weights in place) and may be shared by
 *     concurrent calls on different streams that use different output buffers.
 */
#ifndef FOLD_H_
#define FOLD_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------ */
#define FOLD_OK 0
#define FOLD_E_INVALID -1  /* null pointer, negative count, bad dims/dtype, bad op table, broken graph_ptr/child_ptr */
#define FOLD_E_OP -2       /* node_op out of [0, num_ops) */
#define FOLD_E_ARITY -3    /* a node's child count differs from its operation's arity */
#define FOLD_E_CHILD -4    /* child id out of range or in another graph (-1, the zero state, is allowed) */
#define FOLD_E_INPUT -5    /* input row out of [0, num_inputs), or present/absent against has_input */
#define FOLD_E_CYCLE -6    /* the graph is not acyclic */
#define FOLD_E_NOMEM -7    /* device allocation failed */
#define FOLD_E_DEVICE -8   /* a HIP call failed */
#define FOLD_E_MISMATCH -9 /* schedule / parameters / workspace inconsistent with each other */

/* ---- operation kinds (the operations of the paper's experiments) ------- */
enum {
  FOLD_EMBED = 0,    /* h = table[input]                        (embedding lookup, arity 0, has_input) */
  FOLD_TREERNN = 1,  /* h = tanh([h_l; h_r] W + b)              (binary TreeRNN cell, arity 2) */
  FOLD_TREELSTM = 2, /* binary N-ary Tree-LSTM, gates (i|f_l|f_r|o|u); arity 0 with input = leaf
                        TreeLSTM(x, 0, 0), arity 2 = internal TreeLSTM(x?, h_l, h_r) */
  FOLD_LSTM = 3,     /* one LSTM step, gates (i|f|o|u), arity 1 (child -1 = zero start state) */
  FOLD_PROJ = 4,     /* h = tanh(h_c P + b), c = c_c            (unary projection, arity 1) */
  /* Feed-forward attention (Section 3.4, Appendix A): e_t = a(h_t), alpha = softmax(e),
   * c = sum_t alpha_t h_t, with the scorer a(h) = w . h + b.  The two sums over t are carried as one
   * aggregate of a set of scored items, (m, s, acc) = (max e, sum exp(e - m), sum exp(e - m) h), held in
   * a node's state as h = acc and c = [m, s, 0, ...] (needs hidden >= 2), so that a Reduce over the items
   * batches like any other operation.  Gradients hold m fixed (the value acc / s does not depend on it). */
  FOLD_ATTN_SCORE = 5, /* one item from the child's h: e = w . h_c + b, h = h_c, c = [e, 1, 0..]
                          (arity 1; parameters: W_rec = w as [H, 1], bias = [b]) */
  FOLD_ATTN_SUM = 6,   /* union of the two children's sets: m = max(m_1, m_2), x_k = exp(m_k - m),
                          s = x_1 s_1 + x_2 s_2, acc = x_1 acc_1 + x_2 acc_2; a child with s = 0 (the
                          zero state, an empty set) takes no part; two empty sets give the zero state
                          (arity 2, no parameters: W_rec and bias may be NULL) */
  FOLD_ATTN_OUT = 7    /* the attention output: h = acc / s (the zero vector for an empty set), c = 0
                          (arity 1, no parameters) */
};

/* ---- element types of weights, leaf table and h pool ------------------- */
enum { FOLD_F32 = 0, FOLD_BF16 = 1 };

/* One operation of the op table.  The paper requires every operation to be
 * specified and enumerated in advance (Section 2); the op id is the index in
 * the table, and groups of one depth are ordered by it. */
typedef struct {
  int32_t kind;      /* FOLD_EMBED .. FOLD_ATTN_OUT */
  int32_t arity;     /* number of node children (CSR entries) */
  int32_t has_input; /* 1: reads leaf-table row node_input[v] */
  int32_t param_set; /* index into fold_params.sets */
} fold_op;

/* A batch of graphs as one disconnected DAG (Section 2), CSR form.
 * Node ids are global; node order inside a graph is arbitrary.  Children
 * must belong to the node's own graph; -1 names a zero state. */
typedef struct {
  int32_t num_graphs;        /* G >= 0 */
  int32_t num_nodes;         /* N >= 0 */
  int32_t num_edges;         /* E >= 0, = child_ptr[N] */
  int32_t num_ops;           /* 1 .. 256 (more: FOLD_E_INVALID) */
  int32_t num_inputs;        /* rows of the leaf table that node_input may name */
  const int32_t* graph_ptr;  /* device [G+1], graph_ptr[0] = 0, graph_ptr[G] = N, nondecreasing */
  const int32_t* node_op;    /* device [N] */
  const int32_t* child_ptr;  /* device [N+1], child_ptr[0] = 0, nondecreasing */
  const int32_t* child_idx;  /* device [E] global node ids or -1 */
  const int32_t* node_input; /* device [N] leaf-table row, or -1 */
  const fold_op* ops;        /* host [num_ops] */
} fold_batch;

typedef struct fold_sched fold_sched;
typedef struct fold_packed fold_packed;

/* Read-only view of a schedule.  Device arrays are owned by the schedule. */
typedef struct {
  int32_t num_nodes, num_edges, num_graphs, num_ops;
  int32_t num_levels; /* D = maximum depth = number of batched steps */
  int32_t num_groups; /* non-empty (depth, op) groups */
  int32_t num_roots;  /* nodes that are nobody's child */
  int32_t max_parents;
  /* device, int32 */
  const int32_t* depth;           /* [N]   depth of node v (leaf operations: 1) */
  const int32_t* node_pos;        /* [N]   pool row of node v */
  const int32_t* pos_node;        /* [N]   node at pool row p */
  const int32_t* level_ptr;       /* [D+1] rows of depth <= l end at level_ptr[l] */
  const int32_t* group_level;     /* [num_groups] */
  const int32_t* group_op;        /* [num_groups] */
  const int32_t* group_row_begin; /* [num_groups] first pool row of the group */
  const int32_t* group_rows;      /* [num_groups] */
  const int32_t* group_idx_off;   /* [num_groups] offset of the group's edges in child_pos */
  const int32_t* child_pos;       /* [E]   pool row of child k of the group's row r at
                                     group_idx_off + r * arity + k, or -1 (zero state) */
  const int32_t* input_idx;       /* [N]   leaf-table row read by pool row p, or -1 */
  const int32_t* root_pos;        /* [num_roots] pool rows of the roots, ascending node id */
  /* host copies */
  const int32_t* h_level_ptr;
  const int32_t* h_group_level;
  const int32_t* h_group_op;
  const int32_t* h_group_row_begin;
  const int32_t* h_group_rows;
  const int32_t* h_group_idx_off;
  /* Static-graph layout, per group and child slot k = 0, 1: the pool row of the
   * slot's first child when the slot's children are the consecutive rows
   * base .. base + rows - 1 and each has exactly one parent edge (a batch of
   * identically shaped graphs with one operation per node position, i.e.
   * manual batching, has it on every slot); -1 otherwise.  The forward
   * kernels address such children as base + row, with no child_pos load.
   * Device [num_groups] each, and host copies. */
  const int32_t* group_child_base0;
  const int32_t* group_child_base1;
  const int32_t* h_group_child_base0;
  const int32_t* h_group_child_base1;
} fold_sched_info;

/* Schedule a batch (Section 2, the greedy scheduling algorithm):
 * validates the CSR (codes above), computes every node's depth on the GPU
 * (cycles -> FOLD_E_CYCLE), sorts the nodes by the key (depth - 1) * num_ops
 * + op with ties kept in node-id order (a stable counting sort), and emits
 * the per-group gather indices.  The edge label of the paper (index i into
 * the concatenated outputs of depth d) is the pool row minus
 * level_ptr[d - 1]; pass-throughs are unnecessary because the pool keeps
 * every level.  Synchronises `stream` twice (error flag and depth, then the
 * group table).  On success *out is a new handle to free with
 * fold_sched_free; on error *out is NULL. */
int32_t fold_schedule(const fold_batch* batch, hipStream_t stream, fold_sched** out);
int32_t fold_sched_get_info(const fold_sched* sched, fold_sched_info* out);
int32_t fold_sched_free(fold_sched* sched);

/* ---- the paper's own form of the schedule ---------------------------------
 * Section 2 schedules a typed DAG: source nodes are constants of a tensor
 * type, other nodes invoke operations whose inputs and outputs have fixed
 * tensor types, and an edge connects output k of node u to input j of node
 * v.  Its five steps: (1) depth (constants 0, an operation node 1 + the
 * largest depth it reads); (2) pass-through (identity) operations, so that a
 * node at depth d + 1 reads only results of depth d; (3) one batch per
 * (depth, operation); (4) at each depth the outputs of one type concatenated
 * in the operations' enumeration order; (5) every edge labelled (d, t, i),
 * the depth and type of the value it reads and its index into that
 * concatenation; the schedule is the indices i grouped by depth and
 * operation.  fold_schedule above is the special case of one state type
 * (node and child states travel together) with pass-throughs elided; this
 * call produces the general form, including an int-typed state such as the
 * word ids of Figure 1.
 *
 * Readings (the paper is silent): pass-throughs are operations too, one per
 * type t, numbered num_ops + t (after the caller's operations), with one
 * input and one output of type t; one pass-through per value and depth,
 * shared by all readers of that value; a batch lists its operation nodes in
 * ascending node id and its pass-through instances in ascending value order
 * (node id, then output slot); an operation's outputs of one type enter
 * that type's concatenation in slot order, each with the whole batch in
 * batch order; the depth-0 state of type t holds the constants of type t in
 * ascending node id. */
typedef struct {
  int32_t num_inputs, num_outputs; /* 1..8 each */
  const int32_t* in_type;          /* host [num_inputs], 0..num_types-1 */
  const int32_t* out_type;         /* host [num_outputs] */
} fold_typed_op;

typedef struct {
  int32_t num_graphs, num_nodes, num_edges;
  int32_t num_ops;    /* 1..64 */
  int32_t num_types;  /* 1..16 */
  const int32_t* graph_ptr; /* device [G+1]: graph g is nodes graph_ptr[g] .. graph_ptr[g+1]-1 */
  const int32_t* node_op;   /* device [N]: operation id, or -1 - t for a constant of type t */
  const int32_t* in_ptr;    /* device [N+1]: node v's inputs are edges in_ptr[v] .. in_ptr[v+1]-1 */
  const int32_t* in_node;   /* device [E]: source node of the edge (same graph) */
  const int32_t* in_slot;   /* device [E]: source output slot */
  const fold_typed_op* ops; /* host [num_ops] */
} fold_typed_batch;

typedef struct fold_typed_sched fold_typed_sched;

typedef struct {
  int32_t num_levels;   /* D: the largest depth */
  int32_t num_batches;  /* non-empty (depth, operation) batches, pass-throughs included */
  int32_t num_passes;   /* pass-through instances */
  int32_t num_items;    /* operation nodes + pass-through instances */
  int32_t num_gather;   /* entries of gather */
  int32_t num_ops, num_types;
  /* device, int32 */
  const int32_t* depth;             /* [N] */
  const int32_t* batch_depth;       /* [num_batches] ascending (depth, operation) */
  const int32_t* batch_op;          /* [num_batches] operation, or num_ops + t: pass-through of type t */
  const int32_t* batch_rows;        /* [num_batches] */
  const int32_t* batch_gather_off;  /* [num_batches] input j of row r at gather[off + j * rows + r] */
  const int32_t* batch_item_begin;  /* [num_batches] first entry in item_node */
  const int32_t* item_node;         /* [num_items] node id, or -1 - p for pass-through instance p */
  const int32_t* gather;            /* [num_gather] indices i into the (depth - 1, input type) state */
  const int32_t* pass_node;         /* [num_passes] the value (node, output slot) carried, and the */
  const int32_t* pass_slot;         /*   depth of the instance; ascending value, then depth */
  const int32_t* pass_depth;
  const int32_t* state_size;        /* [(D + 1) * num_types]: rows of the state (d, t) at d * T + t */
  const int32_t* edge_index;        /* [E] label index i of every input edge (its d is the reader's
                                       depth - 1, its t the input's type) */
  /* host copies */
  const int32_t* h_batch_depth;
  const int32_t* h_batch_op;
  const int32_t* h_batch_rows;
  const int32_t* h_batch_gather_off;
  const int32_t* h_state_size;
} fold_typed_sched_info;

/* fold_schedule_typed: validates the batch (FOLD_E_INVALID for a malformed
 * op table, graph_ptr / in_ptr, an edge from a missing node or output or of
 * the wrong type, a constant with inputs or an operation node with the wrong
 * input count; FOLD_E_CHILD for an edge across graphs; FOLD_E_OP for an
 * operation or constant type out of range; FOLD_E_CYCLE), then schedules it
 * on the GPU.  The library allocates and owns the result.  Synchronises
 * `stream` twice: once to size the pass-through arrays, once at the end. */
int32_t fold_schedule_typed(const fold_typed_batch* batch, hipStream_t stream, fold_typed_sched** out);
int32_t fold_typed_sched_get_info(const fold_typed_sched* sched, fold_typed_sched_info* out);
int32_t fold_typed_sched_free(fold_typed_sched* sched);


/* Parameters of one operation family, canonical row-major layout, device
 * memory, element type fold_params.dtype (bias always fp32).  G gate blocks
 * (Tree-LSTM 5, LSTM 4, TreeRNN / PROJ 1, EMBED 0) of `hidden` columns each,
 * in the order given under FOLD_TREELSTM / FOLD_LSTM.  Attention sets
 * (in_dim 0): FOLD_ATTN_SCORE has arity 1, W_rec = the scorer vector w as
 * [hidden, 1] and bias = [b] (one float); FOLD_ATTN_SUM (arity 2) and
 * FOLD_ATTN_OUT (arity 1) hold no values (W_rec and bias may be NULL).  Their
 * gradients (fold_param_grads) are dW_rec [hidden] and dbias [1] for the
 * scorer, none for the other two.  hidden must be at least 2 once an
 * attention set is present. */
typedef struct {
  int32_t kind;
  int32_t in_dim;    /* width of the leaf-table rows the ops read (EMBED: = hidden) */
  int32_t arity;     /* child slots covered by W_rec */
  const void* W_in;  /* [in_dim, G*hidden] or NULL when in_dim == 0 */
  const void* W_rec; /* [arity*hidden, G*hidden]; rows k*hidden.. belong to child k */
  const float* bias; /* [G*hidden] (NULL for EMBED) */
} fold_param_set;

typedef struct {
  int32_t dtype;  /* FOLD_F32 or FOLD_BF16 */
  int32_t hidden; /* H, 1 .. 4096 */
  int32_t num_sets;
  const fold_param_set* sets; /* host [num_sets] */
} fold_params;

/* Copy the parameters into the library's MFMA-friendly layouts (gate blocks
 * interleaved per 32 hidden units, K padded per input segment, transposed
 * copies for the backward).  Reads the caller's arrays once; synchronises.
 * FOLD_E_INVALID for a set whose packed matrix, G * H' * (in_dim' + arity * H')
 * entries (primes: rounded up to 64), would reach 2^32. */
int32_t fold_pack_params(const fold_params* params, hipStream_t stream, fold_packed** out);
int32_t fold_packed_free(fold_packed* packed);

/* Re-pack new values of the same parameters into an existing handle (a
 * training loop after each optimizer step): `params` must match the handle
 * in dtype, hidden, number of sets and each set's kind, in_dim and arity
 * (FOLD_E_MISMATCH otherwise; FOLD_E_INVALID for the checks of
 * fold_pack_params).  Enqueued on `stream`; asynchronous; allocates
 * nothing; the packed buffers keep their addresses, so HIP graphs recorded
 * with the handle stay valid.  The caller orders it after every pass that
 * still reads the old weights and before every pass that needs the new. */
int32_t fold_pack_update(fold_packed* packed, const fold_params* params, hipStream_t stream);

/* Row stride, in elements, that the library uses for a row of `width`
 * elements (pools, root outputs, gradients of node states, leaf tables):
 * width rounded up to a multiple of 64. */
int32_t fold_row_ld(int32_t width);

/* Workspace needed by fold_forward (saved gate activations for the
 * backward) and by fold_backward (the same region plus per-node gradient
 * accumulators).  One buffer of bwd_bytes serves both calls. */
int32_t fold_workspace_size(const fold_sched* sched, const fold_packed* packed,
                            size_t* fwd_bytes, size_t* bwd_bytes);

/* Forward pass over every level: for each (depth, op) group in order, gather
 * the children's (h, c) rows and the leaf-table rows by index, contract
 * with the operation's weights on the matrix cores, apply the cell, and
 * write the group's rows of the pools.
 *   leaf_table  device [leaf_rows, fold_row_ld(in_dim)] of dtype (may be NULL
 *               if no op has an input)
 *   h_pool      device [N, fold_row_ld(H)] of dtype (written)
 *   c_pool      device [N, fold_row_ld(H)] fp32 (written)
 *   roots_out   device [num_roots, fold_row_ld(H)] of dtype (written; NULL skips)
 *   ws          device workspace of >= fwd_bytes; receives the activations
 *               fold_backward needs (NULL with ws_bytes 0: inference only)
 * Asynchronous; allocates nothing. */
int32_t fold_forward(const fold_sched* sched, const fold_packed* packed,
                     const void* leaf_table, int64_t leaf_rows,
                     void* h_pool, float* c_pool, void* roots_out,
                     void* ws, size_t ws_bytes, hipStream_t stream);

/* Gradients of one parameter set, canonical layout, fp32, device memory.
 * Accumulated (+=): the caller zeroes them.  NULL skips that tensor. */
typedef struct {
  float* dW_in;  /* [in_dim, G*H] */
  float* dW_rec; /* [arity*H, G*H] */
  float* dbias;  /* [G*H] */
} fold_param_grads;

typedef struct {
  int32_t num_sets;              /* must equal the packed parameters' */
  const fold_param_grads* sets;  /* host [num_sets] */
  float* d_leaf_table;           /* device [leaf_rows, fold_row_ld(in_dim)] fp32, += ; or NULL */
} fold_grads;

/* Backward pass, levels in reverse order.  The upstream gradient is
 * dh_roots on the roots (row r = root r, in ascending node id) plus, if
 * given, dh_nodes on every pool row; the roots' cell states get none.
 * For each group: dz from the saved gates, dz . W^T scatter-added into the
 * children's (h, c) gradients (every parent lies at a greater depth, so a
 * child's gradient is complete before its own level runs); then, per
 * operation, the weight gradients dW += X^T dz, db += sum dz, and the
 * leaf-table gradient: dz summed over the operation's rows of each
 * leaf-table row, times W_in^T, added into that row (the same sum as adding
 * every row's dz . W_in^T, in another order).
 *   h_pool, c_pool, ws   exactly as left by fold_forward with this schedule
 *   dh_roots             device [num_roots, ld(H)] fp32 or NULL
 *   dh_nodes             device [N, ld(H)] fp32 (pool order) or NULL
 *   dh_out, dc_out       device [N, ld(H)] fp32 (pool order) or NULL: receive every
 *                        node's total upstream gradient of h and c (every row
 *                        written whole)
 * dh_roots, dh_nodes, dh_out, dc_out and ws must be 16-byte aligned
 * (FOLD_E_INVALID otherwise).  Asynchronous; allocates nothing. */
int32_t fold_backward(const fold_sched* sched, const fold_packed* packed,
                      const void* leaf_table, int64_t leaf_rows,
                      const void* h_pool, const float* c_pool,
                      const float* dh_roots, const float* dh_nodes,
                      const fold_grads* grads, float* dh_out, float* dc_out,
                      void* ws, size_t ws_bytes, hipStream_t stream);

/* fold_forward_noalloc: fold_forward for callers that cannot allocate --
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  It computes the same states as fold_forward (inference: no
 * activations are saved for a backward pass) and takes no workspace: the
 * K-split partial sums of narrow levels go to a library-owned 16 MiB device
 * array per GPU (a static __device__ array, held until the process ends).
 * A level whose K split would need more than that splits into fewer slices,
 * or none, so no batch is rejected for its size; results stay within the
 * tolerance of fold_forward's (slices may differ, so not always bit-equal).
 * Arguments, errors and asynchrony are those of fold_forward without ws;
 * FOLD_E_MISMATCH if the handles belong to another device than the current
 * one, FOLD_E_DEVICE if the array's address cannot be looked up.  It calls
 * no hipMalloc, hipFree or allocating routine.  Every call on one GPU shares
 * that GPU's array, so calls that overlap on one GPU (two streams, two host
 * threads) race: serialise them.  No contents carry over between calls that
 * matter (every slice writes its partial sums before they are read). */
int32_t fold_forward_noalloc(const fold_sched* sched, const fold_packed* packed,
                             const void* leaf_table, int64_t leaf_rows,
                             void* h_pool, float* c_pool, void* roots_out,
                             hipStream_t stream);

/* Recurrent dropout (Section 3.5 trains the Tree-LSTM with the recurrent
 * dropout of Semeniuta et al., "Recurrent dropout without memory loss"):
 * the forward and backward passes above with a mask on the candidate update
 * u where it enters the memory cell, c = i*(m*u) + sum_k f_k*c_k, so the
 * forget paths of the cell state are never dropped.  Operations of kind
 * FOLD_TREELSTM (leaf and internal) and FOLD_LSTM use the mask; the other
 * kinds ignore it.
 *   u_mask  device [N, fold_row_ld(H)] fp32, pool order (row p = node
 *           pos_node[p]); any multiplier (0 or 1/(1-p) for inverted
 *           dropout, drawn by the caller).  Caller-owned, read only; the
 *           backward must get the same mask as the forward.  NULL is
 *           FOLD_E_INVALID (use fold_forward / fold_backward instead).
 * Every other argument, error and the asynchrony are as in fold_forward /
 * fold_backward. */
int32_t fold_forward_dropout(const fold_sched* sched, const fold_packed* packed,
                             const void* leaf_table, int64_t leaf_rows,
                             void* h_pool, float* c_pool, void* roots_out,
                             const float* u_mask, void* ws, size_t ws_bytes,
                             hipStream_t stream);
int32_t fold_backward_dropout(const fold_sched* sched, const fold_packed* packed,
                              const void* leaf_table, int64_t leaf_rows,
                              const void* h_pool, const float* c_pool,
                              const float* u_mask, const float* dh_roots,
                              const float* dh_nodes, const fold_grads* grads,
                              float* dh_out, float* dc_out,
                              void* ws, size_t ws_bytes, hipStream_t stream);

/* fold_dropout_mask: draws the recurrent-dropout mask of one training step
 * (the u_mask of fold_forward_dropout / fold_backward_dropout) on the GPU
 * from the counter-based generator Philox4x32-10 (Salmon, Moraes, Dror and
 * Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC 2011).  For node
 * v and hidden unit j < hidden, with r the (j mod 4)-th output word of the
 * call on counter (v, j / 4, low and high 32 bits of step) under the key
 * (low and high 32 bits of seed):
 *     mask[pos(v)][j] = 0 if r < min(floor(p 2^32), 2^32 - 1), else (float)(1 / (1 - p))
 * (inverted dropout: kept units are scaled so the expected multiplier is 1).
 *   mask    device [N, fold_row_ld(hidden)] fp32, POOL order (row q = node
 *           pos_node[q]), 16-byte aligned; written whole, pad columns 0.
 *           Caller-owned.
 *   p       drop probability in [0, 1); p = 0 gives all ones.
 *   seed, step  any 64-bit values; a node's row depends only on (v, seed,
 *           step, p), not on the batch around it.
 * FOLD_E_INVALID for a NULL schedule, hidden outside 1..4096, p outside
 * [0, 1), or a NULL or misaligned mask (N > 0).  Asynchronous; allocates
 * nothing. */
int32_t fold_dropout_mask(const fold_sched* sched, int32_t hidden, double p, uint64_t seed, uint64_t step,
                          float* mask, hipStream_t stream);

/* ---- the training step around the path ------------------------------------
 * Section 3.5 trains the binary Tree-LSTM on trees whose every node carries a
 * class label: a linear layer and a softmax on every node's state h, the
 * cross entropy against the node's label, summed over the nodes, minimised
 * with TensorFlow's Adam optimizer (Section 3.3).  These two calls are that
 * step's loss head and update; fold_backward takes the head's dh_nodes.
 *
 * fold_loss_softmax_ce: per node v with label y_v >= 0
 *     z_v = h_v W_cls + b_cls,  loss_v = log sum_c exp(z_vc) - z_{v,y_v}
 * and the gradients of L = scale * sum_v loss_v:
 *     dz_v = scale (softmax(z_v) - onehot(y_v)),  dh_v = dz_v W_cls^T,
 *     dW_cls += h^T dz,  db_cls += sum_v dz_v;
 * a node with label -1 (or any label outside [0, num_classes)) has loss 0
 * and dh 0.  fp32 arithmetic on h of the packed parameters' dtype.
 *   h_pool     device [N, fold_row_ld(H)] pool (as left by fold_forward)
 *   labels     device [N] int32 in NODE order: class 0..num_classes-1, or -1
 *              (no label)
 *   num_classes  2..8, 10, 16 or 32, with H * num_classes <= 8000
 *   W_cls      device [H, num_classes] fp32 row-major; b_cls device [num_classes] fp32
 *   node_loss  device [N] fp32, NODE order (written)
 *   dh_nodes   device [N, fold_row_ld(H)] fp32, POOL order (written, pad
 *              columns zero): the dh_nodes argument of fold_backward
 *   dW_cls, db_cls  device, fp32, accumulated (+=; the caller zeroes them);
 *              partial sums per block of rows are added in a fixed order,
 *              but the four waves of a block meet in LDS in arrival order,
 *              so the result is reproducible up to the order of those fp32
 *              additions, not bit for bit
 *   ws         device workspace of >= fold_loss_workspace_size bytes (the
 *              per-block partial sums; contents on entry do not matter)
 * FOLD_E_INVALID for an unsupported class count, H * num_classes above
 * 8000, a non-finite scale or a NULL buffer (N > 0); FOLD_E_MISMATCH for a
 * workspace that is too small, and as fold_forward for a schedule and
 * parameters that do not belong together.  Asynchronous; allocates nothing.
 * fold_loss_workspace_size fails with FOLD_E_INVALID as above. */
int32_t fold_loss_workspace_size(const fold_packed* packed, int32_t num_classes, size_t* bytes);
int32_t fold_loss_softmax_ce(const fold_sched* sched, const fold_packed* packed, const void* h_pool,
                             const int32_t* labels, int32_t num_classes, const float* W_cls, const float* b_cls,
                             float scale, float* node_loss, float* dh_nodes, float* dW_cls, float* db_cls,
                             void* ws, size_t ws_bytes, hipStream_t stream);

/* fold_adam_step: step `step` (1, 2, ...) of Adam (Kingma and Ba) in the
 * form of TensorFlow's optimizer, elementwise over n fp32 values:
 *     m = beta1 m + (1 - beta1) g,  v = beta2 v + (1 - beta2) g^2,
 *     p = p - lr_t m / (sqrt(v) + eps),
 *     lr_t = lr sqrt(1 - beta2^step) / (1 - beta1^step)
 * in fp32, with lr_t, 1 - beta1 and 1 - beta2 computed in double first (the
 * hyperparameters are double so that 1 - 0.999 keeps its value).
 * param, m, v are device fp32 arrays updated in place (m, v start at zero);
 * grad is read; param_bf16, if not NULL, receives param rounded to bf16
 * (round to nearest even) for models whose weights are bf16.  Any flat
 * tensor works (weights, biases, a padded leaf table whose pad columns hold
 * zero parameters and gradients, which stay zero).  FOLD_E_INVALID for n < 0,
 * step < 1, beta outside [0, 1), eps < 0, a non-finite lr or a NULL buffer
 * (n > 0).  Asynchronous; allocates nothing. */
int32_t fold_adam_step(int64_t n, float* param, uint16_t* param_bf16, const float* grad, float* m, float* v,
                       double lr, double beta1, double beta2, double eps, int32_t step, hipStream_t stream);

/* ---- a whole step as one HIP graph ----------------------------------------
 * The level loop (Section 2: one batched iteration per depth, so a batch of
 * depth D costs O(D) launches instead of one per node) still issues a few
 * launches per (depth, operation) group.  For deep batches of narrow levels
 * the host launch cost and the gaps between dependent launches dominate.
 * fold_graph_create records, once, exactly the launches that fold_forward
 * (and, with FOLD_STEP_BACKWARD, fold_backward) would enqueue with the
 * buffers below, and instantiates them as a HIP graph; fold_graph_launch
 * submits that step on any stream with one call.
 *   - The buffers are bound at creation: every launch reads and writes the
 *     same device memory (contents may change between launches, addresses
 *     may not).  Recreate the graph to use other buffers.
 *   - With FOLD_STEP_ZERO_GRADS the step first zeroes every gradient tensor
 *     in `grads` (dW_in, dW_rec, dbias of each set, d_leaf_table of
 *     leaf_rows rows), so a launch yields the gradients of this step alone;
 *     without it they accumulate across launches as with fold_backward.
 *   - The recorded step holds kernel nodes only (no memset or copy nodes),
 *     allocates nothing and never synchronises when launched.
 *   - Launches of one graph must not overlap (they share the buffers): keep
 *     them on one stream or order them with events.
 * fold_graph_create synchronises nothing but returns only after
 * instantiation; it fails with the same codes as fold_forward /
 * fold_backward for inconsistent arguments, FOLD_E_DEVICE if capture or
 * instantiation fails, and leaves *out NULL on error.  The graph must be
 * launched on the device that was current at creation (FOLD_E_MISMATCH
 * otherwise).  The schedule and parameter handles must outlive the graph. */
typedef struct fold_graph fold_graph;

typedef struct {
  const void* leaf_table; /* as fold_forward */
  int64_t leaf_rows;
  void* h_pool;
  float* c_pool;
  void* roots_out;        /* or NULL */
  const float* dh_roots;  /* as fold_backward (used with FOLD_STEP_BACKWARD) */
  const float* dh_nodes;
  const fold_grads* grads; /* read at creation; the host arrays may be freed afterwards */
  float* dh_out;
  float* dc_out;
  void* ws;               /* >= fwd_bytes (forward only) or bwd_bytes */
  size_t ws_bytes;
} fold_step_buffers;

#define FOLD_STEP_BACKWARD 1   /* record fold_backward after fold_forward */
#define FOLD_STEP_ZERO_GRADS 2 /* zero the gradients first (needs FOLD_STEP_BACKWARD) */

int32_t fold_graph_create(const fold_sched* sched, const fold_packed* packed, const fold_step_buffers* buffers,
                          int32_t flags, fold_graph** out);
int32_t fold_graph_launch(const fold_graph* graph, hipStream_t stream);
int32_t fold_graph_num_nodes(const fold_graph* graph, int32_t* nodes); /* kernel nodes recorded */
int32_t fold_graph_free(fold_graph* graph);

/* ---- level launches --------------------------------------------------------
 * The groups of one depth are independent, so by default the narrow groups of
 * a level (up to four) run as one launch per kernel stage (one for their
 * contractions, one for their K-split epilogues, one for their cell
 * backwards, one for their dz . W^T), which removes the dependent launches of
 * levels with several operations.  fold_level_launches(0) turns this off for
 * every later call in the process (each group then launches alone, as a static
 * graph of one batched operation per node would run); fold_level_launches(1)
 * turns it back on.  Returns the previous setting (1 or 0).  Results are the
 * same either way up to the order of the atomic additions of shared
 * children. */
int32_t fold_level_launches(int32_t on);

/* ---- per-kernel timing (profiling aid) ----------------------------------
 * While enabled, every kernel the library launches is bracketed by a pair of
 * HIP events recorded on the launch stream, under a short kernel-class name
 * (e.g. "cell_fwd.treelstm.f32").  fold_profile_read waits for the recorded
 * events, returns one entry per class (launch count, summed and largest
 * duration in milliseconds), and clears the record.  Enabling costs one
 * event pair per launch; disabled (the default) it costs nothing. */
typedef struct {
  char name[48];
  int64_t launches;
  double total_ms;
  double max_ms;
} fold_kernel_stat;

int32_t fold_profile_enable(int32_t on);
int32_t fold_profile_read(fold_kernel_stat* out, int32_t capacity, int32_t* count);

/* The same records one by one, in launch order, each with the schedule group
 * it ran for (its index in the group table; -1 for launches of no single
 * group: gradient set-up, roots, the per-operation weight gradients) and its
 * operation id (-1 if none).  This splits a step's time by level and by
 * (depth, op) group (Section 2: one batched operation per group).
 * Writes min(capacity, records) entries to `out` (caller-owned host array),
 * sets *count to the number of records taken, and clears them all, as
 * fold_profile_read does.  With capacity 0 (`out` may be NULL) it only sets
 * *count and keeps the records.  FOLD_E_INVALID for NULL arguments;
 * FOLD_E_DEVICE if an event could not be read. */
typedef struct {
  char name[48];
  int32_t group;
  int32_t op;
  double ms;
} fold_launch_time;

int32_t fold_profile_read_launches(fold_launch_time* out, int32_t capacity, int32_t* count);

/* ---- achievable peaks (diagnostics) --------------------------------------
 * fold_probe_mfma times a loop of independent 32x32 MFMA instructions
 * (fp32 32x32x2 or bf16 32x32x16) on every compute unit and returns the
 * sustained dense TFLOP/s; fold_probe_copy copies `bytes` (a multiple of 16,
 * both buffers 16-byte aligned, caller-owned device memory) five times with
 * 16-byte loads and stores and returns read+write GB/s.  Both synchronise
 * `stream`; fold_probe_mfma allocates a small output buffer.
 * fold_probe_mfma_random is the same loop with random operand bits (four
 * registers a side per lane, uniform in [-1, 1), cycled over the
 * accumulators): the matrix cores' power draw, and so the clock the GPU
 * holds, depends on the operand bits, and random data is what the
 * contractions multiply.  FOLD_E_INVALID for a dtype other than FOLD_F32 /
 * FOLD_BF16 or a NULL result pointer. */
int32_t fold_probe_mfma(int32_t dtype, hipStream_t stream, double* tflops);
int32_t fold_probe_mfma_random(int32_t dtype, hipStream_t stream, double* tflops);
int32_t fold_probe_copy(void* dst, const void* src, size_t bytes, hipStream_t stream, double* gbs);

/* Text of the last error on the calling thread ("" if none). */
const char* fold_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* FOLD_H_ */
