/*
 * rgcn.h -- C ABI of the MI355X (gfx950) relational graph-convolution block library.
 *
 * One call computes one GNN layer on one sampled mini-batch block, the unit the paper's
 * models iterate over (programming-interface appendix, customised-model figure: one
 * layer applied per block, node representations kept per node type).  The layer is the
 * relational GCN the paper lists for heterogeneous graphs (Sec. 3.1.4, model zoo):
 *
 *   M_r[i]  = mean of H_{src(r)}[indices_r[k]] over the sampled in-edges k of row i
 *             (0 when row i has no in-edge in relation r; repeated edges count)
 *   Y_t[i]  = H_t[i] W_self_t + sum_{r : dst(r) = t} M_r[i] W_r (+ b_t)
 *
 * where the destination rows of type t are the first n_dst[t] source rows of type t.
 * At the first layer H_t[j] is row row_ids_t[j] of a feature table or of a learnable
 * embedding table (featureless node types, Sec. 3.3.2); backward then scatter-adds the
 * input gradient into a table-shaped gradient buffer.
 *
 * Conventions (all entry points):
 *  - Pointers marked [host] are host memory; every other pointer is device memory.
 *  - The library allocates no device memory.  The caller owns every buffer, including
 *    the workspace, whose size comes from rgcn_block_workspace_size().  Forward leaves
 *    the per-relation aggregates there for backward, so plan, forward and backward of a
 *    block use the same workspace, in that order, on the same stream.
 *  - Calls enqueue work on `stream` and return without synchronising, except with
 *    RGCN_VALIDATE_DEVICE, which synchronises to report index/CSR errors.
 *  - Device arrays must be 16-byte aligned; d_in and d_out must be multiples of 8
 *    (bf16) or 4 (fp32); ld a multiple of the same; row counts and nnz below 2^31.
 *  - Functions are stateless and thread-safe.  On any non-OK status nothing has been
 *    enqueued (host-detected errors) or the stream has been synchronised (device
 *    validation); rgcn_last_error() returns a message for the calling thread.
 */
#ifndef RGCN_H
#define RGCN_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    RGCN_OK = 0,
    RGCN_ERR_INVALID_ARG = 1,          /* NULL required pointer, bad count, misalignment */
    RGCN_ERR_SHAPE = 2,                /* inconsistent sizes (n_dst > n_src, ld < d_in, ...) */
    RGCN_ERR_DTYPE = 3,                /* unknown dtype */
    RGCN_ERR_INDEX_OOB = 4,            /* device validation: index or row id out of range */
    RGCN_ERR_BAD_CSR = 5,              /* device validation: indptr not a valid CSR offset array */
    RGCN_ERR_WORKSPACE_TOO_SMALL = 6,
    RGCN_ERR_UNSUPPORTED = 7,          /* valid request outside the implemented limits */
    RGCN_ERR_HIP = 8                   /* a HIP runtime call failed */
} rgcn_status;

typedef enum { RGCN_F32 = 0, RGCN_BF16 = 1 } rgcn_dtype;

#define RGCN_MAX_TYPES 16
#define RGCN_MAX_RELS 64

/* flags */
#define RGCN_VALIDATE_DEVICE 0x1u /* check CSR and indices on the device first (synchronises) */
#define RGCN_FUSE_RELU       0x2u /* forward: y = max(0, .) (block followed by ReLU) */
#define RGCN_INPUT_RELU      0x4u /* backward: the input H is a ReLU output, so the input
                                     gradient is multiplied elementwise by [H > 0] */
#define RGCN_IDS_UNIQUE      0x8u /* backward: the caller asserts row_ids are distinct per
                                     type, so demb rows are updated without atomics */
#define RGCN_CLEAR_GRAD      0x10u /* rgcn_sparse_adagrad: zero the gradient rows it read */
#define RGCN_PLAN_FORWARD    0x20u /* rgcn_block_plan: only the part the forward stages read */
#define RGCN_PLAN_BACKWARD   0x40u /* rgcn_block_plan: only the part only the backward reads */
#define RGCN_PLAN_ENUMERATION_ORDER 0x80u /* rgcn_block_plan: keep both schedules in
                                     enumeration order (no degree sort); every result is
                                     bit-identical, only the processing order changes */
#define RGCN_DY_HILO         0x100u /* backward (dense part), bf16: dy[t] is given in the
                                     hi/lo form below instead of fp32 */
#define RGCN_DH_HILO         0x200u /* backward (sparse part), bf16: dh_src[t] is written in
                                     the hi/lo form below instead of fp32 */
/* The hi/lo form of an fp32 gradient row of d values: d bf16 high parts followed by d bf16
 * low parts, hi = x rounded to bf16 (nearest even), lo = (x - hi) rounded to bf16; the same
 * 4 d bytes per row as fp32.  The bf16 backward products take dY as exactly this pair of
 * bf16 operands (16 significant bits); a block's dh_src written in this form is the next
 * (lower) block's dy, read without splitting it again: the weight and input gradients are
 * bit for bit those of the fp32 row, and the bias gradient is the column sum of hi + lo
 * (which differs from x by at most 2^-16 |x|).  Either flag with the fp32 dtype returns
 * RGCN_ERR_UNSUPPORTED. */

/* One relation (canonical edge type src_type -> dst_type) of a block, as a CSR over the
 * destination rows.  indptr[0] = 0, non-decreasing, indptr[n_dst] = nnz; indices are
 * block-local source rows in [0, n_src[src_type]); repeats allowed.
 * src_rows (optional, NULL = not given): the input-table row of each edge's source,
 * src_rows[k] = in[src_type].row_ids[indices[k]] (indices[k] when the input has no row
 * ids), as a sampler that drew the edges from the graph already holds it (the global id
 * of each sampled in-edge's source, before relabelling).  When given, the forward gather
 * reads each edge's table row from it instead of resolving indices[k] through row_ids,
 * which spares a dependent random 8-byte read per edge.  The caller guarantees the
 * equality; RGCN_VALIDATE_DEVICE checks it (RGCN_ERR_INDEX_OOB otherwise).  Everything
 * else (the transpose, the backward, the embedding scatter) uses indices and row_ids. */
typedef struct {
    int32_t src_type;
    int32_t dst_type;
    int64_t nnz;
    const int32_t *indptr;    /* [n_dst[dst_type] + 1] */
    const int32_t *indices;   /* [nnz] */
    const int64_t *src_rows;  /* [nnz] or NULL */
} rgcn_relation;

/* A block: node-type counts and relations.  grad_src_types has bit t set when backward
 * may be asked for dh_src[t] or demb[t]; plan builds the transpose only for those. */
typedef struct {
    int32_t num_types;
    int32_t num_rels;
    const int64_t *n_src;           /* [host][num_types] */
    const int64_t *n_dst;           /* [host][num_types], n_dst[t] <= n_src[t] */
    const rgcn_relation *rels;      /* [host][num_rels] */
    uint32_t grad_src_types;
} rgcn_block;

/* Input rows of one node type: H[j] = base[row_ids[j] * ld + 0 .. d_in) (row_ids NULL:
 * H[j] = base[j * ld ...]).  base has num_rows rows of the block's dtype.
 * relu_mask (optional, read only by the backward under RGCN_INPUT_RELU): the signs of
 * the input as bits, [num_rows x ceil(d_in / 64)] uint64 words, 8-byte aligned, row r's
 * words at relu_mask + r * ceil(d_in / 64), bit c % 64 of word c / 64 set exactly when
 * element c of table row r is positive (rows addressed like base).  The forward of the
 * block that produced the input writes it (rgcn_block_forward's relu_mask); with it the
 * backward reads 1 bit per element instead of the input row.  NULL: the input rows are
 * read. */
typedef struct {
    const void *base;
    const int64_t *row_ids;   /* [n_src[t]] or NULL */
    int64_t num_rows;
    int64_t ld;
    const uint64_t *relu_mask;   /* or NULL */
} rgcn_input;

/* Weights of one block in the block's dtype, row-major [d_in x d_out]. */
typedef struct {
    rgcn_dtype dtype;
    int32_t d_in;
    int32_t d_out;
    const void *const *w_rel;     /* [host][num_rels] */
    const void *const *w_self;    /* [host][num_types]; needed for types with n_dst > 0 */
    const void *const *bias;      /* [host][num_types] entries may be NULL; or NULL = none */
} rgcn_params;

/* Byte offsets inside the workspace of the integer plan (for inspection and tests).
 * An offset of SIZE_MAX means "not built". */
typedef struct {
    int64_t n_fwd_segments;                 /* forward segments (self-loop + relation rows) */
    size_t fwd_order;                       /* int32 [n_fwd_segments]: segment ids in processing
                                               order (a permutation; see rgcn_block_plan) */
    int64_t n_bwd_rows;                     /* source rows of the types in grad_src_types */
    size_t bwd_order;                       /* int32 [n_bwd_rows] */
    size_t csc_indptr[RGCN_MAX_RELS];       /* int32 [n_src[src_type] + 1]: csc_indptr[j+1] -
                                               csc_indptr[j] = in-degree of source row j;
                                               values are offset by csc_indptr[0] */
    size_t csc_dst[RGCN_MAX_RELS];          /* int32 [nnz]: destination row of each edge, edges
                                               of source row j at csc_indptr[j] - csc_indptr[0] */
    size_t total_bytes;                     /* = rgcn_block_workspace_size */
} rgcn_plan_layout;

/* Workspace bytes needed by plan/forward/backward of this block and parameter shape.
 * Host only; enqueues nothing. */
rgcn_status rgcn_block_workspace_size(const rgcn_block *block, const rgcn_params *params,
                                      size_t *bytes /* [host] */);

/* Where the plan arrays sit inside the workspace.  Host only. */
rgcn_status rgcn_block_plan_layout(const rgcn_block *block, const rgcn_params *params,
                                   rgcn_plan_layout *layout /* [host] */);

/* Integer plan of a block (exact, deterministic):
 *  - for every relation whose source type is in grad_src_types, the CSC transpose:
 *    csc_indptr and csc_dst, a stable sort of edges by source row (ascending edge
 *    position inside a source row) -- the transposed adjacency the backward of the
 *    segmented mean runs over;
 *  - two schedules, the order in which the kernels visit work items.  They are library
 *    policy for load balance, not part of the method: no passage of the paper defines
 *    them, every order gives the same results bit for bit, and RGCN_PLAN_ENUMERATION_ORDER
 *    keeps both in enumeration order.  The forward schedule is a permutation of the
 *    forward segments, enumerated type by type (ascending): the type's self-loop rows,
 *    then each relation into the type (ascending relation index), rows ascending.  The
 *    backward schedule holds, for each type in grad_src_types (ascending), a section that
 *    is a permutation of that type's rows (local ids).  The key of an item of degree d
 *    (a segment's edge count; for a backward row, its in-degree in the transpose summed
 *    over the relations leaving the type) is 31 for d <= 32 and max(0, 30 - (floor(log2 d)
 *    - 5)) above; a schedule is the stable sort by ascending key, so items of more than 32
 *    edges come first, the heaviest power of two first, and every lighter item keeps its
 *    enumeration order.
 * Only structural arrays are read.  flags: RGCN_VALIDATE_DEVICE, RGCN_PLAN_FORWARD,
 * RGCN_PLAN_BACKWARD, RGCN_PLAN_ENUMERATION_ORDER.  With neither (or both) of
 * RGCN_PLAN_FORWARD and RGCN_PLAN_BACKWARD the whole plan is built.
 * RGCN_PLAN_FORWARD builds the slot table and the forward schedule, all that
 * rgcn_block_aggregate / rgcn_block_transform read; RGCN_PLAN_BACKWARD builds the CSC
 * transpose and the backward schedule.  The two parts share the workspace's temporary
 * region, so the backward part must be ordered after the forward part (same stream, or an
 * event); the forward stages do not touch that region or anything the backward part
 * writes, so the backward part may run on another stream while they run.  The backward
 * stages need both parts complete. */
rgcn_status rgcn_block_plan(const rgcn_block *block, const rgcn_params *params,
                            void *workspace, size_t workspace_bytes, unsigned flags,
                            hipStream_t stream);

/* Forward: y[t] (device [n_dst[t] x d_out], block dtype, row-major) for every type with
 * n_dst[t] > 0; entries for other types are ignored.  in: [host][num_types].
 * relu_mask ([host][num_types] or NULL; entries may be NULL): with RGCN_FUSE_RELU,
 * relu_mask[t] receives the signs of y[t] as bits, [n_dst[t] x ceil(d_out / 64)] uint64
 * words, 8-byte aligned, bit c % 64 of word c / 64 of row i set exactly when the stored
 * y[t][i][c] is positive (bits past d_out zero) -- the relu_mask of rgcn_input for the
 * next block's backward.  A non-NULL entry without RGCN_FUSE_RELU is an error.
 * flags: RGCN_VALIDATE_DEVICE, RGCN_FUSE_RELU.  Requires rgcn_block_plan first. */
rgcn_status rgcn_block_forward(const rgcn_block *block, const rgcn_input *in,
                               const rgcn_params *params, void *const *y /* [host] */,
                               uint64_t *const *relu_mask /* [host] or NULL */,
                               void *workspace, size_t workspace_bytes, unsigned flags,
                               hipStream_t stream);

/* Backward, after forward on the same workspace.  dy[t]: fp32 [n_dst[t] x d_out].
 * Outputs are fp32 and overwritten unless stated; any array argument may be NULL and any
 * entry NULL to skip that output:
 *   dw_rel[r], dw_self[t]: [d_in x d_out];  dbias[t]: [d_out];
 *   dh_src[t]: [n_src[t] x d_in] gradient w.r.t. the block input H_t;
 *   demb[t]:   [num_rows x d_in] table-shaped; row row_ids[j] += dH_t[j] (scatter-ADD into
 *              caller-initialised memory; rows never named are untouched).
 * dh_src[t] / demb[t] require bit t of grad_src_types.  dw_self entries must not alias.
 * flags: RGCN_VALIDATE_DEVICE, RGCN_INPUT_RELU, RGCN_IDS_UNIQUE, and in bf16 RGCN_DY_HILO
 * (dy in the hi/lo form) and RGCN_DH_HILO (dh_src written in the hi/lo form). */
rgcn_status rgcn_block_backward(const rgcn_block *block, const rgcn_input *in,
                                const rgcn_params *params, const float *const *dy,
                                float *const *dw_rel, float *const *dw_self,
                                float *const *dbias, float *const *dh_src,
                                float *const *demb, void *workspace, size_t workspace_bytes,
                                unsigned flags, hipStream_t stream);

/* The two stages of rgcn_block_forward, for callers that schedule or time them apart.
 * rgcn_block_aggregate: the input gather and per-relation segmented means (self-loop
 *   rows copied, relation rows averaged over their sampled in-edges) into the workspace.
 *   flags: RGCN_VALIDATE_DEVICE.  Requires rgcn_block_plan first.
 * rgcn_block_transform: the per-destination-type transform
 *   Y_t = [H_t | M_r ...] [W_self_t; W_r ...] (+ b_t) on the matrix cores, reading the
 *   aggregates left by rgcn_block_aggregate; relu_mask as in rgcn_block_forward.
 *   flags: RGCN_FUSE_RELU. */
rgcn_status rgcn_block_aggregate(const rgcn_block *block, const rgcn_input *in,
                                 const rgcn_params *params, void *workspace,
                                 size_t workspace_bytes, unsigned flags, hipStream_t stream);
rgcn_status rgcn_block_transform(const rgcn_block *block, const rgcn_params *params,
                                 void *const *y /* [host] */,
                                 uint64_t *const *relu_mask /* [host] or NULL */,
                                 void *workspace, size_t workspace_bytes, unsigned flags,
                                 hipStream_t stream);

/* The two stages of rgcn_block_backward.
 * rgcn_block_backward_dense: weight and bias gradients (dw_rel, dw_self, dbias as in
 *   rgcn_block_backward) and, for the types in grad_src_types, the per-edge input-side
 *   products dY_t W^T / deg kept in the workspace.  flags: RGCN_DY_HILO (bf16).
 * rgcn_block_backward_sparse: the transposed sums over the CSC transpose that turn those
 *   products into dh_src[t] and the scatter-add into demb[t] (as in rgcn_block_backward);
 *   must follow rgcn_block_backward_dense on the same workspace.
 *   flags: RGCN_VALIDATE_DEVICE, RGCN_INPUT_RELU, RGCN_IDS_UNIQUE, RGCN_DH_HILO (bf16). */
rgcn_status rgcn_block_backward_dense(const rgcn_block *block, const rgcn_params *params,
                                      const float *const *dy, float *const *dw_rel,
                                      float *const *dw_self, float *const *dbias,
                                      void *workspace, size_t workspace_bytes, unsigned flags,
                                      hipStream_t stream);
rgcn_status rgcn_block_backward_sparse(const rgcn_block *block, const rgcn_input *in,
                                       const rgcn_params *params, float *const *dh_src,
                                       float *const *demb, void *workspace,
                                       size_t workspace_bytes, unsigned flags,
                                       hipStream_t stream);

/* Sparse Adagrad step of learnable embedding tables (Sec. 3.3.2: the trainable rows of a
 * featureless node type change only where a mini-batch used them; the paper does not
 * name the optimizer, and the rule taken here is row-wise Adagrad with no decay):
 *   state[r] += g[r]^2  (elementwise);   table[r] -= lr * g[r] / (sqrt(state[r]) + eps)
 * computed in fp32; a bf16 table row is rounded to nearest even after the step. */
typedef struct {
    float lr;
    float eps;
    float *const *state;   /* [host][num_types]; entry t NULL, or fp32 [in[t].num_rows x d_in]
                              row-major (ld = d_in), updated in place */
    void *const *table;    /* [host][num_types]; for every t with state[t]: the writable
                              table of in[t] (must equal in[t].base), updated in place */
} rgcn_adagrad;

/* rgcn_block_backward_sparse with the optimizer step fused into the transposed sum: for
 * every type t with opt->state[t] set, the input gradient row dH_t[j] is applied at once to
 * table row row_ids[j] (row j when row_ids is NULL) instead of being scatter-added.  The
 * other types behave as in rgcn_block_backward_sparse (dh_src / demb).  Requires
 * RGCN_IDS_UNIQUE (each table row then takes exactly one step; repeated ids would race),
 * and, for the optimised types, bit t of grad_src_types, demb[t] NULL, a 16-byte aligned
 * state and no RGCN_INPUT_RELU (a learnable table is not a ReLU output).  dh_src[t] may
 * still be requested and is the gradient before the step.
 * flags: RGCN_VALIDATE_DEVICE, RGCN_IDS_UNIQUE (required). */
rgcn_status rgcn_block_backward_sparse_adagrad(const rgcn_block *block, const rgcn_input *in,
                                               const rgcn_params *params,
                                               float *const *dh_src, float *const *demb,
                                               const rgcn_adagrad *opt /* [host] */,
                                               void *workspace, size_t workspace_bytes,
                                               unsigned flags, hipStream_t stream);

/* The same Adagrad step as a pass of its own, for gradients gathered in a table-shaped
 * buffer first (e.g. demb from rgcn_block_backward_sparse when ids repeat).  For each of
 * the n listed rows r = rows[i]: grad row r (fp32 [num_rows x d], ld = d) and state row r
 * (fp32 [num_rows x d]) are read, state and table row r (dtype, [num_rows x ld]) updated in
 * place.  rows must be distinct (repeats race: any mix of the updates may result; no
 * fault); rows outside [0, num_rows) are skipped, never read or written.  d a multiple of
 * 8 (bf16) or 4 (fp32), ld >= d and a multiple of the same; all arrays 16-byte aligned.
 * flags: RGCN_CLEAR_GRAD zeroes each grad row after reading it, leaving the buffer ready
 * for the next scatter-add without a full clear. */
rgcn_status rgcn_sparse_adagrad(int64_t n, const int64_t *rows, int64_t num_rows, int32_t d,
                                float *grad, float *state, void *table, int64_t ld,
                                rgcn_dtype dtype, float lr, float eps, unsigned flags,
                                hipStream_t stream);

/* ---------------------------------------------------------------- neighbour sampling
 * One layer of on-the-fly mini-batch sampling (Sec. 3.1.1 and 3.1.4: neighbourhoods are
 * sampled per mini-batch with a fanout per layer, one block per GNN layer, top-down from
 * the seeds).  The paper leaves the sampler unspecified; the rule implemented:
 *  - for each destination node v of type dst(r) and each relation r: every in-edge of v
 *    in r when its in-degree is at most `fanout`, else `fanout` distinct in-edges, each
 *    subset equally likely (Floyd's algorithm), listed in the graph's CSR order;
 *  - draw k of (v, r) is word k mod 4 of Philox4x64-10 at counter (v, r, k/4, 0) and key
 *    (seed, layer); a uniform integer in [0, m) is the high word of draw * m (results
 *    are a function of the inputs, bit for bit);
 *  - the block's source nodes of type t are its destination nodes (in the given order),
 *    then the sampled sources in order of first appearance (relations in order,
 *    destination rows in order, edges in order); indices are those block-local rows.
 * The output is a block in the form rgcn_block expects (its source ids are the next
 * layer's destination ids, and at the input layer the row ids of the tables). */
typedef struct {
    int32_t src_type;
    int32_t dst_type;
    const int64_t *indptr;    /* [num_nodes[dst_type] + 1] in-edge CSR offsets */
    const int64_t *indices;   /* [indptr[num_nodes[dst_type]]] global source ids */
} rgcn_graph_relation;

typedef struct {
    int32_t num_types;                /* 1 .. RGCN_MAX_TYPES */
    int32_t num_rels;                 /* 0 .. RGCN_MAX_RELS */
    const int64_t *num_nodes;         /* [host][num_types], each below 2^59 */
    const rgcn_graph_relation *rels;  /* [host][num_rels] */
} rgcn_graph;

#define RGCN_MAX_FANOUT 64

/* Workspace bytes for rgcn_sample_block with these destination counts (host only). */
rgcn_status rgcn_sample_workspace_size(const rgcn_graph *graph,
                                       const int64_t *n_dst /* [host][num_types] */,
                                       int32_t fanout, size_t *bytes /* [host] */);

/* Sample one layer's block for the destination nodes dst_ids[t] (device int64 [n_dst[t]],
 * distinct per type).  fanout in [1, RGCN_MAX_FANOUT].  Outputs (device, caller-owned,
 * overwritten):
 *   out_indptr[r]:  int32 [n_dst[dst(r)] + 1]
 *   out_indices[r]: int32, capacity n_dst[dst(r)] * fanout (block-local source rows)
 *   out_src_ids[t]: int64, capacity n_dst[t] + sum over r with src(r) = t of
 *                   n_dst[dst(r)] * fanout (global ids of the block's source nodes)
 *   out_src_rows:   NULL, or per relation NULL or int64 with the capacity of
 *                   out_indices[r]: the global id of each sampled edge's source, in edge
 *                   order (out_src_ids[src(r)][out_indices[r][k]]; at the input layer the
 *                   rgcn_relation.src_rows of the block)
 *   counts:         int64 [num_rels + num_types]: sampled edges per relation, then source
 *                   nodes per type (read it after the stream completes to size the block)
 * Entries for relations or types whose capacity is zero may be NULL.  Capacities must
 * stay below 2^31 in total (RGCN_ERR_UNSUPPORTED otherwise).  Invalid device data (an id
 * out of range, repeated destination ids, an in-degree of 2^32 or more) is never read
 * out of bounds; it leaves the outputs unspecified and is reported only with
 * RGCN_VALIDATE_DEVICE, which synchronises after the work: RGCN_ERR_INDEX_OOB (an id out
 * of range), RGCN_ERR_INVALID_ARG (repeated destination ids), RGCN_ERR_UNSUPPORTED
 * (degree).  flags: RGCN_VALIDATE_DEVICE. */
rgcn_status rgcn_sample_block(const rgcn_graph *graph, const int64_t *const *dst_ids /* [host] */,
                              const int64_t *n_dst /* [host] */, int32_t fanout, uint64_t seed,
                              int32_t layer, int32_t *const *out_indptr /* [host] */,
                              int32_t *const *out_indices /* [host] */,
                              int64_t *const *out_src_ids /* [host] */,
                              int64_t *const *out_src_rows /* [host] or NULL */, int64_t *counts,
                              void *workspace, size_t workspace_bytes, unsigned flags,
                              hipStream_t stream);

/* ---------------------------------------------------------------- link prediction
 * The link-prediction decoder of the paper's appendix on score and loss functions,
 * applied to a batch of B positive edges (src_i, dst_i), rows of the GNN's output
 * embedding matrix, and their negatives, which keep src_i and replace dst_i:
 *   scores:    dot product sum_c h_u[c] h_v[c], or DistMult sum_c h_u[c] r[c] h_v[c] with r
 *              the edge type's embedding (the printed dot product reuses the node index
 *              as the summation index: the sum runs over the embedding dimension);
 *   negatives: RGCN_LP_NEG_PER_EDGE (uniform): K rows per positive, neg[i*K + k];
 *              RGCN_LP_NEG_JOINT: positives i of group g = i / K share neg[g*K + k];
 *              RGCN_LP_NEG_IN_BATCH: the destinations of the other positives, dst_j for
 *              j != i in ascending j (B - 1 negatives), as in the appendix's example;
 *   losses:    RGCN_LP_CE: binary cross entropy on sigmoid(score), label 1 for positives
 *              and 0 for negatives, averaged over all B (1 + K) scored edges (the printed
 *              formula misplaces a sign and a bracket);
 *              RGCN_LP_WEIGHTED_CE: the same with weight pos_weight[i] on positive i and
 *              1 on negatives;
 *              RGCN_LP_CONTRASTIVE: per positive, -log(exp(s_pos) / (exp(s_pos) +
 *              sum_k exp(s_k))) (the positive is in the denominator), averaged over B. */
typedef enum { RGCN_LP_NEG_PER_EDGE = 0, RGCN_LP_NEG_JOINT = 1, RGCN_LP_NEG_IN_BATCH = 2 } rgcn_lp_neg;
typedef enum { RGCN_LP_CE = 0, RGCN_LP_WEIGHTED_CE = 1, RGCN_LP_CONTRASTIVE = 2 } rgcn_lp_loss_kind;

typedef struct {
    rgcn_dtype dtype;
    int32_t d;                  /* embedding width, a multiple of 8 (bf16) or 4 (fp32), <= 2048 (bf16) / 1024 (fp32) */
    int64_t n_rows;             /* rows of emb */
    int64_t ld;                 /* row stride of emb in elements, >= d, a multiple of 8 / 4 */
    const void *emb;            /* [n_rows x ld] in dtype, 16-byte aligned */
    const void *rel;            /* DistMult: [d] in dtype, 16-byte aligned; NULL: dot product */
    int32_t neg_mode;           /* rgcn_lp_neg */
    int32_t loss;               /* rgcn_lp_loss_kind */
    int64_t batch;              /* B */
    const int32_t *src;         /* [B] rows of emb */
    const int32_t *dst;         /* [B] rows of emb */
    int32_t k;                  /* negatives per positive (per edge, joint); in-batch: ignored */
    const int32_t *neg;         /* per edge: [B x K] rows; joint: [ceil(B / K) x K]; in-batch: NULL */
    const float *pos_weight;    /* weighted CE: [B]; otherwise ignored */
} rgcn_lp_batch;

/* Workspace bytes of rgcn_lp_loss for this batch (host only).  It holds the B x N scores
 * and their derivatives (N = K, or B - 1 in-batch); B x N must stay below 2^31. */
rgcn_status rgcn_lp_workspace_size(const rgcn_lp_batch *batch, size_t *bytes /* [host] */);

/* Loss of one batch, its scores and gradients.  Outputs (device, fp32; NULL skips):
 *   loss:      [1] the averaged loss (overwritten);
 *   pos_score: [B]; neg_score: [B x N] in positive-major order (overwritten);
 *   d_emb:     [n_rows x d], row-major: the gradient of the loss with respect to each
 *              embedding row is ADDED (caller-initialised; rows never used untouched;
 *              fp32 atomics, so the order of additions varies);
 *   d_rel:     [d] the gradient with respect to rel (DistMult; overwritten).
 * Rows outside [0, n_rows) are the caller's error: checked only with RGCN_VALIDATE_DEVICE
 * (before any other work; synchronises; RGCN_ERR_INDEX_OOB).  flags: RGCN_VALIDATE_DEVICE. */
rgcn_status rgcn_lp_loss(const rgcn_lp_batch *batch, float *loss, float *pos_score,
                         float *neg_score, float *d_emb, float *d_rel, void *workspace,
                         size_t workspace_bytes, unsigned flags, hipStream_t stream);

/* rgcn_lp_loss for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same computation
 * and outputs, with no workspace argument.  Its temporaries live in one fixed device
 * array of RGCN_LP_NOALLOC_MAX_SCRATCH bytes inside the library, one per device, held
 * until the process ends; the call allocates nothing and calls no allocating routine.
 * A batch whose temporaries (rgcn_lp_workspace_size) exceed that size is rejected with
 * RGCN_ERR_UNSUPPORTED before anything is enqueued.  Every call on a device shares that
 * device's array: calls that overlap on one device (two streams, two threads) race and
 * give unspecified results; calls ordered on one stream are safe, and each call
 * initialises every temporary it reads, whatever the previous call left.
 * flags: RGCN_VALIDATE_DEVICE. */
#define RGCN_LP_NOALLOC_MAX_SCRATCH 33554432u /* 32 MiB */
rgcn_status rgcn_lp_loss_noalloc(const rgcn_lp_batch *batch, float *loss, float *pos_score,
                                 float *neg_score, float *d_emb, float *d_rel, unsigned flags,
                                 hipStream_t stream);

/* Negative node ids for the per-edge (slots = B * K) or joint (slots = ceil(B / K) * K)
 * modes: slot q is the high word of draw * num_nodes, the draw being word q mod 4 of
 * Philox4x64-10 at counter (q / 4, neg_mode, 0, 0) and key (seed, 0x6e6567); uniform over
 * [0, num_nodes) and a function of the arguments only.  out: device int64 [slots]. */
rgcn_status rgcn_lp_negatives(int32_t neg_mode, int64_t slots, int64_t num_nodes, uint64_t seed,
                              int64_t *out, hipStream_t stream);

/* ---------------------------------------------------------------- featureless nodes
 * Feature construction for a node type without features (Sec. 3.3.2, eq. 1, with f the
 * average): over the whole graph, for every node i of the type,
 *   F'_i = mean of F_{src(r)}[j] over the in-edges (j -> i) of the given relations,
 * each relation's source type having a feature table; an edge listed twice counts twice;
 * F'_i = 0 when i has no such in-edge.  fp32 accumulation; bf16 output rounded to nearest
 * even. */
typedef struct {
    const int64_t *indptr;     /* [num_nodes + 1] in-edge CSR over the featureless type */
    const int64_t *indices;    /* [indptr[num_nodes]] rows of `features` */
    const void *features;      /* [rows x ld] source feature table in the dtype, 16-byte aligned */
    int64_t rows;
    int64_t ld;                /* >= d, a multiple of 8 (bf16) or 4 (fp32) */
} rgcn_feature_relation;

#define RGCN_FEATURELESS_WORKSPACE 256   /* bytes of device workspace (a work counter) */

/* out: [num_nodes x out_ld] in dtype (written).  d a multiple of 8 (bf16) or 4 (fp32), at
 * most 2048 / 1024.  rels: [host][num_rels], 1 <= num_rels <= RGCN_MAX_RELS.  workspace:
 * RGCN_FEATURELESS_WORKSPACE bytes, 256-byte aligned.  Neighbour indices outside
 * [0, rows) are skipped (never read); with RGCN_VALIDATE_DEVICE (synchronises after the
 * work) they are reported as RGCN_ERR_INDEX_OOB.  flags: RGCN_VALIDATE_DEVICE. */
rgcn_status rgcn_featureless_mean(int32_t num_rels, const rgcn_feature_relation *rels,
                                  int64_t num_nodes, int32_t d, rgcn_dtype dtype, void *out,
                                  int64_t out_ld, void *workspace, unsigned flags,
                                  hipStream_t stream);

/* Message for the last non-OK status returned on the calling thread ("" if none). */
const char *rgcn_last_error(void);

/* Library version string. */
const char *rgcn_version(void);

#ifdef __cplusplus
}
#endif

#endif /* RGCN_H */
