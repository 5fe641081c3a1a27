// Internal declarations shared by the HIP translation units of librgcn (not installed).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "rgcn.h"

namespace rgcn {

// ------------------------------------------------------------------------------------
// Element helpers
// ------------------------------------------------------------------------------------
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two fp32 values -> packed bf16 pair (low half = lo), round to nearest even; one
// v_cvt_pk_bf16_f32 on gfx950.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    f32x2_t f = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}
// fp32 value rounded to bf16 and widened back to fp32.
__device__ __forceinline__ float round_bf16(float x) {
    return __uint_as_float(pack_bf16x2(x, 0.f) << 16);
}

// Philox4x64-10 block function (Salmon, Moraes, Dror and Shaw, SC 2011): 10 rounds of
// two 64x64 -> 128-bit products of words 0 and 2 by fixed odd constants, the high halves
// mixed into words 1 and 3 with the key, the key advanced by two Weyl constants between
// rounds.  c: counter in, output out.
__device__ __forceinline__ void philox4x64(uint64_t c[4], uint64_t k0, uint64_t k1) {
    const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
    for (int round = 0; round < 10; ++round) {
        const uint64_t hi0 = __umul64hi(M0, c[0]), lo0 = M0 * c[0];
        const uint64_t hi1 = __umul64hi(M1, c[2]), lo1 = M1 * c[2];
        const uint64_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
        c[0] = n0; c[1] = lo1; c[2] = n2; c[3] = lo0;
        k0 += W0;
        k1 += W1;
    }
}

// Broadcast a 64-bit value from absolute lane `src` of the wave.
__device__ __forceinline__ int64_t shfl64(int64_t v, int src) {
    const int lo = __shfl((int)(uint32_t)v, src, 64);
    const int hi = __shfl((int)(uint32_t)((uint64_t)v >> 32), src, 64);
    return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// Number of set bits of `mask` below the calling lane (wave64).
__device__ __forceinline__ int lanes_below(uint64_t mask) {
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                          __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

// Workgroup index remapped so that consecutive logical ids run on the same XCD.  The
// dispatcher hands workgroup w to XCD (w mod 8); logical id = XCD-major order.
__device__ __forceinline__ int64_t xcd_major_id(int64_t wg, int64_t total) {
    const int64_t nx = 8;
    int64_t per = total / nx, rem = total % nx;
    int64_t x = wg % nx, idx = wg / nx;
    return x < rem ? x * (per + 1) + idx : rem * (per + 1) + (x - rem) * per + idx;
}

// ------------------------------------------------------------------------------------
// Limits and launch-side tables
// ------------------------------------------------------------------------------------
constexpr int kMaxTypes = RGCN_MAX_TYPES;
constexpr int kMaxRels = RGCN_MAX_RELS;
constexpr int kMaxSlots = RGCN_MAX_TYPES + RGCN_MAX_RELS;  // forward slots: self + relations
constexpr int kSchedBuckets = 32;                          // schedule keys 0..31
constexpr int kFwdChunk = 64;   // weight per chunk of the flattened forward stream
constexpr int kFwdClaim = 8;    // most chunks per run a gather group claims at a time
// A backward source row with more transpose edges than this (over all relations leaving
// its type) is summed in pieces of this many edges by several lane groups, then reduced:
// one group walking a hub of tens of thousands of edges alone would set the stage's time.
constexpr int kSplitEdges = 128;
// Words of the workspace's flag area: [0] forward schedule flag, [1 + t] backward schedule
// flag of type t, [kGatherClaimWord] the gather's work counter, [kPieceCountWord + t] the
// number of pieces of type t's split rows.
constexpr int kGatherClaimWord = 32;
constexpr int kPieceCountWord = 48;
// Split rows of one backward type (plan output, read by the transposed sum).
struct SplitRows {
    int32_t *np;        // [n_rows] pieces of row j (0: not split)
    int32_t *base;      // [n_rows] index of row j's first piece (split rows only)
    int2 *pieces;       // [cap] (row, piece number) of each piece
    uint32_t *count;    // pieces written (zero before the plan)
    int64_t cap;
};
// Pieces of a type whose relations leaving it hold nnz edges: a split row of deg > P edges
// has ceil(deg / P) <= deg / P + 1 pieces and there are fewer than nnz / P split rows.
inline int64_t split_piece_cap(int64_t nnz) { return 2 * ((nnz + kSplitEdges - 1) / kSplitEdges) + 1; }

// A forward slot: the self-loop rows of a destination type, or the rows of one relation.
struct FwdSlot {
    int64_t seg_base;        // first segment id of this slot
    const int32_t *indptr;   // NULL: self-loop slot (every row has degree 1)
    const int32_t *indices;
    const int64_t *rows;     // table row of each edge's source, or NULL (resolve indices)
    int32_t src_type;
    int32_t dst_type;
    int32_t col_off;         // element offset of this slot inside a row of Mcat_t
    int32_t pad;
};

// A forward segment in schedule order, as the gather kernel reads it (16 bytes):
//   k0, deg: first edge position and degree in the slot's CSR (self-loop: k0 = row, deg 1)
//   out:     byte offset / 16 of the segment's output in the workspace (40 bits: out_lo
//            and info bits 0-7); slot: info bits 8-15
struct SegDesc {
    int32_t k0;
    int32_t deg;
    uint32_t out_lo;
    uint32_t info;
};

struct TypeInput {           // rgcn_input restated for the device
    const void *base;
    const int64_t *row_ids;
    int64_t ld;
};

// ------------------------------------------------------------------------------------
// Host launchers (each enqueues on `stream`; return hipSuccess or the launch error)
// ------------------------------------------------------------------------------------
// sort.hip
size_t scan_temp_bytes(int64_t n);
hipError_t exclusive_scan_i32(const int32_t *in, int32_t *out, int64_t n, void *temp,
                              hipStream_t s);
size_t bucket_sort_temp_bytes(int64_t n, int nbuckets);
// Forward schedule and segment descriptors in schedule order; mcat_off[t]: byte offset of
// Mcat_t in the workspace, mcat_ld[t]: its row length in elements, es: element size.
// weight[p] = balancing weight of segment p in the flattened forward stream: the rows it
// moves, max(deg, 1) entries read plus one written.  *flag
// (zero on entry) ends nonzero when some segment is heavy and the schedule was sorted;
// keep_order != 0 keeps enumeration order (the flag stays zero, nothing is sorted).
hipError_t fwd_plan(const FwdSlot *slots_host, int nslots, int64_t n_seg, int32_t *order,
                    const int64_t *mcat_off, const int64_t *mcat_ld, int es, SegDesc *desc,
                    int32_t *weight, uint32_t *flag, int keep_order, void *temp,
                    hipStream_t s);
// Flattened forward stream split into chunks of kFwdChunk weight (segments whole): cs has
// nc_max + 2 entries, nc_max = fwd_chunk_bound(n_seg, sum of relation nnz); cs[c] = first
// segment of chunk c, cs[nc_max + 1] = total weight.  temp: fwd_chunks_temp_bytes(n_seg);
// `weight` may lie in temp past that size.
int64_t fwd_chunk_bound(int64_t n_seg, int64_t nnz_total);
size_t fwd_chunks_temp_bytes(int64_t n_seg);
hipError_t fwd_chunks(const int32_t *weight, int64_t n_seg, int64_t nc_max, int32_t *cs,
                      void *temp, hipStream_t s);
// Combined transpose of several relations: one stable sort of all their edges by
// key = koff_r + source row.  ip[key] (key in [0, key_range]) = position of the first edge
// with that key; csd = destination rows in sorted order.  Relation r's transpose is
// ip + koff_r (values are positions in csd).
struct CscRels {
    int32_t count;
    int64_t row_base[kMaxRels];   // prefix over the relations' destination-row counts
    const int32_t *indptr[kMaxRels];
    const int32_t *indices[kMaxRels];
    int64_t koff[kMaxRels];
    int64_t e0[kMaxRels];         // position of the relation's first edge
};
hipError_t csc_build_all(const CscRels &rels, int64_t total_rows, int64_t nnz,
                         int64_t key_range, int32_t *ip, int32_t *csd, void *temp,
                         hipStream_t s);
size_t csc_temp_bytes(int64_t nnz, int64_t key_range);
struct BwdKeyRels {          // relations leaving one source type
    int32_t count;
    const int32_t *csc_indptr[kMaxRels];
};
// *flag (zero on entry) ends nonzero when some row is heavy and the schedule was sorted;
// keep_order != 0 keeps enumeration order.
// Also lists the rows of more than kSplitEdges transpose edges in `split`.
hipError_t bwd_schedule(const BwdKeyRels &rels, int64_t n_rows, int32_t *order, void *temp,
                        uint32_t *flag, int keep_order, const SplitRows &split, hipStream_t s);
hipError_t fill_words(void *dst, const void *src_host, size_t bytes, hipStream_t s);

// aggregate.hip
// claims: one device word, the gather's shared work counter (set by the launch)
hipError_t gather_mean(rgcn_dtype dt, int d_in, const SegDesc *desc, int64_t n_seg,
                       const int32_t *chunk_starts, int64_t nc_max, const FwdSlot *slots_dev,
                       int nslots, const TypeInput *in, char *ws_base, uint32_t *claims,
                       hipStream_t s);

struct TsumRel {
    const int32_t *csc_indptr;
    const int32_t *csc_dst;
    const float *dms;        // dMs of the destination type, already offset to this slot
    int64_t dms_ld;
};
struct TsumArgs {
    const int32_t *order;    // backward schedule of this source type
    int64_t n_rows;          // n_src[s]
    int64_t n_dst;           // n_dst[s]
    const float *self_dms;   // dY_s W_self_s^T rows (NULL if n_dst == 0)
    int64_t self_ld;
    TypeInput in;            // block input of type s (for the ReLU mask and row ids)
    const uint64_t *relu_mask;   // the input's sign bits, [num_rows x mask_ld], or NULL
    int64_t mask_ld;
    int32_t input_relu;
    int32_t ids_unique;
    float *dh;               // [n_src x d_in] or NULL
    int32_t dh_hilo;         // dh rows in the hi/lo form (d_in bf16 high parts, then low)
    float *demb;             // table-shaped or NULL
    float *opt_state;        // Adagrad mode: fp32 [num_rows x d_in] squared-gradient sums, or NULL
    void *opt_table;         // Adagrad mode: the table of `in`, updated in place
    float lr, eps;
    int32_t d_in;
    int32_t nrel;
    // rows split into pieces (see kSplitEdges): per row its piece count and first piece,
    // the piece list and its length, and fp32 partial sums [piece_cap x d_in]
    const int32_t *split_np;
    const int32_t *split_base;
    const int2 *pieces;
    const uint32_t *piece_count;
    int64_t piece_cap;
    float *partial;
    TsumRel rel[kMaxRels];
};
hipError_t transpose_sum(rgcn_dtype dt, const TsumArgs &a, hipStream_t s);
hipError_t sparse_adagrad(rgcn_dtype dt, int64_t n, const int64_t *rows, int64_t num_rows,
                          int32_t d, float *grad, int64_t grad_ld, bool clear_grad,
                          float *state, void *table, int64_t ld, float lr, float eps,
                          hipStream_t s);

// sample.hip: one layer's neighbour sampling and block construction (tables in the
// workspace; see the file for the method)
constexpr int kMaxFanout = 64;
struct SampleTab {
    int32_t ntypes, nrel, fanout, layer;
    uint64_t seed;
    int64_t n_seg, cap_total;
    int64_t num_nodes[kMaxTypes], n_dst[kMaxTypes], type_base[kMaxTypes], type_cap[kMaxTypes];
    int64_t node_base[kMaxTypes];   // prefix of num_nodes (the per-node first-position words)
    const int64_t *dst_ids[kMaxTypes];
    int64_t *out_src_ids[kMaxTypes];
    int32_t src_type[kMaxRels], dst_type[kMaxRels];
    int64_t seg_base[kMaxRels], cand_base[kMaxRels];
    const int64_t *g_indptr[kMaxRels];
    const int64_t *g_indices[kMaxRels];
    int32_t *out_indptr[kMaxRels];
    int32_t *out_indices[kMaxRels];
    int64_t *out_src_rows[kMaxRels];   // global source id per sampled edge, or NULL
};
struct SampleLayout {
    size_t off_err, off_tab, off_seg, off_scan, off_cand, off_flag, off_first, total;
    int64_t nodes;
};
// Fills the derived fields of T (segments, candidate regions) and the workspace layout;
// false when positions would not fit int32.
bool sample_layout(SampleTab &T, SampleLayout &L);
// Error word bits (at ws + L.off_err): 1 destination id out of range, 2 repeated
// destination ids, 4 in-degree of 2^32 or more, 8 graph source id out of range.
hipError_t sample_block(const SampleTab &T, const SampleLayout &L, char *ws, int64_t *counts,
                        hipStream_t s);

// lp.hip: link-prediction decoder (see the file for the passes)
struct LpArgs {
    rgcn_dtype dtype;
    int32_t d;
    int64_t ld, n_rows;
    const void *emb;
    const void *rel;          // [d] (DistMult) or NULL (dot product)
    int32_t neg_mode, loss;
    int64_t batch, k, nn;     // nn: negatives per positive
    const int32_t *src, *dst, *neg;
    const float *pos_weight;
};
struct LpLayout {
    size_t off_pos, off_gpos, off_lossp, off_S, off_G, off_U, off_P, off_dU, off_Hn, off_dHn,
        off_colsum, off_err, total;
};
LpLayout lp_layout(const LpArgs &a);
hipError_t lp_loss(const LpArgs &a, const LpLayout &L, char *ws, float *loss, float *pos_score,
                   float *neg_score, float *d_emb, float *d_rel, hipStream_t s);
// error bit 1 at *err when a row is outside [0, n_rows)
hipError_t lp_validate(const LpArgs &a, uint32_t *err, hipStream_t s);
hipError_t lp_negatives(int32_t neg_mode, int64_t slots, int64_t num_nodes, uint64_t seed,
                        int64_t *out, hipStream_t s);

// feature.hip: mean of the featured in-neighbours of every node of a featureless type
struct FeatRel {
    const int64_t *indptr;    // [num_nodes + 1]
    const int64_t *indices;   // global rows of the source feature table
    const void *feat;         // [rows x ld] in the dtype
    int64_t rows, ld;
};
struct FeatArgs {
    FeatRel rel[kMaxRels];
    int32_t nrel, d;
    int64_t num_nodes, out_ld;
    void *out;
    rgcn_dtype dtype;
};
// words: two device words (the work counter and the error word: bit 1 = an index out of
// range, skipped)
hipError_t featureless_mean(const FeatArgs &a, uint32_t *words, hipStream_t s);

hipError_t pack_weights(rgcn_dtype dt, int d_in, int d_out, const void *const *w_slots,
                        int nslots, void *wcat_t, hipStream_t s);
// hilo: dy rows in the hi/lo form (cols bf16 high parts, then cols low parts)
hipError_t column_sums(const float *dy, bool hilo, int64_t rows, int cols, float *out,
                       float *partial, int64_t max_splits, hipStream_t s);
size_t column_sums_temp_bytes(int64_t rows, int cols);
hipError_t validate_csr(const int32_t *indptr, const int32_t *indices, int64_t n_dst,
                        int64_t nnz, int64_t n_src, uint32_t *err, hipStream_t s);
hipError_t validate_ids(const int64_t *ids, int64_t n, int64_t num_rows, uint32_t *err,
                        hipStream_t s);
hipError_t validate_src_rows(const int32_t *indices, const int64_t *rows, int64_t nnz,
                             int64_t n_src, const int64_t *ids, int64_t num_rows, uint32_t *err,
                             hipStream_t s);

// gemm.hip
// Forward: Y = A W + bias (opt. ReLU); A [M x K] row-major (ld K), wcat_t [N x K].
// mask (or NULL): the positive bits of the stored Y, [M x ceil(N / 64)] words.
hipError_t gemm_forward(rgcn_dtype dt, const void *a, int64_t M, int N, int K,
                        const void *wcat_t, const void *bias, int relu, void *y,
                        uint64_t *mask, hipStream_t s);
// Backward input side: C[m][n] = (sum_k dy[m][k] W_slot(n)[c(n)][k]) / deg_slot(n)(m);
// slot(n) = n / d_in, c(n) = n % d_in; indptr[slot] NULL: no scaling (self-loop slot).
struct DmsSlots {
    int32_t count;
    const void *w[kMaxSlots];
    const int32_t *indptr[kMaxSlots];
};
// wpack: device space for N x d_out block-dtype values (the input side's weight rows,
// packed when dy is in the hi/lo form), or NULL
hipError_t gemm_dms(rgcn_dtype dt, const float *dy, bool dy_hilo, int64_t M, int d_out,
                    int d_in, const DmsSlots &slots, float *dms, void *wpack, hipStream_t s);
// Weight side: dWcat[kc][o] = sum_i Mcat[i][kc] dy[i][o], K = rows of Mcat.
size_t gemm_dw_partial_bytes(int64_t M, int Kcat, int d_out);
struct DwOut {
    int32_t count;            // slots
    float *w[kMaxSlots];      // destination of slot s ([d_in x d_out]) or NULL
};
// dy_hilo (bf16): dy rows in the hi/lo form (d_out bf16 high parts, then d_out low parts)
hipError_t gemm_dw(rgcn_dtype dt, const void *mcat, int64_t M, int Kcat, int d_in,
                   const float *dy, bool dy_hilo, int d_out, const DwOut &out, float *partial,
                   hipStream_t s);

}  // namespace rgcn

#define RGCN_HIP_TRY(expr)                         \
    do {                                           \
        hipError_t _e = (expr);                    \
        if (_e != hipSuccess) return _e;           \
    } while (0)
