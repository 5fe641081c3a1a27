// C ABI of librgcn: argument validation, workspace layout and the order of kernel
// launches for plan / forward / backward of one block.  No device memory is allocated
// here; everything lives in the caller's workspace.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <string>

#include "common.h"

using namespace rgcn;

namespace {

thread_local std::string g_err;

rgcn_status fail(rgcn_status st, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return st;
}

rgcn_status hip_fail(hipError_t e, const char *what) {
    return fail(RGCN_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define TRY_HIP(expr, what)                           \
    do {                                              \
        hipError_t _e = (expr);                       \
        if (_e != hipSuccess) return hip_fail(_e, what); \
    } while (0)

// A dtype field of a caller's struct read as the integer it holds: a caller may store any
// value there, and loading a value outside the enumeration as the enum type is undefined.
inline int32_t dtype_code(const rgcn_dtype *p) {
    int32_t v;
    memcpy(&v, p, sizeof(v));
    return v;
}
inline bool dtype_known(const rgcn_dtype *p) {
    const int32_t v = dtype_code(p);
    return v == RGCN_F32 || v == RGCN_BF16;
}

inline size_t align256(size_t x) { return (x + 255) / 256 * 256; }
inline bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }
inline bool aligned4(const void *p) { return ((uintptr_t)p & 3u) == 0; }
constexpr int64_t kI32Max = 2147483647;

// Everything the launches need to know about a block, derived on the host.
struct Layout {
    int T = 0, R = 0, d_in = 0, d_out = 0, es = 0;
    rgcn_dtype dt = RGCN_F32;
    uint32_t grad_mask = 0;
    // forward slots: per destination type with n_dst > 0, self then relations into it
    int nslots = 0;
    FwdSlot slots[kMaxSlots];
    int64_t n_seg = 0;
    int type_slot0[kMaxTypes];          // first slot of type t (-1: no destination rows)
    int type_nslots[kMaxTypes];
    int rel_pos[kMaxRels];              // position of relation r among its type's slots
    int64_t K[kMaxTypes];               // Mcat row length = nslots_t * d_in
    // backward input-side slots (dMs): self if t is a grad type, relations leaving one
    int dms_nslots[kMaxTypes];
    int dms_self[kMaxTypes];            // slot index or -1
    int dms_rel[kMaxRels];              // slot index in dMs_{dst(r)} or -1
    int64_t bwd_base[kMaxTypes];
    int64_t n_bwd_rows = 0;
    // workspace offsets
    size_t off_slots = 0, off_fwd_order = 0, off_fwd_desc = 0, off_bwd_order = 0, off_err = 0;
    size_t off_fwd_chunks = 0;
    size_t off_flags = 0;         // flag words (see kGatherClaimWord, kPieceCountWord)
    // split backward rows: np and base per backward row, the piece list (per type a window
    // of piece_cap[t] pieces from piece_at[t]), partial sums in the backward temporaries
    size_t off_split_np = 0, off_split_base = 0, off_pieces = 0;
    int64_t piece_at[kMaxTypes], piece_cap[kMaxTypes], piece_total = 0;
    size_t off_split_partial = 0;       // relative to scratch
    int64_t nc_max = 0;           // chunk bound of the flattened forward stream
    size_t off_csc_indptr[kMaxRels], off_csc_dst[kMaxRels];
    // combined transpose of the relations leaving grad types
    int64_t koff[kMaxRels], e0[kMaxRels];
    int64_t key_range = 0, csc_nnz = 0, csc_rows = 0;
    size_t off_ip = 0, off_csd = 0;
    size_t off_mcat[kMaxTypes], off_wcat[kMaxTypes];
    size_t off_scratch = 0;
    // scratch (a union: plan temporaries, or backward temporaries)
    size_t plan_temp = 0;
    size_t off_dms[kMaxTypes];          // relative to scratch
    size_t off_partial = 0, off_colsum = 0;
    size_t total = 0;
};

rgcn_status check_block(const rgcn_block *b) {
    if (!b) return fail(RGCN_ERR_INVALID_ARG, "block is NULL");
    if (b->num_types < 1 || b->num_types > kMaxTypes)
        return fail(RGCN_ERR_INVALID_ARG, "num_types %d outside [1, %d]", b->num_types, kMaxTypes);
    if (b->num_rels < 0 || b->num_rels > kMaxRels)
        return fail(RGCN_ERR_INVALID_ARG, "num_rels %d outside [0, %d]", b->num_rels, kMaxRels);
    if (!b->n_src || !b->n_dst) return fail(RGCN_ERR_INVALID_ARG, "n_src / n_dst is NULL");
    if (b->num_rels > 0 && !b->rels) return fail(RGCN_ERR_INVALID_ARG, "rels is NULL");
    if (b->grad_src_types >> b->num_types)
        return fail(RGCN_ERR_INVALID_ARG, "grad_src_types names a type >= num_types");
    for (int t = 0; t < b->num_types; ++t) {
        if (b->n_dst[t] < 0 || b->n_src[t] < b->n_dst[t])
            return fail(RGCN_ERR_SHAPE, "type %d: need 0 <= n_dst (%lld) <= n_src (%lld)", t,
                        (long long)b->n_dst[t], (long long)b->n_src[t]);
        if (b->n_src[t] >= kI32Max)
            return fail(RGCN_ERR_UNSUPPORTED, "type %d: n_src must be below 2^31", t);
    }
    for (int r = 0; r < b->num_rels; ++r) {
        const rgcn_relation &rel = b->rels[r];
        if (rel.src_type < 0 || rel.src_type >= b->num_types || rel.dst_type < 0 ||
            rel.dst_type >= b->num_types)
            return fail(RGCN_ERR_INVALID_ARG, "relation %d: node type out of range", r);
        if (rel.nnz < 0 || rel.nnz >= kI32Max)
            return fail(RGCN_ERR_UNSUPPORTED, "relation %d: nnz must be in [0, 2^31)", r);
        if (!rel.indptr || !aligned4(rel.indptr))
            return fail(RGCN_ERR_INVALID_ARG, "relation %d: indptr NULL or misaligned", r);
        if (rel.nnz > 0 && (!rel.indices || !aligned4(rel.indices)))
            return fail(RGCN_ERR_INVALID_ARG, "relation %d: indices NULL or misaligned", r);
        if (rel.nnz > 0 && b->n_src[rel.src_type] == 0)
            return fail(RGCN_ERR_SHAPE, "relation %d: edges into an empty source type", r);
        if (rel.src_rows && ((uintptr_t)rel.src_rows & 7u))
            return fail(RGCN_ERR_INVALID_ARG, "relation %d: src_rows misaligned", r);
    }
    return RGCN_OK;
}

rgcn_status check_params(const rgcn_block *b, const rgcn_params *p) {
    if (!p) return fail(RGCN_ERR_INVALID_ARG, "params is NULL");
    if (!dtype_known(&p->dtype))
        return fail(RGCN_ERR_DTYPE, "unknown dtype %d", (int)dtype_code(&p->dtype));
    const int vec = p->dtype == RGCN_BF16 ? 8 : 4;
    if (p->d_in <= 0 || p->d_out <= 0)
        return fail(RGCN_ERR_INVALID_ARG, "d_in / d_out must be positive");
    if (p->d_in % vec || p->d_out % vec)
        return fail(RGCN_ERR_UNSUPPORTED, "d_in and d_out must be multiples of %d", vec);
    if (p->d_in > 256 * vec)
        return fail(RGCN_ERR_UNSUPPORTED, "d_in above %d", 256 * vec);
    if (b->num_rels > 0 && !p->w_rel) return fail(RGCN_ERR_INVALID_ARG, "w_rel is NULL");
    for (int r = 0; r < b->num_rels; ++r)
        if (!p->w_rel[r] || !aligned16(p->w_rel[r]))
            return fail(RGCN_ERR_INVALID_ARG, "w_rel[%d] NULL or not 16-byte aligned", r);
    if (!p->w_self) return fail(RGCN_ERR_INVALID_ARG, "w_self is NULL");
    for (int t = 0; t < b->num_types; ++t) {
        if (b->n_dst[t] > 0 && (!p->w_self[t] || !aligned16(p->w_self[t])))
            return fail(RGCN_ERR_INVALID_ARG, "w_self[%d] NULL or not 16-byte aligned", t);
        if (p->bias && p->bias[t] && !aligned16(p->bias[t]))
            return fail(RGCN_ERR_INVALID_ARG, "bias[%d] not 16-byte aligned", t);
    }
    return RGCN_OK;
}

rgcn_status make_layout(const rgcn_block *b, const rgcn_params *p, Layout &L) {
    rgcn_status st = check_block(b);
    if (st != RGCN_OK) return st;
    if ((st = check_params(b, p)) != RGCN_OK) return st;
    L.T = b->num_types;
    L.R = b->num_rels;
    L.d_in = p->d_in;
    L.d_out = p->d_out;
    L.dt = p->dtype;
    L.es = p->dtype == RGCN_BF16 ? 2 : 4;
    L.grad_mask = b->grad_src_types;
    // forward slots
    L.nslots = 0;
    L.n_seg = 0;
    for (int r = 0; r < kMaxRels; ++r) { L.rel_pos[r] = -1; L.dms_rel[r] = -1; }
    for (int t = 0; t < kMaxTypes; ++t) {
        L.type_slot0[t] = -1;
        L.type_nslots[t] = 0;
        L.K[t] = 0;
        L.dms_nslots[t] = 0;
        L.dms_self[t] = -1;
        L.bwd_base[t] = -1;
    }
    for (int t = 0; t < L.T; ++t) {
        const int64_t nd = b->n_dst[t];
        if (nd == 0) continue;
        L.type_slot0[t] = L.nslots;
        FwdSlot self{};
        self.seg_base = L.n_seg;
        self.src_type = t;
        self.dst_type = t;
        self.col_off = 0;
        L.slots[L.nslots++] = self;
        L.n_seg += nd;
        int pos = 1;
        for (int r = 0; r < L.R; ++r) {
            if (b->rels[r].dst_type != t) continue;
            FwdSlot s{};
            s.seg_base = L.n_seg;
            s.indptr = b->rels[r].indptr;
            s.indices = b->rels[r].indices;
            s.rows = b->rels[r].nnz > 0 ? b->rels[r].src_rows : nullptr;
            s.src_type = b->rels[r].src_type;
            s.dst_type = t;
            s.col_off = pos * L.d_in;
            L.rel_pos[r] = pos;
            L.slots[L.nslots++] = s;
            L.n_seg += nd;
            ++pos;
        }
        L.type_nslots[t] = pos;
        L.K[t] = (int64_t)pos * L.d_in;
    }
    if (L.n_seg >= kI32Max) return fail(RGCN_ERR_UNSUPPORTED, "too many forward segments");
    {
        int64_t nnz_total = 0;
        for (int r = 0; r < L.R; ++r)
            if (b->n_dst[b->rels[r].dst_type] > 0) nnz_total += b->rels[r].nnz;
        if (2 * L.n_seg + nnz_total >= kI32Max)
            return fail(RGCN_ERR_UNSUPPORTED, "edges plus twice the forward segments of the block exceed 2^31");
        L.nc_max = fwd_chunk_bound(L.n_seg, nnz_total);
    }
    // backward slots
    for (int t = 0; t < L.T; ++t) {
        if (b->n_dst[t] == 0) continue;
        int n = 0;
        if (L.grad_mask >> t & 1u) L.dms_self[t] = n++;
        for (int r = 0; r < L.R; ++r)
            if (b->rels[r].dst_type == t && (L.grad_mask >> b->rels[r].src_type & 1u))
                L.dms_rel[r] = n++;
        L.dms_nslots[t] = n;
    }
    L.n_bwd_rows = 0;
    for (int t = 0; t < L.T; ++t)
        if (L.grad_mask >> t & 1u) {
            L.bwd_base[t] = L.n_bwd_rows;
            L.n_bwd_rows += b->n_src[t];
        }
    if (L.n_bwd_rows >= kI32Max) return fail(RGCN_ERR_UNSUPPORTED, "too many backward rows");

    // persistent region
    size_t off = 0;
    L.off_err = off;                      off += 256;
    L.off_flags = off;                    off += 256;
    L.off_slots = off;                    off += align256(sizeof(FwdSlot) * kMaxSlots);
    L.off_fwd_order = off;                off += align256((size_t)L.n_seg * 4 + 4);
    L.off_fwd_desc = off;                 off += align256((size_t)L.n_seg * sizeof(SegDesc) + 16);
    L.off_fwd_chunks = off;               off += align256((size_t)(L.nc_max + 2) * 4);
    L.off_bwd_order = off;                off += align256((size_t)L.n_bwd_rows * 4 + 4);
    L.off_split_np = off;                 off += align256((size_t)L.n_bwd_rows * 4 + 4);
    L.off_split_base = off;               off += align256((size_t)L.n_bwd_rows * 4 + 4);
    L.piece_total = 0;
    for (int t = 0; t < kMaxTypes; ++t) L.piece_at[t] = L.piece_cap[t] = 0;
    for (int t = 0; t < L.T; ++t) {
        if (!(L.grad_mask >> t & 1u)) continue;
        int64_t nnz_out = 0;
        for (int r = 0; r < L.R; ++r)
            if (b->rels[r].src_type == t) nnz_out += b->rels[r].nnz;
        L.piece_at[t] = L.piece_total;
        L.piece_cap[t] = split_piece_cap(nnz_out);
        L.piece_total += L.piece_cap[t];
    }
    L.off_pieces = off;                   off += align256((size_t)L.piece_total * 8 + 8);
    for (int r = 0; r < kMaxRels; ++r) {
        L.off_csc_indptr[r] = L.off_csc_dst[r] = SIZE_MAX;
        L.koff[r] = L.e0[r] = -1;
    }
    L.key_range = L.csc_nnz = L.csc_rows = 0;
    for (int r = 0; r < L.R; ++r) {
        const rgcn_relation &rel = b->rels[r];
        if (!(L.grad_mask >> rel.src_type & 1u)) continue;
        L.koff[r] = L.key_range;
        L.e0[r] = L.csc_nnz;
        L.key_range += b->n_src[rel.src_type];
        L.csc_nnz += rel.nnz;
        L.csc_rows += b->n_dst[rel.dst_type];
    }
    if (L.key_range >= kI32Max || L.csc_nnz >= kI32Max)
        return fail(RGCN_ERR_UNSUPPORTED, "transpose of the grad relations exceeds 2^31 entries");
    L.off_ip = off;   off += align256((size_t)(L.key_range + 1) * 4);
    L.off_csd = off;  off += align256((size_t)L.csc_nnz * 4 + 4);
    for (int r = 0; r < L.R; ++r)
        if (L.koff[r] >= 0) {
            L.off_csc_indptr[r] = L.off_ip + 4 * (size_t)L.koff[r];
            L.off_csc_dst[r] = L.off_csd + 4 * (size_t)L.e0[r];
        }
    for (int t = 0; t < kMaxTypes; ++t) L.off_mcat[t] = L.off_wcat[t] = SIZE_MAX;
    for (int t = 0; t < L.T; ++t) {
        if (b->n_dst[t] == 0) continue;
        L.off_mcat[t] = off;  off += align256((size_t)b->n_dst[t] * L.K[t] * L.es);
        L.off_wcat[t] = off;  off += align256((size_t)L.d_out * L.K[t] * L.es);
    }
    L.off_scratch = off;
    // plan temporaries
    size_t pt = bucket_sort_temp_bytes(L.n_seg, kSchedBuckets);
    {
        size_t c = fwd_chunks_temp_bytes(L.n_seg) + align256((size_t)L.n_seg * 4 + 4);
        if (c > pt) pt = c;
    }
    {
        size_t c = csc_temp_bytes(L.csc_nnz, L.key_range);
        if (c > pt) pt = c;
    }
    for (int t = 0; t < L.T; ++t)
        if (L.grad_mask >> t & 1u) {
            size_t c = bucket_sort_temp_bytes(b->n_src[t], kSchedBuckets);
            if (c > pt) pt = c;
        }
    L.plan_temp = align256(pt);
    // backward temporaries
    size_t bt = 0;
    for (int t = 0; t < kMaxTypes; ++t) L.off_dms[t] = SIZE_MAX;
    size_t part = 256, cols = 256;
    for (int t = 0; t < L.T; ++t) {
        if (b->n_dst[t] == 0) continue;
        if (L.dms_nslots[t] > 0) {
            L.off_dms[t] = bt;
            bt += align256((size_t)b->n_dst[t] * L.dms_nslots[t] * L.d_in * 4);
        }
        size_t pb = gemm_dw_partial_bytes(b->n_dst[t], (int)L.K[t], L.d_out);
        if (pb > part) part = pb;
        size_t cb = column_sums_temp_bytes(b->n_dst[t], L.d_out);
        if (cb > cols) cols = cb;
    }
    L.off_partial = bt;   bt += align256(part);
    L.off_colsum = bt;    bt += align256(cols);
    L.off_split_partial = bt;  bt += align256((size_t)L.piece_total * L.d_in * 4 + 16);
    L.total = L.off_scratch + (L.plan_temp > bt ? L.plan_temp : bt);
    return RGCN_OK;
}

rgcn_status check_workspace(const Layout &L, void *ws, size_t bytes) {
    if (!ws) return fail(RGCN_ERR_INVALID_ARG, "workspace is NULL");
    if ((uintptr_t)ws & 255u) return fail(RGCN_ERR_INVALID_ARG, "workspace not 256-byte aligned");
    if (bytes < L.total)
        return fail(RGCN_ERR_WORKSPACE_TOO_SMALL, "workspace %zu bytes, need %zu", bytes, L.total);
    return RGCN_OK;
}

rgcn_status check_inputs(const rgcn_block *b, const rgcn_input *in, const Layout &L,
                         bool need_all_types) {
    if (!in) return fail(RGCN_ERR_INVALID_ARG, "inputs are NULL");
    const int vec = L.dt == RGCN_BF16 ? 8 : 4;
    for (int t = 0; t < L.T; ++t) {
        bool read = b->n_dst[t] > 0 || need_all_types;
        for (int r = 0; r < L.R && !read; ++r)
            read = b->rels[r].src_type == t && b->rels[r].nnz > 0;
        if (!read || b->n_src[t] == 0) continue;
        const rgcn_input &x = in[t];
        if (!x.base || !aligned16(x.base))
            return fail(RGCN_ERR_INVALID_ARG, "input %d: base NULL or not 16-byte aligned", t);
        if (x.ld < L.d_in || x.ld % vec)
            return fail(RGCN_ERR_SHAPE, "input %d: ld %lld must be >= d_in and a multiple of %d", t,
                        (long long)x.ld, vec);
        if (x.row_ids && !((uintptr_t)x.row_ids % 8 == 0))
            return fail(RGCN_ERR_INVALID_ARG, "input %d: row_ids misaligned", t);
        if (!x.row_ids && x.num_rows < b->n_src[t])
            return fail(RGCN_ERR_SHAPE, "input %d: %lld rows < n_src %lld", t,
                        (long long)x.num_rows, (long long)b->n_src[t]);
        if (x.num_rows < 0) return fail(RGCN_ERR_SHAPE, "input %d: negative num_rows", t);
    }
    return RGCN_OK;
}

__global__ void k_zero_word(uint32_t *p) { *p = 0u; }

// Device-side structural check (synchronises the stream).
rgcn_status device_validate(const rgcn_block *b, const rgcn_input *in, const Layout &L,
                            char *ws, hipStream_t s) {
    uint32_t *err = (uint32_t *)(ws + L.off_err);
    hipLaunchKernelGGL(k_zero_word, dim3(1), dim3(1), 0, s, err);
    TRY_HIP(hipGetLastError(), "validate");
    for (int r = 0; r < L.R; ++r) {
        const rgcn_relation &rel = b->rels[r];
        TRY_HIP(validate_csr(rel.indptr, rel.indices, b->n_dst[rel.dst_type], rel.nnz,
                             b->n_src[rel.src_type], err, s), "validate_csr");
    }
    if (in) {
        for (int t = 0; t < L.T; ++t)
            if (in[t].row_ids)
                TRY_HIP(validate_ids(in[t].row_ids, b->n_src[t], in[t].num_rows, err, s),
                        "validate_ids");
        for (int r = 0; r < L.R; ++r) {
            const rgcn_relation &rel = b->rels[r];
            if (rel.src_rows && rel.nnz > 0)
                TRY_HIP(validate_src_rows(rel.indices, rel.src_rows, rel.nnz,
                                          b->n_src[rel.src_type], in[rel.src_type].row_ids,
                                          in[rel.src_type].num_rows, err, s),
                        "validate_src_rows");
        }
    }
    uint32_t host = 0;
    TRY_HIP(hipMemcpyAsync(&host, err, 4, hipMemcpyDeviceToHost, s), "validate copy");
    TRY_HIP(hipStreamSynchronize(s), "validate sync");
    if (host & 1u) return fail(RGCN_ERR_BAD_CSR, "indptr is not a valid CSR offset array");
    if (host & 2u) return fail(RGCN_ERR_INDEX_OOB, "an index or row id is out of range");
    return RGCN_OK;
}

}  // namespace

extern "C" {

const char *rgcn_last_error(void) { return g_err.c_str(); }

const char *rgcn_version(void) { return "rgcn-mi355x 0.1 (gfx950)"; }

rgcn_status rgcn_block_workspace_size(const rgcn_block *block, const rgcn_params *params,
                                      size_t *bytes) {
    if (!bytes) return fail(RGCN_ERR_INVALID_ARG, "bytes is NULL");
    Layout L;
    rgcn_status st = make_layout(block, params, L);
    if (st != RGCN_OK) return st;
    *bytes = L.total;
    return RGCN_OK;
}

rgcn_status rgcn_block_plan_layout(const rgcn_block *block, const rgcn_params *params,
                                   rgcn_plan_layout *out) {
    if (!out) return fail(RGCN_ERR_INVALID_ARG, "layout is NULL");
    Layout L;
    rgcn_status st = make_layout(block, params, L);
    if (st != RGCN_OK) return st;
    memset(out, 0, sizeof(*out));
    out->n_fwd_segments = L.n_seg;
    out->fwd_order = L.off_fwd_order;
    out->n_bwd_rows = L.n_bwd_rows;
    out->bwd_order = L.off_bwd_order;
    for (int r = 0; r < RGCN_MAX_RELS; ++r) {
        out->csc_indptr[r] = L.off_csc_indptr[r];
        out->csc_dst[r] = L.off_csc_dst[r];
    }
    out->total_bytes = L.total;
    return RGCN_OK;
}

rgcn_status rgcn_block_plan(const rgcn_block *block, const rgcn_params *params,
                            void *workspace, size_t workspace_bytes, unsigned flags,
                            hipStream_t stream) {
    Layout L;
    rgcn_status st = make_layout(block, params, L);
    if (st != RGCN_OK) return st;
    if ((st = check_workspace(L, workspace, workspace_bytes)) != RGCN_OK) return st;
    char *ws = (char *)workspace;
    if (flags & RGCN_VALIDATE_DEVICE) {
        if ((st = device_validate(block, nullptr, L, ws, stream)) != RGCN_OK) return st;
    }
    char *scratch = ws + L.off_scratch;
    const int keep_order = (flags & RGCN_PLAN_ENUMERATION_ORDER) ? 1 : 0;
    unsigned parts = flags & (RGCN_PLAN_FORWARD | RGCN_PLAN_BACKWARD);
    if (parts == 0) parts = RGCN_PLAN_FORWARD | RGCN_PLAN_BACKWARD;
    // flag word 0 belongs to the forward schedule, words 1 + t to the backward ones
    uint32_t *sched_flag = (uint32_t *)(ws + L.off_flags);
    const uint32_t zeros[1 + kMaxTypes] = {};
    if (parts & RGCN_PLAN_FORWARD) {
        if (L.nslots > 0)
            TRY_HIP(fill_words(ws + L.off_slots, L.slots, sizeof(FwdSlot) * L.nslots, stream),
                    "slot table");
        TRY_HIP(fill_words(sched_flag, zeros, sizeof(uint32_t), stream), "schedule flags");
    }
    if (parts & RGCN_PLAN_BACKWARD) {
        TRY_HIP(fill_words(sched_flag + 1, zeros, sizeof(uint32_t) * kMaxTypes, stream),
                "schedule flags");
        TRY_HIP(fill_words(sched_flag + kPieceCountWord, zeros, sizeof(uint32_t) * kMaxTypes,
                           stream), "piece counters");
    }
    if (parts & RGCN_PLAN_FORWARD) {
        int64_t moff[kMaxTypes], mld[kMaxTypes];
        for (int t = 0; t < kMaxTypes; ++t) {
            moff[t] = (t < L.T && L.off_mcat[t] != SIZE_MAX) ? (int64_t)L.off_mcat[t] : 0;
            mld[t] = t < L.T ? L.K[t] : 0;
        }
        // segment weights sit in the plan scratch after the chunk pass's own temporaries
        int32_t *weight = (int32_t *)(scratch + fwd_chunks_temp_bytes(L.n_seg));
        TRY_HIP(fwd_plan(L.slots, L.nslots, L.n_seg, (int32_t *)(ws + L.off_fwd_order), moff, mld,
                         L.es, (SegDesc *)(ws + L.off_fwd_desc), weight, sched_flag,
                         keep_order, scratch, stream), "forward schedule");
        TRY_HIP(fwd_chunks(weight, L.n_seg, L.nc_max, (int32_t *)(ws + L.off_fwd_chunks), scratch,
                           stream), "forward chunks");
    }
    if (!(parts & RGCN_PLAN_BACKWARD)) return RGCN_OK;
    if (L.key_range > 0) {
        CscRels cr{};
        int64_t rows = 0;
        for (int r = 0; r < L.R; ++r) {
            if (L.koff[r] < 0) continue;
            const rgcn_relation &rel = block->rels[r];
            cr.row_base[cr.count] = rows;
            cr.indptr[cr.count] = rel.indptr;
            cr.indices[cr.count] = rel.indices;
            cr.koff[cr.count] = L.koff[r];
            cr.e0[cr.count] = L.e0[r];
            ++cr.count;
            rows += block->n_dst[rel.dst_type];
        }
        TRY_HIP(csc_build_all(cr, rows, L.csc_nnz, L.key_range, (int32_t *)(ws + L.off_ip),
                              (int32_t *)(ws + L.off_csd), scratch, stream), "transpose");
    }
    for (int t = 0; t < L.T; ++t) {
        if (!(L.grad_mask >> t & 1u)) continue;
        BwdKeyRels kr{};
        for (int r = 0; r < L.R; ++r)
            if (block->rels[r].src_type == t)
                kr.csc_indptr[kr.count++] = (const int32_t *)(ws + L.off_csc_indptr[r]);
        SplitRows sp;
        sp.np = (int32_t *)(ws + L.off_split_np) + L.bwd_base[t];
        sp.base = (int32_t *)(ws + L.off_split_base) + L.bwd_base[t];
        sp.pieces = (int2 *)(ws + L.off_pieces) + L.piece_at[t];
        sp.count = sched_flag + kPieceCountWord + t;
        sp.cap = L.piece_cap[t];
        TRY_HIP(bwd_schedule(kr, block->n_src[t], (int32_t *)(ws + L.off_bwd_order) + L.bwd_base[t],
                             scratch, sched_flag + 1 + t, keep_order, sp, stream),
                "backward schedule");
    }
    return RGCN_OK;
}

rgcn_status rgcn_block_aggregate(const rgcn_block *block, const rgcn_input *in,
                                 const rgcn_params *params, void *workspace,
                                 size_t workspace_bytes, unsigned flags, hipStream_t stream) {
    Layout L;
    rgcn_status st = make_layout(block, params, L);
    if (st != RGCN_OK) return st;
    if ((st = check_workspace(L, workspace, workspace_bytes)) != RGCN_OK) return st;
    if ((st = check_inputs(block, in, L, false)) != RGCN_OK) return st;
    char *ws = (char *)workspace;
    if (flags & RGCN_VALIDATE_DEVICE) {
        if ((st = device_validate(block, in, L, ws, stream)) != RGCN_OK) return st;
    }
    TypeInput tin[kMaxTypes];
    for (int t = 0; t < kMaxTypes; ++t)
        tin[t] = t < L.T ? TypeInput{in[t].base, in[t].row_ids, in[t].ld} : TypeInput{nullptr, nullptr, 0};
    TRY_HIP(gather_mean(L.dt, L.d_in, (const SegDesc *)(ws + L.off_fwd_desc), L.n_seg,
                        (const int32_t *)(ws + L.off_fwd_chunks), L.nc_max,
                        (const FwdSlot *)(ws + L.off_slots), L.nslots, tin, ws,
                        (uint32_t *)(ws + L.off_flags) + kGatherClaimWord, stream),
            "gather mean");
    return RGCN_OK;
}

// The forward outputs: y[t] for every type with rows, and the optional sign masks (only
// with RGCN_FUSE_RELU, 8-byte aligned).
static rgcn_status check_forward_outputs(const rgcn_block *block, int T, void *const *y,
                                         uint64_t *const *relu_mask, unsigned flags) {
    if (!y) return fail(RGCN_ERR_INVALID_ARG, "y is NULL");
    for (int t = 0; t < T; ++t) {
        if (block->n_dst[t] > 0 && (!y[t] || !aligned16(y[t])))
            return fail(RGCN_ERR_INVALID_ARG, "y[%d] NULL or not 16-byte aligned", t);
        if (relu_mask && relu_mask[t]) {
            if (!(flags & RGCN_FUSE_RELU))
                return fail(RGCN_ERR_INVALID_ARG, "relu_mask[%d] given without RGCN_FUSE_RELU", t);
            if ((uintptr_t)relu_mask[t] % 8)
                return fail(RGCN_ERR_INVALID_ARG, "relu_mask[%d] not 8-byte aligned", t);
        }
    }
    return RGCN_OK;
}

rgcn_status rgcn_block_transform(const rgcn_block *block, const rgcn_params *params,
                                 void *const *y, uint64_t *const *relu_mask, void *workspace,
                                 size_t workspace_bytes, unsigned flags, hipStream_t stream) {
    Layout L;
    rgcn_status st = make_layout(block, params, L);
    if (st != RGCN_OK) return st;
    if ((st = check_workspace(L, workspace, workspace_bytes)) != RGCN_OK) return st;
    if ((st = check_forward_outputs(block, L.T, y, relu_mask, flags)) != RGCN_OK) return st;
    char *ws = (char *)workspace;
    for (int t = 0; t < L.T; ++t) {
        if (block->n_dst[t] == 0) continue;
        // weights of type t, K-contiguous: [W_self_t; W_r for r into t] transposed
        const void *wslots[kMaxSlots];
        wslots[0] = params->w_self[t];
        for (int r = 0; r < L.R; ++r)
            if (L.rel_pos[r] > 0 && block->rels[r].dst_type == t) wslots[L.rel_pos[r]] = params->w_rel[r];
        TRY_HIP(pack_weights(L.dt, L.d_in, L.d_out, wslots, L.type_nslots[t], ws + L.off_wcat[t],
                             stream), "pack weights");
        const void *bias = params->bias ? params->bias[t] : nullptr;
        TRY_HIP(gemm_forward(L.dt, ws + L.off_mcat[t], block->n_dst[t], L.d_out, (int)L.K[t],
                             ws + L.off_wcat[t], bias, (flags & RGCN_FUSE_RELU) ? 1 : 0, y[t],
                             relu_mask ? relu_mask[t] : nullptr, stream),
                "forward transform");
    }
    return RGCN_OK;
}

rgcn_status rgcn_block_forward(const rgcn_block *block, const rgcn_input *in,
                               const rgcn_params *params, void *const *y,
                               uint64_t *const *relu_mask, void *workspace,
                               size_t workspace_bytes, unsigned flags, hipStream_t stream) {
    // check everything the second stage needs before enqueueing the first
    if (!y) return fail(RGCN_ERR_INVALID_ARG, "y is NULL");
    if (block && block->n_dst && block->num_types > 0 && block->num_types <= kMaxTypes) {
        rgcn_status st = check_forward_outputs(block, block->num_types, y, relu_mask, flags);
        if (st != RGCN_OK) return st;
    }
    rgcn_status st = rgcn_block_aggregate(block, in, params, workspace, workspace_bytes, flags,
                                          stream);
    if (st != RGCN_OK) return st;
    return rgcn_block_transform(block, params, y, relu_mask, workspace, workspace_bytes,
                                flags & ~RGCN_VALIDATE_DEVICE, stream);
}

// the hi/lo gradient forms exist for the bf16 products only
static rgcn_status check_hilo_flags(const Layout &L, unsigned flags) {
    if ((flags & (RGCN_DY_HILO | RGCN_DH_HILO)) && L.dt != RGCN_BF16)
        return fail(RGCN_ERR_UNSUPPORTED, "RGCN_DY_HILO / RGCN_DH_HILO need the bf16 dtype");
    return RGCN_OK;
}

static rgcn_status check_dy(const rgcn_block *block, const Layout &L, const float *const *dy) {
    if (!dy) return fail(RGCN_ERR_INVALID_ARG, "dy is NULL");
    for (int t = 0; t < L.T; ++t)
        if (block->n_dst[t] > 0 && (!dy[t] || !aligned16(dy[t])))
            return fail(RGCN_ERR_INVALID_ARG, "dy[%d] NULL or not 16-byte aligned", t);
    return RGCN_OK;
}

static rgcn_status check_sparse_outputs(const rgcn_block *block, const rgcn_input *in,
                                        const Layout &L, float *const *dh_src,
                                        float *const *demb, unsigned flags) {
    for (int t = 0; t < L.T; ++t) {
        const bool want = (dh_src && dh_src[t]) || (demb && demb[t]);
        if (want && !(L.grad_mask >> t & 1u))
            return fail(RGCN_ERR_INVALID_ARG,
                        "dh_src/demb of type %d requested but bit %d of grad_src_types is clear", t, t);
        if (dh_src && dh_src[t] && !aligned16(dh_src[t]))
            return fail(RGCN_ERR_INVALID_ARG, "dh_src[%d] not 16-byte aligned", t);
        if (demb && demb[t] && !aligned16(demb[t]))
            return fail(RGCN_ERR_INVALID_ARG, "demb[%d] not 16-byte aligned", t);
        if (want && block->n_src[t] > 0 && (!in || !in[t].base ||
                                            ((flags & RGCN_INPUT_RELU) && !aligned16(in[t].base))))
            return fail(RGCN_ERR_INVALID_ARG, "input %d needed for its gradient", t);
        if (want && in && in[t].relu_mask && (uintptr_t)in[t].relu_mask % 8)
            return fail(RGCN_ERR_INVALID_ARG, "input %d: relu_mask not 8-byte aligned", t);
    }
    return RGCN_OK;
}

rgcn_status rgcn_block_backward_dense(const rgcn_block *block, const rgcn_params *params,
                                      const float *const *dy, float *const *dw_rel,
                                      float *const *dw_self, float *const *dbias,
                                      void *workspace, size_t workspace_bytes, unsigned flags,
                                      hipStream_t stream) {
    Layout L;
    rgcn_status st = make_layout(block, params, L);
    if (st != RGCN_OK) return st;
    if ((st = check_workspace(L, workspace, workspace_bytes)) != RGCN_OK) return st;
    if ((st = check_hilo_flags(L, flags)) != RGCN_OK) return st;
    if ((st = check_dy(block, L, dy)) != RGCN_OK) return st;
    const bool hilo = (flags & RGCN_DY_HILO) != 0;
    for (int t = 0; t < L.T; ++t)
        if (dw_self && dw_self[t])
            for (int u = 0; u < t; ++u)
                if (dw_self[u] == dw_self[t])
                    return fail(RGCN_ERR_INVALID_ARG, "dw_self[%d] aliases dw_self[%d]", t, u);
    char *ws = (char *)workspace;
    char *scratch = ws + L.off_scratch;
    for (int t = 0; t < L.T; ++t) {
        const int64_t nd = block->n_dst[t];
        // weight side: [dW_self_t; dW_r ...] = Mcat_t^T dY_t
        DwOut out{};
        out.count = nd > 0 ? L.type_nslots[t] : 1;
        out.w[0] = dw_self ? dw_self[t] : nullptr;
        bool any = out.w[0] != nullptr;
        if (nd > 0) {
            for (int r = 0; r < L.R; ++r)
                if (L.rel_pos[r] > 0 && block->rels[r].dst_type == t) {
                    out.w[L.rel_pos[r]] = dw_rel ? dw_rel[r] : nullptr;
                    any |= out.w[L.rel_pos[r]] != nullptr;
                }
        } else {  // no rows: gradients of the weights into t are zero
            for (int r = 0; r < L.R; ++r)
                if (block->rels[r].dst_type == t && dw_rel && dw_rel[r] && out.count < kMaxSlots) {
                    out.w[out.count++] = dw_rel[r];
                    any = true;
                }
        }
        if (any)
            TRY_HIP(gemm_dw(L.dt, nd > 0 ? ws + L.off_mcat[t] : nullptr, nd,
                            nd > 0 ? (int)L.K[t] : out.count * L.d_in, L.d_in,
                            nd > 0 ? dy[t] : nullptr, hilo, L.d_out, out,
                            (float *)(scratch + L.off_partial), stream), "weight gradient");
        if (dbias && dbias[t])
            TRY_HIP(column_sums(nd > 0 ? dy[t] : nullptr, hilo, nd, L.d_out, dbias[t],
                                (float *)(scratch + L.off_colsum), 0, stream), "bias gradient");
        // input side: dMs_t = dY_t [W_self_t | W_r ...]^T, relation slots divided by deg
        if (nd > 0 && L.dms_nslots[t] > 0) {
            DmsSlots ds{};
            ds.count = L.dms_nslots[t];
            if (L.dms_self[t] >= 0) {
                ds.w[L.dms_self[t]] = params->w_self[t];
                ds.indptr[L.dms_self[t]] = nullptr;
            }
            for (int r = 0; r < L.R; ++r)
                if (L.dms_rel[r] >= 0 && block->rels[r].dst_type == t) {
                    ds.w[L.dms_rel[r]] = params->w_rel[r];
                    ds.indptr[L.dms_rel[r]] = block->rels[r].indptr;
                }
            // the packed forward weights of the type are not read again before the next
            // transform packs them anew: their space holds the input side's weight rows
            TRY_HIP(gemm_dms(L.dt, dy[t], hilo, nd, L.d_out, L.d_in, ds,
                             (float *)(scratch + L.off_dms[t]), ws + L.off_wcat[t], stream),
                    "input-side transform");
        }
    }
    return RGCN_OK;
}

}  // extern "C"

namespace {

// Checks of the Adagrad mode of the transposed sum (types with opt->state[t] set).
rgcn_status check_adagrad(const rgcn_block *block, const rgcn_input *in, const Layout &L,
                          float *const *demb, const rgcn_adagrad *opt, unsigned flags) {
    if (!opt) return fail(RGCN_ERR_INVALID_ARG, "opt is NULL");
    if (!opt->state) return fail(RGCN_ERR_INVALID_ARG, "opt->state is NULL");
    if (!(flags & RGCN_IDS_UNIQUE))
        return fail(RGCN_ERR_INVALID_ARG, "the fused Adagrad step requires RGCN_IDS_UNIQUE");
    if (!(opt->lr == opt->lr) || !(opt->eps == opt->eps))
        return fail(RGCN_ERR_INVALID_ARG, "lr or eps is NaN");
    for (int t = 0; t < L.T; ++t) {
        if (!opt->state[t]) continue;
        if (!(L.grad_mask >> t & 1u))
            return fail(RGCN_ERR_INVALID_ARG, "Adagrad on type %d but bit %d of grad_src_types "
                        "is clear", t, t);
        if (flags & RGCN_INPUT_RELU)
            return fail(RGCN_ERR_INVALID_ARG, "Adagrad on type %d with RGCN_INPUT_RELU", t);
        if (demb && demb[t])
            return fail(RGCN_ERR_INVALID_ARG, "type %d has both demb and an Adagrad state", t);
        if (!aligned16(opt->state[t]))
            return fail(RGCN_ERR_INVALID_ARG, "state[%d] not 16-byte aligned", t);
        if (!opt->table || !opt->table[t] || !in || opt->table[t] != in[t].base)
            return fail(RGCN_ERR_INVALID_ARG, "table[%d] must be the writable base of input %d",
                        t, t);
        if (block->n_src[t] > 0 && (!aligned16(in[t].base) || in[t].ld < L.d_in))
            return fail(RGCN_ERR_INVALID_ARG, "table %d misaligned or ld < d_in", t);
    }
    return RGCN_OK;
}

rgcn_status backward_sparse(const rgcn_block *block, const rgcn_input *in,
                            const rgcn_params *params, float *const *dh_src, float *const *demb,
                            const rgcn_adagrad *opt, void *workspace, size_t workspace_bytes,
                            unsigned flags, hipStream_t stream) {
    Layout L;
    rgcn_status st = make_layout(block, params, L);
    if (st != RGCN_OK) return st;
    if ((st = check_workspace(L, workspace, workspace_bytes)) != RGCN_OK) return st;
    if ((st = check_hilo_flags(L, flags)) != RGCN_OK) return st;
    if ((st = check_sparse_outputs(block, in, L, dh_src, demb, flags)) != RGCN_OK) return st;
    if (opt && (st = check_adagrad(block, in, L, demb, opt, flags)) != RGCN_OK) return st;
    char *ws = (char *)workspace;
    if ((flags & RGCN_VALIDATE_DEVICE) && in) {
        if ((st = device_validate(block, in, L, ws, stream)) != RGCN_OK) return st;
    }
    char *scratch = ws + L.off_scratch;
    for (int s = 0; s < L.T; ++s) {
        float *dh = dh_src ? dh_src[s] : nullptr;
        float *de = demb ? demb[s] : nullptr;
        float *state = opt ? opt->state[s] : nullptr;
        if (!dh && !de && !state) continue;
        TsumArgs a;
        memset(&a, 0, sizeof(a));
        a.order = (const int32_t *)(ws + L.off_bwd_order) + L.bwd_base[s];
        a.n_rows = block->n_src[s];
        a.n_dst = block->n_dst[s];
        if (block->n_dst[s] > 0 && L.dms_self[s] >= 0) {
            a.self_dms = (const float *)(scratch + L.off_dms[s]) + (int64_t)L.dms_self[s] * L.d_in;
            a.self_ld = (int64_t)L.dms_nslots[s] * L.d_in;
        }
        a.in = TypeInput{in[s].base, in[s].row_ids, in[s].ld};
        a.input_relu = (flags & RGCN_INPUT_RELU) ? 1 : 0;
        if (a.input_relu && in[s].relu_mask) {   // the input's signs as bits
            a.relu_mask = in[s].relu_mask;
            a.mask_ld = (L.d_in + 63) / 64;
        }
        a.ids_unique = (flags & RGCN_IDS_UNIQUE) ? 1 : 0;
        a.dh = dh;
        a.dh_hilo = (flags & RGCN_DH_HILO) ? 1 : 0;
        a.demb = de;
        if (state) {
            a.opt_state = state;
            a.opt_table = opt->table[s];
            a.lr = opt->lr;
            a.eps = opt->eps;
        }
        a.d_in = L.d_in;
        a.split_np = (const int32_t *)(ws + L.off_split_np) + L.bwd_base[s];
        a.split_base = (const int32_t *)(ws + L.off_split_base) + L.bwd_base[s];
        a.pieces = (const int2 *)(ws + L.off_pieces) + L.piece_at[s];
        a.piece_count = (const uint32_t *)(ws + L.off_flags) + kPieceCountWord + s;
        a.piece_cap = L.piece_cap[s];
        a.partial = (float *)(scratch + L.off_split_partial) + L.piece_at[s] * L.d_in;
        for (int r = 0; r < L.R; ++r) {
            const rgcn_relation &rel = block->rels[r];
            if (rel.src_type != s || block->n_dst[rel.dst_type] == 0) continue;
            const int t = rel.dst_type;
            TsumRel tr;
            tr.csc_indptr = (const int32_t *)(ws + L.off_csc_indptr[r]);
            tr.csc_dst = (const int32_t *)(ws + L.off_csd);
            tr.dms = (const float *)(scratch + L.off_dms[t]) + (int64_t)L.dms_rel[r] * L.d_in;
            tr.dms_ld = (int64_t)L.dms_nslots[t] * L.d_in;
            a.rel[a.nrel++] = tr;
        }
        TRY_HIP(transpose_sum(L.dt, a, stream), "transposed sum");
    }
    return RGCN_OK;
}

}  // namespace

extern "C" {

rgcn_status rgcn_block_backward_sparse(const rgcn_block *block, const rgcn_input *in,
                                       const rgcn_params *params, float *const *dh_src,
                                       float *const *demb, void *workspace,
                                       size_t workspace_bytes, unsigned flags,
                                       hipStream_t stream) {
    return backward_sparse(block, in, params, dh_src, demb, nullptr, workspace, workspace_bytes,
                           flags, stream);
}

rgcn_status rgcn_block_backward_sparse_adagrad(const rgcn_block *block, const rgcn_input *in,
                                               const rgcn_params *params,
                                               float *const *dh_src, float *const *demb,
                                               const rgcn_adagrad *opt, void *workspace,
                                               size_t workspace_bytes, unsigned flags,
                                               hipStream_t stream) {
    if (!opt) return fail(RGCN_ERR_INVALID_ARG, "opt is NULL");
    return backward_sparse(block, in, params, dh_src, demb, opt, workspace, workspace_bytes,
                           flags, stream);
}

rgcn_status rgcn_sparse_adagrad(int64_t n, const int64_t *rows, int64_t num_rows, int32_t d,
                                float *grad, float *state, void *table, int64_t ld,
                                rgcn_dtype dtype, float lr, float eps, unsigned flags,
                                hipStream_t stream) {
    if (!dtype_known(&dtype)) return fail(RGCN_ERR_DTYPE, "unknown dtype");
    const int vec = dtype == RGCN_BF16 ? 8 : 4;
    if (n < 0 || num_rows < 0 || d < 0) return fail(RGCN_ERR_SHAPE, "negative size");
    if (d % vec || ld < d || ld % vec)
        return fail(RGCN_ERR_SHAPE, "d %d and ld %lld must be multiples of %d with ld >= d", d,
                    (long long)ld, vec);
    if (flags & ~(unsigned)RGCN_CLEAR_GRAD)
        return fail(RGCN_ERR_INVALID_ARG, "unsupported flags 0x%x", flags);
    if (!(lr == lr) || !(eps == eps)) return fail(RGCN_ERR_INVALID_ARG, "lr or eps is NaN");
    if (n == 0 || d == 0) return RGCN_OK;
    if (!rows || !grad || !state || !table)
        return fail(RGCN_ERR_INVALID_ARG, "rows, grad, state or table is NULL");
    if ((uintptr_t)rows % 8 || !aligned16(grad) || !aligned16(state) || !aligned16(table))
        return fail(RGCN_ERR_INVALID_ARG, "misaligned array");
    TRY_HIP(sparse_adagrad(dtype, n, rows, num_rows, d, grad, d, (flags & RGCN_CLEAR_GRAD) != 0,
                           state, table, ld, lr, eps, stream), "sparse Adagrad");
    return RGCN_OK;
}

rgcn_status rgcn_block_backward(const rgcn_block *block, const rgcn_input *in,
                                const rgcn_params *params, const float *const *dy,
                                float *const *dw_rel, float *const *dw_self,
                                float *const *dbias, float *const *dh_src, float *const *demb,
                                void *workspace, size_t workspace_bytes, unsigned flags,
                                hipStream_t stream) {
    // validate what both stages need before enqueueing anything
    Layout L;
    rgcn_status st = make_layout(block, params, L);
    if (st != RGCN_OK) return st;
    if ((st = check_workspace(L, workspace, workspace_bytes)) != RGCN_OK) return st;
    if ((st = check_inputs(block, in, L, false)) != RGCN_OK) return st;
    if ((st = check_hilo_flags(L, flags)) != RGCN_OK) return st;
    if ((st = check_dy(block, L, dy)) != RGCN_OK) return st;
    if ((st = check_sparse_outputs(block, in, L, dh_src, demb, flags)) != RGCN_OK) return st;
    if (flags & RGCN_VALIDATE_DEVICE) {
        if ((st = device_validate(block, in, L, (char *)workspace, stream)) != RGCN_OK) return st;
    }
    const unsigned f = flags & ~RGCN_VALIDATE_DEVICE;
    st = rgcn_block_backward_dense(block, params, dy, dw_rel, dw_self, dbias, workspace,
                                   workspace_bytes, f, stream);
    if (st != RGCN_OK) return st;
    return rgcn_block_backward_sparse(block, in, params, dh_src, demb, workspace,
                                      workspace_bytes, f, stream);
}

}  // extern "C"

namespace {

rgcn_status sample_tab(const rgcn_graph *g, const int64_t *n_dst, int32_t fanout,
                       SampleTab &T, SampleLayout &L) {
    if (!g || !n_dst) return fail(RGCN_ERR_INVALID_ARG, "graph or n_dst is NULL");
    if (g->num_types < 1 || g->num_types > kMaxTypes)
        return fail(RGCN_ERR_INVALID_ARG, "num_types %d outside [1, %d]", g->num_types, kMaxTypes);
    if (g->num_rels < 0 || g->num_rels > kMaxRels)
        return fail(RGCN_ERR_INVALID_ARG, "num_rels %d outside [0, %d]", g->num_rels, kMaxRels);
    if (!g->num_nodes || (g->num_rels > 0 && !g->rels))
        return fail(RGCN_ERR_INVALID_ARG, "num_nodes or rels is NULL");
    if (fanout < 1 || fanout > kMaxFanout)
        return fail(RGCN_ERR_UNSUPPORTED, "fanout %d outside [1, %d]", fanout, kMaxFanout);
    memset(&T, 0, sizeof(T));
    T.ntypes = g->num_types;
    T.nrel = g->num_rels;
    T.fanout = fanout;
    for (int t = 0; t < T.ntypes; ++t) {
        if (g->num_nodes[t] < 0 || g->num_nodes[t] >= (int64_t)1 << 59)
            return fail(RGCN_ERR_SHAPE, "num_nodes[%d] outside [0, 2^59)", t);
        if (n_dst[t] < 0) return fail(RGCN_ERR_SHAPE, "n_dst[%d] negative", t);
        T.num_nodes[t] = g->num_nodes[t];
        T.n_dst[t] = n_dst[t];
    }
    for (int r = 0; r < T.nrel; ++r) {
        const rgcn_graph_relation &rel = g->rels[r];
        if (rel.src_type < 0 || rel.src_type >= T.ntypes || rel.dst_type < 0 ||
            rel.dst_type >= T.ntypes)
            return fail(RGCN_ERR_INVALID_ARG, "relation %d: bad node type", r);
        if (!rel.indptr || !rel.indices || ((uintptr_t)rel.indptr | (uintptr_t)rel.indices) & 7u)
            return fail(RGCN_ERR_INVALID_ARG, "relation %d: indptr/indices NULL or misaligned", r);
        T.src_type[r] = rel.src_type;
        T.dst_type[r] = rel.dst_type;
        T.g_indptr[r] = rel.indptr;
        T.g_indices[r] = rel.indices;
    }
    if (!sample_layout(T, L))
        return fail(RGCN_ERR_UNSUPPORTED, "sampling capacity %lld exceeds 2^31",
                    (long long)T.cap_total);
    return RGCN_OK;
}

}  // namespace

extern "C" {

rgcn_status rgcn_sample_workspace_size(const rgcn_graph *graph, const int64_t *n_dst,
                                       int32_t fanout, size_t *bytes) {
    if (!bytes) return fail(RGCN_ERR_INVALID_ARG, "bytes is NULL");
    SampleTab T;
    SampleLayout L;
    rgcn_status st = sample_tab(graph, n_dst, fanout, T, L);
    if (st != RGCN_OK) return st;
    *bytes = L.total;
    return RGCN_OK;
}

rgcn_status rgcn_sample_block(const rgcn_graph *graph, const int64_t *const *dst_ids,
                              const int64_t *n_dst, int32_t fanout, uint64_t seed,
                              int32_t layer, int32_t *const *out_indptr,
                              int32_t *const *out_indices, int64_t *const *out_src_ids,
                              int64_t *const *out_src_rows, int64_t *counts, void *workspace,
                              size_t workspace_bytes, unsigned flags, hipStream_t stream) {
    SampleTab T;
    SampleLayout L;
    rgcn_status st = sample_tab(graph, n_dst, fanout, T, L);
    if (st != RGCN_OK) return st;
    if (flags & ~(unsigned)RGCN_VALIDATE_DEVICE)
        return fail(RGCN_ERR_INVALID_ARG, "unsupported flags 0x%x", flags);
    if (!workspace || ((uintptr_t)workspace & 255u))
        return fail(RGCN_ERR_INVALID_ARG, "workspace NULL or not 256-byte aligned");
    if (workspace_bytes < L.total)
        return fail(RGCN_ERR_WORKSPACE_TOO_SMALL, "workspace %zu bytes, need %zu",
                    workspace_bytes, L.total);
    if (!counts || ((uintptr_t)counts & 7u))
        return fail(RGCN_ERR_INVALID_ARG, "counts NULL or misaligned");
    if (!dst_ids || !out_indptr || !out_indices || !out_src_ids)
        return fail(RGCN_ERR_INVALID_ARG, "an array argument is NULL");
    T.seed = seed;
    T.layer = layer;
    for (int t = 0; t < T.ntypes; ++t) {
        if (T.n_dst[t] > 0 && (!dst_ids[t] || ((uintptr_t)dst_ids[t] & 7u)))
            return fail(RGCN_ERR_INVALID_ARG, "dst_ids[%d] NULL or misaligned", t);
        if (T.type_cap[t] > 0 && (!out_src_ids[t] || ((uintptr_t)out_src_ids[t] & 7u)))
            return fail(RGCN_ERR_INVALID_ARG, "out_src_ids[%d] NULL or misaligned", t);
        T.dst_ids[t] = dst_ids[t];
        T.out_src_ids[t] = out_src_ids[t];
    }
    for (int r = 0; r < T.nrel; ++r) {
        const int64_t cap = T.n_dst[T.dst_type[r]] * (int64_t)fanout;
        if (!out_indptr[r] || ((uintptr_t)out_indptr[r] & 3u))
            return fail(RGCN_ERR_INVALID_ARG, "out_indptr[%d] NULL or misaligned", r);
        if (cap > 0 && (!out_indices[r] || ((uintptr_t)out_indices[r] & 3u)))
            return fail(RGCN_ERR_INVALID_ARG, "out_indices[%d] NULL or misaligned", r);
        T.out_indptr[r] = out_indptr[r];
        T.out_indices[r] = out_indices[r];
        int64_t *rows = out_src_rows ? out_src_rows[r] : nullptr;
        if (rows && ((uintptr_t)rows & 7u))
            return fail(RGCN_ERR_INVALID_ARG, "out_src_rows[%d] misaligned", r);
        T.out_src_rows[r] = cap > 0 ? rows : nullptr;
    }
    char *ws = (char *)workspace;
    TRY_HIP(sample_block(T, L, ws, counts, stream), "sampling");
    if (flags & RGCN_VALIDATE_DEVICE) {
        uint32_t host = 0;
        TRY_HIP(hipMemcpyAsync(&host, ws + L.off_err, 4, hipMemcpyDeviceToHost, stream),
                "validate copy");
        TRY_HIP(hipStreamSynchronize(stream), "validate sync");
        if (host & 1u) return fail(RGCN_ERR_INDEX_OOB, "a destination id is out of range");
        if (host & 8u) return fail(RGCN_ERR_INDEX_OOB, "a graph source id is out of range");
        if (host & 2u) return fail(RGCN_ERR_INVALID_ARG, "repeated destination ids");
        if (host & 4u) return fail(RGCN_ERR_UNSUPPORTED, "an in-degree of 2^32 or more");
    }
    return RGCN_OK;
}

}  // extern "C"

namespace {

rgcn_status lp_args(const rgcn_lp_batch *b, LpArgs &a) {
    if (!b) return fail(RGCN_ERR_INVALID_ARG, "batch is NULL");
    if (!dtype_known(&b->dtype)) return fail(RGCN_ERR_DTYPE, "unknown dtype");
    const int vec = b->dtype == RGCN_BF16 ? 8 : 4;
    if (b->d <= 0 || b->d % vec || b->d > 256 * vec)
        return fail(RGCN_ERR_UNSUPPORTED, "d %d must be a positive multiple of %d, at most %d",
                    b->d, vec, 256 * vec);
    if (b->ld < b->d || b->ld % vec || b->n_rows < 0)
        return fail(RGCN_ERR_SHAPE, "ld %lld must be >= d and a multiple of %d",
                    (long long)b->ld, vec);
    if (b->neg_mode < 0 || b->neg_mode > 2) return fail(RGCN_ERR_INVALID_ARG, "unknown neg_mode");
    if (b->loss < 0 || b->loss > 2) return fail(RGCN_ERR_INVALID_ARG, "unknown loss");
    if (b->batch < 0) return fail(RGCN_ERR_SHAPE, "negative batch");
    if (b->neg_mode != RGCN_LP_NEG_IN_BATCH && b->k < 1)
        return fail(RGCN_ERR_SHAPE, "k must be at least 1");
    memset(&a, 0, sizeof(a));
    a.dtype = b->dtype;
    a.d = b->d;
    a.ld = b->ld;
    a.n_rows = b->n_rows;
    a.emb = b->emb;
    a.rel = b->rel;
    a.neg_mode = b->neg_mode;
    a.loss = b->loss;
    a.batch = b->batch;
    a.k = b->neg_mode == RGCN_LP_NEG_IN_BATCH ? 0 : b->k;
    a.nn = b->neg_mode == RGCN_LP_NEG_IN_BATCH ? (b->batch > 0 ? b->batch - 1 : 0) : b->k;
    a.src = b->src;
    a.dst = b->dst;
    a.neg = b->neg;
    a.pos_weight = b->pos_weight;
    if ((double)a.batch * (double)(a.nn > 0 ? a.nn : 1) >= 2147483647.0 ||
        (double)a.batch * a.d >= 2147483647.0)
        return fail(RGCN_ERR_UNSUPPORTED, "batch x negatives or batch x d reaches 2^31");
    if (a.batch > 0) {
        if (!a.emb || !aligned16(a.emb)) return fail(RGCN_ERR_INVALID_ARG, "emb NULL or misaligned");
        if (a.rel && !aligned16(a.rel)) return fail(RGCN_ERR_INVALID_ARG, "rel misaligned");
        if (!a.src || !a.dst || !aligned4(a.src) || !aligned4(a.dst))
            return fail(RGCN_ERR_INVALID_ARG, "src or dst NULL or misaligned");
        if (a.neg_mode != RGCN_LP_NEG_IN_BATCH && (!a.neg || !aligned4(a.neg)))
            return fail(RGCN_ERR_INVALID_ARG, "neg NULL or misaligned");
        if (a.loss == RGCN_LP_WEIGHTED_CE && (!a.pos_weight || !aligned4(a.pos_weight)))
            return fail(RGCN_ERR_INVALID_ARG, "pos_weight NULL or misaligned");
    }
    return RGCN_OK;
}

}  // namespace

extern "C" {

rgcn_status rgcn_lp_workspace_size(const rgcn_lp_batch *batch, size_t *bytes) {
    if (!bytes) return fail(RGCN_ERR_INVALID_ARG, "bytes is NULL");
    LpArgs a;
    rgcn_status st = lp_args(batch, a);
    if (st != RGCN_OK) return st;
    *bytes = lp_layout(a).total;
    return RGCN_OK;
}

}  // extern "C"

namespace {

// Argument checks of the decoder shared by both entry points (the workspace aside).
rgcn_status lp_check_outputs(const LpArgs &a, float *loss, float *pos_score, float *neg_score,
                             float *d_emb, float *d_rel, unsigned flags) {
    if (flags & ~(unsigned)RGCN_VALIDATE_DEVICE)
        return fail(RGCN_ERR_INVALID_ARG, "unsupported flags 0x%x", flags);
    if (!loss || !aligned4(loss)) return fail(RGCN_ERR_INVALID_ARG, "loss NULL or misaligned");
    if ((pos_score && !aligned4(pos_score)) || (neg_score && !aligned4(neg_score)) ||
        (d_emb && !aligned4(d_emb)) || (d_rel && !aligned4(d_rel)))
        return fail(RGCN_ERR_INVALID_ARG, "an output is misaligned");
    if (d_rel && !a.rel) return fail(RGCN_ERR_INVALID_ARG, "d_rel requested for a dot product");
    return RGCN_OK;
}

// The decoder's launches on temporaries at `ws` (L.total bytes, 256-byte aligned).
rgcn_status lp_run(const LpArgs &a, const LpLayout &L, char *ws, float *loss, float *pos_score,
                   float *neg_score, float *d_emb, float *d_rel, unsigned flags,
                   hipStream_t stream) {
    if ((flags & RGCN_VALIDATE_DEVICE) && a.batch > 0) {
        uint32_t *err = (uint32_t *)(ws + L.off_err);
        const uint32_t zero = 0;
        TRY_HIP(fill_words(err, &zero, 4, stream), "validate");
        TRY_HIP(lp_validate(a, err, stream), "validate");
        uint32_t host = 0;
        TRY_HIP(hipMemcpyAsync(&host, err, 4, hipMemcpyDeviceToHost, stream), "validate copy");
        TRY_HIP(hipStreamSynchronize(stream), "validate sync");
        if (host) return fail(RGCN_ERR_INDEX_OOB, "a row index is outside [0, n_rows)");
    }
    TRY_HIP(lp_loss(a, L, ws, loss, pos_score, neg_score, d_emb, d_rel, stream), "link prediction");
    return RGCN_OK;
}

}  // namespace

extern "C" {

rgcn_status rgcn_lp_loss(const rgcn_lp_batch *batch, float *loss, float *pos_score,
                         float *neg_score, float *d_emb, float *d_rel, void *workspace,
                         size_t workspace_bytes, unsigned flags, hipStream_t stream) {
    LpArgs a;
    rgcn_status st = lp_args(batch, a);
    if (st != RGCN_OK) return st;
    if ((st = lp_check_outputs(a, loss, pos_score, neg_score, d_emb, d_rel, flags)) != RGCN_OK)
        return st;
    const LpLayout L = lp_layout(a);
    if (!workspace || ((uintptr_t)workspace & 255u))
        return fail(RGCN_ERR_INVALID_ARG, "workspace NULL or not 256-byte aligned");
    if (workspace_bytes < L.total)
        return fail(RGCN_ERR_WORKSPACE_TOO_SMALL, "workspace %zu bytes, need %zu",
                    workspace_bytes, L.total);
    return lp_run(a, L, (char *)workspace, loss, pos_score, neg_score, d_emb, d_rel, flags,
                  stream);
}

}  // extern "C"

// ------------------------------------------------ the decoder without a caller workspace
// Temporaries of rgcn_lp_loss_noalloc: one fixed array per device, part of the library's
// code object (each GPU the library runs on holds it until the process ends).  Host code
// never uses its name as an address: the per-device address comes from
// hipGetSymbolAddress, taken once per device with that device current.
static __device__ __align__(256) char scratch[RGCN_LP_NOALLOC_MAX_SCRATCH];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char *g_scratch_ptr[kMaxDevices] = {};

// The current device's scratch address (looked up on the first call on each device).
rgcn_status current_scratch(char **out) {
    int dev = -1;
    TRY_HIP(hipGetDevice(&dev), "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices)
        return fail(RGCN_ERR_UNSUPPORTED, "device index %d outside [0, %d)", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        TRY_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "scratch address");
        if (!p || ((uintptr_t)p & 255u))
            return fail(RGCN_ERR_HIP, "scratch array address missing or misaligned");
        g_scratch_ptr[dev] = (char *)p;
    }
    *out = g_scratch_ptr[dev];
    return RGCN_OK;
}

}  // namespace

extern "C" {

rgcn_status rgcn_lp_loss_noalloc(const rgcn_lp_batch *batch, float *loss, float *pos_score,
                                 float *neg_score, float *d_emb, float *d_rel, unsigned flags,
                                 hipStream_t stream) {
    LpArgs a;
    rgcn_status st = lp_args(batch, a);
    if (st != RGCN_OK) return st;
    if ((st = lp_check_outputs(a, loss, pos_score, neg_score, d_emb, d_rel, flags)) != RGCN_OK)
        return st;
    const LpLayout L = lp_layout(a);
    if (L.total > (size_t)RGCN_LP_NOALLOC_MAX_SCRATCH)
        return fail(RGCN_ERR_UNSUPPORTED,
                    "this batch needs %zu bytes of temporaries, above the %zu of the fixed "
                    "scratch array; call rgcn_lp_loss with a workspace", L.total,
                    (size_t)RGCN_LP_NOALLOC_MAX_SCRATCH);
    char *ws = nullptr;
    if ((st = current_scratch(&ws)) != RGCN_OK) return st;
    return lp_run(a, L, ws, loss, pos_score, neg_score, d_emb, d_rel, flags, stream);
}

rgcn_status rgcn_lp_negatives(int32_t neg_mode, int64_t slots, int64_t num_nodes, uint64_t seed,
                              int64_t *out, hipStream_t stream) {
    if (neg_mode != RGCN_LP_NEG_PER_EDGE && neg_mode != RGCN_LP_NEG_JOINT)
        return fail(RGCN_ERR_INVALID_ARG, "negative ids are drawn for per-edge or joint modes");
    if (slots < 0 || num_nodes < 1) return fail(RGCN_ERR_SHAPE, "slots < 0 or num_nodes < 1");
    if (slots > 0 && (!out || ((uintptr_t)out & 7u)))
        return fail(RGCN_ERR_INVALID_ARG, "out NULL or misaligned");
    TRY_HIP(lp_negatives(neg_mode, slots, num_nodes, seed, out, stream), "negatives");
    return RGCN_OK;
}

}  // extern "C"

extern "C" {

rgcn_status rgcn_featureless_mean(int32_t num_rels, const rgcn_feature_relation *rels,
                                  int64_t num_nodes, int32_t d, rgcn_dtype dtype, void *out,
                                  int64_t out_ld, void *workspace, unsigned flags,
                                  hipStream_t stream) {
    if (!dtype_known(&dtype)) return fail(RGCN_ERR_DTYPE, "unknown dtype");
    const int vec = dtype == RGCN_BF16 ? 8 : 4;
    if (num_rels < 1 || num_rels > kMaxRels || !rels)
        return fail(RGCN_ERR_INVALID_ARG, "num_rels %d outside [1, %d] or rels NULL", num_rels,
                    kMaxRels);
    if (d <= 0 || d % vec || d > 256 * vec)
        return fail(RGCN_ERR_UNSUPPORTED, "d %d must be a positive multiple of %d, at most %d", d,
                    vec, 256 * vec);
    if (num_nodes < 0 || out_ld < d || out_ld % vec)
        return fail(RGCN_ERR_SHAPE, "num_nodes negative or out_ld %lld bad", (long long)out_ld);
    if (flags & ~(unsigned)RGCN_VALIDATE_DEVICE)
        return fail(RGCN_ERR_INVALID_ARG, "unsupported flags 0x%x", flags);
    if (num_nodes > 0 && (!out || !aligned16(out)))
        return fail(RGCN_ERR_INVALID_ARG, "out NULL or not 16-byte aligned");
    if (!workspace || ((uintptr_t)workspace & 255u))
        return fail(RGCN_ERR_INVALID_ARG, "workspace NULL or not 256-byte aligned");
    FeatArgs a;
    memset(&a, 0, sizeof(a));
    for (int r = 0; r < num_rels; ++r) {
        const rgcn_feature_relation &x = rels[r];
        if (!x.indptr || !x.indices || ((uintptr_t)x.indptr | (uintptr_t)x.indices) & 7u)
            return fail(RGCN_ERR_INVALID_ARG, "relation %d: indptr/indices NULL or misaligned", r);
        if (x.rows < 0 || x.ld < d || x.ld % vec || (x.rows > 0 && (!x.features ||
                                                                    !aligned16(x.features))))
            return fail(RGCN_ERR_SHAPE, "relation %d: feature table misaligned or ld < d", r);
        a.rel[r] = FeatRel{x.indptr, x.indices, x.features, x.rows, x.ld};
    }
    a.nrel = num_rels;
    a.d = d;
    a.num_nodes = num_nodes;
    a.out_ld = out_ld;
    a.out = out;
    a.dtype = dtype;
    uint32_t *words = (uint32_t *)workspace;
    TRY_HIP(featureless_mean(a, words, stream), "featureless mean");
    if ((flags & RGCN_VALIDATE_DEVICE) && num_nodes > 0) {
        uint32_t host = 0;
        TRY_HIP(hipMemcpyAsync(&host, words + 1, 4, hipMemcpyDeviceToHost, stream),
                "validate copy");
        TRY_HIP(hipStreamSynchronize(stream), "validate sync");
        if (host & 1u) return fail(RGCN_ERR_INDEX_OOB, "a neighbour index is out of range");
    }
    return RGCN_OK;
}

}  // extern "C"
