/*
 * rgcn_oracle.c -- plain, slow CPU oracle of the relational graph-convolution (RGCN)
 * layer applied to one sampled mini-batch block, forward and backward.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or call this
 * file; only the tests, the smoke check and the CPU-baseline leg of the benchmark do.
 * It shares no code, header, table or helper with the HIP library.
 *
 * What it computes (all arithmetic in IEEE double, plain loops, no blocking or fusion):
 *
 *  The paper names RGCN as its encoder for heterogeneous graphs (Sec. 3.1.4 "Model
 *  zoo", and Sec. 3 "Design", the heterogeneous-graph models) and applies one GNN
 *  layer per sampled block (programming-interface appendix, customised-model figure:
 *  h = gcs[i](blocks[i], h) with h a dict keyed by node type).  Featureless node types
 *  read a learnable embedding table (Sec. 3.3.2).  The paper does not print the RGCN
 *  formula; the oracle uses the relational GCN form with a self-loop,
 *
 *      Y_t[i] = H_t[i] W_self_t + sum_{r : dst(r) = t} M_r[i] W_r + b_t,
 *      M_r[i] = (1 / deg_r(i)) * sum_{k in segment i of r} H_{src(r)}[indices_r[k]],
 *
 *  with deg_r(i) the number of sampled in-edges of destination row i in relation r
 *  (duplicates count) and M_r[i] = 0 when deg_r(i) = 0.  Destination rows of type t are
 *  the first n_dst[t] source rows of type t (block convention), so the self-loop reads
 *  H_t[0 .. n_dst[t]).  Its backward, given dY_t, is
 *
 *      db_t       = sum_i dY_t[i]
 *      dW_self_t  = sum_{i < n_dst[t]} H_t[i]^T dY_t[i]
 *      dW_r       = sum_i M_r[i]^T dY_{dst(r)}[i]
 *      dH_s[j]    = sum_{r: src(r)=s} sum_{(i,k): indices_r[k]=j} dY_{dst(r)}[i] W_r^T / deg_r(i)
 *                   + [j < n_dst[s]] dY_s[j] W_self_s^T
 *      dE_t[ids_t[j]] += dH_t[j]                (embedding-gradient scatter-add)
 *
 *  and the integer plan (degrees, and the CSC transpose of every relation as a stable
 *  counting sort of edge positions by source row), and a sparse Adagrad step on the
 *  touched rows of a learnable table.  The order in which a GPU processes segments is
 *  not part of the method (any order gives the same sums) and is not modelled here.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Threads of the loops below.  Each loop marked "omp" hands whole output elements to one
 * thread, which computes them in exactly the order written, so every result is the same
 * bit for bit whatever the thread count. */
void orc_set_threads(int n)
{
#ifdef _OPENMP
    omp_set_num_threads(n > 0 ? n : 1);
#else
    (void)n;
#endif
}

int orc_get_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

typedef struct {
    int32_t src_type;
    int32_t dst_type;
    const int32_t *indptr;   /* [n_dst[dst_type] + 1] */
    const int32_t *indices;  /* [indptr[n_dst]] local source rows */
} orc_relation;

typedef struct {
    int32_t num_types;
    int32_t num_rels;
    const int64_t *n_src;    /* [num_types] */
    const int64_t *n_dst;    /* [num_types] */
    const orc_relation *rels;
} orc_block;

/* Structural check of a block: CSR shape and index ranges.  0 = valid, -1 = invalid. */
int orc_check_block(const orc_block *b)
{
    for (int t = 0; t < b->num_types; ++t)
        if (b->n_dst[t] < 0 || b->n_src[t] < b->n_dst[t]) return -1;
    for (int r = 0; r < b->num_rels; ++r) {
        const orc_relation *rel = &b->rels[r];
        if (rel->src_type < 0 || rel->src_type >= b->num_types) return -1;
        if (rel->dst_type < 0 || rel->dst_type >= b->num_types) return -1;
        int64_t nd = b->n_dst[rel->dst_type], ns = b->n_src[rel->src_type];
        if (rel->indptr[0] != 0) return -1;
        for (int64_t i = 0; i < nd; ++i)
            if (rel->indptr[i + 1] < rel->indptr[i]) return -1;
        for (int64_t k = 0; k < rel->indptr[nd]; ++k)
            if (rel->indices[k] < 0 || rel->indices[k] >= ns) return -1;
    }
    return 0;
}

/* deg_r(i) = indptr[i+1] - indptr[i]. */
void orc_degrees(const int32_t *indptr, int64_t n_dst, int32_t *deg)
{
    for (int64_t i = 0; i < n_dst; ++i) deg[i] = indptr[i + 1] - indptr[i];
}

/* Segmented mean of one relation: M[i] = sum of the segment's source rows / deg, or 0.
 * The sum runs in ascending edge position, then one division. */
void orc_mean_aggregate(const int32_t *indptr, const int32_t *indices, int64_t n_dst,
                        const double *h_src, int64_t d, double *m)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n_dst; ++i) {
        int64_t deg = indptr[i + 1] - indptr[i];
        for (int64_t c = 0; c < d; ++c) {
            double acc = 0.0;
            for (int64_t k = indptr[i]; k < indptr[i + 1]; ++k)
                acc += h_src[(int64_t)indices[k] * d + c];
            m[i * d + c] = deg > 0 ? acc / (double)deg : 0.0;
        }
    }
}

/* Forward of one block.  h_src[t]: [n_src[t] x d_in]; w_rel[r], w_self[t]: [d_in x d_out]
 * row-major; bias[t]: [d_out] or NULL; y[t]: [n_dst[t] x d_out] (written for every type
 * with n_dst[t] > 0).  relu != 0 applies max(0, .) to the output.  Returns 0 or -1. */
int orc_block_forward(const orc_block *b, int64_t d_in, int64_t d_out,
                      const double *const *h_src, const double *const *w_rel,
                      const double *const *w_self, const double *const *bias, int relu,
                      double *const *y)
{
    if (orc_check_block(b) != 0) return -1;
    for (int t = 0; t < b->num_types; ++t) {
        int64_t nd = b->n_dst[t];
        if (nd == 0) continue;
        double *yt = y[t];
        /* self-loop term (and bias) */
#pragma omp parallel for schedule(static)
        for (int64_t i = 0; i < nd; ++i)
            for (int64_t o = 0; o < d_out; ++o) {
                double acc = bias && bias[t] ? bias[t][o] : 0.0;
                for (int64_t c = 0; c < d_in; ++c)
                    acc += h_src[t][i * d_in + c] * w_self[t][c * d_out + o];
                yt[i * d_out + o] = acc;
            }
        /* sum over relations into t of M_r W_r */
        for (int r = 0; r < b->num_rels; ++r) {
            const orc_relation *rel = &b->rels[r];
            if (rel->dst_type != t) continue;
            double *m = (double *)malloc((size_t)(nd * d_in) * sizeof(double));
            if (!m) return -1;
            orc_mean_aggregate(rel->indptr, rel->indices, nd, h_src[rel->src_type], d_in, m);
#pragma omp parallel for schedule(static)
            for (int64_t i = 0; i < nd; ++i)
                for (int64_t o = 0; o < d_out; ++o) {
                    double acc = 0.0;
                    for (int64_t c = 0; c < d_in; ++c)
                        acc += m[i * d_in + c] * w_rel[r][c * d_out + o];
                    yt[i * d_out + o] += acc;
                }
            free(m);
        }
        if (relu)
            for (int64_t e = 0; e < nd * d_out; ++e)
                if (!(yt[e] > 0.0)) yt[e] = 0.0;
    }
    return 0;
}

/* Backward of one block.  dy[t]: [n_dst[t] x d_out].  Outputs (any may be NULL, and
 * any per-type / per-relation entry may be NULL to skip it), all overwritten:
 *   dw_rel[r], dw_self[t]: [d_in x d_out]; dbias[t]: [d_out]; dh_src[t]: [n_src[t] x d_in].
 * input_relu != 0: the block's input is the output of a ReLU, so dh_src is multiplied
 * elementwise by [h_src > 0].  Returns 0 or -1. */
int orc_block_backward(const orc_block *b, int64_t d_in, int64_t d_out,
                       const double *const *h_src, const double *const *w_rel,
                       const double *const *w_self, const double *const *dy, int input_relu,
                       double *const *dw_rel, double *const *dw_self, double *const *dbias,
                       double *const *dh_src)
{
    if (orc_check_block(b) != 0) return -1;
    /* db_t and dW_self_t */
    for (int t = 0; t < b->num_types; ++t) {
        int64_t nd = b->n_dst[t];
        if (dbias && dbias[t])
#pragma omp parallel for schedule(static)
            for (int64_t o = 0; o < d_out; ++o) {
                double acc = 0.0;
                for (int64_t i = 0; i < nd; ++i) acc += dy[t][i * d_out + o];
                dbias[t][o] = acc;
            }
        if (dw_self && dw_self[t])
#pragma omp parallel for schedule(static)
            for (int64_t c = 0; c < d_in; ++c)
                for (int64_t o = 0; o < d_out; ++o) {
                    double acc = 0.0;
                    for (int64_t i = 0; i < nd; ++i)
                        acc += h_src[t][i * d_in + c] * dy[t][i * d_out + o];
                    dw_self[t][c * d_out + o] = acc;
                }
    }
    /* dW_r = M_r^T dY */
    if (dw_rel)
        for (int r = 0; r < b->num_rels; ++r) {
            if (!dw_rel[r]) continue;
            const orc_relation *rel = &b->rels[r];
            int64_t nd = b->n_dst[rel->dst_type];
            double *m = (double *)malloc((size_t)(nd * d_in + 1) * sizeof(double));
            if (!m) return -1;
            orc_mean_aggregate(rel->indptr, rel->indices, nd, h_src[rel->src_type], d_in, m);
#pragma omp parallel for schedule(static)
            for (int64_t c = 0; c < d_in; ++c)
                for (int64_t o = 0; o < d_out; ++o) {
                    double acc = 0.0;
                    for (int64_t i = 0; i < nd; ++i)
                        acc += m[i * d_in + c] * dy[rel->dst_type][i * d_out + o];
                    dw_rel[r][c * d_out + o] = acc;
                }
            free(m);
        }
    /* dH_src */
    if (dh_src)
        for (int s = 0; s < b->num_types; ++s) {
            if (!dh_src[s]) continue;
            int64_t ns = b->n_src[s], nds = b->n_dst[s];
            double *g = dh_src[s];
            for (int64_t e = 0; e < ns * d_in; ++e) g[e] = 0.0;
            /* self-loop: rows j < n_dst[s] receive dY_s[j] W_self_s^T */
#pragma omp parallel for schedule(static)
            for (int64_t j = 0; j < nds; ++j)
                for (int64_t c = 0; c < d_in; ++c) {
                    double acc = 0.0;
                    for (int64_t o = 0; o < d_out; ++o)
                        acc += dy[s][j * d_out + o] * w_self[s][c * d_out + o];
                    g[j * d_in + c] += acc;
                }
            /* every edge (i <- j) of a relation leaving s sends dY[i] W_r^T / deg_r(i);
             * column c of every row takes its terms in ascending (r, i, k) order */
            for (int r = 0; r < b->num_rels; ++r) {
                const orc_relation *rel = &b->rels[r];
                if (rel->src_type != s) continue;
                int t = rel->dst_type;
#pragma omp parallel for schedule(static)
                for (int64_t c = 0; c < d_in; ++c)
                    for (int64_t i = 0; i < b->n_dst[t]; ++i) {
                        int64_t deg = rel->indptr[i + 1] - rel->indptr[i];
                        for (int64_t k = rel->indptr[i]; k < rel->indptr[i + 1]; ++k) {
                            int64_t j = rel->indices[k];
                            double acc = 0.0;
                            for (int64_t o = 0; o < d_out; ++o)
                                acc += dy[t][i * d_out + o] * w_rel[r][c * d_out + o];
                            g[j * d_in + c] += acc / (double)deg;
                        }
                    }
            }
            if (input_relu)
                for (int64_t e = 0; e < ns * d_in; ++e)
                    if (!(h_src[s][e] > 0.0)) g[e] = 0.0;
        }
    return 0;
}

/* Embedding-gradient scatter-add (Sec. 3.3.2 learnable tables): for j ascending,
 * demb[ids[j]] += dh[j].  Repeated ids accumulate; rows never named are untouched. */
void orc_scatter_add(int64_t n, int64_t d, const int64_t *ids, const double *dh, double *demb)
{
    for (int64_t j = 0; j < n; ++j)
        for (int64_t c = 0; c < d; ++c)
            demb[ids[j] * d + c] += dh[j * d + c];
}

/* Sparse Adagrad step on the rows of a learnable embedding table that a mini-batch
 * touched (Sec. 3.3.2 trains such tables; the paper does not name the optimizer, and the
 * reading here is the row-wise Adagrad rule applied to touched rows only).  For each
 * listed row e, with g = grad[e] (the table-shaped gradient of the scatter-add above),
 * elementwise:
 *     state[e] <- state[e] + g * g
 *     table[e] <- table[e] - lr * g / (sqrt(state[e]) + eps)
 * Rows are listed at most once (the block's source ids of a type are distinct); rows not
 * listed are left exactly as they were.  Returns 0, or -1 for an out-of-range or repeated
 * row. */
int orc_sparse_adagrad(int64_t n, int64_t d, int64_t num_rows, const int64_t *rows,
                       const double *grad, double *state, double *table, double lr, double eps)
{
    unsigned char *seen = (unsigned char *)calloc((size_t)num_rows + 1, 1);
    if (!seen) return -1;
    for (int64_t i = 0; i < n; ++i) {
        const int64_t e = rows[i];
        if (e < 0 || e >= num_rows || seen[e]) { free(seen); return -1; }
        seen[e] = 1;
    }
    free(seen);
    for (int64_t i = 0; i < n; ++i) {
        const int64_t e = rows[i];
        for (int64_t c = 0; c < d; ++c) {
            const double g = grad[e * d + c];
            const double s = state[e * d + c] + g * g;
            state[e * d + c] = s;
            table[e * d + c] = table[e * d + c] - lr * g / (sqrt(s) + eps);
        }
    }
    return 0;
}

/* CSC transpose of one relation as a stable counting sort of edge positions k by
 * source row indices[k]: csc_indptr [n_src + 1], and for each slot p of the sorted order
 * csc_dst[p] = destination row of the edge, csc_eid[p] = its position k (ascending k
 * within a source row).  Returns 0 or -1. */
int orc_csc(int64_t n_src, int64_t n_dst, const int32_t *indptr, const int32_t *indices,
            int32_t *csc_indptr, int32_t *csc_dst, int32_t *csc_eid)
{
    int64_t nnz = indptr[n_dst];
    int64_t *fill = (int64_t *)calloc((size_t)n_src + 1, sizeof(int64_t));
    if (!fill) return -1;
    for (int64_t j = 0; j <= n_src; ++j) csc_indptr[j] = 0;
    for (int64_t k = 0; k < nnz; ++k) csc_indptr[indices[k] + 1] += 1;
    for (int64_t j = 0; j < n_src; ++j) csc_indptr[j + 1] += csc_indptr[j];
    for (int64_t i = 0; i < n_dst; ++i)
        for (int64_t k = indptr[i]; k < indptr[i + 1]; ++k) {
            int64_t j = indices[k];
            int64_t p = csc_indptr[j] + fill[j]++;
            csc_dst[p] = (int32_t)i;
            csc_eid[p] = (int32_t)k;
        }
    free(fill);
    return 0;
}
