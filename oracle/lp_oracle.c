/*
 * lp_oracle.c -- plain CPU oracle of the link-prediction decoder: scores, losses, their
 * gradients, and negative-edge construction (the paper's appendix on link-prediction
 * score and loss functions and negative sampling).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or call this
 * file; only the tests and the benchmark's CPU baseline do.  It shares no code, header,
 * table or helper with the HIP library.  All arithmetic in IEEE double.
 *
 * Scores of an edge (u, v) with n-dimensional embeddings (appendix, score functions):
 *   dot product:  sum_c emb_u[c] * emb_v[c]
 *   DistMult:     sum_c emb_u[c] * rel[c] * emb_v[c]      (rel: the edge type's embedding)
 * (the printed dot product reuses the node index i as the summation index; the sum runs
 * over the embedding dimension.)
 *
 * Negatives of positive edge i = (src_i, dst_i), which keep src_i and replace dst_i
 * (appendix, negative sampling):
 *   per edge (uniform): K nodes of its own, neg[i*K + k];
 *   joint: the K positives of group g = i / K share K nodes, neg[g*K + k];
 *   in-batch: the destinations of the other positives, dst_j for j != i in ascending j
 *     (B - 1 negatives), as in the appendix's three-edge example.
 *
 * Losses (appendix, loss functions), with s the score:
 *   cross entropy: the printed formula misplaces a sign and a bracket; read as binary
 *     cross entropy on sigmoid(s) with label 1 for positives and 0 for negatives,
 *     averaged over all B (1 + K) scored edges;
 *   weighted cross entropy: the same with weight w_i on positive edge i and weight 1 on
 *     negatives (the printed w_e is 1 for edges of the training graph, which every
 *     positive is), averaged over all scored edges;
 *   contrastive: per positive, -log(exp(s_pos) / (exp(s_pos) + sum_k exp(s_k))) over the
 *     positive and its negatives (the printed lower limit "1=0" read as i = 0 .. N with
 *     the positive included), averaged over the B positives.
 * Gradients are those of the averaged loss with respect to every embedding row used and
 * to rel, written out by the chain rule.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

void orc_philox4x64(const uint64_t *ctr, const uint64_t *key, uint64_t *out);

enum { LP_DOT = 0, LP_DISTMULT = 1 };
enum { NEG_PER_EDGE = 0, NEG_JOINT = 1, NEG_IN_BATCH = 2 };
enum { LOSS_CE = 0, LOSS_WCE = 1, LOSS_CONTRASTIVE = 2 };

/* Number of negatives of each positive. */
int64_t orc_lp_num_neg(int32_t neg_mode, int64_t batch, int64_t k)
{
    return neg_mode == NEG_IN_BATCH ? (batch > 0 ? batch - 1 : 0) : k;
}

/* Row of negative k of positive i. */
int64_t orc_lp_neg_row(int32_t neg_mode, int64_t i, int64_t k, int64_t kk, const int64_t *neg,
                       const int64_t *dst)
{
    if (neg_mode == NEG_PER_EDGE) return neg[i * kk + k];
    if (neg_mode == NEG_JOINT) return neg[(i / kk) * kk + k];
    return dst[k < i ? k : k + 1];
}

static double score(const double *a, const double *b, const double *rel, int64_t d)
{
    double s = 0.0;
    for (int64_t c = 0; c < d; ++c) s += a[c] * (rel ? rel[c] : 1.0) * b[c];
    return s;
}

static double softplus(double x)   /* log(1 + exp(x)) without overflow */
{
    return x > 0 ? x + log1p(exp(-x)) : log1p(exp(x));
}

static double sigmoid(double x) { return 1.0 / (1.0 + exp(-x)); }

/* emb [n_rows x d]; rel [d] (DistMult) or NULL (dot).  Outputs: *loss; pos_score [B];
 * neg_score [B x N]; d_emb [n_rows x d] (added to) and d_rel [d] (overwritten) when not
 * NULL.  Returns 0, or -1 on an invalid mode or row. */
int orc_lp_loss(int64_t n_rows, int64_t d, const double *emb, const double *rel,
                int32_t neg_mode, int32_t loss_kind, int64_t batch, const int64_t *src,
                const int64_t *dst, int64_t k, const int64_t *neg, const double *pos_weight,
                double *loss, double *pos_score, double *neg_score, double *d_emb,
                double *d_rel)
{
    if (neg_mode < 0 || neg_mode > 2 || loss_kind < 0 || loss_kind > 2) return -1;
    const int64_t nn = orc_lp_num_neg(neg_mode, batch, k);
    for (int64_t i = 0; i < batch; ++i) {
        if (src[i] < 0 || src[i] >= n_rows || dst[i] < 0 || dst[i] >= n_rows) return -1;
        for (int64_t q = 0; q < nn; ++q) {
            int64_t r = orc_lp_neg_row(neg_mode, i, q, k, neg, dst);
            if (r < 0 || r >= n_rows) return -1;
        }
    }
    /* scores */
    for (int64_t i = 0; i < batch; ++i) {
        pos_score[i] = score(emb + src[i] * d, emb + dst[i] * d, rel, d);
        for (int64_t q = 0; q < nn; ++q) {
            int64_t r = orc_lp_neg_row(neg_mode, i, q, k, neg, dst);
            neg_score[i * nn + q] = score(emb + src[i] * d, emb + r * d, rel, d);
        }
    }
    /* loss and its derivative with respect to every score */
    double *gpos = (double *)calloc((size_t)(batch > 0 ? batch : 1), sizeof(double));
    double *gneg = (double *)calloc((size_t)(batch * nn > 0 ? batch * nn : 1), sizeof(double));
    double total = 0.0;
    if (loss_kind == LOSS_CONTRASTIVE) {
        for (int64_t i = 0; i < batch; ++i) {
            double m = pos_score[i];
            for (int64_t q = 0; q < nn; ++q) m = fmax(m, neg_score[i * nn + q]);
            double z = exp(pos_score[i] - m);
            for (int64_t q = 0; q < nn; ++q) z += exp(neg_score[i * nn + q] - m);
            total += m + log(z) - pos_score[i];
            gpos[i] = (exp(pos_score[i] - m) / z - 1.0) / (double)batch;
            for (int64_t q = 0; q < nn; ++q)
                gneg[i * nn + q] = exp(neg_score[i * nn + q] - m) / z / (double)batch;
        }
        total /= (double)batch;
    } else {
        const double n_edges = (double)(batch * (1 + nn));
        for (int64_t i = 0; i < batch; ++i) {
            double w = (loss_kind == LOSS_WCE && pos_weight) ? pos_weight[i] : 1.0;
            total += w * softplus(-pos_score[i]);        /* -log sigmoid(s) */
            gpos[i] = w * (sigmoid(pos_score[i]) - 1.0) / n_edges;
            for (int64_t q = 0; q < nn; ++q) {
                double s = neg_score[i * nn + q];
                total += softplus(s);                     /* -log(1 - sigmoid(s)) */
                gneg[i * nn + q] = sigmoid(s) / n_edges;
            }
        }
        total /= n_edges;
    }
    *loss = total;
    /* chain rule: d score(a, b) / d a = rel * b, / d b = rel * a, / d rel = a * b */
    if (d_rel) memset(d_rel, 0, (size_t)d * sizeof(double));
    for (int64_t i = 0; i < batch; ++i) {
        const double *a = emb + src[i] * d;
        for (int64_t q = -1; q < nn; ++q) {
            int64_t r = q < 0 ? dst[i] : orc_lp_neg_row(neg_mode, i, q, k, neg, dst);
            double g = q < 0 ? gpos[i] : gneg[i * nn + q];
            const double *b = emb + r * d;
            for (int64_t c = 0; c < d; ++c) {
                double rc = rel ? rel[c] : 1.0;
                if (d_emb) {
                    d_emb[src[i] * d + c] += g * rc * b[c];
                    d_emb[r * d + c] += g * rc * a[c];
                }
                if (d_rel && rel) d_rel[c] += g * a[c] * b[c];
            }
        }
    }
    free(gpos);
    free(gneg);
    return 0;
}

/* Negative node ids: slot q (per edge: q = i*K + k, joint: q = g*K + k) takes the high word
 * of draw * num_nodes, the draw being word q mod 4 of Philox4x64-10 at counter
 * (q / 4, mode, 0, 0) and key (seed, 0x6e6567). */
void orc_lp_negatives(int32_t neg_mode, int64_t slots, int64_t num_nodes, uint64_t seed,
                      int64_t *out)
{
    for (int64_t q = 0; q < slots; ++q) {
        uint64_t ctr[4] = {(uint64_t)q / 4, (uint64_t)neg_mode, 0, 0};
        uint64_t key[2] = {seed, 0x6e6567ULL}, w[4];
        orc_philox4x64(ctr, key, w);
        unsigned __int128 p = (unsigned __int128)w[q % 4] * (unsigned __int128)(uint64_t)num_nodes;
        out[q] = (int64_t)(uint64_t)(p >> 64);
    }
}
