/*
 * feature_oracle.c -- plain CPU oracle of feature construction for featureless nodes
 * (Sec. 3.3.2, eq. 1: the features of a node without features are built from its
 * neighbours that have features, with f an average or a learned function).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or call this
 * file; only the tests and the benchmark's CPU baseline do.  It shares no code, header,
 * table or helper with the HIP library.  Arithmetic in IEEE double.
 *
 * Reading (f the average): for node i of the featureless type, N_i is the multiset of
 * in-neighbours over the given relations, each from a type with features (an edge
 * listed twice counts twice, as in the layer's mean), and
 *   F'_i = (1 / |N_i|) sum_{j in N_i} F_{src(r)}[j],      F'_i = 0 when N_i is empty.
 * Relation r: in-edge CSR over the featureless type (indptr [num_nodes + 1], indices =
 * global rows of its source type's feature table).
 */
#include <stdint.h>
#include <string.h>

/* feat[r]: [src_rows[r] x d] source features of relation r.  out: [num_nodes x d].
 * Returns 0, or -1 when an index is out of range. */
int orc_featureless_mean(int32_t num_rels, const int64_t *const *indptr,
                         const int64_t *const *indices, const double *const *feat,
                         const int64_t *src_rows, int64_t num_nodes, int64_t d, double *out)
{
    for (int64_t i = 0; i < num_nodes; ++i) {
        double *o = out + i * d;
        memset(o, 0, (size_t)d * sizeof(double));
        int64_t count = 0;
        for (int32_t r = 0; r < num_rels; ++r) {
            for (int64_t k = indptr[r][i]; k < indptr[r][i + 1]; ++k) {
                int64_t j = indices[r][k];
                if (j < 0 || j >= src_rows[r]) return -1;
                for (int64_t c = 0; c < d; ++c) o[c] += feat[r][j * d + c];
                ++count;
            }
        }
        if (count > 0)
            for (int64_t c = 0; c < d; ++c) o[c] /= (double)count;
    }
    return 0;
}
