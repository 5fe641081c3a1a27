/*
 * sample_oracle.c -- plain CPU oracle of on-the-fly neighbour sampling and block
 * construction for one layer of a mini-batch.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or call this
 * file; only the tests and the benchmark's CPU baseline do.  It shares no code, header,
 * table or helper with the HIP library.
 *
 * The paper trains on mini-batches whose neighbourhoods are sampled on the fly with a
 * fanout per layer (Sec. 3.1.1, the distributed graph engine's sampling; Sec. 3.1.4,
 * mini-batch training), one block per GNN layer, built top-down from the seeds.  It does
 * not spell out the sampler; the reading taken here:
 *
 *  - For every destination node v (global id) of type dst(r) and every relation r, the
 *    in-neighbours of v in r are the positions [indptr_r[v], indptr_r[v+1]) of the
 *    graph's in-edge CSR.  With deg <= fanout all of them are taken; otherwise fanout
 *    distinct positions, every subset of that size equally likely, chosen by Floyd's
 *    algorithm (for j = deg-fanout .. deg-1: t uniform in [0, j]; take t, or j if t was
 *    already taken).  Taken positions are listed in ascending order.
 *  - Randomness: draw k of (v, r) is word k mod 4 of the Philox4x64-10 block function
 *    (Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3",
 *    SC 2011) at counter (v, r, floor(k / 4), 0) with key (seed, layer).  A uniform
 *    integer in [0, m) is the high word of the 128-bit product draw * m.
 *  - Block: the destination nodes of type t are the first n_dst[t] source nodes of type
 *    t; the other source nodes follow in order of first appearance over the sampled
 *    edges (relations in order, destination rows in order, taken positions in order);
 *    edge indices are these block-local source rows.  Destination ids of a type must be
 *    distinct.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ---------------------------------------------------------------- Philox4x64-10 */
/* The round function multiplies words 0 and 2 by two fixed odd constants, keeping both
 * halves of the 128-bit products, and mixes the high halves with words 1 and 3 and the
 * key; the key is advanced by two Weyl constants between rounds. */
static const uint64_t PHILOX_M0 = 0xD2E7470EE14C6C93ULL;
static const uint64_t PHILOX_M1 = 0xCA5A826395121157ULL;
static const uint64_t PHILOX_W0 = 0x9E3779B97F4A7C15ULL;
static const uint64_t PHILOX_W1 = 0xBB67AE8584CAA73BULL;

static void mulhilo64(uint64_t a, uint64_t b, uint64_t *hi, uint64_t *lo)
{
    unsigned __int128 p = (unsigned __int128)a * (unsigned __int128)b;
    *hi = (uint64_t)(p >> 64);
    *lo = (uint64_t)p;
}

void orc_philox4x64(const uint64_t *ctr, const uint64_t *key, uint64_t *out)
{
    uint64_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint64_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += PHILOX_W0;
            k1 += PHILOX_W1;
        }
        uint64_t hi0, lo0, hi1, lo1;
        mulhilo64(PHILOX_M0, c0, &hi0, &lo0);
        mulhilo64(PHILOX_M1, c2, &hi1, &lo1);
        uint64_t n0 = hi1 ^ c1 ^ k0, n1 = lo1, n2 = hi0 ^ c3 ^ k1, n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Draw k of segment (v, r) at (seed, layer). */
uint64_t orc_sample_draw(uint64_t seed, uint64_t layer, uint64_t v, uint64_t r, uint64_t k)
{
    uint64_t ctr[4] = {v, r, k / 4, 0}, key[2] = {seed, layer}, out[4];
    orc_philox4x64(ctr, key, out);
    return out[k % 4];
}

/* Uniform integer in [0, m): high word of draw * m. */
static uint64_t uniform_below(uint64_t draw, uint64_t m)
{
    uint64_t hi, lo;
    mulhilo64(draw, m, &hi, &lo);
    return hi;
}

static int cmp_i64(const void *a, const void *b)
{
    int64_t x = *(const int64_t *)a, y = *(const int64_t *)b;
    return (x > y) - (x < y);
}

/* Positions taken from a segment of n in-edges with the given fanout, ascending.
 * Returns the count (min(n, fanout)); pos must hold that many.  fanout >= 1. */
int64_t orc_sample_segment(int64_t n, int64_t fanout, uint64_t seed, int32_t layer,
                           int64_t v, int32_t r, int64_t *pos)
{
    if (n <= fanout) {
        for (int64_t i = 0; i < n; ++i) pos[i] = i;
        return n;
    }
    int64_t taken = 0;
    for (int64_t k = 0; k < fanout; ++k) {
        int64_t j = n - fanout + k;
        uint64_t d = orc_sample_draw(seed, (uint64_t)(uint32_t)layer, (uint64_t)v,
                                     (uint64_t)(uint32_t)r, (uint64_t)k);
        int64_t t = (int64_t)uniform_below(d, (uint64_t)(j + 1));
        int seen = 0;
        for (int64_t q = 0; q < taken; ++q)
            if (pos[q] == t) seen = 1;
        pos[taken++] = seen ? j : t;
    }
    qsort(pos, (size_t)taken, sizeof(int64_t), cmp_i64);
    return taken;
}

/* ---------------------------------------------------------------- block construction */
typedef struct {
    int64_t id;
    int64_t pos;
} id_pos;

static int cmp_id_pos(const void *a, const void *b)
{
    const id_pos *x = (const id_pos *)a, *y = (const id_pos *)b;
    if (x->id != y->id) return (x->id > y->id) - (x->id < y->id);
    return (x->pos > y->pos) - (x->pos < y->pos);
}

/* One layer's block.  Graph relation r: src type rel_src[r], dst type rel_dst[r], in-edge
 * CSR g_indptr[r] ([num_nodes[rel_dst[r]] + 1]) and g_indices[r] (global source ids).
 * dst_ids[t]: n_dst[t] distinct global ids of type t.
 * Outputs (caller-allocated): out_indptr[r] [n_dst[rel_dst[r]] + 1]; out_indices[r]
 * (capacity n_dst * fanout); out_src_ids[t] (capacity n_dst[t] + the sampled edges leaving
 * type t); counts[r] = sampled edges of r, counts[num_rels + t] = source nodes of type t.
 * Returns 0, -1 (a destination id out of range) or -2 (repeated destination ids). */
int orc_sample_block(int32_t num_types, int32_t num_rels, const int32_t *rel_src,
                     const int32_t *rel_dst, const int64_t *const *g_indptr,
                     const int64_t *const *g_indices, const int64_t *num_nodes,
                     const int64_t *const *dst_ids, const int64_t *n_dst, int64_t fanout,
                     uint64_t seed, int32_t layer, int32_t *const *out_indptr,
                     int32_t *const *out_indices, int64_t *const *out_src_ids,
                     int64_t *counts)
{
    /* 1. sample every (destination, relation) segment: global source ids per edge */
    int64_t **cand = (int64_t **)calloc((size_t)num_rels, sizeof(int64_t *));
    int64_t *pos = (int64_t *)malloc((size_t)(fanout > 0 ? fanout : 1) * sizeof(int64_t));
    int rc = 0;
    for (int32_t r = 0; r < num_rels && rc == 0; ++r) {
        int32_t t = rel_dst[r];
        cand[r] = (int64_t *)malloc((size_t)(n_dst[t] * fanout + 1) * sizeof(int64_t));
        out_indptr[r][0] = 0;
        int64_t e = 0;
        for (int64_t i = 0; i < n_dst[t]; ++i) {
            int64_t v = dst_ids[t][i];
            if (v < 0 || v >= num_nodes[t]) { rc = -1; break; }
            int64_t b = g_indptr[r][v], n = g_indptr[r][v + 1] - b;
            int64_t c = orc_sample_segment(n, fanout, seed, layer, v, r, pos);
            for (int64_t q = 0; q < c; ++q) cand[r][e++] = g_indices[r][b + pos[q]];
            out_indptr[r][i + 1] = (int32_t)e;
        }
        counts[r] = e;
    }
    /* 2. per source type: destination ids first, then sampled sources; the first
     *    occurrence of each id gets the next block-local row */
    for (int32_t s = 0; s < num_types && rc == 0; ++s) {
        int64_t m = n_dst[s];
        for (int32_t r = 0; r < num_rels; ++r)
            if (rel_src[r] == s) m += counts[r];
        id_pos *all = (id_pos *)malloc((size_t)(m + 1) * sizeof(id_pos));
        int64_t p = 0;
        for (int64_t i = 0; i < n_dst[s]; ++i, ++p) all[p].id = dst_ids[s][i], all[p].pos = p;
        for (int32_t r = 0; r < num_rels; ++r)
            if (rel_src[r] == s)
                for (int64_t e = 0; e < counts[r]; ++e, ++p) all[p].id = cand[r][e], all[p].pos = p;
        qsort(all, (size_t)m, sizeof(id_pos), cmp_id_pos);
        int64_t *first_of = (int64_t *)malloc((size_t)(m + 1) * sizeof(int64_t));
        unsigned char *is_first = (unsigned char *)calloc((size_t)(m + 1), 1);
        for (int64_t q = 0; q < m; ++q) {
            int64_t f = (q > 0 && all[q].id == all[q - 1].id) ? first_of[all[q - 1].pos]
                                                               : all[q].pos;
            first_of[all[q].pos] = f;
            if (f == all[q].pos) is_first[f] = 1;
        }
        for (int64_t i = 0; i < n_dst[s]; ++i)
            if (!is_first[i]) rc = -2;
        int64_t *local = (int64_t *)malloc((size_t)(m + 1) * sizeof(int64_t));
        int64_t n_src = 0;
        /* ids by position, to number first occurrences in position order */
        int64_t *id_at = (int64_t *)malloc((size_t)(m + 1) * sizeof(int64_t));
        for (int64_t q = 0; q < m; ++q) id_at[all[q].pos] = all[q].id;
        for (int64_t q = 0; q < m; ++q)
            if (is_first[q]) {
                local[q] = n_src;
                out_src_ids[s][n_src++] = id_at[q];
            }
        counts[num_rels + s] = n_src;
        p = n_dst[s];
        for (int32_t r = 0; r < num_rels; ++r)
            if (rel_src[r] == s)
                for (int64_t e = 0; e < counts[r]; ++e, ++p)
                    out_indices[r][e] = (int32_t)local[first_of[p]];
        free(all); free(first_of); free(is_first); free(local); free(id_at);
    }
    for (int32_t r = 0; r < num_rels; ++r) free(cand[r]);
    free(cand);
    free(pos);
    return rc;
}
