// Feature construction for featureless nodes (Sec. 3.3.2, eq. 1, f the average): for
// every node i of the featureless type, the mean of the feature rows of its in-neighbours
// over the given relations (each relation's source type has a feature table; repeated
// edges count twice; zeros for a node without such neighbours), over the whole graph.
//
// One group of G lanes per node (G = 16-byte chunks per row, rounded up to a power of
// two, at least 8, at least the number of relations, at most 64; CPL chunks per lane
// beyond 64 chunks).  A persistent grid whose groups claim runs of 16 nodes from a
// counter, so a node of very high degree delays only the group that holds it.  A node's
// in-edges over all relations form one list: the offsets of every relation are loaded at
// once (the next node's while this one's rows are in flight), the group loads G ids of the
// list at a time, and every lane keeps up to 16 row chunks in flight before adding them in
// fp32 with compensation.  The mean is written in the table dtype (bf16 rounded to
// nearest even).
#include "common.h"

namespace rgcn {

namespace {

constexpr int kThreads = 256;
constexpr int kNodeRun = 16;   // nodes claimed at a time
constexpr int kMinGroup = 8;

__host__ __device__ inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Compensated (Kahan) accumulation: a node can have 1e5 in-neighbours, where a plain fp32
// running sum loses about n 2^-24 of its magnitude; the compensation term keeps the error
// near 2^-23 of the sum of magnitudes whatever the degree.
__device__ __forceinline__ void kahan_add(float &s, float &c, float x) {
    const float y = x - c;
    const float t = s + y;
    c = (t - s) - y;
    s = t;
}

template <bool BF16>
__device__ __forceinline__ void add_chunk(float *acc, float *comp, const uint4 w) {
    if constexpr (BF16) {
        kahan_add(acc[0], comp[0], bf16_lo(w.x)); kahan_add(acc[1], comp[1], bf16_hi(w.x));
        kahan_add(acc[2], comp[2], bf16_lo(w.y)); kahan_add(acc[3], comp[3], bf16_hi(w.y));
        kahan_add(acc[4], comp[4], bf16_lo(w.z)); kahan_add(acc[5], comp[5], bf16_hi(w.z));
        kahan_add(acc[6], comp[6], bf16_lo(w.w)); kahan_add(acc[7], comp[7], bf16_hi(w.w));
    } else {
        kahan_add(acc[0], comp[0], __uint_as_float(w.x));
        kahan_add(acc[1], comp[1], __uint_as_float(w.y));
        kahan_add(acc[2], comp[2], __uint_as_float(w.z));
        kahan_add(acc[3], comp[3], __uint_as_float(w.w));
    }
}

// Kernel body.  A node's in-edges over all relations are one flattened list: the group's
// lanes r < nrel hold relation r's [begin, end) for the node (an inclusive scan over
// them gives each relation's offset in the list), lane e of a batch loads the id of list
// entry e0 + e (its relation found from the offsets), and every lane then loads its
// chunk(s) of U of the batch's rows at a time, all U loads in flight before any is added.
// The next node's offsets are requested before the current node's rows.
template <bool BF16, int CPL>
__global__ __launch_bounds__(kThreads) void k_feature_mean(FeatArgs a, int G, uint32_t *claims,
                                                           uint32_t *err) {
    constexpr int VEC = BF16 ? 8 : 4;
    constexpr int U = 16 / CPL;                  // rows in flight per lane
    constexpr int ES = BF16 ? 2 : 4;
    __shared__ FeatRel s_rel[kMaxRels];
    for (int i = threadIdx.x; i < a.nrel; i += kThreads) s_rel[i] = a.rel[i];
    __syncthreads();
    const int lane = threadIdx.x & 63;
    const int lg = lane & (G - 1);
    const int g0 = lane - lg;
    const int chunks = a.d / VEC;
    const int nrel = a.nrel;
    const int64_t runs = cdiv(a.num_nodes, kNodeRun);
    // this lane's relation (lg < nrel): begin and end of node v's in-edges
    auto load_range = [&](int64_t v, int64_t &b, int64_t &e) {
        b = e = 0;
        if (lg < nrel && v < a.num_nodes) {
            b = s_rel[lg].indptr[v];
            e = s_rel[lg].indptr[v + 1];
        }
    };
    while (true) {
        uint32_t run = 0;
        if (lg == 0) run = atomicAdd(claims, 1u);
        run = __shfl(run, g0, 64);
        if ((int64_t)run >= runs) break;
        const int64_t vb = (int64_t)run * kNodeRun;
        const int64_t v1 = vb + kNodeRun < a.num_nodes ? vb + kNodeRun : a.num_nodes;
        int64_t nb, ne;
        load_range(vb, nb, ne);
        for (int64_t v = vb; v < v1; ++v) {
            const int64_t rb = nb, re = ne;
            load_range(v + 1 < v1 ? v + 1 : a.num_nodes, nb, ne);   // next node, in flight
            // flattened list: relation r covers [start_r, start_r + deg_r)
            const int64_t deg = re - rb;
            int64_t incl = deg;
            for (int off = 1; off < G; off <<= 1) {
                const int64_t o = shfl64(incl, g0 + (lg >= off ? lg - off : lg));
                if (lg >= off) incl += o;
            }
            const int64_t total = shfl64(incl, g0 + G - 1);
            const int64_t start = incl - deg;
            float acc[CPL][VEC], comp[CPL][VEC];
#pragma unroll
            for (int p = 0; p < CPL; ++p)
#pragma unroll
                for (int e = 0; e < VEC; ++e) acc[p][e] = comp[p][e] = 0.f;
            for (int64_t e0 = 0; e0 < total; e0 += G) {
                // lane lg: entry f = e0 + lg -> its relation (last r with start_r <= f and
                // deg_r > 0) and id
                const int64_t f = e0 + lg;
                int rel = 0;
                int64_t pos = 0;
                for (int r = 0; r < nrel; ++r) {
                    const int64_t sr = shfl64(start, g0 + r);
                    const int64_t dr = shfl64(deg, g0 + r);
                    const int64_t br = shfl64(rb, g0 + r);
                    if (f >= sr && f < sr + dr) {
                        rel = r;
                        pos = br + (f - sr);
                    }
                }
                int64_t id = -1;
                if (f < total) {
                    id = s_rel[rel].indices[pos];
                    if (id < 0 || id >= s_rel[rel].rows) {
                        atomicOr(err, 1u);
                        id = -1;
                    }
                }
                const int cnt = total - e0 < G ? (int)(total - e0) : G;
                for (int u0 = 0; u0 < cnt; u0 += U) {
                    uint4 w[U][CPL];
#pragma unroll
                    for (int u = 0; u < U; ++u) {
                        const int src = g0 + ((u0 + u) & (G - 1));
                        const int64_t idu = shfl64(id, src);
                        const int relu = __shfl(rel, src, 64);
                        const bool ok = u0 + u < cnt && idu >= 0;
                        const FeatRel &R = s_rel[relu];
#pragma unroll
                        for (int p = 0; p < CPL; ++p) {
                            const int c = lg + p * G;
                            if (ok && c < chunks)
                                w[u][p] = *(const uint4 *)((const char *)R.feat +
                                                           idu * R.ld * ES + (int64_t)c * 16);
                            else
                                w[u][p] = make_uint4(0u, 0u, 0u, 0u);
                        }
                    }
#pragma unroll
                    for (int u = 0; u < U; ++u)
#pragma unroll
                        for (int p = 0; p < CPL; ++p) add_chunk<BF16>(acc[p], comp[p], w[u][p]);
                }
            }
            const float fc = (float)total;
            const float rc = total > 0 ? 1.f / fc : 0.f;
#pragma unroll
            for (int p = 0; p < CPL; ++p) {
                const int c = lg + p * G;
                if (c >= chunks) continue;
                float q[VEC];
#pragma unroll
                for (int e = 0; e < VEC; ++e) {
                    // one correction step from the exact remainder keeps fp32 output
                    // within an ulp of the quotient
                    const float sum = acc[p][e] - comp[p][e];
                    const float q0 = sum * rc;
                    q[e] = total > 0 ? __builtin_fmaf(__builtin_fmaf(-q0, fc, sum), rc, q0) : 0.f;
                }
                char *o = (char *)a.out + (v * a.out_ld + (int64_t)c * VEC) * ES;
                if constexpr (BF16) {
                    *(uint4 *)o = make_uint4(pack_bf16x2(q[0], q[1]), pack_bf16x2(q[2], q[3]),
                                             pack_bf16x2(q[4], q[5]), pack_bf16x2(q[6], q[7]));
                } else {
                    *(uint4 *)o = make_uint4(__float_as_uint(q[0]), __float_as_uint(q[1]),
                                             __float_as_uint(q[2]), __float_as_uint(q[3]));
                }
            }
        }
    }
}

template <class K>
int64_t resident(K kernel) {
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, kThreads, 0) != hipSuccess ||
        per_cu < 1)
        per_cu = 1;
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) == hipSuccess) {
        hipDeviceProp_t prop;
        if (hipGetDeviceProperties(&prop, dev) == hipSuccess) cus = prop.multiProcessorCount;
    }
    return (int64_t)per_cu * cus;
}

template <bool B, int C>
hipError_t launch(const FeatArgs &a, int G, uint32_t *claims, uint32_t *err, hipStream_t s) {
    const int64_t groups_needed = cdiv(a.num_nodes, kNodeRun);
    int64_t wgs = cdiv(groups_needed, kThreads / G);
    const int64_t cap = resident(k_feature_mean<B, C>);
    if (wgs > cap) wgs = cap;
    if (wgs < 1) wgs = 1;
    hipLaunchKernelGGL((k_feature_mean<B, C>), dim3((unsigned)wgs), dim3(kThreads), 0, s, a, G,
                       claims, err);
    return hipGetLastError();
}

}  // namespace

hipError_t featureless_mean(const FeatArgs &a, uint32_t *words, hipStream_t s) {
    if (a.num_nodes == 0) return hipSuccess;
    const uint32_t zero[2] = {0u, 0u};
    RGCN_HIP_TRY(fill_words(words, zero, sizeof zero, s));   // claims counter, error word
    const bool bf = a.dtype == RGCN_BF16;
    const int chunks = a.d / (bf ? 8 : 4);
    // a group is at least kMinGroup lanes wide, and at least one lane per relation (the
    // lanes r < nrel hold relation r's edge range of the node)
    int G = kMinGroup;
    while ((G < chunks || G < a.nrel) && G < 64) G *= 2;
    const int cpl = (int)cdiv(chunks, G);
    if (cpl == 1) return bf ? launch<true, 1>(a, G, words, words + 1, s)
                            : launch<false, 1>(a, G, words, words + 1, s);
    if (cpl == 2) return bf ? launch<true, 2>(a, G, words, words + 1, s)
                            : launch<false, 2>(a, G, words, words + 1, s);
    if (cpl <= 4) return bf ? launch<true, 4>(a, G, words, words + 1, s)
                            : launch<false, 4>(a, G, words, words + 1, s);
    return hipErrorInvalidValue;
}

}  // namespace rgcn
