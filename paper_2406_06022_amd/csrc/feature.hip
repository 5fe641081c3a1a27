// Feature construction for featureless nodes (Sec. 3.3.2, eq. 1, f the average): for
// every node i of the featureless type, the mean of the feature rows of its in-neighbours
// over the given relations (each relation's source type has a feature table; repeated
// edges count twice; zeros for a node without such neighbours), over the whole graph.
//
// One group of G lanes per node (G = 16-byte chunks per row, rounded up to a power of
// two, at least 8 and at most 64; CPL chunks per lane beyond that).  A persistent grid whose groups
// claim runs of nodes from a counter, so a node of very high degree delays only the group
// that holds it.  A node's in-edges are walked relation by relation: the group's lanes
// load up to 8 neighbour ids at once, then every lane loads its chunk of those 8 rows
// (8 rows in flight per lane) and accumulates in fp32 with compensation.  The mean is
// written in the
// table dtype (bf16 rounded to nearest even).
#include "common.h"

namespace rgcn {

namespace {

constexpr int kThreads = 256;
constexpr int kNodeRun = 16;   // nodes claimed at a time
constexpr int kRowsInFlight = 8;

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
__device__ __forceinline__ void add_chunk(float *acc, float *comp, const FeatRel &r, int64_t row,
                                          int c) {
    const uint4 w = *(const uint4 *)((const char *)r.feat + row * r.ld * (BF16 ? 2 : 4) +
                                     (int64_t)c * 16);
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

template <bool BF16, int CPL>
__global__ __launch_bounds__(kThreads) void k_feature_mean(FeatArgs a, int G, uint32_t *claims,
                                                           uint32_t *err) {
    constexpr int VEC = BF16 ? 8 : 4;
    __shared__ FeatRel s_rel[kMaxRels];
    for (int i = threadIdx.x; i < a.nrel; i += kThreads) s_rel[i] = a.rel[i];
    __syncthreads();
    const int lane = threadIdx.x & 63;
    const int lg = lane & (G - 1);
    const int g0 = lane - lg;
    const int chunks = a.d / VEC;
    const int64_t runs = cdiv(a.num_nodes, kNodeRun);
    while (true) {
        uint32_t run = 0;
        if (lg == 0) run = atomicAdd(claims, 1u);
        run = __shfl(run, g0, 64);
        if ((int64_t)run >= runs) break;
        const int64_t v1 = ((int64_t)run + 1) * kNodeRun < a.num_nodes
                               ? ((int64_t)run + 1) * kNodeRun : a.num_nodes;
        for (int64_t v = (int64_t)run * kNodeRun; v < v1; ++v) {
            float acc[CPL][VEC], comp[CPL][VEC];
#pragma unroll
            for (int p = 0; p < CPL; ++p)
#pragma unroll
                for (int e = 0; e < VEC; ++e) acc[p][e] = comp[p][e] = 0.f;
            int64_t count = 0;
            for (int r = 0; r < a.nrel; ++r) {
                const FeatRel &R = s_rel[r];
                const int64_t b = R.indptr[v], e1 = R.indptr[v + 1];
                count += e1 - b;
                for (int64_t k0 = b; k0 < e1; k0 += kRowsInFlight) {
                    int64_t id = -1;
                    if (lg < kRowsInFlight && k0 + lg < e1) {
                        id = R.indices[k0 + lg];
                        if (id < 0 || id >= R.rows) {
                            atomicOr(err, 1u);
                            id = -1;
                        }
                    }
                    int64_t ids[kRowsInFlight];
#pragma unroll
                    for (int u = 0; u < kRowsInFlight; ++u) ids[u] = shfl64(id, g0 + u);
#pragma unroll
                    for (int p = 0; p < CPL; ++p) {
                        const int c = lg + p * G;
                        if (c >= chunks) continue;
#pragma unroll
                        for (int u = 0; u < kRowsInFlight; ++u)
                            if (ids[u] >= 0) add_chunk<BF16>(acc[p], comp[p], R, ids[u], c);
                    }
                }
            }
            const float fc = (float)count;
            const float rc = count > 0 ? 1.f / fc : 0.f;
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
                    q[e] = count > 0 ? __builtin_fmaf(__builtin_fmaf(-q0, fc, sum), rc, q0) : 0.f;
                }
                char *o = (char *)a.out + (v * a.out_ld + (int64_t)c * VEC) * (BF16 ? 2 : 4);
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
    // a group is at least kRowsInFlight lanes wide: its lanes load the ids it broadcasts
    int G = kRowsInFlight;
    while (G < chunks && G < 64) G *= 2;
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
