// HBM-bound kernels of the block: the forward gather + per-relation segmented mean, the
// backward transposed sum (with the ReLU-input mask and the embedding-gradient
// scatter-add fused in), weight packing, column sums and device-side validation.
//
// Row traffic is done in 16-byte chunks: a "group" of G lanes covers one row of d
// elements (G = chunks per row, at most 64; rows wider than 64 chunks give each lane
// CPL chunks), so a wave moves 64/G rows per load instruction and every row access is a
// run of contiguous 16-byte pieces.
#include "common.h"

namespace rgcn {
namespace {

constexpr int kThreads = 256;
__host__ __device__ inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

struct GroupShape {
    int G;       // lanes per row
    int gpw;     // groups per wave
    int cpl;     // chunks per lane
};
GroupShape group_shape(int chunks) {
    GroupShape g;
    g.cpl = (int)cdiv(chunks, 64);
    g.G = (int)cdiv(chunks, g.cpl);
    g.gpw = 64 / g.G;
    return g;
}

// Accumulate one 16-byte chunk of a source row into 8 (bf16) or 4 (fp32) floats.
template <bool BF16>
__device__ __forceinline__ void acc_chunk(float *acc, const uint4 &v) {
    if constexpr (BF16) {
        acc[0] += bf16_lo(v.x); acc[1] += bf16_hi(v.x);
        acc[2] += bf16_lo(v.y); acc[3] += bf16_hi(v.y);
        acc[4] += bf16_lo(v.z); acc[5] += bf16_hi(v.z);
        acc[6] += bf16_lo(v.w); acc[7] += bf16_hi(v.w);
    } else {
        acc[0] += __uint_as_float(v.x); acc[1] += __uint_as_float(v.y);
        acc[2] += __uint_as_float(v.z); acc[3] += __uint_as_float(v.w);
    }
}

// Broadcast a 64-bit value from absolute lane `src` of the wave.
__device__ __forceinline__ int64_t shfl64(int64_t v, int src) {
    const int lo = __shfl((int)(uint32_t)v, src, 64);
    const int hi = __shfl((int)(uint32_t)((uint64_t)v >> 32), src, 64);
    return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// Forward segments in schedule order (heaviest first), one group of G lanes per segment,
// persistent: group q handles segments q, q + ngroups, ...  A segment is the self-loop
// row of a destination (copied) or the sampled in-edges of a destination row in one
// relation (mean of the gathered source rows; 0 if none).  Lane lg of the group fetches
// edge lg's source index and global row id, the group walks the edges broadcasting row
// addresses, U row loads in flight.  Software pipeline, two round trips per segment:
//   {row ids of this segment, descriptor of the next}  then
//   {rows of this segment, source indices of the next}.
// The sum runs in ascending edge position; one division by the degree.
struct GatherTabs {
    TypeInput in[kMaxTypes];
};

template <bool BF16, int CPL>
__global__ __launch_bounds__(kThreads) void k_gather_mean(const SegDesc *__restrict__ desc,
                                                          int64_t n_seg,
                                                          const FwdSlot *__restrict__ slots,
                                                          int nslots, GatherTabs tabs,
                                                          char *__restrict__ ws, int G, int gpw,
                                                          int chunks) {
    constexpr int VEC = BF16 ? 8 : 4;
    constexpr int ES = BF16 ? 2 : 4;
    constexpr int U = CPL == 1 ? 8 : 4;  // row loads in flight per lane
    __shared__ const int32_t *s_idx[kMaxSlots];
    __shared__ int32_t s_src[kMaxSlots];
    for (int i = threadIdx.x; i < nslots; i += kThreads) {
        s_idx[i] = slots[i].indices;
        s_src[i] = slots[i].src_type;
    }
    __syncthreads();

    const int lane = threadIdx.x & 63;
    const int gi = lane / G;
    const int lg = lane - gi * G;
    const int g0 = gi * G;
    if (gi >= gpw) return;
    const int64_t stride = (int64_t)gridDim.x * (kThreads / 64) * gpw;
    int64_t sg = ((int64_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6)) * gpw + gi;
    if (sg >= n_seg) return;

    // source index of edge e of segment d (self-loop slot: the row itself), -1 past the end
    auto edge_src = [&](const SegDesc &d, int e) -> int64_t {
        if (e >= d.deg) return -1;
        const int32_t *ix = s_idx[(d.info >> 8) & 0xff];
        return ix ? (int64_t)ix[d.k0 + e] : (int64_t)d.k0 + e;
    };
    // byte offset of that source row in its table
    auto row_off = [&](const SegDesc &d, int64_t j) -> int64_t {
        if (j < 0) return 0;
        const TypeInput &in = tabs.in[s_src[(d.info >> 8) & 0xff]];
        const int64_t grow = in.row_ids ? in.row_ids[j] : j;
        return grow * in.ld * ES;
    };

    SegDesc d = desc[sg];
    int64_t j = edge_src(d, lg);
    while (true) {
        const int64_t off0 = row_off(d, j);
        const int64_t sn = sg + stride;
        SegDesc dn = d;
        if (sn < n_seg) dn = desc[sn];
        const char *src = (const char *)tabs.in[s_src[(d.info >> 8) & 0xff]].base;
        const int deg = d.deg;

        float acc[CPL][VEC];
#pragma unroll
        for (int p = 0; p < CPL; ++p)
#pragma unroll
            for (int e = 0; e < VEC; ++e) acc[p][e] = 0.f;

        int64_t jn = -1;
        bool next_issued = false;
        for (int kc = 0; kc < deg; kc += G) {
            const int64_t off = kc == 0 ? off0 : row_off(d, edge_src(d, kc + lg));
            const int n = (deg - kc) < G ? (deg - kc) : G;
            for (int q = 0; q < n; q += U) {
                int64_t o[U];
#pragma unroll
                for (int u = 0; u < U; ++u) o[u] = shfl64(off, g0 + ((q + u) < n ? q + u : 0));
                uint4 v[U][CPL];
#pragma unroll
                for (int u = 0; u < U; ++u)
#pragma unroll
                    for (int p = 0; p < CPL; ++p) {
                        const int c = lg + p * G;
                        v[u][p] = (q + u < n && c < chunks)
                                      ? *(const uint4 *)(src + o[u] + (int64_t)c * 16)
                                      : make_uint4(0, 0, 0, 0);
                    }
                if (!next_issued) {  // next segment's source indices, alongside these rows
                    next_issued = true;
                    if (sn < n_seg) jn = edge_src(dn, lg);
                }
#pragma unroll
                for (int u = 0; u < U; ++u)
#pragma unroll
                    for (int p = 0; p < CPL; ++p) acc_chunk<BF16>(acc[p], v[u][p]);
            }
        }
        if (!next_issued && sn < n_seg) jn = edge_src(dn, lg);

        const float fdeg = (float)deg;
        const uint64_t out16 = ((uint64_t)(d.info & 0xffu) << 32) | d.out_lo;
        char *out = ws + (out16 << 4);
#pragma unroll
        for (int p = 0; p < CPL; ++p) {
            const int c = lg + p * G;
            if (c >= chunks) continue;
            float r[VEC];
#pragma unroll
            for (int e = 0; e < VEC; ++e) r[e] = deg > 0 ? acc[p][e] / fdeg : 0.f;
            uint4 w;
            if constexpr (BF16) {
                w.x = pack_bf16x2(r[0], r[1]); w.y = pack_bf16x2(r[2], r[3]);
                w.z = pack_bf16x2(r[4], r[5]); w.w = pack_bf16x2(r[6], r[7]);
            } else {
                w.x = __float_as_uint(r[0]); w.y = __float_as_uint(r[1]);
                w.z = __float_as_uint(r[2]); w.w = __float_as_uint(r[3]);
            }
            *(uint4 *)(out + (int64_t)c * 16) = w;
        }
        if (sn >= n_seg) break;
        sg = sn;
        d = dn;
        j = jn;
    }
}

// Backward, one group per source row j of one node type, in schedule order:
//   acc = [j < n_dst] dMs_self[j] + sum over relations leaving the type, over the
//         transpose segment of j (ascending destination row), of dMs_r[i]
// where dMs rows already carry the 1/deg factor.  Then the optional ReLU-input mask,
// the dh_src store and the embedding scatter-add demb[row_ids[j]] += acc.
// Lanes first fetch the transpose offsets of up to G relations at once, then the
// destination rows of up to G edges at once (flattened relation by relation), then walk
// the edges broadcasting row addresses, U row loads in flight; the embedding-gradient
// row and the ReLU mask input are requested before the walk.
template <bool BF16IN, int CPL>
__global__ __launch_bounds__(kThreads) void k_transpose_sum(TsumArgs a, int G, int gpw,
                                                            int chunks) {
    constexpr int HES = BF16IN ? 2 : 4;  // element size of the block input (ReLU mask)
    constexpr int U = CPL == 1 ? 8 : 4;
    const int lane = threadIdx.x & 63;
    const int gi = lane / G;
    const int lg = lane - gi * G;
    const int g0 = gi * G;
    if (gi >= gpw) return;
    const int64_t wave = ((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6;
    const int64_t g = wave * gpw + gi;
    if (g >= a.n_rows) return;
    const int64_t j = a.order[g];
    const int64_t grow = a.in.row_ids ? a.in.row_ids[j] : j;

    // early requests: embedding-gradient row (read-add-write), ReLU mask input, self term
    float4 old[CPL];
    float hm[CPL][4];
    float acc[CPL][4];
#pragma unroll
    for (int p = 0; p < CPL; ++p) {
        const int c = lg + p * G;
        const bool okc = c < chunks;
        old[p] = (a.demb && a.ids_unique && okc)
                     ? *(const float4 *)(a.demb + grow * a.d_in + (int64_t)c * 4)
                     : make_float4(0.f, 0.f, 0.f, 0.f);
        if (a.input_relu && okc) {
            const char *hp = (const char *)a.in.base + (grow * a.in.ld + (int64_t)c * 4) * HES;
            if constexpr (BF16IN) {
                const uint2 hv = *(const uint2 *)hp;
                hm[p][0] = bf16_lo(hv.x); hm[p][1] = bf16_hi(hv.x);
                hm[p][2] = bf16_lo(hv.y); hm[p][3] = bf16_hi(hv.y);
            } else {
                const float4 hv = *(const float4 *)hp;
                hm[p][0] = hv.x; hm[p][1] = hv.y; hm[p][2] = hv.z; hm[p][3] = hv.w;
            }
        } else {
            hm[p][0] = hm[p][1] = hm[p][2] = hm[p][3] = 1.f;
        }
        float4 sv = make_float4(0.f, 0.f, 0.f, 0.f);
        if (a.self_dms && j < a.n_dst && okc)
            sv = *(const float4 *)(a.self_dms + j * a.self_ld + (int64_t)c * 4);
        acc[p][0] = sv.x; acc[p][1] = sv.y; acc[p][2] = sv.z; acc[p][3] = sv.w;
    }

    for (int r0 = 0; r0 < a.nrel; r0 += G) {
        // lane lg: transpose segment of relation r0 + lg
        const int nr = (a.nrel - r0) < G ? (a.nrel - r0) : G;
        int p0 = 0, cnt = 0;
        if (lg < nr) {
            const int32_t *ip = a.rel[r0 + lg].csc_indptr;
            p0 = ip[j];
            cnt = ip[j + 1] - p0;
        }
        int total = 0;
        for (int r = 0; r < nr; ++r) total += __shfl(cnt, g0 + r, 64);
        for (int ec = 0; ec < total; ec += G) {
            // lane lg: flattened edge ec + lg -> (relation, position) -> dMs row address.
            // Every lane of the group runs the shuffles; only the owner loads.
            const int e = ec + lg;
            uint64_t addr = 0;
            int base = 0;
            for (int r = 0; r < nr; ++r) {
                const int cr = __shfl(cnt, g0 + r, 64);
                const int pr = __shfl(p0, g0 + r, 64);
                if (e < total && e >= base && e < base + cr) {
                    const TsumRel &rel = a.rel[r0 + r];
                    const int64_t i = rel.csc_dst[pr + (e - base)];
                    addr = (uint64_t)(uintptr_t)(rel.dms + i * rel.dms_ld);
                }
                base += cr;
            }
            const int n = (total - ec) < G ? (total - ec) : G;
            for (int q = 0; q < n; q += U) {
                int64_t o[U];
#pragma unroll
                for (int u = 0; u < U; ++u)
                    o[u] = shfl64((int64_t)addr, g0 + ((q + u) < n ? q + u : 0));
                float4 v[U][CPL];
#pragma unroll
                for (int u = 0; u < U; ++u)
#pragma unroll
                    for (int p = 0; p < CPL; ++p) {
                        const int c = lg + p * G;
                        const float *rp = (const float *)(uintptr_t)(uint64_t)o[u];
                        v[u][p] = (q + u < n && c < chunks) ? *(const float4 *)(rp + (int64_t)c * 4)
                                                            : make_float4(0.f, 0.f, 0.f, 0.f);
                    }
#pragma unroll
                for (int u = 0; u < U; ++u)
#pragma unroll
                    for (int p = 0; p < CPL; ++p) {
                        acc[p][0] += v[u][p].x; acc[p][1] += v[u][p].y;
                        acc[p][2] += v[u][p].z; acc[p][3] += v[u][p].w;
                    }
            }
        }
    }
#pragma unroll
    for (int p = 0; p < CPL; ++p) {
        const int c = lg + p * G;
        if (c >= chunks) continue;
        if (a.input_relu) {
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[p][e] = hm[p][e] > 0.f ? acc[p][e] : 0.f;
        }
        const float4 res = make_float4(acc[p][0], acc[p][1], acc[p][2], acc[p][3]);
        if (a.dh) *(float4 *)(a.dh + j * a.d_in + (int64_t)c * 4) = res;
        if (a.demb) {
            float *dp = a.demb + grow * a.d_in + (int64_t)c * 4;
            if (a.ids_unique) {
                *(float4 *)dp = make_float4(old[p].x + res.x, old[p].y + res.y, old[p].z + res.z,
                                            old[p].w + res.w);
            } else {
                unsafeAtomicAdd(dp + 0, res.x);
                unsafeAtomicAdd(dp + 1, res.y);
                unsafeAtomicAdd(dp + 2, res.z);
                unsafeAtomicAdd(dp + 3, res.w);
            }
        }
    }
}

// WcatT[n][s*d_in + c] = W_s[c][n]: the forward transform's weights, K-contiguous.
struct WSlots {
    const void *w[kMaxSlots];
};
template <typename T>
__global__ __launch_bounds__(kThreads) void k_pack_weights(WSlots ws, int nslots, int d_in,
                                                           int d_out, T *out) {
    const int64_t K = (int64_t)nslots * d_in;
    const int64_t total = K * d_out;
    for (int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * kThreads) {
        const int64_t n = e / K, kk = e - n * K;
        const int64_t s = kk / d_in, c = kk - s * d_in;
        out[e] = ((const T *)ws.w[s])[c * d_out + n];
    }
}

// Deterministic column sums: partial[split][o] over a fixed row range, then a fixed-order
// sum over splits.
__global__ __launch_bounds__(kThreads) void k_colsum_partial(const float *dy, int64_t rows,
                                                             int cols, int64_t rows_per_split,
                                                             float *partial) {
    const int o = blockIdx.x * kThreads + threadIdx.x;
    if (o >= cols) return;
    const int64_t r0 = (int64_t)blockIdx.y * rows_per_split;
    const int64_t r1 = r0 + rows_per_split < rows ? r0 + rows_per_split : rows;
    float acc = 0.f;
    for (int64_t r = r0; r < r1; ++r) acc += dy[r * cols + o];
    partial[(int64_t)blockIdx.y * cols + o] = acc;
}
__global__ __launch_bounds__(kThreads) void k_colsum_final(const float *partial, int splits,
                                                           int cols, float *out) {
    const int o = blockIdx.x * kThreads + threadIdx.x;
    if (o >= cols) return;
    float acc = 0.f;
    for (int sp = 0; sp < splits; ++sp) acc += partial[(int64_t)sp * cols + o];
    out[o] = acc;
}

__global__ __launch_bounds__(kThreads) void k_zero_f32(float *p, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i < n) p[i] = 0.f;
}

// err bit 1: malformed CSR offsets; bit 2: index out of range.
__global__ __launch_bounds__(kThreads) void k_validate_csr(const int32_t *indptr,
                                                           const int32_t *indices,
                                                           int64_t n_dst, int64_t nnz,
                                                           int64_t n_src, uint32_t *err) {
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i > n_dst) return;
    uint32_t bad = 0;
    const int64_t a = indptr[i];
    if (i == 0 && a != 0) bad |= 1u;
    if (i == n_dst && a != nnz) bad |= 1u;
    if (i < n_dst) {
        const int64_t b = indptr[i + 1];
        if (b < a || a < 0 || b > nnz) {
            bad |= 1u;
        } else {
            for (int64_t k = a; k < b; ++k) {
                const int64_t x = indices[k];
                if (x < 0 || x >= n_src) { bad |= 2u; break; }
            }
        }
    }
    if (bad) atomicOr(err, bad);
}
__global__ __launch_bounds__(kThreads) void k_validate_ids(const int64_t *ids, int64_t n,
                                                           int64_t num_rows, uint32_t *err) {
    const int64_t j = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (j >= n) return;
    const int64_t x = ids[j];
    if (x < 0 || x >= num_rows) atomicOr(err, 2u);
}

}  // namespace

// Workgroups of `kernel` that fit on the device at once (persistent grids).
template <class K>
int64_t resident_wgs(K kernel) {
    static int cus = 0;
    if (cus == 0) {
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            cus <= 0)
            cus = 256;
    }
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, kThreads, 0) != hipSuccess ||
        per_cu <= 0)
        per_cu = 1;
    return (int64_t)per_cu * cus;
}

template <bool B, int C>
hipError_t launch_gather(const SegDesc *desc, int64_t n_seg, const FwdSlot *slots_dev,
                         int nslots, const GatherTabs &tabs, char *ws_base, const GroupShape &gs,
                         int chunks, hipStream_t s) {
    const int64_t groups_per_wg = (int64_t)(kThreads / 64) * gs.gpw;
    int64_t wgs = cdiv(n_seg, groups_per_wg);
    const int64_t cap = resident_wgs(k_gather_mean<B, C>);
    if (wgs > cap) wgs = cap;
    hipLaunchKernelGGL((k_gather_mean<B, C>), dim3((unsigned)wgs), dim3(kThreads), 0, s, desc,
                       n_seg, slots_dev, nslots, tabs, ws_base, gs.G, gs.gpw, chunks);
    return hipGetLastError();
}

hipError_t gather_mean(rgcn_dtype dt, int d_in, const SegDesc *desc, int64_t n_seg,
                       const FwdSlot *slots_dev, int nslots, const TypeInput *in,
                       char *ws_base, hipStream_t s) {
    if (n_seg == 0) return hipSuccess;
    const bool bf = dt == RGCN_BF16;
    const int chunks = bf ? d_in / 8 : d_in / 4;
    const GroupShape gs = group_shape(chunks);
    GatherTabs tabs;
    for (int t = 0; t < kMaxTypes; ++t) tabs.in[t] = in[t];
    if (gs.cpl == 1)
        return bf ? launch_gather<true, 1>(desc, n_seg, slots_dev, nslots, tabs, ws_base, gs, chunks, s)
                  : launch_gather<false, 1>(desc, n_seg, slots_dev, nslots, tabs, ws_base, gs, chunks, s);
    if (gs.cpl == 2)
        return bf ? launch_gather<true, 2>(desc, n_seg, slots_dev, nslots, tabs, ws_base, gs, chunks, s)
                  : launch_gather<false, 2>(desc, n_seg, slots_dev, nslots, tabs, ws_base, gs, chunks, s);
    if (gs.cpl <= 4)
        return bf ? launch_gather<true, 4>(desc, n_seg, slots_dev, nslots, tabs, ws_base, gs, chunks, s)
                  : launch_gather<false, 4>(desc, n_seg, slots_dev, nslots, tabs, ws_base, gs, chunks, s);
    return hipErrorInvalidValue;
}

hipError_t transpose_sum(rgcn_dtype dt, const TsumArgs &a, hipStream_t s) {
    if (a.n_rows == 0) return hipSuccess;
    const int chunks = a.d_in / 4;
    const GroupShape gs = group_shape(chunks);
    const int64_t waves = cdiv(a.n_rows, gs.gpw);
    const dim3 grid((unsigned)cdiv(waves, kThreads / 64));
    const bool bf = dt == RGCN_BF16;
#define RGCN_TS(B, C) \
    hipLaunchKernelGGL((k_transpose_sum<B, C>), grid, dim3(kThreads), 0, s, a, gs.G, gs.gpw, chunks)
    if (gs.cpl == 1) { if (bf) RGCN_TS(true, 1); else RGCN_TS(false, 1); }
    else if (gs.cpl == 2) { if (bf) RGCN_TS(true, 2); else RGCN_TS(false, 2); }
    else if (gs.cpl <= 4) { if (bf) RGCN_TS(true, 4); else RGCN_TS(false, 4); }
    else return hipErrorInvalidValue;
#undef RGCN_TS
    return hipGetLastError();
}

hipError_t pack_weights(rgcn_dtype dt, int d_in, int d_out, const void *const *w_slots,
                        int nslots, void *wcat_t, hipStream_t s) {
    WSlots ws;
    for (int i = 0; i < kMaxSlots; ++i) ws.w[i] = i < nslots ? w_slots[i] : nullptr;
    const int64_t total = (int64_t)nslots * d_in * d_out;
    if (total == 0) return hipSuccess;
    const int64_t blocks = cdiv(total, kThreads) < 65536 ? cdiv(total, kThreads) : 65536;
    if (dt == RGCN_BF16)
        hipLaunchKernelGGL(k_pack_weights<uint16_t>, dim3((unsigned)blocks), dim3(kThreads), 0,
                           s, ws, nslots, d_in, d_out, (uint16_t *)wcat_t);
    else
        hipLaunchKernelGGL(k_pack_weights<float>, dim3((unsigned)blocks), dim3(kThreads), 0, s,
                           ws, nslots, d_in, d_out, (float *)wcat_t);
    return hipGetLastError();
}

static int64_t colsum_splits(int64_t rows) {
    int64_t sp = cdiv(rows, 2048);
    return sp < 1 ? 1 : (sp > 1024 ? 1024 : sp);
}
size_t column_sums_temp_bytes(int64_t rows, int cols) {
    return (size_t)colsum_splits(rows) * cols * 4 + 256;
}
hipError_t column_sums(const float *dy, int64_t rows, int cols, float *out, float *partial,
                       int64_t max_splits, hipStream_t s) {
    (void)max_splits;
    if (cols == 0) return hipSuccess;
    if (rows == 0) {
        hipLaunchKernelGGL(k_zero_f32, dim3((unsigned)cdiv(cols, kThreads)), dim3(kThreads), 0, s,
                           out, (int64_t)cols);
        return hipGetLastError();
    }
    const int64_t sp = colsum_splits(rows);
    const int64_t rps = cdiv(rows, sp);
    const int64_t nsp = cdiv(rows, rps);
    hipLaunchKernelGGL(k_colsum_partial, dim3((unsigned)cdiv(cols, kThreads), (unsigned)nsp),
                       dim3(kThreads), 0, s, dy, rows, cols, rps, partial);
    RGCN_HIP_TRY(hipGetLastError());
    hipLaunchKernelGGL(k_colsum_final, dim3((unsigned)cdiv(cols, kThreads)), dim3(kThreads), 0, s,
                       partial, (int)nsp, cols, out);
    return hipGetLastError();
}

hipError_t validate_csr(const int32_t *indptr, const int32_t *indices, int64_t n_dst,
                        int64_t nnz, int64_t n_src, uint32_t *err, hipStream_t s) {
    hipLaunchKernelGGL(k_validate_csr, dim3((unsigned)cdiv(n_dst + 1, kThreads)), dim3(kThreads),
                       0, s, indptr, indices, n_dst, nnz, n_src, err);
    return hipGetLastError();
}

hipError_t validate_ids(const int64_t *ids, int64_t n, int64_t num_rows, uint32_t *err,
                        hipStream_t s) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(k_validate_ids, dim3((unsigned)cdiv(n, kThreads)), dim3(kThreads), 0, s,
                       ids, n, num_rows, err);
    return hipGetLastError();
}

}  // namespace rgcn
