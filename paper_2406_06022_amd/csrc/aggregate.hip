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

struct GatherIO {
    TypeInput in[kMaxTypes];
    void *mcat[kMaxTypes];
    int64_t mcat_ld[kMaxTypes];   // elements per Mcat row
};

// One group per forward segment, in schedule order (heaviest segments first).  A
// segment is the self-loop row of a destination (copied) or the sampled in-edges of a
// destination row in one relation (mean of the gathered source rows; 0 if none).  The
// sum runs in ascending edge position; the result is divided once by the degree.
template <bool BF16, int CPL>
__global__ __launch_bounds__(kThreads) void k_gather_mean(const int32_t *__restrict__ order,
                                                          int64_t n_seg,
                                                          const FwdSlot *__restrict__ slots,
                                                          int nslots, GatherIO io, int G,
                                                          int gpw, int chunks) {
    constexpr int VEC = BF16 ? 8 : 4;
    constexpr int ES = BF16 ? 2 : 4;
    constexpr int U = 4;  // independent row loads in flight per lane
    __shared__ int64_t s_base[kMaxSlots];
    for (int i = threadIdx.x; i < nslots; i += kThreads) s_base[i] = slots[i].seg_base;
    __syncthreads();

    const int lane = threadIdx.x & 63;
    const int gi = lane / G;
    const int lg = lane - gi * G;
    if (gi >= gpw) return;
    const int64_t wave = ((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6;
    const int64_t g = wave * gpw + gi;
    if (g >= n_seg) return;

    const int64_t seg = order[g];
    int lo = 0, hi = nslots - 1;
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if (s_base[mid] <= seg) lo = mid; else hi = mid - 1;
    }
    const FwdSlot sl = slots[lo];
    const int64_t row = seg - sl.seg_base;
    const TypeInput in = io.in[sl.src_type];
    const char *src = (const char *)in.base;
    const int64_t ld_bytes = in.ld * ES;

    int64_t k0 = row, k1 = row + 1;  // self-loop slot: the row itself
    if (sl.indptr) {
        k0 = sl.indptr[row];
        k1 = sl.indptr[row + 1];
    }
    float acc[CPL][VEC];
#pragma unroll
    for (int p = 0; p < CPL; ++p)
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[p][e] = 0.f;

    for (int64_t k = k0; k < k1; k += U) {
        const char *rp[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t kk = k + u;
            rp[u] = nullptr;
            if (kk < k1) {
                const int64_t j = sl.indices ? (int64_t)sl.indices[kk] : kk;
                const int64_t grow = in.row_ids ? in.row_ids[j] : j;
                rp[u] = src + grow * ld_bytes;
            }
        }
        uint4 v[U][CPL];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int p = 0; p < CPL; ++p) {
                const int c = lg + p * G;
                if (rp[u] && c < chunks) v[u][p] = *(const uint4 *)(rp[u] + (int64_t)c * 16);
                else v[u][p] = make_uint4(0, 0, 0, 0);
            }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int p = 0; p < CPL; ++p) acc_chunk<BF16>(acc[p], v[u][p]);
    }

    const int64_t deg = k1 - k0;
    const float fdeg = (float)deg;
    char *out = (char *)io.mcat[sl.dst_type] +
                (row * io.mcat_ld[sl.dst_type] + sl.col_off) * ES;
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
}

// Backward, one group per source row j of one node type, in schedule order:
//   acc = [j < n_dst] dMs_self[j] + sum over relations leaving the type, over the
//         transpose segment of j (ascending destination row), of dMs_r[i]
// where dMs rows already carry the 1/deg factor.  Then the optional ReLU-input mask,
// the dh_src store and the embedding scatter-add demb[row_ids[j]] += acc.
template <bool BF16IN, int CPL>
__global__ __launch_bounds__(kThreads) void k_transpose_sum(TsumArgs a, int G, int gpw,
                                                            int chunks) {
    constexpr int HES = BF16IN ? 2 : 4;  // element size of the block input (ReLU mask)
    constexpr int U = 4;
    const int lane = threadIdx.x & 63;
    const int gi = lane / G;
    const int lg = lane - gi * G;
    if (gi >= gpw) return;
    const int64_t wave = ((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6;
    const int64_t g = wave * gpw + gi;
    if (g >= a.n_rows) return;
    const int64_t j = a.order[g];

    float acc[CPL][4];
#pragma unroll
    for (int p = 0; p < CPL; ++p) {
        const int c = lg + p * G;
        float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
        if (a.self_dms && j < a.n_dst && c < chunks)
            s = *(const float4 *)(a.self_dms + j * a.self_ld + (int64_t)c * 4);
        acc[p][0] = s.x; acc[p][1] = s.y; acc[p][2] = s.z; acc[p][3] = s.w;
    }
    for (int r = 0; r < a.nrel; ++r) {
        const TsumRel rel = a.rel[r];
        const int64_t p0 = rel.csc_indptr[j], p1 = rel.csc_indptr[j + 1];
        for (int64_t q = p0; q < p1; q += U) {
            const float *rp[U];
#pragma unroll
            for (int u = 0; u < U; ++u)
                rp[u] = (q + u < p1) ? rel.dms + (int64_t)rel.csc_dst[q + u] * rel.dms_ld : nullptr;
            float4 v[U][CPL];
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int p = 0; p < CPL; ++p) {
                    const int c = lg + p * G;
                    v[u][p] = (rp[u] && c < chunks) ? *(const float4 *)(rp[u] + (int64_t)c * 4)
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
    const int64_t grow = a.in.row_ids ? a.in.row_ids[j] : j;
#pragma unroll
    for (int p = 0; p < CPL; ++p) {
        const int c = lg + p * G;
        if (c >= chunks) continue;
        if (a.input_relu) {
            const char *hp = (const char *)a.in.base + (grow * a.in.ld + (int64_t)c * 4) * HES;
            float h[4];
            if constexpr (BF16IN) {
                const uint2 hv = *(const uint2 *)hp;
                h[0] = bf16_lo(hv.x); h[1] = bf16_hi(hv.x); h[2] = bf16_lo(hv.y); h[3] = bf16_hi(hv.y);
            } else {
                const float4 hv = *(const float4 *)hp;
                h[0] = hv.x; h[1] = hv.y; h[2] = hv.z; h[3] = hv.w;
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[p][e] = h[e] > 0.f ? acc[p][e] : 0.f;
        }
        const float4 res = make_float4(acc[p][0], acc[p][1], acc[p][2], acc[p][3]);
        if (a.dh) *(float4 *)(a.dh + j * a.d_in + (int64_t)c * 4) = res;
        if (a.demb) {
            float *dp = a.demb + grow * a.d_in + (int64_t)c * 4;
            if (a.ids_unique) {
                float4 old = *(float4 *)dp;
                old.x += res.x; old.y += res.y; old.z += res.z; old.w += res.w;
                *(float4 *)dp = old;
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

hipError_t gather_mean(rgcn_dtype dt, int d_in, const int32_t *order, int64_t n_seg,
                       const FwdSlot *slots_dev, int nslots, const TypeInput *in,
                       void *const *mcat, const int64_t *mcat_ld, hipStream_t s) {
    if (n_seg == 0) return hipSuccess;
    const bool bf = dt == RGCN_BF16;
    const int chunks = bf ? d_in / 8 : d_in / 4;
    const GroupShape gs = group_shape(chunks);
    GatherIO io;
    for (int t = 0; t < kMaxTypes; ++t) {
        io.in[t] = in[t];
        io.mcat[t] = mcat[t];
        io.mcat_ld[t] = mcat_ld[t];
    }
    const int64_t waves = cdiv(n_seg, gs.gpw);
    const dim3 grid((unsigned)cdiv(waves, kThreads / 64));
#define RGCN_GM(B, C)                                                                        \
    hipLaunchKernelGGL((k_gather_mean<B, C>), grid, dim3(kThreads), 0, s, order, n_seg,      \
                       slots_dev, nslots, io, gs.G, gs.gpw, chunks)
    if (gs.cpl == 1) { if (bf) RGCN_GM(true, 1); else RGCN_GM(false, 1); }
    else if (gs.cpl == 2) { if (bf) RGCN_GM(true, 2); else RGCN_GM(false, 2); }
    else if (gs.cpl <= 4) { if (bf) RGCN_GM(true, 4); else RGCN_GM(false, 4); }
    else return hipErrorInvalidValue;
#undef RGCN_GM
    return hipGetLastError();
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
