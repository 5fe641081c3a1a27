// Integer plan of a block: exclusive scans, stable counting sorts by small keys (the
// degree-sorted schedules) and LSD radix sorts of edges by source row (the CSC
// transpose).  Everything here is integer arithmetic and deterministic: the result does
// not depend on scheduling, so it is bit-exact against a sequential stable sort.
#include "common.h"

namespace rgcn {
// exclusive scan whose kernels do nothing while *gate is zero (gate NULL: always run)
hipError_t scan_gated(const int32_t *in, int32_t *out, int64_t n, void *temp,
                      const uint32_t *gate, hipStream_t s);

namespace {

constexpr int kThreads = 256;
constexpr int kScanRounds = 4;                        // int4 per thread per round
constexpr int kScanTile = kThreads * 4 * kScanRounds;  // 4096
constexpr int kSortItems = 16;
constexpr int kSortTile = kThreads * kSortItems;     // 4096

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
__host__ __device__ inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Exclusive scan of one value per thread over a 256-thread workgroup: inclusive scans
// within the waves (shuffles), then the four wave totals through LDS (two barriers).
__device__ int wg_exclusive_scan(int v, int *total) {
    __shared__ int wsum[kThreads / 64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int x = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(x, off, 64);
        if (lane >= off) x += y;
    }
    if (lane == 63) wsum[wave] = x;
    __syncthreads();
    int below = 0, all = 0;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) {
        const int t = wsum[w];
        below += w < wave ? t : 0;
        all += t;
    }
    __syncthreads();   // wsum is rewritten by the next call
    *total = all;
    return below + x - v;
}

// ---------------------------------------------------------------- scan (3 kernels)
// A gate (NULL = none) is a device word: kernels given one do nothing while it is zero.
// Tiles of 4096 values: in round u thread t holds values 4 (256 u + t) .. + 3 (one 16-byte
// access when the arrays are 16-byte aligned, VEC), so every access of a round is
// contiguous across the workgroup.
__device__ __forceinline__ bool gated_off(const uint32_t *gate) { return gate && *gate == 0u; }

template <bool VEC>
__device__ __forceinline__ void scan_load4(const int32_t *in, int64_t i, int64_t n, int v[4]) {
    if (VEC && i + 4 <= n) {
        const int4 q = *(const int4 *)(in + i);
        v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
        return;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = i + e < n ? in[i + e] : 0;
}

template <bool VEC>
__global__ __launch_bounds__(kThreads) void k_scan_reduce(const int32_t *in, int64_t n,
                                                          int32_t *partial, const uint32_t *gate) {
    if (gated_off(gate)) return;
    const int64_t base = (int64_t)blockIdx.x * kScanTile;
    int sum = 0;
#pragma unroll
    for (int u = 0; u < kScanRounds; ++u) {
        int v[4];
        scan_load4<VEC>(in, base + 4 * ((int64_t)u * kThreads + threadIdx.x), n, v);
        sum += v[0] + v[1] + v[2] + v[3];
    }
    int total;
    wg_exclusive_scan(sum, &total);
    if (threadIdx.x == 0) partial[blockIdx.x] = total;
}

__global__ __launch_bounds__(kThreads) void k_scan_partials(int32_t *partial, int64_t nb,
                                                            const uint32_t *gate) {
    if (gated_off(gate)) return;
    constexpr int kItems = kScanTile / kThreads;
    int carry = 0;
    for (int64_t c0 = 0; c0 < nb; c0 += kScanTile) {
        int v[kItems];
        int sum = 0;
        for (int u = 0; u < kItems; ++u) {
            int64_t i = c0 + (int64_t)threadIdx.x * kItems + u;
            v[u] = i < nb ? partial[i] : 0;
            sum += v[u];
        }
        int total;
        int pre = wg_exclusive_scan(sum, &total) + carry;
        for (int u = 0; u < kItems; ++u) {
            int64_t i = c0 + (int64_t)threadIdx.x * kItems + u;
            if (i < nb) partial[i] = pre;
            pre += v[u];
        }
        carry += total;
    }
}

// partial NULL: a single tile (offset 0).  in may equal out: every value of a round is
// read before that round's values are written.
template <bool VEC>
__global__ __launch_bounds__(kThreads) void k_scan_apply(const int32_t *in, int32_t *out,
                                                         int64_t n, const int32_t *partial,
                                                         const uint32_t *gate) {
    if (gated_off(gate)) return;
    const int64_t base = (int64_t)blockIdx.x * kScanTile;
    int carry = partial ? partial[blockIdx.x] : 0;
#pragma unroll
    for (int u = 0; u < kScanRounds; ++u) {
        const int64_t i = base + 4 * ((int64_t)u * kThreads + threadIdx.x);
        int v[4];
        scan_load4<VEC>(in, i, n, v);
        int total;
        const int pre = wg_exclusive_scan(v[0] + v[1] + v[2] + v[3], &total) + carry;
        const int o[4] = {pre, pre + v[0], pre + v[0] + v[1], pre + v[0] + v[1] + v[2]};
        if (VEC && i + 4 <= n) {
            *(int4 *)(out + i) = make_int4(o[0], o[1], o[2], o[3]);
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (i + e < n) out[i + e] = o[e];
        }
        carry += total;
    }
}

// ---------------------------------------------------------------- stable bucket sort
// Items of a tile are visited in "striped" order: round u, thread t -> item
// tile*4096 + u*256 + t.  That order is ascending item index, so ranking items of equal
// key in that order keeps the sort stable.
template <int NB, class KeyFn>
__global__ __launch_bounds__(kThreads) void k_bucket_hist(KeyFn kf, int64_t n, int32_t *hist,
                                                          int32_t ntiles, const uint32_t *gate) {
    if (gated_off(gate)) return;
    __shared__ int32_t h[NB];
    for (int b = threadIdx.x; b < NB; b += kThreads) h[b] = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kSortTile;
    for (int u = 0; u < kSortItems; ++u) {
        int64_t idx = base + (int64_t)u * kThreads + threadIdx.x;
        if (idx < n) atomicAdd(&h[kf(idx)], 1);
    }
    __syncthreads();
    for (int b = threadIdx.x; b < NB; b += kThreads)
        hist[(int64_t)b * ntiles + blockIdx.x] = h[b];
}

template <int NB, int BITS, class KeyFn, class PutFn>
__global__ __launch_bounds__(kThreads) void k_bucket_scatter(KeyFn kf, PutFn put, int64_t n,
                                                             const int32_t *offs,
                                                             int32_t ntiles,
                                                             const uint32_t *gate) {
    if (gated_off(gate)) return;
    __shared__ int32_t run[NB];
    __shared__ int32_t wcnt[kThreads / 64][NB];
    for (int b = threadIdx.x; b < NB; b += kThreads) {
        run[b] = offs[(int64_t)b * ntiles + blockIdx.x];
        for (int w = 0; w < kThreads / 64; ++w) wcnt[w][b] = 0;
    }
    __syncthreads();
    const int wave = threadIdx.x >> 6;
    const int64_t base = (int64_t)blockIdx.x * kSortTile;
    for (int u = 0; u < kSortItems; ++u) {
        const int64_t idx = base + (int64_t)u * kThreads + threadIdx.x;
        const bool valid = idx < n;
        const int key = valid ? kf(idx) : 0;
        // lanes of this wave holding the same key (all lanes take part in every ballot)
        uint64_t peers = __ballot(valid);
        for (int b = 0; b < BITS; ++b) {
            const bool bit = (key >> b) & 1;
            const uint64_t m = __ballot(bit);
            peers &= bit ? m : ~m;
        }
        const int rank = lanes_below(peers);
        if (valid && rank == 0) wcnt[wave][key] = __popcll(peers);
        __syncthreads();
        if (valid) {
            int pos = run[key] + rank;
            for (int w = 0; w < wave; ++w) pos += wcnt[w][key];
            put(pos, idx);
        }
        __syncthreads();
        for (int b = threadIdx.x; b < NB; b += kThreads) {
            int add = 0;
            for (int w = 0; w < kThreads / 64; ++w) {
                add += wcnt[w][b];
                wcnt[w][b] = 0;
            }
            run[b] += add;
        }
        __syncthreads();
    }
}

template <int NB, int BITS, class KeyFn, class PutFn>
hipError_t bucket_sort(const KeyFn &kf, const PutFn &put, int64_t n, void *temp,
                       hipStream_t s, const uint32_t *gate = nullptr) {
    if (n == 0) return hipSuccess;
    const int64_t ntiles = cdiv(n, kSortTile);
    int32_t *hist = (int32_t *)temp;
    void *scan_tmp = (char *)temp + align_up((size_t)NB * ntiles * 4, 256);
    hipLaunchKernelGGL((k_bucket_hist<NB, KeyFn>), dim3((unsigned)ntiles), dim3(kThreads), 0,
                       s, kf, n, hist, (int32_t)ntiles, gate);
    RGCN_HIP_TRY(hipGetLastError());
    RGCN_HIP_TRY(scan_gated(hist, hist, (int64_t)NB * ntiles, scan_tmp, gate, s));
    hipLaunchKernelGGL((k_bucket_scatter<NB, BITS, KeyFn, PutFn>), dim3((unsigned)ntiles),
                       dim3(kThreads), 0, s, kf, put, n, hist, (int32_t)ntiles, gate);
    return hipGetLastError();
}

// Schedule key of a segment of degree deg: segments of at most 32 edges share the last key
// (they keep their enumeration order, so neighbours stay together); heavier ones come
// first, one key per power of two, heaviest first.
__device__ __forceinline__ int degree_key(int64_t deg) {
    if (deg <= 32) return kSchedBuckets - 1;
    const int lg = 63 - __clzll((unsigned long long)deg);   // floor(log2 deg) >= 5
    const int k = (kSchedBuckets - 2) - (lg - 5);
    return k > 0 ? k : 0;
}

// Forward segments: key of segment id = degree key of its (slot, row).
struct FwdKey {
    int32_t nslots;
    int64_t base[kMaxSlots];
    const int32_t *indptr[kMaxSlots];
    __device__ int operator()(int64_t seg) const {
        int lo = 0, hi = nslots - 1;           // last slot with base <= seg
        while (lo < hi) {
            int mid = (lo + hi + 1) >> 1;
            if (base[mid] <= seg) lo = mid; else hi = mid - 1;
        }
        const int32_t *ip = indptr[lo];
        if (!ip) return degree_key(1);
        int64_t row = seg - base[lo];
        return degree_key((int64_t)ip[row + 1] - ip[row]);
    }
};

struct PutIndex {
    int32_t *order;
    __device__ void operator()(int pos, int64_t idx) const { order[pos] = (int32_t)idx; }
};

// Backward rows of one source type: key = degree key of the in-degree summed over the
// relations leaving the type.
struct BwdKey {
    BwdKeyRels rels;
    // transpose degree of row j summed over the relations leaving the type
    // (four relations' loads in flight at a time: past the last relation the first one is
    // read again and not counted, so the loads need no branch)
    __device__ int64_t degree(int64_t j) const {
        int64_t deg = 0;
        for (int r0 = 0; r0 < rels.count; r0 += 4) {
            int32_t a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int32_t *ip = rels.csc_indptr[r0 + i < rels.count ? r0 + i : 0] + j;
                a[i] = ip[0];
                b[i] = ip[1];
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) deg += r0 + i < rels.count ? (int64_t)b[i] - a[i] : 0;
        }
        return deg;
    }
    __device__ int operator()(int64_t j) const { return degree_key(degree(j)); }
};

// Radix pass: the digit (key >> shift) & mask.
struct RadixKey {
    const uint32_t *keys;
    int shift;
    uint32_t mask;
    __device__ int operator()(int64_t i) const { return (int)((keys[i] >> shift) & mask); }
};
struct RadixPut {
    const uint32_t *kin;
    const int32_t *vin;
    uint32_t *kout;
    int32_t *vout;
    __device__ void operator()(int pos, int64_t i) const {
        kout[pos] = kin[i];
        vout[pos] = vin[i];
    }
};

// Edges of every relation taking part in the combined transpose, as (key, value) pairs:
// key = koff_r + source row (disjoint key ranges per relation), value = destination row;
// relation r's edges occupy positions [E_r, E_r + nnz_r) in input order.  Also counts the
// edges per key.  The relations' destination rows are concatenated, and so are their
// edges, in the same order, so the edges of 64 consecutive rows are one contiguous range:
// a wave takes 64 rows (lane l: row x0 + l, its relation and first edge), then walks the
// range 64 edges at a time, lane l on edge g, whose row it finds by a binary search over
// the lanes' first edges (wave shuffles).  Index reads and key / value writes are
// contiguous across the wave.
__global__ __launch_bounds__(kThreads) void k_expand_edges(CscRels a, int64_t total_rows,
                                                           uint32_t *keys, int32_t *vals,
                                                           int32_t *cnt) {
    __shared__ const int32_t *s_ix[kMaxRels];
    __shared__ const int32_t *s_ip[kMaxRels];
    __shared__ int64_t s_koff[kMaxRels], s_e0[kMaxRels], s_rb[kMaxRels];
    for (int r = threadIdx.x; r < a.count; r += kThreads) {
        s_ix[r] = a.indices[r];
        s_ip[r] = a.indptr[r];
        s_koff[r] = a.koff[r];
        s_e0[r] = a.e0[r];
        s_rb[r] = a.row_base[r];
    }
    __syncthreads();
    const int lane = threadIdx.x & 63;
    const int64_t x0 = ((int64_t)blockIdx.x * kThreads + (threadIdx.x & ~63));
    if (x0 >= total_rows) return;                       // whole wave
    const int64_t x = x0 + lane;
    const bool live = x < total_rows;
    // this lane's row: relation c (last with row_base <= x), local row i, first edge eb
    int c = 0;
    for (int r = 1; r < a.count; ++r)
        if (s_rb[r] <= x) c = r;
    const int64_t i = live ? x - s_rb[c] : 0;
    const int32_t *ip = s_ip[c];
    const int32_t eb = live ? (int32_t)(s_e0[c] + ip[i]) : 0;
    const int32_t ee = live ? (int32_t)(s_e0[c] + ip[i + 1]) : 0;
    // the wave's edge range [E0, E1): first edge of row x0, end of its last live row
    const int last = (int)((total_rows - x0 < 64 ? total_rows - x0 : 64) - 1);
    const int32_t E0 = __shfl(eb, 0, 64), E1 = __shfl(ee, last, 64);
    const int32_t ebs = live ? eb : INT32_MAX;          // dead lanes never match
    for (int32_t g0 = E0; g0 < E1; g0 += 64) {
        const int32_t g = g0 + lane;
        int lo = 0;
#pragma unroll
        for (int step = 32; step >= 1; step >>= 1) {
            const int cand = lo + step;
            const int32_t v = __shfl(ebs, cand, 64);
            if (v <= g) lo = cand;
        }
        const int cg = __shfl(c, lo, 64);
        const int32_t ig = (int32_t)__shfl((int)i, lo, 64);
        if (g < E1) {
            const uint32_t key = (uint32_t)(s_koff[cg] + s_ix[cg][g - s_e0[cg]]);
            keys[g] = key;
            vals[g] = ig;
            atomicAdd(&cnt[key], 1);
        }
    }
}

// p[0, n) = v; 16-byte stores over the grid (p 16-byte aligned), a grid-stride loop
__global__ __launch_bounds__(kThreads) void k_fill_i32(int32_t *p, int64_t n, int32_t v) {
    const int64_t n4 = n / 4;
    const int4 q = make_int4(v, v, v, v);
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n4; i += stride)
        ((int4 *)p)[i] = q;
    const int64_t t = 4 * n4 + (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (t < n) p[t] = v;
}

// ---------------------------------------------------------------- CSC by placement
// The per-key offsets are known from the counts, so each edge takes a slot of its key's
// segment with one atomic decrement of the key's remaining count (cur, which returns to
// zero), and the segment is then sorted by value.  Within a key the stable order is
// ascending edge position, i.e. ascending destination row (a relation's edges are listed
// by destination row), and edges with the same destination row have equal values, so the
// sorted segment is the stable result whatever order the slots were taken in.
__global__ __launch_bounds__(kThreads) void k_csc_place(const uint32_t *keys, const int32_t *vals,
                                                        int64_t nnz, const int32_t *ip,
                                                        int32_t *cur, int32_t *csd) {
    const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (e >= nnz) return;
    const uint32_t k = keys[e];
    const int32_t slot = atomicSub(&cur[k], 1) - 1;
    csd[ip[k] + slot] = vals[e];
}

constexpr int kSegNet = 16;        // segments up to this length: a sorting network per thread
constexpr int kSegLds = 16384;     // longer ones up to this length: a workgroup sort in LDS

__device__ __forceinline__ void cswap(int32_t &a, int32_t &b) {
    const int32_t lo = a < b ? a : b, hi = a < b ? b : a;
    a = lo;
    b = hi;
}

// One thread per key: segments of 2..kSegNet values sorted in registers (bitonic network
// over 16 slots, unused slots +inf); longer segments are queued for k_csc_sort_long.
__global__ __launch_bounds__(kThreads) void k_csc_sort_short(const int32_t *ip, int64_t nkeys,
                                                             int32_t *csd, int32_t *long_keys,
                                                             uint32_t *long_count) {
    const int64_t k = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (k >= nkeys) return;
    const int32_t b = ip[k], n = ip[k + 1] - b;
    if (n <= 1) return;
    if (n == 2) {
        int32_t x = csd[b], y = csd[b + 1];
        if (y < x) {
            csd[b] = y;
            csd[b + 1] = x;
        }
        return;
    }
    if (n > kSegNet) {
        long_keys[atomicAdd(long_count, 1u)] = (int32_t)k;
        return;
    }
    int32_t v[kSegNet];
#pragma unroll
    for (int i = 0; i < kSegNet; ++i) v[i] = i < n ? csd[b + i] : INT32_MAX;
#pragma unroll
    for (int sz = 2; sz <= kSegNet; sz <<= 1)
#pragma unroll
        for (int st = sz >> 1; st > 0; st >>= 1)
#pragma unroll
            for (int i = 0; i < kSegNet; ++i) {
                const int j = i ^ st;
                if (j > i) {
                    if ((i & sz) == 0) cswap(v[i], v[j]);
                    else cswap(v[j], v[i]);
                }
            }
#pragma unroll
    for (int i = 0; i < kSegNet; ++i)
        if (i < n) csd[b + i] = v[i];
}

// One workgroup per queued segment (grid-stride over the queue): bitonic sort of up to
// kSegLds values in LDS.  A longer segment raises *overflow, which runs the radix sort
// of all edges instead.
__global__ __launch_bounds__(kThreads) void k_csc_sort_long(const int32_t *ip, int32_t *csd,
                                                            const int32_t *long_keys,
                                                            const uint32_t *long_count,
                                                            uint32_t *overflow) {
    __shared__ int32_t buf[kSegLds];
    const uint32_t total = *long_count;
    for (uint32_t q = blockIdx.x; q < total; q += gridDim.x) {
        const int32_t k = long_keys[q];
        const int32_t b = ip[k], n = ip[k + 1] - b;
        if (n > kSegLds) {
            if (threadIdx.x == 0) atomicOr(overflow, 1u);
            continue;
        }
        int P = 1;
        while (P < n) P <<= 1;
        __syncthreads();
        for (int i = threadIdx.x; i < P; i += kThreads) buf[i] = i < n ? csd[b + i] : INT32_MAX;
        __syncthreads();
        for (int sz = 2; sz <= P; sz <<= 1) {
            for (int st = sz >> 1; st > 0; st >>= 1) {
                for (int i = threadIdx.x; i < P; i += kThreads) {
                    const int j = i ^ st;
                    if (j > i) {
                        const int32_t x = buf[i], y = buf[j];
                        const bool up = (i & sz) == 0;
                        if (up ? y < x : x < y) {
                            buf[i] = y;
                            buf[j] = x;
                        }
                    }
                }
                __syncthreads();
            }
        }
        for (int i = threadIdx.x; i < n; i += kThreads) csd[b + i] = buf[i];
    }
}

// dst[i] = src[i] for i < n, only when *gate is raised
__global__ __launch_bounds__(kThreads) void k_copy_i32_gated(const int32_t *src, int32_t *dst,
                                                             int64_t n, const uint32_t *gate) {
    if (*gate == 0u) return;
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i < n) dst[i] = src[i];
}


// Descriptor of the segment at schedule position p (see SegDesc).
struct DescArgs {
    int32_t nslots;
    int64_t base[kMaxSlots];
    const int32_t *indptr[kMaxSlots];
    int16_t dst[kMaxSlots];
    int32_t col_off[kMaxSlots];
    int64_t mcat_off[kMaxTypes];
    int64_t mcat_ld[kMaxTypes];
    int32_t es;
};
// Descriptor of segment seg written at schedule position p; returns its degree.
__device__ __forceinline__ int32_t desc_of(const DescArgs &a, int64_t seg, int64_t p,
                                           SegDesc *desc, int32_t *weight) {
    int lo = 0, hi = a.nslots - 1;
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if (a.base[mid] <= seg) lo = mid; else hi = mid - 1;
    }
    const int64_t row = seg - a.base[lo];
    SegDesc d;
    if (a.indptr[lo]) {
        d.k0 = a.indptr[lo][row];
        d.deg = a.indptr[lo][row + 1] - d.k0;
    } else {
        d.k0 = (int32_t)row;
        d.deg = 1;
    }
    const int t = a.dst[lo];
    const uint64_t out = (uint64_t)(a.mcat_off[t] + (row * a.mcat_ld[t] + a.col_off[lo]) * a.es) >> 4;
    d.out_lo = (uint32_t)out;
    d.info = (uint32_t)((out >> 32) & 0xffu) | ((uint32_t)lo << 8);
    desc[p] = d;
    // balancing weight: the rows a segment moves, its entries read plus the row it writes
    weight[p] = (d.deg > 0 ? d.deg : 1) + 1;
    return d.deg;
}

// IDENT: schedule position p holds segment p; order[p] = p, and *flag is raised when some
// segment is heavy (a schedule key other than the last), i.e. when the sorted schedule is
// not the identity, unless `keep` asks for enumeration order.  Otherwise (gated on that
// flag): segment order[p].
// The slot tables are copied into LDS first: the slot search indexes them per lane, which
// from the kernel arguments is a chain of dependent global loads.
template <bool IDENT>
__global__ __launch_bounds__(kThreads) void k_fwd_desc(DescArgs a, int32_t *order,
                                                       int64_t n_seg, SegDesc *desc,
                                                       int32_t *weight, uint32_t *flag, int keep) {
    if (!IDENT && *flag == 0u) return;
    __shared__ DescArgs s_a;
    static_assert(sizeof(DescArgs) % 4 == 0, "copied in words");
    for (int i = threadIdx.x; i < (int)(sizeof(DescArgs) / 4); i += kThreads)
        ((uint32_t *)&s_a)[i] = ((const uint32_t *)&a)[i];
    __syncthreads();
    const int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const bool in = p < n_seg;
    int64_t seg = p;
    if (!IDENT && in) seg = order[p];
    if (IDENT && in) order[p] = (int32_t)p;
    bool heavy = false;
    if (in) heavy = desc_of(s_a, seg, p, desc, weight) > 32;
    if (IDENT && !keep && __ballot(heavy) != 0 && (threadIdx.x & 63) == 0) atomicOr(flag, 1u);
}

// Backward rows of one type in enumeration order (order[j] = j); *flag is raised when some
// row is heavy, i.e. when the sorted schedule is not the identity, unless `keep` asks for
// enumeration order.  Rows of more than kSplitEdges transpose edges are split into pieces
// of kSplitEdges edges: np[j] = their count (0 for other rows), and the pieces (j, 0),
// (j, 1), ... take consecutive slots from the shared counter (the slots' places vary from
// run to run; what is summed, and in which order, does not).
__global__ __launch_bounds__(kThreads) void k_bwd_ident(BwdKey kf, int64_t n, int32_t *order,
                                                        uint32_t *flag, int keep, SplitRows sp) {
    const int64_t j = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const bool in = j < n;
    int64_t deg = 0;
    if (in) {
        order[j] = (int32_t)j;
        deg = kf.degree(j);
        const int32_t np = deg > kSplitEdges ? (int32_t)((deg + kSplitEdges - 1) / kSplitEdges) : 0;
        sp.np[j] = np;
        if (np > 0) {
            const uint32_t b = atomicAdd(sp.count, (uint32_t)np);
            sp.base[j] = (int32_t)b;
            // the capacity bounds every count the edges allow; the test keeps a corrupt
            // transpose from writing past the list
            if ((int64_t)b + np <= sp.cap)
                for (int32_t q = 0; q < np; ++q) sp.pieces[b + q] = make_int2((int)j, q);
        }
    }
    const bool heavy = in && !keep && degree_key(deg) != kSchedBuckets - 1;
    if (__ballot(heavy) != 0 && (threadIdx.x & 63) == 0) atomicOr(flag, 1u);
}


// Chunk starts of the flattened forward stream.  pre = exclusive prefix of the segment
// weights (rows a segment moves).  Segment p belongs to chunk pre[p] / kFwdChunk; cs[c] is
// the first segment of chunk c or later (chunks no segment starts in are empty), for
// c <= ceil(total / kFwdChunk); cs[nc_max + 1] = total weight.
__global__ __launch_bounds__(kThreads) void k_chunk_starts(const int32_t *pre, const int32_t *weight,
                                                           int64_t n_seg, int64_t nc_max, int32_t *cs) {
    const int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (p >= n_seg) return;
    const int64_t cur = pre[p] / kFwdChunk;
    const int64_t prev = p == 0 ? -1 : pre[p - 1] / kFwdChunk;
    for (int64_t c = prev + 1; c <= cur; ++c) cs[c] = (int32_t)p;
    if (p == n_seg - 1) {
        const int64_t total = (int64_t)pre[p] + weight[p];
        const int64_t nc = (total + kFwdChunk - 1) / kFwdChunk;
        for (int64_t c = cur + 1; c <= nc; ++c) cs[c] = (int32_t)n_seg;
        cs[nc_max + 1] = (int32_t)total;
    }
}

struct Words {
    uint32_t n;
    uint32_t w[512];
};
__global__ void k_fill_words(uint32_t *dst, Words a) {
    for (uint32_t i = threadIdx.x; i < a.n; i += blockDim.x) dst[i] = a.w[i];
}

}  // namespace

size_t scan_temp_bytes(int64_t n) { return align_up((size_t)cdiv(n, kScanTile) * 4 + 4, 256); }

hipError_t scan_gated(const int32_t *in, int32_t *out, int64_t n, void *temp,
                      const uint32_t *gate, hipStream_t s) {
    if (n == 0) return hipSuccess;
    const int64_t nb = cdiv(n, kScanTile);
    const bool vec = ((uintptr_t)in % 16) == 0 && ((uintptr_t)out % 16) == 0;
    if (nb == 1) {   // one tile: the apply pass alone
        if (vec)
            hipLaunchKernelGGL(k_scan_apply<true>, dim3(1), dim3(kThreads), 0, s, in, out, n,
                               (const int32_t *)nullptr, gate);
        else
            hipLaunchKernelGGL(k_scan_apply<false>, dim3(1), dim3(kThreads), 0, s, in, out, n,
                               (const int32_t *)nullptr, gate);
        return hipGetLastError();
    }
    int32_t *partial = (int32_t *)temp;
    if (vec)
        hipLaunchKernelGGL(k_scan_reduce<true>, dim3((unsigned)nb), dim3(kThreads), 0, s, in, n,
                           partial, gate);
    else
        hipLaunchKernelGGL(k_scan_reduce<false>, dim3((unsigned)nb), dim3(kThreads), 0, s, in, n,
                           partial, gate);
    RGCN_HIP_TRY(hipGetLastError());
    hipLaunchKernelGGL(k_scan_partials, dim3(1), dim3(kThreads), 0, s, partial, nb, gate);
    RGCN_HIP_TRY(hipGetLastError());
    if (vec)
        hipLaunchKernelGGL(k_scan_apply<true>, dim3((unsigned)nb), dim3(kThreads), 0, s, in, out,
                           n, (const int32_t *)partial, gate);
    else
        hipLaunchKernelGGL(k_scan_apply<false>, dim3((unsigned)nb), dim3(kThreads), 0, s, in, out,
                           n, (const int32_t *)partial, gate);
    return hipGetLastError();
}

hipError_t exclusive_scan_i32(const int32_t *in, int32_t *out, int64_t n, void *temp,
                              hipStream_t s) {
    return scan_gated(in, out, n, temp, nullptr, s);
}

size_t bucket_sort_temp_bytes(int64_t n, int nbuckets) {
    const int64_t ntiles = cdiv(n, kSortTile);
    return align_up((size_t)nbuckets * ntiles * 4, 256) +
           scan_temp_bytes((int64_t)nbuckets * ntiles);
}

hipError_t fwd_plan(const FwdSlot *slots_host, int nslots, int64_t n_seg, int32_t *order,
                    const int64_t *mcat_off, const int64_t *mcat_ld, int es, SegDesc *desc,
                    int32_t *weight, uint32_t *flag, int keep_order, void *temp,
                    hipStream_t s) {
    if (n_seg == 0) return hipSuccess;
    DescArgs a;
    a.nslots = nslots;
    FwdKey kf;
    kf.nslots = nslots;
    for (int i = 0; i < kMaxSlots; ++i) {
        a.base[i] = kf.base[i] = i < nslots ? slots_host[i].seg_base : 0;
        a.indptr[i] = kf.indptr[i] = i < nslots ? slots_host[i].indptr : nullptr;
        a.dst[i] = (int16_t)(i < nslots ? slots_host[i].dst_type : 0);
        a.col_off[i] = i < nslots ? slots_host[i].col_off : 0;
    }
    for (int t = 0; t < kMaxTypes; ++t) {
        a.mcat_off[t] = mcat_off[t];
        a.mcat_ld[t] = mcat_ld[t];
    }
    a.es = es;
    const dim3 grid((unsigned)cdiv(n_seg, kThreads));
    // enumeration order first; the sort and the second descriptor pass run only when some
    // segment is heavy (otherwise the stable sort by key is the identity)
    hipLaunchKernelGGL(k_fwd_desc<true>, grid, dim3(kThreads), 0, s, a, order, n_seg, desc,
                       weight, flag, keep_order);
    RGCN_HIP_TRY(hipGetLastError());
    RGCN_HIP_TRY((bucket_sort<kSchedBuckets, 5>(kf, PutIndex{order}, n_seg, temp, s, flag)));
    hipLaunchKernelGGL(k_fwd_desc<false>, grid, dim3(kThreads), 0, s, a, order, n_seg, desc,
                       weight, flag, keep_order);
    return hipGetLastError();
}

int64_t fwd_chunk_bound(int64_t n_seg, int64_t nnz_total) {
    return cdiv(2 * n_seg + nnz_total, kFwdChunk);
}

size_t fwd_chunks_temp_bytes(int64_t n_seg) {
    return 2 * align_up((size_t)n_seg * 4 + 4, 256) + scan_temp_bytes(n_seg);
}

hipError_t fwd_chunks(const int32_t *weight, int64_t n_seg, int64_t nc_max, int32_t *cs,
                      void *temp, hipStream_t s) {
    if (n_seg == 0) return hipSuccess;
    int32_t *pre = (int32_t *)temp;
    void *stemp = (char *)temp + align_up((size_t)n_seg * 4 + 4, 256);
    RGCN_HIP_TRY(exclusive_scan_i32(weight, pre, n_seg, stemp, s));
    hipLaunchKernelGGL(k_chunk_starts, dim3((unsigned)cdiv(n_seg, kThreads)), dim3(kThreads), 0, s,
                       pre, weight, n_seg, nc_max, cs);
    return hipGetLastError();
}

hipError_t bwd_schedule(const BwdKeyRels &rels, int64_t n_rows, int32_t *order, void *temp,
                        uint32_t *flag, int keep_order, const SplitRows &split, hipStream_t s) {
    if (n_rows == 0) return hipSuccess;
    hipLaunchKernelGGL(k_bwd_ident, dim3((unsigned)cdiv(n_rows, kThreads)), dim3(kThreads), 0, s,
                       BwdKey{rels}, n_rows, order, flag, keep_order, split);
    RGCN_HIP_TRY(hipGetLastError());
    return bucket_sort<kSchedBuckets, 5>(BwdKey{rels}, PutIndex{order}, n_rows, temp, s, flag);
}

// Digit plan of an LSD radix sort of keys < key_range: the fewest passes of at most 10
// bits, digits as even as possible.
static void radix_plan(int64_t key_range, int *passes, int *bits) {
    int nb = 0;
    while (nb < 32 && ((int64_t)1 << nb) < key_range) ++nb;  // keys < 2^nb
    *passes = (nb + 9) / 10;
    *bits = *passes ? (nb + *passes - 1) / *passes : 0;
}

size_t csc_temp_bytes(int64_t nnz, int64_t key_range) {
    int passes, bits;
    radix_plan(key_range, &passes, &bits);
    const int nbk = bits <= 8 ? 256 : (1 << bits);
    const size_t sort = bucket_sort_temp_bytes(nnz, nbk);
    const size_t scan = scan_temp_bytes(key_range + 1);
    // values, two key buffers, sort / scan scratch, then the per-key cursors and two
    // words (queue length, overflow flag)
    return 3 * align_up((size_t)nnz * 4 + 4, 256) + align_up(sort > scan ? sort : scan, 256) +
           align_up((size_t)(key_range + 3) * 4, 256);
}

// The transpose: (key, value) pairs of every edge (k_expand_edges, which also counts edges
// per key), offsets by an exclusive scan of the counts, each edge placed in its key's
// segment, segments sorted by value.  If some segment is longer than kSegLds, the LSD
// radix sort of all pairs (stable, digits of at most 10 bits) runs instead, gated on a
// device flag so the host never waits.
hipError_t csc_build_all(const CscRels &rels, int64_t total_rows, int64_t nnz,
                         int64_t key_range, int32_t *ip, int32_t *csd, void *temp,
                         hipStream_t s) {
    int passes, bits;
    radix_plan(key_range, &passes, &bits);
    if (nnz == 0) passes = 0;
    const int nbk = bits <= 8 ? 256 : (1 << bits);
    const size_t sort = bucket_sort_temp_bytes(nnz, nbk);
    const size_t scan = scan_temp_bytes(key_range + 1);
    const size_t arr = align_up((size_t)nnz * 4 + 4, 256);
    int32_t *tmp_vals = (int32_t *)temp;
    uint32_t *kb[2] = {(uint32_t *)((char *)temp + arr), (uint32_t *)((char *)temp + 2 * arr)};
    void *sort_tmp = (char *)temp + 3 * arr;   // also the scan's scratch
    int32_t *cur = (int32_t *)((char *)sort_tmp + align_up(sort > scan ? sort : scan, 256));
    uint32_t *words = (uint32_t *)(cur + key_range + 1);   // queue length, overflow
    int32_t *long_keys = (int32_t *)kb[0];                 // at most nnz / (kSegNet + 1)

    // cursors and the two words start at zero
    {
        int64_t blocks = cdiv(cdiv(key_range + 3, 4), kThreads);
        blocks = blocks < 1 ? 1 : (blocks > 2048 ? 2048 : blocks);
        hipLaunchKernelGGL(k_fill_i32, dim3((unsigned)blocks), dim3(kThreads), 0, s, cur,
                           key_range + 3, 0);
    }
    RGCN_HIP_TRY(hipGetLastError());
    if (total_rows > 0 && nnz > 0) {
        hipLaunchKernelGGL(k_expand_edges, dim3((unsigned)cdiv(total_rows, kThreads)),
                           dim3(kThreads), 0, s, rels, total_rows, kb[1], tmp_vals, cur);
        RGCN_HIP_TRY(hipGetLastError());
    }
    RGCN_HIP_TRY(exclusive_scan_i32(cur, ip, key_range + 1, sort_tmp, s));
    if (nnz == 0) return hipSuccess;
    hipLaunchKernelGGL(k_csc_place, dim3((unsigned)cdiv(nnz, kThreads)), dim3(kThreads), 0, s,
                       kb[1], tmp_vals, nnz, ip, cur, csd);
    RGCN_HIP_TRY(hipGetLastError());
    hipLaunchKernelGGL(k_csc_sort_short, dim3((unsigned)cdiv(key_range, kThreads)), dim3(kThreads),
                       0, s, ip, key_range, csd, long_keys, words);
    RGCN_HIP_TRY(hipGetLastError());
    hipLaunchKernelGGL(k_csc_sort_long, dim3(512), dim3(kThreads), 0, s, ip, csd, long_keys,
                       words, words + 1);
    RGCN_HIP_TRY(hipGetLastError());

    // fallback, gated on the overflow word: values ping-pong between tmp_vals and csd
    // from tmp_vals; with an even number of passes they end in tmp_vals and are copied
    const uint32_t *gate = words + 1;
    const uint32_t *keys = kb[1];
    const uint32_t mask = bits ? (uint32_t)((1u << bits) - 1u) : 0u;
    int32_t *vb[2] = {tmp_vals, csd};
    for (int p = 0; p < passes; ++p) {
        RadixKey kf{keys, bits * p, mask};
        uint32_t *kout = kb[p % 2] == keys ? kb[(p + 1) % 2] : kb[p % 2];
        RadixPut put{keys, vb[p % 2], kout, vb[(p + 1) % 2]};
        if (bits <= 8) {
            RGCN_HIP_TRY((bucket_sort<256, 8>(kf, put, nnz, sort_tmp, s, gate)));
        } else if (bits == 9) {
            RGCN_HIP_TRY((bucket_sort<512, 9>(kf, put, nnz, sort_tmp, s, gate)));
        } else {
            RGCN_HIP_TRY((bucket_sort<1024, 10>(kf, put, nnz, sort_tmp, s, gate)));
        }
        keys = kout;
    }
    if (passes % 2 == 0) {
        hipLaunchKernelGGL(k_copy_i32_gated, dim3((unsigned)cdiv(nnz, kThreads)), dim3(kThreads),
                           0, s, tmp_vals, csd, nnz, gate);
        RGCN_HIP_TRY(hipGetLastError());
    }
    return hipSuccess;
}

hipError_t fill_words(void *dst, const void *src_host, size_t bytes, hipStream_t s) {
    const uint32_t *src = (const uint32_t *)src_host;
    size_t nw = bytes / 4;
    for (size_t off = 0; off < nw; off += 512) {
        Words a;
        a.n = (uint32_t)((nw - off) < 512 ? (nw - off) : 512);
        for (uint32_t i = 0; i < a.n; ++i) a.w[i] = src[off + i];
        hipLaunchKernelGGL(k_fill_words, dim3(1), dim3(256), 0, s, (uint32_t *)dst + off, a);
        RGCN_HIP_TRY(hipGetLastError());
    }
    return hipSuccess;
}

}  // namespace rgcn
