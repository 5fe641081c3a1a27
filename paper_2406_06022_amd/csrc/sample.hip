// On-the-fly neighbour sampling and block construction for one GNN layer (the paper
// samples each mini-batch's neighbourhoods with a per-layer fanout, Sec. 3.1.1 and
// 3.1.4; one block per layer).  For every destination node v of every relation r, all
// in-edges when deg <= fanout, otherwise a uniform subset of fanout positions chosen
// by Floyd's algorithm, listed in CSR order.  Draw k of (v, r) is word k mod 4 of
// Philox4x64-10 (Salmon et al., SC 2011) at counter (v, r, k / 4, 0), key (seed, layer);
// a uniform integer in [0, m) is the high word of draw * m.  The block's source nodes
// of a type are its destination nodes, then the sampled sources in order of first
// appearance (relations in order, destination rows in order, positions in order);
// edges are relabelled to those block-local rows.
//
// Layout of the work: every (relation, destination row) is a segment; a count pass and
// an exclusive scan give each segment's edge offset; the draw pass writes the sampled
// global ids into a candidate array laid out per source type by capacity (destination
// ids first, then each relation leaving the type, fanout slots per destination row), so
// candidate positions follow first-appearance order with gaps.  One word per graph node
// keeps the smallest position holding that node (atomicMin: one atomic per candidate, no
// probing, where a hash table keyed by id needs a compare-and-swap and a min per
// candidate); a flag per position that holds its
// node's first occurrence, scanned, numbers the source rows.
#include "common.h"

namespace rgcn {

namespace {

constexpr int kThreads = 256;
constexpr int kDrawThreads = 128;

__host__ __device__ inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

__device__ __forceinline__ int find_le(const int64_t *base, int n, int64_t x) {
    // last index i < n with base[i] <= x (base ascending, base[0] <= x)
    int i = 0;
    for (int j = 1; j < n; ++j) i = base[j] <= x ? j : i;
    return i;
}

__device__ __forceinline__ void load_tab(SampleTab *dst, const SampleTab *src) {
    const int n = (int)(sizeof(SampleTab) / 4);
    for (int i = threadIdx.x; i < n; i += blockDim.x) ((uint32_t *)dst)[i] = ((const uint32_t *)src)[i];
    __syncthreads();
}

// Segment s -> relation, row, node id and in-edge range; false (with error bits) when
// the id or the degree is out of range.
struct Seg {
    int r;
    int64_t i, v, base, deg;
};
__device__ __forceinline__ bool seg_of(const SampleTab &T, int64_t s, Seg &g, uint32_t *err) {
    g.r = find_le(T.seg_base, T.nrel, s);
    g.i = s - T.seg_base[g.r];
    const int t = T.dst_type[g.r];
    g.v = T.dst_ids[t][g.i];
    g.base = 0;
    g.deg = 0;
    if (g.v < 0 || g.v >= T.num_nodes[t]) {
        atomicOr(err, 1u);
        return false;
    }
    const int64_t *ip = T.g_indptr[g.r];
    g.base = ip[g.v];
    g.deg = ip[g.v + 1] - g.base;
    if (g.deg < 0 || g.deg > 0xFFFFFFFFll) {
        atomicOr(err, 4u);
        g.deg = 0;
        return false;
    }
    return true;
}

__global__ __launch_bounds__(kThreads) void k_sample_count(const SampleTab *tab, int32_t *cnt,
                                                           uint32_t *err) {
    __shared__ SampleTab T;
    load_tab(&T, tab);
    for (int64_t s = (int64_t)blockIdx.x * kThreads + threadIdx.x; s <= T.n_seg;
         s += (int64_t)gridDim.x * kThreads) {
        if (s == T.n_seg) {
            cnt[s] = 0;
            continue;
        }
        Seg g;
        seg_of(T, s, g, err);
        cnt[s] = (int32_t)(g.deg < T.fanout ? g.deg : T.fanout);
    }
}

// Destination ids of each type at the head of its candidate region.
__global__ __launch_bounds__(kThreads) void k_sample_prefix(const SampleTab *tab, int64_t *cand) {
    __shared__ SampleTab T;
    load_tab(&T, tab);
    for (int t = 0; t < T.ntypes; ++t)
        for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < T.n_dst[t];
             i += (int64_t)gridDim.x * kThreads)
        {
            const int64_t v = T.dst_ids[t][i];   // out of range: reported by the count pass
            cand[T.type_base[t] + i] = (v >= 0 && v < T.num_nodes[t]) ? v : 0;
        }
}

// One thread per segment: the positions taken (sorted, in LDS, one column per thread),
// then the global ids of those in-edges into the candidate array, and the block indptr.
__global__ __launch_bounds__(kDrawThreads) void k_sample_draw(const SampleTab *tab,
                                                              const int32_t *off, int64_t *cand,
                                                              uint32_t *err) {
    __shared__ SampleTab T;
    __shared__ uint32_t pos[kMaxFanout][kDrawThreads];
    load_tab(&T, tab);
    const int lane = threadIdx.x;
    for (int64_t s = (int64_t)blockIdx.x * kDrawThreads + lane; s < T.n_seg;
         s += (int64_t)gridDim.x * kDrawThreads) {
        Seg g;
        seg_of(T, s, g, err);
        const int r = g.r;
        const int64_t e = (int64_t)off[s] - off[T.seg_base[r]];
        T.out_indptr[r][g.i] = (int32_t)e;
        const int f = T.fanout;
        const int c = off[s + 1] - off[s];
        if (c == 0) continue;
        const int src = T.src_type[r];
        const int64_t *gx = T.g_indices[r];
        int64_t *out = cand + T.cand_base[r] + e;
        const int64_t nsrc = T.num_nodes[src];
        auto put = [&](int q, int64_t p) {
            int64_t x = gx[g.base + p];
            if (x < 0 || x >= nsrc) {
                atomicOr(err, 8u);
                x = 0;
            }
            out[q] = x;
        };
        if (g.deg <= f) {
            for (int q = 0; q < c; ++q) put(q, q);
            continue;
        }
        // Floyd: for j = deg - f .. deg - 1, t uniform in [0, j]; take t, or j when t is
        // already taken (j exceeds every position taken so far, so it goes last).
        int taken = 0;
        uint64_t w[4];
        for (int k = 0; k < f; ++k) {
            if ((k & 3) == 0) {
                w[0] = (uint64_t)g.v;
                w[1] = (uint64_t)r;
                w[2] = (uint64_t)(k >> 2);
                w[3] = 0;
                philox4x64(w, T.seed, (uint64_t)(uint32_t)T.layer);
            }
            const uint64_t j = (uint64_t)g.deg - (uint64_t)f + (uint64_t)k;
            const uint64_t d = w[k & 3];
            const uint32_t t = (uint32_t)__umul64hi(d, j + 1);
            int lo = 0, hi = taken;
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (pos[mid][lane] < t) lo = mid + 1; else hi = mid;
            }
            if (lo < taken && pos[lo][lane] == t) {
                pos[taken][lane] = (uint32_t)j;
            } else {
                for (int q = taken; q > lo; --q) pos[q][lane] = pos[q - 1][lane];
                pos[lo][lane] = t;
            }
            ++taken;
        }
        for (int q = 0; q < f; ++q) put(q, pos[q][lane]);
    }
}

// Per relation: the last indptr entry and the edge count; per type the source count is
// written by k_dedup_counts.
__global__ void k_sample_tails(const SampleTab *tab, const int32_t *off, int64_t *counts) {
    __shared__ SampleTab T;
    load_tab(&T, tab);
    for (int r = threadIdx.x; r < T.nrel; r += blockDim.x) {
        const int64_t n = T.n_dst[T.dst_type[r]];
        const int32_t tot = off[T.seg_base[r] + n] - off[T.seg_base[r]];
        T.out_indptr[r][n] = tot;
        counts[r] = tot;
    }
}

// Candidate position p -> type, relation (-1: destination prefix) and edge; false for
// the unused capacity slots.
__device__ __forceinline__ bool slot_info(const SampleTab &T, const int32_t *off, int64_t p,
                                          int &t, int &r, int64_t &e) {
    t = find_le(T.type_base, T.ntypes, p);
    const int64_t q = p - T.type_base[t];
    if (q < T.n_dst[t]) {
        r = -1;
        e = q;
        return true;
    }
    r = -1;
    for (int x = 0; x < T.nrel; ++x)
        if (T.src_type[x] == t && p >= T.cand_base[x]) r = x;
    if (r < 0) return false;
    e = p - T.cand_base[r];
    const int64_t tot = off[T.seg_base[r] + T.n_dst[T.dst_type[r]]] - off[T.seg_base[r]];
    return e < tot;
}

// first[node_base[t] + id]: the smallest candidate position holding node id of type t
// (INT32_MAX: none), one word per graph node, cleared every call.
__global__ __launch_bounds__(kThreads) void k_fill_first(int32_t *first, int64_t n) {
    const int64_t n4 = n / 4;
    int4 *f4 = (int4 *)first;
    const int big = 0x7FFFFFFF;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n4;
         i += (int64_t)gridDim.x * kThreads)
        f4[i] = make_int4(big, big, big, big);
    for (int64_t i = n4 * 4 + (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * kThreads)
        first[i] = big;
}

__global__ __launch_bounds__(kThreads) void k_dedup_insert(const SampleTab *tab, const int32_t *off,
                                                           const int64_t *cand, int32_t *first) {
    __shared__ SampleTab T;
    load_tab(&T, tab);
    for (int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x; p < T.cap_total;
         p += (int64_t)gridDim.x * kThreads) {
        int t, r;
        int64_t e;
        if (!slot_info(T, off, p, t, r, e)) continue;
        atomicMin(&first[T.node_base[t] + cand[p]], (int32_t)p);
    }
}

__global__ __launch_bounds__(kThreads) void k_dedup_flag(const SampleTab *tab, const int32_t *off,
                                                         const int64_t *cand, const int32_t *first,
                                                         int32_t *flag, uint32_t *err) {
    __shared__ SampleTab T;
    load_tab(&T, tab);
    for (int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x; p <= T.cap_total;
         p += (int64_t)gridDim.x * kThreads) {
        if (p == T.cap_total) {
            flag[p] = 0;
            continue;
        }
        int t, r;
        int64_t e;
        if (!slot_info(T, off, p, t, r, e)) {
            flag[p] = 0;
            continue;
        }
        const int32_t f = first[T.node_base[t] + cand[p]] == (int32_t)p ? 1 : 0;
        flag[p] = f;
        if (r < 0 && !f) atomicOr(err, 2u);   // a repeated destination id
    }
}

__global__ __launch_bounds__(kThreads) void k_dedup_emit(const SampleTab *tab, const int32_t *off,
                                                         const int64_t *cand,
                                                         const int32_t *first,
                                                         const int32_t *rank) {
    __shared__ SampleTab T;
    load_tab(&T, tab);
    for (int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x; p < T.cap_total;
         p += (int64_t)gridDim.x * kThreads) {
        int t, r;
        int64_t e;
        if (!slot_info(T, off, p, t, r, e)) continue;
        const int64_t id = cand[p];
        const int32_t f = first[T.node_base[t] + id];
        const int32_t loc = rank[f] - rank[T.type_base[t]];
        if (f == (int32_t)p) T.out_src_ids[t][loc] = id;
        if (r >= 0) T.out_indices[r][e] = loc;
        if (r >= 0 && T.out_src_rows[r]) T.out_src_rows[r][e] = id;
    }
}

__global__ void k_dedup_counts(const SampleTab *tab, const int32_t *rank, int64_t *counts) {
    __shared__ SampleTab T;
    load_tab(&T, tab);
    for (int t = threadIdx.x; t < T.ntypes; t += blockDim.x)
        counts[T.nrel + t] = rank[T.type_base[t] + T.type_cap[t]] - rank[T.type_base[t]];
}

// Grid-stride launches: at most 8 workgroups per CU of 256 (each copies the tables).
int64_t grid_for(int64_t n, int threads) {
    int64_t g = cdiv(n, threads);
    if (g < 1) g = 1;
    return g > 2048 ? 2048 : g;
}

}  // namespace

bool sample_layout(SampleTab &T, SampleLayout &L) {
    // segments and candidate regions
    int64_t s = 0;
    for (int r = 0; r < T.nrel; ++r) {
        T.seg_base[r] = s;
        s += T.n_dst[T.dst_type[r]];
    }
    T.n_seg = s;
    int64_t c = 0;
    for (int t = 0; t < T.ntypes; ++t) {
        T.type_base[t] = c;
        int64_t cap = T.n_dst[t];
        for (int r = 0; r < T.nrel; ++r)
            if (T.src_type[r] == t) {
                T.cand_base[r] = c + cap;
                cap += T.n_dst[T.dst_type[r]] * (int64_t)T.fanout;
            }
        T.type_cap[t] = cap;
        c += cap;
    }
    for (int t = T.ntypes; t < kMaxTypes; ++t) T.type_base[t] = c, T.type_cap[t] = 0;
    T.cap_total = c;
    if (T.n_seg + 1 > 0x7FFFFFFFll || c + 1 > 0x7FFFFFFFll) return false;
    int64_t nodes = 0;
    for (int t = 0; t < T.ntypes; ++t) {
        T.node_base[t] = nodes;
        nodes += T.num_nodes[t];
    }
    auto al = [](size_t x) { return (x + 255) / 256 * 256; };
    size_t o = 0;
    L.off_err = o; o += 256;
    L.off_tab = o; o += al(sizeof(SampleTab));
    L.off_seg = o; o += al((size_t)(T.n_seg + 1) * 4);
    const int64_t scan_n = (T.n_seg + 1) > (c + 1) ? (T.n_seg + 1) : (c + 1);
    L.off_scan = o; o += al(scan_temp_bytes(scan_n));
    L.off_cand = o; o += al((size_t)c * 8 + 8);
    L.off_flag = o; o += al((size_t)(c + 1) * 4);
    L.off_first = o; o += al((size_t)nodes * 4);
    L.nodes = nodes;
    L.total = o;
    return true;
}

hipError_t sample_block(const SampleTab &T, const SampleLayout &L, char *ws, int64_t *counts,
                        hipStream_t s) {
    uint32_t *err = (uint32_t *)(ws + L.off_err);
    SampleTab *tab = (SampleTab *)(ws + L.off_tab);
    int32_t *seg = (int32_t *)(ws + L.off_seg);
    int64_t *cand = (int64_t *)(ws + L.off_cand);
    int32_t *flag = (int32_t *)(ws + L.off_flag);
    int32_t *first = (int32_t *)(ws + L.off_first);
    const uint32_t zero = 0;
    RGCN_HIP_TRY(fill_words(err, &zero, 4, s));
    RGCN_HIP_TRY(fill_words(tab, &T, sizeof(SampleTab), s));
    hipLaunchKernelGGL(k_sample_count, dim3((unsigned)grid_for(T.n_seg + 1, kThreads)),
                       dim3(kThreads), 0, s, tab, seg, err);
    RGCN_HIP_TRY(hipGetLastError());
    RGCN_HIP_TRY(exclusive_scan_i32(seg, seg, T.n_seg + 1, ws + L.off_scan, s));
    int64_t maxdst = 0;
    for (int t = 0; t < T.ntypes; ++t) maxdst = T.n_dst[t] > maxdst ? T.n_dst[t] : maxdst;
    hipLaunchKernelGGL(k_sample_prefix, dim3((unsigned)grid_for(maxdst, kThreads)),
                       dim3(kThreads), 0, s, tab, cand);
    RGCN_HIP_TRY(hipGetLastError());
    hipLaunchKernelGGL(k_sample_draw, dim3((unsigned)grid_for(T.n_seg, kDrawThreads)),
                       dim3(kDrawThreads), 0, s, tab, seg, cand, err);
    RGCN_HIP_TRY(hipGetLastError());
    hipLaunchKernelGGL(k_sample_tails, dim3(1), dim3(64), 0, s, tab, seg, counts);
    RGCN_HIP_TRY(hipGetLastError());
    hipLaunchKernelGGL(k_fill_first, dim3((unsigned)grid_for(L.nodes / 4 + 1, kThreads)),
                       dim3(kThreads), 0, s, first, L.nodes);
    RGCN_HIP_TRY(hipGetLastError());
    hipLaunchKernelGGL(k_dedup_insert, dim3((unsigned)grid_for(T.cap_total, kThreads)),
                       dim3(kThreads), 0, s, tab, seg, cand, first);
    RGCN_HIP_TRY(hipGetLastError());
    hipLaunchKernelGGL(k_dedup_flag, dim3((unsigned)grid_for(T.cap_total + 1, kThreads)),
                       dim3(kThreads), 0, s, tab, seg, cand, first, flag, err);
    RGCN_HIP_TRY(hipGetLastError());
    RGCN_HIP_TRY(exclusive_scan_i32(flag, flag, T.cap_total + 1, ws + L.off_scan, s));
    hipLaunchKernelGGL(k_dedup_emit, dim3((unsigned)grid_for(T.cap_total, kThreads)),
                       dim3(kThreads), 0, s, tab, seg, cand, first, flag);
    RGCN_HIP_TRY(hipGetLastError());
    hipLaunchKernelGGL(k_dedup_counts, dim3(1), dim3(64), 0, s, tab, flag, counts);
    return hipGetLastError();
}

}  // namespace rgcn
