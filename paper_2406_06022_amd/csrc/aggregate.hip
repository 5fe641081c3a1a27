// HBM-bound kernels of the block: the forward gather + per-relation segmented mean, the
// backward transposed sum (with the ReLU-input mask and the embedding-gradient
// scatter-add fused in), weight packing, column sums and device-side validation.
//
// Row traffic is done in 16-byte chunks: a "group" of G lanes covers one row of d
// elements (G = chunks per row, at most 64, rounded up to a power of two in the forward
// gather; rows wider than 64 chunks give each lane CPL chunks), so a wave moves 64/G rows
// per load instruction and every row access is a run of contiguous 16-byte pieces.
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

// A pointer known to address global memory, as a global-address-space pointer (loads
// through it are global loads rather than flat loads).
template <class T>
__device__ __forceinline__ const __attribute__((address_space(1))) T *gbl(const T *p) {
    return (const __attribute__((address_space(1))) T *)p;
}

// ReLU mask of the block input at chunk c (columns 4 c .. 4 c + 3) of input row grow, as
// 1 / 0 per column, from the sign bits the caller passed (bit c' % 64 of word c' / 64 of
// the row): one 8-byte word read, shared by the 16 chunks it covers.  !ok reads `zero`.
__device__ __forceinline__ f32x4 relu_bits4(const uint64_t *mask, int64_t ld, int64_t grow, int c,
                                            bool ok, const char *zero) {
    const uint64_t w = *gbl(ok ? mask + grow * ld + (c >> 4) : (const uint64_t *)zero);
    const uint32_t b = (uint32_t)(w >> (4 * (c & 15)));
    return f32x4{(b & 1u) ? 1.f : 0.f, (b & 2u) ? 1.f : 0.f, (b & 4u) ? 1.f : 0.f,
                 (b & 8u) ? 1.f : 0.f};
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Gathered rows are read once (no locality over a table of many GB): streaming loads, so
// they do not push the index, row-id and descriptor lines out of L2.
__device__ __forceinline__ u32x4 ld_row(const char *p) {
    const __attribute__((address_space(1))) u32x4 *g = (const __attribute__((address_space(1))) u32x4 *)p;
    return __builtin_nontemporal_load(g);
}
// 16-byte global load
__device__ __forceinline__ uint4 ld16(const char *p) {
    const u32x4 v = *gbl((const u32x4 *)p);
    return make_uint4(v.x, v.y, v.z, v.w);
}

// Forward segments in schedule order (heaviest first), one group of G lanes per segment,
// persistent: group q handles segments q, q + ngroups, ...  A segment is the self-loop
// row of a destination (copied) or the sampled in-edges of a destination row in one
// relation (mean of the gathered source rows; 0 if none).
//
// The address of a gathered row takes three dependent loads: the segment descriptor, the
// source index of the edge, the global row id of that source.  They are software-
// pipelined over the group's successive segments, so that while the rows of segment i
// are in flight the row ids of segment i+1, the source indices of segment i+2 and the
// descriptor of segment i+3 are too.  Lane lg holds edges lg, lg+G, ... (EPL of them) of
// each segment in the pipeline; edges past EPL*G (degrees above the pipelined width)
// are resolved in place.  Row byte offsets are published to the group's LDS slots and
// read back as broadcasts while U rows per lane are in flight.
// The sum runs in ascending edge position; one division by the degree.
// Read (never written) by loads whose value is not needed; zero-initialised.  g_zero_row
// covers the widest row a group reads (256 chunks of 16 bytes), so a lane's chunk offset
// into it stays in bounds.
__device__ int64_t g_zero[2];
__device__ u32x4 g_zero_row[256];

// Row batches: rows [q, q + r) of a group, B loads per lane in flight; slots past r read
// the zero row.  The batch size is chosen per wave from ballots (uniform branches): the
// largest of UMAX, 4, 2, 1 that some group of the wave can fill past half.
template <int B, class LoadAcc>
__device__ __forceinline__ void row_batch(const int64_t *goff, int q, int r, LoadAcc &&la) {
    int64_t o[B];
    bool ok[B];
#pragma unroll
    for (int u = 0; u < B; ++u) {
        ok[u] = u < r;
        o[u] = goff[ok[u] ? q + u : 0];
    }
    la.template run<B>(o, ok);
}
template <int UMAX, class LoadAcc>
__device__ __forceinline__ void row_walk(const int64_t *goff, int n, LoadAcc &&la) {
    int q = 0;
    while (true) {
        const int r = n - q;
        if (__ballot(r > 0) == 0) break;
        if (UMAX > 4 && __ballot(r > 4) != 0) {
            row_batch<UMAX>(goff, q, r, la);
            q += UMAX;
        } else if (__ballot(r > 2) != 0) {
            row_batch<4>(goff, q, r, la);
            q += 4;
        } else if (__ballot(r > 1) != 0) {
            row_batch<2>(goff, q, r, la);
            q += 2;
        } else {
            row_batch<1>(goff, q, r, la);
            q += 1;
        }
    }
}

// Batch bodies: load B rows' chunks (16 bytes per lane per chunk) and add them into acc.
// SumLoad: fp32 rows at absolute addresses.  COMP: added with compensation (Kahan), comp
// holding the low-order part each addition lost, for the pieces of split rows: the terms
// of a hub's transpose cancel over thousands of edges, and plain fp32 sums of its pieces
// lost a digit against the exact sum (the rows of at most kSplitEdges edges that the
// plain kernels sum do not need it, and its registers cost those kernels a wave per
// SIMD).
// A slot that holds no row (padding of a batch) must leave acc and comp as they are:
// adding a zero would apply the pending compensation, and how many padding slots a row
// sees depends on its neighbours in the wave, i.e. on the processing order.
__device__ __forceinline__ void kahan_add(f32x4 &acc, f32x4 &comp, f32x4 x, bool take) {
    const f32x4 y = x - comp;
    const f32x4 t = acc + y;
    const f32x4 c = (t - acc) - y;
    acc = take ? t : acc;
    comp = take ? c : comp;
}
template <int CPL, bool COMP>
struct SumLoad {
    int lg, G, chunks;
    f32x4 *acc;
    f32x4 *comp;   // COMP only
    template <int B>
    __device__ __forceinline__ void run(const int64_t (&o)[B], const bool (&ok)[B]) const {
        f32x4 v[B][CPL];
#pragma unroll
        for (int u = 0; u < B; ++u)
#pragma unroll
            for (int p = 0; p < CPL; ++p) {
                const int c = lg + p * G;
                const char *pa = (ok[u] && c < chunks) ? (const char *)(uintptr_t)o[u] + (int64_t)c * 16
                                                       : (const char *)g_zero_row + c * 16;
                v[u][p] = *gbl((const f32x4 *)pa);
            }
#pragma unroll
        for (int u = 0; u < B; ++u)
#pragma unroll
            for (int p = 0; p < CPL; ++p) {
                if constexpr (COMP)
                    kahan_add(acc[p], comp[p], v[u][p], ok[u]);
                else
                    acc[p] += v[u][p];
            }
    }
};

struct GatherTabs {
    TypeInput in[kMaxTypes];
};


// Forward gather over the flattened stream of the schedule: every in-edge of a segment is
// one entry, and a self-loop row or a segment of degree 0 is one entry as well.  The
// stream is cut into balanced contiguous ranges of whole segments (chunks of kFwdChunk
// rows moved -- entries read plus one row written per segment -- split evenly over the
// groups of the grid), so every group moves about the same number of rows whatever the
// degrees, and consecutive segments' indices and row ids are read by the same group.
//
// A group of G lanes takes S = G entries per step.  A step's entries are resolved with one
// entry per lane: the G segment descriptors from the step's first segment are loaded one
// per lane, an inclusive scan of their entry counts and a binary search give each lane its
// segment and edge, and the source index and global row id of that edge follow.  Those
// three dependent loads are software-pipelined over the steps (descriptors of step i+3,
// source indices of step i+2, row ids of step i+1 in flight with the rows of step i).
// The rows of a step are loaded U at a time by all G lanes (16 bytes per lane per chunk),
// with the next batch in flight while one is summed; after the last entry of a segment
// the group writes its mean (sum in ascending edge order, one division by the degree; 0
// for degree 0).
template <bool BF16, int G, int CPL, int U, bool FULL>
__global__ __launch_bounds__(kThreads) void k_gather_flat(const SegDesc *__restrict__ desc,
                                                          const int32_t *__restrict__ cs,
                                                          int64_t nc_max,
                                                          const FwdSlot *__restrict__ slots,
                                                          int nslots, GatherTabs tabs,
                                                          char *__restrict__ ws, int chunks,
                                                          uint32_t *claims, int claim) {
    constexpr int VEC = BF16 ? 8 : 4;
    constexpr int ES = BF16 ? 2 : 4;
    constexpr int S = G;
    constexpr int GPW = 64 / G;
    constexpr int W = kThreads / 64;
    constexpr int NB = S / U;
    static_assert(S % U == 0 && (G & (G - 1)) == 0, "power-of-two groups, whole batches");
    __shared__ const int32_t *s_idx[kMaxSlots];
    __shared__ const int64_t *s_rows[kMaxSlots];
    __shared__ int32_t s_src[kMaxSlots];
    __shared__ TypeInput s_tab[kMaxTypes];
    __shared__ int64_t s_addr[W][64];
    __shared__ int64_t s_out[W][64];
    __shared__ int32_t s_deg[W][64];
    for (int i = threadIdx.x; i < nslots; i += kThreads) {
        s_idx[i] = slots[i].indices;
        s_rows[i] = slots[i].rows;
        s_src[i] = slots[i].src_type;
    }
    for (int i = threadIdx.x; i < kMaxTypes; i += kThreads) s_tab[i] = tabs.in[i];
    __syncthreads();

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int gb = lane & ~(G - 1);    // first lane of this lane's group
    const int lg = lane & (G - 1);
    const int64_t ngroups = (int64_t)gridDim.x * W * GPW;
    const int64_t gid = ((int64_t)blockIdx.x * W + wave) * GPW + lane / G;
    const int64_t total = cs[nc_max + 1];
    const int64_t nc = (total + kFwdChunk - 1) / kFwdChunk;
    // Work is claimed in runs of `claim` chunks: run gid first, then runs from the shared
    // counter (which starts at ngroups), each time this group's window stage reaches the
    // end of its run, so the stream continues without a pipeline restart.  Costs per row
    // differ between source tables (a row of the largest one costs more), which a static
    // split cannot know.
    auto run_of = [&](int64_t c, int32_t &lo, int32_t &hi) {
        const int64_t a = c * claim, b = a + claim < nc ? a + claim : nc;
        lo = a < nc ? cs[a] : 0;
        hi = a < nc ? cs[b] : 0;
        return a < nc;
    };
    int32_t s_lo, s_hi;
    bool live = run_of(gid, s_lo, s_hi);
    const char *zero = (const char *)g_zero;
    const int64_t zrow = (int64_t)(uintptr_t)g_zero_row;

    // window of the step starting at segment sc: lane lg holds segment sc + lg (degree -1
    // past the group's range)
    auto load_win = [&](int32_t sc) -> SegDesc {
        const int64_t sw = (int64_t)sc + lg;
        const bool in = sw < s_hi;
        SegDesc d = desc[in ? sw : 0];
        d.deg = in ? d.deg : -1;
        return d;
    };
    // per-lane entry of a step, after the scan
    struct Ent {
        int32_t k;      // edge position (edge entry) or row (self-loop entry)
        int32_t deg;    // degree of the entry's segment
        int64_t out;    // workspace byte offset of the segment's output
        int slot;
        int kind;       // 0 none, 1 degree-0 segment, 2 self-loop row, 3 edge
        bool last;      // last entry of its segment
    };
    // Resolve the step at (sc, e0) from its window d; advance (sc, e0) to the next step.
    auto scan = [&](const SegDesc &d, int32_t &sc, int32_t &e0) -> Ent {
        int w = d.deg < 0 ? 0 : (d.deg > 0 ? d.deg : 1);
        if (lg == 0) w -= e0;
        int incl = w;
#pragma unroll
        for (int o = 1; o < G; o <<= 1) {
            const int up = __shfl_up(incl, o, G);
            incl += lg >= o ? up : 0;
        }
        const int excl = incl - w;
        const int tot = __shfl(incl, gb + G - 1, 64);
        // segment of entry p: the last window lane whose first entry is <= p
        auto find = [&](int p) -> int {
            int j = 0;
#pragma unroll
            for (int st = G / 2; st >= 1; st >>= 1) {
                const int ex = __shfl(excl, gb + j + st, 64);
                j = ex <= p ? j + st : j;
            }
            return j;
        };
        const int j = find(lg);
        const int jx = __shfl(excl, gb + j, 64), ji = __shfl(incl, gb + j, 64);
        const int32_t k0 = __shfl(d.k0, gb + j, 64), dg = __shfl(d.deg, gb + j, 64);
        const uint32_t olo = __shfl(d.out_lo, gb + j, 64), inf = __shfl(d.info, gb + j, 64);
        Ent e;
        const bool valid = lg < tot;
        e.slot = (int)((inf >> 8) & 0xffu);
        const int ein = lg - jx + (j == 0 ? e0 : 0);
        const bool self = s_idx[e.slot] == nullptr;
        e.kind = !valid ? 0 : (dg == 0 ? 1 : (self ? 2 : 3));
        e.k = self ? k0 : k0 + ein;
        e.deg = dg;
        e.out = (int64_t)((((uint64_t)(inf & 0xffu) << 32) | olo) << 4);
        e.last = valid && lg == ji - 1;
        // next step: the segment holding entry S of this window
        const int js = find(S);
        const int sx = __shfl(excl, gb + js, 64), si = __shfl(incl, gb + js, 64);
        if (si <= S) {
            sc += js + 1;
            e0 = 0;
        } else {
            e0 = S - sx + (js == 0 ? e0 : 0);
            sc += js;
        }
        return e;
    };
    // source of an entry: its row within its type, or, for an edge of a relation whose
    // table rows are given per edge, that table row; -1 for none
    auto load_src = [&](const Ent &e) -> int64_t {
        const bool edge = e.kind == 3;
        const int64_t *pr = s_rows[e.slot];
        int64_t v;
        if (pr != nullptr) {
            v = *gbl(edge ? pr + e.k : (const int64_t *)zero);
        } else {
            v = *gbl(edge ? s_idx[e.slot] + e.k : (const int32_t *)zero);
        }
        return edge ? v : (e.kind == 2 ? (int64_t)e.k : -1);
    };
    // absolute address of that row (the zero row for none): a row within the type goes
    // through the type's row ids, a per-edge table row is used as it is
    auto load_addr = [&](int slot, int64_t j) -> int64_t {
        const int t = s_src[slot];
        const int64_t *rid = s_tab[t].row_ids;
        const bool ids = rid != nullptr && s_rows[slot] == nullptr;
        const int64_t v = *gbl((j >= 0 && ids) ? rid + j : (const int64_t *)zero);
        const int64_t row = ids ? v : j;
        return j < 0 ? zrow : (int64_t)(uintptr_t)s_tab[t].base + row * (s_tab[t].ld * ES);
    };

    int32_t sc = s_lo, e0 = 0;
    // after a scan: at the end of the run, continue with the next claimed run
    // with no more runs than groups every run is taken first and nobody claims
    const bool shared = (nc + claim - 1) / claim > ngroups;
    auto next_run = [&]() {
        const bool need = live && sc >= s_hi;
        uint32_t c = (uint32_t)ngroups;   // past the last run when nothing is shared
        if (shared && need && lg == 0) c = atomicAdd(claims, 1u);
        c = __shfl(c, gb, 64);
        if (need) {
            live = run_of(c, s_lo, s_hi);
            sc = live ? s_lo : sc;
            e0 = 0;
        }
    };

    // pipeline prologue: steps 0, 1, 2
    SegDesc dw = load_win(sc);
    Ent ez = scan(dw, sc, e0);
    next_run();
    dw = load_win(sc);
    int64_t jz = load_src(ez);
    Ent ey = scan(dw, sc, e0);
    next_run();
    dw = load_win(sc);
    int64_t jy = load_src(ey);
    int64_t az = load_addr(ez.slot, jz);

    float acc[CPL][VEC];
#pragma unroll
    for (int p = 0; p < CPL; ++p)
#pragma unroll
        for (int v = 0; v < VEC; ++v) acc[p][v] = 0.f;

    // a step with no entries (the end of a run, an empty run) does not end a group: it
    // ends when nothing is in flight and it can claim no more
    while (__ballot(ez.kind != 0 || ey.kind != 0 || dw.deg >= 0 || live) != 0) {
        __builtin_amdgcn_wave_barrier();
        s_addr[wave][lane] = az;
        s_out[wave][lane] = ez.out;
        s_deg[wave][lane] = ez.deg;
        uint64_t lm = __ballot(ez.last);
        if constexpr (G < 64) lm = (lm >> gb) & ((1ull << G) - 1);
        __builtin_amdgcn_wave_barrier();

        u32x4 v[2][U][CPL];
        auto issue = [&](int b, u32x4 (&dst)[U][CPL]) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t a = s_addr[wave][gb + b * U + u];
#pragma unroll
                for (int p = 0; p < CPL; ++p) {
                    const int c = lg + p * G;
                    const int64_t pa = (FULL || c < chunks) ? a + (int64_t)c * 16 : zrow + (int64_t)c * 16;
                    dst[u][p] = ld_row((const char *)(uintptr_t)pa);
                }
            }
        };
        // this step's first rows, then the later pipeline stages while they are in flight
        issue(0, v[0]);
        Ent ex = scan(dw, sc, e0);
        next_run();
        dw = load_win(sc);
        const int64_t jx = load_src(ex);
        const int64_t ay = load_addr(ey.slot, jy);
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            if (b + 1 < NB) issue(b + 1, v[(b + 1) & 1]);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int q = b * U + u;
#pragma unroll
                for (int p = 0; p < CPL; ++p) {
                    const u32x4 x = v[b & 1][u][p];
                    acc_chunk<BF16>(acc[p], make_uint4(x.x, x.y, x.z, x.w));
                }
                if ((lm >> q) & 1u) {
                    const int64_t ob = s_out[wave][gb + q];
                    const int dg = s_deg[wave][gb + q];
                    // sum / deg by the reciprocal; fp32 output takes one correction from
                    // the exact remainder (fma), bf16 output is rounded to 8 bits anyway.
                    // Degree 0 has a zero sum and gives 0.
                    const float fdeg = (float)dg;
                    const float rc = dg > 0 ? __builtin_amdgcn_rcpf(fdeg) : 0.f;
                    char *out = ws + ob;
#pragma unroll
                    for (int p = 0; p < CPL; ++p) {
                        const int c = lg + p * G;
                        float r[VEC];
#pragma unroll
                        for (int e = 0; e < VEC; ++e) {
                            const float q0 = acc[p][e] * rc;
                            if constexpr (BF16)
                                r[e] = q0;
                            else
                                r[e] = __builtin_fmaf(__builtin_fmaf(-q0, fdeg, acc[p][e]), rc, q0);
                            acc[p][e] = 0.f;
                        }
                        if (!FULL && c >= chunks) continue;
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
            }
        }
        ez = ey;
        az = ay;
        ey = ex;
        jy = jx;
    }
}

// Stores of one 4-column chunk `res` of source row j's input gradient (global row grow),
// all non-temporal (each row is written once here and read only by a later kernel, long
// after it would have left L2; streaming stores took block 1's hi/lo input-gradient
// writes from 1.85 to 1.76 ms):
// the dh_src row, then one of
//  - Adagrad mode: the table row takes one step, state += res^2 and
//    w -= lr res / (sqrt(state) + eps), with `old` the state and `cur` the table values
//    read before the sum (each row belongs to one group, so no other lane touches it);
//  - demb += res, as a read-add-write of `old` when ids are unique, else by atomics.
// OFF_HERE: the lane's byte offset is formed at the store (kept across the row loop as
// part of a 64-bit address it costs two registers for the whole kernel, which the bit
// form at two chunks per lane cannot spare)
template <bool BF16IN, bool OPT, bool OFF_HERE = false>
__device__ __forceinline__ void tsum_store(const TsumArgs &a, int64_t j, int64_t grow, int c,
                                           f32x4 res, f32x4 old, f32x4 cur) {
    int co = c * 16;
    if constexpr (OFF_HERE) asm volatile("" : "+v"(co));
    if (a.dh) {
        if (a.dh_hilo) {
            // the 4 values' bf16 high parts at element 4 c of the row's first half, their
            // low parts at the same place in the second half
            const uint32_t h0 = pack_bf16x2(res[0], res[1]), h1 = pack_bf16x2(res[2], res[3]);
            const uint32_t l0 = pack_bf16x2(res[0] - bf16_lo(h0), res[1] - bf16_hi(h0));
            const uint32_t l1 = pack_bf16x2(res[2] - bf16_lo(h1), res[3] - bf16_hi(h1));
            char *rp = (char *)(a.dh + j * a.d_in) + co / 2;
            __builtin_nontemporal_store(u32x2{h0, h1}, (u32x2 *)rp);
            __builtin_nontemporal_store(u32x2{l0, l1}, (u32x2 *)(rp + (int64_t)a.d_in * 2));
        } else if constexpr (OFF_HERE) {
            __builtin_nontemporal_store(res, (f32x4 *)((char *)(a.dh + j * a.d_in) + co));
        } else {
            __builtin_nontemporal_store(res, (f32x4 *)(a.dh + j * a.d_in + (int64_t)c * 4));
        }
    }
    if constexpr (OPT) {
        const f32x4 st = old + res * res;
        f32x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e) w[e] = cur[e] - a.lr * res[e] / (sqrtf(st[e]) + a.eps);
        __builtin_nontemporal_store(st, (f32x4 *)(a.opt_state + grow * a.d_in + (int64_t)c * 4));
        char *tp = (char *)a.opt_table + (grow * a.in.ld + (int64_t)c * 4) * (BF16IN ? 2 : 4);
        if constexpr (BF16IN) {
            typedef uint32_t u2 __attribute__((ext_vector_type(2)));
            __builtin_nontemporal_store(u2{pack_bf16x2(w[0], w[1]), pack_bf16x2(w[2], w[3])}, (u2 *)tp);
        } else {
            __builtin_nontemporal_store(w, (f32x4 *)tp);
        }
    } else if (a.demb) {
        float *dp = OFF_HERE ? (float *)((char *)(a.demb + grow * a.d_in) + co)
                             : a.demb + grow * a.d_in + (int64_t)c * 4;
        if (a.ids_unique) {
            __builtin_nontemporal_store(old + res, (f32x4 *)dp);
        } else {
            unsafeAtomicAdd(dp + 0, res[0]);
            unsafeAtomicAdd(dp + 1, res[1]);
            unsafeAtomicAdd(dp + 2, res[2]);
            unsafeAtomicAdd(dp + 3, res[3]);
        }
    }
}

// Backward, one group per source row j of one node type, in schedule order:
//   acc = [j < n_dst] dMs_self[j] + sum over relations leaving the type, over the
//         transpose segment of j (ascending destination row), of dMs_r[i]
// where dMs rows already carry the 1/deg factor.  Then the optional ReLU-input mask,
// the dh_src store and the embedding scatter-add demb[row_ids[j]] += acc, or (OPT) the
// Adagrad step of table row row_ids[j] with gradient acc.
// Lanes first fetch the transpose offsets of up to G relations at once, then the
// destination rows of up to G edges at once (flattened relation by relation), then walk
// the edges broadcasting row addresses, U row loads in flight; the embedding-gradient
// row and the ReLU mask input are requested before the walk.
template <bool BF16IN, int CPL, bool OPT, bool MASK>
__device__ __forceinline__ void transpose_sum_body(const TsumArgs &a, int G, int gpw,
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
    if (a.split_np != nullptr && a.split_np[j] > 0) return;   // summed by the piece kernels
    const int64_t grow = a.in.row_ids ? a.in.row_ids[j] : j;

    // early requests: embedding-gradient row (read-add-write) or Adagrad state, ReLU mask
    // input or the table row the step updates, self term
    float4 old[CPL];
    float hm[CPL][4];
    float acc[CPL][4];
#pragma unroll
    for (int p = 0; p < CPL; ++p) {
        const int c = lg + p * G;
        const bool okc = c < chunks;
        const float *ob = OPT ? a.opt_state : (a.ids_unique ? a.demb : nullptr);
        old[p] = (ob && okc) ? *(const float4 *)(ob + grow * a.d_in + (int64_t)c * 4)
                             : make_float4(0.f, 0.f, 0.f, 0.f);
        if constexpr (MASK) {
            const f32x4 b = relu_bits4(a.relu_mask, a.mask_ld, grow, c, okc, (const char *)g_zero);
            hm[p][0] = b[0]; hm[p][1] = b[1]; hm[p][2] = b[2]; hm[p][3] = b[3];
        } else if ((a.input_relu || OPT) && okc) {
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
        tsum_store<BF16IN, OPT>(a, j, grow, c, f32x4{acc[p][0], acc[p][1], acc[p][2], acc[p][3]},
                           f32x4{old[p].x, old[p].y, old[p].z, old[p].w},
                           f32x4{hm[p][0], hm[p][1], hm[p][2], hm[p][3]});
    }
}

// The same sum, persistent and software-pipelined over a group's successive source rows
// (used when the relations leaving the type fit in one group, nrel <= G).  A row takes
// four dependent steps: its schedule entry j; the global row id and, on lane r, the
// transpose offsets of relation r; on lane e, the destination row of flattened edge e
// (with the embedding-gradient or Adagrad-state row, the ReLU-mask input or table row, and
// the self term); the dMs rows.
// While the rows of one source row are in flight, the earlier steps of the next three
// rows are too.  Edges past the group width are resolved in place.  Every load is
// unconditional (unused lanes read a zero word).

// PF (one chunk per lane): a fourth stage loads the first edge's dMs row of the next row
// while the current one is summed, so each wave has two rows' reads in flight instead of
// one.  (At two chunks per lane, where sources of a hidden block mostly have one edge, it
// measured slower: the registers of the extra stage cost a wave per SIMD.)
template <bool BF16IN, int CPL, bool OPT, bool MASK>
__device__ __forceinline__ void transpose_pipe_body(const TsumArgs &a, int G, int gpw,
                                                    int chunks) {
    constexpr int HES = BF16IN ? 2 : 4;
    constexpr int U = 4;   // rows in flight per lane
    constexpr bool PF = CPL == 1;
    constexpr int W = kThreads / 64;
    __shared__ TsumRel s_rel[kMaxRels];
    __shared__ int64_t s_off[W][64];
    for (int i = threadIdx.x; i < a.nrel; i += kThreads) s_rel[i] = a.rel[i];
    __syncthreads();

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int gi = lane / G;
    const int lg = lane - gi * G;
    const int g0 = gi * G;
    if (gi >= gpw) return;
    int64_t *goff = &s_off[wave][g0];
    const int64_t stride = (int64_t)gridDim.x * W * gpw;
    int64_t g = ((int64_t)blockIdx.x * W + wave) * gpw + gi;
    if (g >= a.n_rows) return;
    const char *zero = (const char *)g_zero;
    const int nrel = a.nrel;
    const int rl = lg < nrel ? lg : 0;   // this lane's relation (stage 2)

    struct Meta {
        int32_t j, p0, cnt;
        int64_t grow;
    };
    struct Row {
        Meta m;
        int32_t total, ei, er;
        bool split;     // more than kSplitEdges edges: the piece kernels sum this row
        f32x4 old[CPL], self[CPL], hm[CPL];
        uint32_t hb[CPL];   // MASK: the 4 sign bits of each chunk (hm unused)
        f32x4 pre[CPL];     // PF: the first edge's dMs row (zero if the row has no edge)
    };
    // stage 1: source row at schedule position q (-1 past the end)
    auto s1 = [&](int64_t q) -> int32_t {
        const int32_t v = *gbl(a.order + (q < a.n_rows ? q : a.n_rows - 1));
        return q < a.n_rows ? v : -1;
    };
    // stage 2: global row id; lane r < nrel: transpose segment of relation r
    auto s2 = [&](int32_t j) -> Meta {
        Meta m;
        m.j = j;
        const bool okj = j >= 0;
        const int64_t *rid = a.in.row_ids;
        const int64_t gv = *gbl((okj && rid != nullptr) ? rid + j : (const int64_t *)zero);
        m.grow = gv + (rid != nullptr ? 0 : (int64_t)j);
        const bool okr = okj && lg < nrel;
        const int32_t *ip = okr ? s_rel[rl].csc_indptr + j : (const int32_t *)zero;
        const int32_t v0 = *gbl(ip), v1 = *gbl(ip + (okr ? 1 : 0));
        m.p0 = v0;
        m.cnt = v1 - v0;
        return m;
    };
    // flattened edge e of a row -> (relation, position in the shared transpose arrays)
    auto locate = [&](const Meta &m, int e, int &r_out, int &pos_out) -> int {
        int total = 0, ridx = 0, pos = 0;
        for (int r = 0; r < nrel; ++r) {
            const int cr = __shfl(m.cnt, g0 + r, 64);
            const int pr = __shfl(m.p0, g0 + r, 64);
            const bool in = e >= total && e < total + cr;
            ridx = in ? r : ridx;
            pos = in ? pr + (e - total) : pos;
            total += cr;
        }
        r_out = ridx;
        pos_out = pos;
        return total;
    };
    // stage 3: destination row of this lane's edge, and the row's per-chunk side data
    auto s3 = [&](const Meta &m, Row &rw) {
        rw.m = m;
        int ridx, pos;
        rw.total = locate(m, lg, ridx, pos);
        // the plan split exactly the rows whose degree passes the threshold
        rw.split = a.split_np != nullptr && rw.total > kSplitEdges;
        if (rw.split) rw.total = 0;
        const bool oke = lg < rw.total;
        rw.ei = *gbl(oke ? s_rel[ridx].csc_dst + pos : (const int32_t *)zero);
        rw.er = ridx;
#pragma unroll
        for (int p = 0; p < CPL; ++p) {
            const int c = lg + p * G;
            const bool okc = c < chunks && m.j >= 0 && !rw.split;
            // row read before the sum: Adagrad state, or the embedding gradient when ids
            // are unique.  (Written this way, pointer chosen here and the flag test in the
            // predicate: forms that pick the pointer once before the loop measured 9%
            // slower at d = 128.)
            if constexpr (MASK) {
                rw.old[p] = f32x4{0.f, 0.f, 0.f, 0.f};   // never read (see transpose_sum_dt)
            } else {
                const bool ok_old = OPT ? okc : (okc && a.demb != nullptr && a.ids_unique);
                const float *ob = OPT ? a.opt_state : a.demb;
                rw.old[p] = *gbl(ok_old ? (const f32x4 *)(ob + m.grow * a.d_in + (int64_t)c * 4)
                                        : (const f32x4 *)zero);
            }
            const bool ok_self = okc && a.self_dms != nullptr && m.j < a.n_dst;
            rw.self[p] = *gbl(ok_self ? (const f32x4 *)(a.self_dms + m.j * a.self_ld + (int64_t)c * 4)
                                      : (const f32x4 *)zero);
            const bool ok_h = okc && (a.input_relu || OPT);
            if constexpr (MASK) {
                const uint64_t w = *gbl(ok_h ? a.relu_mask + m.grow * a.mask_ld + (c >> 4)
                                             : (const uint64_t *)zero);
                rw.hb[p] = (uint32_t)(w >> (4 * (c & 15))) & 0xFu;
            } else {
                const char *hp = ok_h ? (const char *)a.in.base +
                                            (m.grow * a.in.ld + (int64_t)c * 4) * HES
                                      : zero;
                if constexpr (BF16IN) {
                    const u32x2 hv = *gbl((const u32x2 *)hp);
                    rw.hm[p] = f32x4{bf16_lo(hv.x), bf16_hi(hv.x), bf16_lo(hv.y), bf16_hi(hv.y)};
                } else {
                    rw.hm[p] = *gbl((const f32x4 *)hp);
                }
            }
        }
    };
    // rows [0, n) whose addresses are in goff, added into acc; a batch's unused slots re-read
    // the last row and are dropped
    auto rows = [&](const int64_t *go, int n, f32x4 (&acc)[CPL]) {
        row_walk<U>(go, n, SumLoad<CPL, false>{lg, G, chunks, acc, nullptr});
    };
    auto edge_addr = [&](int r, int32_t i) -> int64_t {
        return (int64_t)(uintptr_t)(s_rel[r].dms + (int64_t)i * s_rel[r].dms_ld);
    };
    // stage 4 (PF): edge 0 of the row is held by the group's first lane
    auto s4 = [&](Row &rw) {
        const int er0 = __shfl(rw.er, g0, 64);
        const int32_t ei0 = __shfl(rw.ei, g0, 64);
        const bool okp = rw.total > 0;
        const char *base = okp ? (const char *)(uintptr_t)edge_addr(er0, ei0)
                               : (const char *)g_zero_row;
#pragma unroll
        for (int p = 0; p < CPL; ++p) {
            const int c = lg + p * G;
            const char *pa = (okp && c < chunks) ? base + (int64_t)c * 16
                                                 : (const char *)g_zero_row + c * 16;
            rw.pre[p] = *gbl((const f32x4 *)pa);
        }
    };
    // last step of a row: its dMs rows, the mask, the stores
    auto finish = [&](const Row &rw) {
        f32x4 acc[CPL];
#pragma unroll
        for (int p = 0; p < CPL; ++p) acc[p] = rw.self[p];
        const int n1 = rw.total < G ? rw.total : G;
        goff[lg] = edge_addr(rw.er, rw.ei);
        __builtin_amdgcn_wave_barrier();
        if constexpr (PF) {
            if (rw.total > 0) {
#pragma unroll
                for (int p = 0; p < CPL; ++p) acc[p] += rw.pre[p];
            }
            rows(goff + 1, n1 > 1 ? n1 - 1 : 0, acc);
        } else {
            rows(goff, n1, acc);
        }
        for (int ec = G; ec < rw.total; ec += G) {
            int ridx, pos;
            locate(rw.m, ec + lg, ridx, pos);
            const bool oke = ec + lg < rw.total;
            const int32_t i = *gbl(oke ? s_rel[ridx].csc_dst + pos : (const int32_t *)zero);
            __builtin_amdgcn_wave_barrier();
            goff[lg] = edge_addr(ridx, i);
            __builtin_amdgcn_wave_barrier();
            rows(goff, rw.total - ec < G ? rw.total - ec : G, acc);
        }
        __builtin_amdgcn_wave_barrier();
        if (rw.split) return;
#pragma unroll
        for (int p = 0; p < CPL; ++p) {
            const int c = lg + p * G;
            if (c >= chunks) continue;
            f32x4 res = acc[p];
            if constexpr (MASK) {
#pragma unroll
                for (int e = 0; e < 4; ++e) res[e] = (rw.hb[p] >> e) & 1u ? res[e] : 0.f;
            } else if (a.input_relu) {
#pragma unroll
                for (int e = 0; e < 4; ++e) res[e] = rw.hm[p][e] > 0.f ? res[e] : 0.f;
            }
            tsum_store<BF16IN, OPT, MASK>(a, rw.m.j, rw.m.grow, c, res, rw.old[p],
                                    MASK ? f32x4{0.f, 0.f, 0.f, 0.f} : rw.hm[p]);
        }
    };

    if constexpr (PF) {
        // prologue: row g through stage 4, g+stride through stage 3, g+2 stride through
        // stage 2, g+3 stride through stage 1
        Row cur, nxt;
        s3(s2(s1(g)), cur);
        s4(cur);
        s3(s2(s1(g + stride)), nxt);
        Meta mn = s2(s1(g + 2 * stride));
        int32_t jnn = s1(g + 3 * stride);
        while (true) {
            Row nn;
            s3(mn, nn);
            const Meta mnn = s2(jnn);
            const int32_t jn4 = s1(g + 4 * stride);
            s4(nxt);
            finish(cur);
            g += stride;
            if (g >= a.n_rows) break;
            cur = nxt;
            nxt = nn;
            mn = mnn;
            jnn = jn4;
        }
    } else {
        // prologue: row g through stage 3, row g+stride through stage 2, row g+2*stride
        // through stage 1
        Row cur;
        s3(s2(s1(g)), cur);
        Meta mn = s2(s1(g + stride));
        int32_t jnn = s1(g + 2 * stride);
        while (true) {
            Row nxt;
            s3(mn, nxt);
            const Meta mnn = s2(jnn);
            const int32_t jn3 = s1(g + 3 * stride);
            finish(cur);
            g += stride;
            if (g >= a.n_rows) break;
            cur = nxt;
            mn = mnn;
            jnn = jn3;
        }
    }
}

// Rows split into pieces (transpose degree above kSplitEdges).  Piece p = (row j, number q)
// is the sum of the dMs rows of edges [q P, min((q + 1) P, deg)) of row j's transpose,
// flattened relation by relation in order, edges in order; it goes to partial[p].  Lanes
// r < nrel of a group hold relation r's segment of row j (in blocks of G relations), the
// group resolves G edges at a time and keeps the rows' loads in flight through row_walk.
template <int CPL>
__device__ __forceinline__ void pieces_body(const TsumArgs &a, int G, int gpw, int chunks) {
    constexpr int U = CPL == 1 ? 8 : 4;
    constexpr int W = kThreads / 64;
    __shared__ TsumRel s_rel[kMaxRels];
    __shared__ int64_t s_off[W][64];
    for (int i = threadIdx.x; i < a.nrel; i += kThreads) s_rel[i] = a.rel[i];
    __syncthreads();
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int gi = lane / G;
    const int lg = lane - gi * G;
    const int g0 = gi * G;
    if (gi >= gpw) return;
    int64_t *goff = &s_off[wave][g0];
    const uint32_t cnt_all = *a.piece_count;
    const int64_t n = (int64_t)cnt_all < a.piece_cap ? (int64_t)cnt_all : a.piece_cap;
    const int64_t stride = (int64_t)gridDim.x * W * gpw;
    const int64_t zrow = (int64_t)(uintptr_t)g_zero_row;
    for (int64_t p = ((int64_t)blockIdx.x * W + wave) * gpw + gi; p < n; p += stride) {
        const int2 pc = a.pieces[p];
        const int64_t j = pc.x;
        const int e0 = pc.y * kSplitEdges, e1 = e0 + kSplitEdges;
        f32x4 acc[CPL], comp[CPL];
#pragma unroll
        for (int q = 0; q < CPL; ++q) acc[q] = comp[q] = f32x4{0.f, 0.f, 0.f, 0.f};
        int base = 0;   // flattened index of the first edge of relation block r0
        for (int r0 = 0; r0 < a.nrel && base < e1; r0 += G) {
            const int nr = (a.nrel - r0) < G ? (a.nrel - r0) : G;
            int p0 = 0, cnt = 0;
            if (lg < nr) {
                const int32_t *ip = s_rel[r0 + lg].csc_indptr;
                p0 = ip[j];
                cnt = ip[j + 1] - p0;
            }
            int tot = 0;
            for (int r = 0; r < nr; ++r) tot += __shfl(cnt, g0 + r, 64);
            const int lo = e0 - base > 0 ? e0 - base : 0;
            const int hi = e1 - base < tot ? e1 - base : tot;
            for (int ec = lo; ec < hi; ec += G) {
                const int e = ec + lg;
                int64_t addr = zrow;
                int b = 0;
                for (int r = 0; r < nr; ++r) {
                    const int cr = __shfl(cnt, g0 + r, 64);
                    const int pr = __shfl(p0, g0 + r, 64);
                    if (e < hi && e >= b && e < b + cr) {
                        const TsumRel &rel = s_rel[r0 + r];
                        const int64_t i = rel.csc_dst[pr + (e - b)];
                        addr = (int64_t)(uintptr_t)(rel.dms + i * rel.dms_ld);
                    }
                    b += cr;
                }
                __builtin_amdgcn_wave_barrier();
                goff[lg] = addr;
                __builtin_amdgcn_wave_barrier();
                row_walk<U>(goff, hi - ec < G ? hi - ec : G, SumLoad<CPL, true>{lg, G, chunks, acc, comp});
                __builtin_amdgcn_wave_barrier();
            }
            base += tot;
        }
#pragma unroll
        for (int q = 0; q < CPL; ++q) {
            const int c = lg + q * G;
            if (c < chunks) *(f32x4 *)(a.partial + p * a.d_in + (int64_t)c * 4) = acc[q];
        }
    }
}

// The rows split into pieces, finished: one group per split row (found through its first
// piece) adds its self term and its pieces' partial sums in piece order, then applies the
// mask and the stores of the transposed sum (dh_src, the embedding gradient or the Adagrad
// step).
template <bool BF16IN, int CPL, bool OPT, bool MASK>
__device__ __forceinline__ void split_finish_body(const TsumArgs &a, int G, int gpw, int chunks) {
    constexpr int HES = BF16IN ? 2 : 4;
    constexpr int U = CPL == 1 ? 8 : 4;
    constexpr int W = kThreads / 64;
    __shared__ int64_t s_off[W][64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int gi = lane / G;
    const int lg = lane - gi * G;
    const int g0 = gi * G;
    if (gi >= gpw) return;
    int64_t *goff = &s_off[wave][g0];
    const uint32_t cnt_all = *a.piece_count;
    const int64_t n = (int64_t)cnt_all < a.piece_cap ? (int64_t)cnt_all : a.piece_cap;
    const int64_t stride = (int64_t)gridDim.x * W * gpw;
    for (int64_t p = ((int64_t)blockIdx.x * W + wave) * gpw + gi; p < n; p += stride) {
        const int2 pc = a.pieces[p];
        if (pc.y != 0) continue;
        const int64_t j = pc.x;
        const int np = a.split_np[j];
        const int64_t pb = a.split_base[j];
        const int64_t grow = a.in.row_ids ? a.in.row_ids[j] : j;
        f32x4 acc[CPL], comp[CPL], old[CPL], hm[CPL];
#pragma unroll
        for (int q = 0; q < CPL; ++q) {
            const int c = lg + q * G;
            const bool okc = c < chunks;
            const float *ob = OPT ? a.opt_state : (a.ids_unique ? a.demb : nullptr);
            old[q] = (ob && okc) ? *(const f32x4 *)(ob + grow * a.d_in + (int64_t)c * 4)
                                 : f32x4{0.f, 0.f, 0.f, 0.f};
            hm[q] = f32x4{1.f, 1.f, 1.f, 1.f};
            if constexpr (MASK) {
                hm[q] = relu_bits4(a.relu_mask, a.mask_ld, grow, c, okc, (const char *)g_zero);
            } else if ((a.input_relu || OPT) && okc) {
                const char *hp = (const char *)a.in.base + (grow * a.in.ld + (int64_t)c * 4) * HES;
                if constexpr (BF16IN) {
                    const uint2 hv = *(const uint2 *)hp;
                    hm[q] = f32x4{bf16_lo(hv.x), bf16_hi(hv.x), bf16_lo(hv.y), bf16_hi(hv.y)};
                } else {
                    hm[q] = *(const f32x4 *)hp;
                }
            }
            acc[q] = (a.self_dms && j < a.n_dst && okc)
                         ? *(const f32x4 *)(a.self_dms + j * a.self_ld + (int64_t)c * 4)
                         : f32x4{0.f, 0.f, 0.f, 0.f};
            comp[q] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
        for (int q0 = 0; q0 < np; q0 += G) {
            __builtin_amdgcn_wave_barrier();
            goff[lg] = (int64_t)(uintptr_t)(a.partial + (pb + q0 + (q0 + lg < np ? lg : 0)) * a.d_in);
            __builtin_amdgcn_wave_barrier();
            row_walk<U>(goff, np - q0 < G ? np - q0 : G, SumLoad<CPL, true>{lg, G, chunks, acc, comp});
        }
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int q = 0; q < CPL; ++q) {
            const int c = lg + q * G;
            if (c >= chunks) continue;
            f32x4 res = acc[q];
            if (a.input_relu) {
#pragma unroll
                for (int e = 0; e < 4; ++e) res[e] = hm[q][e] > 0.f ? res[e] : 0.f;
            }
            tsum_store<BF16IN, OPT>(a, j, grow, c, res, old[q], hm[q]);
        }
    }
}

template <int CPL>
__global__ __launch_bounds__(kThreads) void k_transpose_pieces(TsumArgs a, int G, int gpw,
                                                               int chunks) {
    pieces_body<CPL>(a, G, gpw, chunks);
}
template <bool BF16IN, int CPL, bool OPT, bool MASK>
__global__ __launch_bounds__(kThreads) void k_transpose_split_finish(TsumArgs a, int G, int gpw,
                                                                     int chunks) {
    split_finish_body<BF16IN, CPL, OPT, MASK>(a, G, gpw, chunks);
}

// The transposed sums as kernels; the Adagrad forms carry a name of their own so that
// traces and counters keep them apart.
template <bool BF16IN, int CPL, bool MASK>
__global__ __launch_bounds__(kThreads) void k_transpose_sum(TsumArgs a, int G, int gpw,
                                                            int chunks) {
    transpose_sum_body<BF16IN, CPL, false, MASK>(a, G, gpw, chunks);
}
template <bool BF16IN, int CPL>
__global__ __launch_bounds__(kThreads) void k_transpose_sum_adagrad(TsumArgs a, int G, int gpw,
                                                                    int chunks) {
    transpose_sum_body<BF16IN, CPL, true, false>(a, G, gpw, chunks);
}
// the bit form at two chunks per lane (hidden layers of 512) is held to 128 registers, so
// four of its waves share a SIMD
template <bool BF16IN, int CPL, bool MASK>
__global__ __launch_bounds__(kThreads, (MASK && CPL == 2) ? 4 : 1) void k_transpose_pipe(
    TsumArgs a, int G, int gpw, int chunks) {
    transpose_pipe_body<BF16IN, CPL, false, MASK>(a, G, gpw, chunks);
}
template <bool BF16IN, int CPL>
__global__ __launch_bounds__(kThreads) void k_transpose_pipe_adagrad(TsumArgs a, int G, int gpw,
                                                                     int chunks) {
    transpose_pipe_body<BF16IN, CPL, true, false>(a, G, gpw, chunks);
}

// WcatT[n][s*d_in + c] = W_s[c][n]: the forward transform's weights, K-contiguous.
struct WSlots {
    const void *w[kMaxSlots];
};
// The slots stacked as one [K x d_out] matrix (row kk = s d_in + c) are transposed in
// 64 x 64 tiles through LDS: a tile's rows are read along n and written along kk, so both
// sides are whole contiguous pieces; the padded LDS row keeps the column reads off one
// bank.
constexpr int kPackTile = 64;
template <typename T>
__global__ __launch_bounds__(kThreads) void k_pack_weights(WSlots ws, int nslots, int d_in,
                                                           int d_out, T *out) {
    __shared__ T tile[kPackTile][kPackTile + 1];
    const int K = nslots * d_in;
    const int kk0 = blockIdx.x * kPackTile, n0 = blockIdx.y * kPackTile;
    const int tx = threadIdx.x % kPackTile, ty = threadIdx.x / kPackTile;
    constexpr int kRowsPerPass = kThreads / kPackTile;
    for (int r = ty; r < kPackTile; r += kRowsPerPass) {
        const int kk = kk0 + r, n = n0 + tx;
        if (kk < K && n < d_out) {
            const int sl = kk / d_in, c = kk - sl * d_in;
            tile[r][tx] = ((const T *)ws.w[sl])[(int64_t)c * d_out + n];
        }
    }
    __syncthreads();
    for (int r = ty; r < kPackTile; r += kRowsPerPass) {
        const int n = n0 + r, kk = kk0 + tx;
        if (n < d_out && kk < K) out[(int64_t)n * K + kk] = tile[tx][r];
    }
}

// Deterministic column sums: partial[split][o] over a fixed row range, then a fixed-order
// sum over splits.
// hilo: dy rows in the hi/lo form (cols bf16 high parts, then cols low parts); an element
// is then hi + lo
__global__ __launch_bounds__(kThreads) void k_colsum_partial(const float *dy, int hilo,
                                                             int64_t rows, int cols,
                                                             int64_t rows_per_split,
                                                             float *partial) {
    const int o = blockIdx.x * kThreads + threadIdx.x;
    if (o >= cols) return;
    const int64_t r0 = (int64_t)blockIdx.y * rows_per_split;
    const int64_t r1 = r0 + rows_per_split < rows ? r0 + rows_per_split : rows;
    float acc = 0.f;
    if (hilo) {
        const uint16_t *h = (const uint16_t *)dy;
        for (int64_t r = r0; r < r1; ++r)
            acc += __uint_as_float((uint32_t)h[r * 2 * cols + o] << 16) +
                   __uint_as_float((uint32_t)h[r * 2 * cols + cols + o] << 16);
    } else {
        for (int64_t r = r0; r < r1; ++r) acc += dy[r * cols + o];
    }
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

// rows in flight per lane in the gather (for one chunk per lane)
constexpr int kFlatRows = 8;

template <bool B, int G, int C, bool FULL>
hipError_t launch_flat_k(const SegDesc *desc, const int32_t *cs, int64_t nc_max,
                         const FwdSlot *slots_dev, int nslots, const GatherTabs &tabs,
                         char *ws_base, int chunks, uint32_t *claims, hipStream_t s) {
    constexpr int U0 = kFlatRows / C > 0 ? kFlatRows / C : 1;
    constexpr int U = U0 < G ? U0 : G;
    const int64_t groups_per_wg = (int64_t)(kThreads / 64) * (64 / G);
    const int64_t cap = resident_wgs(k_gather_flat<B, G, C, U, FULL>);
    // runs of up to kFwdClaim chunks, fewer when that would leave about three runs or less
    // per resident group (a small block then still spreads over the grid)
    int64_t claim = nc_max / (3 * cap * groups_per_wg);
    claim = claim < 1 ? 1 : (claim > kFwdClaim ? kFwdClaim : claim);
    int64_t wgs = cdiv(cdiv(nc_max, claim), groups_per_wg);
    if (wgs > cap) wgs = cap;
    if (wgs < 1) wgs = 1;
    // the shared run counter starts past the runs the groups take first
    const uint32_t first = (uint32_t)(wgs * groups_per_wg);
    RGCN_HIP_TRY(fill_words(claims, &first, 4, s));
    hipLaunchKernelGGL((k_gather_flat<B, G, C, U, FULL>), dim3((unsigned)wgs), dim3(kThreads), 0,
                       s, desc, cs, nc_max, slots_dev, nslots, tabs, ws_base, chunks, claims,
                       (int)claim);
    return hipGetLastError();
}
template <bool B, int G, int C>
hipError_t launch_flat(const SegDesc *desc, const int32_t *cs, int64_t nc_max,
                       const FwdSlot *slots_dev, int nslots, const GatherTabs &tabs,
                       char *ws_base, int chunks, uint32_t *claims, hipStream_t s) {
    // every lane of a group owns a chunk of the row: no per-lane range checks
    if (chunks == G * C)
        return launch_flat_k<B, G, C, true>(desc, cs, nc_max, slots_dev, nslots, tabs, ws_base,
                                            chunks, claims, s);
    return launch_flat_k<B, G, C, false>(desc, cs, nc_max, slots_dev, nslots, tabs, ws_base,
                                         chunks, claims, s);
}

template <bool B>
hipError_t flat_dispatch(const SegDesc *desc, const int32_t *cs, int64_t nc_max,
                         const FwdSlot *slots_dev, int nslots, const GatherTabs &tabs,
                         char *ws_base, int chunks, uint32_t *claims, hipStream_t s) {
    // lanes per row: the next power of two >= chunks / chunks-per-lane, at least 4
    const int cpl = (int)cdiv(chunks, 64);
    const int need = (int)cdiv(chunks, cpl);
    int g = 4;
    while (g < need) g <<= 1;
#define RGCN_FLAT(G_, C_) \
    return launch_flat<B, G_, C_>(desc, cs, nc_max, slots_dev, nslots, tabs, ws_base, chunks, \
                                  claims, s)
    if (cpl == 1) {
        if (g == 4) RGCN_FLAT(4, 1);
        if (g == 8) RGCN_FLAT(8, 1);
        if (g == 16) RGCN_FLAT(16, 1);
        if (g == 32) RGCN_FLAT(32, 1);
        RGCN_FLAT(64, 1);
    }
    if (cpl == 2) RGCN_FLAT(64, 2);
    if (cpl <= 4) RGCN_FLAT(64, 4);
#undef RGCN_FLAT
    return hipErrorInvalidValue;
}

hipError_t gather_mean(rgcn_dtype dt, int d_in, const SegDesc *desc, int64_t n_seg,
                       const int32_t *chunk_starts, int64_t nc_max, const FwdSlot *slots_dev,
                       int nslots, const TypeInput *in, char *ws_base, uint32_t *claims,
                       hipStream_t s) {
    if (n_seg == 0) return hipSuccess;
    const bool bf = dt == RGCN_BF16;
    const int chunks = bf ? d_in / 8 : d_in / 4;
    GatherTabs tabs;
    for (int t = 0; t < kMaxTypes; ++t) tabs.in[t] = in[t];
    return bf ? flat_dispatch<true>(desc, chunk_starts, nc_max, slots_dev, nslots, tabs, ws_base,
                                    chunks, claims, s)
              : flat_dispatch<false>(desc, chunk_starts, nc_max, slots_dev, nslots, tabs, ws_base,
                                     chunks, claims, s);
}

template <bool B, int C, bool O, bool K>
hipError_t launch_transpose_pipe(const TsumArgs &a, const GroupShape &gs, int chunks,
                                 hipStream_t s) {
    const int64_t groups_per_wg = (int64_t)(kThreads / 64) * gs.gpw;
    int64_t wgs = cdiv(a.n_rows, groups_per_wg);
    auto kern = O ? k_transpose_pipe_adagrad<B, C> : k_transpose_pipe<B, C, K>;
    const int64_t cap = resident_wgs(kern);
    if (wgs > cap) wgs = cap;
    hipLaunchKernelGGL(kern, dim3((unsigned)wgs), dim3(kThreads), 0, s, a,
                       gs.G, gs.gpw, chunks);
    return hipGetLastError();
}

// The piece and finishing kernels of split rows: persistent grids that read the piece
// count on the device (no piece: every group exits at once).
template <bool B, int C, bool O, bool K>
hipError_t launch_split(const TsumArgs &a, const GroupShape &gs, int chunks, bool finish,
                        hipStream_t s) {
    if (a.piece_cap <= 0 || !a.pieces) return hipSuccess;
    const int64_t groups_per_wg = (int64_t)(kThreads / 64) * gs.gpw;
    int64_t wgs = cdiv(a.piece_cap, groups_per_wg);
    if (finish) {
        auto kern = k_transpose_split_finish<B, C, O, K>;
        const int64_t cap = resident_wgs(kern);
        hipLaunchKernelGGL(kern, dim3((unsigned)(wgs < cap ? wgs : cap)), dim3(kThreads), 0, s,
                           a, gs.G, gs.gpw, chunks);
    } else {
        auto kern = k_transpose_pieces<C>;
        const int64_t cap = resident_wgs(kern);
        hipLaunchKernelGGL(kern, dim3((unsigned)(wgs < cap ? wgs : cap)), dim3(kThreads), 0, s,
                           a, gs.G, gs.gpw, chunks);
    }
    return hipGetLastError();
}

template <bool B, int C, bool O, bool K>
hipError_t launch_transpose_rows(const TsumArgs &a, const GroupShape &gs, int chunks,
                                 hipStream_t s) {
    if (a.nrel <= gs.G) return launch_transpose_pipe<B, C, O, K>(a, gs, chunks, s);
    const int64_t waves = cdiv(a.n_rows, gs.gpw);
    const dim3 grid((unsigned)cdiv(waves, kThreads / 64));
    auto kern = O ? k_transpose_sum_adagrad<B, C> : k_transpose_sum<B, C, K>;
    hipLaunchKernelGGL(kern, grid, dim3(kThreads), 0, s, a, gs.G, gs.gpw,
                       chunks);
    return hipGetLastError();
}

template <bool B, int C, bool O, bool K>
hipError_t launch_transpose(const TsumArgs &a, const GroupShape &gs, int chunks, hipStream_t s) {
    // split rows: pieces first, then every other row, then the split rows' reductions
    RGCN_HIP_TRY((launch_split<B, C, O, K>(a, gs, chunks, false, s)));
    RGCN_HIP_TRY((launch_transpose_rows<B, C, O, K>(a, gs, chunks, s)));
    return launch_split<B, C, O, K>(a, gs, chunks, true, s);
}

template <bool B, bool O, bool K>
hipError_t launch_transpose_cpl(const TsumArgs &a, const GroupShape &gs, int chunks,
                                hipStream_t s) {
    if (gs.cpl == 1) return launch_transpose<B, 1, O, K>(a, gs, chunks, s);
    if (gs.cpl == 2) return launch_transpose<B, 2, O, K>(a, gs, chunks, s);
    if (gs.cpl <= 4) return launch_transpose<B, 4, O, K>(a, gs, chunks, s);
    return hipErrorInvalidValue;
}

// kernel forms: the block dtype (B), Adagrad (O), the input's ReLU signs read as bits (K;
// never with O: a learnable table is not a ReLU output).  The bit form reads no row
// before the sum, so an embedding gradient updated in place (unique ids) takes the form
// that reads the input rows instead.
template <bool B>
hipError_t transpose_sum_dt(const TsumArgs &a, const GroupShape &gs, int chunks, hipStream_t s) {
    if (a.opt_state != nullptr) return launch_transpose_cpl<B, true, false>(a, gs, chunks, s);
    if (a.input_relu && a.relu_mask != nullptr && !(a.demb != nullptr && a.ids_unique))
        return launch_transpose_cpl<B, false, true>(a, gs, chunks, s);
    return launch_transpose_cpl<B, false, false>(a, gs, chunks, s);
}

hipError_t transpose_sum(rgcn_dtype dt, const TsumArgs &a, hipStream_t s) {
    if (a.n_rows == 0) return hipSuccess;
    const int chunks = a.d_in / 4;
    const GroupShape gs = group_shape(chunks);
    return dt == RGCN_BF16 ? transpose_sum_dt<true>(a, gs, chunks, s)
                           : transpose_sum_dt<false>(a, gs, chunks, s);
}

hipError_t pack_weights(rgcn_dtype dt, int d_in, int d_out, const void *const *w_slots,
                        int nslots, void *wcat_t, hipStream_t s) {
    WSlots ws;
    for (int i = 0; i < kMaxSlots; ++i) ws.w[i] = i < nslots ? w_slots[i] : nullptr;
    const int64_t K = (int64_t)nslots * d_in;
    if (K == 0 || d_out == 0) return hipSuccess;
    const dim3 grid((unsigned)cdiv(K, kPackTile), (unsigned)cdiv(d_out, kPackTile));
    if (dt == RGCN_BF16)
        hipLaunchKernelGGL(k_pack_weights<uint16_t>, grid, dim3(kThreads), 0, s, ws, nslots, d_in,
                           d_out, (uint16_t *)wcat_t);
    else
        hipLaunchKernelGGL(k_pack_weights<float>, grid, dim3(kThreads), 0, s, ws, nslots, d_in,
                           d_out, (float *)wcat_t);
    return hipGetLastError();
}

static int64_t colsum_splits(int64_t rows) {
    int64_t sp = cdiv(rows, 2048);
    return sp < 1 ? 1 : (sp > 1024 ? 1024 : sp);
}
size_t column_sums_temp_bytes(int64_t rows, int cols) {
    return (size_t)colsum_splits(rows) * cols * 4 + 256;
}
hipError_t column_sums(const float *dy, bool hilo, int64_t rows, int cols, float *out,
                       float *partial, int64_t max_splits, hipStream_t s) {
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
                       dim3(kThreads), 0, s, dy, hilo ? 1 : 0, rows, cols, rps, partial);
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

// Per-edge table rows must be those the indices and row ids name (and inside the table).
__global__ __launch_bounds__(kThreads) void k_validate_src_rows(const int32_t *indices,
                                                                const int64_t *rows, int64_t nnz,
                                                                int64_t n_src, const int64_t *ids,
                                                                int64_t num_rows, uint32_t *err) {
    const int64_t k = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (k >= nnz) return;
    const int64_t j = indices[k], x = rows[k];
    if (j < 0 || j >= n_src) return;   // reported by the CSR check
    const int64_t want = ids ? ids[j] : j;
    if (x != want || x < 0 || x >= num_rows) atomicOr(err, 2u);
}
hipError_t validate_src_rows(const int32_t *indices, const int64_t *rows, int64_t nnz,
                             int64_t n_src, const int64_t *ids, int64_t num_rows, uint32_t *err,
                             hipStream_t s) {
    if (nnz == 0) return hipSuccess;
    hipLaunchKernelGGL(k_validate_src_rows, dim3((unsigned)cdiv(nnz, kThreads)), dim3(kThreads), 0,
                       s, indices, rows, nnz, n_src, ids, num_rows, err);
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
