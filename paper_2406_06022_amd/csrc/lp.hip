// Link-prediction decoder on the GNN's output embeddings (the paper's appendix on
// link-prediction score and loss functions): per positive edge (src_i, dst_i) and its
// negatives (per edge, joint, or in-batch), the dot-product or DistMult score
// s = sum_c h_src[c] r[c] h_other[c], the cross-entropy, weighted cross-entropy or
// contrastive loss averaged over the batch, and the gradients with respect to every
// embedding row used (added into a table-shaped fp32 buffer) and to r.
//
// Passes: (1) scores, one lane group per positive with u_i = h_src_i * r held in
// registers (u_i also stored for the later passes), negatives four at a time;
// (2) the loss per positive and the derivative of the loss with respect to each score;
// (3) a fixed-order sum of the per-positive losses; (4) per positive, the gradient of
// u_i (gpos h_dst + sum_k G_ik h_neg), scattered into the source row (times r) and, per
// edge, G_ik u_i into each negative row, plus gpos u_i into the destination row; the
// products dU_i * h_src_i for the gradient of r; (5) for shared negatives (joint,
// in-batch) the negative rows' gradients per column, sum_i G_ik u_i, one add per column;
// (6) the column sums that give the gradient of r.
#include "common.h"

namespace rgcn {

namespace {

constexpr int kThreads = 256;

__host__ __device__ inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

template <bool BF16>
struct Row {
    static constexpr int VEC = BF16 ? 8 : 4;   // elements per 16-byte chunk
};

// Chunk c of row `row` as floats.
template <bool BF16>
__device__ __forceinline__ void load_chunk(const LpArgs &a, int64_t row, int c, float *v) {
    const uint4 w = *(const uint4 *)((const char *)a.emb + (row * a.ld * (BF16 ? 2 : 4)) +
                                     (int64_t)c * 16);
    if constexpr (BF16) {
        v[0] = bf16_lo(w.x); v[1] = bf16_hi(w.x); v[2] = bf16_lo(w.y); v[3] = bf16_hi(w.y);
        v[4] = bf16_lo(w.z); v[5] = bf16_hi(w.z); v[6] = bf16_lo(w.w); v[7] = bf16_hi(w.w);
    } else {
        v[0] = __uint_as_float(w.x); v[1] = __uint_as_float(w.y);
        v[2] = __uint_as_float(w.z); v[3] = __uint_as_float(w.w);
    }
}

template <bool BF16>
__device__ __forceinline__ void load_rel(const LpArgs &a, int c, float *v) {
    constexpr int VEC = Row<BF16>::VEC;
    if (!a.rel) {
        for (int e = 0; e < VEC; ++e) v[e] = 1.f;
        return;
    }
    const uint4 w = *(const uint4 *)((const char *)a.rel + (int64_t)c * 16);
    if constexpr (BF16) {
        v[0] = bf16_lo(w.x); v[1] = bf16_hi(w.x); v[2] = bf16_lo(w.y); v[3] = bf16_hi(w.y);
        v[4] = bf16_lo(w.z); v[5] = bf16_hi(w.z); v[6] = bf16_lo(w.w); v[7] = bf16_hi(w.w);
    } else {
        v[0] = __uint_as_float(w.x); v[1] = __uint_as_float(w.y);
        v[2] = __uint_as_float(w.z); v[3] = __uint_as_float(w.w);
    }
}

// Sum over the G lanes of a group (G a power of two, groups aligned).
__device__ __forceinline__ float group_sum(float x, int G) {
    for (int o = G >> 1; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
    return x;
}

// Row of negative k of positive i.
__device__ __forceinline__ int64_t neg_row(const LpArgs &a, int64_t i, int64_t k) {
    if (a.neg_mode == RGCN_LP_NEG_PER_EDGE) return a.neg[i * a.k + k];
    if (a.neg_mode == RGCN_LP_NEG_JOINT) return a.neg[(i / a.k) * a.k + k];
    return a.dst[k < i ? k : k + 1];
}

// (1) scores and u_i.  One group of G lanes per positive; lane lg holds chunks
// lg + p G (p < CPL) of u_i.
template <bool BF16, int CPL>
__global__ __launch_bounds__(kThreads) void k_lp_scores(LpArgs a, int G, float *pos, float *S,
                                                        float *U, int loop_negs) {
    constexpr int VEC = Row<BF16>::VEC;
    const int lane = threadIdx.x & 63;
    const int lg = lane & (G - 1);
    const int64_t groups = (int64_t)gridDim.x * (kThreads / G);
    const int chunks = a.d / VEC;
    for (int64_t i = ((int64_t)blockIdx.x * kThreads + threadIdx.x) / G; i < a.batch; i += groups) {
        float u[CPL][VEC];
        const int64_t s = a.src[i];
#pragma unroll
        for (int p = 0; p < CPL; ++p) {
            const int c = lg + p * G;
            float h[VEC], r[VEC];
            if (c < chunks) {
                load_chunk<BF16>(a, s, c, h);
                load_rel<BF16>(a, c, r);
            } else {
                for (int e = 0; e < VEC; ++e) h[e] = r[e] = 0.f;
            }
            for (int e = 0; e < VEC; ++e) u[p][e] = h[e] * r[e];
            if (c < chunks)
                for (int e = 0; e < VEC; ++e) U[i * a.d + (int64_t)c * VEC + e] = u[p][e];
        }
        // positive
        {
            float acc = 0.f;
#pragma unroll
            for (int p = 0; p < CPL; ++p) {
                const int c = lg + p * G;
                if (c < chunks) {
                    float h[VEC];
                    load_chunk<BF16>(a, a.dst[i], c, h);
                    for (int e = 0; e < VEC; ++e) acc += u[p][e] * h[e];
                }
            }
            acc = group_sum(acc, G);
            if (lg == 0) pos[i] = acc;
        }
        for (int64_t k0 = 0; loop_negs && k0 < a.nn; k0 += 4) {
            float acc[4] = {0.f, 0.f, 0.f, 0.f};
            int64_t rows[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) rows[q] = k0 + q < a.nn ? neg_row(a, i, k0 + q) : a.src[i];
#pragma unroll
            for (int p = 0; p < CPL; ++p) {
                const int c = lg + p * G;
                if (c >= chunks) continue;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    float h[VEC];
                    load_chunk<BF16>(a, rows[q], c, h);
                    for (int e = 0; e < VEC; ++e) acc[q] += u[p][e] * h[e];
                }
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float t = group_sum(acc[q], G);
                if (lg == 0 && k0 + q < a.nn) S[i * a.nn + k0 + q] = t;
            }
        }
    }
}

__device__ __forceinline__ float softplus_f(float x) {   // log(1 + e^x)
    return x > 0.f ? x + log1pf(expf(-x)) : log1pf(expf(x));
}
__device__ __forceinline__ float sigmoid_f(float x) { return 1.f / (1.f + expf(-x)); }

// (2) loss per positive and d loss / d score: one wave per positive.
// In-batch scores are the full B x B product (row i: positive i, column j: destination
// j, the positive on the diagonal): negative k of row i is column k < i ? k : k + 1, and
// the derivative of the positive is written on the diagonal of G.
__device__ __forceinline__ int64_t loss_col(bool full, int64_t i, int64_t k) {
    return full ? (k < i ? k : k + 1) : k;
}

__global__ __launch_bounds__(kThreads) void k_lp_loss(LpArgs a, const float *pos, const float *S,
                                                      float *gpos, float *Gm, float *lossp) {
    const int lane = threadIdx.x & 63;
    const int64_t waves = (int64_t)gridDim.x * (kThreads / 64);
    const double n_edges = (double)a.batch * (double)(1 + a.nn);
    const bool full = a.neg_mode == RGCN_LP_NEG_IN_BATCH;
    const int64_t ld = full ? a.batch : a.nn;
    for (int64_t i = ((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6; i < a.batch; i += waves) {
        const float sp = pos[i];
        const float *Si = S + i * ld;
        float *Gi = Gm + i * ld;
        if (a.loss == RGCN_LP_CONTRASTIVE) {
            float m = sp;
            for (int64_t k = lane; k < a.nn; k += 64) m = fmaxf(m, Si[loss_col(full, i, k)]);
            for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
            float z = 0.f;
            for (int64_t k = lane; k < a.nn; k += 64) z += expf(Si[loss_col(full, i, k)] - m);
            for (int o = 32; o > 0; o >>= 1) z += __shfl_xor(z, o, 64);
            z += expf(sp - m);
            const float inv = 1.f / (z * (float)a.batch);
            for (int64_t k = lane; k < a.nn; k += 64) {
                const int64_t c = loss_col(full, i, k);
                Gi[c] = expf(Si[c] - m) * inv;
            }
            if (lane == 0) {
                gpos[i] = expf(sp - m) * inv - 1.f / (float)a.batch;
                if (full) Gi[i] = gpos[i];
                lossp[i] = (m + logf(z) - sp) / (float)a.batch;
            }
        } else {
            const float w = (a.loss == RGCN_LP_WEIGHTED_CE && a.pos_weight) ? a.pos_weight[i] : 1.f;
            const float inv = (float)(1.0 / n_edges);
            float l = 0.f;
            for (int64_t k = lane; k < a.nn; k += 64) {
                const int64_t c = loss_col(full, i, k);
                const float s = Si[c];
                l += softplus_f(s);
                Gi[c] = sigmoid_f(s) * inv;
            }
            for (int o = 32; o > 0; o >>= 1) l += __shfl_xor(l, o, 64);
            if (lane == 0) {
                gpos[i] = w * (sigmoid_f(sp) - 1.f) * inv;
                lossp[i] = (l + w * softplus_f(-sp)) * inv;
                if (full) Gi[i] = gpos[i];
            }
        }
    }
}

// (3) the batch loss: one workgroup, fixed order (deterministic).
__global__ __launch_bounds__(kThreads) void k_lp_sum(const float *lossp, int64_t n, float *out) {
    __shared__ float buf[kThreads];
    float acc = 0.f;
    for (int64_t i = threadIdx.x; i < n; i += kThreads) acc += lossp[i];
    buf[threadIdx.x] = acc;
    __syncthreads();
    for (int o = kThreads / 2; o > 0; o >>= 1) {
        if ((int)threadIdx.x < o) buf[threadIdx.x] += buf[threadIdx.x + o];
        __syncthreads();
    }
    if (threadIdx.x == 0) *out = buf[0];
}

// Shared negatives as dense products, per group of positives (joint: K positives and
// their K shared rows; in-batch: all B positives and the B destination rows):
//   S_g = U_g Hn_g^T,  dU_g = G_g Hn_g,  dHn_g = G_g^T U_g.
// A generic batched fp32 tile product C = A B^T over strided operands: 32 x 32 tiles, one
// wave each (a batch of 1,024 positives makes 1,024 tiles, four per CU), K steps of 16
// through LDS, fp32 MFMA.  Rows of A (or the reduction, for dHn) that lie past the batch
// in a group's last tile are left out.
constexpr int kLpTile = 32;
struct LpGemm {
    const float *A, *B;
    float *C;
    int64_t M, N, K;
    int64_t sam, sak, sbn, sbk, scm, scn;
    int64_t bsa, bsb, bsc;
    int64_t pos_total, pos_per_group;
    int32_t pos_dim;   // 0: M counts positives; 2: K counts positives; -1: neither
};

__global__ __launch_bounds__(64) void k_lp_gemm(LpGemm g) {
    const int64_t grp = blockIdx.z;
    int64_t M = g.M, K = g.K;
    if (g.pos_dim >= 0) {
        const int64_t rest = g.pos_total - grp * g.pos_per_group;
        const int64_t lim = rest < g.pos_per_group ? rest : g.pos_per_group;
        if (g.pos_dim == 0) M = lim; else K = lim;
    }
    const int64_t m0 = (int64_t)blockIdx.y * kLpTile, n0 = (int64_t)blockIdx.x * kLpTile;
    if (m0 >= M) return;   // the whole workgroup leaves together
    const float *A = g.A + grp * g.bsa;
    const float *B = g.B + grp * g.bsb;
    float *C = g.C + grp * g.bsc;
    __shared__ float As[16][kLpTile + 1], Bs[16][kLpTile + 1];
    // one wave per 32 x 32 tile on fp32 MFMA tiles of 32 x 32 x 2: lane l supplies row
    // l % 32 of the A slice and column l % 32 of the B slice at k = l / 32, and holds
    // column l % 32, rows 8 (e / 4) + 4 (l / 32) + e % 4 of the result.  The next K step's
    // operands are loaded into registers while the current one is multiplied.
    const int lane = threadIdx.x, l32 = lane & 31, kh = lane >> 5;
    float ra[8], rb[8];
    auto load = [&](int64_t k0) {
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int idx = lane + q * 64;
            const int r = idx >> 4, kk = idx & 15;
            const int64_t m = m0 + r, n = n0 + r, k = k0 + kk;
            ra[q] = (m < M && k < K) ? A[m * g.sam + k * g.sak] : 0.f;
            rb[q] = (n < g.N && k < K) ? B[n * g.sbn + k * g.sbk] : 0.f;
        }
    };
    f32x16 acc;
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[e] = 0.f;
    load(0);
    for (int64_t k0 = 0; k0 < K; k0 += 16) {
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int idx = lane + q * 64;
            As[idx & 15][idx >> 4] = ra[q];
            Bs[idx & 15][idx >> 4] = rb[q];
        }
        __syncthreads();
        if (k0 + 16 < K) load(k0 + 16);
#pragma unroll
        for (int kp = 0; kp < 8; ++kp)
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(As[2 * kp + kh][l32], Bs[2 * kp + kh][l32],
                                                       acc, 0, 0, 0);
        __syncthreads();
    }
    const int64_t n = n0 + l32;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
        const int64_t m = m0 + 8 * (e / 4) + 4 * kh + (e % 4);
        if (m < M && n < g.N) C[m * g.scm + n * g.scn] = acc[e];
    }
}

// Row of shared-negative column c: joint neg[c], in-batch dst[c].
__device__ __forceinline__ int64_t col_row(const LpArgs &a, int64_t c) {
    return a.neg_mode == RGCN_LP_NEG_JOINT ? a.neg[c] : a.dst[c];
}

// Hn[c] = emb[col_row(c)] in fp32.
template <bool BF16>
__global__ __launch_bounds__(kThreads) void k_lp_gather(LpArgs a, int64_t ncols, float *Hn) {
    const int64_t total = ncols * a.d;
    for (int64_t t = (int64_t)blockIdx.x * kThreads + threadIdx.x; t < total;
         t += (int64_t)gridDim.x * kThreads) {
        const int64_t c = t / a.d, e = t - c * a.d;
        const int64_t row = col_row(a, c);
        if constexpr (BF16) {
            const uint16_t v = ((const uint16_t *)a.emb)[row * a.ld + e];
            Hn[t] = __uint_as_float((uint32_t)v << 16);
        } else {
            Hn[t] = ((const float *)a.emb)[row * a.ld + e];
        }
    }
}

// d_emb[col_row(c)] += dHn[c], consecutive lanes on consecutive elements.
__global__ __launch_bounds__(kThreads) void k_lp_scatter_cols(LpArgs a, int64_t ncols,
                                                              const float *dHn, float *d_emb) {
    const int64_t total = ncols * a.d;
    for (int64_t t = (int64_t)blockIdx.x * kThreads + threadIdx.x; t < total;
         t += (int64_t)gridDim.x * kThreads) {
        const int64_t c = t / a.d, e = t - c * a.d;
        unsafeAtomicAdd(d_emb + col_row(a, c) * a.d + e, dHn[t]);
    }
}

template <bool BF16>
__device__ __forceinline__ float elem(const LpArgs &a, int64_t row, int64_t e) {
    if constexpr (BF16)
        return __uint_as_float((uint32_t)((const uint16_t *)a.emb)[row * a.ld + e] << 16);
    else
        return ((const float *)a.emb)[row * a.ld + e];
}
template <bool BF16>
__device__ __forceinline__ float rel_elem(const LpArgs &a, int64_t e) {
    if (!a.rel) return 1.f;
    if constexpr (BF16)
        return __uint_as_float((uint32_t)((const uint16_t *)a.rel)[e] << 16);
    else
        return ((const float *)a.rel)[e];
}

// (4) one wave per positive, element e = lane + 64 j: the gradient of u_i,
//   du = [dense] dU_i + [not in-batch] gpos h_dst + [per edge] sum_k G_ik h_neg_k,
// added into the source row (times r); gpos u into the destination row (not in-batch:
// there the diagonal of the products carries it); per edge, G_ik u into each negative
// row; P_i = du * h_src for the gradient of r.  Atomics of a wave cover 64 consecutive
// floats.
template <bool BF16, int J>
__global__ __launch_bounds__(kThreads) void k_lp_finish(LpArgs a, const float *gpos, const float *Gm,
                                                        const float *U, const float *dU,
                                                        float *d_emb, float *P) {
    const int lane = threadIdx.x & 63;
    const int64_t waves = (int64_t)gridDim.x * (kThreads / 64);
    const bool per_edge = a.neg_mode == RGCN_LP_NEG_PER_EDGE;
    const bool inbatch = a.neg_mode == RGCN_LP_NEG_IN_BATCH;
    for (int64_t i = ((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6; i < a.batch; i += waves) {
        float u[J], du[J];
        const float gp = gpos[i];
        const int64_t sr = a.src[i], dr = a.dst[i];
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const int64_t e = lane + 64 * j;
            u[j] = e < a.d ? U[i * a.d + e] : 0.f;
            du[j] = 0.f;
            if (e < a.d) {
                if (dU) du[j] = dU[i * a.d + e];
                if (!inbatch) du[j] += gp * elem<BF16>(a, dr, e);
            }
        }
        if (!inbatch && d_emb)
#pragma unroll
            for (int j = 0; j < J; ++j) {
                const int64_t e = lane + 64 * j;
                if (e < a.d) unsafeAtomicAdd(d_emb + dr * a.d + e, gp * u[j]);
            }
        if (per_edge) {
            // Per chunk of 64 negatives, lane l loads negative l's row and weight once (the
            // loop broadcasts them); each negative's embedding row is loaded one negative
            // ahead, and one word of every 128-byte line of its gradient row two ahead, so
            // the atomics find the lines in L2 (the value read is not used).
            const int64_t lo_off = (int64_t)lane * 32;   // lane's line of a gradient row
            for (int64_t k0 = 0; k0 < a.nn; k0 += 64) {
                const int kn = a.nn - k0 < 64 ? (int)(a.nn - k0) : 64;
                const bool okl = lane < kn;
                const int32_t nrow_l = okl ? a.neg[i * a.k + k0 + lane] : 0;
                const float g_l = okl ? Gm[i * a.nn + k0 + lane] : 0.f;
                auto load_row = [&](int kk, float (&v)[J]) {
                    const int64_t row = __shfl(nrow_l, kk, 64);
#pragma unroll
                    for (int j = 0; j < J; ++j) {
                        const int64_t e = lane + 64 * j;
                        v[j] = e < a.d ? elem<BF16>(a, row, e) : 0.f;
                    }
                };
                auto touch = [&](int kk) -> float {
                    const int64_t row = __shfl(nrow_l, kk, 64);
                    return (d_emb && lo_off < a.d) ? d_emb[row * a.d + lo_off] : 0.f;
                };
                float nx[J];
                load_row(0, nx);
                float t0 = touch(0), t1 = kn > 1 ? touch(1) : 0.f;
                for (int kk = 0; kk < kn; ++kk) {
                    float cur[J];
#pragma unroll
                    for (int j = 0; j < J; ++j) cur[j] = nx[j];
                    if (kk + 1 < kn) load_row(kk + 1, nx);
                    const float t2 = kk + 2 < kn ? touch(kk + 2) : 0.f;
                    asm volatile("" ::"v"(t0));   // this negative's lines have been fetched
                    const int64_t row = __shfl(nrow_l, kk, 64);
                    const float g = __shfl(g_l, kk, 64);
#pragma unroll
                    for (int j = 0; j < J; ++j) {
                        const int64_t e = lane + 64 * j;
                        if (e < a.d) {
                            du[j] += g * cur[j];
                            if (d_emb) unsafeAtomicAdd(d_emb + row * a.d + e, g * u[j]);
                        }
                    }
                    t0 = t1;
                    t1 = t2;
                }
            }
        }
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const int64_t e = lane + 64 * j;
            if (e >= a.d) continue;
            if (d_emb) unsafeAtomicAdd(d_emb + sr * a.d + e, du[j] * rel_elem<BF16>(a, e));
            if (P) P[i * a.d + e] = du[j] * elem<BF16>(a, sr, e);
        }
    }
}

// (6) d_rel = sum_i P_i: a workgroup takes 64 columns of a slice of rows with 4 row
// lanes per column (coalesced 256-byte rows), the lanes combined in LDS; then the slices
// of each column in order.
constexpr int kRelCols = 64, kRelLanes = kThreads / kRelCols;
__global__ __launch_bounds__(kThreads) void k_lp_rel_partial(const float *P, int64_t rows, int d,
                                                             int64_t per, float *part) {
    __shared__ float buf[kRelLanes][kRelCols];
    const int c = threadIdx.x % kRelCols, rl = threadIdx.x / kRelCols;
    const int64_t e = (int64_t)blockIdx.x * kRelCols + c;
    const int64_t r0 = (int64_t)blockIdx.y * per;
    const int64_t r1 = r0 + per < rows ? r0 + per : rows;
    float acc = 0.f;
    if (e < d)
        for (int64_t r = r0 + rl; r < r1; r += kRelLanes) acc += P[r * d + e];
    buf[rl][c] = acc;
    __syncthreads();
    if (rl == 0 && e < d) {
        float t = 0.f;
        for (int q = 0; q < kRelLanes; ++q) t += buf[q][c];
        part[(int64_t)blockIdx.y * d + e] = t;
    }
}
__global__ __launch_bounds__(kThreads) void k_lp_rel_final(const float *part, int64_t nparts, int d,
                                                           float *out) {
    const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (e >= d) return;
    float acc = 0.f;
    for (int64_t p = 0; p < nparts; ++p) acc += part[p * d + e];
    out[e] = acc;
}

// Row slices of the d_rel reduction: 64 rows each, at most 256 slices.
int64_t rel_parts(int64_t rows) {
    int64_t p = cdiv(rows, 64);
    return p < 1 ? 1 : (p > 256 ? 256 : p);
}

// neg_score[i][k] = S[i][k < i ? k : k + 1] for the in-batch product.
__global__ __launch_bounds__(kThreads) void k_lp_offdiag(const float *S, int64_t B, float *out) {
    const int64_t total = B * (B - 1);
    for (int64_t t = (int64_t)blockIdx.x * kThreads + threadIdx.x; t < total;
         t += (int64_t)gridDim.x * kThreads) {
        const int64_t i = t / (B - 1), k = t - i * (B - 1);
        out[t] = S[i * B + (k < i ? k : k + 1)];
    }
}


__global__ __launch_bounds__(kThreads) void k_lp_validate(LpArgs a, uint32_t *err) {
    const int64_t nneg = a.neg_mode == RGCN_LP_NEG_PER_EDGE ? a.batch * a.k
                       : a.neg_mode == RGCN_LP_NEG_JOINT ? cdiv(a.batch, a.k) * a.k : 0;
    const int64_t n = a.batch > nneg ? a.batch : nneg;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * kThreads) {
        bool bad = false;
        if (i < a.batch) bad |= a.src[i] < 0 || a.src[i] >= a.n_rows || a.dst[i] < 0 ||
                                a.dst[i] >= a.n_rows;
        if (i < nneg) bad |= a.neg[i] < 0 || a.neg[i] >= a.n_rows;
        if (bad) atomicOr(err, 1u);
    }
}

// Negative ids: slot q takes the high word of draw * num_nodes, the draw being word
// q mod 4 of Philox4x64-10 at counter (q / 4, mode, 0, 0), key (seed, 0x6e6567).
__global__ __launch_bounds__(kThreads) void k_lp_negatives(int32_t mode, int64_t slots,
                                                           uint64_t num_nodes, uint64_t seed,
                                                           int64_t *out) {
    for (int64_t q = (int64_t)blockIdx.x * kThreads + threadIdx.x; q < slots;
         q += (int64_t)gridDim.x * kThreads) {
        uint64_t w[4] = {(uint64_t)q >> 2, (uint64_t)(uint32_t)mode, 0, 0};
        philox4x64(w, seed, 0x6e6567ull);
        out[q] = (int64_t)__umul64hi(w[q & 3], num_nodes);
    }
}

int64_t grid_for(int64_t items, int per_wg) {
    int64_t g = cdiv(items, per_wg);
    if (g < 1) g = 1;
    return g > 4096 ? 4096 : g;
}

template <bool BF16, int CPL>
hipError_t run_scores(const LpArgs &a, int G, float *pos, float *S, float *U, int loop_negs,
                      hipStream_t s) {
    hipLaunchKernelGGL((k_lp_scores<BF16, CPL>), dim3((unsigned)grid_for(a.batch, kThreads / G)),
                       dim3(kThreads), 0, s, a, G, pos, S, U, loop_negs);
    return hipGetLastError();
}

template <bool BF16>
hipError_t dispatch_scores(const LpArgs &a, float *pos, float *S, float *U, int loop_negs,
                           hipStream_t s) {
    const int chunks = a.d / Row<BF16>::VEC;
    int G = 1;
    while (G < chunks && G < 64) G *= 2;
    const int cpl = (int)cdiv(chunks, G);
    if (cpl == 1) return run_scores<BF16, 1>(a, G, pos, S, U, loop_negs, s);
    if (cpl == 2) return run_scores<BF16, 2>(a, G, pos, S, U, loop_negs, s);
    if (cpl <= 4) return run_scores<BF16, 4>(a, G, pos, S, U, loop_negs, s);
    return hipErrorInvalidValue;
}

template <bool BF16>
hipError_t dispatch_finish(const LpArgs &a, const float *gpos, const float *Gm, const float *U,
                           const float *dU, float *d_emb, float *P, hipStream_t s) {
    const dim3 grid((unsigned)grid_for(a.batch, kThreads / 64)), block(kThreads);
    const int J = (int)cdiv(a.d, 64);
#define RGCN_FIN(JJ) \
    hipLaunchKernelGGL((k_lp_finish<BF16, JJ>), grid, block, 0, s, a, gpos, Gm, U, dU, d_emb, P)
    if (J <= 1) RGCN_FIN(1);
    else if (J <= 2) RGCN_FIN(2);
    else if (J <= 4) RGCN_FIN(4);
    else if (J <= 8) RGCN_FIN(8);
    else if (J <= 16) RGCN_FIN(16);
    else if (J <= 32) RGCN_FIN(32);
    else return hipErrorInvalidValue;
#undef RGCN_FIN
    return hipGetLastError();
}

hipError_t gemm(const LpGemm &g, int64_t groups, hipStream_t s) {
    if (groups == 0 || g.M == 0 || g.N == 0) return hipSuccess;
    hipLaunchKernelGGL(k_lp_gemm, dim3((unsigned)cdiv(g.N, kLpTile), (unsigned)cdiv(g.M, kLpTile),
                                       (unsigned)groups), dim3(64), 0, s, g);
    return hipGetLastError();
}

// Shared-negative layout: groups, positives per group (M), columns per group (N).
void dense_shape(const LpArgs &a, int64_t &groups, int64_t &M, int64_t &N) {
    if (a.neg_mode == RGCN_LP_NEG_JOINT) {
        groups = cdiv(a.batch, a.k);
        M = a.k;
        N = a.k;
    } else {
        groups = 1;
        M = a.batch;
        N = a.batch;
    }
}

}  // namespace

LpLayout lp_layout(const LpArgs &a) {
    auto al = [](size_t x) { return (x + 255) / 256 * 256; };
    LpLayout L;
    size_t o = 0;
    const bool dense = a.neg_mode != RGCN_LP_NEG_PER_EDGE;
    // scores and their derivatives: per edge and joint [B x K]; in-batch the full [B x B]
    const size_t bn = (size_t)a.batch * (size_t)(a.neg_mode == RGCN_LP_NEG_IN_BATCH ? a.batch : a.nn);
    int64_t groups = 0, M = 0, N = 0;
    if (dense) dense_shape(a, groups, M, N);
    const size_t ncols = (size_t)(groups * N);
    const size_t bd = (size_t)a.batch * a.d;
    L.off_pos = o; o += al((size_t)a.batch * 4 + 4);
    L.off_gpos = o; o += al((size_t)a.batch * 4 + 4);
    L.off_lossp = o; o += al((size_t)a.batch * 4 + 4);
    L.off_S = o; o += al(bn * 4 + 4);
    L.off_G = o; o += al(bn * 4 + 4);
    L.off_U = o; o += al(bd * 4 + 4);
    L.off_P = o; o += al(bd * 4 + 4);
    L.off_dU = o; o += dense ? al(bd * 4 + 4) : 0;
    L.off_Hn = o; o += dense ? al(ncols * a.d * 4 + 4) : 0;
    L.off_dHn = o; o += dense ? al(ncols * a.d * 4 + 4) : 0;
    L.off_colsum = o; o += al((size_t)rel_parts(a.batch) * a.d * 4 + 4);
    L.off_err = o; o += 256;
    L.total = o;
    return L;
}

hipError_t lp_loss(const LpArgs &a, const LpLayout &L, char *ws, float *loss, float *pos_score,
                   float *neg_score, float *d_emb, float *d_rel, hipStream_t s) {
    const bool bf = a.dtype == RGCN_BF16;
    const bool dense = a.neg_mode != RGCN_LP_NEG_PER_EDGE;
    const bool inbatch = a.neg_mode == RGCN_LP_NEG_IN_BATCH;
    float *pos = pos_score ? pos_score : (float *)(ws + L.off_pos);
    // per edge and joint write the caller's neg_score directly; in-batch keeps the full
    // product in the workspace and copies the off-diagonal entries out at the end
    float *S = (neg_score && !inbatch) ? neg_score : (float *)(ws + L.off_S);
    float *gpos = (float *)(ws + L.off_gpos);
    float *lossp = (float *)(ws + L.off_lossp);
    float *Gm = (float *)(ws + L.off_G);
    float *U = (float *)(ws + L.off_U);
    float *P = d_rel ? (float *)(ws + L.off_P) : nullptr;
    float *dU = dense ? (float *)(ws + L.off_dU) : nullptr;
    float *Hn = (float *)(ws + L.off_Hn);
    float *dHn = (float *)(ws + L.off_dHn);
    if (a.batch == 0) {
        const uint32_t zero = 0;
        RGCN_HIP_TRY(fill_words(loss, &zero, 4, s));
        if (d_rel) RGCN_HIP_TRY(column_sums(nullptr, false, 0, a.d, d_rel, nullptr, 0, s));
        return hipSuccess;
    }
    // (1) scores: u_i and the positives; per edge also the negatives
    RGCN_HIP_TRY(bf ? dispatch_scores<true>(a, pos, S, U, dense ? 0 : 1, s)
                    : dispatch_scores<false>(a, pos, S, U, dense ? 0 : 1, s));
    int64_t groups = 0, M = 0, N = 0;
    if (dense) {
        dense_shape(a, groups, M, N);
        const int64_t ncols = groups * N;
        if (bf)
            hipLaunchKernelGGL(k_lp_gather<true>, dim3((unsigned)grid_for(ncols * a.d, kThreads)),
                               dim3(kThreads), 0, s, a, ncols, Hn);
        else
            hipLaunchKernelGGL(k_lp_gather<false>, dim3((unsigned)grid_for(ncols * a.d, kThreads)),
                               dim3(kThreads), 0, s, a, ncols, Hn);
        RGCN_HIP_TRY(hipGetLastError());
        // S_g = U_g Hn_g^T  (rows: positives of the group; row stride N)
        LpGemm g{};
        g.A = U; g.B = Hn; g.C = S;
        g.M = M; g.N = N; g.K = a.d;
        g.sam = a.d; g.sak = 1; g.sbn = a.d; g.sbk = 1; g.scm = N; g.scn = 1;
        g.bsa = M * a.d; g.bsb = N * a.d; g.bsc = M * N;
        g.pos_total = a.batch; g.pos_per_group = M; g.pos_dim = 0;
        RGCN_HIP_TRY(gemm(g, groups, s));
    }
    // (2), (3) loss
    hipLaunchKernelGGL(k_lp_loss, dim3((unsigned)grid_for(a.batch, kThreads / 64)), dim3(kThreads),
                       0, s, a, pos, S, gpos, Gm, lossp);
    RGCN_HIP_TRY(hipGetLastError());
    hipLaunchKernelGGL(k_lp_sum, dim3(1), dim3(kThreads), 0, s, lossp, a.batch, loss);
    RGCN_HIP_TRY(hipGetLastError());
    if (d_emb || d_rel) {
        if (dense) {
            // dU_g = G_g Hn_g: C[m][e] = sum_n G[m][n] Hn[n][e]
            LpGemm g{};
            g.A = Gm; g.B = Hn; g.C = dU;
            g.M = M; g.N = a.d; g.K = N;
            g.sam = N; g.sak = 1; g.sbn = 1; g.sbk = a.d; g.scm = a.d; g.scn = 1;
            g.bsa = M * N; g.bsb = N * a.d; g.bsc = M * a.d;
            g.pos_total = a.batch; g.pos_per_group = M; g.pos_dim = 0;
            RGCN_HIP_TRY(gemm(g, groups, s));
            if (d_emb) {
                // dHn_g = G_g^T U_g: C[n][e] = sum_m G[m][n] U[m][e] (m: positives)
                LpGemm h{};
                h.A = Gm; h.B = U; h.C = dHn;
                h.M = N; h.N = a.d; h.K = M;
                h.sam = 1; h.sak = N; h.sbn = 1; h.sbk = a.d; h.scm = a.d; h.scn = 1;
                h.bsa = M * N; h.bsb = M * a.d; h.bsc = N * a.d;
                h.pos_total = a.batch; h.pos_per_group = M; h.pos_dim = 2;
                RGCN_HIP_TRY(gemm(h, groups, s));
                const int64_t ncols = groups * N;
                hipLaunchKernelGGL(k_lp_scatter_cols, dim3((unsigned)grid_for(ncols * a.d, kThreads)),
                                   dim3(kThreads), 0, s, a, ncols, dHn, d_emb);
                RGCN_HIP_TRY(hipGetLastError());
            }
        }
        RGCN_HIP_TRY(bf ? dispatch_finish<true>(a, gpos, Gm, U, dU, d_emb, P, s)
                        : dispatch_finish<false>(a, gpos, Gm, U, dU, d_emb, P, s));
        if (d_rel) {
            const int64_t parts = rel_parts(a.batch);
            const int64_t per = cdiv(a.batch, parts);
            float *part = (float *)(ws + L.off_colsum);
            hipLaunchKernelGGL(k_lp_rel_partial, dim3((unsigned)cdiv(a.d, kRelCols), (unsigned)parts),
                               dim3(kThreads), 0, s, P, a.batch, a.d, per, part);
            RGCN_HIP_TRY(hipGetLastError());
            hipLaunchKernelGGL(k_lp_rel_final, dim3((unsigned)cdiv(a.d, kThreads)), dim3(kThreads), 0,
                               s, part, parts, a.d, d_rel);
            RGCN_HIP_TRY(hipGetLastError());
        }
    }
    if (neg_score && inbatch) {
        hipLaunchKernelGGL(k_lp_offdiag, dim3((unsigned)grid_for(a.batch * a.nn, kThreads)),
                           dim3(kThreads), 0, s, S, a.batch, neg_score);
        RGCN_HIP_TRY(hipGetLastError());
    }
    return hipSuccess;
}

hipError_t lp_validate(const LpArgs &a, uint32_t *err, hipStream_t s) {
    const int64_t n = a.batch * (a.k > 1 ? a.k : 1) + a.batch;
    hipLaunchKernelGGL(k_lp_validate, dim3((unsigned)grid_for(n, kThreads)), dim3(kThreads), 0, s,
                       a, err);
    return hipGetLastError();
}

hipError_t lp_negatives(int32_t neg_mode, int64_t slots, int64_t num_nodes, uint64_t seed,
                        int64_t *out, hipStream_t s) {
    if (slots == 0) return hipSuccess;
    hipLaunchKernelGGL(k_lp_negatives, dim3((unsigned)grid_for(slots, kThreads)), dim3(kThreads),
                       0, s, neg_mode, slots, (uint64_t)num_nodes, seed, out);
    return hipGetLastError();
}

}  // namespace rgcn
