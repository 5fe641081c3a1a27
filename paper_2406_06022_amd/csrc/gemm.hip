// Dense transforms of the block on the CDNA4 matrix cores.
//
// One kernel body serves three products, differing only in how tiles reach LDS and how
// results leave:
//   forward      Y_t   = Mcat_t  [n_dst x K]      . WcatT_t^T  (+ bias, opt. ReLU)
//                K = (1 + R_t) * d_in: the self-loop and every relation into t are one
//                K-concatenated product, so the sum over relations is the K reduction.
//   input side   dMs_t = dY_t [n_dst x d_out]    . [W_s rows]^T, slot columns / deg
//   weight side  dW    = Mcat_t^T [K x n_dst]    . dY_t [n_dst x d_out]   (split over rows)
//
// Workgroup tile 128 x 128, four waves in a 2 x 2 arrangement of 64 x 64, each wave a 4 x 4
// grid of 16 x 16 MFMA tiles.  LDS holds both operands K-contiguous ("row r, k..."), one
// row = 64 bytes of K (32 bf16 or 16 fp32) + 16 bytes of padding, so the 16 rows read by a
// 16-lane group for an MFMA operand fall in distinct bank groups.  Double-buffered:
// global loads of step k+1 are in flight while step k is multiplied.
//
// bf16 mode: v_mfma_f32_16x16x32_bf16, fp32 accumulation.  The fp32 output gradient dY
// enters the weight-side product rounded to bf16 (nearest-even) and the input-side
// product as a hi + lo pair of bf16 values.  fp32 mode: v_mfma_f32_16x16x4_f32 (full fp32).
#include "common.h"

namespace rgcn {
namespace {

constexpr int kThreads = 256;
constexpr int kTile = 128;
constexpr int kPitch = 80;                        // LDS bytes per operand row
constexpr int kTileBytes = kTile * kPitch;        // 10240
constexpr int kStagePitch = 68;                   // epilogue staging row (floats)
__host__ __device__ inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// ------------------------------------------------------------------ MFMA cores
struct MmaBf16 {
    static constexpr int BK = 32;
    __device__ static void run(const char *As, const char *Bs, f32x4 (&acc)[4][4], int wm,
                               int wn, int lane) {
        bf16x8 a[4], b[4];
        const int r = lane & 15, q = lane >> 4;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            a[i] = *(const bf16x8 *)(As + (wm * 64 + i * 16 + r) * kPitch + q * 16);
            b[i] = *(const bf16x8 *)(Bs + (wn * 64 + i * 16 + r) * kPitch + q * 16);
        }
#pragma unroll
        for (int mi = 0; mi < 4; ++mi)
#pragma unroll
            for (int ni = 0; ni < 4; ++ni)
                acc[mi][ni] =
                    __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[mi], b[ni], acc[mi][ni], 0, 0, 0);
    }
};

// fp32: lane group q holds k = 4q..4q+3 of its row; MFMA step s uses element s, so the
// four steps together cover k = 0..15 (the sum over k is taken in a different order, not
// a different set).
struct MmaF32 {
    static constexpr int BK = 16;
    __device__ static void run(const char *As, const char *Bs, f32x4 (&acc)[4][4], int wm,
                               int wn, int lane) {
        f32x4 a[4], b[4];
        const int r = lane & 15, q = lane >> 4;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            a[i] = *(const f32x4 *)(As + (wm * 64 + i * 16 + r) * kPitch + q * 16);
            b[i] = *(const f32x4 *)(Bs + (wn * 64 + i * 16 + r) * kPitch + q * 16);
        }
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int mi = 0; mi < 4; ++mi)
#pragma unroll
                for (int ni = 0; ni < 4; ++ni)
                    acc[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[mi][s], b[ni][s],
                                                                       acc[mi][ni], 0, 0, 0);
    }
};

// ------------------------------------------------------------------ tile loaders
// K-contiguous rows, element type equal to the LDS type.  Each thread moves 2 of the 512
// 16-byte chunks of a 128-row x 64-byte tile.  Row addresses come from a policy.
struct PlainRows {
    const char *base;
    int64_t ld_bytes;
    int64_t rows;
    __device__ const char *row(int64_t r) const { return r < rows ? base + r * ld_bytes : nullptr; }
};
struct SlotRows {  // row n = (slot n / d_in, column c = n % d_in) of W_slot [d_in x d_out]
    const void *w[kMaxSlots];
    int32_t d_in;
    int32_t es_dout;   // bytes per W row (d_out * element size)
    int64_t rows;
    __device__ const char *row(int64_t r) const {
        if (r >= rows) return nullptr;
        const int64_t sl = r / d_in, c = r - sl * d_in;
        return (const char *)w[sl] + c * es_dout;
    }
};

template <class RowPolicy, bool WRAP = false>
struct LoadRows {
    RowPolicy pol;
    int64_t kbytes;     // bytes of K per row
    int es;             // element size
    int64_t wrap_bytes; // WRAP: the product's K is twice the row; k >= row length re-reads it
    const char *rp[2];
    int lr[2], lq[2];
    uint4 reg[2];
    __device__ void init(int64_t row0) {
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            const int chunk = threadIdx.x + c * kThreads;
            lr[c] = chunk >> 2;
            lq[c] = chunk & 3;
            rp[c] = pol.row(row0 + lr[c]);
        }
    }
    __device__ void load(int64_t k0) {
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            int64_t kb = k0 * es + lq[c] * 16;
            if constexpr (WRAP) {
                if (kb >= wrap_bytes) kb -= wrap_bytes;
            }
            reg[c] = (rp[c] && kb < kbytes) ? *(const uint4 *)(rp[c] + kb) : make_uint4(0, 0, 0, 0);
        }
    }
    __device__ void store(char *lds) const {
#pragma unroll
        for (int c = 0; c < 2; ++c) *(uint4 *)(lds + lr[c] * kPitch + lq[c] * 16) = reg[c];
    }
};

// K-contiguous fp32 rows rounded to bf16 (bf16 mode): a 16-byte LDS chunk = 8 values =
// 32 source bytes.
struct LoadRowsF32ToBf16 {
    PlainRows pol;
    int64_t K;
    const char *rp[2];
    int lr[2], lq[2];
    float4 reg[2][2];
    __device__ void init(int64_t row0) {
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            const int chunk = threadIdx.x + c * kThreads;
            lr[c] = chunk >> 2;
            lq[c] = chunk & 3;
            rp[c] = pol.row(row0 + lr[c]);
        }
    }
    __device__ void load(int64_t k0) {
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            const int64_t k = k0 + lq[c] * 8;
            if (rp[c] && k < K) {
                reg[c][0] = *(const float4 *)(rp[c] + k * 4);
                reg[c][1] = *(const float4 *)(rp[c] + k * 4 + 16);
            } else {
                reg[c][0] = reg[c][1] = make_float4(0.f, 0.f, 0.f, 0.f);
            }
        }
    }
    __device__ void store(char *lds) const {
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            uint4 w;
            w.x = pack_bf16x2(reg[c][0].x, reg[c][0].y);
            w.y = pack_bf16x2(reg[c][0].z, reg[c][0].w);
            w.z = pack_bf16x2(reg[c][1].x, reg[c][1].y);
            w.w = pack_bf16x2(reg[c][1].z, reg[c][1].w);
            *(uint4 *)(lds + lr[c] * kPitch + lq[c] * 16) = w;
        }
    }
};

// fp32 rows entering a bf16 product as two bf16 terms: for k < K the high part
// hi = bf16(x), for K <= k < 2K the low part lo = bf16(x - hi) of element k - K.  With
// the other operand repeated along K (LoadRows<..., true>), the product accumulates
// hi.W + lo.W, which carries x to ~16 significant bits instead of 8.
struct LoadRowsF32Split {
    PlainRows pol;
    int64_t K;
    const char *rp[2];
    int lr[2], lq[2];
    float4 reg[2][2];
    bool low;
    __device__ void init(int64_t row0) {
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            const int chunk = threadIdx.x + c * kThreads;
            lr[c] = chunk >> 2;
            lq[c] = chunk & 3;
            rp[c] = pol.row(row0 + lr[c]);
        }
    }
    __device__ void load(int64_t k0) {
        low = k0 >= K;
        const int64_t kbase = low ? k0 - K : k0;
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            const int64_t k = kbase + lq[c] * 8;
            if (rp[c] && k < K) {
                reg[c][0] = *(const float4 *)(rp[c] + k * 4);
                reg[c][1] = *(const float4 *)(rp[c] + k * 4 + 16);
            } else {
                reg[c][0] = reg[c][1] = make_float4(0.f, 0.f, 0.f, 0.f);
            }
        }
    }
    __device__ static float part(float x, bool low) {
        const float hi = __uint_as_float(f32_to_bf16_bits(x) << 16);
        return low ? x - hi : x;
    }
    __device__ void store(char *lds) const {
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            uint4 w;
            w.x = pack_bf16x2(part(reg[c][0].x, low), part(reg[c][0].y, low));
            w.y = pack_bf16x2(part(reg[c][0].z, low), part(reg[c][0].w, low));
            w.z = pack_bf16x2(part(reg[c][1].x, low), part(reg[c][1].y, low));
            w.w = pack_bf16x2(part(reg[c][1].z, low), part(reg[c][1].w, low));
            *(uint4 *)(lds + lr[c] * kPitch + lq[c] * 16) = w;
        }
    }
};

// Transposed operand for the weight-side product: source [Ksrc rows x C cols] row-major;
// LDS row = source column (128 of them from col0), LDS k = source row.  Global reads are
// row-contiguous; the transpose happens in the LDS writes.
//   SRC_BF16 && LDS bf16:  32 k x 16 chunks of 8 columns, 2 chunks per thread
//   SRC_F32  && LDS f32:   16 k x 32 chunks of 4 columns, 2 chunks per thread
//   SRC_F32  && LDS bf16:  32 k x 32 chunks of 4 columns, 4 chunks per thread
template <bool SRC_BF16, bool LDS_BF16>
struct LoadTrans {
    static constexpr int NCH = (!SRC_BF16 && LDS_BF16) ? 4 : 2;
    static constexpr int CPR = SRC_BF16 ? 16 : 32;       // chunks per source row
    static constexpr int VEC = SRC_BF16 ? 8 : 4;         // columns per chunk
    static constexpr int SES = SRC_BF16 ? 2 : 4;         // source element size
    static constexpr int LES = LDS_BF16 ? 2 : 4;         // LDS element size
    const char *base;
    int64_t ld_bytes;
    int64_t ksrc;       // source rows (the reduction length)
    int64_t cols;       // source columns
    int64_t col0;
    int ik[NCH], cq[NCH];
    uint4 reg[NCH];
    __device__ void init(int64_t c0) {
        col0 = c0;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const int chunk = threadIdx.x + c * kThreads;
            ik[c] = chunk / CPR;
            cq[c] = chunk % CPR;
        }
    }
    __device__ void load(int64_t k0) {
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const int64_t i = k0 + ik[c];
            const int64_t col = col0 + (int64_t)cq[c] * VEC;
            reg[c] = (i < ksrc && col < cols)
                         ? *(const uint4 *)(base + i * ld_bytes + col * SES)
                         : make_uint4(0, 0, 0, 0);
        }
    }
    __device__ void store(char *lds) const {
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const uint32_t w[4] = {reg[c].x, reg[c].y, reg[c].z, reg[c].w};
            if constexpr (SRC_BF16) {
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const uint16_t h = (uint16_t)(w[e >> 1] >> ((e & 1) * 16));
                    *(uint16_t *)(lds + (cq[c] * 8 + e) * kPitch + ik[c] * 2) = h;
                }
            } else if constexpr (LDS_BF16) {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    *(uint16_t *)(lds + (cq[c] * 4 + e) * kPitch + ik[c] * 2) =
                        (uint16_t)f32_to_bf16_bits(__uint_as_float(w[e]));
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    *(uint32_t *)(lds + (cq[c] * 4 + e) * kPitch + ik[c] * 4) = w[e];
            }
        }
        (void)LES;
    }
};

// ------------------------------------------------------------------ epilogues
// Each call gets 16 consecutive columns of one row.
template <bool OUT_BF16>
struct EpiForward {
    void *y;
    const void *bias;    // block dtype, [N] or NULL
    int64_t M;
    int32_t N;
    int32_t relu;
    __device__ void operator()(int64_t m, int64_t n0, const float *v) const {
        if (m >= M) return;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int64_t n = n0 + 4 * q;
            if (n >= N) return;
            float r[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                float b = 0.f;
                if (bias) {
                    if constexpr (OUT_BF16)
                        b = __uint_as_float((uint32_t)((const uint16_t *)bias)[n + e] << 16);
                    else
                        b = ((const float *)bias)[n + e];
                }
                r[e] = v[4 * q + e] + b;
                if (relu) r[e] = r[e] > 0.f ? r[e] : 0.f;
            }
            if constexpr (OUT_BF16) {
                uint2 w;
                w.x = pack_bf16x2(r[0], r[1]);
                w.y = pack_bf16x2(r[2], r[3]);
                *(uint2 *)((uint16_t *)y + m * N + n) = w;
            } else {
                *(float4 *)((float *)y + m * N + n) = make_float4(r[0], r[1], r[2], r[3]);
            }
        }
    }
};

struct EpiDms {
    float *out;
    int64_t M;
    int32_t N;
    int32_t d_in;
    const int32_t *indptr[kMaxSlots];
    __device__ void operator()(int64_t m, int64_t n0, const float *v) const {
        if (m >= M) return;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int64_t n = n0 + 4 * q;
            if (n >= N) return;
            const int sl = (int)(n / d_in);
            float scale = 1.f;
            bool zero = false;
            if (indptr[sl]) {
                const int32_t deg = indptr[sl][m + 1] - indptr[sl][m];
                zero = deg == 0;
                scale = (float)deg;
            }
            float4 r;
            r.x = zero ? 0.f : v[4 * q + 0] / scale;
            r.y = zero ? 0.f : v[4 * q + 1] / scale;
            r.z = zero ? 0.f : v[4 * q + 2] / scale;
            r.w = zero ? 0.f : v[4 * q + 3] / scale;
            *(float4 *)(out + m * N + n) = r;
        }
    }
};

struct EpiPartial {
    float *out;          // [splits][M][N]
    int64_t M;
    int32_t N;
    __device__ void operator()(int64_t m, int64_t n0, const float *v) const {
        if (m >= M) return;
        float *o = out + (int64_t)blockIdx.y * M * N + m * N;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int64_t n = n0 + 4 * q;
            if (n >= N) return;
            *(float4 *)(o + n) = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
        }
    }
};

// ------------------------------------------------------------------ the kernel
// Grid: x = output tiles (XCD-major so tiles sharing an A row-block share an L2),
// y = splits of the reduction (weight side only).
template <class Mma, class LA, class LB, class Epi>
__global__ __launch_bounds__(kThreads, 2) void k_gemm(LA la, LB lb, Epi epi, int64_t K,
                                                      int64_t tiles_n, int64_t k_per_split) {
    __shared__ __attribute__((aligned(16))) char lds[4 * kTileBytes];
    const int64_t total = (int64_t)gridDim.x;
    const int64_t t = xcd_major_id(blockIdx.x, total);
    const int64_t tm = t / tiles_n, tn = t - tm * tiles_n;
    const int64_t m0 = tm * kTile, n0 = tn * kTile;
    const int64_t kb = (int64_t)blockIdx.y * k_per_split;
    const int64_t ke = kb + k_per_split < K ? kb + k_per_split : K;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave >> 1, wn = wave & 1;

    la.init(m0);
    lb.init(n0);
    f32x4 acc[4][4];
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) acc[mi][ni] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int64_t nk = ke > kb ? cdiv(ke - kb, Mma::BK) : 0;
    if (nk > 0) {
        la.load(kb);
        lb.load(kb);
    }
    for (int64_t it = 0; it < nk; ++it) {
        char *As = lds + (it & 1) * 2 * kTileBytes;
        char *Bs = As + kTileBytes;
        la.store(As);
        lb.store(Bs);
        __syncthreads();
        if (it + 1 < nk) {
            la.load(kb + (it + 1) * Mma::BK);
            lb.load(kb + (it + 1) * Mma::BK);
        }
        Mma::run(As, Bs, acc, wm, wn, lane);
    }
    __syncthreads();

    // epilogue: per wave, 16 rows at a time through LDS, then 16 contiguous columns/lane
    float *stage = (float *)lds + wave * 16 * kStagePitch;
    const int rq = lane >> 4, cc = lane & 15;
#pragma unroll
    for (int mi = 0; mi < 4; ++mi) {
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                stage[(4 * rq + v) * kStagePitch + ni * 16 + cc] = acc[mi][ni][v];
        __syncthreads();
        const int r = lane >> 2, c0 = (lane & 3) * 16;
        float vals[16];
#pragma unroll
        for (int e = 0; e < 16; e += 4) {
            const float4 x = *(const float4 *)(stage + r * kStagePitch + c0 + e);
            vals[e] = x.x; vals[e + 1] = x.y; vals[e + 2] = x.z; vals[e + 3] = x.w;
        }
        epi(m0 + wm * 64 + mi * 16 + r, n0 + wn * 64 + c0, vals);
        __syncthreads();
    }
}

template <class Mma, class LA, class LB, class Epi>
hipError_t launch_gemm(const LA &la, const LB &lb, const Epi &epi, int64_t M, int64_t N,
                       int64_t K, int64_t splits, int64_t k_per_split, hipStream_t s) {
    const int64_t tiles_m = cdiv(M, kTile), tiles_n = cdiv(N, kTile);
    if (tiles_m == 0 || tiles_n == 0 || splits == 0) return hipSuccess;
    hipLaunchKernelGGL((k_gemm<Mma, LA, LB, Epi>), dim3((unsigned)(tiles_m * tiles_n),
                       (unsigned)splits), dim3(kThreads), 0, s, la, lb, epi, K, tiles_n,
                       k_per_split);
    return hipGetLastError();
}

// Split of the weight-side reduction over rows: enough workgroups to fill the chip
// (~4 per CU), each split a whole number of K steps and at least 8 of them.
void dw_split(int64_t M, int Kcat, int d_out, int bk, int64_t *splits, int64_t *per) {
    const int64_t tiles = cdiv(Kcat, kTile) * cdiv(d_out, kTile);
    int64_t want = cdiv(1024, tiles);
    const int64_t max_by_len = cdiv(M, (int64_t)bk * 8);
    if (want > max_by_len) want = max_by_len;
    if (want < 1) want = 1;
    int64_t p = cdiv(cdiv(M, want), bk) * bk;
    if (p < bk) p = bk;
    *per = p;
    *splits = M > 0 ? cdiv(M, p) : 0;
}

// dW_slot[c][o] = sum over splits (in order) of partial[split][slot * d_in + c][o]
__global__ __launch_bounds__(kThreads) void k_dw_reduce(const float *partial, int64_t splits,
                                                        int Kcat, int d_in, int d_out, DwOut out) {
    const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const int64_t total = (int64_t)Kcat * d_out;
    if (e >= total) return;
    const int64_t row = e / d_out, o = e - row * d_out;
    const int sl = (int)(row / d_in);
    float *dst = out.w[sl];
    if (!dst) return;
    float acc = 0.f;
    for (int64_t sp = 0; sp < splits; ++sp) acc += partial[sp * total + e];
    dst[(row - (int64_t)sl * d_in) * d_out + o] = acc;
}

__global__ __launch_bounds__(kThreads) void k_zero_outputs(DwOut out, int d_in, int d_out) {
    const int64_t per = (int64_t)d_in * d_out;
    const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const int sl = (int)blockIdx.y;
    if (e < per && out.w[sl]) out.w[sl][e] = 0.f;
}

}  // namespace

hipError_t gemm_forward(rgcn_dtype dt, const void *a, int64_t M, int N, int K,
                        const void *wcat_t, const void *bias, int relu, void *y,
                        hipStream_t s) {
    const int es = dt == RGCN_BF16 ? 2 : 4;
    LoadRows<PlainRows> la{PlainRows{(const char *)a, (int64_t)K * es, M}, (int64_t)K * es, es, 0};
    LoadRows<PlainRows> lb{PlainRows{(const char *)wcat_t, (int64_t)K * es, N}, (int64_t)K * es,
                           es, 0};
    if (dt == RGCN_BF16)
        return launch_gemm<MmaBf16>(la, lb, EpiForward<true>{y, bias, M, N, relu}, M, N, K, 1, K, s);
    return launch_gemm<MmaF32>(la, lb, EpiForward<false>{y, bias, M, N, relu}, M, N, K, 1, K, s);
}

hipError_t gemm_dms(rgcn_dtype dt, const float *dy, int64_t M, int d_out, int d_in,
                    const DmsSlots &slots, float *dms, hipStream_t s) {
    const int es = dt == RGCN_BF16 ? 2 : 4;
    const int64_t N = (int64_t)slots.count * d_in;
    SlotRows sr;
    for (int i = 0; i < kMaxSlots; ++i) sr.w[i] = i < slots.count ? slots.w[i] : nullptr;
    sr.d_in = d_in;
    sr.es_dout = d_out * es;
    sr.rows = N;
    LoadRows<SlotRows> lb{sr, (int64_t)d_out * es, es, 0};
    EpiDms epi;
    epi.out = dms;
    epi.M = M;
    epi.N = (int32_t)N;
    epi.d_in = d_in;
    for (int i = 0; i < kMaxSlots; ++i) epi.indptr[i] = i < slots.count ? slots.indptr[i] : nullptr;
    PlainRows pa{(const char *)dy, (int64_t)d_out * 4, M};
    if (dt == RGCN_BF16) {
        // dY enters as hi + lo bf16 parts: K = 2 d_out, the weight rows read twice
        LoadRowsF32Split la{pa, d_out};
        LoadRows<SlotRows, true> lbw{sr, (int64_t)d_out * es, es, (int64_t)d_out * es};
        return launch_gemm<MmaBf16>(la, lbw, epi, M, N, 2 * (int64_t)d_out, 1, 2 * (int64_t)d_out, s);
    }
    LoadRows<PlainRows> la{pa, (int64_t)d_out * 4, 4, 0};
    return launch_gemm<MmaF32>(la, lb, epi, M, N, d_out, 1, d_out, s);
}

size_t gemm_dw_partial_bytes(int64_t M, int Kcat, int d_out) {
    int64_t sp16, p16, sp32, p32;
    dw_split(M, Kcat, d_out, 16, &sp16, &p16);
    dw_split(M, Kcat, d_out, 32, &sp32, &p32);
    const int64_t sp = sp16 > sp32 ? sp16 : sp32;
    return (size_t)(sp > 0 ? sp : 1) * Kcat * d_out * 4 + 256;
}

hipError_t gemm_dw(rgcn_dtype dt, const void *mcat, int64_t M, int Kcat, int d_in,
                   const float *dy, int d_out, const DwOut &out, float *partial,
                   hipStream_t s) {
    const bool bf = dt == RGCN_BF16;
    const int bk = bf ? MmaBf16::BK : MmaF32::BK;
    int64_t splits, per;
    dw_split(M, Kcat, d_out, bk, &splits, &per);
    if (splits == 0) {  // no rows: every requested gradient is zero
        hipLaunchKernelGGL(k_zero_outputs, dim3((unsigned)cdiv((int64_t)d_in * d_out, kThreads),
                           (unsigned)out.count), dim3(kThreads), 0, s, out, d_in, d_out);
        return hipGetLastError();
    }
    EpiPartial epi{partial, Kcat, d_out};
    if (bf) {
        LoadTrans<true, true> la{(const char *)mcat, (int64_t)Kcat * 2, M, Kcat};
        LoadTrans<false, true> lb{(const char *)dy, (int64_t)d_out * 4, M, d_out};
        RGCN_HIP_TRY(launch_gemm<MmaBf16>(la, lb, epi, Kcat, d_out, M, splits, per, s));
    } else {
        LoadTrans<false, false> la{(const char *)mcat, (int64_t)Kcat * 4, M, Kcat};
        LoadTrans<false, false> lb{(const char *)dy, (int64_t)d_out * 4, M, d_out};
        RGCN_HIP_TRY(launch_gemm<MmaF32>(la, lb, epi, Kcat, d_out, M, splits, per, s));
    }
    const int64_t total = (int64_t)Kcat * d_out;
    hipLaunchKernelGGL(k_dw_reduce, dim3((unsigned)cdiv(total, kThreads)), dim3(kThreads), 0, s,
                       partial, splits, Kcat, d_in, d_out, out);
    return hipGetLastError();
}

}  // namespace rgcn
