// Dense transforms of the block on the CDNA4 matrix cores:
//   forward      Y_t   = Mcat_t  [n_dst x K]      . WcatT_t^T  (+ bias, opt. ReLU)
//                K = (1 + R_t) * d_in: the self-loop and every relation into t are one
//                K-concatenated product, so the sum over relations is the K reduction.
//   input side   dMs_t = dY_t [n_dst x d_out]    . [W_s rows]^T, slot columns / deg
//   weight side  dW    = Mcat_t^T [K x n_dst]    . dY_t [n_dst x d_out]   (split over rows)
//
// bf16 mode, fp32 accumulation, one kernel per product:
//   k_gemm_fwd  forward: both operands are K-contiguous bf16 rows, loaded straight from
//               global memory into LDS, 256 x 256 tiles (16 waves of 64 x 64),
//               v_mfma_f32_16x16x32_bf16; persistent, one K-step pipeline across a
//               workgroup's tiles, epilogue stored from registers;
//   k_dms_stream input side with at most 128 output columns and d_out 256 or 512 (the
//               input layer's embedding slots): K split over the waves, the weights held
//               in registers, dY read once in whole rows, partial sums met in LDS;
//   k_gemm      input side otherwise: the register-staged kernel below with 128 x 128
//               tiles (N is one or two slots of d_in columns; a 256-wide tile would be half
//               empty), on v_mfma_f32_32x32x16_bf16 (the 16 x 16 x 32 form issues at half
//               its rate on gfx950);
//   k_gemm_dw   weight side: reduces over the rows of both operands; 256 x 256 tiles whose
//               operands are loaded straight into LDS (one row per m) and read down the
//               columns, on v_mfma_f32_32x32x16_bf16.
// These products are skinny (K and N of a few hundred against up to millions of rows), so
// what limits them is how often the long operand is re-read: a 256-wide tile reads it half
// as often as a 128-wide one.  The fp32 output gradient dY enters both backward products as
// a hi + lo pair of bf16 values (hi = bf16(x), lo = bf16(x - hi)), ~16 significant bits:
// each fp32 tile is read from memory once and split on the way to the MFMA operands, and
// every fragment of the other operand meets both parts.
//
// k_gemm (input side, and every product in fp32 mode with v_mfma_f32_16x16x4_f32): LDS
// holds both operands K-contiguous ("row r, k..."), one row = BK elements of K + 16 bytes
// of padding; the row pitch is an odd number of 16-byte units, so the 16 rows a 16-lane
// group reads for one MFMA operand fall in distinct bank groups.  Global loads are staged
// through registers, issued in a fixed order and always unconditionally (rows past the end
// and K past the range read a zero buffer), so each LDS store waits only for its own
// loads.  The fp32 weight side transposes its tiles on the way to LDS with scalar writes.
#include <type_traits>

#include "common.h"

namespace rgcn {
namespace {

constexpr int kThreads = 256;                     // small helper kernels
constexpr int kStagePitch = 68;                   // epilogue staging row (floats)
__host__ __device__ inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Workgroup tile TM x TN, WM x WN waves; each wave FM x FN MFMA tiles of 16 x 16.
template <int TM_, int TN_, int WM_, int WN_>
struct Cfg {
    static constexpr int TM = TM_, TN = TN_, WM = WM_, WN = WN_;
    static constexpr int NT = 64 * WM * WN;
    static constexpr int FM = TM / WM / 16, FN = TN / WN / 16;
    static_assert(FN * 16 == 64, "epilogue stages 64 columns per wave");
};
using CfgWide = Cfg<256, 256, 2, 4>;
using CfgNarrow = Cfg<128, 128, 2, 2>;
using CfgFwd = Cfg<256, 256, 4, 4>;   // bf16 forward: 16 waves of 64 x 64
using CfgDms = CfgNarrow;   // bf16 input side: N is one or two slots of d_in columns
// bf16 weight side (k_gemm_dw): 256 x 256 tiles of 8 waves, one workgroup per CU (16
// waves of 64 x 64 measured 1 % slower)
using CfgDw = CfgWide;
constexpr int kDwMinWaves = CfgDw::NT / 64 / 4;   // waves per SIMD
using CfgF32 = Cfg<128, 128, 2, 2>;

template <int ROWS_, int BK_, int ES_>
struct Tile {
    static constexpr int ROWS = ROWS_;            // rows of the operand tile
    static constexpr int BK = BK_;                // K elements per step
    static constexpr int ES = ES_;                // LDS element size
    static constexpr int PAYLOAD = BK_ * ES_;     // bytes of K per LDS row
    static constexpr int PITCH = PAYLOAD + 16;
    static constexpr int CPR = PAYLOAD / 16;      // 16-byte chunks per LDS row
    static constexpr int BYTES = ROWS_ * PITCH;   // one operand tile
    static_assert((PITCH / 16) % 2 == 1, "pitch must be an odd number of 16-byte units");
};
template <class C> using TileBf16 = Tile<C::TM, 64, 2>;
using TileF32 = Tile<CfgF32::TM, 16, 4>;

// Register staging uses the compiler's native vector types (one 16-byte load or LDS store,
// no struct copies).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
// Loads a thread does not need (rows past the end, K past the range) read these zero bytes
// instead, so the registers hold zeros without a select; never written.
__device__ u32x4 g_zero16[2];

// ------------------------------------------------------------------ MFMA cores
// A held as two bf16 tiles (hi at As, lo two tiles further, after B) of one fp32 operand:
// acc += A_hi.B + A_lo.B, fp32 accumulation, on 32 x 32 x 16 MFMA tiles (the 16 x 16 x 32
// form issues at half the rate on gfx950): the wave's 16 x 16 grid of FM x FN fragments
// is (FM / 2) x (FN / 2) accumulators of 32 x 32.  Lane l reads row l % 32 of the operand
// tile at K chunk 2 s + l / 32 of K sub-step s (16 elements); it holds column l % 32 of
// each accumulator and rows 8 (e / 4) + 4 (l / 32) + e % 4 for its 16 values e.
template <class TL, int FM, int FN>
struct MmaBf16SplitA32 {
    using T = TL;
    using Acc = f32x16;
    static constexpr int AM = FM / 2, AN = FN / 2;
    static_assert(AM * 2 == FM && AN * 2 == FN, "pairs of 16 x 16 fragments");
    static constexpr int STAGE_BYTES = 3 * TL::BYTES;   // A_hi, B, A_lo
    __device__ __forceinline__ static void run(const char *As, const char *Bs,
                                               f32x16 (&acc)[AM][AN], int wm, int wn, int lane) {
        const int r = lane & 31, h = lane >> 5;
        const char *Al = As + 2 * TL::BYTES;
#pragma unroll
        for (int s = 0; s < TL::BK / 16; ++s) {
            bf16x8 b[AN];
#pragma unroll
            for (int i = 0; i < AN; ++i)
                b[i] = *(const bf16x8 *)(Bs + (wn * AN * 32 + i * 32 + r) * TL::PITCH + s * 32 + h * 16);
#pragma unroll
            for (int mi = 0; mi < AM; ++mi) {
                const int ao = (wm * AM * 32 + mi * 32 + r) * TL::PITCH + s * 32 + h * 16;
                const bf16x8 ah = *(const bf16x8 *)(As + ao);
                const bf16x8 al = *(const bf16x8 *)(Al + ao);
#pragma unroll
                for (int ni = 0; ni < AN; ++ni) {
                    acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, b[ni], acc[mi][ni],
                                                                          0, 0, 0);
                    acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, b[ni], acc[mi][ni],
                                                                          0, 0, 0);
                }
            }
        }
    }
};

// fp32: lane group q holds k = 4q..4q+3 of its row; MFMA step s uses element s, so the
// four steps together cover k = 0..15 (the sum over k is taken in a different order, not
// a different set).
template <int FM, int FN>
struct MmaF32 {
    using T = TileF32;
    using Acc = f32x4;
    static constexpr int AM = FM, AN = FN;
    static constexpr int STAGE_BYTES = 2 * T::BYTES;
    __device__ __forceinline__ static void run(const char *As, const char *Bs,
                                               f32x4 (&acc)[FM][FN], int wm, int wn, int lane) {
        f32x4 a[FM], b[FN];
        const int r = lane & 15, q = lane >> 4;
#pragma unroll
        for (int i = 0; i < FM; ++i)
            a[i] = *(const f32x4 *)(As + (wm * FM * 16 + i * 16 + r) * T::PITCH + q * 16);
#pragma unroll
        for (int i = 0; i < FN; ++i)
            b[i] = *(const f32x4 *)(Bs + (wn * FN * 16 + i * 16 + r) * T::PITCH + q * 16);
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int mi = 0; mi < FM; ++mi)
#pragma unroll
                for (int ni = 0; ni < FN; ++ni)
                    acc[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[mi][s], b[ni][s],
                                                                       acc[mi][ni], 0, 0, 0);
    }
};

// ------------------------------------------------------------------ tile loaders
// Row addressing policies.  row(r) always returns a readable row (out-of-range rows are
// clamped to the last one); loads of rows r >= rows read the zero buffer instead.
struct PlainRows {
    const char *base;
    int64_t ld_bytes;
    int64_t rows;
    __device__ __forceinline__ const char *row(int64_t r) const {
        return base + (r < rows ? r : rows - 1) * ld_bytes;
    }
};
struct SlotRows {  // row n = (slot n / d_in, column c = n % d_in) of W_slot [d_in x d_out]
    const void *w[kMaxSlots];
    int32_t d_in;
    int32_t es_dout;   // bytes per W row (d_out * element size)
    int64_t rows;
    __device__ __forceinline__ const char *row(int64_t r) const {
        const int64_t rr = r < rows ? r : rows - 1;
        const int64_t sl = rr / d_in, c = rr - sl * d_in;
        return (const char *)w[sl] + c * es_dout;
    }
};

// K-contiguous rows whose element type is the LDS type.
template <class TL, int NT, class RowPolicy>
struct LoadRows {
    static constexpr int NCH = TL::ROWS * TL::CPR / NT;
    static_assert(NCH * NT == TL::ROWS * TL::CPR, "threads must divide the tile's chunks");
    RowPolicy pol;
    int64_t kbytes;       // bytes of K per source row
    struct State {
        const char *rp[NCH];
        bool rok[NCH];
        int lr[NCH], lq[NCH];
        u32x4 reg[NCH];
    };
    __device__ __forceinline__ void init(State &st, int64_t row0) const {
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const int chunk = threadIdx.x + c * NT;
            st.lr[c] = chunk / TL::CPR;
            st.lq[c] = chunk % TL::CPR;
            st.rok[c] = row0 + st.lr[c] < pol.rows;
            st.rp[c] = pol.row(row0 + st.lr[c]);
        }
    }
    __device__ __forceinline__ void load(State &st, int64_t k0, int64_t kend) const {
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const int64_t k = k0 + st.lq[c] * (16 / TL::ES);
            const int64_t kb = k * TL::ES;
            const bool ok = st.rok[c] && kb < kbytes && k < kend;
            st.reg[c] = *(const u32x4 *)(ok ? st.rp[c] + kb : (const char *)g_zero16);
        }
    }
    __device__ __forceinline__ void store(const State &st, char *lds) const {
#pragma unroll
        for (int c = 0; c < NCH; ++c)
            *(u32x4 *)(lds + st.lr[c] * TL::PITCH + st.lq[c] * 16) = st.reg[c];
    }
};

// fp32 rows entering a bf16 product as a hi + lo pair read once: each 32-byte piece (8
// values) goes to the hi tile at lds (hi = bf16(x)) and to the lo tile at lds + LO_OFF
// (lo = bf16(x - hi)), for MmaBf16SplitA.
template <class TL, int NT, int LO_OFF>
struct LoadRowsF32HiLo {
    static constexpr int CPR = TL::BK / 8;        // 8 bf16 per 16-byte LDS chunk
    static constexpr int NCH = TL::ROWS * CPR / NT;
    static_assert(NCH * NT == TL::ROWS * CPR, "threads must divide the tile's chunks");
    PlainRows pol;
    int64_t K;
    struct State {
        const char *rp[NCH];
        bool rok[NCH];
        int lr[NCH], lq[NCH];
        f32x4 reg[NCH][2];
    };
    __device__ __forceinline__ void init(State &st, int64_t row0) const {
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const int chunk = threadIdx.x + c * NT;
            st.lr[c] = chunk / CPR;
            st.lq[c] = chunk % CPR;
            st.rok[c] = row0 + st.lr[c] < pol.rows;
            st.rp[c] = pol.row(row0 + st.lr[c]);
        }
    }
    __device__ __forceinline__ void load(State &st, int64_t k0, int64_t kend) const {
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const int64_t k = k0 + st.lq[c] * 8;
            const bool ok = st.rok[c] && k < K && k < kend;
            const char *p = ok ? st.rp[c] + k * 4 : (const char *)g_zero16;
            st.reg[c][0] = *(const f32x4 *)p;
            st.reg[c][1] = *(const f32x4 *)(p + 16);
        }
    }
    __device__ __forceinline__ void store(const State &st, char *lds) const {
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const f32x4 a = st.reg[c][0], b = st.reg[c][1];
            u32x4 h, l;
            h.x = pack_bf16x2(a.x, a.y);
            h.y = pack_bf16x2(a.z, a.w);
            h.z = pack_bf16x2(b.x, b.y);
            h.w = pack_bf16x2(b.z, b.w);
            l.x = pack_bf16x2(a.x - bf16_lo(h.x), a.y - bf16_hi(h.x));
            l.y = pack_bf16x2(a.z - bf16_lo(h.y), a.w - bf16_hi(h.y));
            l.z = pack_bf16x2(b.x - bf16_lo(h.z), b.y - bf16_hi(h.z));
            l.w = pack_bf16x2(b.z - bf16_lo(h.w), b.w - bf16_hi(h.w));
            char *d = lds + st.lr[c] * TL::PITCH + st.lq[c] * 16;
            *(u32x4 *)d = h;
            *(u32x4 *)(d + LO_OFF) = l;
        }
    }
};

// The same tiles from dY rows in the hi/lo form (K bf16 high parts, then K low parts; a
// row's byte pitch is that of its fp32 form): each chunk's high and low parts are loaded
// as they are and stored without a split.
template <class TL, int NT, int LO_OFF>
struct LoadRowsHiLoBf16 {
    static constexpr int CPR = TL::BK / 8;
    static constexpr int NCH = TL::ROWS * CPR / NT;
    static_assert(NCH * NT == TL::ROWS * CPR, "threads must divide the tile's chunks");
    PlainRows pol;   // ld_bytes = 4 K
    int64_t K;
    struct State {
        const char *rp[NCH];
        bool rok[NCH];
        int lr[NCH], lq[NCH];
        u32x4 reg[NCH][2];
    };
    __device__ __forceinline__ void init(State &st, int64_t row0) const {
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const int chunk = threadIdx.x + c * NT;
            st.lr[c] = chunk / CPR;
            st.lq[c] = chunk % CPR;
            st.rok[c] = row0 + st.lr[c] < pol.rows;
            st.rp[c] = pol.row(row0 + st.lr[c]);
        }
    }
    __device__ __forceinline__ void load(State &st, int64_t k0, int64_t kend) const {
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const int64_t k = k0 + st.lq[c] * 8;
            const bool ok = st.rok[c] && k < K && k < kend;
            const char *p = ok ? st.rp[c] + k * 2 : (const char *)g_zero16;
            const int64_t lo = ok ? K * 2 : 0;
            st.reg[c][0] = *(const u32x4 *)p;
            st.reg[c][1] = *(const u32x4 *)(p + lo);
        }
    }
    __device__ __forceinline__ void store(const State &st, char *lds) const {
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            char *d = lds + st.lr[c] * TL::PITCH + st.lq[c] * 16;
            *(u32x4 *)d = st.reg[c][0];
            *(u32x4 *)(d + LO_OFF) = st.reg[c][1];
        }
    }
};

// fp32 weight side: 16 k x (ROWS / 4) chunks of 4 columns, transposed by scalar LDS writes
// (used only in fp32 mode).
template <int NT>
struct LoadTransF32 {
    using TL = TileF32;
    static constexpr int NCH = 16 * (TL::ROWS / 4) / NT;
    static_assert(NCH * NT == 16 * (TL::ROWS / 4), "threads must divide the tile's chunks");
    const char *base;
    int64_t ld_bytes;
    int64_t ksrc;
    int64_t cols;
    struct State {
        int64_t col0;
        int ik[NCH], cq[NCH];
        u32x4 reg[NCH];
    };
    __device__ __forceinline__ void init(State &st, int64_t c0) const {
        st.col0 = c0;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const int chunk = threadIdx.x + c * NT;
            st.ik[c] = chunk / (TL::ROWS / 4);
            st.cq[c] = chunk % (TL::ROWS / 4);
        }
    }
    __device__ __forceinline__ void load(State &st, int64_t k0, int64_t kend) const {
        const int64_t lim = kend < ksrc ? kend : ksrc;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const int64_t i = k0 + st.ik[c];
            const int64_t col = st.col0 + (int64_t)st.cq[c] * 4;
            const bool ok = i < lim && col < cols;
            st.reg[c] = *(const u32x4 *)(ok ? base + i * ld_bytes + col * 4 : (const char *)g_zero16);
        }
    }
    __device__ __forceinline__ void store(const State &st, char *lds) const {
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const u32x4 v = st.reg[c];
#pragma unroll
            for (int e = 0; e < 4; ++e)
                *(uint32_t *)(lds + (st.cq[c] * 4 + e) * TL::PITCH + st.ik[c] * 4) = v[e];
        }
    }
};

// ------------------------------------------------------------------ epilogues
// Each call gets 16 consecutive columns of one row.
// ReLU sign words: bit c % 64 of word c / 64 of row m is set when the stored value (m, c)
// is positive.  A lane hands in the bits of its own columns, already shifted to their place
// in the 64-column word of its wave; the lanes that share a row OR theirs together (xor
// shuffles over `span` lanes at stride `step`) and the first of them stores the word.
struct ReluMask {
    uint64_t *w;         // [M x ld] or NULL
    int64_t ld;
    __device__ __forceinline__ void put(int64_t m, int64_t M, int64_t col0, int64_t N,
                                        uint64_t bits, int step, int span, bool first) const {
        for (int o = step; o < step * span; o <<= 1) bits |= (uint64_t)shfl64((int64_t)bits, (int)(__lane_id() ^ o));
        if (first && m < M && col0 < N) w[m * ld + col0 / 64] = bits;
    }
};

template <bool OUT_BF16>
struct EpiForward {
    static constexpr bool kPrefetch = false;
    static constexpr bool kMask = true;
    void *y;
    const void *bias;    // block dtype, [N] or NULL
    int64_t M;
    int32_t N;
    int32_t relu;
    ReluMask mask;
    // v: columns n0 + 16 q .. + 3 for q = 0 .. 3; returns their positive bits (bit 4 q + e:
    // column n0 + 16 q + e)
    __device__ __forceinline__ uint32_t operator()(int64_t m, int64_t n0, const float *v, int64_t) const {
        if (m >= M) return 0u;
        // N is a multiple of 4: each group of 4 columns is either whole or absent.  The
        // bias loads are issued together (clamped, then zeroed) before any is used; with no
        // bias (a uniform test) nothing is loaded.
        float bq[4][4] = {};
        if (bias != nullptr) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int64_t n = n0 + 16 * q;
                const bool ok = n < N;
                if constexpr (OUT_BF16) {
                    const uint2 w = *(const uint2 *)((const uint16_t *)bias + (ok ? n : 0));
                    bq[q][0] = ok ? bf16_lo(w.x) : 0.f;
                    bq[q][1] = ok ? bf16_hi(w.x) : 0.f;
                    bq[q][2] = ok ? bf16_lo(w.y) : 0.f;
                    bq[q][3] = ok ? bf16_hi(w.y) : 0.f;
                } else {
                    const float4 w = *(const float4 *)((const float *)bias + (ok ? n : 0));
                    bq[q][0] = ok ? w.x : 0.f;
                    bq[q][1] = ok ? w.y : 0.f;
                    bq[q][2] = ok ? w.z : 0.f;
                    bq[q][3] = ok ? w.w : 0.f;
                }
            }
        }
        uint32_t bits = 0u;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int64_t n = n0 + 16 * q;
            if (n >= N) break;
            float r[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                r[e] = v[4 * q + e] + bq[q][e];
                if (relu) r[e] = r[e] > 0.f ? r[e] : 0.f;
            }
            if constexpr (OUT_BF16) {
                uint2 w;
                w.x = pack_bf16x2(r[0], r[1]);
                w.y = pack_bf16x2(r[2], r[3]);
                *(uint2 *)((uint16_t *)y + m * N + n) = w;
                bits |= (uint32_t)(((w.x & 0xffffu) != 0u) | (((w.x >> 16) != 0u) << 1) |
                                   (((w.y & 0xffffu) != 0u) << 2) | (((w.y >> 16) != 0u) << 3))
                        << (4 * q);
            } else {
                *(float4 *)((float *)y + m * N + n) = make_float4(r[0], r[1], r[2], r[3]);
#pragma unroll
                for (int e = 0; e < 4; ++e) bits |= (uint32_t)(r[e] > 0.f) << (4 * q + e);
            }
        }
        return bits;
    }
};

// The forward epilogue of the persistent kernel: 4 consecutive columns of one row per call,
// their bias loaded only when there is one.
struct EpiForwardBf16 {
    static constexpr bool kDms = false;
    void *y;
    const void *bias;    // bf16 [N] or NULL
    int64_t M;
    int32_t N;
    int32_t relu;
    ReluMask mask;
    // 4 columns from n (N is a multiple of 4: whole or absent)
    __device__ __forceinline__ void load_bias4(int64_t n, float *bq) const {
        bq[0] = bq[1] = bq[2] = bq[3] = 0.f;
        if (bias == nullptr || n >= N) return;
        const uint2 w = *(const uint2 *)((const uint16_t *)bias + n);
        bq[0] = bf16_lo(w.x);
        bq[1] = bf16_hi(w.x);
        bq[2] = bf16_lo(w.y);
        bq[3] = bf16_hi(w.y);
    }
    // the 4 values of columns n .. n + 3 with bias (and ReLU) as bf16 pairs lo, hi; returns
    // their positive bits (bit e: column n + e), none outside the output.  No branches: the
    // callers exchange the results between lanes.
    __device__ __forceinline__ uint32_t pack4(int64_t m, int64_t n, const f32x4 v,
                                              const float *bq, uint32_t &lo,
                                              uint32_t &hi) const {
        float r[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            r[e] = v[e] + bq[e];
            if (relu) r[e] = r[e] > 0.f ? r[e] : 0.f;
        }
        lo = pack_bf16x2(r[0], r[1]);
        hi = pack_bf16x2(r[2], r[3]);
        const uint32_t bits = (uint32_t)((lo & 0xffffu) != 0u) |
                              ((uint32_t)((lo >> 16) != 0u) << 1) |
                              ((uint32_t)((hi & 0xffffu) != 0u) << 2) |
                              ((uint32_t)((hi >> 16) != 0u) << 3);
        return m < M && n < N ? bits : 0u;
    }
    // 8 bf16 at columns n .. n + 7 of row m (N is a multiple of 8: whole or absent)
    __device__ __forceinline__ void store8(int64_t m, int64_t n, uint4 v) const {
        if (m < M && n < N) *(uint4 *)((uint16_t *)y + m * N + n) = v;
    }
};

// The input-side product dMs = dY W^T / deg in k_gemm_fwd, with dY in the hi/lo form: a
// row of d_out hi then d_out lo bf16 values is a bf16 row of K = 2 d_out, and the weight
// rows (packed [N x d_out]) serve K index k and k + d_out alike (kwrap = d_out), so each
// weight meets hi and lo.  fp32 output, divided by the degree of the row's segment in the
// column's slot (0 for an empty segment, as is for the self slot).  d_in is a multiple of
// 64, so a wave's 64 columns lie in one slot; inv_din = ceil(2^32 / d_in) gives the slot
// of a column as umulhi(n, inv_din) (exact for n < 2^21).
struct EpiDmsFwd {
    static constexpr bool kDms = true;
    float *out;
    int64_t M;
    int32_t N;
    int32_t kwrap;
    uint32_t inv_din;
    const int32_t *indptr[kMaxSlots];
};

// dMs rows divided by the segment's degree.  The degrees a lane's epilogue needs are read
// before the K loop (deg_of), so the epilogue waits for no load (store).
struct EpiDms {
    static constexpr bool kPrefetch = true;
    float *out;
    int64_t M;
    int32_t N;
    int32_t d_in;
    const int32_t *indptr[kMaxSlots];
    // degree of row m in the slot of column n; -1 where the slot has none (scale 1) or the
    // element is outside the output
    __device__ __forceinline__ int32_t deg_of(int64_t m, int64_t n) const {
        if (m >= M || n >= N) return -1;
        const int sl = (int)(n / d_in);
        if (!indptr[sl]) return -1;
        return indptr[sl][m + 1] - indptr[sl][m];
    }
    // v: columns n0 + 16 q .. + 3, which take degree deg[q]
    __device__ __forceinline__ void store(int64_t m, int64_t n0, const float *v,
                                          const int32_t *deg) const {
        if (m >= M) return;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int64_t n = n0 + 16 * q;
            if (n >= N) return;
            const bool zero = deg[q] == 0;
            const float scale = deg[q] > 0 ? (float)deg[q] : 1.f;
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
    static constexpr bool kPrefetch = false;
    static constexpr bool kMask = false;
    float *out;          // [splits][M][N]
    int64_t M;
    int32_t N;
    __device__ __forceinline__ void operator()(int64_t m, int64_t n0, const float *v,
                                               int64_t split) const {
        if (m >= M) return;
        float *o = out + split * M * N + m * N;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int64_t n = n0 + 16 * q;   // v: columns n0 + 16 q .. + 3
            if (n >= N) return;
            *(float4 *)(o + n) = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
        }
    }
};

// ------------------------------------------------------------------ the kernel
// One-dimensional grid over (split, output tile), numbered XCD-major: the dispatcher
// sends workgroup w to XCD w mod 8, and consecutive logical ids -- the tiles of one
// split, and within a split the tiles sharing a row block of A -- land on the same XCD
// and share its L2.
// STAGES = 2: double-buffered LDS (one barrier per step); STAGES = 1: one buffer.
// R register stages: the global loads of step k + R are issued right after step k's tiles
// reach LDS, so R multiplies overlap each load's latency.
template <class C, class Mma, class LA, class LB, class Epi, int STAGES, int R>
__global__ __launch_bounds__(C::NT) void k_gemm(const LA la, const LB lb, const Epi epi,
                                                int64_t K, int64_t tiles_m, int64_t tiles_n,
                                                int64_t k_per_split) {
    using TL = typename Mma::T;
    constexpr int FM = C::FM, FN = C::FN;
    constexpr int STAGE_BYTES = Mma::STAGE_BYTES;
    constexpr int NW = C::NT / 64;
    __shared__ __attribute__((aligned(16))) char lds[STAGES * STAGE_BYTES];
    static_assert(STAGES * STAGE_BYTES >= NW * 16 * kStagePitch * 4, "epilogue staging space");
    const int64_t logical = xcd_major_id(blockIdx.x, (int64_t)gridDim.x);
    const int64_t tiles = tiles_m * tiles_n;
    const int64_t split = logical / tiles;
    const int64_t t = logical - split * tiles;
    const int64_t tm = t / tiles_n, tn = t - tm * tiles_n;
    const int64_t m0 = tm * C::TM, n0 = tn * C::TN;
    const int64_t kb = split * k_per_split;
    const int64_t ke = kb + k_per_split < K ? kb + k_per_split : K;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave / C::WN, wn = wave % C::WN;

    typename LA::State sa[R];
    typename LB::State sb[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        la.init(sa[r], m0);
        lb.init(sb[r], n0);
    }
    using Acc = typename Mma::Acc;
    constexpr int AM = Mma::AM, AN = Mma::AN;
    constexpr int AV = (int)(sizeof(Acc) / sizeof(float));   // values per lane per accumulator
    Acc acc[AM][AN];
#pragma unroll
    for (int mi = 0; mi < AM; ++mi)
#pragma unroll
        for (int ni = 0; ni < AN; ++ni)
#pragma unroll
            for (int e = 0; e < AV; ++e) acc[mi][ni][e] = 0.f;

    // the epilogue's per-row data (EpiDms: degrees), read before the tiles so the loads
    // are long done when the epilogue needs them; slice e of the wave covers rows
    // m0 + wm FM 16 + 16 e + er, the lane columns n0 + wn FN 16 + ec + 16 q
    const int er = lane & 15, ec = 4 * (lane >> 4);
    int32_t pdeg[FM][4];
    if constexpr (Epi::kPrefetch) {
#pragma unroll
        for (int e = 0; e < FM; ++e)
#pragma unroll
            for (int q = 0; q < 4; ++q)
                pdeg[e][q] = epi.deg_of(m0 + wm * FM * 16 + 16 * e + er,
                                        n0 + wn * FN * 16 + ec + 16 * q);
    }

    // Steps are padded to a multiple of R and every load is issued unconditionally
    // (steps past the range load zero tiles), so all paths through the loop have the same
    // loads in flight and the waits before each LDS store cover only its own register set.
    const int64_t nk = ke > kb ? cdiv(ke - kb, TL::BK) : 0;
    const int64_t nkp = cdiv(nk, R) * R;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        la.load(sa[r], kb + r * TL::BK, ke);
        lb.load(sb[r], kb + r * TL::BK, ke);
        __builtin_amdgcn_sched_barrier(0);   // register set r's loads all precede set r+1's
    }
    for (int64_t it0 = 0; it0 < nkp; it0 += R) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int64_t it = it0 + r;
            char *As = lds + (STAGES == 2 ? (it & 1) * STAGE_BYTES : 0);
            char *Bs = As + TL::BYTES;
            if constexpr (STAGES == 1) __syncthreads();
            la.store(sa[r], As);
            lb.store(sb[r], Bs);
            __syncthreads();
            la.load(sa[r], kb + (it + R) * TL::BK, ke);
            lb.load(sb[r], kb + (it + R) * TL::BK, ke);
            // keep the loads ahead of the multiplies and their consumers after them
            __builtin_amdgcn_sched_barrier(0);
            Mma::run(As, Bs, acc, wm, wn, lane);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
    __syncthreads();

    // epilogue: per wave, 16 rows at a time through the wave's own LDS area; lane L takes
    // row L % 16 and columns 4 (L / 16) + 16 q .. + 3 (q = 0 .. 3), so the 4 lanes of a row
    // store 64 contiguous bytes in each store instruction
    float *stage = (float *)lds + wave * 16 * kStagePitch;
    auto emit = [&](int64_t row, int slice) {
        __builtin_amdgcn_wave_barrier();
        float vals[16];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float4 x = *(const float4 *)(stage + er * kStagePitch + ec + 16 * q);
            vals[4 * q] = x.x; vals[4 * q + 1] = x.y; vals[4 * q + 2] = x.z; vals[4 * q + 3] = x.w;
        }
        __builtin_amdgcn_wave_barrier();
        if constexpr (Epi::kPrefetch) {
            epi.store(row + er, n0 + wn * FN * 16 + ec, vals, pdeg[slice]);
        } else if constexpr (Epi::kMask) {
            // the 4 lanes of a row (L, L + 16, L + 32, L + 48) hold its 64 columns
            const uint32_t bits = epi(row + er, n0 + wn * FN * 16 + ec, vals, split);
            if (epi.mask.w != nullptr) {
                uint64_t b64 = 0u;
#pragma unroll
                for (int q = 0; q < 4; ++q) b64 |= (uint64_t)((bits >> (4 * q)) & 0xFu) << (ec + 16 * q);
                epi.mask.put(row + er, epi.M, n0 + wn * FN * 16, epi.N, b64, 16, 4, (lane >> 4) == 0);
            }
        } else {
            epi(row + er, n0 + wn * FN * 16 + ec, vals, split);
        }
    };
    if constexpr (AV == 4) {
        const int rq = lane >> 4, cc = lane & 15;
#pragma unroll
        for (int mi = 0; mi < AM; ++mi) {
#pragma unroll
            for (int ni = 0; ni < AN; ++ni)
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    stage[(4 * rq + v) * kStagePitch + ni * 16 + cc] = acc[mi][ni][v];
            emit(m0 + wm * FM * 16 + mi * 16, mi);
        }
    } else {
        // 32 x 32 accumulators: values e = 8 hh .. 8 hh + 7 are rows 16 hh + 8 (e / 4 % 2)
        // + 4 (lane / 32) + e % 4 of the 32-row slice
        const int h = lane >> 5, r32 = lane & 31;
#pragma unroll
        for (int mi = 0; mi < AM; ++mi) {
#pragma unroll
            for (int hh = 0; hh < 2; ++hh) {
#pragma unroll
                for (int ni = 0; ni < AN; ++ni)
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        stage[(8 * (e / 4) + 4 * h + (e % 4)) * kStagePitch + ni * 32 + r32] =
                            acc[mi][ni][8 * hh + e];
                emit(m0 + wm * FM * 16 + mi * 32 + hh * 16, 2 * mi + hh);
            }
        }
    }
}

// ------------------------------------------------------------------ direct-load kernel
// bf16 products whose operands are both K-contiguous rows (the forward transform).  Tiles
// go from global memory straight into LDS (16 bytes per lane per instruction, lane L's
// piece landing at base + 16 L), S stages deep, so no registers stage them and S - 1 K
// steps are in flight while one is multiplied.  An LDS row is the BK elements of K of one
// operand row (RB bytes, CPR 16-byte chunks); chunk c of row r sits in slot c ^ swz(r), so
// the 16 rows an MFMA operand read touches fall in distinct bank groups.  A lane picks the
// global chunk that belongs in its fixed LDS slot.  Rows past the end and K past the range
// read the zero buffer.  Waits are explicit (vector-memory count, then a plain barrier).
template <int BK_>
struct DlGeom {
    static constexpr int BK = BK_;
    static constexpr int RB = BK * 2;             // bytes per LDS row
    static constexpr int CPR = RB / 16;           // chunks per row
    static constexpr int RPI = 64 / CPR;          // rows per wave instruction
    static_assert(CPR == 4 || CPR == 8, "BK 32 or 64");
    __device__ __forceinline__ static int swz(int r) { return CPR == 8 ? (r & 7) : ((r >> 1) & 3); }
    __device__ __forceinline__ static int off(int r, int c) { return r * RB + ((c ^ swz(r)) << 4); }
};

__device__ __forceinline__ void lds_dma16(const char *g, char *l) {
    __builtin_amdgcn_global_load_lds((const void __attribute__((address_space(1))) *)g,
                                     (void __attribute__((address_space(3))) *)l, 16, 0, 0);
}
// wait until at most n vector-memory operations of this wave are outstanding (other
// counters untouched), then a workgroup barrier with no memory fence: the fence of
// __syncthreads would wait for every LDS load in flight
template <int N>
__device__ __forceinline__ void vm_wait_barrier() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// The forward product as a persistent kernel: one workgroup per CU walks a sequence of
// output tiles with one K-step pipeline across them, so the first steps of the next tile
// are in flight while the current tile's epilogue stores its results.  XCD x (workgroups
// b with b % 8 == x) takes a contiguous range of the tiles, its workgroups the tiles
// lo + j, lo + j + (workgroups per XCD), ..., so the two column halves of a row block are
// worked on at the same time on the same XCD and share its L2.  The MFMA operands are
// swapped (weights as the first operand), which leaves each lane 4 consecutive output
// columns of one row: the epilogue stores straight from registers, and LDS holds only the
// pipeline stages.  Steps past the last tile load zero tiles, so every step issues the
// same loads; everything lands before a workgroup exits.
template <class C, int BK, int S, class E>
__global__ __launch_bounds__(C::NT, C::NT / 256) void k_gemm_fwd(
    const char *__restrict__ a, int64_t lda, int64_t M, const char *__restrict__ b,
    int64_t ldb, int64_t N, int64_t K, const E epi, int64_t tiles_m, int64_t tiles_n) {
    using Gm = DlGeom<BK>;
    constexpr int FM = C::FM, FN = C::FN, NW = C::NT / 64;
    constexpr int A_BYTES = C::TM * Gm::RB, B_BYTES = C::TN * Gm::RB;
    constexpr int IA = C::TM / Gm::RPI / NW, IB = C::TN / Gm::RPI / NW;
    static_assert(IA * Gm::RPI * NW == C::TM && IB * Gm::RPI * NW == C::TN, "whole instructions");
    // A tiles (rows of the long operand, from HBM) are loaded AH + 1 steps ahead, B tiles
    // (weights, mostly L2 hits) one step ahead: SA = 2 + AH stages of A, two of B.  The
    // forward form takes AH = 1 (three A stages and two B stages fill the 160 KB of LDS;
    // block-0 transform 1.95 -> 1.86 ms); the input-side form measured slower with it.
    static_assert(S == 2, "two B stages");
    constexpr int AH = E::kDms ? 0 : 1;
    constexpr int SA = 2 + AH, SB = 2;
    __shared__ __attribute__((aligned(1024))) char lds[SA * A_BYTES + SB * B_BYTES];

    const int64_t T = tiles_m * tiles_n;
    const int64_t wpx = (int64_t)gridDim.x / 8;          // workgroups per XCD (grid % 8 == 0)
    const int64_t per = (T + 7) / 8;
    const int64_t x = blockIdx.x % 8, jx = blockIdx.x / 8;
    const int64_t lo = x * per + jx, hi = (x + 1) * per < T ? (x + 1) * per : T;
    const int64_t ntile = lo < hi ? (hi - lo + wpx - 1) / wpx : 0;
    const int64_t nk = (K + BK - 1) / BK;
    const int64_t nsteps = ntile * nk;

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int wm = wave / C::WN, wn = wave % C::WN;
    const char *zp = (const char *)g_zero16;
    asm volatile("" : "+v"(zp));
    const int lr = lane / Gm::CPR, ls = lane % Gm::CPR;
    int ra[IA], rb[IB], ca[IA], cb[IB];
#pragma unroll
    for (int j = 0; j < IA; ++j) {
        ra[j] = (wave * IA + j) * Gm::RPI + lr;
        ca[j] = ls ^ Gm::swz(ra[j]);
    }
#pragma unroll
    for (int j = 0; j < IB; ++j) {
        rb[j] = (wave * IB + j) * Gm::RPI + lr;
        cb[j] = ls ^ Gm::swz(rb[j]);
    }
    // Tile origins, stepped: a workgroup's tiles are lo, lo + wpx, ..., so each cursor
    // keeps (row block, column block) and adds wpx as a quotient and remainder of
    // tiles_n (a division in the loop kept its divisor in a spilled register, whose reload
    // waited for every load in flight).
    const int tn_n = (int)tiles_n;
    const int dq = (int)(wpx / tiles_n), dr = (int)(wpx - (int64_t)dq * tiles_n);
    const int tm_0 = (int)(lo / tiles_n), tn_0 = (int)(lo - (int64_t)tm_0 * tiles_n);
    auto step_tile = [&](int &tm, int &tn) {
        tn += dr;
        tm += dq;
        if (tn >= tn_n) {
            tn -= tn_n;
            ++tm;
        }
    };
    // issue cursors: with AH, A runs AH steps ahead of B
    int ia_t = 0, ia_k = 0, ga = 0, ib_t = 0, ib_k = 0, gb = 0;
    int a_tm = tm_0, a_tn = tn_0, b_tm = tm_0, b_tn = tn_0;
    auto issueA = [&]() {
        char *st = lds + (ga % SA) * A_BYTES;
        const bool live = ia_t < ntile;
        const int64_t k0 = (int64_t)ia_k * BK;
#pragma unroll
        for (int j = 0; j < IA; ++j) {
            const int64_t k = k0 + ca[j] * 8, m = (int64_t)a_tm * C::TM + ra[j];
            const char *g = (live && m < M && k < K) ? a + m * lda + k * 2 : zp;
            lds_dma16(g, st + (wave * IA + j) * 1024);
        }
        ++ga;
        if (++ia_k == nk) {
            ia_k = 0;
            ++ia_t;
            step_tile(a_tm, a_tn);
        }
    };
    auto issueB = [&]() {
        char *st = lds + SA * A_BYTES + (gb % SB) * B_BYTES;
        const bool live = ib_t < ntile;
        const int64_t k0 = (int64_t)ib_k * BK;
#pragma unroll
        for (int j = 0; j < IB; ++j) {
            const int64_t k = k0 + cb[j] * 8, n = (int64_t)b_tn * C::TN + rb[j];
            int64_t kb = k;
            if constexpr (E::kDms) kb = k < epi.kwrap ? k : k - epi.kwrap;
            const char *g = (live && n < N && k < K) ? b + n * ldb + kb * 2 : zp;
            lds_dma16(g, st + (wave * IB + j) * 1024);
        }
        ++gb;
        if (++ib_k == nk) {
            ib_k = 0;
            ++ib_t;
            step_tile(b_tm, b_tn);
        }
    };

    f32x4 acc[FM][FN];
    for (int i = 0; i < AH; ++i) issueA();
    issueB();
    issueA();
    const int r16 = lane & 15, q = lane >> 4;
    int64_t m0 = 0, n0 = 0, kk = 0;
    int c_tm = tm_0, c_tn = tn_0;
    // kDms: indptr[m] and indptr[m + 1] of each of the lane's rows in the wave's slot,
    // loaded at the tile's start and subtracted only in its epilogue (a use right after
    // the load would wait for the K step's loads issued before it)
    int32_t dlo[FM], dhi[FM];
    for (int64_t gs = 0; gs < nsteps; ++gs) {
        if (kk == 0) {
            m0 = (int64_t)c_tm * C::TM;
            n0 = (int64_t)c_tn * C::TN;
#pragma unroll
            for (int mi = 0; mi < FM; ++mi)
#pragma unroll
                for (int ni = 0; ni < FN; ++ni) acc[mi][ni] = f32x4{0.f, 0.f, 0.f, 0.f};
            if constexpr (E::kDms) {
                // the segment offsets of the lane's rows (the zero buffer where the slot has
                // no segments or the row is outside the output)
                const int64_t nw = n0 + wn * FN * 16;
                const int sl = nw < N ? (int)__umulhi((uint32_t)nw, epi.inv_din) : 0;
                const int32_t *ip = nw < N ? epi.indptr[sl] : nullptr;
#pragma unroll
                for (int mi = 0; mi < FM; ++mi) {
                    const int64_t m = m0 + wm * FM * 16 + mi * 16 + r16;
                    const bool ok = ip != nullptr && m < M;
                    const int32_t *p = ok ? ip + m : (const int32_t *)zp;
                    dlo[mi] = p[0];
                    dhi[mi] = p[1];
                }
            }
        }
        // A(gs) and B(gs) have landed; with AH, A(gs + 1) may still be in flight
        vm_wait_barrier<AH ? IA : 0>();
        issueB();
        issueA();
        const char *As = lds + (int)(gs % SA) * A_BYTES;
        const char *Bs = lds + SA * A_BYTES + (int)(gs % SB) * B_BYTES;
#pragma unroll
        for (int s = 0; s < BK / 32; ++s) {
            bf16x8 bv[FN];
#pragma unroll
            for (int i = 0; i < FN; ++i)
                bv[i] = *(const bf16x8 *)(Bs + Gm::off(wn * FN * 16 + i * 16 + r16, s * 4 + q));
#pragma unroll
            for (int mi = 0; mi < FM; ++mi) {
                const bf16x8 av = *(const bf16x8 *)(As + Gm::off(wm * FM * 16 + mi * 16 + r16, s * 4 + q));
#pragma unroll
                for (int ni = 0; ni < FN; ++ni)
                    acc[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bv[ni], av, acc[mi][ni], 0, 0, 0);
            }
        }
        if constexpr (E::kDms) {
            if (kk == nk - 1) {
                // lane: row m0 + wm FM 16 + 16 mi + (lane % 16), columns n0 + wn FN 16 +
                // 16 ni + 4 (lane / 16) .. + 3, stored as they are (16 bytes)
                const int64_t nw = n0 + wn * FN * 16;
                const int sl = nw < N ? (int)__umulhi((uint32_t)nw, epi.inv_din) : 0;
                const bool seg = nw < N && epi.indptr[sl] != nullptr;
#pragma unroll
                for (int mi = 0; mi < FM; ++mi) {
                    const int64_t m = m0 + wm * FM * 16 + mi * 16 + r16;
                    // -1 where the slot has no segments (self slot) or the row is outside
                    const int32_t deg = seg && m < M ? dhi[mi] - dlo[mi] : -1;
                    const bool zero = deg == 0;
                    const float scale = deg > 0 ? (float)deg : 1.f;
#pragma unroll
                    for (int ni = 0; ni < FN; ++ni) {
                        const int64_t n = nw + 16 * ni + 4 * q;
                        f32x4 r;
#pragma unroll
                        for (int e = 0; e < 4; ++e) r[e] = zero ? 0.f : acc[mi][ni][e] / scale;
                        if (m < M && n < N) *(f32x4 *)(epi.out + m * N + n) = r;
                    }
                }
            }
        } else if (kk == nk - 1) {
            // lane: row m0 + wm FM 16 + 16 mi + (lane % 16), columns n0 + wn FN 16 + 16 ni +
            // 4 (lane / 16) .. + 3; the wave's 64 columns are one word of the sign mask, of
            // which the lane holds bits 16 ni + 4 (lane / 16) + e, kept packed as bits
            // 16 (mi % 2) + 4 ni + e of word mi / 2 while the results are stored
            // The packed bf16 results of fragments 2 p and 2 p + 1 are exchanged between the
            // lane rows (16 lanes) 0 and 1, and 2 and 3, of the wave: lane row q then holds
            // 8 consecutive columns, 16 (q % 2) + 8 (q / 2) .. of the pair's 32, and the 4
            // lanes of an output row store 64 contiguous bytes.
            static_assert(FM % 2 == 0 && FN == 4, "packed sign bits");
            uint32_t pk[FM / 2];
#pragma unroll
            for (int i = 0; i < FM / 2; ++i) pk[i] = 0u;
            const int cofs = 16 * (q & 1) + 8 * (q >> 1);
#pragma unroll
            for (int p = 0; p < FN / 2; ++p) {
                const int64_t na = n0 + wn * FN * 16 + p * 32 + 4 * q, nb = na + 16;
                const int64_t ns = n0 + wn * FN * 16 + p * 32 + cofs;
                float ba[4], bb[4];
                epi.load_bias4(na, ba);
                epi.load_bias4(nb, bb);
#pragma unroll
                for (int mi = 0; mi < FM; ++mi) {
                    const int64_t m = m0 + wm * FM * 16 + mi * 16 + r16;
                    uint32_t a0, a1, b0, b1;
                    const uint32_t bits = epi.pack4(m, na, acc[mi][2 * p], ba, a0, a1) |
                                          (epi.pack4(m, nb, acc[mi][2 * p + 1], bb, b0, b1) << 4);
                    pk[mi / 2] |= bits << (16 * (mi % 2) + 8 * p);
                    // odd lane rows of the first operand trade places with even lane rows
                    // of the second
                    const auto s0 = __builtin_amdgcn_permlane16_swap(a0, b0, false, false);
                    const auto s1 = __builtin_amdgcn_permlane16_swap(a1, b1, false, false);
                    epi.store8(m, ns, make_uint4(s0[0], s1[0], s0[1], s1[1]));
                }
            }
            if (epi.mask.w != nullptr) {
#pragma unroll
                for (int mi = 0; mi < FM; ++mi) {
                    const uint32_t c16 = pk[mi / 2] >> (16 * (mi % 2));
                    uint64_t bits = 0u;
#pragma unroll
                    for (int ni = 0; ni < FN; ++ni)
                        bits |= (uint64_t)((c16 >> (4 * ni)) & 0xFu) << (16 * ni + 4 * q);
                    epi.mask.put(m0 + wm * FM * 16 + mi * 16 + r16, epi.M, n0 + wn * FN * 16,
                                 epi.N, bits, 16, 4, q == 0);
                }
            }
        }
        if (++kk == nk) {
            kk = 0;
            step_tile(c_tm, c_tn);
        }
    }
    __builtin_amdgcn_s_waitcnt(0);   // padded steps' loads landed before the workgroup exits
}

// ------------------------------------------------------------------ weight side
// dW partial of one split: out[c][o] = sum over the split's rows m of Mcat[m][c] dY[m][o].
// The reduction runs over rows of both operands, so both tiles sit in LDS as loaded (row
// = one m, TM or TN consecutive columns) and the MFMA fragments, which want 8 consecutive
// m per lane, are read down the columns: the bf16 Mcat tile with the LDS transpose read (a
// 16-lane group hands in sixteen 8-byte pieces, four columns of one row each, and every
// lane gets one column of four rows), the fp32 dY tile one row at a time.  Mcat tile:
// 512-byte LDS rows, 16-byte chunk c of row r at slot c ^ SWZ (r & 3).  A transpose read
// of 32 lanes takes 64 bytes of each of four rows; with SWZ = 4 the four rows fall in
// distinct 64-byte bank windows.
template <int BK_, int COLS>
struct DwGeom {
    static constexpr int BK = BK_;                 // rows (m) per K step
    static constexpr int RB = COLS * 2;            // bytes per LDS row (COLS bf16)
    static constexpr int CPR = RB / 16;            // 16-byte chunks per row
    static constexpr int RPI = 1024 / RB;          // rows per wave load instruction
    static constexpr int TILE = BK * RB;
    static constexpr int SWZ = 4;
    static_assert(CPR >= 4 * SWZ, "the slot swizzle stays within a row");
    __device__ __forceinline__ static int slot(int r, int c) { return c ^ ((r & 3) * SWZ); }
};
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
// LDS transpose read from inline assembly.  Before the builtin form of this read the
// compiler waits for every direct-to-LDS load in flight (vmcnt(0)), since it cannot tell
// which LDS bytes they write; in a pipelined loop that stalls each step on the loads just
// issued for the steps ahead.  The compiler does not track these reads: lds_reads_done must
// run on the fragment before it is used.
__device__ __forceinline__ s16x4 lds_tr16_untracked(const char *p) {
    s16x4 v;
    const uint32_t a = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char *)p;
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(v) : "v"(a));
    return v;
}
// Fragment of 16 columns [col0, col0 + 16) x rows [row0, row0 + 8) of a DwGeom tile for
// lane j of a 16-lane group.
template <class Gm>
__device__ __forceinline__ bf16x8 dw_frag_untracked(const char *tile, int row0, int col0, int j) {
    const int col = col0 + 4 * (j & 3);
    const int r0 = row0 + (j >> 2), r1 = r0 + 4;
    const int c = col >> 3, byte = (col & 7) * 2;
    const s16x4 lo = lds_tr16_untracked(tile + r0 * Gm::RB + (Gm::slot(r0, c) << 4) + byte);
    const s16x4 hi = lds_tr16_untracked(tile + r1 * Gm::RB + (Gm::slot(r1, c) << 4) + byte);
    const s16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(bf16x8, v);
}
// Waits until every LDS read of the wave has returned; `v` depends on the wait, so no use
// of it is scheduled before it.
__device__ __forceinline__ void lds_reads_done(bf16x8 &v) {
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(v));
}

// fp32 dY tile of k_gemm_dw: BK rows of COLS floats as loaded, 16-byte chunk c of row r in
// slot c ^ 8 ((r / 8) % 2).  A fragment read takes rows r and r + 8 of the same 32 columns
// in its two half-waves; the slot flip puts them 128 bytes apart, on disjoint banks.
template <int BK_, int COLS>
struct DwRawGeom {
    static constexpr int BK = BK_;
    static constexpr int RB = COLS * 4;            // bytes per LDS row
    static constexpr int CPR = RB / 16;            // 16-byte chunks per row
    static constexpr int RPI = 1024 / RB;          // rows per wave load instruction
    static constexpr int TILE = BK * RB;
    static_assert(CPR >= 16 && RPI >= 1, "the slot flip needs 16 chunks per row");
    __device__ __forceinline__ static int slot(int r, int c) { return c ^ (((r >> 3) & 1) << 3); }
};
// B fragment of a 32 x 32 x 16 product from an fp32 tile: column `col`, rows row0 .. + 7
// (row0 a multiple of 8), split into hi = bf16(x) and lo = bf16(x - hi) for the two
// products that carry dY's 16 significant bits.
template <class Gr>
__device__ __forceinline__ void dw_raw_frag(const char *tile, int row0, int col, bf16x8 &hi,
                                            bf16x8 &lo) {
    const char *p = tile + row0 * Gr::RB + (Gr::slot(row0, col >> 2) << 4) + (col & 3) * 4;
    float x[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = *(const float *)(p + i * Gr::RB);
    u32x4 h, l;
    h.x = pack_bf16x2(x[0], x[1]); h.y = pack_bf16x2(x[2], x[3]);
    h.z = pack_bf16x2(x[4], x[5]); h.w = pack_bf16x2(x[6], x[7]);
    l.x = pack_bf16x2(x[0] - bf16_lo(h.x), x[1] - bf16_hi(h.x));
    l.y = pack_bf16x2(x[2] - bf16_lo(h.y), x[3] - bf16_hi(h.y));
    l.z = pack_bf16x2(x[4] - bf16_lo(h.z), x[5] - bf16_hi(h.z));
    l.w = pack_bf16x2(x[6] - bf16_lo(h.w), x[7] - bf16_hi(h.w));
    hi = __builtin_bit_cast(bf16x8, h);
    lo = __builtin_bit_cast(bf16x8, l);
}

// The weight-side product with both operands loaded straight into LDS (no register
// staging), S stages deep: the loads of the next S - 1 steps are in flight while a step is
// multiplied.  dY stays fp32 in LDS and each fragment is split into its hi and lo bf16
// parts in registers.  32 x 32 x 16 MFMA tiles (see the input-side core): the 16-lane
// group g of a fragment read takes columns 16 (g % 2) .. of the 32 and rows 8 (g / 2) ..
// of the 16-row K sub-step.
// HILO: dY rows come in the hi/lo form (d_out bf16 high parts, then d_out low parts): the
// hi and lo tiles are loaded like the Mcat tile and read by the same transpose reads, with
// no split in registers.
template <class C, int BK, int S, int MINW, bool HILO>
__global__ __launch_bounds__(C::NT, MINW) void k_gemm_dw(const char *__restrict__ mcat, int64_t M,
                                                    int64_t Kcat, const float *__restrict__ dy,
                                                    int64_t d_out, int64_t tiles_m,
                                                    int64_t tiles_n, int64_t per,
                                                    const EpiPartial epi) {
    using Ga = DwGeom<BK, C::TM>;
    using Gb = DwRawGeom<BK, C::TN>;
    using Gh = DwGeom<BK, C::TN>;                  // HILO: each of the hi and lo tiles
    constexpr int FM = C::FM, FN = C::FN, NW = C::NT / 64;
    constexpr int B_TILE = HILO ? 2 * Gh::TILE : Gb::TILE;
    constexpr int STAGE = Ga::TILE + B_TILE;
    constexpr int IA = BK / Ga::RPI / NW;
    constexpr int IB = HILO ? BK / Gh::RPI / NW : BK / Gb::RPI / NW;   // per B tile
    static_assert(IA * Ga::RPI * NW == BK, "whole instructions");
    static_assert(HILO ? IB * Gh::RPI * NW == BK : IB * Gb::RPI * NW == BK, "whole instructions");
    constexpr int LPS = IA + (HILO ? 2 : 1) * IB;
    static_assert(S >= 2 && (S - 2) * LPS < 64, "vmcnt range");
    __shared__ __attribute__((aligned(1024))) char lds[S * STAGE];
    static_assert(S * STAGE >= NW * 16 * kStagePitch * 4, "epilogue staging space");

    const int64_t logical = xcd_major_id(blockIdx.x, (int64_t)gridDim.x);
    const int64_t tiles = tiles_m * tiles_n;
    const int64_t split = logical / tiles;
    const int64_t t = logical - split * tiles;
    const int64_t tm = t / tiles_n, tn = t - tm * tiles_n;
    const int64_t c0 = tm * C::TM, o0 = tn * C::TN;
    const int64_t kb = split * per;
    const int64_t ke = kb + per < M ? kb + per : M;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int wm = wave / C::WN, wn = wave % C::WN;
    const char *zp = (const char *)g_zero16;
    asm volatile("" : "+v"(zp));

    // instruction j of this wave: A rows RPI (IA wave + j) .., B rows RPI (IB wave + j) ..;
    // lane L fills slot L % CPR of row L / CPR with the chunk that belongs there
    const int64_t nk = ke > kb ? (ke - kb + BK - 1) / BK : 0;
    auto issue = [&](int64_t step) {
        char *st = lds + (int)(step % S) * STAGE;
        const int64_t m0 = kb + step * BK;
#pragma unroll
        for (int j = 0; j < IA; ++j) {
            const int r = (wave * IA + j) * Ga::RPI + lane / Ga::CPR;
            const int64_t m = m0 + r, col = c0 + Ga::slot(r, lane % Ga::CPR) * 8;
            const char *g = (m < ke && col < Kcat) ? mcat + m * Kcat * 2 + col * 2 : zp;
            lds_dma16(g, st + (wave * IA + j) * 1024);
        }
        if constexpr (HILO) {
#pragma unroll
            for (int j = 0; j < IB; ++j) {
                const int r = (wave * IB + j) * Gh::RPI + lane / Gh::CPR;
                const int64_t m = m0 + r, col = o0 + Gh::slot(r, lane % Gh::CPR) * 8;
                const bool ok = m < ke && col < d_out;
                const char *row = (const char *)dy + m * d_out * 4 + col * 2;
                lds_dma16(ok ? row : zp, st + Ga::TILE + (wave * IB + j) * 1024);
                lds_dma16(ok ? row + d_out * 2 : zp, st + Ga::TILE + Gh::TILE + (wave * IB + j) * 1024);
            }
        } else {
#pragma unroll
            for (int j = 0; j < IB; ++j) {
                const int r = (wave * IB + j) * Gb::RPI + lane / Gb::CPR;
                const int64_t m = m0 + r, col = o0 + Gb::slot(r, lane % Gb::CPR) * 4;
                const char *g = (m < ke && col < d_out) ? (const char *)(dy + m * d_out + col) : zp;
                lds_dma16(g, st + Ga::TILE + (wave * IB + j) * 1024);
            }
        }
    };

    constexpr int AM = FM / 2, AN = FN / 2;
    f32x16 acc[AM][AN];
#pragma unroll
    for (int mi = 0; mi < AM; ++mi)
#pragma unroll
        for (int ni = 0; ni < AN; ++ni)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[mi][ni][e] = 0.f;

    for (int st = 0; st < S - 1; ++st)
        if (st < nk) issue(st);
    const int j16 = lane & 15, q = lane >> 4;
    const int gc = 16 * (q & 1), gr = 8 * (q >> 1);
    for (int64_t it = 0; it < nk; ++it) {
        // this step's tiles have landed in every wave, and every wave is done with the stage
        // the next issue overwrites (the loads of later steps stay in flight)
        if (it + S - 2 < nk)
            vm_wait_barrier<(S - 2) * LPS>();
        else
            vm_wait_barrier<0>();
        if (it + S - 1 < nk) issue(it + S - 1);
        const char *As = lds + (int)(it % S) * STAGE;
        const char *Bs = As + Ga::TILE;
#pragma unroll
        for (int s = 0; s < BK / 16; ++s) {
            bf16x8 bh[AN], bl[AN];
            if constexpr (HILO) {
#pragma unroll
                for (int ni = 0; ni < AN; ++ni) {
                    bh[ni] = dw_frag_untracked<Gh>(Bs, s * 16 + gr, wn * FN * 16 + ni * 32 + gc, j16);
                    bl[ni] = dw_frag_untracked<Gh>(Bs + Gh::TILE, s * 16 + gr,
                                                   wn * FN * 16 + ni * 32 + gc, j16);
                }
            } else {
#pragma unroll
                for (int ni = 0; ni < AN; ++ni)
                    dw_raw_frag<Gb>(Bs, s * 16 + 8 * (lane >> 5),
                                    wn * FN * 16 + ni * 32 + (lane & 31), bh[ni], bl[ni]);
            }
            bf16x8 av[AM];
#pragma unroll
            for (int mi = 0; mi < AM; ++mi)
                av[mi] = dw_frag_untracked<Ga>(As, s * 16 + gr, wm * FM * 16 + mi * 32 + gc, j16);
#pragma unroll
            for (int mi = 0; mi < AM; ++mi) lds_reads_done(av[mi]);
            if constexpr (HILO) {
#pragma unroll
                for (int ni = 0; ni < AN; ++ni) {
                    lds_reads_done(bh[ni]);
                    lds_reads_done(bl[ni]);
                }
            }
#pragma unroll
            for (int mi = 0; mi < AM; ++mi) {
#pragma unroll
                for (int ni = 0; ni < AN; ++ni) {
                    acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[mi], bh[ni], acc[mi][ni], 0, 0, 0);
                    acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[mi], bl[ni], acc[mi][ni], 0, 0, 0);
                }
            }
        }
    }
    // every load has landed (the last steps wait for all) and every wave is done with the
    // stages before the epilogue reuses them
    __syncthreads();

    // lane L: row L % 16, columns 4 (L / 16) + 16 q .. + 3 of the staged 16 x 64 slice
    float *stage = (float *)lds + wave * 16 * kStagePitch;
    const int er = lane & 15, ec = 4 * (lane >> 4);
    auto emit = [&](int64_t row) {
        __builtin_amdgcn_wave_barrier();
        float vals[16];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float4 x = *(const float4 *)(stage + er * kStagePitch + ec + 16 * q);
            vals[4 * q] = x.x; vals[4 * q + 1] = x.y; vals[4 * q + 2] = x.z; vals[4 * q + 3] = x.w;
        }
        __builtin_amdgcn_wave_barrier();
        epi(row + er, o0 + wn * FN * 16 + ec, vals, split);
    };
    const int h = lane >> 5, r32 = lane & 31;
#pragma unroll
    for (int mi = 0; mi < AM; ++mi) {
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
#pragma unroll
            for (int ni = 0; ni < AN; ++ni)
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    stage[(8 * (e / 4) + 4 * h + (e % 4)) * kStagePitch + ni * 32 + r32] =
                        acc[mi][ni][8 * hh + e];
            emit(c0 + wm * FM * 16 + mi * 32 + hh * 16);
        }
    }
}

// ------------------------------------------------------------------ input side, streamed
// dMs with at most 128 output columns (one slot of d_in <= 128, or a few narrower ones),
// d_out a multiple of 256 up to 512: K (= d_out) is split over the 8 waves of a workgroup.
// Each wave keeps its K slice of the weights of all 128 columns in registers and the
// workgroup walks blocks of 16 dY rows: every wave reads its slice of the 16 rows straight
// into registers (so the workgroup reads the 16 rows whole, at once), splits each fp32
// value into its hi and lo bf16 parts, multiplies both against its weights, and leaves its
// partial products in LDS; the waves then sum the 8 partials of 2 rows each, divide by the
// degree and store whole rows.  dY is read exactly once, in whole rows; the register-
// staged kernel reads it in 256-byte row pieces, once per column tile.
// v_mfma_f32_16x16x32_bf16 with the weights as the first operand: lane l supplies weight
// row 16 t + l % 16 and dY row m0 + l % 16, K group q = l / 16, and holds output row
// m0 + l % 16, columns 16 t + 4 q .. + 3.  Wave w's slice is K values [KW w, KW w + KW),
// KW = d_out / 8; MFMA step s gives group q the 8 values at KW w + 32 s + 8 q (S = KW / 32
// steps), so the 4 groups of a step read 128 contiguous bytes of each row and every load
// instruction stays within one 128-byte window per row.  Partial row r, 4-column
// piece c sits at slot c ^ r of the row's 512 bytes, so the 16 rows a partial store
// writes and the 32 pieces a summing read takes fall in distinct banks.  Two LDS buffers
// alternate between row blocks (one barrier per block); each wave's register copies of
// the next NB blocks are in flight while it multiplies one.
constexpr int kDmsStreamCols = 128;                  // output columns
constexpr int kDmsStreamWaves = 8;
constexpr int kDmsStreamPart = 16 * kDmsStreamCols * 4;   // one wave's partial block
struct DmsStream {
    const void *w[kMaxSlots];          // W_slot [d_in x d_out] bf16
    const int32_t *indptr[kMaxSlots];  // relation slot: degrees; NULL: the self slot
    float *out;                        // [M x N]
    int32_t N;
    int32_t d_in;
};
// HILO: dY rows in the hi/lo form; the loads fetch the bf16 parts as they are.
template <int S, int NB, bool HILO>
__global__ __launch_bounds__(kDmsStreamWaves * 64, 1) void k_dms_stream(
    const float *__restrict__ dy, int64_t M, const DmsStream p) {
    constexpr int KW = 32 * S;                       // K values per wave
    constexpr int D = KW * kDmsStreamWaves;          // d_out
    __shared__ __attribute__((aligned(16))) char lds[2 * kDmsStreamWaves * kDmsStreamPart];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int r16 = lane & 15, q = lane >> 4;
    // weight fragments: tile t, step s: row n = 16 t + r16 (W_{n / d_in} row n % d_in, zero
    // past N), K values KW wave + 32 s + 8 q ..
    bf16x8 wf[8][S];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
        const int n = t * 16 + r16;
        const int sl = n < p.N ? n / p.d_in : 0;
        const char *wr = (const char *)p.w[sl] + (int64_t)(n < p.N ? n - sl * p.d_in : 0) * D * 2 +
                         (wave * KW + q * 8) * 2;
#pragma unroll
        for (int s = 0; s < S; ++s) {
            u32x4 v = *(const u32x4 *)(wr + s * 64);
            if (n >= p.N) v = u32x4{0u, 0u, 0u, 0u};
            wf[t][s] = __builtin_bit_cast(bf16x8, v);
        }
    }
    const int64_t nblocks = (M + 15) / 16;
    const int64_t P = gridDim.x;
    const int nmine = blockIdx.x < nblocks ? (int)((nblocks - blockIdx.x + P - 1) / P) : 0;
    const float *zp = (const float *)g_zero16;
    // summing role: row rr of the block, columns 4 cq .. + 3 (slot cq 4 / d_in)
    const int rr = 2 * wave + (lane >> 5), cq = lane & 31;
    const bool col_ok = cq * 4 < p.N;
    const int32_t *ipc = col_ok ? p.indptr[cq * 4 / p.d_in] : nullptr;
    // block bi of this workgroup: rows 16 (blockIdx.x + bi P) ..; the lane's slice of its
    // row, and indptr[m], indptr[m + 1] of its summing row and slot (the self slot and
    // rows past M read the zero buffer).  Loads are issued unconditionally (blocks past the
    // last read the zero buffer), so every path has the same loads in flight.
    struct Blk {
        f32x4 v[2 * S];
        int32_t i0, i1;
    };
    auto load = [&](int bi, Blk &b) {
        const bool live = bi < nmine;
        const int64_t m0 = ((int64_t)blockIdx.x + (int64_t)(live ? bi : 0) * P) * 16;
        const int64_t m = m0 + r16;
        const bool ok = live && m < M;
        if constexpr (HILO) {
            // step s: the high parts of the 8 values in v[2 s], the low parts in v[2 s + 1]
            const char *src = ok ? (const char *)dy + m * D * 4 + (wave * KW + q * 8) * 2
                                 : (const char *)zp;
            const int st = ok ? 1 : 0;
#pragma unroll
            for (int i = 0; i < 2 * S; ++i)
                b.v[i] = *(const f32x4 *)(src + (64 * (i / 2) + D * 2 * (i % 2)) * st);
        } else {
            const float *src = ok ? dy + m * D + wave * KW + q * 8 : zp;
            const int st = ok ? 1 : 0;
#pragma unroll
            for (int i = 0; i < 2 * S; ++i)
                b.v[i] = *(const f32x4 *)(src + (32 * (i / 2) + 4 * (i % 2)) * st);
        }
        const int64_t mr = m0 + rr;
        const int32_t *d = (live && ipc != nullptr && mr < M) ? ipc + mr : (const int32_t *)zp;
        b.i0 = d[0];
        b.i1 = d[1];
    };
    Blk bufs[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) load(b, bufs[b]);
    for (int bi0 = 0; bi0 < nmine; bi0 += NB) {
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            const int bi = bi0 + b;
            if (bi >= nmine) break;
            f32x4 acc[8];
#pragma unroll
            for (int t = 0; t < 8; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < S; ++s) {
                const f32x4 a = bufs[b].v[2 * s], c = bufs[b].v[2 * s + 1];
                u32x4 hv, lv;
                if constexpr (HILO) {
                    hv = __builtin_bit_cast(u32x4, a);
                    lv = __builtin_bit_cast(u32x4, c);
                } else {
                    hv.x = pack_bf16x2(a.x, a.y);
                    hv.y = pack_bf16x2(a.z, a.w);
                    hv.z = pack_bf16x2(c.x, c.y);
                    hv.w = pack_bf16x2(c.z, c.w);
                    lv.x = pack_bf16x2(a.x - bf16_lo(hv.x), a.y - bf16_hi(hv.x));
                    lv.y = pack_bf16x2(a.z - bf16_lo(hv.y), a.w - bf16_hi(hv.y));
                    lv.z = pack_bf16x2(c.x - bf16_lo(hv.z), c.y - bf16_hi(hv.z));
                    lv.w = pack_bf16x2(c.z - bf16_lo(hv.w), c.w - bf16_hi(hv.w));
                }
                const bf16x8 bh = __builtin_bit_cast(bf16x8, hv), bl = __builtin_bit_cast(bf16x8, lv);
#pragma unroll
                for (int t = 0; t < 8; ++t) {
                    acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[t][s], bh, acc[t], 0, 0, 0);
                    acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[t][s], bl, acc[t], 0, 0, 0);
                }
            }
            const int32_t i0 = bufs[b].i0, i1 = bufs[b].i1;
            char *part = lds + (bi & 1) * (kDmsStreamWaves * kDmsStreamPart);
            char *mine = part + wave * kDmsStreamPart;
#pragma unroll
            for (int t = 0; t < 8; ++t)
                *(f32x4 *)(mine + r16 * 512 + (((4 * t + q) ^ r16) * 16)) = acc[t];
            load(bi + NB, bufs[b]);
            // every wave's partials of this block are in LDS; the buffer written next was
            // last read before this barrier
            __syncthreads();
            f32x4 sum = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int w = 0; w < kDmsStreamWaves; ++w)
                sum += *(const f32x4 *)(part + w * kDmsStreamPart + rr * 512 + ((cq ^ rr) * 16));
            const int64_t m = ((int64_t)blockIdx.x + (int64_t)bi * P) * 16 + rr;
            if (col_ok && m < M) {
                const int32_t deg = i1 - i0;
                const bool zero = ipc != nullptr && deg == 0;
                const float scale = ipc != nullptr && deg > 0 ? (float)deg : 1.f;
                f32x4 r;
                r.x = zero ? 0.f : sum.x / scale;
                r.y = zero ? 0.f : sum.y / scale;
                r.z = zero ? 0.f : sum.z / scale;
                r.w = zero ? 0.f : sum.w / scale;
                *(f32x4 *)(p.out + m * p.N + cq * 4) = r;
            }
        }
    }
}

template <class C, class Mma, class LA, class LB, class Epi, int STAGES, int R>
hipError_t launch_gemm(const LA &la, const LB &lb, const Epi &epi, int64_t M, int64_t N,
                       int64_t K, int64_t splits, int64_t k_per_split, hipStream_t s) {
    const int64_t tiles_m = cdiv(M, C::TM), tiles_n = cdiv(N, C::TN);
    if (tiles_m == 0 || tiles_n == 0 || splits == 0) return hipSuccess;
    hipLaunchKernelGGL((k_gemm<C, Mma, LA, LB, Epi, STAGES, R>),
                       dim3((unsigned)(tiles_m * tiles_n * splits)), dim3(C::NT), 0, s, la, lb,
                       epi, K, tiles_m, tiles_n, k_per_split);
    return hipGetLastError();
}

// Split of the weight-side reduction over rows: at most `target` workgroups in total (one
// wave of them where a workgroup fills a CU, so no partial second wave trails), each split
// a whole number of K steps and at least 8 of them.
template <class C>
void dw_split(int64_t M, int Kcat, int d_out, int bk, int64_t target, int64_t *splits,
              int64_t *per) {
    const int64_t tiles = cdiv(Kcat, C::TM) * cdiv(d_out, C::TN);
    int64_t want = target / tiles;
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

// The input side's weight rows stacked as one bf16 [N x d_out] matrix (row s d_in + c =
// row c of W_s), in 16-byte chunks (cpr per row).
__global__ __launch_bounds__(kThreads) void k_pack_rows(SlotRows sr, int64_t chunks, int cpr,
                                                        u32x4 *out) {
    for (int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x; e < chunks;
         e += (int64_t)gridDim.x * kThreads) {
        const int64_t n = e / cpr, ch = e - n * cpr;
        out[e] = *(const u32x4 *)(sr.row(n) + ch * 16);
    }
}

constexpr int kDwBK = 32;   // rows per K step of the bf16 weight-side kernel
constexpr int kDwStages = 2;   // LDS stages of k_gemm_dw (three measured 2 % slower)
// workgroups of one weight-side product: the bf16 kernel holds a CU by itself (96 KB of
// LDS), so one per CU of the 256 (a 2.02-wave grid left most CUs idle behind its last
// few workgroups); the fp32 kernel fits two per CU
constexpr int64_t kDwTargetBf16 = 256;
constexpr int64_t kDwTargetF32 = 512;
// compute units of the current device (cached per device)
int64_t device_cus() {
    static int64_t cache[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    if (cache[dev] == 0) {
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            cus <= 0)
            cus = 256;
        cache[dev] = cus;
    }
    return cache[dev];
}
// forward transform: K step (elements) and LDS stages of k_gemm_fwd
constexpr int kFwdBK = 64;
constexpr int kFwdStages = 2;
// input side: one LDS stage (two workgroups share a CU), one register stage
constexpr int kDmsStages = 1;
constexpr int kDmsRegStages = 1;

}  // namespace

hipError_t gemm_forward(rgcn_dtype dt, const void *a, int64_t M, int N, int K,
                        const void *wcat_t, const void *bias, int relu, void *y,
                        uint64_t *mask, hipStream_t s) {
    const ReluMask rm{mask, (int64_t)(N + 63) / 64};
    if (dt == RGCN_BF16) {
        using C = CfgFwd;
        const int64_t tiles_m = cdiv(M, C::TM), tiles_n = cdiv(N, C::TN);
        if (tiles_m == 0 || tiles_n == 0) return hipSuccess;
        // one workgroup per CU (a multiple of 8 so every XCD has the same count)
        int64_t P = tiles_m * tiles_n;
        const int64_t cus = device_cus();
        if (P > cus) P = cus;
        P = (P + 7) / 8 * 8;
        hipLaunchKernelGGL((k_gemm_fwd<C, kFwdBK, kFwdStages, EpiForwardBf16>), dim3((unsigned)P),
                           dim3(C::NT), 0, s, (const char *)a, (int64_t)K * 2, M,
                           (const char *)wcat_t, (int64_t)K * 2, (int64_t)N, (int64_t)K,
                           EpiForwardBf16{y, bias, M, N, relu, rm}, tiles_m, tiles_n);
        return hipGetLastError();
    }
    using C = CfgF32;
    using TL = TileF32;
    LoadRows<TL, C::NT, PlainRows> la{PlainRows{(const char *)a, (int64_t)K * 4, M}, (int64_t)K * 4};
    LoadRows<TL, C::NT, PlainRows> lb{PlainRows{(const char *)wcat_t, (int64_t)K * 4, N},
                                      (int64_t)K * 4};
    return launch_gemm<C, MmaF32<C::FM, C::FN>, decltype(la), decltype(lb), EpiForward<false>, 2, 2>(
        la, lb, EpiForward<false>{y, bias, M, N, relu, rm}, M, N, K, 1, K, s);
}

hipError_t gemm_dms(rgcn_dtype dt, const float *dy, bool dy_hilo, int64_t M, int d_out,
                    int d_in, const DmsSlots &slots, float *dms, void *wpack, hipStream_t s) {
    const int es = dt == RGCN_BF16 ? 2 : 4;
    const int64_t N = (int64_t)slots.count * d_in;
    SlotRows sr;
    for (int i = 0; i < kMaxSlots; ++i) sr.w[i] = i < slots.count ? slots.w[i] : nullptr;
    sr.d_in = d_in;
    sr.es_dout = d_out * es;
    sr.rows = N;
    if (dt == RGCN_BF16 && dy_hilo && wpack != nullptr && d_in % 64 == 0 && N > kDmsStreamCols) {
        // the persistent product over the hi/lo rows (K = 2 d_out) and the packed weight rows
        using C = CfgFwd;
        const int64_t tiles_m = cdiv(M, C::TM), tiles_n = cdiv(N, C::TN);
        if (tiles_m == 0) return hipSuccess;
        const int64_t chunks = N * (d_out / 8);
        const int64_t pb = cdiv(chunks, kThreads) < 4096 ? cdiv(chunks, kThreads) : 4096;
        hipLaunchKernelGGL(k_pack_rows, dim3((unsigned)pb), dim3(kThreads), 0, s, sr, chunks,
                           d_out / 8, (u32x4 *)wpack);
        RGCN_HIP_TRY(hipGetLastError());
        EpiDmsFwd e{};
        e.out = dms;
        e.M = M;
        e.N = (int32_t)N;
        e.kwrap = d_out;
        e.inv_din = (uint32_t)(((1ull << 32) + (uint64_t)d_in - 1) / (uint64_t)d_in);
        for (int i = 0; i < kMaxSlots; ++i) e.indptr[i] = i < slots.count ? slots.indptr[i] : nullptr;
        int64_t P = tiles_m * tiles_n;
        const int64_t cus = device_cus();
        if (P > cus) P = cus;
        P = (P + 7) / 8 * 8;
        hipLaunchKernelGGL((k_gemm_fwd<C, kFwdBK, kFwdStages, EpiDmsFwd>), dim3((unsigned)P),
                           dim3(C::NT), 0, s, (const char *)dy, (int64_t)d_out * 4, M,
                           (const char *)wpack, (int64_t)d_out * 2, N, (int64_t)d_out * 2, e,
                           tiles_m, tiles_n);
        return hipGetLastError();
    }
    EpiDms epi;
    epi.out = dms;
    epi.M = M;
    epi.N = (int32_t)N;
    epi.d_in = d_in;
    for (int i = 0; i < kMaxSlots; ++i) epi.indptr[i] = i < slots.count ? slots.indptr[i] : nullptr;
    PlainRows pa{(const char *)dy, (int64_t)d_out * 4, M};
    if (dt == RGCN_BF16 && N <= kDmsStreamCols && d_in % 16 == 0 &&
        (d_out == 256 || d_out == 512)) {
        if (M == 0) return hipSuccess;
        DmsStream ps{};
        for (int i = 0; i < kMaxSlots; ++i) {
            ps.w[i] = sr.w[i];
            ps.indptr[i] = epi.indptr[i];
        }
        ps.out = dms;
        ps.N = (int32_t)N;
        ps.d_in = d_in;
        // one workgroup per CU (128 KB of LDS), no more than there are 16-row blocks
        int64_t P = cdiv(M, 16);
        const int64_t cus = device_cus();
        if (P > cus) P = cus;
        // register blocks in flight per wave: as many as fit beside the weights
#define RGCN_DMS_STREAM(S_, NB_)                                                             \
    do {                                                                                     \
        if (dy_hilo)                                                                         \
            hipLaunchKernelGGL((k_dms_stream<S_, NB_, true>), dim3((unsigned)P),             \
                               dim3(kDmsStreamWaves * 64), 0, s, dy, M, ps);                 \
        else                                                                                 \
            hipLaunchKernelGGL((k_dms_stream<S_, NB_, false>), dim3((unsigned)P),            \
                               dim3(kDmsStreamWaves * 64), 0, s, dy, M, ps);                 \
    } while (0)
        if (d_out == 512)
            RGCN_DMS_STREAM(2, 5);
        else
            RGCN_DMS_STREAM(1, 8);
#undef RGCN_DMS_STREAM
        return hipGetLastError();
    }
    if (dt == RGCN_BF16) {
        // dY enters as hi + lo bf16 tiles from one read of each fp32 row; each weight
        // fragment meets both
        using C = CfgDms;
        using TL = TileBf16<C>;
        LoadRows<TL, C::NT, SlotRows> lb{sr, (int64_t)d_out * 2};
        using Core = MmaBf16SplitA32<TL, C::FM, C::FN>;
        if (dy_hilo) {
            LoadRowsHiLoBf16<TL, C::NT, 2 * TL::BYTES> la{pa, d_out};
            return launch_gemm<C, Core, decltype(la), decltype(lb), EpiDms, kDmsStages,
                               kDmsRegStages>(la, lb, epi, M, N, d_out, 1, d_out, s);
        }
        LoadRowsF32HiLo<TL, C::NT, 2 * TL::BYTES> la{pa, d_out};
        return launch_gemm<C, Core, decltype(la), decltype(lb), EpiDms, kDmsStages,
                           kDmsRegStages>(la, lb, epi, M, N, d_out, 1, d_out, s);
    }
    using C = CfgF32;
    using TL = TileF32;
    LoadRows<TL, C::NT, PlainRows> la{pa, (int64_t)d_out * 4};
    LoadRows<TL, C::NT, SlotRows> lb{sr, (int64_t)d_out * 4};
    return launch_gemm<C, MmaF32<C::FM, C::FN>, decltype(la), decltype(lb), EpiDms, 2, 2>(
        la, lb, epi, M, N, d_out, 1, d_out, s);
}

size_t gemm_dw_partial_bytes(int64_t M, int Kcat, int d_out) {
    int64_t sp16, p16, sp64, p64;
    dw_split<CfgF32>(M, Kcat, d_out, TileF32::BK, kDwTargetF32, &sp16, &p16);
    dw_split<CfgDw>(M, Kcat, d_out, kDwBK, kDwTargetBf16, &sp64, &p64);
    const int64_t sp = sp16 > sp64 ? sp16 : sp64;
    return (size_t)(sp > 0 ? sp : 1) * Kcat * d_out * 4 + 256;
}

hipError_t gemm_dw(rgcn_dtype dt, const void *mcat, int64_t M, int Kcat, int d_in,
                   const float *dy, bool dy_hilo, int d_out, const DwOut &out, float *partial,
                   hipStream_t s) {
    const bool bf = dt == RGCN_BF16;
    int64_t splits, per;
    if (bf)
        dw_split<CfgDw>(M, Kcat, d_out, kDwBK, kDwTargetBf16, &splits, &per);
    else
        dw_split<CfgF32>(M, Kcat, d_out, TileF32::BK, kDwTargetF32, &splits, &per);
    if (splits == 0) {  // no rows: every requested gradient is zero
        hipLaunchKernelGGL(k_zero_outputs, dim3((unsigned)cdiv((int64_t)d_in * d_out, kThreads),
                           (unsigned)out.count), dim3(kThreads), 0, s, out, d_in, d_out);
        return hipGetLastError();
    }
    EpiPartial epi{partial, Kcat, d_out};
    if (bf) {
        using C = CfgDw;
        const int64_t tiles_m = cdiv(Kcat, C::TM), tiles_n = cdiv(d_out, C::TN);
        if (dy_hilo)
            hipLaunchKernelGGL((k_gemm_dw<C, kDwBK, kDwStages, kDwMinWaves, true>),
                               dim3((unsigned)(tiles_m * tiles_n * splits)),
                               dim3(C::NT), 0, s, (const char *)mcat, M, (int64_t)Kcat, dy,
                               (int64_t)d_out, tiles_m, tiles_n, per, epi);
        else
            hipLaunchKernelGGL((k_gemm_dw<C, kDwBK, kDwStages, kDwMinWaves, false>),
                               dim3((unsigned)(tiles_m * tiles_n * splits)),
                               dim3(C::NT), 0, s, (const char *)mcat, M, (int64_t)Kcat, dy,
                               (int64_t)d_out, tiles_m, tiles_n, per, epi);
        RGCN_HIP_TRY(hipGetLastError());
    } else {
        using C = CfgF32;
        LoadTransF32<C::NT> la{(const char *)mcat, (int64_t)Kcat * 4, M, Kcat};
        LoadTransF32<C::NT> lb{(const char *)dy, (int64_t)d_out * 4, M, d_out};
        RGCN_HIP_TRY((launch_gemm<C, MmaF32<C::FM, C::FN>, decltype(la), decltype(lb), EpiPartial,
                                  2, 2>(la, lb, epi, Kcat, d_out, M, splits, per, s)));
    }
    const int64_t total = (int64_t)Kcat * d_out;
    hipLaunchKernelGGL(k_dw_reduce, dim3((unsigned)cdiv(total, kThreads)), dim3(kThreads), 0, s,
                       partial, splits, Kcat, d_in, d_out, out);
    return hipGetLastError();
}

}  // namespace rgcn
