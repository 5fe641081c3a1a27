// Sparse optimizer step of learnable embedding tables (Sec. 3.3.2: the trainable rows of
// a featureless node type are updated only where a mini-batch used them).  The rule is
// row-wise Adagrad on the listed rows:
//   state[r] += g[r]^2;   table[r] -= lr * g[r] / (sqrt(state[r]) + eps)
// with g the table-shaped fp32 gradient, state fp32 and the table in the block dtype
// (bf16 rounded to nearest even after the step).  The fused form of the same step inside
// the backward transposed sum lives with that kernel; this one serves gradients that
// were scatter-added first (repeated ids in a block).
#include "common.h"

namespace rgcn {

namespace {

constexpr int kThreads = 256;

// One group of G lanes per listed row (G = the power of two covering the row's 4-column
// chunks, at most 64); lane lg handles chunks lg, lg + G, ...  Rows outside
// [0, num_rows) are skipped.
template <bool BF16>
__global__ __launch_bounds__(kThreads) void k_sparse_adagrad(int64_t n, const int64_t *rows,
                                                             int64_t num_rows, int d, int G,
                                                             float *grad, int64_t grad_ld,
                                                             int clear, float *state,
                                                             char *table, int64_t ld, float lr,
                                                             float eps) {
    const int lane = threadIdx.x & 63;
    const int lg = lane & (G - 1);
    const int per_wave = 64 / G;
    const int chunks = d / 4;
    const int64_t wave = ((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6;
    const int64_t stride = ((int64_t)gridDim.x * kThreads >> 6) * per_wave;
    constexpr int ES = BF16 ? 2 : 4;
    for (int64_t i = wave * per_wave + lane / G; i < n; i += stride) {
        const int64_t r = rows[i];
        if (r < 0 || r >= num_rows) continue;
        for (int c = lg; c < chunks; c += G) {
            float *gp = grad + r * grad_ld + (int64_t)c * 4;
            float *sp = state + r * (int64_t)d + (int64_t)c * 4;
            char *tp = table + (r * ld + (int64_t)c * 4) * ES;
            const f32x4 g = *(const f32x4 *)gp;
            const f32x4 st = *(const f32x4 *)sp + g * g;
            f32x4 w;
            if constexpr (BF16) {
                typedef uint32_t u2 __attribute__((ext_vector_type(2)));
                const u2 v = *(const u2 *)tp;
                w = f32x4{bf16_lo(v.x), bf16_hi(v.x), bf16_lo(v.y), bf16_hi(v.y)};
            } else {
                w = *(const f32x4 *)tp;
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) w[e] = w[e] - lr * g[e] / (sqrtf(st[e]) + eps);
            *(f32x4 *)sp = st;
            if constexpr (BF16) {
                typedef uint32_t u2 __attribute__((ext_vector_type(2)));
                *(u2 *)tp = u2{pack_bf16x2(w[0], w[1]), pack_bf16x2(w[2], w[3])};
            } else {
                *(f32x4 *)tp = w;
            }
            if (clear) *(f32x4 *)gp = f32x4{0.f, 0.f, 0.f, 0.f};
        }
    }
}

}  // namespace

hipError_t sparse_adagrad(rgcn_dtype dt, int64_t n, const int64_t *rows, int64_t num_rows,
                          int32_t d, float *grad, int64_t grad_ld, bool clear_grad,
                          float *state, void *table, int64_t ld, float lr, float eps,
                          hipStream_t s) {
    if (n == 0 || d == 0) return hipSuccess;
    const int chunks = d / 4;
    int G = 1;
    while (G < chunks && G < 64) G *= 2;
    const int64_t per_wg = (int64_t)(kThreads / 64) * (64 / G);
    int64_t wgs = (n + per_wg - 1) / per_wg;
    if (wgs > 65536) wgs = 65536;
    if (dt == RGCN_BF16)
        hipLaunchKernelGGL(k_sparse_adagrad<true>, dim3((unsigned)wgs), dim3(kThreads), 0, s, n,
                           rows, num_rows, (int)d, G, grad, grad_ld, clear_grad ? 1 : 0, state,
                           (char *)table, ld, lr, eps);
    else
        hipLaunchKernelGGL(k_sparse_adagrad<false>, dim3((unsigned)wgs), dim3(kThreads), 0, s, n,
                           rows, num_rows, (int)d, G, grad, grad_ld, clear_grad ? 1 : 0, state,
                           (char *)table, ld, lr, eps);
    return hipGetLastError();
}

}  // namespace rgcn
