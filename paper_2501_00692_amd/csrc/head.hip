// head.hip -- the language head's loss and logit gradients (Sec. 3.2: o^t =
// Omega Norm(y_K^t); the per-token losses and dl/do^t that Alg. 1 evaluates once
// before the layers' gradients).  The products with Omega run on the bf16 MFMA
// GEMMs of gemm.hip; this file holds the row-wise step between them:
//   k_head_xent : per row of fp32 logits o [V] and target t, the cross-entropy
//                 l = log sum_v exp(o_v) - o_t and the logit gradient
//                 G = softmax(o) - onehot(t) as bf16 (round to nearest even).
//                 t < 0: no loss (l = 0, G = 0); t >= V: l = NaN, G = 0.
// Vocabularies up to 65,536: one workgroup of 1024 threads per row holds the row
// in registers (one read of the logits: 6 bytes per logit with G).  Larger ones:
// 256 threads per row, pass 1 keeps a running maximum and the sum of
// exp(o - max) per thread over float4 pieces of the row (the sum rescaled when
// the maximum grows), combined over the workgroup in a fixed tree; pass 2 reads
// the row again (from L2) and writes G.
#include <cmath>

#include "internal.h"

namespace ssmk {
namespace {

constexpr int kXentThreads = 256;

// fp32 -> bf16, round to nearest even (the hardware conversion, v_cvt_pk_bf16_f32)
__device__ __forceinline__ uint16_t bf16_rne(float v) { return __builtin_bit_cast(uint16_t, static_cast<__bf16>(v)); }

__global__ __launch_bounds__(kXentThreads) void k_head_xent(const float* o, int64_t ldo, const int32_t* tgt,
                                                            float* loss, uint16_t* G, int64_t ldg, int64_t V) {
    __shared__ float smax[kXentThreads], ssum[kXentThreads];
    const int tid = threadIdx.x;
    const int64_t row = blockIdx.x;
    const float4* orow = reinterpret_cast<const float4*>(o + row * ldo);
    const int64_t nv4 = V / 4;
    float mx = -INFINITY, s = 0.f;
    for (int64_t i = tid; i < nv4; i += kXentThreads) {
        const float4 x = orow[i];
        const float m4 = fmaxf(fmaxf(x.x, x.y), fmaxf(x.z, x.w));
        const float mn = fmaxf(mx, m4);
        // exp(-inf) = 0 covers the first piece (mx = -inf)
        s = s * __expf(mx - mn) + ((__expf(x.x - mn) + __expf(x.y - mn)) + (__expf(x.z - mn) + __expf(x.w - mn)));
        mx = mn;
    }
    smax[tid] = mx;
    ssum[tid] = s;
    __syncthreads();
#pragma unroll
    for (int h = kXentThreads / 2; h > 0; h >>= 1) {
        if (tid < h) {
            const float ma = smax[tid], mb = smax[tid + h];
            const float mn = fmaxf(ma, mb);
            // pieces that never saw a value (-inf) contribute 0
            const float sa = ma == -INFINITY ? 0.f : ssum[tid] * __expf(ma - mn);
            const float sb = mb == -INFINITY ? 0.f : ssum[tid + h] * __expf(mb - mn);
            smax[tid] = mn;
            ssum[tid] = sa + sb;
        }
        __syncthreads();
    }
    const float m = smax[0], tot = ssum[0];
    const int32_t t = tgt[row];
    const bool valid = t >= 0 && t < V;
    if (tid == 0) {
        const float* orw = o + row * ldo;
        loss[row] = valid ? (m + __logf(tot)) - orw[t] : (t < 0 ? 0.f : NAN);
    }
    const float inv = 1.f / tot;
    const float keep = valid ? 1.f : 0.f;
    uint2* grow = reinterpret_cast<uint2*>(G + row * ldg);
    for (int64_t i = tid; i < nv4; i += kXentThreads) {
        const float4 x = orow[i];
        float g[4] = {__expf(x.x - m) * inv, __expf(x.y - m) * inv, __expf(x.z - m) * inv, __expf(x.w - m) * inv};
        const int64_t v0 = 4 * i;
        if (valid && t >= v0 && t < v0 + 4) g[t - v0] -= 1.f;
        uint16_t b[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) b[k] = bf16_rne(g[k] * keep);
        grow[i] = make_uint2(static_cast<uint32_t>(b[0]) | (static_cast<uint32_t>(b[1]) << 16),
                             static_cast<uint32_t>(b[2]) | (static_cast<uint32_t>(b[3]) << 16));
    }
}

// The same with the row held in registers (one read of the logits): 1024 threads,
// PER float4 pieces of the row per thread (V <= 4096 PER).  The maximum and the
// rescaled sum are combined over each wave with shuffles and over the 16 waves in
// LDS, in a fixed order.
template <int PER>
__global__ __launch_bounds__(1024) void k_head_xent_reg(const float* o, int64_t ldo, const int32_t* tgt, float* loss,
                                                        uint16_t* G, int64_t ldg, int64_t V) {
    __shared__ float smax[16], ssum[16];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int64_t row = blockIdx.x;
    const float4* orow = reinterpret_cast<const float4*>(o + row * ldo);
    const int64_t nv4 = V / 4;
    float4 x[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int64_t i = tid + 1024 * j;
        x[j] = i < nv4 ? orow[i] : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
    }
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < PER; ++j) mx = fmaxf(mx, fmaxf(fmaxf(x[j].x, x[j].y), fmaxf(x[j].z, x[j].w)));
    for (int m = 1; m < 64; m <<= 1) mx = fmaxf(mx, __shfl_xor(mx, m));
    if (lane == 0) smax[wv] = mx;
    __syncthreads();
    float m = smax[0];
    for (int w = 1; w < 16; ++w) m = fmaxf(m, smax[w]);
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < PER; ++j)  // padding pieces are -inf: exp gives 0
        s += (__expf(x[j].x - m) + __expf(x[j].y - m)) + (__expf(x[j].z - m) + __expf(x[j].w - m));
    for (int k = 1; k < 64; k <<= 1) s += __shfl_xor(s, k);
    if (lane == 0) ssum[wv] = s;
    __syncthreads();
    float tot = ssum[0];
    for (int w = 1; w < 16; ++w) tot += ssum[w];
    const int32_t t = tgt[row];
    const bool valid = t >= 0 && t < V;
    if (tid == 0) loss[row] = valid ? (m + __logf(tot)) - o[row * ldo + t] : (t < 0 ? 0.f : NAN);
    const float inv = 1.f / tot;
    const float keep = valid ? 1.f : 0.f;
    uint2* grow = reinterpret_cast<uint2*>(G + row * ldg);
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int64_t i = tid + 1024 * j;
        if (i >= nv4) break;
        float g[4] = {__expf(x[j].x - m) * inv, __expf(x[j].y - m) * inv, __expf(x[j].z - m) * inv,
                      __expf(x[j].w - m) * inv};
        const int64_t v0 = 4 * i;
        if (valid && t >= v0 && t < v0 + 4) g[t - v0] -= 1.f;
        uint16_t b[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) b[k] = bf16_rne(g[k] * keep);
        grow[i] = make_uint2(static_cast<uint32_t>(b[0]) | (static_cast<uint32_t>(b[1]) << 16),
                             static_cast<uint32_t>(b[2]) | (static_cast<uint32_t>(b[3]) << 16));
    }
}

}  // namespace

hipError_t launch_head_xent(const float* logits, int64_t ldo, const int32_t* targets, float* loss, uint16_t* G,
                            int64_t ldg, int64_t rows, int64_t V, hipStream_t s) {
    if (V % 4 || ldo % 4 || ldg % 4) return hipErrorInvalidValue;
    SSMK_TIMED("head_xent", s);
    const dim3 grid(static_cast<unsigned>(rows));
    const int64_t per = (V / 4 + 1023) / 1024;  // float4 pieces per thread with the row in registers
#define SSMK_XENT_REG(P) hipLaunchKernelGGL(k_head_xent_reg<P>, grid, dim3(1024), 0, s, logits, ldo, targets, loss, G, ldg, V)
    if (per <= 1) SSMK_XENT_REG(1);
    else if (per <= 2) SSMK_XENT_REG(2);
    else if (per <= 4) SSMK_XENT_REG(4);
    else if (per <= 8) SSMK_XENT_REG(8);
    else if (per <= 16) SSMK_XENT_REG(16);
    else hipLaunchKernelGGL(k_head_xent, grid, dim3(kXentThreads), 0, s, logits, ldo, targets, loss, G, ldg, V);
#undef SSMK_XENT_REG
    return hipGetLastError();
}

}  // namespace ssmk
