// stack.hip -- kernels of the K-layer residual stack (Sec. 3.2, Alg. 1) around
// the per-layer SSM kernels:
//   k_rms_fwd   : u = y / sqrt(mean_d y^2 + eps) as bf16, and 1/rms per row;
//   k_rms_bwd   : g (+)= (du - u mean_d(du u)) / rms with u = y / rms recomputed in
//                 fp32 (the cotangent of the normalisation), plus g's bf16 copy
//                 when asked;
//   k_residual  : y_out = y_in + ytil (ytil bf16);
//   k_transpose : bf16 [R][C] -> [C][R] (the forward projections read W^T);
//   k_to_bf16   : fp32 -> bf16 (round to nearest even).
// One workgroup per row for the normalisation; sums over the row in a fixed
// order (per-thread strided partials, then a tree over the workgroup).
#include "internal.h"

namespace ssmk {
namespace {

constexpr int kRowThreads = 256;
constexpr float kRmsEps = 1e-6f;

// fp32 -> bf16, round to nearest even (the hardware conversion, v_cvt_pk_bf16_f32)
__device__ __forceinline__ uint16_t to_bf16(float v) { return __builtin_bit_cast(uint16_t, static_cast<__bf16>(v)); }
__device__ __forceinline__ float from_bf16(uint16_t b) { return __uint_as_float(static_cast<uint32_t>(b) << 16); }

// Sum of v over the workgroup (kRowThreads threads), the same on every thread.
__device__ __forceinline__ float row_sum(float v, float* sh) {
    const int tid = threadIdx.x;
    sh[tid] = v;
    __syncthreads();
#pragma unroll
    for (int s = kRowThreads / 2; s > 0; s >>= 1) {
        if (tid < s) sh[tid] += sh[tid + s];
        __syncthreads();
    }
    const float r = sh[0];
    __syncthreads();
    return r;
}

__global__ __launch_bounds__(kRowThreads) void k_rms_fwd(const float* y, uint16_t* u, float* rinv, int64_t D) {
    __shared__ float sh[kRowThreads];
    const int64_t row = blockIdx.x;
    const float* yr = y + row * D;
    float ss = 0.f;
    for (int64_t d = threadIdx.x; d < D; d += kRowThreads) ss = fmaf(yr[d], yr[d], ss);
    const float r = 1.f / sqrtf(row_sum(ss, sh) / static_cast<float>(D) + kRmsEps);
    for (int64_t d = threadIdx.x; d < D; d += kRowThreads) u[row * D + d] = to_bf16(yr[d] * r);
    if (threadIdx.x == 0) rinv[row] = r;
}

__global__ __launch_bounds__(kRowThreads) void k_rms_bwd(const float* y, const float* rinv, const float* du,
                                                          float* g, uint16_t* g16, int64_t D, bool accum) {
    __shared__ float sh[kRowThreads];
    const int64_t row = blockIdx.x;
    const float r = rinv[row];
    const float* yr = y + row * D;
    const float* dr = du + row * D;
    float s = 0.f;
    for (int64_t d = threadIdx.x; d < D; d += kRowThreads) s = fmaf(dr[d], yr[d] * r, s);
    const float m = row_sum(s, sh) / static_cast<float>(D);
    for (int64_t d = threadIdx.x; d < D; d += kRowThreads) {
        const float v = (accum ? g[row * D + d] : 0.f) + (dr[d] - yr[d] * r * m) * r;
        g[row * D + d] = v;
        if (g16) g16[row * D + d] = to_bf16(v);
    }
}

__global__ __launch_bounds__(256) void k_residual(const float* yin, const uint16_t* ytil, float* yout, int64_t n) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i < n) yout[i] = yin[i] + from_bf16(ytil[i]);
}

__global__ __launch_bounds__(256) void k_to_bf16(const float* x, uint16_t* y, int64_t n) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i < n) y[i] = to_bf16(x[i]);
}

// grid (ceil(C/32), ceil(R/32)), 32 x 8 threads; a 32 x 32 tile through LDS.
__global__ __launch_bounds__(256) void k_transpose(const uint16_t* in, uint16_t* out, int64_t R, int64_t C) {
    __shared__ uint16_t tile[32][33];
    const int64_t c0 = static_cast<int64_t>(blockIdx.x) * 32, r0 = static_cast<int64_t>(blockIdx.y) * 32;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
    for (int j = ty; j < 32; j += 8) {
        const int64_t r = r0 + j, c = c0 + tx;
        if (r < R && c < C) tile[j][tx] = in[r * C + c];
    }
    __syncthreads();
    for (int j = ty; j < 32; j += 8) {
        const int64_t c = c0 + j, r = r0 + tx;
        if (r < R && c < C) out[c * R + r] = tile[tx][j];
    }
}

inline unsigned blocks(int64_t n, int64_t per) { return static_cast<unsigned>((n + per - 1) / per); }

}  // namespace

hipError_t launch_rms_fwd(const float* y, uint16_t* u, float* rinv, int64_t M, int64_t D, hipStream_t s) {
    SSMK_TIMED("rms_fwd", s);
    hipLaunchKernelGGL(k_rms_fwd, dim3(static_cast<unsigned>(M)), dim3(kRowThreads), 0, s, y, u, rinv, D);
    return hipGetLastError();
}

hipError_t launch_rms_bwd(const float* y, const float* rinv, const float* du, float* g, uint16_t* g16, int64_t M,
                          int64_t D, hipStream_t s, bool accum) {
    SSMK_TIMED("rms_bwd", s);
    hipLaunchKernelGGL(k_rms_bwd, dim3(static_cast<unsigned>(M)), dim3(kRowThreads), 0, s, y, rinv, du, g, g16, D,
                       accum);
    return hipGetLastError();
}

hipError_t launch_residual(const float* yin, const uint16_t* ytil, float* yout, int64_t n, hipStream_t s) {
    SSMK_TIMED("residual", s);
    hipLaunchKernelGGL(k_residual, dim3(blocks(n, 256)), dim3(256), 0, s, yin, ytil, yout, n);
    return hipGetLastError();
}

hipError_t launch_to_bf16(const float* x, uint16_t* y, int64_t n, hipStream_t s) {
    hipLaunchKernelGGL(k_to_bf16, dim3(blocks(n, 256)), dim3(256), 0, s, x, y, n);
    return hipGetLastError();
}

hipError_t launch_transpose16(const uint16_t* in, uint16_t* out, int64_t R, int64_t C, hipStream_t s) {
    hipLaunchKernelGGL(k_transpose, dim3(blocks(C, 32), blocks(R, 32)), dim3(256), 0, s, in, out, R, C);
    return hipGetLastError();
}

}  // namespace ssmk
