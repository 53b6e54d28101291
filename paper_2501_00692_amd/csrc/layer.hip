// layer.hip -- the step between the layer's weight-gradient launch and the
// product that finishes dW_in when the input projection's gradient is
// reassociated (d_model < D):
//   dW_in[:, :D] = u^T dx + (u^T dZx) W_x^T,   dW_in[:, D:] = u^T dz,
// where one launch has produced G = u^T [dx | dz | dZx] (fp32 [d_model][3D+2N]).
// k_layer_split copies G[:, D:2D] into dW_in[:, D:2D] and splits G[:, 2D:]
// = u^T dZx into two bf16 parts, hi = bf16(v) and lo = bf16(v - hi) (round to
// nearest even), so that the product with W_x^T that follows sees v to about
// 2^-17 relative instead of bf16's 2^-9.
#include "internal.h"

namespace ssmk {
namespace {

// fp32 -> bf16, round to nearest even (the hardware conversion, v_cvt_pk_bf16_f32)
__device__ __forceinline__ uint16_t rne16(float v) { return __builtin_bit_cast(uint16_t, static_cast<__bf16>(v)); }

// grid (ceil(max(D, nx) / 256), min(dm, 65535)); one thread per column of each
// part, rows strided by the grid's height
__global__ __launch_bounds__(256) void k_layer_split(const float* __restrict__ G, int64_t ldg, int64_t dm,
                                                     int64_t D, int64_t nx, float* __restrict__ dW_in, int64_t ldw,
                                                     uint16_t* __restrict__ hi, uint16_t* __restrict__ lo) {
    const int64_t c = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    for (int64_t r = blockIdx.y; r < dm; r += gridDim.y) {
        const float* g = G + r * ldg;
        if (c < D) dW_in[r * ldw + D + c] = g[D + c];
        if (c < nx) {
            const float v = g[2 * D + c];
            const uint16_t h = rne16(v);
            hi[r * nx + c] = h;
            lo[r * nx + c] = rne16(v - __uint_as_float(static_cast<uint32_t>(h) << 16));
        }
    }
}

}  // namespace

hipError_t launch_layer_split(const float* G, int64_t ldg, int64_t dm, int64_t D, int64_t nx, float* dW_in,
                              int64_t ldw, uint16_t* hi, uint16_t* lo, hipStream_t s) {
    const int64_t w = D > nx ? D : nx;
    SSMK_TIMED("layer_split", s);
    const int64_t gy = dm < 65535 ? dm : 65535;
    hipLaunchKernelGGL(k_layer_split, dim3(static_cast<unsigned>((w + 255) / 256), static_cast<unsigned>(gy)),
                       dim3(256), 0, s, G, ldg, dm, D, nx, dW_in, ldw, hi, lo);
    return hipGetLastError();
}

}  // namespace ssmk
