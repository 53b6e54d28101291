// da_debug.hip -- the optional debug output of the gradient: the cotangent of
// each decay value, da_t[d,n] = mubar_t[d,n] h_{t-1}[d,n] (Prop. 2's vjp_A term
// before it is chained into Delta and A_log; mubar is the full adjoint, or the
// windowed adjoint of Eq. "capped" in truncated mode).  It is not on the hot
// path: one thread per (batch, channel, state) walks the sequence forward,
// leaving h_{t-1} in the output, then backwards, multiplying it by mubar_t.
// The windowed adjoint follows the same recurrence as the fused gradient
// kernel: mubar_t = g_t C_t + a_{t+1} mubar_{t+1} - P(t, t+tbar) g_{t+tbar} C_{t+tbar},
// with P(t, t+tbar) = 2^{cn W_t} from the fp64 window sum of Delta.
#include "internal.h"

namespace ssmk {
namespace {

__device__ __forceinline__ float ld_in(const void* p, int64_t i, bool bf16) {
    if (bf16) return __uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t*>(p)[i]) << 16);
    return static_cast<const float*>(p)[i];
}

__device__ __forceinline__ float softplus_ref(float v) { return v > 0.f ? v + log1pf(expf(-v)) : log1pf(expf(v)); }

// Delta_t and the gated upstream g_t of channel d at row (bb, t).
__device__ __forceinline__ void step_scalars(const ScanProblem& p, int64_t td, float* dl, float* g) {
    const float pr = ld_in(p.delta, td, p.bf16);
    *dl = p.softplus ? softplus_ref(pr) : pr;
    const float dy = ld_in(p.dy, td, p.bf16);
    if (p.gate) {
        const float z = ld_in(p.z, td, p.bf16);
        *g = dy * z / (1.f + expf(-z));
    } else {
        *g = dy;
    }
}

// grid (ceil(D * N / 256), b); thread (d, n) with n fastest, so that the output
// rows [b][t][d][n] are written contiguously
__global__ __launch_bounds__(256) void k_da_debug(const ScanProblem p, float* __restrict__ da) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i >= p.D * p.N) return;
    const int64_t d = i / p.N, n = i % p.N, bb = blockIdx.y;
    const float cn = -expf(p.A_log[p.ascalar ? d : d * p.N + n]) * 1.4426950408889634f;
    const int64_t T = p.T;
    float h = p.h0 ? p.h0[(bb * p.D + d) * p.N + n] : 0.f;
    for (int64_t t = 0; t < T; ++t) {
        const int64_t td = (bb * T + t) * p.D + d;
        float dl, g;
        step_scalars(p, td, &dl, &g);
        const float u = p.bdelta ? dl * ld_in(p.x, td, p.bf16) : ld_in(p.x, td, p.bf16);
        da[td * p.N + n] = h;  // h_{t-1}
        h = exp2f(cn * dl) * h + ld_in(p.B, (bb * T + t) * p.N + n, p.bf16) * u;
    }
    const bool trunc = p.trunc && p.tbar < T;
    float mu = 0.f;      // a_{t+1} mubar_{t+1}
    double W = 0.0;      // W_t = sum_{j=t+1}^{t+tbar} Delta_j, steps past T counting 0
    float dl_next = 0.f; // Delta_{t+1}
    for (int64_t t = T - 1; t >= 0; --t) {
        const int64_t td = (bb * T + t) * p.D + d;
        float dl, g;
        step_scalars(p, td, &dl, &g);
        float m = fmaf(g, ld_in(p.C, (bb * T + t) * p.N + n, p.bf16), mu);
        if (trunc) {
            // W_t = W_{t+1} + Delta_{t+1} - Delta_{t+1+tbar}
            if (t + 1 < T) W += static_cast<double>(dl_next);
            const int64_t s = t + p.tbar;  // the step that leaves the window
            if (s + 1 < T) {
                float dl1, g1;
                step_scalars(p, (bb * T + s + 1) * p.D + d, &dl1, &g1);
                W -= static_cast<double>(dl1);
            }
            if (s < T) {
                float dls, gs;
                step_scalars(p, (bb * T + s) * p.D + d, &dls, &gs);
                m = fmaf(-exp2f(cn * static_cast<float>(W)), gs * ld_in(p.C, (bb * T + s) * p.N + n, p.bf16), m);
            }
        }
        da[td * p.N + n] *= m;  // held h_{t-1}
        mu = exp2f(cn * dl) * m;
        dl_next = dl;
    }
}

}  // namespace

hipError_t launch_da_debug(const ScanProblem& p, float* da, hipStream_t s) {
    SSMK_TIMED("da_debug", s);
    hipLaunchKernelGGL(k_da_debug, dim3(static_cast<unsigned>((p.D * p.N + 255) / 256), static_cast<unsigned>(p.nb)),
                       dim3(256), 0, s, p, da);
    return hipGetLastError();
}

}  // namespace ssmk
