// scan_kernels.h -- gfx950 kernels for the selective diagonal SSM layer:
//   k_chunk_aggr : per carry chunk, the local end state (from a zero carry-in),
//                  the local adjoint aggregate and the chunk sum of Delta;
//   k_carry      : sequential scan of the chunk aggregates (forward state
//                  carries, reverse adjoint carries, prefix sums of Delta);
//   k_forward    : forward recurrence from the carries, writes y;
//   k_grad       : fused reverse adjoint scan with the vjp epilogue (Prop. 2),
//                  and the truncated window of Eq. "capped";
//   k_reduce_*   : deterministic reductions of the dB/dC and dA_log partials.
//
// Thread layout of the per-step kernels: one wave of 64 lanes covers 16
// channels; the 4 lanes of a quad share a channel and hold 4 of its 16 states
// each, so per-channel sums over the state are two DPP quad swaps.  Loads of
// x, Delta, dy, z are coalesced along the contiguous channel dimension; B_t and
// C_t are the same for every channel and are vector-loaded per lane.
#pragma once

#include "internal.h"

namespace ssmk {
namespace {

constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ float fexp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ float ldf(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float ldf(const uint16_t* p, int64_t i) {
    return __uint_as_float(static_cast<uint32_t>(p[i]) << 16);
}
__device__ __forceinline__ void stf(float* p, int64_t i, float v) { p[i] = v; }
__device__ __forceinline__ void stf(uint16_t* p, int64_t i, float v) {
    uint32_t u = __float_as_uint(v);
    uint16_t r;
    if ((u & 0x7fffffffu) > 0x7f800000u) {
        r = 0x7fc0;  // NaN
    } else {
        u += 0x7fffu + ((u >> 16) & 1u);  // round to nearest even
        r = static_cast<uint16_t>(u >> 16);
    }
    p[i] = r;
}

__device__ __forceinline__ float softplus_f(float p) {
    return fmaxf(p, 0.f) + log1pf(__expf(-fabsf(p)));
}
__device__ __forceinline__ float sigmoid_f(float z) { return 1.f / (1.f + __expf(-z)); }

// DPP quad permutations: [1,0,3,2] and [2,3,0,1].
__device__ __forceinline__ float dpp_swap1(float v) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xF, 0xF, true));
}
__device__ __forceinline__ float dpp_swap2(float v) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xF, 0xF, true));
}
// Sum over the 4 lanes of a quad; every lane gets the same value.
__device__ __forceinline__ float quad_sum(float v) {
    v += dpp_swap1(v);
    v += dpp_swap2(v);
    return v;
}

// Load 4 consecutive states (r*4 .. r*4+3) of row `row` of a [rows][N] tensor.
template <typename TI, bool N16>
__device__ __forceinline__ void ld4(const TI* p, int64_t row, int r, int64_t N, bool valid,
                                    float v[4]) {
    if constexpr (N16) {
        if (!valid) {
            v[0] = v[1] = v[2] = v[3] = 0.f;
            return;
        }
        if constexpr (sizeof(TI) == 2) {
            const uint2 u = *reinterpret_cast<const uint2*>(p + row * 16 + r * 4);
            v[0] = __uint_as_float(u.x << 16);
            v[1] = __uint_as_float(u.x & 0xffff0000u);
            v[2] = __uint_as_float(u.y << 16);
            v[3] = __uint_as_float(u.y & 0xffff0000u);
        } else {
            const float4 f = *reinterpret_cast<const float4*>(p + row * 16 + r * 4);
            v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
        }
    } else {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int n = r * 4 + k;
            v[k] = (valid && n < N) ? ldf(p, row * N + n) : 0.f;
        }
    }
}

// Per-lane decay constants: cn = -e^{A_log} log2(e) (a = 2^{cn Delta}) and
// wn = -e^{A_log} (da/dDelta = a wn).  Padding states get cn = wn = 0.
__device__ __forceinline__ void lane_consts(const float* A_log, int64_t d, int r, int64_t N,
                                            bool dv, float cn[4], float wn[4]) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int n = r * 4 + k;
        const float e = (dv && n < N) ? __expf(A_log[d * N + n]) : 0.f;
        wn[k] = -e;
        cn[k] = -e * kLog2e;
    }
}

// ---------------------------------------------------------------------------
// k_chunk_aggr: grid (ceil(D/64), nc, b), 256 threads (64 channels).
// For chunk c = [s, e]: hloc = state at e from a zero carry-in,
// mloc = sum_{t in c} g_t C_t prod_{j=s}^{t} a_j  (the adjoint that the chunk
// hands to h_{s-1} from a zero carry at its end), sdel = sum_t Delta_t.
// ---------------------------------------------------------------------------
template <typename TI, bool SP, bool GATE, bool WANT_M, bool N16>
__global__ __launch_bounds__(256) void k_chunk_aggr(const ScanProblem p) {
    const int lane = threadIdx.x;
    const int r = lane & 3;
    const int64_t d = static_cast<int64_t>(blockIdx.x) * 64 + (lane >> 2);
    const int64_t c = blockIdx.y, bb = blockIdx.z;
    const bool dv = d < p.D;
    const TI* X = static_cast<const TI*>(p.x);
    const TI* DL = static_cast<const TI*>(p.delta);
    const TI* Bp = static_cast<const TI*>(p.B);
    const TI* Cp = static_cast<const TI*>(p.C);
    const TI* DY = static_cast<const TI*>(p.dy);
    const TI* Z = static_cast<const TI*>(p.z);

    float cn[4], wn[4];
    lane_consts(p.A_log, d, r, p.N, dv, cn, wn);
    float h[4] = {0.f, 0.f, 0.f, 0.f}, m[4] = {0.f, 0.f, 0.f, 0.f}, P[4] = {1.f, 1.f, 1.f, 1.f};
    double sd = 0.0;
    const int64_t t0 = c * p.L;
    const int64_t t1 = min(t0 + p.L, p.T);
    for (int64_t t = t0; t < t1; ++t) {
        const int64_t td = (bb * p.T + t) * p.D + d;
        float xv = 0.f, dl = 0.f, g = 0.f;
        if (dv) {
            xv = ldf(X, td);
            const float pv = ldf(DL, td);
            dl = SP ? softplus_f(pv) : pv;
            if constexpr (WANT_M) {
                const float gy = ldf(DY, td);
                if constexpr (GATE) {
                    const float zv = ldf(Z, td);
                    g = gy * zv * sigmoid_f(zv);
                } else {
                    g = gy;
                }
            }
        }
        float Bv[4], Cv[4];
        ld4<TI, N16>(Bp, bb * p.T + t, r, p.N, true, Bv);
        if constexpr (WANT_M) ld4<TI, N16>(Cp, bb * p.T + t, r, p.N, true, Cv);
        sd += static_cast<double>(dl);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const float av = fexp2(cn[k] * dl);
            h[k] = fmaf(av, h[k], Bv[k] * xv);
            if constexpr (WANT_M) {
                P[k] *= av;
                m[k] = fmaf(g * Cv[k], P[k], m[k]);
            }
        }
    }
    if (!dv) return;
    const int64_t cb = ((bb * p.nc + c) * p.N) * p.D + d;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int n = r * 4 + k;
        if (n < p.N) {
            p.hbuf[cb + n * p.D] = h[k];
            if constexpr (WANT_M) p.mbuf[cb + n * p.D] = m[k];
        }
    }
    if (r == 0) p.sdel[(bb * p.nc + c) * p.D + d] = sd;
}

// ---------------------------------------------------------------------------
// k_carry: grid (ceil(D/256), N, 2b), 256 threads; blockIdx.z = 2*bb + dir.
// dir 0: H_c = state before chunk c: H_0 = h0, H_{c+1} = Pc H_c + hloc_c, with
//        Pc = prod over the chunk of a = 2^{cn sdel_c}; hbuf := H_c; h_last.
//        Thread n == 0 also writes the exclusive prefix sums of sdel (psum).
// dir 1: M_c = a_{e_c+1} mu_{e_c+1}: M_{nc-1} = 0, M_{c-1} = mloc_c + Pc M_c;
//        mbuf := M_c; dh0 = M_{-1}.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_carry(const ScanProblem p) {
    const int64_t d = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (d >= p.D) return;
    const int64_t n = blockIdx.y;
    const int64_t bb = blockIdx.z >> 1;
    const int dir = blockIdx.z & 1;
    const float cn = -__expf(p.A_log[d * p.N + n]) * kLog2e;
    const int64_t st = p.N * p.D;
    const int64_t base = (bb * p.nc * p.N + n) * p.D + d;
    const int64_t sbase = bb * p.nc * p.D + d;
    constexpr int U = 8;
    if (dir == 0) {
        float H = p.h0 ? p.h0[(bb * p.D + d) * p.N + n] : 0.f;
        const bool wps = (p.psum != nullptr) && n == 0;
        const int64_t pbase = bb * (p.nc + 1) * p.D + d;
        double ps = 0.0;
        for (int64_t c0 = 0; c0 < p.nc; c0 += U) {
            float hl[U];
            double sd[U];
#pragma unroll
            for (int j = 0; j < U; ++j) {
                const int64_t c = c0 + j;
                if (c < p.nc) {
                    hl[j] = p.hbuf[base + c * st];
                    sd[j] = p.sdel[sbase + c * p.D];
                }
            }
#pragma unroll
            for (int j = 0; j < U; ++j) {
                const int64_t c = c0 + j;
                if (c < p.nc) {
                    p.hbuf[base + c * st] = H;
                    H = fmaf(fexp2(cn * static_cast<float>(sd[j])), H, hl[j]);
                    if (wps) {
                        p.psum[pbase + c * p.D] = ps;
                        ps += sd[j];
                    }
                }
            }
        }
        if (wps) p.psum[pbase + p.nc * p.D] = ps;
        if (p.h_last) p.h_last[(bb * p.D + d) * p.N + n] = H;
    } else {
        if (!p.mbuf) return;
        float M = 0.f;
        for (int64_t c0 = p.nc - 1; c0 >= 0; c0 -= U) {
            float ml[U];
            double sd[U];
#pragma unroll
            for (int j = 0; j < U; ++j) {
                const int64_t c = c0 - j;
                if (c >= 0) {
                    ml[j] = p.mbuf[base + c * st];
                    sd[j] = p.sdel[sbase + c * p.D];
                }
            }
#pragma unroll
            for (int j = 0; j < U; ++j) {
                const int64_t c = c0 - j;
                if (c >= 0) {
                    p.mbuf[base + c * st] = M;
                    M = fmaf(fexp2(cn * static_cast<float>(sd[j])), M, ml[j]);
                }
            }
        }
        if (p.dh0) p.dh0[(bb * p.D + d) * p.N + n] = M;
    }
}

// ---------------------------------------------------------------------------
// k_forward: grid (ceil(D/64), nc, b), 256 threads.  y_t = sum_n C_t h_t
// (times silu(z_t) with the gate), state recomputed from the chunk carry-in.
// ---------------------------------------------------------------------------
template <typename TI, bool SP, bool GATE, bool N16>
__global__ __launch_bounds__(256) void k_forward(const ScanProblem p) {
    const int lane = threadIdx.x;
    const int r = lane & 3;
    const int64_t d = static_cast<int64_t>(blockIdx.x) * 64 + (lane >> 2);
    const int64_t c = blockIdx.y, bb = blockIdx.z;
    const bool dv = d < p.D;
    const TI* X = static_cast<const TI*>(p.x);
    const TI* DL = static_cast<const TI*>(p.delta);
    const TI* Bp = static_cast<const TI*>(p.B);
    const TI* Cp = static_cast<const TI*>(p.C);
    const TI* Z = static_cast<const TI*>(p.z);
    TI* Y = static_cast<TI*>(p.y);
    float cn[4], wn[4];
    lane_consts(p.A_log, d, r, p.N, dv, cn, wn);
    float h[4];
    const int64_t cb = ((bb * p.nc + c) * p.N) * p.D + d;
#pragma unroll
    for (int k = 0; k < 4; ++k) h[k] = (dv && r * 4 + k < p.N) ? p.hbuf[cb + (r * 4 + k) * p.D] : 0.f;
    const int64_t t0 = c * p.L;
    const int64_t t1 = min(t0 + p.L, p.T);
    for (int64_t t = t0; t < t1; ++t) {
        const int64_t td = (bb * p.T + t) * p.D + d;
        float xv = 0.f, dl = 0.f;
        if (dv) {
            xv = ldf(X, td);
            const float pv = ldf(DL, td);
            dl = SP ? softplus_f(pv) : pv;
        }
        float Bv[4], Cv[4];
        ld4<TI, N16>(Bp, bb * p.T + t, r, p.N, true, Bv);
        ld4<TI, N16>(Cp, bb * p.T + t, r, p.N, true, Cv);
        float yp = 0.f;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            h[k] = fmaf(fexp2(cn[k] * dl), h[k], Bv[k] * xv);
            yp = fmaf(Cv[k], h[k], yp);
        }
        float y = quad_sum(yp);
        if (r == 0 && dv) {
            if constexpr (GATE) {
                const float zv = ldf(Z, td);
                y *= zv * sigmoid_f(zv);
            }
            stf(Y, td, y);
        }
    }
}

// Checkpoint storage indexed by a wave-uniform segment number (scalar branches).
template <int NCK, int I = 0>
__device__ __forceinline__ void ck_put(float (&ck)[NCK][4], int q, const float (&h)[4]) {
    if constexpr (I < NCK) {
        if (q == I) {
#pragma unroll
            for (int k = 0; k < 4; ++k) ck[I][k] = h[k];
        } else {
            ck_put<NCK, I + 1>(ck, q, h);
        }
    }
}
template <int NCK, int I = 0>
__device__ __forceinline__ void ck_get(const float (&ck)[NCK][4], int q, float (&h)[4]) {
    if constexpr (I < NCK) {
        if (q == I) {
#pragma unroll
            for (int k = 0; k < 4; ++k) h[k] = ck[I][k];
        } else {
            ck_get<NCK, I + 1>(ck, q, h);
        }
    }
}

// Sum over the 16 channels of the wave of a per-(channel, state) value, for one
// time step, and add it into acc_row[off + n].  Fixed summation order.
__device__ __forceinline__ void channel_sum_add(float (*buf)[17], const float v[4], int lane,
                                                float* acc_row, int off) {
    const int ch = lane >> 2, r = lane & 3;
#pragma unroll
    for (int k = 0; k < 4; ++k) buf[r * 4 + k][ch] = v[k];
    __syncthreads();
    const int n = lane >> 2, part = lane & 3;
    float s = ((buf[n][part * 4 + 0] + buf[n][part * 4 + 1]) + buf[n][part * 4 + 2]) +
              buf[n][part * 4 + 3];
    s = quad_sum(s);
    if (part == 0) acc_row[off + n] += s;
    __syncthreads();
}

// ---------------------------------------------------------------------------
// k_grad: grid (nsplit, nc, b), one wave (64 lanes) per workgroup.  The
// workgroup owns carry chunk c (L = S*NCK steps) and a range of 16-channel
// tiles.  Per tile:
//   1. checkpoint sweep: from the carry-in state H_c, the state at the start of
//      each S-step segment (registers, NCK x 4 per lane);
//   2. segments in reverse order: recompute the segment's states forward
//      (keeping h_{t-1} and a_t), write dz and the dC partial; then run the
//      adjoint backwards, mu_t = g_t C_t + a_{t+1} mu_{t+1}, starting from the
//      chunk's reverse carry M_c, and apply the vjp epilogue:
//        s = mubar * a_t * h_{t-1};  ddelta = sum_n s wn;  dA_log += s Delta wn;
//        dx = sum_n mubar B_t;  dB_t[n] += mubar x_t  (over channels).
//      Truncated mode: mubar_t = mu_t - P(t, t+tbar) mu_{t+tbar}; mu at the
//      shifted position t+tbar comes from a second reverse sweep run in lockstep
//      from the carry of its own chunk, and P(t, t+tbar) = 2^{cn W_t} with the
//      window sum W_t = sum_{j=t+1}^{t+tbar} Delta_j kept in fp64.
// dB/dC are summed over channels per step in LDS, accumulated over the tiles,
// and written once per chunk (partials per split when nsplit > 1).  The dA_log
// partial of (chunk, channel, state) is written into that chunk's hbuf slot.
// ---------------------------------------------------------------------------
template <typename TI, bool SP, bool GATE, bool TRUNC, bool N16, int S, int NCK>
__global__ __launch_bounds__(64) void k_grad(const ScanProblem p) {
    constexpr int L = S * NCK;
    __shared__ float acc[L][32];  // [t][0..15] dB, [t][16..31] dC
    __shared__ float buf[16][17];
    const int lane = threadIdx.x;
    const int r = lane & 3, chl = lane >> 2;
    const int64_t c = blockIdx.y, bb = blockIdx.z;
    const int split = blockIdx.x;
    const int64_t t0 = c * L;
    const TI* X = static_cast<const TI*>(p.x);
    const TI* DL = static_cast<const TI*>(p.delta);
    const TI* Bp = static_cast<const TI*>(p.B);
    const TI* Cp = static_cast<const TI*>(p.C);
    const TI* DY = static_cast<const TI*>(p.dy);
    const TI* Z = static_cast<const TI*>(p.z);

    for (int i = lane; i < L * 32; i += 64) (&acc[0][0])[i] = 0.f;
    __syncthreads();

    const int64_t ntile = (p.D + 15) / 16;
    const int64_t per = (ntile + p.nsplit - 1) / p.nsplit;
    const int64_t tile_lo = split * per;
    const int64_t tile_hi = min(ntile, tile_lo + per);

    for (int64_t tile = tile_lo; tile < tile_hi; ++tile) {
        const int64_t d = tile * 16 + chl;
        const bool dv = d < p.D;
        float cn[4], wn[4];
        lane_consts(p.A_log, d, r, p.N, dv, cn, wn);
        bool nv[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) nv[k] = dv && (r * 4 + k < p.N);
        const int64_t cb = ((bb * p.nc + c) * p.N + r * 4) * p.D + d;

        // 1. checkpoint sweep
        float h[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) h[k] = nv[k] ? p.hbuf[cb + k * p.D] : 0.f;
        float ck[NCK][4];
        for (int q = 0; q < NCK; ++q) {
            ck_put<NCK>(ck, q, h);
#pragma unroll 4
            for (int j = 0; j < S; ++j) {
                const int64_t t = t0 + q * S + j;
                const bool tv = t < p.T;
                float xv = 0.f, dl = 0.f;
                if (tv && dv) {
                    const int64_t td = (bb * p.T + t) * p.D + d;
                    xv = ldf(X, td);
                    const float pv = ldf(DL, td);
                    dl = SP ? softplus_f(pv) : pv;
                }
                float Bv[4];
                ld4<TI, N16>(Bp, bb * p.T + t, r, p.N, tv, Bv);
#pragma unroll
                for (int k = 0; k < 4; ++k) h[k] = fmaf(fexp2(cn[k] * dl), h[k], Bv[k] * xv);
            }
        }

        // 2. reverse over segments
        float Mp[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) Mp[k] = nv[k] ? p.mbuf[cb + k * p.D] : 0.f;
        float dA[4] = {0.f, 0.f, 0.f, 0.f};

        // truncated-mode state: shifted adjoint carry and the window sum
        float Msh[4] = {0.f, 0.f, 0.f, 0.f};
        double W = 0.0;
        if constexpr (TRUNC) {
            const int64_t tb = p.tbar;
            const int64_t pstart = t0 + L - 1 + tb;
            const int64_t pb = bb * (p.nc + 1) * p.D + d;
            if (pstart < p.T) {
                const int64_t cp = pstart / L;
                const int64_t cpend = (cp + 1) * L - 1;
                const int64_t mb = ((bb * p.nc + cp) * p.N + r * 4) * p.D + d;
#pragma unroll
                for (int k = 0; k < 4; ++k) Msh[k] = nv[k] ? p.mbuf[mb + k * p.D] : 0.f;
                double pre = 0.0;
                for (int64_t ps = cpend; ps > pstart; --ps) {
                    const bool pv = ps < p.T;
                    float dlp = 0.f, gp = 0.f;
                    if (pv && dv) {
                        const int64_t td = (bb * p.T + ps) * p.D + d;
                        const float pr = ldf(DL, td);
                        dlp = SP ? softplus_f(pr) : pr;
                        const float gy = ldf(DY, td);
                        if constexpr (GATE) {
                            const float zv = ldf(Z, td);
                            gp = gy * zv * sigmoid_f(zv);
                        } else {
                            gp = gy;
                        }
                    }
                    float Cv[4];
                    ld4<TI, N16>(Cp, bb * p.T + ps, r, p.N, pv, Cv);
#pragma unroll
                    for (int k = 0; k < 4; ++k)
                        Msh[k] = fexp2(cn[k] * dlp) * fmaf(gp, Cv[k], Msh[k]);
                    pre += static_cast<double>(dlp);
                }
                if (dv)
                    W = (p.psum[pb + cp * p.D] - p.psum[pb + (c + 1) * p.D]) +
                        (p.sdel[(bb * p.nc + cp) * p.D + d] - pre);
            } else if (dv) {
                W = p.psum[pb + p.nc * p.D] - p.psum[pb + (c + 1) * p.D];
            }
        }

        for (int q = NCK - 1; q >= 0; --q) {
            ck_get<NCK>(ck, q, h);
            float hp[S][4], ah[S][4], gh[S], dlh[S], xh[S];
#pragma unroll
            for (int j = 0; j < S; ++j) {
                const int64_t t = t0 + q * S + j;
                const bool tv = t < p.T;
                const int64_t td = (bb * p.T + t) * p.D + d;
                float xv = 0.f, dl = 0.f, g = 0.f, gy = 0.f, zv = 0.f;
                if (tv && dv) {
                    xv = ldf(X, td);
                    const float pv = ldf(DL, td);
                    dl = SP ? softplus_f(pv) : pv;
                    gy = ldf(DY, td);
                    if constexpr (GATE) {
                        zv = ldf(Z, td);
                        g = gy * zv * sigmoid_f(zv);
                    } else {
                        g = gy;
                    }
                }
                float Bv[4], Cv[4];
                ld4<TI, N16>(Bp, bb * p.T + t, r, p.N, tv, Bv);
                ld4<TI, N16>(Cp, bb * p.T + t, r, p.N, tv, Cv);
                float yp = 0.f, gv[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    hp[j][k] = h[k];
                    const float av = fexp2(cn[k] * dl);
                    ah[j][k] = av;
                    h[k] = fmaf(av, h[k], Bv[k] * xv);
                    yp = fmaf(Cv[k], h[k], yp);
                    gv[k] = g * h[k];
                }
                channel_sum_add(buf, gv, lane, acc[q * S + j], 16);
                if constexpr (GATE) {
                    const float y = quad_sum(yp);
                    if (r == 0 && tv && dv) {
                        const float sg = sigmoid_f(zv);
                        p.dz[td] = gy * y * sg * (1.f + zv * (1.f - sg));
                    }
                }
                gh[j] = g;
                dlh[j] = dl;
                xh[j] = xv;
            }
#pragma unroll
            for (int j = S - 1; j >= 0; --j) {
                const int64_t t = t0 + q * S + j;
                const bool tv = t < p.T;
                const int64_t td = (bb * p.T + t) * p.D + d;
                float Bv[4], Cv[4];
                ld4<TI, N16>(Bp, bb * p.T + t, r, p.N, tv, Bv);
                ld4<TI, N16>(Cp, bb * p.T + t, r, p.N, tv, Cv);
                float mu[4], mb[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    mu[k] = fmaf(gh[j], Cv[k], Mp[k]);
                    mb[k] = mu[k];
                }
                if constexpr (TRUNC) {
                    const int64_t ps = t + p.tbar;
                    const bool pv = ps < p.T;
                    float dlp = 0.f, gp = 0.f;
                    if (pv && dv) {
                        const int64_t tdp = (bb * p.T + ps) * p.D + d;
                        const float pr = ldf(DL, tdp);
                        dlp = SP ? softplus_f(pr) : pr;
                        const float gy = ldf(DY, tdp);
                        if constexpr (GATE) {
                            const float zv = ldf(Z, tdp);
                            gp = gy * zv * sigmoid_f(zv);
                        } else {
                            gp = gy;
                        }
                    }
                    float Cs[4];
                    ld4<TI, N16>(Cp, bb * p.T + ps, r, p.N, pv, Cs);
                    const float wf = static_cast<float>(W);
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        const float musp = fmaf(gp, Cs[k], Msh[k]);
                        mb[k] = fmaf(-fexp2(cn[k] * wf), musp, mu[k]);
                        Msh[k] = fexp2(cn[k] * dlp) * musp;
                    }
                    W += static_cast<double>(dlh[j]) - static_cast<double>(dlp);
                }
                float dxp = 0.f, ddp = 0.f, bv[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    dxp = fmaf(mb[k], Bv[k], dxp);
                    const float s = mb[k] * ah[j][k] * hp[j][k];
                    ddp = fmaf(s, wn[k], ddp);
                    dA[k] = fmaf(s, dlh[j], dA[k]);
                    bv[k] = mb[k] * xh[j];
                    Mp[k] = ah[j][k] * mu[k];
                }
                channel_sum_add(buf, bv, lane, acc[q * S + j], 0);
                const float dxv = quad_sum(dxp);
                const float ddv = quad_sum(ddp);
                if (r == 0 && tv && dv) {
                    p.dx[td] = dxv;
                    // softplus'(Delta_pre) = sigmoid(Delta_pre) = 1 - e^{-Delta}
                    p.ddelta[td] = SP ? ddv * (1.f - __expf(-dlh[j])) : ddv;
                }
            }
        }
#pragma unroll
        for (int k = 0; k < 4; ++k)
            if (nv[k]) p.hbuf[cb + k * p.D] = dA[k] * wn[k];
    }
    __syncthreads();
    float* dBo = p.nsplit == 1 ? p.dB : p.pB + static_cast<int64_t>(split) * p.nb * p.T * p.N;
    float* dCo = p.nsplit == 1 ? p.dC : p.pC + static_cast<int64_t>(split) * p.nb * p.T * p.N;
    for (int i = lane; i < L * 32; i += 64) {
        const int tl = i >> 5, col = i & 31, n = col & 15;
        const int64_t t = t0 + tl;
        if (t >= p.T || n >= p.N) continue;
        const int64_t o = (bb * p.T + t) * p.N + n;
        if (col < 16)
            dBo[o] = acc[tl][col];
        else
            dCo[o] = acc[tl][col];
    }
}

// dB, dC = sum over splits of the partials (fixed order).
__global__ __launch_bounds__(256) void k_reduce_bc(const ScanProblem p) {
    const int64_t total = p.nb * p.T * p.N;
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i >= total) return;
    float sb = 0.f, sc = 0.f;
    for (int s = 0; s < p.nsplit; ++s) {
        sb += p.pB[s * total + i];
        sc += p.pC[s * total + i];
    }
    p.dB[i] = sb;
    p.dC[i] = sc;
}

// dA_log, stage 1: grid (ceil(D/256), N, nslice); slice s sums the (b, chunk)
// partials q in its contiguous range, in order.
__global__ __launch_bounds__(256) void k_reduce_da1(const ScanProblem p) {
    const int64_t d = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (d >= p.D) return;
    const int64_t n = blockIdx.y, s = blockIdx.z;
    const int64_t nq = p.nb * p.nc;
    const int64_t per = (nq + p.nslice - 1) / p.nslice;
    const int64_t q0 = s * per, q1 = min(nq, q0 + per);
    float acc = 0.f;
    for (int64_t q = q0; q < q1; ++q) acc += p.hbuf[(q * p.N + n) * p.D + d];
    p.dAtmp[(s * p.N + n) * p.D + d] = acc;
}

// dA_log, stage 2: sum of the slices, transposed to [D][N].
__global__ __launch_bounds__(256) void k_reduce_da2(const ScanProblem p) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i >= p.D * p.N) return;
    const int64_t d = i / p.N, n = i % p.N;
    float acc = 0.f;
    for (int s = 0; s < p.nslice; ++s) acc += p.dAtmp[(s * p.N + n) * p.D + d];
    p.dA_log[i] = acc;
}

inline unsigned cdiv(int64_t a, int64_t b) { return static_cast<unsigned>((a + b - 1) / b); }

template <typename TI, bool SP, bool GATE, bool N16>
hipError_t forward_impl(const ScanProblem& p, hipStream_t s) {
    dim3 g1(cdiv(p.D, 64), static_cast<unsigned>(p.nc), static_cast<unsigned>(p.nb));
    {
        SSMK_TIMED("chunk_aggr", s);
        hipLaunchKernelGGL((k_chunk_aggr<TI, SP, GATE, false, N16>), g1, dim3(256), 0, s, p);
    }
    SSMK_TIMED("carry", s);
    hipLaunchKernelGGL(k_carry, dim3(cdiv(p.D, 256), static_cast<unsigned>(p.N),
                                     static_cast<unsigned>(2 * p.nb)),
                       dim3(256), 0, s, p);
    SSMK_TIMED("forward", s);
    hipLaunchKernelGGL((k_forward<TI, SP, GATE, N16>), g1, dim3(256), 0, s, p);
    return hipGetLastError();
}

template <typename TI, bool SP, bool GATE, bool TRUNC, bool N16, int S, int NCK>
void grad_main(const ScanProblem& p, hipStream_t s) {
    dim3 g(static_cast<unsigned>(p.nsplit), static_cast<unsigned>(p.nc),
           static_cast<unsigned>(p.nb));
    SSMK_TIMED("grad_fused", s);
    hipLaunchKernelGGL((k_grad<TI, SP, GATE, TRUNC, N16, S, NCK>), g, dim3(64), 0, s, p);
}

template <typename TI, bool SP, bool GATE, bool TRUNC, bool N16>
hipError_t grad_impl(const ScanProblem& p, hipStream_t s) {
    dim3 g1(cdiv(p.D, 64), static_cast<unsigned>(p.nc), static_cast<unsigned>(p.nb));
    {
        SSMK_TIMED("chunk_aggr", s);
        hipLaunchKernelGGL((k_chunk_aggr<TI, SP, GATE, true, N16>), g1, dim3(256), 0, s, p);
    }
    {
        SSMK_TIMED("carry", s);
        hipLaunchKernelGGL(k_carry, dim3(cdiv(p.D, 256), static_cast<unsigned>(p.N),
                                         static_cast<unsigned>(2 * p.nb)),
                           dim3(256), 0, s, p);
    }
    switch (p.L) {
        case 16: grad_main<TI, SP, GATE, TRUNC, N16, 8, 2>(p, s); break;
        case 32: grad_main<TI, SP, GATE, TRUNC, N16, 8, 4>(p, s); break;
        case 64: grad_main<TI, SP, GATE, TRUNC, N16, 8, 8>(p, s); break;
        case 128: grad_main<TI, SP, GATE, TRUNC, N16, 8, 16>(p, s); break;
        default: grad_main<TI, SP, GATE, TRUNC, N16, 16, 16>(p, s); break;  // 256
    }
    SSMK_TIMED("reduce", s);
    if (p.nsplit > 1)
        hipLaunchKernelGGL(k_reduce_bc, dim3(cdiv(p.nb * p.T * p.N, 256)), dim3(256), 0, s, p);
    hipLaunchKernelGGL(k_reduce_da1, dim3(cdiv(p.D, 256), static_cast<unsigned>(p.N),
                                          static_cast<unsigned>(p.nslice)),
                       dim3(256), 0, s, p);
    hipLaunchKernelGGL(k_reduce_da2, dim3(cdiv(p.D * p.N, 256)), dim3(256), 0, s, p);
    return hipGetLastError();
}

// Dispatch of the gradient kernels for one input dtype and one mode; each
// (dtype, mode) pair is instantiated in its own translation unit.
template <typename TI, bool TRUNC>
hipError_t grad_sel(const ScanProblem& p, hipStream_t s) {
    const bool n16 = p.N == 16;
#define SSMK_GRAD(SP, GT) \
    return n16 ? grad_impl<TI, SP, GT, TRUNC, true>(p, s) : grad_impl<TI, SP, GT, TRUNC, false>(p, s)
    if (p.softplus) {
        if (p.gate) SSMK_GRAD(true, true);
        SSMK_GRAD(true, false);
    }
    if (p.gate) SSMK_GRAD(false, true);
    SSMK_GRAD(false, false);
#undef SSMK_GRAD
}

}  // namespace

// Entry points of the per-(dtype, mode) translation units.
hipError_t grad_f32_full(const ScanProblem& p, hipStream_t s);
hipError_t grad_f32_trunc(const ScanProblem& p, hipStream_t s);
hipError_t grad_bf16_full(const ScanProblem& p, hipStream_t s);
hipError_t grad_bf16_trunc(const ScanProblem& p, hipStream_t s);

}  // namespace ssmk
