// scan_kernels.h -- gfx950 kernels for the selective diagonal SSM layer:
//   k_chunk_aggr : per carry chunk, the local end state (from a zero carry-in),
//                  the local adjoint aggregate and the chunk sum of Delta
//                  (k_chunk_aggr_quad for small grids);
//   k_carry      : sequential scan of the chunk aggregates (forward state
//                  carries, reverse adjoint carries, prefix sums of Delta);
//   k_forward    : forward recurrence from the carries, writes y
//                  (k_forward_quad for small grids);
//   k_grad       : fused reverse adjoint scan with the vjp epilogue (Prop. 2),
//                  and the truncated window of Eq. "capped";
//   k_reduce_*   : deterministic reductions of the dB/dC and dA_log partials.
//
// Thread layouts: the chunk-aggregate and forward kernels give each lane one
// channel with all of its states in registers, B_t and C_t being scalar operands
// (their _quad forms, for grids too small to hide latency that way, and the fused
// gradient kernel give a wave 16 channels, the 4 lanes of a quad sharing a channel
// and holding 4 of its 16 states each, so per-channel sums over the state are two
// DPP quad swaps).
// Loads of x, Delta, dy, z are coalesced along the contiguous channel
// dimension; B_t and C_t are the same for every channel.
#pragma once

#include <type_traits>

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

// Masked loads without a branch: a lane whose element is not valid reads
// element 0 of the same array (which exists) and clears the value with a bit
// mask.  The load is then issued unconditionally and waited on at its first use;
// a load under a condition is waited on inside its own branch, right after
// issue, and a select between the loaded value and 0 is turned by the compiler
// into exactly such a branch (hence the mask, not a select).
template <typename T>
__device__ __forceinline__ float ldm(const T* p, int64_t i, bool v) {
    const float r = ldf(p, v ? i : 0);
    return __uint_as_float(__float_as_uint(r) & (v ? 0xffffffffu : 0u));
}
// bf16 store, rounded to nearest even by the hardware conversion (v_cvt_pk_bf16_f32;
// checked bit for bit against the integer rounding on every non-NaN pattern class)
__device__ __forceinline__ void stf(uint16_t* p, int64_t i, float v) {
    p[i] = __builtin_bit_cast(uint16_t, static_cast<__bf16>(v));
}

constexpr float kLn2 = 0.6931471805599453f;

// e^x from the hardware base-2 exponential (no denormal results: arguments
// below about -87 give 0, which none of the uses below can tell apart).
__device__ __forceinline__ float fexp(float x) { return __builtin_amdgcn_exp2f(x * kLog2e); }

// log(1 + e) for e in [0, 1] from the hardware base-2 logarithm (1 + e is in
// [1, 2], a normal number); the factor e / ((1 + e) - 1) cancels the rounding
// of 1 + e (Goldberg's log1p).
__device__ __forceinline__ float log1p_small(float e) {
    const float u = 1.f + e;
    const float d = u - 1.f;
    return d == 0.f ? e : (__builtin_amdgcn_logf(u) * kLn2) * (e * __builtin_amdgcn_rcpf(d));
}
__device__ __forceinline__ float softplus_f(float p) {
    return fmaxf(p, 0.f) + log1p_small(fexp(-fabsf(p)));
}
// softplus(p) where `on`, else p: evaluated on every lane and then selected, so
// that no divergent branch splits the surrounding code into basic blocks
__device__ __forceinline__ float softplus_sel(float p, bool on) {
    const float sp = softplus_f(p);
    return on ? sp : p;
}
__device__ __forceinline__ float sigmoid_f(float z) {
    return __builtin_amdgcn_rcpf(1.f + fexp(-z));
}

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
// Quad sums of four per-lane partials v[0..3] (of four consecutive steps): lane r
// of the quad receives the sum of v[r] over the quad.  Two exchange rounds (lane
// r^1, then r^2) send each lane the partials it does not keep: 9 instructions
// where four quad_sum calls and the selection of lane r's value take 12.  The
// additions group as quad_sum's, (v_r + v_{r^1}) + (v_{r^2} + v_{r^3}), so each
// sum is bit-identical to quad_sum's.
__device__ __forceinline__ float quad_sum_transposed(const float v[4], int r) {
    const bool b0 = (r & 1) != 0, b1 = (r & 2) != 0;
    const float s01 = (b0 ? v[1] : v[0]) + dpp_swap1(b0 ? v[0] : v[1]);
    const float s23 = (b0 ? v[3] : v[2]) + dpp_swap1(b0 ? v[2] : v[3]);
    return (b1 ? s23 : s01) + dpp_swap2(b1 ? s01 : s23);
}

// Workgroup barrier for LDS traffic only: waits for this wave's LDS operations
// but leaves its global loads and stores in flight (a plain __syncthreads also
// drains those, which would stall the loads issued ahead of their use).
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Load 4 consecutive states (r*4 .. r*4+3) of row `row` of a [rows][N] tensor.
template <typename TI, bool N16>
__device__ __forceinline__ void ld4(const TI* p, int64_t row, int r, int64_t N, bool valid,
                                    float v[4]) {
    if constexpr (N16) {
        const int64_t o = valid ? row * 16 + r * 4 : 0;  // no branch around the load
        if constexpr (sizeof(TI) == 2) {
            const uint2 u = *reinterpret_cast<const uint2*>(p + o);
            v[0] = valid ? __uint_as_float(u.x << 16) : 0.f;
            v[1] = valid ? __uint_as_float(u.x & 0xffff0000u) : 0.f;
            v[2] = valid ? __uint_as_float(u.y << 16) : 0.f;
            v[3] = valid ? __uint_as_float(u.y & 0xffff0000u) : 0.f;
        } else {
            const float4 f = *reinterpret_cast<const float4*>(p + o);
            v[0] = valid ? f.x : 0.f; v[1] = valid ? f.y : 0.f;
            v[2] = valid ? f.z : 0.f; v[3] = valid ? f.w : 0.f;
        }
    } else {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int n = r * 4 + k;
            v[k] = ldm(p, row * N + n, valid && n < N);
        }
    }
}

// Per-lane decay constants: cn = -e^{A_log} log2(e) (a = 2^{cn Delta}) and
// wn = -e^{A_log} (da/dDelta = a wn), with A_log per (channel, state) or, for the
// scalar-decay variant, per channel.  Padding states get cn = wn = 0.
__device__ __forceinline__ void lane_consts(const float* A_log, int64_t d, int r, int64_t N,
                                            bool dv, bool ascalar, float cn[4], float wn[4]) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int n = r * 4 + k;
        const bool v = dv && n < N;
        const float al = ldm(A_log, ascalar ? d : d * N + n, v);  // one rate per channel, or per state
        const float e = v ? __expf(al) : 0.f;
        wn[k] = -e;
        cn[k] = -e * kLog2e;
    }
}

// Rows of C at the truncated window's shifted steps (16 states), staged per
// segment: the S rows x 16 states of a segment are spread over the 64 lanes of a
// wave, CPL = S/4 consecutive states per lane, and loaded through a raw buffer
// resource over the rows that exist (rows past it read as zero).  Loading them
// per step instead, next to their use, left every step waiting for a load: the
// row's validity is wave-uniform, the compiler branched around the load, and the
// branch's merge waited for all outstanding memory operations.
template <typename TI, int S>
struct ShiftedC {
    static constexpr int CPL = S / 4;                    // states per lane
    static constexpr int BYTES = CPL * sizeof(TI);       // 4, 8 or 16
    using Raw = typename std::conditional<BYTES == 4, uint32_t,
                typename std::conditional<BYTES == 8, uint32_t __attribute__((ext_vector_type(2))),
                                          uint32_t __attribute__((ext_vector_type(4)))>::type>::type;
    static_assert(BYTES == 4 || BYTES == 8 || BYTES == 16, "segment length");

    // raw bits of the rows of segment qs (in-chunk steps qs*S ..) that lane `lane` stages
    static __device__ __forceinline__ Raw load(__amdgpu_buffer_rsrc_t rs, int qs, int lane) {
        const int row = qs * S + lane / (16 / CPL), n0 = (lane % (16 / CPL)) * CPL;
        const int off = (row * 16 + n0) * static_cast<int>(sizeof(TI));
        if constexpr (BYTES == 4) return __builtin_amdgcn_raw_buffer_load_b32(rs, off, 0, 0);
        else if constexpr (BYTES == 8) return __builtin_amdgcn_raw_buffer_load_b64(rs, off, 0, 0);
        else return __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0);
    }
    // fp32 values of the lane's CPL states: into w[j][n / 4][16 + n % 4] (the spare
    // column of the wave's padded channel-sum rows; states 4r .. 4r+3 of step j end
    // up at w[j][r][16 .. 19]), or into w[j][n ..] of the wave's own rows of shifted C
    static __device__ __forceinline__ void stage(const Raw& u, float (&w)[S][16][20], int lane) {
        const int j = lane / (16 / CPL), n0 = (lane % (16 / CPL)) * CPL;
        put(u, &w[j][n0 / 4][16 + n0 % 4]);
    }
    static __device__ __forceinline__ void stage(const Raw& u, float (&w)[S][16], int lane) {
        const int j = lane / (16 / CPL), n0 = (lane % (16 / CPL)) * CPL;
        put(u, &w[j][n0]);
    }
    static __device__ __forceinline__ void put(const Raw& u, float* dst) {
        float v[CPL];
        if constexpr (sizeof(TI) == 2) {
#pragma unroll
            for (int i = 0; i < CPL / 2; ++i) {
                uint32_t x;
                if constexpr (BYTES == 4) x = u;
                else x = u[i];
                v[2 * i] = __uint_as_float(x << 16);
                v[2 * i + 1] = __uint_as_float(x & 0xffff0000u);
            }
        } else {
#pragma unroll
            for (int i = 0; i < CPL; ++i) v[i] = __uint_as_float(u[i]);
        }
        if constexpr (CPL == 2) *reinterpret_cast<float2*>(dst) = make_float2(v[0], v[1]);
        else *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
    }
};

// Uniform loads of the (up to) 16 states of row `row` of a [rows][N] tensor:
// the same for every lane of the wave.
template <typename TI>
__device__ __forceinline__ void ld_row16(const TI* p, int64_t row, int64_t N, float v[16]) {
#pragma unroll
    for (int n = 0; n < 16; ++n) v[n] = n < N ? ldf(p, row * N + n) : 0.f;
}

// Broadcast lane `src` (0..3, a compile-time constant after unrolling) of each
// quad to the whole quad.
__device__ __forceinline__ float quad_bcast(float v, int src) {
    const int iv = __float_as_int(v);
    switch (src & 3) {
        case 0: return __int_as_float(__builtin_amdgcn_mov_dpp(iv, 0x00, 0xF, 0xF, true));
        case 1: return __int_as_float(__builtin_amdgcn_mov_dpp(iv, 0x55, 0xF, 0xF, true));
        case 2: return __int_as_float(__builtin_amdgcn_mov_dpp(iv, 0xAA, 0xF, 0xF, true));
        default: return __int_as_float(__builtin_amdgcn_mov_dpp(iv, 0xFF, 0xF, 0xF, true));
    }
}

// Value of lane `src` of each quad, for a double.
__device__ __forceinline__ double quad_bcast_d(double v, int src) {
    const uint64_t u = __double_as_longlong(v);
    const float lo = quad_bcast(__uint_as_float(static_cast<uint32_t>(u)), src);
    const float hi = quad_bcast(__uint_as_float(static_cast<uint32_t>(u >> 32)), src);
    return __longlong_as_double(static_cast<long long>((static_cast<uint64_t>(__float_as_uint(hi)) << 32) |
                                                       __float_as_uint(lo)));
}

// Raw per-(step, channel) inputs of the steps a lane prepares for its quad, as
// element bits: they are loaded a group or segment ahead and converted at their
// first use, so that nothing waits for the loads before then.
template <typename TI, int SPL>
struct RawIn {
    // element bits at their own width (16 for bf16: the conversion's shift then
    // needs no zero-extension of a loaded register)
    using Bits = typename std::conditional<sizeof(TI) == 2, uint16_t, uint32_t>::type;
    Bits x[SPL], p[SPL], dy[SPL], z[SPL];
};

__device__ __forceinline__ uint32_t ldbits(const float* p, int64_t i) { return __float_as_uint(p[i]); }
__device__ __forceinline__ uint16_t ldbits(const uint16_t* p, int64_t i) { return p[i]; }
// Value of element bits loaded by ldbits; 0 where the element is padding.
template <typename TI>
__device__ __forceinline__ float fin(uint32_t b, bool v) {
    const float f = sizeof(TI) == 2 ? __uint_as_float(b << 16) : __uint_as_float(b);
    return v ? f : 0.f;
}

// Load the raw inputs of the steps j = r + 4*jj of segment [ts, ts+S); lanes whose
// step (t >= T) or channel is padding load element 0 instead.  `full` also loads
// dy and z.
template <typename TI, bool GATE, int SPL>
__device__ __forceinline__ void load_raw(const ScanProblem& p, int64_t bb, int64_t ts, int64_t d,
                                         bool dv, int r, bool full, RawIn<TI, SPL>& o) {
    const TI* X = static_cast<const TI*>(p.x);
    const TI* DL = static_cast<const TI*>(p.delta);
    const TI* DY = static_cast<const TI*>(p.dy);
    const TI* Z = static_cast<const TI*>(p.z);
#pragma unroll
    for (int jj = 0; jj < SPL; ++jj) {
        const int64_t t = ts + r + 4 * jj;
        const bool v = dv && t < p.T;
        const int64_t td = v ? (bb * p.T + t) * p.D + d : 0;
        o.x[jj] = ldbits(X, td);
        o.p[jj] = ldbits(DL, td);
        if (full) {
            o.dy[jj] = ldbits(DY, td);
            o.z[jj] = GATE ? ldbits(Z, td) : 0;
        }
    }
}

// Scalar-load views of global memory: loads through them at an address that is
// the same for every lane of the wave become scalar loads.
typedef const __attribute__((address_space(4))) uint32_t* ConstDw;

// One row of B or C (up to 16 states) as raw bits in scalar registers: with 16
// states the row is contiguous and read with wide scalar loads (bf16: the packed
// pairs, fp32: the values); with fewer, each state is read on its own and held
// as fp32 bits (states past N are 0).  Scalar loads read whole aligned dwords:
// element e of a bf16 tensor (16-byte aligned) is half (e & 1) of dword e >> 1
// (for a last element that starts a dword, the dword's other half lies past the
// tensor but in the same aligned dword, so in mapped memory).
template <typename TI, bool N16>
struct SRow {
    static constexpr bool PACKED = N16 && sizeof(TI) == 2;
    static constexpr int NW = PACKED ? 8 : 16;
    uint32_t w[NW];
    __device__ __forceinline__ void load(const TI* base, int64_t row, int64_t N) {
        if constexpr (N16) {
            const ConstDw q = (ConstDw)(base + row * 16);
#pragma unroll
            for (int i = 0; i < NW; ++i) w[i] = q[i];  // merged into wide scalar loads
        } else {
            const ConstDw q = (ConstDw)(base);
#pragma unroll
            for (int n = 0; n < 16; ++n) {
                const int64_t e = row * N + n;
                if (n >= N) w[n] = 0u;
                else if constexpr (sizeof(TI) == 4) w[n] = q[e];
                else w[n] = (e & 1) ? (q[e >> 1] & 0xffff0000u) : (q[e >> 1] << 16);
            }
        }
    }
    __device__ __forceinline__ float at(int k) const {
        if constexpr (PACKED) return __uint_as_float((k & 1) ? (w[k >> 1] & 0xffff0000u) : (w[k >> 1] << 16));
        else return __uint_as_float(w[k]);
    }
};

// Decay constants cn = -e^{A_log} log2(e) (a = 2^{cn Delta}) of the 16 states of
// channel d (one rate per channel with the scalar-decay variant); padding
// states and channels get 0.
__device__ __forceinline__ void lane_rates16(const ScanProblem& p, int64_t d, bool dv, float cn[16]) {
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        const bool v = dv && k < p.N;
        const float al = ldm(p.A_log, p.ascalar ? d : d * p.N + k, v);
        const float e = v ? __expf(al) : 0.f;
        cn[k] = -e * kLog2e;
    }
}

// The [b][T][D] inputs x, Delta, dy, z of one chunk for a wave of 64 channels
// (one per lane): buffer resources over the chunk's rows, the lane's fixed byte
// offset (padding channels read out of range, i.e. zero) and the step's row
// offset as a scalar.  Step indices are local to the chunk and 32-bit, so that
// their compares and minima stay on the scalar unit (which has no 64-bit signed
// compare); byte offsets within a chunk fit 31 bits (L <= 256, D <= 2^20).
template <typename TI>
struct ChunkRows {
    static constexpr uint32_t kEl = sizeof(TI);
    __amdgpu_buffer_rsrc_t x, p, dy, z;
    uint32_t voff;
    int rowbytes;

    __device__ __forceinline__ void init(const ScanProblem& q, int64_t row0, int nl, int64_t d, bool dv) {
        const int64_t e0 = row0 * q.D;  // the chunk's first element
        const int nbytes = static_cast<int>(nl * q.D * kEl);
        auto rs = [&](const void* base) {
            return __builtin_amdgcn_make_buffer_rsrc(const_cast<TI*>(static_cast<const TI*>(base) + e0), 0, nbytes,
                                                     0x00020000);
        };
        x = rs(q.x);
        p = rs(q.delta);
        dy = q.dy ? rs(q.dy) : x;
        z = q.z ? rs(q.z) : x;
        voff = dv ? static_cast<uint32_t>(d) * kEl : 0x80000000u;
        rowbytes = static_cast<int>(q.D * kEl);
    }
    // element bits of local step tl
    __device__ __forceinline__ uint32_t ld(__amdgpu_buffer_rsrc_t r, int tl) const {
        if constexpr (kEl == 2) return __builtin_amdgcn_raw_buffer_load_b16(r, voff, tl * rowbytes, 0);
        else return __builtin_amdgcn_raw_buffer_load_b32(r, voff, tl * rowbytes, 0);
    }
    static __device__ __forceinline__ float cvt(uint32_t b) { return __uint_as_float(kEl == 2 ? b << 16 : b); }
};

// ---------------------------------------------------------------------------
// k_chunk_aggr: grid (ceil(D/64), nc, b), one wave per workgroup; each lane owns
// one channel and all 16 of its states.  For chunk c = [s, e]:
//   hloc = state at e from a zero carry-in,
//   mloc = sum_{t in c} g_t C_t prod_{j=s}^{t} a_j  (the adjoint that the chunk
//          hands to h_{s-1} from a zero carry at its end),
//   sdel = sum_{t in c} Delta_t (fp64);
// with WANT_M (the gradient) also, for each segment of SEG steps of the chunk,
// the state at the segment start from a zero carry-in (hseg) and the sum of
// Delta from the chunk start to the segment start (cseg): the fused gradient
// kernel rebuilds its segment-start states from them and the chunk carry.
// B_t and C_t are the same for every channel: they are read with scalar loads
// (the rows of step t+1 while step t runs) and enter the arithmetic as scalar
// operands, so nothing is staged in LDS or exchanged between lanes, and the
// per-(channel, step) preparation (softplus, gate, the Delta sum) is done once
// per step for all 16 states.  The raw inputs x, Delta, dy, z are loaded one
// 4-step group ahead.  Steps past the end of the sequence (in the last group)
// have Delta = x = g = 0 and leave h, P, m and the sum unchanged.
// ---------------------------------------------------------------------------
template <typename TI, bool SP, bool GATE, bool WANT_M, bool N16, int SEG>
__global__ __launch_bounds__(64) void k_chunk_aggr(const ScanProblem p) {
    constexpr int G = 4;  // steps per group
    static_assert(SEG % G == 0, "segments are whole groups");
    const int lane = threadIdx.x;
    const int64_t d = static_cast<int64_t>(blockIdx.x) * 64 + lane;  // < Dp
    const int64_t c = blockIdx.y, bb = blockIdx.z;
    const bool dv = d < p.D;
    float cn[16];
    lane_rates16(p, d, dv, cn);
    float h[16], m[16], P[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        h[k] = 0.f;
        m[k] = 0.f;
        P[k] = 1.f;
    }
    double sd = 0.0;
    const int64_t t0 = c * p.L;
    const int64_t t1 = min(t0 + p.L, p.T);
    const int64_t rowb = bb * p.T;  // first row of the sequence
    const TI* Bp = static_cast<const TI*>(p.B);
    const TI* Cp = static_cast<const TI*>(p.C);
    const int nl = static_cast<int>(t1 - t0);  // the chunk's steps
    ChunkRows<TI> cr;
    cr.init(p, rowb + t0, nl, d, dv);
    auto ld = [&](__amdgpu_buffer_rsrc_t r, int tl) { return cr.ld(r, tl); };
    auto cvt = [](uint32_t b) { return ChunkRows<TI>::cvt(b); };
    // segment records (WANT_M): slot q holds the record of segment q; padding
    // channels record zero sums
    const int64_t nseg = WANT_M ? p.L / SEG : 0;
    const int64_t sgb = (bb * p.nc + c) * nseg * p.Dp;
    auto put_seg = [&](int64_t q) {
        float4* rec = reinterpret_cast<float4*>(p.hseg + (sgb + q * p.Dp) * 16) + 4 * static_cast<uint32_t>(d);
        rec[0] = make_float4(h[0], h[1], h[2], h[3]);
        rec[1] = make_float4(h[4], h[5], h[6], h[7]);
        rec[2] = make_float4(h[8], h[9], h[10], h[11]);
        rec[3] = make_float4(h[12], h[13], h[14], h[15]);
        (p.cseg + sgb + q * p.Dp)[static_cast<uint32_t>(d)] = dv ? static_cast<float>(sd) : 0.f;
    };
    // one step from its raw inputs and its rows of B and C
    auto step = [&](float xr, float pr, float dyr, float zr, const SRow<TI, N16>& cB,
                    const SRow<TI, N16>& cC) __attribute__((always_inline)) {
        const float dl = SP ? softplus_f(pr) : pr;
        if (p.bdelta) xr *= dl;  // input term Delta B x
        float g = 0.f;
        if constexpr (WANT_M) g = GATE ? dyr * zr * sigmoid_f(zr) : dyr;
        sd += static_cast<double>(dl);
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            const float av = fexp2(cn[k] * dl);
            h[k] = fmaf(av, h[k], cB.at(k) * xr);
            if constexpr (WANT_M) {
                P[k] *= av;
                m[k] = fmaf(g * cC.at(k), P[k], m[k]);
            }
        }
    };
    // Whole groups: the raw inputs of each step are loaded one group ahead into
    // its slot (past the chunk: its last row again, not used), the rows of B and C
    // one step ahead.
    const int ngrp = nl / G;
    RawIn<TI, G> raw;
    auto load_slot = [&](int tl, int j) __attribute__((always_inline)) {
        const int tc = min(tl, nl - 1);
        raw.x[j] = ld(cr.x, tc);
        raw.p[j] = ld(cr.p, tc);
        if constexpr (WANT_M) {
            raw.dy[j] = ld(cr.dy, tc);
            raw.z[j] = GATE ? ld(cr.z, tc) : 0;
        }
    };
    SRow<TI, N16> nB, nC;  // B and C rows of the next step
    if (ngrp > 0) {
#pragma unroll
        for (int j = 0; j < G; ++j) load_slot(j, j);
        nB.load(Bp, rowb + t0, p.N);
        if constexpr (WANT_M) nC.load(Cp, rowb + t0, p.N);
    }
    for (int gi = 0; gi < ngrp; ++gi) {
        const int s0 = gi * G;
        if constexpr (WANT_M)
            if (s0 % SEG == 0) put_seg(s0 / SEG);  // uniform
#pragma unroll
        for (int j = 0; j < G; ++j) {
            const int t = s0 + j;
            // this step's raw inputs are converted first, then the slot is refilled: a
            // register is reloaded only once its value is used, so the compiler never
            // copies a load still in flight (it would wait for it).  The scheduler is
            // left free here: it sinks the refills towards the end of the group and
            // overlaps each step's per-channel chain (softplus, gate) with the previous
            // step's state updates, which measured 4 % faster than keeping the loads
            // a full group ahead (k_forward, with less arithmetic per step, keeps them
            // there).
            const float xr = cvt(raw.x[j]), pr = cvt(raw.p[j]);
            const float dyr = WANT_M ? cvt(raw.dy[j]) : 0.f, zr = (WANT_M && GATE) ? cvt(raw.z[j]) : 0.f;
            load_slot(t + G, j);
            const SRow<TI, N16> cB = nB;
            SRow<TI, N16> cC;
            const int64_t rn = rowb + t0 + min(t + 1, nl - 1);
            nB.load(Bp, rn, p.N);
            if constexpr (WANT_M) {
                cC = nC;
                nC.load(Cp, rn, p.N);
            }
            step(xr, pr, dyr, zr, cB, cC);
        }
    }
    // the steps after the last whole group (fewer than G: the end of the sequence)
    for (int t = ngrp * G; t < nl; ++t) {
        if constexpr (WANT_M)
            if (t % SEG == 0) put_seg(t / SEG);
        SRow<TI, N16> cB, cC;
        cB.load(Bp, rowb + t0 + t, p.N);
        if constexpr (WANT_M) cC.load(Cp, rowb + t0 + t, p.N);
        step(cvt(ld(cr.x, t)), cvt(ld(cr.p, t)), WANT_M ? cvt(ld(cr.dy, t)) : 0.f,
             (WANT_M && GATE) ? cvt(ld(cr.z, t)) : 0.f, cB, cC);
    }
    if constexpr (WANT_M) {
        // segments that start past the end of the sequence hold the final state
        for (int64_t q = (nl + SEG - 1) / SEG; q < nseg; ++q) put_seg(q);
    }
    if (!dv) return;
    const int64_t cb = (bb * p.nc + c) * p.N * p.D + d;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        if (k < p.N) {
            p.hbuf[cb + k * p.D] = h[k];
            if constexpr (WANT_M) p.mbuf[cb + k * p.D] = m[k];
        }
    }
    p.sdel[(bb * p.nc + c) * p.D + d] = sd;
}

inline dim3 aggr_grid(const ScanProblem& p) {
    return dim3(static_cast<unsigned>((p.D + 63) / 64), static_cast<unsigned>(p.nc), static_cast<unsigned>(p.nb));
}
// Grids of fewer than 2,048 waves at one lane per channel (about two per SIMD: a
// short or narrow problem, e.g. b = 2, T = 4,096, D = 1,536) take the quad layout,
// whose four times as many waves hide the latency that one lane per channel then
// leaves exposed (there 78 against 98 us for the chunk aggregates, 60 against 68
// us for the forward).
inline bool aggr_quad(const ScanProblem& p) { return (p.D + 63) / 64 * p.nc * p.nb < 2048; }

// ---------------------------------------------------------------------------
// k_chunk_aggr_quad: the chunk aggregates of k_chunk_aggr for small grids: grid
// (ceil(D/64), nc, b), 256 threads; the 4 lanes of a quad share a channel and
// hold 4 states each (four times the waves of one lane per channel).  For chunk c = [s, e]:
//   hloc = state at e from a zero carry-in,
//   mloc = sum_{t in c} g_t C_t prod_{j=s}^{t} a_j  (the adjoint that the chunk
//          hands to h_{s-1} from a zero carry at its end),
//   sdel = sum_{t in c} Delta_t (fp64);
// with WANT_M (the gradient) also, for each segment of p.seg steps of the
// chunk, the state at the segment start from a zero carry-in (hseg) and the sum
// of Delta from the chunk start to the segment start (cseg): the fused gradient
// kernel rebuilds its segment-start states from them and the chunk carry.
// B and C are staged in LDS as fp32, 64 steps at a time, for the whole
// workgroup, double-buffered: the next block's loads are in flight while the
// current block is processed, and one barrier per block publishes it.  Lane r
// prepares the per-channel quantities of steps s+r, s+r+4, ... and broadcasts
// them to its quad; its raw inputs are loaded two 4-step groups ahead, so a
// whole group of arithmetic lies between the issue of a load and its use.
// ---------------------------------------------------------------------------
template <typename TI, bool SP, bool GATE, bool WANT_M, int SEG>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4, 8))) void k_chunk_aggr_quad(const ScanProblem p) {
    constexpr int SB = 64;  // steps per staged block
    constexpr int PT = SB * 32 / 256;  // staged values per thread
    static_assert(SB % SEG == 0 && SEG % 4 == 0, "segments tile the staged blocks");
    __shared__ __attribute__((aligned(16))) float bcs[2][SB][32];
    const int tid = threadIdx.x;
    const int r = tid & 3;
    const int64_t d = static_cast<int64_t>(blockIdx.x) * 64 + (tid >> 2);  // < Dp
    const int64_t c = blockIdx.y, bb = blockIdx.z;
    const bool dv = d < p.D;
    const TI* Bp = static_cast<const TI*>(p.B);
    const TI* Cp = static_cast<const TI*>(p.C);
    float cn[4], wn[4];
    lane_consts(p.A_log, d, r, p.N, dv, p.ascalar, cn, wn);
    float h[4] = {0.f, 0.f, 0.f, 0.f}, m[4] = {0.f, 0.f, 0.f, 0.f}, P[4] = {1.f, 1.f, 1.f, 1.f};
    double sd = 0.0;
    const int64_t t0 = c * p.L;
    const int64_t t1 = min(t0 + p.L, p.T);
    // segment records (WANT_M): slot q holds the record of segment q
    const uint32_t nseg = WANT_M ? static_cast<uint32_t>(p.L / SEG) : 0u;
    const int64_t sgb = (bb * p.nc + c) * nseg * p.Dp + d;
    auto put_seg = [&](uint32_t q, float cum) {
        *reinterpret_cast<float4*>(p.hseg + (sgb + q * p.Dp) * 16 + 4 * r) = make_float4(h[0], h[1], h[2], h[3]);
        p.cseg[sgb + q * p.Dp] = cum;
    };
    // the quad's Delta sum so far, added in lane order
    auto quad_total = [&]() {
        return ((quad_bcast_d(sd, 0) + quad_bcast_d(sd, 1)) + quad_bcast_d(sd, 2)) + quad_bcast_d(sd, 3);
    };
    // B/C values of the staged block starting at step sb (padding and steps past
    // the chunk read as 0)
    // raw element bits and validity masks, applied when the block is stored (a
    // masked value right after its load would make each load wait on the spot)
    typename RawIn<TI, 1>::Bits bcv[PT];
    uint32_t bcm[PT];
    auto load_bc = [&](int64_t sb) {
#pragma unroll
        for (int e = 0; e < PT; ++e) {
            const int i = tid + 256 * e;
            const int t = i >> 5, cc = i & 31, n = cc & 15;
            const int64_t tg = sb + t;
            const bool ok = (cc < 16 || WANT_M) && tg < t1 && n < p.N;
            bcm[e] = ok ? 0xffffffffu : 0u;
            bcv[e] = ldbits(cc < 16 ? Bp : Cp, ok ? (bb * p.T + tg) * p.N + n : 0);
        }
    };
    auto store_bc = [&](int buf) {
#pragma unroll
        for (int e = 0; e < PT; ++e) {
            const int i = tid + 256 * e;
            const uint32_t b = sizeof(TI) == 2 ? static_cast<uint32_t>(bcv[e]) << 16 : static_cast<uint32_t>(bcv[e]);
            bcs[buf][i >> 5][i & 31] = __uint_as_float(b & bcm[e]);
        }
    };
    load_bc(t0);
    store_bc(0);
    load_bc(t0 + SB);  // block 1 (all padding when the chunk has one block)
    // raw inputs of the next two groups of 4 steps, in two buffers used
    // alternately (no copies of data still in flight)
    RawIn<TI, 1> n1, n2;
    load_raw<TI, GATE, 1>(p, bb, t0, d, dv, r, WANT_M, n1);
    load_raw<TI, GATE, 1>(p, bb, t0 + 4, d, dv, r, WANT_M, n2);
    lds_barrier();
    int buf = 0;
    // One group of 4 steps from s0, its raw inputs in `nb`, which is then
    // refilled with the group two ahead.  Steps past the end of the sequence have
    // Delta = x = g = 0 and B = C = 0, so they leave h, P, m and the Delta sum
    // unchanged; every group of the chunk runs (no tail branch).
    auto group = [&](int64_t s0, int64_t sb, RawIn<TI, 1>& nb) {
        if constexpr (WANT_M) {
            const uint32_t tl = static_cast<uint32_t>(s0 - t0);
            if (tl % SEG == 0) put_seg(tl / SEG, static_cast<float>(quad_total()));  // uniform
        }
        // this group's raw inputs are converted first, then `nb` is refilled: a
        // register is only reloaded once its value has been used, so the
        // compiler never copies a load that is still in flight
        const bool v = dv && s0 + r < t1;
        const float pr = fin<TI>(nb.p[0], v);
        float xr = fin<TI>(nb.x[0], v);
        const float dyr = WANT_M ? fin<TI>(nb.dy[0], v) : 0.f;
        const float zr = (WANT_M && GATE) ? fin<TI>(nb.z[0], v) : 0.f;
        // issued on every path (past the end it reloads valid data that is not
        // used), so that later waits count exactly; the scheduling barrier keeps
        // the loads ahead of this group's arithmetic
        load_raw<TI, GATE, 1>(p, bb, s0 + 8, d, dv, r, WANT_M, nb);
        __builtin_amdgcn_sched_barrier(0);
        const float dlr = SP ? softplus_sel(pr, v) : pr;
        if (p.bdelta) xr *= dlr;  // input term Delta B x
        float gr = 0.f;
        if constexpr (WANT_M) gr = GATE ? dyr * zr * sigmoid_f(zr) : dyr;
        sd += static_cast<double>(dlr);
        const int tb = static_cast<int>(s0 - sb);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const float xv = quad_bcast(xr, j);
            const float dl = quad_bcast(dlr, j);
            const float4 b4 = *reinterpret_cast<const float4*>(&bcs[buf][tb + j][4 * r]);
            const float Bv[4] = {b4.x, b4.y, b4.z, b4.w};
            float Cv[4] = {0.f, 0.f, 0.f, 0.f};
            if constexpr (WANT_M) {
                const float4 c4 = *reinterpret_cast<const float4*>(&bcs[buf][tb + j][16 + 4 * r]);
                Cv[0] = c4.x; Cv[1] = c4.y; Cv[2] = c4.z; Cv[3] = c4.w;
            }
            const float g = WANT_M ? quad_bcast(gr, j) : 0.f;
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
    };
    for (int64_t sb = t0; sb < t1; sb += SB) {
        // the block's groups, up to the chunk edge (L and SB are multiples of 8)
        const int64_t se = min(sb + SB, t0 + p.L);
        for (int64_t s0 = sb; s0 < se; s0 += 8) {
            group(s0, sb, n1);
            group(s0 + 4, sb, n2);
        }
        // publish the next block (its buffer was last read before the previous
        // barrier) and start loading the one after it
        store_bc(buf ^ 1);
        load_bc(sb + 2 * SB);
        lds_barrier();
        buf ^= 1;
    }
    if constexpr (WANT_M) {
        // segments that start in a block past the end of the sequence hold the final state
        const float cum = static_cast<float>(quad_total());
        const uint32_t done = static_cast<uint32_t>((t1 - t0 + SB - 1) / SB * SB / SEG);
        for (uint32_t q = done; q < nseg; ++q) put_seg(q, cum);
    }
    // sum of Delta over the quad's prepared steps, in a fixed order
    const double s1 = __shfl_xor(sd, 1);
    const double s2 = __shfl_xor(sd, 2);
    const double s3 = __shfl_xor(sd, 3);
    if (!dv) return;
    const int64_t cb = ((bb * p.nc + c) * p.N + r * 4) * p.D + d;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        if (r * 4 + k < p.N) {
            p.hbuf[cb + k * p.D] = h[k];
            if constexpr (WANT_M) p.mbuf[cb + k * p.D] = m[k];
        }
    }
    if (r == 0) p.sdel[(bb * p.nc + c) * p.D + d] = ((sd + s1) + s2) + s3;
}

// ---------------------------------------------------------------------------
// k_carry: 256 threads (4 waves); a unit is (sequence bb, direction, block of 64
// channels), a workgroup takes one unit and 4 of its states (wave w: state
// 4q + w, lane: channel).  The carries are sequential over chunks:
// dir 0: H_c = state before chunk c: H_0 = h0, H_{c+1} = Pc H_c + hloc_c, with
//        Pc = prod over the chunk of a = 2^{cn sdel_c}; hbuf := H_c; h_last.
//        State 0 also writes the exclusive prefix sums of sdel (psum).
// dir 1: M_c = a_{e_c+1} mu_{e_c+1}: M_{nc-1} = 0, M_{c-1} = mloc_c + Pc M_c;
//        mbuf := M_c; dh0 = M_{-1}.
// The walk is bound by memory latency: each wave keeps the loads of the next
// kCarryU chunks in flight while it consumes the current kCarryU (two register
// buffers used alternately).  The workgroups of one unit run on one XCD
// (workgroups are dealt to the XCDs in turn by linear id), so the four waves of
// a workgroup and the workgroups of the unit's other states read each chunk's
// Delta sums through one L2.
// ---------------------------------------------------------------------------
constexpr int kCarryU = 16;

__global__ __launch_bounds__(256) void k_carry(const ScanProblem p) {
    const int64_t nd64 = (p.D + 63) / 64;
    const int64_t nunits = 2 * p.nb * nd64;
    const int nq = static_cast<int>((p.N + 3) / 4);
    const int lin = static_cast<int>(blockIdx.x);
    const int64_t slot = lin / 8;
    const int64_t unit = lin % 8 + 8 * (slot / nq);
    if (unit >= nunits) return;
    const int64_t n = 4 * (slot % nq) + (threadIdx.x >> 6);
    if (n >= p.N) return;
    const int64_t d = (unit % nd64) * 64 + (threadIdx.x & 63);
    if (d >= p.D) return;
    const int dir = static_cast<int>((unit / nd64) & 1);
    const int64_t bb = unit / nd64 / 2;
    const float cn = -__expf(p.A_log[p.ascalar ? d : d * p.N + n]) * kLog2e;
    const int64_t st = p.N * p.D;
    const int64_t base = (bb * p.nc * p.N + n) * p.D + d;
    const int64_t sbase = bb * p.nc * p.D + d;
    const int64_t nc = p.nc;
    constexpr int U = kCarryU;
    float* buf = dir == 0 ? p.hbuf : p.mbuf;
    if (dir == 1 && !buf) return;
    // block k covers chunks kU .. kU+U-1 in walk order (dir 1 walks backwards);
    // positions past the end load a valid chunk and are not used
    auto chunk = [&](int64_t k, int j) { const int64_t i = k * U + j; return dir == 0 ? i : nc - 1 - i; };
    auto load = [&](int64_t k, float (&v)[U], double (&sd)[U]) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < U; ++j) {
            const int64_t c = min(max<int64_t>(chunk(k, j), 0), nc - 1);
            v[j] = buf[base + c * st];
            sd[j] = p.sdel[sbase + c * p.D];
        }
    };
    float V = 0.f;  // H (dir 0) or M (dir 1)
    if (dir == 0 && p.h0) V = p.h0[(bb * p.D + d) * p.N + n];
    const bool wps = dir == 0 && p.psum != nullptr && n == 0;
    const int64_t pbase = bb * (nc + 1) * p.D + d;
    double ps = 0.0;
    auto consume = [&](int64_t k, const float (&v)[U], const double (&sd)[U]) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < U; ++j) {
            const int64_t i = k * U + j;
            if (i < nc) {
                const int64_t c = chunk(k, j);
                buf[base + c * st] = V;
                V = fmaf(fexp2(cn * static_cast<float>(sd[j])), V, v[j]);
                if (wps) {
                    p.psum[pbase + c * p.D] = ps;
                    ps += sd[j];
                }
            }
        }
    };
    const int64_t nblk = (nc + U - 1) / U;
    float va[U], vb[U];
    double sa[U], sb[U];
    load(0, va, sa);
    for (int64_t k = 0; k < nblk; k += 2) {
        load(k + 1, vb, sb);
        consume(k, va, sa);
        if (k + 1 >= nblk) break;
        load(k + 2, va, sa);
        consume(k + 1, vb, sb);
    }
    if (dir == 0) {
        if (wps) p.psum[pbase + nc * p.D] = ps;
        if (p.h_last) p.h_last[(bb * p.D + d) * p.N + n] = V;
    } else if (p.dh0) {
        p.dh0[(bb * p.D + d) * p.N + n] = V;
    }
}

// Grid of k_carry: 8 x (units per XCD) x (groups of 4 states).
inline dim3 carry_grid(const ScanProblem& p) {
    const int64_t nunits = 2 * p.nb * ((p.D + 63) / 64);
    return dim3(static_cast<unsigned>(8 * ((nunits + 7) / 8) * ((p.N + 3) / 4)));
}

// ---------------------------------------------------------------------------
// k_forward: grid (ceil(D/64), nc, b), one wave per workgroup; as in
// k_chunk_aggr each lane owns one channel and all 16 of its states, recomputed
// from the chunk carry-in H_c, with B and C through scalar loads (one step
// ahead) and the raw inputs through the chunk's buffer resources (one group
// ahead; the steps after the last whole group run one by one).
// y_t = sum_n C_t h_t (times silu(z_t) with the gate): four partial sums of four
// states each, (S0 + S1) + (S2 + S3).
// ---------------------------------------------------------------------------
template <typename TI, bool SP, bool GATE, bool N16>
__global__ __launch_bounds__(64) void k_forward(const ScanProblem p) {
    constexpr int G = 4;  // steps per group
    const int lane = threadIdx.x;
    const int64_t d = static_cast<int64_t>(blockIdx.x) * 64 + lane;
    const int64_t c = blockIdx.y, bb = blockIdx.z;
    const bool dv = d < p.D;
    float cn[16];
    lane_rates16(p, d, dv, cn);
    const int64_t cb = (bb * p.nc + c) * p.N * p.D + d;
    float h[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) h[k] = ldm(p.hbuf, cb + k * p.D, dv && k < p.N);
    const int64_t t0 = c * p.L;
    const int64_t t1 = min(t0 + p.L, p.T);
    const int64_t rowb = bb * p.T;
    const TI* Bp = static_cast<const TI*>(p.B);
    const TI* Cp = static_cast<const TI*>(p.C);
    const int nl = static_cast<int>(t1 - t0);
    ChunkRows<TI> cr;
    cr.init(p, rowb + t0, nl, d, dv);
    // y of the chunk's rows through a buffer resource like the inputs' (padding
    // channels store out of range, which writes nothing: no branch around the stores)
    const __amdgpu_buffer_rsrc_t rY = __builtin_amdgcn_make_buffer_rsrc(
        static_cast<TI*>(p.y) + (rowb + t0) * p.D, 0, static_cast<int>(nl * p.D * sizeof(TI)), 0x00020000);
    auto step = [&](int tl, float xr, float pr, float zr, const SRow<TI, N16>& cB,
                    const SRow<TI, N16>& cC) __attribute__((always_inline)) {
        const float dl = SP ? softplus_f(pr) : pr;
        if (p.bdelta) xr *= dl;  // input term Delta B x
        float yq[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            float yp = 0.f;
#pragma unroll
            for (int k = 4 * i; k < 4 * i + 4; ++k) {
                h[k] = fmaf(fexp2(cn[k] * dl), h[k], cB.at(k) * xr);
                yp = fmaf(cC.at(k), h[k], yp);
            }
            yq[i] = yp;
        }
        float y = (yq[0] + yq[1]) + (yq[2] + yq[3]);
        if constexpr (GATE) y *= zr * sigmoid_f(zr);
        if constexpr (sizeof(TI) == 2)
            __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(uint16_t, static_cast<__bf16>(y)), rY, cr.voff,
                                                  tl * cr.rowbytes, 0);
        else
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(y), rY, cr.voff, tl * cr.rowbytes, 0);
    };
    const int ngrp = nl / G;
    RawIn<TI, G> raw;
    auto load_slot = [&](int tl, int j) __attribute__((always_inline)) {
        const int tc = min(tl, nl - 1);
        raw.x[j] = cr.ld(cr.x, tc);
        raw.p[j] = cr.ld(cr.p, tc);
        raw.z[j] = GATE ? cr.ld(cr.z, tc) : 0;
    };
    SRow<TI, N16> nB, nC;
    if (ngrp > 0) {
#pragma unroll
        for (int j = 0; j < G; ++j) {
            load_slot(j, j);
            __builtin_amdgcn_sched_barrier(0);  // issued in the loop's order: the waits at its head count these
        }
        nB.load(Bp, rowb + t0, p.N);
        nC.load(Cp, rowb + t0, p.N);
    }
    for (int gi = 0; gi < ngrp; ++gi) {
#pragma unroll
        for (int j = 0; j < G; ++j) {
            const int t = gi * G + j;
            // converted before the slot is refilled (see k_chunk_aggr); the scheduling
            // barriers keep the refills a full group ahead of their use (left free, the
            // scheduler sinks them next to it)
            const float xr = ChunkRows<TI>::cvt(raw.x[j]), pr = ChunkRows<TI>::cvt(raw.p[j]);
            const float zr = GATE ? ChunkRows<TI>::cvt(raw.z[j]) : 0.f;
            __builtin_amdgcn_sched_barrier(0);
            load_slot(t + G, j);
            const SRow<TI, N16> cB = nB, cC = nC;
            const int64_t rn = rowb + t0 + min(t + 1, nl - 1);
            nB.load(Bp, rn, p.N);
            nC.load(Cp, rn, p.N);
            __builtin_amdgcn_sched_barrier(0);  // the loads stay ahead of the step's arithmetic
            step(t, xr, pr, zr, cB, cC);
        }
    }
    for (int t = ngrp * G; t < nl; ++t) {
        SRow<TI, N16> cB, cC;
        cB.load(Bp, rowb + t0 + t, p.N);
        cC.load(Cp, rowb + t0 + t, p.N);
        step(t, ChunkRows<TI>::cvt(cr.ld(cr.x, t)), ChunkRows<TI>::cvt(cr.ld(cr.p, t)),
             GATE ? ChunkRows<TI>::cvt(cr.ld(cr.z, t)) : 0.f, cB, cC);
    }
}

// ---------------------------------------------------------------------------
// k_forward_quad: the forward of k_forward for small grids (see aggr_quad): grid
// (ceil(D/64), nc, b), 256 threads; as in k_chunk_aggr_quad the 4 lanes of a quad
// share a channel and hold 4 of its states.  y_t = sum_n C_t h_t
// (times silu(z_t) with the gate), the state recomputed from the chunk carry-in
// H_c.  B and C are staged in LDS 64 steps at a time for the workgroup; lane r
// prepares the per-channel quantities of step s0+r of each group of 4 steps and
// broadcasts them to its quad (its raw inputs loaded one group ahead); the
// quad's sum over its states gives y_t, which the lane that prepared step t
// finishes and stores.  Steps past the end of the chunk have Delta = x = 0 and
// B = C = 0, so every group runs (no tail branch around the arithmetic).
// ---------------------------------------------------------------------------
template <typename TI, bool SP, bool GATE>
__global__ __launch_bounds__(256) void k_forward_quad(const ScanProblem p) {
    constexpr int SB = 64;             // steps per staged block
    constexpr int PT = SB * 32 / 256;  // staged values per thread
    __shared__ __attribute__((aligned(16))) float bcs[SB][32];
    const int tid = threadIdx.x;
    const int r = tid & 3;
    const int64_t d = static_cast<int64_t>(blockIdx.x) * 64 + (tid >> 2);
    const int64_t c = blockIdx.y, bb = blockIdx.z;
    const bool dv = d < p.D;
    const TI* Bp = static_cast<const TI*>(p.B);
    const TI* Cp = static_cast<const TI*>(p.C);
    TI* Y = static_cast<TI*>(p.y);
    float cn[4], wn[4];
    lane_consts(p.A_log, d, r, p.N, dv, p.ascalar, cn, wn);
    const int64_t cb = ((bb * p.nc + c) * p.N + r * 4) * p.D + d;
    float h[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) h[k] = ldm(p.hbuf, cb + k * p.D, dv && r * 4 + k < p.N);
    const int64_t t0 = c * p.L;
    const int64_t t1 = min(t0 + p.L, p.T);
    RawIn<TI, 1> nb;
    load_raw<TI, GATE, 1>(p, bb, t0, d, dv, r, false, nb);
    uint32_t zb = 0;
    if constexpr (GATE) zb = ldbits(static_cast<const TI*>(p.z), dv && t0 + r < p.T ? (bb * p.T + t0 + r) * p.D + d : 0);
    for (int64_t sb = t0; sb < t1; sb += SB) {
        // the block's loads all issued before any is used (raw bits, masks
        // applied at the store)
        typename RawIn<TI, 1>::Bits bcv[PT];
        uint32_t bcm[PT];
#pragma unroll
        for (int e = 0; e < PT; ++e) {
            const int i = tid + 256 * e;
            const int t = i >> 5, cc = i & 31, n = cc & 15;
            const int64_t tg = sb + t;
            const bool ok = tg < t1 && n < p.N;
            bcm[e] = ok ? 0xffffffffu : 0u;
            bcv[e] = ldbits(cc < 16 ? Bp : Cp, ok ? (bb * p.T + tg) * p.N + n : 0);
        }
        __builtin_amdgcn_sched_barrier(0);
        lds_barrier();  // the previous block's reads are done
#pragma unroll
        for (int e = 0; e < PT; ++e) {
            const int i = tid + 256 * e;
            const uint32_t b = sizeof(TI) == 2 ? static_cast<uint32_t>(bcv[e]) << 16 : static_cast<uint32_t>(bcv[e]);
            bcs[i >> 5][i & 31] = __uint_as_float(b & bcm[e]);
        }
        lds_barrier();
        const int64_t se = min(sb + SB, t1);
        for (int64_t s0 = sb; s0 < se; s0 += 4) {
            // this group's inputs, then the next group's loads
            const bool v = dv && s0 + r < t1;
            const float pr = fin<TI>(nb.p[0], v);
            float xr = fin<TI>(nb.x[0], v);
            float zr = 0.f;
            if constexpr (GATE) zr = fin<TI>(zb, v);
            load_raw<TI, GATE, 1>(p, bb, s0 + 4, d, dv, r, false, nb);
            if constexpr (GATE) {
                const int64_t tz = s0 + 4 + r;
                zb = ldbits(static_cast<const TI*>(p.z), dv && tz < p.T ? (bb * p.T + tz) * p.D + d : 0);
            }
            const float dlr = SP ? softplus_sel(pr, v) : pr;
            if (p.bdelta) xr *= dlr;  // input term Delta B x
            float ypart[4];
            const int tb = static_cast<int>(s0 - sb);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const float xv = quad_bcast(xr, j);
                const float dl = quad_bcast(dlr, j);
                const float4 b4 = *reinterpret_cast<const float4*>(&bcs[tb + j][4 * r]);
                const float4 c4 = *reinterpret_cast<const float4*>(&bcs[tb + j][16 + 4 * r]);
                const float Bv[4] = {b4.x, b4.y, b4.z, b4.w};
                const float Cv[4] = {c4.x, c4.y, c4.z, c4.w};
                float yp = 0.f;
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    h[k] = fmaf(fexp2(cn[k] * dl), h[k], Bv[k] * xv);
                    yp = fmaf(Cv[k], h[k], yp);
                }
                ypart[j] = yp;
            }
            float yk = quad_sum_transposed(ypart, r);  // y of step s0 + r
            if constexpr (GATE) yk *= zr * sigmoid_f(zr);
            if (v) stf(Y, (bb * p.T + s0 + r) * p.D + d, yk);
        }
    }
}

// ---------------------------------------------------------------------------
// B_t and C_t of one chunk, staged in LDS as fp32 once per workgroup and read
// by all of its waves.  Row t holds B (states 0..15) then C; padding is zero.
// ---------------------------------------------------------------------------
template <typename TI, int L>
struct __attribute__((aligned(16))) BCStage {
    float w[L][32];

    // NTH threads; each issues all of its loads (raw element bits) before it
    // masks and writes any to LDS (the scheduling barrier keeps the compiler from
    // placing each load's wait and use right behind it).
    template <int NTH>
    __device__ __forceinline__ void load(const ScanProblem& p, int64_t bb, int64_t t0, int tid) {
        constexpr int PT = (L * 32 + NTH - 1) / NTH;
        const TI* Bp = static_cast<const TI*>(p.B);
        const TI* Cp = static_cast<const TI*>(p.C);
        typename RawIn<TI, 1>::Bits v[PT];
        uint32_t mk[PT];
#pragma unroll
        for (int e = 0; e < PT; ++e) {
            const int i = tid + NTH * e;
            const int t = i >> 5, c = i & 31, n = c & 15;
            const int64_t tg = t0 + t;
            const bool ok = i < L * 32 && tg < p.T && n < p.N;
            mk[e] = ok ? 0xffffffffu : 0u;
            v[e] = ldbits(c < 16 ? Bp : Cp, ok ? (bb * p.T + tg) * p.N + n : 0);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int e = 0; e < PT; ++e) {
            const int i = tid + NTH * e;
            const uint32_t b = sizeof(TI) == 2 ? static_cast<uint32_t>(v[e]) << 16 : static_cast<uint32_t>(v[e]);
            if ((L * 32) % NTH == 0 || i < L * 32) w[i >> 5][i & 31] = __uint_as_float(b & mk[e]);
        }
    }
    // States 4r..4r+3 of B and C at in-chunk step t.
    __device__ __forceinline__ void get(int t, int r, float Bv[4], float Cv[4]) const {
        const float4 b = *reinterpret_cast<const float4*>(&w[t][4 * r]);
        const float4 c = *reinterpret_cast<const float4*>(&w[t][16 + 4 * r]);
        Bv[0] = b.x; Bv[1] = b.y; Bv[2] = b.z; Bv[3] = b.w;
        Cv[0] = c.x; Cv[1] = c.y; Cv[2] = c.z; Cv[3] = c.w;
    }
    __device__ __forceinline__ void getB(int t, int r, float Bv[4]) const {
        const float4 b = *reinterpret_cast<const float4*>(&w[t][4 * r]);
        Bv[0] = b.x; Bv[1] = b.y; Bv[2] = b.z; Bv[3] = b.w;
    }
};

// One chunk's rows of a [b*T][ld] tensor for the quad layout of k_grad: a buffer
// resource over the rows that exist; the lane of channel d at quad position r
// reaches row tq + r + 4jj of a segment at its fixed byte offset d*el + r*rb (rb:
// bytes per row) plus the scalar (tq + 4jj)*rb.  Padding channels, and rows past
// the resource, take offsets with bit 31 set, past every range: loads read zero and
// stores write nothing, with no branch and no address arithmetic per access.  Byte
// offsets within a chunk fit 31 bits (L <= 256 rows of at most 2^20 fp32 values,
// or of the bf16 copies' strides).
struct QuadRows {
    static constexpr uint32_t kOff = 0x80000000u;
    __amdgpu_buffer_rsrc_t rs;
    int rb;
    __device__ __forceinline__ void init(const void* base, int64_t row0, int64_t rows, int64_t ld, int el) {
        rb = static_cast<int>(ld * el);
        rs = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<char*>(static_cast<const char*>(base)) + row0 * ld * el, 0,
            static_cast<int>(max<int64_t>(0, rows) * rb), 0x00020000);
    }
    __device__ __forceinline__ uint32_t lane(uint32_t d, int r, int el, bool dv) const {
        return dv ? d * static_cast<uint32_t>(el) + static_cast<uint32_t>(r * rb) : kOff;
    }
    __device__ __forceinline__ void st(uint32_t vo, int row, float v, std::true_type /*bf16*/) const {
        __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(uint16_t, static_cast<__bf16>(v)), rs, vo, row * rb, 0);
    }
    __device__ __forceinline__ void st(uint32_t vo, int row, float v, std::false_type /*fp32*/) const {
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), rs, vo, row * rb, 0);
    }
};

// The [b][T][D] inputs x, Delta, dy, z of one chunk (or of the chunk's steps shifted
// by the window) in the quad layout.
template <typename TI>
struct QuadIn {
    QuadRows x, p, dy, z;
    int rows;  // rows that exist
    __device__ __forceinline__ void init(const ScanProblem& q, int64_t row0, int64_t nrows) {
        const int64_t n = min<int64_t>(max<int64_t>(nrows, 0), 1 << 20);
        rows = static_cast<int>(n);
        x.init(q.x, row0, n, q.D, sizeof(TI));
        p.init(q.delta, row0, n, q.D, sizeof(TI));
        dy.init(q.dy ? q.dy : q.x, row0, n, q.D, sizeof(TI));
        z.init(q.z ? q.z : q.x, row0, n, q.D, sizeof(TI));
    }
    __device__ __forceinline__ uint32_t ld(const QuadRows& t, uint32_t vo, int so) const {
        if constexpr (sizeof(TI) == 2) return __builtin_amdgcn_raw_buffer_load_b16(t.rs, vo, so, 0);
        else return __builtin_amdgcn_raw_buffer_load_b32(t.rs, vo, so, 0);
    }
    // raw bits of the steps tq + r + 4jj this lane prepares (vb: its byte offset);
    // steps past the rows that exist read zero
    template <bool GATE, int SPL>
    __device__ __forceinline__ void load(uint32_t vb, int tq, int r, RawIn<TI, SPL>& o) const {
#pragma unroll
        for (int jj = 0; jj < SPL; ++jj) {
            const uint32_t vo = tq + r + 4 * jj < rows ? vb : QuadRows::kOff;
            const int so = (tq + 4 * jj) * x.rb;
            o.x[jj] = ld(x, vo, so);
            o.p[jj] = ld(p, vo, so);
            o.dy[jj] = ld(dy, vo, so);
            o.z[jj] = GATE ? ld(z, vo, so) : 0;
        }
    }
};

// The same inputs at the window-shifted steps (truncated mode) through wave-uniform
// base pointers and 32-bit lane offsets: a 64-bit address add per load, but two
// scalar registers per tensor where a buffer resource takes four (the truncated
// kernel's scalar registers are all in use, and resources it spills come back as
// per-lane values whose loads the compiler serialises over their distinct values).
// Lanes whose step (tl >= lim) or channel is padding load element 0 and the caller
// masks the value.
template <typename TI>
struct QuadInPtr {
    const TI* p;
    const TI* dy;
    const TI* z;
    __device__ __forceinline__ void init(const ScanProblem& q, int64_t row) {
        const int64_t base = row * q.D;
        p = static_cast<const TI*>(q.delta) + base;
        dy = static_cast<const TI*>(q.dy) + base;
        z = static_cast<const TI*>(q.z ? q.z : q.delta) + base;
    }
    template <bool GATE, int SPL>
    __device__ __forceinline__ void load(uint32_t D, uint32_t d, int tq, int r, int64_t lim, bool dv,
                                         RawIn<TI, SPL>& o) const {
#pragma unroll
        for (int jj = 0; jj < SPL; ++jj) {
            const int tl = tq + r + 4 * jj;
            const uint32_t off = dv && tl < lim ? static_cast<uint32_t>(tl) * D + d : 0u;
            o.x[jj] = 0;
            o.p[jj] = ldbits(p, off);
            o.dy[jj] = ldbits(dy, off);
            o.z[jj] = GATE ? ldbits(z, off) : 0;
        }
    }
};

// Orders one wave's LDS writes before its own later LDS reads of other lanes'
// data (LDS executes a wave's operations in order; this only stops the compiler
// from moving them).
__device__ __forceinline__ void wave_lds_sync() { __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront"); }

// ---------------------------------------------------------------------------
// k_grad: grid (nsplit, nc, b), kGradWaves waves per workgroup.  The workgroup
// owns carry chunk c (L = S*NCK steps) and the 16-channel tiles of its split;
// wave w takes tiles tile_lo + w, tile_lo + w + kGradWaves, ..., so the waves
// read adjacent channels together.  Lanes of a quad share a channel and hold 4
// of its states.  B and C of the chunk are staged in LDS once.  Per tile:
//   1. the state at the start of each S-step segment is the chunk-local one
//      from the chunk-aggregate pass (hseg) plus the carry-in H_c decayed over
//      the steps before the segment (2^{cn cseg});
//   2. segments in reverse order: recompute the segment's states forward
//      (keeping a_t and a_t h_{t-1}), form dz, sum g_t h_t over the channels
//      (dC); then run the adjoint backwards, mu_t = g_t C_t + a_{t+1} mu_{t+1},
//      from the chunk's reverse carry M_c, and apply the vjp epilogue:
//        s = mubar a_t h_{t-1};  ddelta = sum_n s wn;  dA_log += s Delta wn;
//        dx = sum_n mubar B_t;  dB_t[n] += mubar x_t (over channels).
//      Truncated mode: the windowed adjoint mubar_t = sum_{s=t}^{t+tbar-1} g_s C_s
//      P(t, s) obeys its own recurrence, mubar_t = g_t C_t + a_{t+1} mubar_{t+1}
//      - P(t, t+tbar) g_{t+tbar} C_{t+tbar} (the step that leaves the window is
//      taken out as it leaves), so it is carried at its own magnitude and never
//      formed as the difference of two full-horizon adjoints.  Its value entering
//      the chunk from the right, a_{e+1} mubar_{e+1}, is summed directly over the
//      steps (e, e+tbar] when the window is shorter than the chunk; longer windows
//      take M_c - P(e, e+tbar) a_{e+tbar+1} mu_{e+tbar+1}, with the full adjoint
//      carry at the shifted position (that of the chunk holding it, swept back to
//      it); P(t, t+tbar) = 2^{cn W_t} with the window sum W_t = sum_{j=t+1}^{t+tbar}
//      Delta_j kept in fp64.
// Per-channel quantities (softplus, the gate) are computed once per step: lane
// r of a quad prepares steps r, r+4, ... of the segment, DPP-broadcasts them,
// keeps that step's per-channel outputs and stores them after the segment; the
// next segment's raw inputs are loaded ahead.
// Sums over channels of dB/dC: each wave sums its 16 channels per (step, state)
// through LDS, the wave sums are added in wave order into a chunk accumulator
// in LDS, and the workgroup writes the accumulator once at the end (into dB/dC,
// or into its split's partial when nsplit > 1).  All orders are fixed.
// ---------------------------------------------------------------------------
template <typename TI, bool SP, bool GATE, bool TRUNC, bool N16, int S, int NCK, int OUT>
__global__ __launch_bounds__(64 * kGradWaves) __attribute__((amdgpu_waves_per_eu(2, 8))) void k_grad(const ScanProblem p) {
    constexpr int NW = kGradWaves;
    constexpr int NTH = 64 * NW;
    constexpr int L = S * NCK;
    constexpr int SPL = S / 4;  // steps each lane prepares per segment
    constexpr int NP = S * 16;  // (step, state) pairs of a segment
    static_assert(NP % 64 == 0 && NP <= NTH, "pair layout");
    // LDS per workgroup, two per CU: up to 128-step chunks 80 KB: the chunk's B and C,
    // channel-sum rows padded to 20 (free of bank conflicts; the spare column holds
    // the window-shifted C); longer chunks (RING) 76 KB: B and C in a ring of two
    // segments refilled one segment ahead, unpadded rows, shifted C in rows of its own
    // (at 128 steps the ring and the unpadded rows cost 10 %)
    constexpr bool RING = L > 128;
    __shared__ BCStage<TI, RING ? 2 * S : L> bc;
    __shared__ __attribute__((aligned(16))) float red[NW][S][16][RING ? 16 : 20];  // per wave [step][state][channel]
    __shared__ __attribute__((aligned(16))) float csh[(RING && TRUNC && N16) ? NW : 1][S][16];  // per wave: shifted C
    __shared__ float wsum[4][NW][NP];  // per-wave channel sums: (dC, dB) of a segment, two segments alternating
    __shared__ float acc[L][32];       // chunk totals: dB in columns 0..15, dC in 16..31
    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63;
    const int r = lane & 3, chl = lane >> 2;
    // Column of this lane's channel in red[]: rows of states 8..15 hold the two
    // 8-channel halves swapped, so that the lanes of a quad (rows 20 floats
    // apart) write distinct banks; the 16-channel sum tree in flush adds the two
    // halves last, so the swap leaves every sum unchanged.
    const int chs = chl ^ ((r & 2) << 2);
    const int64_t c = blockIdx.y, bb = blockIdx.z;
    const int split = blockIdx.x;
    const int64_t t0 = c * L;
    const int64_t lim = p.T - t0;  // in-chunk steps tl < lim are real
    const int64_t row0 = bb * p.T + t0;
    QuadIn<TI> qin;  // the chunk's inputs
    qin.init(p, row0, min<int64_t>(L, lim));
    // Per-step outputs over the same rows.  OUT 1: also write the bf16 copies of
    // ddelta and dz (and of dx when dx16 is given); OUT 2: write only the bf16
    // copies of dx, ddelta and dz (no fp32 dx, ddelta and dz), for callers that want
    // only the projection GEMMs' operands.  Outputs a variant does not write get an
    // empty resource.
    constexpr bool OUT16 = OUT > 0;
    auto out_rows = [&](const void* ptr, int64_t ld, int el) {
        QuadRows o;
        o.init(ptr ? ptr : p.x, row0, ptr ? qin.rows : 0, ld, el);
        return o;
    };
    const QuadRows odx = out_rows(OUT != 2 ? p.dx : nullptr, p.D, 4);
    const QuadRows odd = out_rows(OUT != 2 ? p.ddelta : nullptr, p.D, 4);
    const QuadRows odz = out_rows(OUT != 2 && GATE ? p.dz : nullptr, p.D, 4);
    const QuadRows o16x = out_rows(OUT16 ? p.dx16 : nullptr, p.ld_dx16, 2);
    const QuadRows o16d = out_rows(OUT16 ? p.dd16 : nullptr, p.ld_dd16, 2);
    const QuadRows o16z = out_rows(OUT16 ? p.dz16 : nullptr, p.ld_dz16, 2);
    // Padding lanes of the per-tile dA_log store write into the sink instead, so
    // that the store is issued without a branch.
    float* const sinkf = p.sink + lane;

    const int64_t ntile = (p.D + 15) / 16;
    const int64_t tile_lo = static_cast<int64_t>(split) * p.tps;
    const int64_t tile_hi = min(ntile, tile_lo + p.tps);
    const int64_t nit = (tile_hi - tile_lo + NW - 1) / NW;  // the same for every wave

    // truncated mode: the chunk's steps shifted by tbar, and (16 states) a buffer
    // resource over the rows of C at the shifted steps that exist
    QuadInPtr<TI> qis;
    int64_t lims = 0;
    if constexpr (TRUNC) {
        lims = p.T - (t0 + p.tbar);
        qis.init(p, bb * p.T + min(t0 + p.tbar, p.T - 1));
    }
    const uint32_t D32 = static_cast<uint32_t>(p.D);
    const int64_t c_rows = (TRUNC && N16) ? max<int64_t>(0, min<int64_t>(L, lims)) : 0;
    const __amdgpu_buffer_rsrc_t rsC = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<TI*>(static_cast<const TI*>(p.C) + (bb * p.T + min(t0 + p.tbar, p.T)) * 16), 0,
        static_cast<int>(c_rows * 16 * static_cast<int64_t>(sizeof(TI))), 0x00020000);

    // The ring's rows of segment qs (in-chunk steps qs*S ..) go to slot qs & 1: each
    // thread fetches its raw element bits one segment ahead and writes them (masked)
    // before the barrier that ends the segment (NCK is even, so the first segment of
    // the next tile, NCK - 1, follows segment 0 in the other slot).
    constexpr int BPT = (S * 32 + NTH - 1) / NTH;
    typename RawIn<TI, 1>::Bits bcv[BPT];
    auto bc_ok = [&](int qs, int e) {
        const int i = tid + NTH * e, n = i & 15;
        return i < S * 32 && t0 + qs * S + (i >> 5) < p.T && n < p.N;
    };
    auto bc_fetch = [&](int qs) {
        const TI* Bp = static_cast<const TI*>(p.B);
        const TI* Cp = static_cast<const TI*>(p.C);
#pragma unroll
        for (int e = 0; e < BPT; ++e) {
            const int i = tid + NTH * e;
            bcv[e] = ldbits((i & 31) < 16 ? Bp : Cp,
                            bc_ok(qs, e) ? (bb * p.T + t0 + qs * S + (i >> 5)) * p.N + (i & 15) : 0);
        }
    };
    auto bc_put = [&](int qs) {
#pragma unroll
        for (int e = 0; e < BPT; ++e) {
            const int i = tid + NTH * e;
            const uint32_t b = sizeof(TI) == 2 ? static_cast<uint32_t>(bcv[e]) << 16 : static_cast<uint32_t>(bcv[e]);
            if ((S * 32) % NTH == 0 || i < S * 32)
                bc.w[(qs & 1) * S + (i >> 5)][i & 31] = __uint_as_float(bc_ok(qs, e) ? b : 0u);
        }
    };
    static_assert(!RING || NCK % 2 == 0, "the ring alternates slots across tiles");

    for (int i = tid; i < L * 32; i += NTH) (&acc[0][0])[i] = 0.f;
    if constexpr (RING) {
        bc_fetch(NCK - 1);  // the first segment the tiles run
        bc_put(NCK - 1);
    } else {
        bc.template load<NTH>(p, bb, t0, tid);
    }
    __syncthreads();

    int pair = 0;
    // Channel sums of red[wave] (16 channels per (step, state) pair of the
    // segment) into this wave's slot of wsum; every wave calls it.
    auto wave_sums = [&](int slot) {
        wave_lds_sync();
#pragma unroll
        for (int i = 0; i < NP / 64; ++i) {
            const int o = lane + 64 * i;
            const int j = o >> 4, n = o & 15;
            const float4 a0 = *reinterpret_cast<const float4*>(&red[wave][j][n][0]);
            const float4 a1 = *reinterpret_cast<const float4*>(&red[wave][j][n][4]);
            const float4 a2 = *reinterpret_cast<const float4*>(&red[wave][j][n][8]);
            const float4 a3 = *reinterpret_cast<const float4*>(&red[wave][j][n][12]);
            wsum[slot][wave][o] = (((a0.x + a0.y) + (a0.z + a0.w)) + ((a1.x + a1.y) + (a1.z + a1.w))) +
                                  (((a2.x + a2.y) + (a2.z + a2.w)) + ((a3.x + a3.y) + (a3.z + a3.w)));
        }
    };
    // After both halves of segment q: one barrier, then the wave sums of dC
    // (slot 2 pair) and dB (slot 2 pair + 1) are added in wave order into acc.
    // The two pairs of slots alternate between segments, so a fast wave writing
    // the next segment's sums never meets a slow wave still reading these.
    auto flush = [&](int q) {
        lds_barrier();
        for (int o2 = tid; o2 < 2 * NP; o2 += NTH) {
            const int half = o2 >= NP ? 1 : 0, o = o2 - half * NP;
            const int slot = 2 * pair + half;
            float sum = wsum[slot][0][o];
#pragma unroll
            for (int w = 1; w < NW; ++w) sum += wsum[slot][w][o];
            acc[q * S + (o >> 4)][(half ? 0 : 16) + (o & 15)] += sum;
        }
        pair ^= 1;
    };

    for (int64_t it = 0; it < nit; ++it) {
        const int64_t tile = tile_lo + it * NW + wave;
        const int64_t d = tile * 16 + chl;
        const bool dv = tile < tile_hi && d < p.D;
        float cn[4], wn[4];
        lane_consts(p.A_log, d, r, p.N, dv, p.ascalar, cn, wn);
        bool nv[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) nv[k] = dv && (r * 4 + k < p.N);
        const int64_t cb = ((bb * p.nc + c) * p.N + r * 4) * p.D + d;
        const uint32_t d32 = dv ? static_cast<uint32_t>(d) : 0u;
        // the lane's byte offsets (row r of a quad's step group, channel d) in the
        // inputs, the fp32 outputs and the bf16 copies
        const uint32_t vbi = qin.x.lane(d32, r, sizeof(TI), dv);
        const uint32_t vbo = odx.lane(d32, r, 4, dv);
        const uint32_t vbx16 = o16x.lane(d32, r, 2, dv), vbd16 = o16d.lane(d32, r, 2, dv);
        const uint32_t vbz16 = o16z.lane(d32, r, 2, dv);

        // inputs of the last segment, for the reverse sweep
        RawIn<TI, SPL> nxt;
        RawIn<TI, SPL> nxs;  // raw inputs at the shifted positions (truncated mode)
        qin.template load<GATE, SPL>(vbi, (NCK - 1) * S, r, nxt);
        if constexpr (TRUNC) qis.template load<GATE, SPL>(D32, d32, (NCK - 1) * S, r, lims, dv, nxs);
        using SC = ShiftedC<TI, S>;
        typename SC::Raw nxc{};  // shifted C rows of the next segment (truncated mode, 16 states)
        if constexpr (TRUNC && N16) nxc = SC::load(rsC, NCK - 1, lane);

        // segment-start states: hseg[q] + (prod of a from the chunk start) H_c, the
        // product being 2^{cn cseg[q]}; loaded one segment ahead
        float Hc[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) Hc[k] = ldm(p.hbuf, cb + k * p.D, nv[k]);
        const int64_t sgb = (bb * p.nc + c) * NCK * p.Dp + (dv ? d : 0);
        float4 hq = *reinterpret_cast<const float4*>(p.hseg + (sgb + (NCK - 1) * p.Dp) * 16 + 4 * r);
        float cq = p.cseg[sgb + (NCK - 1) * p.Dp];
        float h[4];

        // 2. reverse over segments
        float Mp[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) Mp[k] = ldm(p.mbuf, cb + k * p.D, nv[k]);
        float dA[4] = {0.f, 0.f, 0.f, 0.f};

        // truncated-mode state: the swept adjoint carry and the window sum
        float Msh[4] = {0.f, 0.f, 0.f, 0.f};
        double W = 0.0;
        if constexpr (TRUNC) {
            const TI* Cp = static_cast<const TI*>(p.C);
            const int64_t tb = p.tbar;
            const int64_t e = t0 + L - 1;  // the chunk's last step
            const int64_t pstart = e + tb;
            const int64_t pb = bb * (p.nc + 1) * p.D + d;
            // Windows shorter than the chunk: the carry a_{e+1} mubar_{e+1} = sum over
            // s in (e, e+tbar] of g_s C_s P(e, s) is summed directly over those steps
            // from zero (no difference of full-horizon adjoints at all).  Longer
            // windows: the full adjoint carry of the chunk holding e+tbar, swept back
            // to it, is subtracted from the chunk's own carry below.
            const bool direct = tb < L;
            int64_t cpk = 0, sw_hi = e, sw_lo = e;  // the sweep covers steps (sw_lo, sw_hi]
            if (direct) {
                sw_hi = pstart;
            } else if (pstart < p.T) {
                cpk = pstart / L;
                sw_hi = (cpk + 1) * L - 1;
                sw_lo = pstart;
                const int64_t mb = ((bb * p.nc + cpk) * p.N + r * 4) * p.D + d;
#pragma unroll
                for (int k = 0; k < 4; ++k) Msh[k] = ldm(p.mbuf, mb + k * p.D, nv[k]);
            }
            {
                // steps sw_hi down to sw_lo + 1, eight at a time: the loads of a batch
                // (from clamped, always valid addresses) are issued before its
                // arithmetic, and steps outside the sweep are masked to exact no-ops
                // (Delta = g = C = 0 leave Msh and the Delta sum unchanged) with bit
                // masks: selecting a loaded value instead lets the compiler turn the
                // select into a branch around the load, whose merge then waits for it.
                const TI* DL = static_cast<const TI*>(p.delta);
                const TI* DY = static_cast<const TI*>(p.dy);
                const TI* Z = static_cast<const TI*>(p.z);
                constexpr int PB = 8;
                double pre = 0.0;
                for (int64_t p0 = sw_hi; p0 > sw_lo; p0 -= PB) {
                    typename RawIn<TI, PB>::Bits prb[PB], gyb[PB], zb[PB];
                    uint32_t mk[PB];
                    // raw C bits: 4 bf16 (two words) or 4 fp32 words per step
                    uint32_t cw[PB][sizeof(TI) == 2 ? 2 : 4];
                    float Cb[PB][4];
#pragma unroll
                    for (int u = 0; u < PB; ++u) {
                        const int64_t ps = p0 - u;
                        const bool ok = dv && ps > sw_lo && ps < p.T;
                        mk[u] = ok ? 0xffffffffu : 0u;
                        const int64_t row = bb * p.T + min(max<int64_t>(ps, 0), p.T - 1);
                        const int64_t td = row * p.D + (dv ? d : 0);
                        prb[u] = ldbits(DL, td);
                        gyb[u] = ldbits(DY, td);
                        zb[u] = GATE ? ldbits(Z, td) : 0;
                        if constexpr (N16) {
                            if constexpr (sizeof(TI) == 2) {
                                const uint2 w = *reinterpret_cast<const uint2*>(Cp + row * 16 + r * 4);
                                cw[u][0] = w.x;
                                cw[u][1] = w.y;
                            } else {
                                const uint4 w = *reinterpret_cast<const uint4*>(Cp + row * 16 + r * 4);
                                cw[u][0] = w.x;
                                cw[u][1] = w.y;
                                cw[u][2] = w.z;
                                cw[u][3] = w.w;
                            }
                        } else {
                            ld4<TI, N16>(Cp, bb * p.T + ps, r, p.N, ok, Cb[u]);
                        }
                    }
                    // keep the batch's loads ahead of its arithmetic
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int u = 0; u < PB; ++u) {
                        const uint32_t m = mk[u];
                        if constexpr (N16) {
                            if constexpr (sizeof(TI) == 2) {
                                Cb[u][0] = __uint_as_float((cw[u][0] << 16) & m);
                                Cb[u][1] = __uint_as_float((cw[u][0] & 0xffff0000u) & m);
                                Cb[u][2] = __uint_as_float((cw[u][1] << 16) & m);
                                Cb[u][3] = __uint_as_float((cw[u][1] & 0xffff0000u) & m);
                            } else {
#pragma unroll
                                for (int k = 0; k < 4; ++k) Cb[u][k] = __uint_as_float(cw[u][k] & m);
                            }
                        }
                        const float pr = fin<TI>(prb[u], true);
                        const float dlp = __uint_as_float(__float_as_uint(SP ? softplus_f(pr) : pr) & m);
                        const float gy = fin<TI>(gyb[u], true);
                        float g0 = gy;
                        if constexpr (GATE) {
                            const float zv = fin<TI>(zb[u], true);
                            g0 = gy * zv * sigmoid_f(zv);
                        }
                        const float gp = __uint_as_float(__float_as_uint(g0) & m);
#pragma unroll
                        for (int k = 0; k < 4; ++k)
                            Msh[k] = fexp2(cn[k] * dlp) * fmaf(gp, Cb[u][k], Msh[k]);
                        pre += static_cast<double>(dlp);
                    }
                }
                if (direct) {
                    W = pre;  // the window's Delta sum, steps past T counting 0
                } else if (dv) {
                    W = pstart < p.T ? (p.psum[pb + cpk * p.D] - p.psum[pb + (c + 1) * p.D]) +
                                           (p.sdel[(bb * p.nc + cpk) * p.D + d] - pre)
                                     : p.psum[pb + p.nc * p.D] - p.psum[pb + (c + 1) * p.D];
                }
            }
            if (direct) {
#pragma unroll
                for (int k = 0; k < 4; ++k) Mp[k] = Msh[k];
            } else {
                // a_{e+1} mubar_{e+1} = a_{e+1} mu_{e+1} - P(e, e+tbar) (a_{e+tbar+1} mu_{e+tbar+1}):
                // one difference of full-horizon adjoints per tile, whose rounding then
                // decays; with windows of a chunk or more the two are of comparable size
                const float wf0 = static_cast<float>(W);
#pragma unroll
                for (int k = 0; k < 4; ++k) Mp[k] = fmaf(-fexp2(cn[k] * wf0), Msh[k], Mp[k]);
            }
        }

        // Everything the tile's prologue loaded is waited for here, once: the waits
        // at the head of the segment loop are computed for the loop's entry and its
        // back edge together, and with the prologue's loads (issued in another
        // order) still in flight they came out as a full drain, every segment, of
        // the next segment's inputs and the last segment's stores.
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0), other counters unchanged
#pragma unroll 1
        for (int q = NCK - 1; q >= 0; --q) {
            {
                const float hl[4] = {hq.x, hq.y, hq.z, hq.w};
#pragma unroll
                for (int k = 0; k < 4; ++k) h[k] = fmaf(fexp2(cn[k] * cq), Hc[k], hl[k]);
                // the next segment's record (segment 0 reloads its own: no branch around the loads)
                const int64_t qn = q > 0 ? q - 1 : 0;
                hq = *reinterpret_cast<const float4*>(p.hseg + (sgb + qn * p.Dp) * 16 + 4 * r);
                cq = p.cseg[sgb + qn * p.Dp];
            }
            const RawIn<TI, SPL> cur = nxt;
            RawIn<TI, SPL> cus;
            if constexpr (TRUNC) cus = nxs;
            {
                // the next segment (segment 0 reloads itself; see the checkpoint sweep)
                const int qn = q > 0 ? q - 1 : 0;
                qin.template load<GATE, SPL>(vbi, qn * S, r, nxt);
                if constexpr (TRUNC) qis.template load<GATE, SPL>(D32, d32, qn * S, r, lims, dv, nxs);
            }
            typename SC::Raw curc{};
            if constexpr (TRUNC && N16) {
                curc = nxc;
                nxc = SC::load(rsC, q > 0 ? q - 1 : 0, lane);
            }
            // per-channel quantities of the steps this lane prepares
            float dls[SPL], xs[SPL], xr[SPL], gs[SPL], gfs[SPL], dlps[SPL], gps[SPL];
            bool sv[SPL];
#pragma unroll
            for (int jj = 0; jj < SPL; ++jj) {
                sv[jj] = dv && q * S + r + 4 * jj < lim;
                // (the loads read zero for padding steps and channels; softplus(0) is not 0)
                const float pr = fin<TI>(cur.p[jj], true), dyr = fin<TI>(cur.dy[jj], true);
                dls[jj] = SP ? softplus_sel(pr, sv[jj]) : pr;
                xr[jj] = fin<TI>(cur.x[jj], true);
                xs[jj] = p.bdelta ? xr[jj] * dls[jj] : xr[jj];  // the input term is (Delta) B x
                if constexpr (GATE) {
                    const float zr = fin<TI>(cur.z[jj], true);
                    const float sg = sigmoid_f(zr);
                    gs[jj] = dyr * zr * sg;
                    gfs[jj] = dyr * sg * (1.f + zr * (1.f - sg));
                } else {
                    gs[jj] = dyr;
                    gfs[jj] = 0.f;
                }
                if constexpr (TRUNC) {
                    const bool vs = dv && q * S + r + 4 * jj < lims;
                    const float psr = fin<TI>(cus.p[jj], vs), dysr = fin<TI>(cus.dy[jj], vs);
                    dlps[jj] = SP ? softplus_sel(psr, vs) : psr;
                    if constexpr (GATE) {
                        const float zsr = fin<TI>(cus.z[jj], vs);
                        gps[jj] = dysr * zsr * sigmoid_f(zsr);
                    } else {
                        gps[jj] = dysr;
                    }
                }
            }

            float ahp[S][4], ah[S][4], gh[S], dlh[S], xh[S];
            float yk[SPL], ypart[4];
#pragma unroll
            for (int jj = 0; jj < SPL; ++jj) yk[jj] = 0.f;
            // B and C are read from LDS one step ahead of their use
            float Bn[4], Cn[4];
            const int brow = RING ? (q & 1) * S : q * S;  // the segment's first staged row
            bc.get(brow, r, Bn, Cn);
#pragma unroll
            for (int j = 0; j < S; ++j) {
                const int tl = q * S + j;
                const float xv = quad_bcast(xs[j >> 2], j & 3);
                const float dl = quad_bcast(dls[j >> 2], j & 3);
                const float g = quad_bcast(gs[j >> 2], j & 3);
                float Bv[4], Cv[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    Bv[k] = Bn[k];
                    Cv[k] = Cn[k];
                }
                if (j + 1 < S) bc.get(brow + j + 1, r, Bn, Cn);
                float yp = 0.f;
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const float av = fexp2(cn[k] * dl);
                    ah[j][k] = av;
                    ahp[j][k] = av * h[k];
                    h[k] = fmaf(Bv[k], xv, ahp[j][k]);
                    if constexpr (GATE) yp = fmaf(Cv[k], h[k], yp);
                    red[wave][j][r * 4 + k][chs] = g * h[k];
                }
                if constexpr (GATE) {
                    ypart[j & 3] = yp;
                    if ((j & 3) == 3) yk[j >> 2] = quad_sum_transposed(ypart, r);  // y of step 4(j/4) + r
                }
                gh[j] = g;
                dlh[j] = dl;
                xh[j] = xv;
            }
            if constexpr (GATE) {
#pragma unroll
                for (int jj = 0; jj < SPL; ++jj) {
                    const int row = q * S + 4 * jj;  // the quad's first row (the lane adds r)
                    const uint32_t m = sv[jj] ? 0u : QuadRows::kOff;
                    const float v = gfs[jj] * yk[jj];
                    if constexpr (OUT != 2) odz.st(vbo | m, row, v, std::false_type{});
                    if constexpr (OUT16) o16z.st(vbz16 | m, row, v, std::true_type{});
                }
            }
            wave_sums(2 * pair);  // dC
            if constexpr (TRUNC && N16) {
                if constexpr (RING) SC::stage(curc, csh[wave], lane);
                else SC::stage(curc, red[wave], lane);
                wave_lds_sync();
            }

            float dxk[SPL], ddk[SPL], dxpart[4], ddpart[4];
#pragma unroll
            for (int jj = 0; jj < SPL; ++jj) dxk[jj] = ddk[jj] = 0.f;
            // the segment's dA_log terms are summed on their own and then added to
            // the tile's sum: the rounding of the sequential sum grows with S + L/S
            // terms instead of L
            float dAs[4] = {0.f, 0.f, 0.f, 0.f};
            if constexpr (RING) bc_fetch(q > 0 ? q - 1 : NCK - 1);  // the next segment's B and C
            bc.get(brow + S - 1, r, Bn, Cn);
#pragma unroll
            for (int j = S - 1; j >= 0; --j) {
                const int tl = q * S + j;
                float Bv[4], Cv[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    Bv[k] = Bn[k];
                    Cv[k] = Cn[k];
                }
                if (j > 0) bc.get(brow + j - 1, r, Bn, Cn);
                float mb[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) mb[k] = fmaf(gh[j], Cv[k], Mp[k]);
                if constexpr (TRUNC) {
                    const int64_t ps = t0 + tl + p.tbar;
                    const bool pv = ps < p.T;
                    const float dlp = quad_bcast(dlps[j >> 2], j & 3);
                    const float gp = quad_bcast(gps[j >> 2], j & 3);
                    float Cs[4];
                    if constexpr (N16) {
                        const float4 c4 = *reinterpret_cast<const float4*>(RING ? &csh[wave][j][4 * r] : &red[wave][j][r][16]);
                        Cs[0] = c4.x; Cs[1] = c4.y; Cs[2] = c4.z; Cs[3] = c4.w;
                    } else {
                        ld4<TI, N16>(static_cast<const TI*>(p.C), bb * p.T + ps, r, p.N, pv, Cs);
                    }
                    const float wf = static_cast<float>(W);
#pragma unroll
                    for (int k = 0; k < 4; ++k)  // the step t+tbar leaves the window
                        mb[k] = fmaf(-fexp2(cn[k] * wf), gp * Cs[k], mb[k]);
                    W += static_cast<double>(dlh[j]) - static_cast<double>(dlp);
                }
                float dxp = 0.f, ddp = 0.f;
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    dxp = fmaf(mb[k], Bv[k], dxp);
                    const float s = mb[k] * ahp[j][k];
                    ddp = fmaf(s, wn[k], ddp);
                    dAs[k] = fmaf(s, dlh[j], dAs[k]);
                    red[wave][j][r * 4 + k][chs] = mb[k] * xh[j];
                    Mp[k] = ah[j][k] * mb[k];
                }
                dxpart[j & 3] = dxp;
                ddpart[j & 3] = ddp;
                if ((j & 3) == 0) {  // the group's last step in reverse order: lane r takes step 4(j/4) + r
                    dxk[j >> 2] = quad_sum_transposed(dxpart, r);
                    ddk[j >> 2] = quad_sum_transposed(ddpart, r);
                }
            }
#pragma unroll
            for (int jj = 0; jj < SPL; ++jj) {
                const int row = q * S + 4 * jj;  // the quad's first row (the lane adds r)
                const uint32_t m = sv[jj] ? 0u : QuadRows::kOff;
                // with the Delta-scaled input, dx' = sum_n mubar B gives dx = dx' Delta and
                // adds dx' x to dDelta
                const float dd0 = p.bdelta ? fmaf(dxk[jj], xr[jj], ddk[jj]) : ddk[jj];
                const float ddv = SP ? dd0 * (1.f - fexp(-dls[jj])) : dd0;  // d softplus / d Delta_pre
                const float dxv = p.bdelta ? dxk[jj] * dls[jj] : dxk[jj];
                if constexpr (OUT != 2) odx.st(vbo | m, row, dxv, std::false_type{});
                // the bf16 copy of dx (OUT 1: when given; without it the resource is empty)
                if constexpr (OUT16) o16x.st(vbx16 | m, row, dxv, std::true_type{});
                if constexpr (OUT != 2) odd.st(vbo | m, row, ddv, std::false_type{});
                if constexpr (OUT16) o16d.st(vbd16 | m, row, ddv, std::true_type{});
            }
#pragma unroll
            for (int k = 0; k < 4; ++k) dA[k] += dAs[k];
            wave_sums(2 * pair + 1);  // dB
            if constexpr (RING) bc_put(q > 0 ? q - 1 : NCK - 1);
            flush(q);
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) *(nv[k] ? p.hbuf + (cb + k * p.D) : sinkf) = dA[k] * wn[k];
    }

    lds_barrier();
    const int64_t btn = p.nb * p.T * p.N;
    float* dBo = p.nsplit == 1 ? p.dB : p.pB + static_cast<int64_t>(split) * btn;
    float* dCo = p.nsplit == 1 ? p.dC : p.pC + static_cast<int64_t>(split) * btn;
    for (int i = tid; i < L * 32; i += NTH) {
        const int t = i >> 5, cc = i & 31, n = cc & 15;
        if (t < lim && n < p.N) {
            const int64_t row = bb * p.T + t0 + t;
            float* dst = cc < 16 ? dBo : dCo;
            dst[row * p.N + n] = acc[t][cc];
            if (p.nsplit == 1 && p.bc16) stf(p.bc16, row * p.ld_bc16 + (cc < 16 ? 0 : p.N) + n, acc[t][cc]);
        }
    }
}

// dB, dC = sum over splits of the partials (fixed order).
[[maybe_unused]] __global__ __launch_bounds__(256) void k_reduce_bc(const ScanProblem p) {
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
    if (p.bc16) {
        const int64_t row = i / p.N, n = i % p.N;
        stf(p.bc16, row * p.ld_bc16 + n, sb);
        stf(p.bc16, row * p.ld_bc16 + p.N + n, sc);
    }
}

// dA_log, stage 1: grid (ceil(D/256), N, nslice); slice s sums the (b, chunk)
// partials q in its contiguous range, in order.
[[maybe_unused]] __global__ __launch_bounds__(256) void k_reduce_da1(const ScanProblem p) {
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

// dA_log, stage 2: sum of the slices, transposed to [D][N]; with one rate per
// channel also summed over the states (in slice, then state order) into [D].
[[maybe_unused]] __global__ __launch_bounds__(256) void k_reduce_da2(const ScanProblem p) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (p.ascalar) {
        if (i >= p.D) return;
        float acc = 0.f;
        for (int s = 0; s < p.nslice; ++s)
            for (int64_t n = 0; n < p.N; ++n) acc += p.dAtmp[(s * p.N + n) * p.D + i];
        p.dA_log[i] = acc;
        return;
    }
    if (i >= p.D * p.N) return;
    const int64_t d = i / p.N, n = i % p.N;
    float acc = 0.f;
    for (int s = 0; s < p.nslice; ++s) acc += p.dAtmp[(s * p.N + n) * p.D + d];
    p.dA_log[i] = acc;
}

// The tail reductions of the gradient in one launch: blocks [0, nbc) sum the
// dB/dC split partials (as k_reduce_bc); the rest reduce the dA_log partials --
// with one slice straight to the final [D][N] (or [D]) values, each thread
// summing the (b, chunk) partials of one output in order (and, with one rate per
// channel, over the states in order), else stage 1 of the sliced sum
// (k_reduce_da1, with k_reduce_da2 launched after).
[[maybe_unused]] __global__ __launch_bounds__(256) void k_reduce_tail(const ScanProblem p, int nbc) {
    const int tid = threadIdx.x;
    if (static_cast<int>(blockIdx.x) < nbc) {
        const int64_t total = p.nb * p.T * p.N;
        const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + tid;
        if (i >= total) return;
        float sb = 0.f, sc = 0.f;
        for (int s0 = 0; s0 < p.nsplit; s0 += 8) {  // loads of a batch issued before the adds
            float vb[8], vc[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const bool in = s0 + j < p.nsplit;
                vb[j] = in ? p.pB[(s0 + j) * total + i] : 0.f;
                vc[j] = in ? p.pC[(s0 + j) * total + i] : 0.f;
            }
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                sb += vb[j];
                sc += vc[j];
            }
        }
        p.dB[i] = sb;
        p.dC[i] = sc;
        if (p.bc16) {
            const int64_t row = i / p.N, n = i % p.N;
            stf(p.bc16, row * p.ld_bc16 + n, sb);
            stf(p.bc16, row * p.ld_bc16 + p.N + n, sc);
        }
        return;
    }
    const int64_t i = static_cast<int64_t>(static_cast<int>(blockIdx.x) - nbc) * 256 + tid;
    const int64_t nq = p.nb * p.nc;
    // acc += hbuf[(q N + n) D + d] for q = 0..nq-1 in order; the loads of a batch
    // of 8 are issued before any of them is added
    auto sum_q = [&](int64_t n, int64_t d, float acc) {
        const int64_t stride = p.N * p.D;
        const float* src = p.hbuf + n * p.D + d;
        for (int64_t q0 = 0; q0 < nq; q0 += 8) {
            float v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) v[j] = q0 + j < nq ? src[(q0 + j) * stride] : 0.f;
#pragma unroll
            for (int j = 0; j < 8; ++j) acc += v[j];
        }
        return acc;
    };
    if (p.nslice == 1) {
        if (p.ascalar) {
            if (i >= p.D) return;
            float acc = 0.f;
            for (int64_t n = 0; n < p.N; ++n) acc = sum_q(n, i, acc);
            p.dA_log[i] = acc;
            return;
        }
        if (i >= p.D * p.N) return;
        const int64_t n = i / p.D, d = i % p.D;  // consecutive threads read consecutive channels
        p.dA_log[d * p.N + n] = sum_q(n, d, 0.f);
        return;
    }
    if (i >= static_cast<int64_t>(p.nslice) * p.N * p.D) return;
    const int64_t d = i % p.D, n = (i / p.D) % p.N, sl = i / (p.D * p.N);
    const int64_t per = (nq + p.nslice - 1) / p.nslice;
    const int64_t q0 = sl * per, q1 = min(nq, q0 + per);
    float acc = 0.f;
    for (int64_t q = q0; q < q1; ++q) acc += p.hbuf[(q * p.N + n) * p.D + d];
    p.dAtmp[(sl * p.N + n) * p.D + d] = acc;
}

inline unsigned cdiv(int64_t a, int64_t b) { return static_cast<unsigned>((a + b - 1) / b); }

template <typename TI, bool SP, bool GATE, bool N16>
hipError_t forward_impl(const ScanProblem& p, hipStream_t s) {
    {
        SSMK_TIMED("chunk_aggr", s);
        if (aggr_quad(p))
            hipLaunchKernelGGL((k_chunk_aggr_quad<TI, SP, GATE, false, 8>), aggr_grid(p), dim3(256), 0, s, p);
        else
            hipLaunchKernelGGL((k_chunk_aggr<TI, SP, GATE, false, N16, 8>), aggr_grid(p), dim3(64), 0, s, p);
    }
    {
        SSMK_TIMED("carry", s);
        hipLaunchKernelGGL(k_carry, carry_grid(p), dim3(256), 0, s, p);
    }
    SSMK_TIMED("forward", s);
    if (aggr_quad(p))
        hipLaunchKernelGGL((k_forward_quad<TI, SP, GATE>), aggr_grid(p), dim3(256), 0, s, p);
    else
        hipLaunchKernelGGL((k_forward<TI, SP, GATE, N16>), aggr_grid(p), dim3(64), 0, s, p);
    return hipGetLastError();
}

template <typename TI, bool SP, bool GATE, bool TRUNC, bool N16, int S, int NCK>
void grad_main(const ScanProblem& p, hipStream_t s) {
    dim3 g(static_cast<unsigned>(p.nsplit), static_cast<unsigned>(p.nc),
           static_cast<unsigned>(p.nb));
    SSMK_TIMED(TRUNC ? "grad_fused_trunc" : "grad_fused", s);
    // the bf16 copies exist for the whole-layer path (bf16 inputs, softplus, gate)
    if constexpr (sizeof(TI) == 2 && SP && GATE) {
        if (p.dd16 && p.only16) {
            hipLaunchKernelGGL((k_grad<TI, SP, GATE, TRUNC, N16, S, NCK, 2>), g, dim3(64 * kGradWaves), 0, s, p);
            return;
        }
        if (p.dd16) {
            hipLaunchKernelGGL((k_grad<TI, SP, GATE, TRUNC, N16, S, NCK, 1>), g, dim3(64 * kGradWaves), 0, s, p);
            return;
        }
    }
    hipLaunchKernelGGL((k_grad<TI, SP, GATE, TRUNC, N16, S, NCK, 0>), g, dim3(64 * kGradWaves), 0, s, p);
}

template <typename TI, bool SP, bool GATE, bool TRUNC, bool N16>
hipError_t grad_impl(const ScanProblem& p, hipStream_t s) {
    if ((p.dd16 || p.dz16 || p.bc16 || p.dx16) && !(sizeof(TI) == 2 && SP && GATE)) return hipErrorInvalidValue;
    if (p.dd16 && !(p.dz16 && p.bc16)) return hipErrorInvalidValue;
    if ((p.dx16 || p.only16) && !p.dd16) return hipErrorInvalidValue;
    if (p.only16 && !p.dx16) return hipErrorInvalidValue;
    {
        SSMK_TIMED("chunk_aggr", s);
        const bool quad = aggr_quad(p);
        // records every 8 steps at every chunk length
        if (p.seg != 8) return hipErrorInvalidValue;
        if (quad) hipLaunchKernelGGL((k_chunk_aggr_quad<TI, SP, GATE, true, 8>), aggr_grid(p), dim3(256), 0, s, p);
        else hipLaunchKernelGGL((k_chunk_aggr<TI, SP, GATE, true, N16, 8>), aggr_grid(p), dim3(64), 0, s, p);
    }
    {
        SSMK_TIMED("carry", s);
        hipLaunchKernelGGL(k_carry, carry_grid(p), dim3(256), 0, s, p);
    }
    switch (p.L) {
        case 16: grad_main<TI, SP, GATE, TRUNC, N16, 8, 2>(p, s); break;
        case 32: grad_main<TI, SP, GATE, TRUNC, N16, 8, 4>(p, s); break;
        case 64: grad_main<TI, SP, GATE, TRUNC, N16, 8, 8>(p, s); break;
        case 128: grad_main<TI, SP, GATE, TRUNC, N16, 8, 16>(p, s); break;
        default: grad_main<TI, SP, GATE, TRUNC, N16, 8, 32>(p, s); break;  // 256
    }
    SSMK_TIMED("reduce", s);
    const int nbc = p.nsplit > 1 ? static_cast<int>(cdiv(p.nb * p.T * p.N, 256)) : 0;
    const int64_t nda = p.nslice == 1 ? (p.ascalar ? p.D : p.D * p.N) : static_cast<int64_t>(p.nslice) * p.N * p.D;
    hipLaunchKernelGGL(k_reduce_tail, dim3(static_cast<unsigned>(nbc) + cdiv(nda, 256)), dim3(256), 0, s, p, nbc);
    if (p.nslice > 1) hipLaunchKernelGGL(k_reduce_da2, dim3(cdiv(p.D * p.N, 256)), dim3(256), 0, s, p);
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
