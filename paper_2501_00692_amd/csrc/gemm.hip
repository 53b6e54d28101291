// gemm.hip -- bf16 MFMA GEMMs for the projection gradients (gfx950,
// v_mfma_f32_32x32x16_bf16, fp32 accumulation), one templated kernel:
//   dW[K][N] = X^T dZ  (X [M][K], dZ [M][N]): the reduction runs over the row
//       index of both operands, so 8x8 blocks are transposed in registers on
//       their way into LDS; split over M when the output has few tiles, with a
//       fixed-order second-stage reduction;
//   dX[M][K] = dZ W^T  (dZ [M][N], W [K][N]): both operands are contiguous along
//       the reduction and are staged as they are; the epilogue adds an optional
//       fp32 addend, accumulates, and can write a bf16 copy into a strided buffer.
// Workgroup: 512 threads = 4x2 waves, two per SIMD (one wave's MFMAs run while
// the other waits for its loads or the barrier); a wave owns a 64 x (BN/2) block
// of 32x32 MFMA tiles.  Tile BM x BN with BM = 256 and BN in {128, 192, 256};
// interior tiles with whole reduction steps run a loop without bounds checks,
// other loads read a clamped in-range address and select zero (no branches).
// LDS is double-buffered over 64-deep reduction steps (one barrier per step);
// the next step's global loads are in flight while the MFMAs run, and below
// 256 columns the next 16-deep sub-step's fragments are read from LDS while the
// current sub-step's MFMAs run.
// Output tiles and reduction splits are assigned so that each XCD runs one
// contiguous run of (split, row block, column block) (consecutive workgroups go
// to different XCDs), which keeps a row block of the first operand and its
// reduction range in one L2.
#include "internal.h"

namespace ssmk {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int BK = 64;   // reduction depth per step
constexpr int LDK = BK;  // LDS row length (bf16): 8 blocks of 16 bytes, XOR-swizzled

// Physical 16-byte block of logical block `blk` in LDS row `row`: the XOR keeps
// fragment reads (8 consecutive rows), row-wise staging writes (8 blocks of one
// row) and transposed staging writes (rows 8 apart) free of bank conflicts.
__device__ __forceinline__ int swz(int row, int blk) { return (blk ^ (row ^ (row >> 3))) & 7; }

__device__ __forceinline__ uint16_t f2bf(float v) {
    uint32_t u = __float_as_uint(v);
    if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;
    u += 0x7fffu + ((u >> 16) & 1u);
    return static_cast<uint16_t>(u >> 16);
}

__device__ __forceinline__ bf16x8 lds_frag(const uint16_t* p) {
    const uint4 v = *reinterpret_cast<const uint4*>(p);
    return __builtin_bit_cast(bf16x8, v);
}

// Transpose an 8x8 block of bf16: in[r] holds row r (8 values, 4 words); out[c]
// receives column c as 8 values (4 words).
__device__ __forceinline__ void transpose8x8(const uint4 (&in)[8], uint4 (&out)[8]) {
    uint32_t w[8][4];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
        w[r][0] = in[r].x; w[r][1] = in[r].y; w[r][2] = in[r].z; w[r][3] = in[r].w;
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        uint32_t lo[4], hi[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint32_t a = w[2 * j][c], b = w[2 * j + 1][c];
            lo[j] = (a & 0xffffu) | (b << 16);          // column 2c, rows 2j, 2j+1
            hi[j] = (a >> 16) | (b & 0xffff0000u);      // column 2c+1
        }
        out[2 * c] = make_uint4(lo[0], lo[1], lo[2], lo[3]);
        out[2 * c + 1] = make_uint4(hi[0], hi[1], hi[2], hi[3]);
    }
}

struct GemmArgs {
    int64_t R, Cc, Kr;    // output rows, output cols, reduction length
    const uint16_t* A;    // TR: [Kr][R] (reduction-major); else [R][Kr]
    int64_t lda;
    const uint16_t* B;    // TR: [Kr][Cc];                  else [Cc][Kr]
    int64_t ldb;
    float* C;             // output [R][Cc] (ldc = Cc), or split partials
    int64_t kper;         // reduction range per split (multiple of BK)
    int direct;           // write C (else the partial of the workgroup's split)
    int accum;            // C += result
    const float* add;     // optional fp32 addend [R][Cc]
    uint16_t* out16;      // optional bf16 copy of the result
    int64_t ld16;
};

constexpr int kXcds = 8;

// Staging of both operand tiles (BM and BN rows x BK reduction) into LDS rows of
// LDK bf16.  TR (reduction-major sources): 8x8 blocks, numbered A blocks first
// (BM of them) then B blocks (BN); thread tid takes blocks tid and tid + NT,
// transposed in registers.  Otherwise: 16-byte pieces spread over all threads.
// FULL: the tile's rows and columns are in bounds; KF: so is the whole
// reduction step (no checks at all when both hold).  Reduction ranges end on a multiple of 8 except in the row-wise (TR)
// case, where each of the 8 rows of a block is checked.
template <bool TR, int BM, int BN, int NT>
struct Stager {
    static constexpr int PA = TR ? BM : BM * 8;
    static constexpr int PB = TR ? BN : BN * 8;
    static constexpr int PER = TR ? (PA + PB + NT - 1) / NT : (PA + PB) / NT;
    static constexpr int REGS = TR ? 8 : 1;
    static_assert(TR || (PA % NT == 0 && PB % NT == 0), "pieces divide evenly");
    uint4 v[PER][REGS];

    template <bool FULL, bool KF>
    __device__ __forceinline__ void load(const GemmArgs& g, int64_t r0, int64_t c0, int64_t k,
                                         int64_t k_hi, int tid) {
        if constexpr (TR) {
#pragma unroll
            for (int e = 0; e < PER; ++e) {
                const int q = tid + NT * e;
                if (q >= PA + PB) break;  // uniform per wave (PA + PB is a multiple of 64)
                const bool isA = q < PA;
                const int pc = isA ? q : q - PA;
                const int rows8 = (isA ? BM : BN) / 8;
                const int rb = pc / rows8, cb = pc % rows8;  // reduction block, row block
                const uint16_t* src = isA ? g.A : g.B;
                const int64_t ld = isA ? g.lda : g.ldb;
                const int64_t col = (isA ? r0 : c0) + cb * 8;
                const int64_t ncol = isA ? g.R : g.Cc;
                // out-of-range pieces load an in-range one (clamped row and column)
                // and select zero, so that every load is issued without a branch
                const bool cok = FULL || col < ncol;
                const int64_t cs = cok ? col : ncol - 8;
#pragma unroll
                for (int r = 0; r < 8; ++r) {
                    const int64_t kr = k + rb * 8 + r;
                    const bool ok = cok && (KF || kr < k_hi);
                    const uint4 t = *reinterpret_cast<const uint4*>(src + (ok ? kr : k_hi - 1) * ld + cs);
                    v[e][r] = ok ? t : make_uint4(0u, 0u, 0u, 0u);
                }
            }
        } else {
#pragma unroll
            for (int e = 0; e < PER; ++e) {
                constexpr int EA = PA / NT;  // pieces of A per thread; the rest are B
                const bool isA = e < EA;
                const int q = tid + NT * (isA ? e : e - EA);
                const int row = q >> 3, seg = q & 7;
                const int64_t gr = (isA ? r0 : c0) + row, kk = k + seg * 8;
                const uint16_t* src = isA ? g.A : g.B;
                const int64_t ld = isA ? g.lda : g.ldb;
                const int64_t nrow = isA ? g.R : g.Cc;
                const bool ok = (FULL || gr < nrow) && (KF || kk < k_hi);
                const uint4 t = *reinterpret_cast<const uint4*>(src + (FULL || gr < nrow ? gr : nrow - 1) * ld +
                                                                (KF || kk < k_hi ? kk : k_hi - 8));
                v[e][0] = ok ? t : make_uint4(0u, 0u, 0u, 0u);
            }
        }
    }
    __device__ __forceinline__ void store(uint16_t (*As)[LDK], uint16_t (*Bs)[LDK], int tid) const {
        if constexpr (TR) {
#pragma unroll
            for (int e = 0; e < PER; ++e) {
                const int q = tid + NT * e;
                if (q >= PA + PB) break;
                const bool isA = q < PA;
                const int pc = isA ? q : q - PA;
                const int rows8 = (isA ? BM : BN) / 8;
                const int rb = pc / rows8, cb = pc % rows8;
                uint16_t(*dst)[LDK] = isA ? As : Bs;
                uint4 tr[8];
                transpose8x8(v[e], tr);
#pragma unroll
                for (int c = 0; c < 8; ++c) {
                    const int row = cb * 8 + c;
                    *reinterpret_cast<uint4*>(&dst[row][swz(row, rb) * 8]) = tr[c];
                }
            }
        } else {
#pragma unroll
            for (int e = 0; e < PER; ++e) {
                constexpr int EA = PA / NT;
                const bool isA = e < EA;
                const int q = tid + NT * (isA ? e : e - EA);
                const int row = q >> 3, seg = q & 7;
                uint16_t(*dst)[LDK] = isA ? As : Bs;
                *reinterpret_cast<uint4*>(&dst[row][swz(row, seg) * 8]) = v[e][0];
            }
        }
    }
};

// Main loop over the workgroup's reduction range; FULL drops the row and column
// bounds checks.
template <bool TR, int BM, int BN, int NT, bool FULL, bool KF, int MI, int NJ, bool PF2>
__device__ __forceinline__ void gemm_mainloop(const GemmArgs& g, uint16_t (*As)[BM][LDK],
                                              uint16_t (*Bs)[BN][LDK], int64_t r0, int64_t c0,
                                              int64_t k_lo, int64_t k_hi, int tid, int wr, int wc,
                                              f32x16 (&acc)[MI][NJ]) {
    const int lane = tid & 63;
    const int li = lane & 31;
    const int lk = (lane >> 5) * 8;
    Stager<TR, BM, BN, NT> st;
    if (k_lo < k_hi) {
        st.template load<FULL, KF>(g, r0, c0, k_lo, k_hi, tid);
        st.store(As[0], Bs[0], tid);
    }
    // fragments of one 16-deep sub-step, double-buffered in registers: the next
    // sub-step's LDS reads are issued before the current sub-step's MFMAs, and the
    // scheduling barriers keep them there, so that one wave per SIMD does not wait
    // for LDS between MFMAs
    auto frags = [&](int buf, int ks, bf16x8 (&a)[MI], bf16x8 (&b)[NJ]) {
#pragma unroll
        for (int i = 0; i < MI; ++i) {
            const int row = wr + i * 32 + li;
            a[i] = lds_frag(&As[buf][row][swz(row, (ks + lk) >> 3) * 8]);
        }
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int row = wc + j * 32 + li;
            b[j] = lds_frag(&Bs[buf][row][swz(row, (ks + lk) >> 3) * 8]);
        }
    };
    auto mfmas = [&](const bf16x8 (&a)[MI], const bf16x8 (&b)[NJ]) {
#pragma unroll
        for (int i = 0; i < MI; ++i)
#pragma unroll
            for (int j = 0; j < NJ; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    };
    // 256-wide tiles have no registers to spare for a second fragment set: they
    // read each sub-step's fragments right before its MFMAs
    constexpr bool DB = BN < 256 && !(TR && PF2);
    bf16x8 a0[MI], b0[NJ], a1[MI], b1[NJ];
    // the MFMAs of one 64-deep step on LDS buffer `cur`, with `between` (the
    // staging store for the next step) issued before the last sub-step
    auto step = [&](int cur, auto&& between) {
        static_assert(BK == 64, "four sub-steps per step");
        if constexpr (DB) {
            frags(cur, 16, a1, b1);
            __builtin_amdgcn_sched_barrier(0);
            mfmas(a0, b0);
            __builtin_amdgcn_sched_barrier(0);
            frags(cur, 32, a0, b0);
            __builtin_amdgcn_sched_barrier(0);
            mfmas(a1, b1);
            __builtin_amdgcn_sched_barrier(0);
            frags(cur, 48, a1, b1);
            __builtin_amdgcn_sched_barrier(0);
            mfmas(a0, b0);
            __builtin_amdgcn_sched_barrier(0);
            between();
            mfmas(a1, b1);
        } else {
#pragma unroll
            for (int ks = 0; ks < BK; ks += 16) {
                frags(cur, ks, a0, b0);
                mfmas(a0, b0);
            }
            between();
        }
    };
    const int64_t nsteps = (k_hi - k_lo + BK - 1) / BK;
    if constexpr (PF2) {
        // global loads two steps ahead in two staging sets used alternately: at
        // the top of step j the set of step j+1 is in flight and the other one,
        // stored to LDS at the end of step j-1, takes the loads of step j+2
        Stager<TR, BM, BN, NT> st1;
        if (nsteps > 1) st1.template load<FULL, KF>(g, r0, c0, k_lo + BK, k_hi, tid);
        __syncthreads();
        if (DB) frags(0, 0, a0, b0);
        auto pair_step = [&](int64_t j, Stager<TR, BM, BN, NT>& mine, Stager<TR, BM, BN, NT>& other) {
            const int cur = static_cast<int>(j & 1);
            if (j + 2 < nsteps) mine.template load<FULL, KF>(g, r0, c0, k_lo + (j + 2) * BK, k_hi, tid);
            step(cur, [&]() {
                if (j + 1 < nsteps) other.store(As[cur ^ 1], Bs[cur ^ 1], tid);
            });
            __syncthreads();
            if (DB && j + 1 < nsteps) frags(cur ^ 1, 0, a0, b0);
        };
        for (int64_t j = 0; j < nsteps; j += 2) {
            pair_step(j, st, st1);
            if (j + 1 < nsteps) pair_step(j + 1, st1, st);
        }
        return;
    }
    __syncthreads();
    int cur = 0;
    if (DB) frags(0, 0, a0, b0);
    for (int64_t j = 0; j < nsteps; ++j) {
        const bool more = j + 1 < nsteps;
        if (more) st.template load<FULL, KF>(g, r0, c0, k_lo + (j + 1) * BK, k_hi, tid);
        step(cur, [&]() {
            if (more) st.store(As[cur ^ 1], Bs[cur ^ 1], tid);
        });
        __syncthreads();
        cur ^= 1;
        if (DB && more) frags(cur, 0, a0, b0);
    }
}

template <bool TR, int BM, int BN, int WM>
__global__ __launch_bounds__(128 * WM) void k_gemm(const GemmArgs g) {
    constexpr int NT = 128 * WM;  // WM x 2 waves
    constexpr int MI = BM / (32 * WM), NJ = BN / 64;  // 32x32 MFMA tiles per wave
#ifndef SSMK_GEMM_PF2
#define SSMK_GEMM_PF2 1
#endif
    constexpr bool PF2 = SSMK_GEMM_PF2 && BN == 128;  // registers for a second staging set
    __shared__ __attribute__((aligned(16))) uint16_t As[2][BM][LDK];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BN][LDK];
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    // output tile and reduction split: workgroups are dispatched to the XCDs in
    // turn (workgroup i to XCD i % 8), so the linear id is mapped to a logical
    // index that gives every XCD one contiguous run of (split, row block, column
    // block) -- the workgroups of one XCD share the first operand's row block and
    // reduction range in its L2.  The map is a bijection for any count.
    const int ncb = static_cast<int>(gridDim.x);
    const int ntl = ncb * static_cast<int>(gridDim.y);
    const int nwg = ntl * static_cast<int>(gridDim.z);
    const int lin = static_cast<int>(blockIdx.x) + ncb * (static_cast<int>(blockIdx.y) +
                                                          static_cast<int>(gridDim.y) * static_cast<int>(blockIdx.z));
    const int xq = nwg / kXcds, xr = nwg % kXcds, xcd = lin % kXcds;
    const int logical = (xcd < xr ? xcd * (xq + 1) : xr * (xq + 1) + (xcd - xr) * xq) + lin / kXcds;
    const int tile = logical % ntl, split = logical / ntl;
    const int64_t c0 = static_cast<int64_t>(tile % ncb) * BN;
    const int64_t r0 = static_cast<int64_t>(tile / ncb) * BM;
    const int64_t k_lo = static_cast<int64_t>(split) * g.kper;
    const int64_t k_hi = min(g.Kr, k_lo + g.kper);
    const int wr = (wave >> 1) * (BM / WM);
    const int wc = (wave & 1) * (BN / 2);

    f32x16 acc[MI][NJ];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    const bool full = r0 + BM <= g.R && c0 + BN <= g.Cc;
    const bool kfull = (k_hi - k_lo) % BK == 0;
    if (full && kfull)
        gemm_mainloop<TR, BM, BN, NT, true, true, MI, NJ, PF2>(g, As, Bs, r0, c0, k_lo, k_hi, tid, wr, wc, acc);
    else if (full)
        gemm_mainloop<TR, BM, BN, NT, true, false, MI, NJ, PF2>(g, As, Bs, r0, c0, k_lo, k_hi, tid, wr, wc, acc);
    else
        gemm_mainloop<TR, BM, BN, NT, false, false, MI, NJ, PF2>(g, As, Bs, r0, c0, k_lo, k_hi, tid, wr, wc, acc);

    // acc element v of lane l is row 8*(v/4) + 4*(l/32) + v%4, col l%32 of its tile
    float* __restrict__ dst = g.C ? g.C + (g.direct ? 0 : static_cast<int64_t>(split) * g.R * g.Cc) : nullptr;
    const float* __restrict__ addp = g.direct ? g.add : nullptr;
    const bool accum = g.direct && g.accum;
    uint16_t* __restrict__ o16 = g.direct ? g.out16 : nullptr;
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int64_t col = c0 + wc + j * 32 + (lane & 31);
            const int64_t rb = r0 + wr + i * 32 + 4 * (lane >> 5);
            // the tile's addends first, so that their loads overlap
            float extra[16];
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t row = rb + 8 * (v >> 2) + (v & 3);
                const bool in = row < g.R && col < g.Cc;
                const int64_t o = row * g.Cc + col;
                float e = 0.f;
                if (addp && in) e = addp[o];
                if (accum && dst && in) e += dst[o];
                extra[v] = e;
            }
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t row = rb + 8 * (v >> 2) + (v & 3);
                if (row < g.R && col < g.Cc) {
                    const float val = acc[i][j][v] + extra[v];
                    if (dst) dst[row * g.Cc + col] = val;
                    if (o16) o16[row * g.ld16 + col] = f2bf(val);
                }
            }
        }
}

// dW = (dW +) sum over splits, in split order.
__global__ __launch_bounds__(256) void k_splitk_reduce(int64_t KN, int splits, const float* part,
                                                       float* dW, int accum) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i >= KN) return;
    float s = 0.f;
    for (int q = 0; q < splits; ++q) s += part[q * KN + i];
    dW[i] = accum ? dW[i] + s : s;
}

inline unsigned cdiv(int64_t a, int64_t b) { return static_cast<unsigned>((a + b - 1) / b); }

constexpr int kCUs = 256;

// Output-tile width and reduction splits for an R x Cc output with reduction Kr,
// from a simple time model: rounds of 256 workgroups x the MFMA time of one
// workgroup's share (about 1.2 us per 256x256x64 step), plus the HBM time of
// writing and re-reading the split partials (4 TB/s).
struct Plan {
    int bn;
    int splits;
};

Plan plan_gemm(int64_t R, int64_t Cc, int64_t Kr, bool allow_split) {
    Plan best{192, 1};
    double best_us = 1e300;
    const int bns[3] = {256, 192, 128};
    for (int bn : bns) {
        const int64_t tiles = ((R + 255) / 256) * ((Cc + bn - 1) / bn);
        const int64_t iters = (Kr + BK - 1) / BK;
        for (int s = 1; s <= (allow_split ? 32 : 1); ++s) {
            if (s > 1 && iters / s < 8) break;
            const int64_t wgs = tiles * s;
            const double rounds = static_cast<double>((wgs + kCUs - 1) / kCUs);
            double us = rounds * 1.2 * (bn / 256.0) * (static_cast<double>(Kr) / s / BK);
            if (s > 1) us += static_cast<double>(s) * R * Cc * 8.0 / 4e12 * 1e6;
            if (us < best_us * 0.999) {
                best_us = us;
                best = Plan{bn, s};
            }
        }
    }
    return best;
}

template <bool TR, int BN>
void launch_tile(const GemmArgs& g, int splits, hipStream_t s) {
    constexpr int WM = 4;  // 4 x 2 waves, two per SIMD
    dim3 grid(cdiv(g.Cc, BN), cdiv(g.R, 256), static_cast<unsigned>(splits));
    hipLaunchKernelGGL((k_gemm<TR, 256, BN, WM>), grid, dim3(128 * WM), 0, s, g);
}

template <bool TR>
void launch_plan(const GemmArgs& g, const Plan& pl, hipStream_t s) {
    switch (pl.bn) {
        case 128: launch_tile<TR, 128>(g, pl.splits, s); break;
        case 192: launch_tile<TR, 192>(g, pl.splits, s); break;
        default: launch_tile<TR, 256>(g, pl.splits, s); break;
    }
}

}  // namespace

size_t gemm_dw_workspace(int64_t M, int64_t K, int64_t N) {
    const Plan pl = plan_gemm(K, N, M, true);
    return pl.splits > 1 ? static_cast<size_t>(pl.splits) * K * N * sizeof(float) : 0;
}

hipError_t launch_gemm_dw(int64_t M, int64_t K, int64_t N, const uint16_t* X, int64_t ldx,
                          const uint16_t* dZ, int64_t lddz, float* dW, bool accum, void* ws,
                          hipStream_t s) {
    const Plan pl = plan_gemm(K, N, M, true);
    int64_t per = (M + pl.splits - 1) / pl.splits;
    per = (per + BK - 1) / BK * BK;
    const bool direct = pl.splits == 1;
    GemmArgs g{K, N, M, X, ldx, dZ, lddz, direct ? dW : static_cast<float*>(ws), per,
               direct ? 1 : 0, accum ? 1 : 0, nullptr, nullptr, 0};
    {
        SSMK_TIMED("gemm_dw", s);
        launch_plan<true>(g, pl, s);
    }
    if (!direct) {
        SSMK_TIMED("splitk_reduce", s);
        hipLaunchKernelGGL(k_splitk_reduce, dim3(cdiv(K * N, 256)), dim3(256), 0, s, K * N, pl.splits,
                           static_cast<const float*>(ws), dW, accum ? 1 : 0);
    }
    return hipGetLastError();
}

hipError_t launch_gemm_dx(int64_t M, int64_t K, int64_t N, const uint16_t* dZ, int64_t lddz,
                          const uint16_t* W, int64_t ldw, float* dX, bool accum, const float* add,
                          uint16_t* out16, int64_t ld16, hipStream_t s) {
    const Plan pl = plan_gemm(M, K, N, false);
    GemmArgs g{M, K, N, dZ, lddz, W, ldw, dX, (N + BK - 1) / BK * BK, 1, accum ? 1 : 0, add, out16, ld16};
    SSMK_TIMED("gemm_dx", s);
    launch_plan<false>(g, pl, s);
    return hipGetLastError();
}

}  // namespace ssmk
