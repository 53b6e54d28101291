// gemm.hip -- bf16 MFMA GEMMs for the projection gradients (gfx950,
// v_mfma_f32_32x32x16_bf16, fp32 accumulation):
//   k_gemm_dw : dW[K][N] = X^T dZ,  X [M][K], dZ [M][N]; the reduction runs over
//               the row index M of both operands, so 8x8 blocks are transposed
//               in registers on their way into LDS (LDS holds [k][m] and [n][m]);
//               split over M with a deterministic second-stage reduction.
//   k_gemm_dx : dX[M][K] = dZ W^T,  dZ [M][N], W [K][N]; both operands are
//               contiguous along the reduction, staged through LDS as is;
//               epilogue adds an optional fp32 addend, accumulates, and can
//               write a bf16 copy into a strided buffer.
//   k_pack    : fp32 -> bf16 (round to nearest even) strided copy.
#include "internal.h"

namespace ssmk {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int BM = 128;   // output rows per workgroup
constexpr int BN = 128;   // output cols per workgroup
constexpr int BK = 64;    // reduction depth per iteration
constexpr int LDK = BK + 8;  // LDS row length (bf16), padded

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

// ---------------------------------------------------------------------------
// dW partial: grid (ceil(N/BN), ceil(K/BM), splits), 256 threads.
// Workgroup tile: rows k0..k0+127 of dW, cols n0..n0+127, reduction rows
// m in [m_lo, m_hi).  Threads 0..127 stage the X block, 128..255 the dZ block:
// each thread loads an 8(m) x 8 block and writes it transposed.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_gemm_dw(int64_t M, int64_t K, int64_t N,
                                                 const uint16_t* __restrict__ X, int64_t ldx,
                                                 const uint16_t* __restrict__ dZ, int64_t lddz,
                                                 float* __restrict__ out, int64_t m_per_split,
                                                 int direct, int accum) {
    __shared__ __attribute__((aligned(16))) uint16_t At[BM][LDK];  // [k][m]
    __shared__ __attribute__((aligned(16))) uint16_t Bt[BN][LDK];  // [n][m]
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int64_t n0 = static_cast<int64_t>(blockIdx.x) * BN;
    const int64_t k0 = static_cast<int64_t>(blockIdx.y) * BM;
    const int64_t m_lo = static_cast<int64_t>(blockIdx.z) * m_per_split;
    const int64_t m_hi = min(M, m_lo + m_per_split);

    // staging role
    const bool isA = tid < 128;
    const int st = tid & 127;
    const int bcol = st & 15;   // 8-wide column block within the 128 columns
    const int brow = st >> 4;   // 8-row block within BK = 64
    const uint16_t* src = isA ? X : dZ;
    const int64_t ld = isA ? ldx : lddz;
    const int64_t colg = (isA ? k0 : n0) + bcol * 8;
    const int64_t ncol = isA ? K : N;
    const bool colv = colg < ncol;  // K, N are multiples of 8

    uint4 regs[8];
    auto load_tile = [&](int64_t m0) {
#pragma unroll
        for (int r = 0; r < 8; ++r) {
            const int64_t m = m0 + brow * 8 + r;
            if (colv && m < m_hi)
                regs[r] = *reinterpret_cast<const uint4*>(src + m * ld + colg);
            else
                regs[r] = make_uint4(0u, 0u, 0u, 0u);
        }
    };

    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    const int wr = (wave >> 1) * 64;  // wave's row offset within the tile
    const int wc = (wave & 1) * 64;   // wave's col offset
    const int li = lane & 31;
    const int lk = (lane >> 5) * 8;

    load_tile(m_lo);
    for (int64_t m0 = m_lo; m0 < m_hi; m0 += BK) {
        uint4 tr[8];
        transpose8x8(regs, tr);
        __syncthreads();  // previous iteration's fragment reads are done
        uint16_t(*dst)[LDK] = isA ? At : Bt;
#pragma unroll
        for (int c = 0; c < 8; ++c)
            *reinterpret_cast<uint4*>(&dst[bcol * 8 + c][brow * 8]) = tr[c];
        __syncthreads();
        if (m0 + BK < m_hi) load_tile(m0 + BK);
#pragma unroll
        for (int ks = 0; ks < BK; ks += 16) {
            bf16x8 a[2], b[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) a[i] = lds_frag(&At[wr + i * 32 + li][ks + lk]);
#pragma unroll
            for (int j = 0; j < 2; ++j) b[j] = lds_frag(&Bt[wc + j * 32 + li][ks + lk]);
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
        }
    }

    // write: acc element v of lane l is row 8*(v/4) + 4*(l/32) + v%4, col l%32
    float* dst = out + (direct ? 0 : static_cast<int64_t>(blockIdx.z) * K * N);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t row = k0 + wr + i * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
                const int64_t col = n0 + wc + j * 32 + (lane & 31);
                if (row < K && col < N) {
                    const int64_t o = row * N + col;
                    if (direct && accum)
                        dst[o] += acc[i][j][v];
                    else
                        dst[o] = acc[i][j][v];
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

// ---------------------------------------------------------------------------
// dX: grid (ceil(K/BN), ceil(M/BM)), 256 threads.  Tile rows m0.., cols k0..
// A = dZ rows (m, reduction n contiguous), B = W rows (k, reduction n contiguous).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_gemm_dx(int64_t M, int64_t K, int64_t N,
                                                 const uint16_t* __restrict__ dZ, int64_t lddz,
                                                 const uint16_t* __restrict__ W, int64_t ldw,
                                                 float* __restrict__ dX, int accum,
                                                 const float* __restrict__ add,
                                                 uint16_t* __restrict__ out16, int64_t ld16) {
    __shared__ __attribute__((aligned(16))) uint16_t As[BM][LDK];  // [m][n]
    __shared__ __attribute__((aligned(16))) uint16_t Bs[BN][LDK];  // [k][n]
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int64_t k0 = static_cast<int64_t>(blockIdx.x) * BN;
    const int64_t m0 = static_cast<int64_t>(blockIdx.y) * BM;

    // staging: each operand tile is 128 rows x 64 values = 1024 16-byte pieces;
    // thread tid loads pieces tid + 256*e, e = 0..3, for each operand.
    uint4 ra[4], rb[4];
    auto load_tile = [&](int64_t n0) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int piece = tid + 256 * e;
            const int row = piece >> 3, cb = (piece & 7) * 8;
            const int64_t n = n0 + cb;
            const int64_t m = m0 + row, k = k0 + row;
            ra[e] = (m < M && n < N) ? *reinterpret_cast<const uint4*>(dZ + m * lddz + n)
                                     : make_uint4(0u, 0u, 0u, 0u);
            rb[e] = (k < K && n < N) ? *reinterpret_cast<const uint4*>(W + k * ldw + n)
                                     : make_uint4(0u, 0u, 0u, 0u);
        }
    };

    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
    const int wr = (wave >> 1) * 64;
    const int wc = (wave & 1) * 64;
    const int li = lane & 31;
    const int lk = (lane >> 5) * 8;

    load_tile(0);
    for (int64_t n0 = 0; n0 < N; n0 += BK) {
        __syncthreads();
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int piece = tid + 256 * e;
            const int row = piece >> 3, cb = (piece & 7) * 8;
            *reinterpret_cast<uint4*>(&As[row][cb]) = ra[e];
            *reinterpret_cast<uint4*>(&Bs[row][cb]) = rb[e];
        }
        __syncthreads();
        if (n0 + BK < N) load_tile(n0 + BK);
#pragma unroll
        for (int ks = 0; ks < BK; ks += 16) {
            bf16x8 a[2], b[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) a[i] = lds_frag(&As[wr + i * 32 + li][ks + lk]);
#pragma unroll
            for (int j = 0; j < 2; ++j) b[j] = lds_frag(&Bs[wc + j * 32 + li][ks + lk]);
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
        }
    }

#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t m = m0 + wr + i * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
                const int64_t k = k0 + wc + j * 32 + (lane & 31);
                if (m < M && k < K) {
                    const int64_t o = m * K + k;
                    float val = acc[i][j][v];
                    if (add) val += add[o];
                    if (accum) val += dX[o];
                    dX[o] = val;
                    if (out16) out16[m * ld16 + k] = f2bf(val);
                }
            }
}

__global__ __launch_bounds__(256) void k_pack(int64_t rows, int64_t cols, const float* src,
                                              int64_t lds, uint16_t* dst, int64_t ldd, int64_t col0) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i >= rows * cols) return;
    const int64_t r = i / cols, c = i % cols;
    dst[r * ldd + col0 + c] = f2bf(src[r * lds + c]);
}

int dw_splits(int64_t M, int64_t K, int64_t N) {
    const int64_t tiles = ((K + BM - 1) / BM) * ((N + BN - 1) / BN);
    const int64_t iters = (M + BK - 1) / BK;
    int64_t s = (512 + tiles - 1) / tiles;  // aim for >= 2 workgroups per CU
    if (s > iters / 8) s = iters / 8;        // keep >= 8 iterations per split
    if (s < 1) s = 1;
    if (s > 64) s = 64;
    return static_cast<int>(s);
}

inline unsigned cdiv(int64_t a, int64_t b) { return static_cast<unsigned>((a + b - 1) / b); }

}  // namespace

size_t gemm_dw_workspace(int64_t M, int64_t K, int64_t N) {
    const int s = dw_splits(M, K, N);
    return s > 1 ? static_cast<size_t>(s) * K * N * sizeof(float) : 0;
}

hipError_t launch_gemm_dw(int64_t M, int64_t K, int64_t N, const uint16_t* X, int64_t ldx,
                          const uint16_t* dZ, int64_t lddz, float* dW, bool accum, void* ws,
                          hipStream_t s) {
    const int splits = dw_splits(M, K, N);
    int64_t per = (M + splits - 1) / splits;
    per = (per + BK - 1) / BK * BK;
    dim3 grid(cdiv(N, BN), cdiv(K, BM), static_cast<unsigned>(splits));
    const bool direct = splits == 1;
    float* out = direct ? dW : static_cast<float*>(ws);
    SSMK_TIMED("gemm_dw", s);
    hipLaunchKernelGGL(k_gemm_dw, grid, dim3(256), 0, s, M, K, N, X, ldx, dZ, lddz, out, per,
                       direct ? 1 : 0, accum ? 1 : 0);
    if (!direct)
        hipLaunchKernelGGL(k_splitk_reduce, dim3(cdiv(K * N, 256)), dim3(256), 0, s, K * N, splits,
                           static_cast<const float*>(ws), dW, accum ? 1 : 0);
    return hipGetLastError();
}

hipError_t launch_gemm_dx(int64_t M, int64_t K, int64_t N, const uint16_t* dZ, int64_t lddz,
                          const uint16_t* W, int64_t ldw, float* dX, bool accum, const float* add,
                          uint16_t* out16, int64_t ld16, hipStream_t s) {
    dim3 grid(cdiv(K, BN), cdiv(M, BM));
    SSMK_TIMED("gemm_dx", s);
    hipLaunchKernelGGL(k_gemm_dx, grid, dim3(256), 0, s, M, K, N, dZ, lddz, W, ldw, dX,
                       accum ? 1 : 0, add, out16, ld16);
    return hipGetLastError();
}

hipError_t launch_pack_bf16(int64_t rows, int64_t cols, const float* src, int64_t lds,
                            uint16_t* dst, int64_t ldd, int64_t col0, hipStream_t s) {
    SSMK_TIMED("pack", s);
    hipLaunchKernelGGL(k_pack, dim3(cdiv(rows * cols, 256)), dim3(256), 0, s, rows, cols, src, lds,
                       dst, ldd, col0);
    return hipGetLastError();
}

}  // namespace ssmk
