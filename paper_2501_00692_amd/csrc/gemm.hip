// gemm.hip -- bf16 MFMA GEMMs for the projection gradients (gfx950,
// v_mfma_f32_32x32x16_bf16, fp32 accumulation), one templated kernel:
//   dW[K][N] = X^T dZ  (X [M][K], dZ [M][N]): both operands are reduction-major
//       (TR); their tiles are kept reduction-major in LDS and the MFMA fragments
//       are read with the transposing LDS read (ds_read_b64_tr_b16, two per
//       fragment); split over M when the output has few tiles, with a
//       fixed-order second-stage reduction;
//   dX[M][K] = dZ W^T  (dZ [M][N], W [K][N]): both operands are contiguous along
//       the reduction; fragments are plain 16-byte LDS reads.  The epilogue adds
//       an optional fp32 addend, accumulates, and can write a bf16 copy into a
//       strided buffer; narrow outputs split the reduction like dW, and the
//       second stage applies the same epilogue.
// Staging: operand tiles go from global memory straight into LDS (buffer loads
// with the LDS destination, 16 bytes per lane, no registers on the way) through
// a ring of NS stages of BK = 32 reduction steps.  dX: step t waits (vmcnt) until
// its own loads of step t+1 have landed and meets the other waves at a barrier;
// then the loads of step t+NS-1 go into the stage that step t-1 used, and step
// t+1's first fragments are read while step t's second half of MFMAs runs.  dW:
// the two waves of a SIMD alternate between reading/loading and multiplying,
// half a step apart (ping-pong), with a barrier between phases.  Pieces
// outside the matrix (rows, columns, or the reduction tail) read as zero through
// the buffer range check.  Workgroup: 512 threads = 4x2 waves, two per SIMD;
// a wave owns a 64 x (BN/2) block of 32x32 MFMA tiles; tile 256 x BN with BN 128
// or 192.  256 x 256 tiles (dW, and dX with a plain epilogue) run on a kernel of
// their own (k_gemm4): 256 threads, one wave per SIMD owning a 128 x 128 block
// with its accumulators in the AGPRs, a five-stage ring (160 KB of LDS), one
// barrier per step and the MFMAs interleaved one by one with the fragment reads
// and stage loads.
// Output tiles and reduction splits are assigned so that each XCD runs one
// contiguous run of (split, tile) (consecutive workgroups go to different XCDs),
// tiles ordered in groups of four row blocks, so that the tiles one XCD runs at
// a time share row blocks of the first operand and column blocks of the second
// in its L2.
#include <type_traits>

#include "internal.h"

namespace ssmk {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));

constexpr int BK = 32;       // reduction steps per LDS stage
constexpr int BM = 256;      // output tile rows
constexpr int NS = 4;        // stages in the LDS ring
constexpr int kMaxW = 256;   // widest LDS row of the second operand (TR) / most rows (non-TR)
constexpr int kXcds = 8;
constexpr int kGroupRows = 4;  // row blocks per group of the tile order
constexpr uint32_t kOutOfRange = 0x80000000u;  // a buffer offset past every range
constexpr int kRsrcWord3 = 0x00020000;         // raw buffer, 32-bit data format

// The LDS ring: separate arrays per stage, so that the compiler sees reads of
// one stage as independent of the loads in flight into the others.
__shared__ __attribute__((aligned(1024))) uint16_t sA0[BM * BK];
__shared__ __attribute__((aligned(1024))) uint16_t sA1[BM * BK];
__shared__ __attribute__((aligned(1024))) uint16_t sA2[BM * BK];
__shared__ __attribute__((aligned(1024))) uint16_t sA3[BM * BK];
__shared__ __attribute__((aligned(1024))) uint16_t sB0[kMaxW * BK];
__shared__ __attribute__((aligned(1024))) uint16_t sB1[kMaxW * BK];
__shared__ __attribute__((aligned(1024))) uint16_t sB2[kMaxW * BK];
__shared__ __attribute__((aligned(1024))) uint16_t sB3[kMaxW * BK];
// a fifth stage, used by the four-wave dW kernel only (160 KB of LDS in all)
__shared__ __attribute__((aligned(1024))) uint16_t sA4[BM * BK];
__shared__ __attribute__((aligned(1024))) uint16_t sB4[kMaxW * BK];

template <int S>
__device__ __forceinline__ uint16_t* stage_a() {
    static_assert(S >= 0 && S <= NS, "stage");
    if constexpr (S == 0) return sA0;
    else if constexpr (S == 1) return sA1;
    else if constexpr (S == 2) return sA2;
    else if constexpr (S == 3) return sA3;
    else return sA4;
}
template <int S>
__device__ __forceinline__ uint16_t* stage_b() {
    static_assert(S >= 0 && S <= NS, "stage");
    if constexpr (S == 0) return sB0;
    else if constexpr (S == 1) return sB1;
    else if constexpr (S == 2) return sB2;
    else if constexpr (S == 3) return sB3;
    else return sB4;
}
template <int S>
using Stage = std::integral_constant<int, S>;

// Workgroup barrier that orders LDS accesses for the compiler only: the waits
// for the direct-to-LDS loads are explicit (wait_vm), and no other memory
// operation needs to complete at it.
__device__ __forceinline__ void ring_barrier() {
    __builtin_amdgcn_sched_barrier(0);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_sched_barrier(0);
}
// Wait until at most N of this wave's vector-memory operations are outstanding.
template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N >= 0 && N < 64, "vmcnt");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// 16 bytes per lane from buffer offset voff into LDS at lds + 16 * lane (lds is
// wave-uniform).
__device__ __forceinline__ void load_lds16(__amdgpu_buffer_rsrc_t rs, uint32_t voff, uint16_t* lds) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)lds, 16, voff, 0, 0, 0);
}
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const uint16_t* base, int64_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(base), 0, static_cast<int>(bytes), kRsrcWord3);
}
// The same from values every lane holds alike, taken from the first lane, so that
// the resource stays in scalar registers: a resource the compiler cannot prove
// uniform is kept in vector registers and every buffer load through it becomes a
// loop over its distinct values.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc_uniform(const uint16_t* base, int64_t bytes) {
    const uint64_t b = reinterpret_cast<uint64_t>(base);
    const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(b));
    const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(b >> 32));
    const int n = __builtin_amdgcn_readfirstlane(static_cast<int>(bytes));
    void* p = reinterpret_cast<void*>((static_cast<uint64_t>(hi) << 32) | lo);
    return __builtin_amdgcn_make_buffer_rsrc(p, 0, n, kRsrcWord3);
}

// fp32 -> bf16, round to nearest even (the hardware conversion, v_cvt_pk_bf16_f32)
__device__ __forceinline__ uint16_t f2bf(float v) { return __builtin_bit_cast(uint16_t, static_cast<__bf16>(v)); }

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
    const float* add;     // optional fp32 addend [R][Cc] (row stride ldadd)
    uint16_t* out16;      // optional bf16 copy of the result
    int64_t ld16;
    int64_t ldc;          // row stride of C when written directly (split partials: Cc)
    int64_t ldadd;        // row stride of add
};

// One launch covers the output tiles of one product, or of two products with the
// same reduction length and split (the layer's two weight gradients): in every
// split, tiles [0, tiles0) belong to product 0 and [tiles0, tiles) to product 1.
struct GemmLaunch {
    GemmArgs p[2];
    int tiles0;  // output tiles of product 0
    int tiles;   // output tiles of all products
    int cb[2];   // column blocks of each product
};

// Operands contiguous along the reduction (dX = dZ W^T).  A stage holds BM rows
// of A and BN rows of B, each a 64-byte LDS row of BK values whose four 16-byte
// blocks are XOR-swizzled by (row >> 2) & 3: a 16-byte fragment read by 32 lanes
// of consecutive rows then covers all 64 banks in every group of 16 lanes.
// A 1 KB wave load fills 16 rows; lane l supplies row l/4's logical block.
template <int BN>
struct RowMajorOps {
    static constexpr int NB = BN * BK * 2 / 1024;  // wave loads of B per stage
    __amdgpu_buffer_rsrc_t ra, rb;
    uint32_t oa[2], ob[2];
    int ka[2], kb[2];
    int64_t k_hi;
    int offa[2][2], offb[2][BN / 64];  // fragment offsets (elements) per sub-step

    static __device__ __forceinline__ int swz(int row) { return (row >> 2) & 3; }

    __device__ __forceinline__ void init(const GemmArgs& g, int64_t r0, int64_t c0, int64_t khi, int wave,
                                         int lane, int wr, int wc) {
        k_hi = khi;
        // resources over the tile's rows: rows past the matrix read as zero
        ra = rsrc_uniform(g.A + r0 * g.lda, min<int64_t>(BM, g.R - r0) * g.lda * 2);
        rb = rsrc_uniform(g.B + c0 * g.ldb, min<int64_t>(BN, g.Cc - c0) * g.ldb * 2);
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int row = (wave + 8 * i) * 16 + (lane >> 2);
            ka[i] = kb[i] = ((lane & 3) ^ swz(row)) * 8;
            oa[i] = static_cast<uint32_t>((row * g.lda + ka[i]) * 2);
            ob[i] = static_cast<uint32_t>((row * g.ldb + kb[i]) * 2);
        }
        const int li = lane & 31, hk = lane >> 5;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int row = wr + i * 32 + li;
                offa[ks][i] = row * BK + (((ks * 2 + hk) ^ swz(row)) * 8);
            }
#pragma unroll
            for (int j = 0; j < BN / 64; ++j) {
                const int row = wc + j * 32 + li;
                offb[ks][j] = row * BK + (((ks * 2 + hk) ^ swz(row)) * 8);
            }
        }
    }
    // pieces past the reduction range read out of range (zero)
    __device__ __forceinline__ uint32_t off(uint32_t o0, int kq, int64_t k) const {
        return k + kq < k_hi ? o0 + static_cast<uint32_t>(k * 2) : kOutOfRange;
    }
    template <int S>
    __device__ __forceinline__ void issue(Stage<S>, int64_t k, int wave) const {
#pragma unroll
        for (int i = 0; i < 2; ++i) load_lds16(ra, off(oa[i], ka[i], k), stage_a<S>() + (wave + 8 * i) * 512);
        if (wave < NB) load_lds16(rb, off(ob[0], kb[0], k), stage_b<S>() + wave * 512);
        if (wave + 8 < NB) load_lds16(rb, off(ob[1], kb[1], k), stage_b<S>() + (wave + 8) * 512);
    }
    template <int S>
    __device__ __forceinline__ void read(Stage<S>, int ks, bf16x8 (&a)[2], bf16x8 (&b)[BN / 64], int) const {
#pragma unroll
        for (int i = 0; i < 2; ++i)
            a[i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(stage_a<S>() + offa[ks][i]));
#pragma unroll
        for (int j = 0; j < BN / 64; ++j)
            b[j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(stage_b<S>() + offb[ks][j]));
    }
};

// Reduction-major operands (dW = X^T dZ).  A stage holds BK rows (reduction
// steps) of WA = BM values of A and WB values of B (BN, or 256 for BN = 192 so
// that a row stays a power of two of 16-byte blocks); block b of row k sits at
// b ^ 4(k & 3).  A fragment (8 consecutive reduction steps of one column per
// lane) is two transposing 8-byte reads: in each group of 16 lanes, lane 4q+r
// receives element r of the 8-byte chunk addressed by lane 4j+q, j = 0..3, so
// lane l addresses (step 8(l/32) + 4h + (l%16)/4, columns 16((l/16)%2) + 4(l%4)
// .. +3) and receives column l%32 at steps 8(l/32) + 4h + j.  The swizzle keeps
// each 32-lane half free of bank conflicts.
template <int BN>
struct ColMajorOps {
    static constexpr int WA = BM, WB = BN == 192 ? 256 : BN;
    static constexpr int NB = BK * WB * 2 / 1024;
    static_assert(WB <= kMaxW, "LDS row");
    const uint16_t* A;
    const uint16_t* B;
    int64_t lda, ldb, k_hi;
    uint32_t oa[2], ob[2];
    int fa[2][2][2], fb[2][BN / 64][2];  // fragment read byte offsets [sub-step][tile][half]

    static __device__ __forceinline__ int swz(int k) { return (k & 3) << 2; }
    // byte offset of the 8-byte chunk lane `lane` addresses for the fragment of
    // columns col0 .. col0+31 at reduction steps ks + 8(lane/32) + 4h .. +3
    static __device__ __forceinline__ int chunk(int W, int ks, int h, int col0, int lane) {
        const int col = col0 + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
        const int k = ks + 8 * (lane >> 5) + 4 * h + ((lane & 15) >> 2);
        return k * W * 2 + (((col >> 3) ^ swz(k)) << 4) + (((col >> 2) & 1) << 3);
    }

    __device__ __forceinline__ void init(const GemmArgs& g, int64_t r0, int64_t c0, int64_t khi, int wave,
                                         int lane, int wr, int wc) {
        A = g.A;
        B = g.B;
        lda = g.lda;
        ldb = g.ldb;
        k_hi = khi;
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int byte = (wave + 8 * i) * 1024 + lane * 16;
            {
                const int row = byte / (WA * 2), col = ((byte % (WA * 2)) / 16 ^ swz(row)) * 8;
                oa[i] = r0 + col < g.R ? static_cast<uint32_t>((row * g.lda + r0 + col) * 2) : kOutOfRange;
            }
            {
                const int row = byte / (WB * 2), col = ((byte % (WB * 2)) / 16 ^ swz(row)) * 8;
                ob[i] = (col < BN && c0 + col < g.Cc) ? static_cast<uint32_t>((row * g.ldb + c0 + col) * 2)
                                                      : kOutOfRange;
            }
        }
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
#pragma unroll
                for (int i = 0; i < 2; ++i) fa[ks][i][h] = chunk(WA, ks * 16, h, wr + i * 32, lane);
#pragma unroll
                for (int j = 0; j < BN / 64; ++j) fb[ks][j][h] = chunk(WB, ks * 16, h, wc + j * 32, lane);
            }
    }
    template <int S>
    __device__ __forceinline__ void issue(Stage<S>, int64_t k, int wave) const {
        // resources over reduction rows k .. min(k + BK, k_hi): later rows read zero
        const int64_t rows = min<int64_t>(BK, k_hi - k);
        const __amdgpu_buffer_rsrc_t ra = rsrc(A + k * lda, rows * lda * 2);
        const __amdgpu_buffer_rsrc_t rb = rsrc(B + k * ldb, rows * ldb * 2);
#pragma unroll
        for (int i = 0; i < 2; ++i) load_lds16(ra, oa[i], stage_a<S>() + (wave + 8 * i) * 512);
        if (wave < NB) load_lds16(rb, ob[0], stage_b<S>() + wave * 512);
        if (wave + 8 < NB) load_lds16(rb, ob[1], stage_b<S>() + (wave + 8) * 512);
    }
    static __device__ __forceinline__ bf16x8 frag(const uint16_t* T, const int (&o)[2]) {
        const char* base = reinterpret_cast<const char*>(T);
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(base + o[0]));
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(base + o[1]));
        const s16x8 w = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        return __builtin_bit_cast(bf16x8, w);
    }
    template <int S>
    __device__ __forceinline__ void read(Stage<S>, int ks, bf16x8 (&a)[2], bf16x8 (&b)[BN / 64], int) const {
#pragma unroll
        for (int i = 0; i < 2; ++i) a[i] = frag(stage_a<S>(), fa[ks][i]);
#pragma unroll
        for (int j = 0; j < BN / 64; ++j) b[j] = frag(stage_b<S>(), fb[ks][j]);
    }
};

// Epilogue of one wave's MI x NJ block of 32x32 tiles (rows from row0, columns
// from col0): result = acc (+ add) (+ C if ACC), written to C (DST) and/or as
// bf16 (O16).  acc element v of lane l is row 8(v/4) + 4(l/32) + v%4, column
// l%32 of its tile.  FULL: the block lies inside the output (no checks).
template <bool ADD, bool ACC, bool DST, bool O16, bool FULL, int MI, int NJ>
__device__ __forceinline__ void store_tile(const f32x16 (&acc)[MI][NJ], float* __restrict__ dst, int64_t ldc,
                                           const float* __restrict__ addp, int64_t ldadd, uint16_t* __restrict__ o16,
                                           int64_t ld16, int64_t R, int64_t Cc, int64_t row0, int64_t col0, int lane) {
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int64_t col = col0 + j * 32 + (lane & 31);
            const int64_t rb = row0 + i * 32 + 4 * (lane >> 5);
            // the tile's addends first, so that their loads overlap
            float extra[16];
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t row = rb + 8 * (v >> 2) + (v & 3);
                const bool in = FULL || (row < R && col < Cc);
                // out-of-range lanes read element 0
                float e = 0.f;
                if constexpr (ADD) e = addp[in ? row * ldadd + col : 0];
                if constexpr (ACC) e += dst[in ? row * ldc + col : 0];
                extra[v] = e;
            }
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t row = rb + 8 * (v >> 2) + (v & 3);
                if (FULL || (row < R && col < Cc)) {
                    const float val = acc[i][j][v] + extra[v];
                    if constexpr (DST) dst[row * ldc + col] = val;
                    if constexpr (O16) o16[row * ld16 + col] = f2bf(val);
                }
            }
        }
}

template <bool TR, int BN>
__global__ __launch_bounds__(512) void k_gemm(const GemmLaunch gl) {
    constexpr int MI = 2, NJ = BN / 64;  // 32x32 MFMA tiles per wave
    using Ops = typename std::conditional<TR, ColMajorOps<BN>, RowMajorOps<BN>>::type;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // output tile and reduction split: workgroups are dispatched to the XCDs in
    // turn (workgroup i to XCD i % 8), so the linear id is mapped to a logical
    // index that gives every XCD one contiguous run of (split, product, row block,
    // column block) -- the workgroups of one XCD share the first operand's row
    // block and reduction range in its L2.  The map is a bijection for any count.
    const int nwg = static_cast<int>(gridDim.x);
    const int lin = static_cast<int>(blockIdx.x);
    const int xq = nwg / kXcds, xr = nwg % kXcds, xcd = lin % kXcds;
    const int logical = (xcd < xr ? xcd * (xq + 1) : xr * (xq + 1) + (xcd - xr) * xq) + lin / kXcds;
    const int tile_all = logical % gl.tiles, split = logical / gl.tiles;
    // the product (wave-uniform; taken from the first lane so that the compiler
    // keeps its pointers and the buffer resources built from them in SGPRs)
    const int q = __builtin_amdgcn_readfirstlane(tile_all >= gl.tiles0 ? 1 : 0);
    const GemmArgs g = q ? gl.p[1] : gl.p[0];
    const int tile = tile_all - (q ? gl.tiles0 : 0);
    const int ncb = q ? gl.cb[1] : gl.cb[0];  // a select: an indexed kernel argument would not be uniform
    const int nrb = (q ? gl.tiles - gl.tiles0 : gl.tiles0) / ncb;
    // tiles in groups of kGroupRows row blocks, column-major inside a group, so
    // that the 32 consecutive tiles one XCD runs at a time form a block of about
    // 4 row blocks x 8 column blocks (both operands reused from its L2)
    const int grp = tile / (kGroupRows * ncb), first = grp * kGroupRows;
    const int gh = min(kGroupRows, nrb - first), within = tile - grp * kGroupRows * ncb;
    const int64_t r0 = static_cast<int64_t>(first + within % gh) * BM;
    const int64_t c0 = static_cast<int64_t>(within / gh) * BN;
    const int64_t k_lo = static_cast<int64_t>(split) * g.kper;
    const int64_t k_hi = min(g.Kr, k_lo + g.kper);
    const int wr = (wave >> 1) * 64;
    const int wc = (wave & 1) * (BN / 2);
    const int64_t nsteps = k_hi > k_lo ? (k_hi - k_lo + BK - 1) / BK : 0;

    Ops ops;
    ops.init(g, r0, c0, k_hi, wave, lane, wr, wc);
    f32x16 acc[MI][NJ];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
    typedef bf16x8 FA[MI];
    typedef bf16x8 FB[NJ];
    auto mm = [&](const FA& a, const FB& b) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < MI; ++i)
#pragma unroll
            for (int j = 0; j < NJ; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    };
    auto read_any = [&](int s, int ks, FA& a, FB& b) __attribute__((always_inline)) {
        switch (s) {
            case 0: ops.read(Stage<0>{}, ks, a, b, lane); break;
            case 1: ops.read(Stage<1>{}, ks, a, b, lane); break;
            case 2: ops.read(Stage<2>{}, ks, a, b, lane); break;
            default: ops.read(Stage<3>{}, ks, a, b, lane); break;
        }
    };
    // loads per wave per stage: two of A, one or two (or none) of B
    const int per = 2 + (wave < Ops::NB ? 1 : 0) + (wave + 8 < Ops::NB ? 1 : 0);
    auto wait_groups = [&](auto Gt) __attribute__((always_inline)) {  // G later stages may stay in flight
        constexpr int G = decltype(Gt)::value;
        if (per == 4) wait_vm<4 * G>();
        else if (per == 3) wait_vm<3 * G>();
        else wait_vm<2 * G>();
    };
    static_assert(NS == 4, "the ring code below is written for four stages");
    if constexpr (TR) {
        // dW: ping-pong schedule.  The two waves of a SIMD (w and w + 4) take turns,
        // half a step apart, between a memory phase -- wait for the wave's own loads
        // of the next stages, read the step's fragments from LDS, issue the loads
        // three stages ahead -- and an MFMA phase (the step's 2 x MI x NJ MFMAs), with
        // a workgroup barrier between phases: while one wave of a SIMD multiplies,
        // the other feeds (dW at the layer workload 93 -> 85 us; the dX form, whose
        // plain fragment reads are cheaper, gained nothing from it and keeps the
        // schedule below).
        if (nsteps > 0) ops.issue(Stage<0>{}, k_lo, wave);
        if (nsteps > 1) ops.issue(Stage<1>{}, k_lo + BK, wave);
        if (nsteps > 2) ops.issue(Stage<2>{}, k_lo + 2 * BK, wave);
        FA a0, a1;
        FB b0, b1;
        // memory phase of step s: this wave's loads of stages <= s + 1 have landed
        // (stage s + 2 may stay in flight; every wave waited for its share of stage s
        // before an earlier barrier), the fragments of stage s are read and in
        // registers before the next barrier (the other group reloads the slot read
        // one step before), and stage s + 3 is issued into the slot of step s - 1
        auto mem = [&](auto St, int64_t s) __attribute__((always_inline)) {
            constexpr int S = decltype(St)::value;
            if (s + 2 < nsteps) wait_groups(std::integral_constant<int, 1>{});
            else wait_vm<0>();
            ops.read(St, 0, a0, b0, lane);
            ops.read(St, 1, a1, b1, lane);
            if (s + 3 < nsteps) ops.issue(Stage<(S + 3) % NS>{}, k_lo + (s + 3) * BK, wave);
            __builtin_amdgcn_s_waitcnt(0xC07F);  // LDS reads done (vmcnt and expcnt unchanged)
        };
        if (nsteps > 2) wait_groups(std::integral_constant<int, 1>{});
        else wait_vm<0>();
        ring_barrier();
        auto mfma = [&]() __attribute__((always_inline)) {
            mm(a0, b0);
            mm(a1, b1);
        };
        // one step: its memory phase, a barrier, its MFMA phase, and the barrier that
        // ends the interval unless it is the wave's last
        auto pp_step = [&](auto St, int64_t s, bool last_barrier) __attribute__((always_inline)) {
            mem(St, s);
            ring_barrier();
            mfma();
            if (last_barrier) ring_barrier();
        };
        // group 0 (waves 0-3) starts with the memory phase of step 0; group 1 (waves
        // 4-7) one interval later and so skips the barrier after its last MFMA phase:
        // both groups pass 2 nsteps barriers
        const bool g1 = wave >= 4;
        if (g1 && nsteps > 0) ring_barrier();
        int64_t t = 0;
        for (; t + NS <= nsteps; t += NS) {
            pp_step(Stage<0>{}, t, !g1 || t + 1 < nsteps);
            pp_step(Stage<1>{}, t + 1, !g1 || t + 2 < nsteps);
            pp_step(Stage<2>{}, t + 2, !g1 || t + 3 < nsteps);
            pp_step(Stage<3>{}, t + 3, !g1 || t + 4 < nsteps);
        }
        const int64_t rem = nsteps - t;
        if (rem > 0) pp_step(Stage<0>{}, t, !g1 || t + 1 < nsteps);
        if (rem > 1) pp_step(Stage<1>{}, t + 1, !g1 || t + 2 < nsteps);
        if (rem > 2) pp_step(Stage<2>{}, t + 2, !g1 || t + 3 < nsteps);
    } else {
        // dX: every wave reads, multiplies and loads in each step, one barrier per
        // step.
        if (nsteps > 0) ops.issue(Stage<0>{}, k_lo, wave);
        if (nsteps > 1) ops.issue(Stage<1>{}, k_lo + BK, wave);
        if (nsteps > 2) ops.issue(Stage<2>{}, k_lo + 2 * BK, wave);
        // steady steps issue a load group each; the last NS-1 steps only drain
        const int64_t steady = nsteps >= NS - 1 ? nsteps - (NS - 1) : 0;
        if (steady > 0) wait_groups(std::integral_constant<int, NS - 2>{});
        else wait_vm<0>();
        ring_barrier();
        FA a0, a1;
        FB b0, b1;
        if (nsteps > 0) ops.read(Stage<0>{}, 0, a0, b0, lane);
        auto step = [&](auto St, int64_t t) __attribute__((always_inline)) {
            constexpr int S = decltype(St)::value;
            ops.read(St, 1, a1, b1, lane);
            __builtin_amdgcn_sched_barrier(0);
            mm(a0, b0);
            wait_groups(std::integral_constant<int, NS - 3>{});  // step t+1's loads, every wave
            ring_barrier();
            ops.issue(Stage<(S + NS - 1) % NS>{}, k_lo + (t + NS - 1) * BK, wave);
            ops.read(Stage<(S + 1) % NS>{}, 0, a0, b0, lane);
            __builtin_amdgcn_sched_barrier(0);
            mm(a1, b1);
            __builtin_amdgcn_sched_barrier(0);
        };
        int64_t t = 0;
        auto ring = [&](int64_t t) __attribute__((always_inline)) {
            step(Stage<0>{}, t);
            step(Stage<1>{}, t + 1);
            step(Stage<2>{}, t + 2);
            step(Stage<3>{}, t + 3);
        };
        // four rings per loop iteration: the compiler's own drain of the loads in
        // flight at the loop head (see k_gemm4) comes once per 16 steps
        constexpr int kRings = 4;
        for (; t + kRings * NS <= steady; t += kRings * NS) {
#pragma unroll
            for (int u = 0; u < kRings; ++u) ring(t + u * NS);
        }
        for (; t + NS <= steady; t += NS) ring(t);
        const int64_t rem = steady - t;  // t is a multiple of NS here
        if (rem > 0) step(Stage<0>{}, t);
        if (rem > 1) step(Stage<1>{}, t + 1);
        if (rem > 2) step(Stage<2>{}, t + 2);
        if (steady > 0 && steady < nsteps) {
            wait_vm<0>();
            ring_barrier();
        }
        for (int64_t u = steady; u < nsteps; ++u) {
            const int s = static_cast<int>(u % NS);
            read_any(s, 1, a1, b1);
            mm(a0, b0);
            if (u + 1 < nsteps) read_any(s + 1 == NS ? 0 : s + 1, 0, a0, b0);
            mm(a1, b1);
        }
    }

    float* dst = g.C ? g.C + (g.direct ? 0 : static_cast<int64_t>(split) * g.R * g.Cc) : nullptr;
    const float* addp = g.direct ? g.add : nullptr;
    uint16_t* o16 = g.direct ? g.out16 : nullptr;
    const bool accum = g.direct && g.accum && dst;
    const bool full = r0 + BM <= g.R && c0 + BN <= g.Cc;
    // one specialised store per combination of outputs in use (uniform per tile)
    const int mask = (addp ? 1 : 0) | (accum ? 2 : 0) | (dst ? 4 : 0) | (o16 ? 8 : 0);
    auto store = [&](auto Ft, auto Mt) __attribute__((always_inline)) {
        constexpr int M = decltype(Mt)::value;
        store_tile<(M & 1) != 0, (M & 2) != 0, (M & 4) != 0, (M & 8) != 0, decltype(Ft)::value>(
            acc, dst, g.direct ? g.ldc : g.Cc, addp, g.ldadd, o16, g.ld16, g.R, g.Cc, r0 + wr, c0 + wc, lane);
    };
    auto by_mask = [&](auto Ft) __attribute__((always_inline)) {
        if constexpr (TR) {  // dW: C or C += (split partials are C)
            if (mask == 6) store(Ft, std::integral_constant<int, 6>{});
            else store(Ft, std::integral_constant<int, 4>{});
            return;
        }
        switch (mask) {
            case 4: store(Ft, std::integral_constant<int, 4>{}); break;     // C
            case 6: store(Ft, std::integral_constant<int, 6>{}); break;     // C +=
            case 5: store(Ft, std::integral_constant<int, 5>{}); break;     // C = . + add
            case 7: store(Ft, std::integral_constant<int, 7>{}); break;     // C += . + add
            case 8: store(Ft, std::integral_constant<int, 8>{}); break;     // bf16 copy only
            case 9: store(Ft, std::integral_constant<int, 9>{}); break;     // bf16 of . + add
            case 12: store(Ft, std::integral_constant<int, 12>{}); break;   // C and its bf16 copy
            case 13: store(Ft, std::integral_constant<int, 13>{}); break;
            case 14: store(Ft, std::integral_constant<int, 14>{}); break;
            case 15: store(Ft, std::integral_constant<int, 15>{}); break;
            default: break;                                                 // no output
        }
    };
    if (full) by_mask(std::true_type{});
    else by_mask(std::false_type{});
}

// The dW form with four waves, one per SIMD, each owning a 128 x 128 block of
// the 256 x 256 tile (4 x 4 MFMA tiles, 256 accumulator registers): per 32-step
// stage the waves read 64 KB of fragments from LDS instead of the 96 KB that
// eight 64 x 128 blocks read.  Operand staging as in ColMajorOps (four wave
// loads of A and four of B per wave and stage).  Schedule as the dX form's: one
// barrier per step; a step's second-half fragments are read while its first half
// of MFMAs runs, and the next step's first-half fragments while its second half
// runs.
struct ColMajorOps4 {
    static constexpr int W = 256;  // LDS row of both operands (values)
    const uint16_t* A;
    const uint16_t* B;
    int64_t lda, ldb, k_hi;
    uint32_t oa[4], ob[4];
    int fa[2][4][2], fb[2][4][2];

    __device__ __forceinline__ void init(const GemmArgs& g, int64_t r0, int64_t c0, int64_t khi, int wave,
                                         int lane, int wr, int wc) {
        A = g.A;
        B = g.B;
        lda = g.lda;
        ldb = g.ldb;
        k_hi = khi;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int byte = (wave + 4 * i) * 1024 + lane * 16;
            const int row = byte / (W * 2), col = ((byte % (W * 2)) / 16 ^ ColMajorOps<256>::swz(row)) * 8;
            oa[i] = r0 + col < g.R ? static_cast<uint32_t>((row * g.lda + r0 + col) * 2) : kOutOfRange;
            ob[i] = c0 + col < g.Cc ? static_cast<uint32_t>((row * g.ldb + c0 + col) * 2) : kOutOfRange;
        }
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    fa[ks][i][h] = ColMajorOps<256>::chunk(W, ks * 16, h, wr + i * 32, lane);
                    fb[ks][i][h] = ColMajorOps<256>::chunk(W, ks * 16, h, wc + i * 32, lane);
                }
    }
    template <int S>
    __device__ __forceinline__ void issue(Stage<S>, int64_t k, int wave) const {
        const int64_t rows = min<int64_t>(BK, k_hi - k);
        const __amdgpu_buffer_rsrc_t ra = rsrc(A + k * lda, rows * lda * 2);
        const __amdgpu_buffer_rsrc_t rb = rsrc(B + k * ldb, rows * ldb * 2);
#pragma unroll
        for (int i = 0; i < 4; ++i) load_lds16(ra, oa[i], stage_a<S>() + (wave + 4 * i) * 512);
#pragma unroll
        for (int i = 0; i < 4; ++i) load_lds16(rb, ob[i], stage_b<S>() + (wave + 4 * i) * 512);
    }
    template <int S>
    __device__ __forceinline__ void read(Stage<S>, int ks, bf16x8 (&a)[4], bf16x8 (&b)[4]) const {
#pragma unroll
        for (int i = 0; i < 4; ++i) a[i] = ColMajorOps<256>::frag(stage_a<S>(), fa[ks][i]);
#pragma unroll
        for (int j = 0; j < 4; ++j) b[j] = ColMajorOps<256>::frag(stage_b<S>(), fb[ks][j]);
    }
};

// The dX form (operands contiguous along the reduction) on the four-wave
// kernel: the LDS layout of RowMajorOps (64-byte rows of 32 steps, 16-byte
// blocks XOR-swizzled by (row >> 2) & 3), 256 rows of each operand per stage,
// four wave loads of A and four of B per wave and stage; each wave reads the
// 16-byte fragments of its 128 rows of A and 128 rows of B.
struct RowMajorOps4 {
    __amdgpu_buffer_rsrc_t ra, rb;
    uint32_t oa[4], ob[4];
    int ka[4], kb[4];
    int64_t k_hi;
    int offa[2][4], offb[2][4];  // fragment offsets (elements) per sub-step

    __device__ __forceinline__ void init(const GemmArgs& g, int64_t r0, int64_t c0, int64_t khi, int wave,
                                         int lane, int wr, int wc) {
        k_hi = khi;
        // resources over the tile's rows: rows past the matrix read as zero
        ra = rsrc_uniform(g.A + r0 * g.lda, min<int64_t>(BM, g.R - r0) * g.lda * 2);
        rb = rsrc_uniform(g.B + c0 * g.ldb, min<int64_t>(256, g.Cc - c0) * g.ldb * 2);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int row = (wave + 4 * i) * 16 + (lane >> 2);
            ka[i] = kb[i] = ((lane & 3) ^ RowMajorOps<128>::swz(row)) * 8;
            oa[i] = static_cast<uint32_t>((row * g.lda + ka[i]) * 2);
            ob[i] = static_cast<uint32_t>((row * g.ldb + kb[i]) * 2);
        }
        const int li = lane & 31, hk = lane >> 5;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int ra_ = wr + i * 32 + li, rb_ = wc + i * 32 + li;
                offa[ks][i] = ra_ * BK + (((ks * 2 + hk) ^ RowMajorOps<128>::swz(ra_)) * 8);
                offb[ks][i] = rb_ * BK + (((ks * 2 + hk) ^ RowMajorOps<128>::swz(rb_)) * 8);
            }
    }
    // pieces past the reduction range read out of range (zero)
    __device__ __forceinline__ uint32_t off(uint32_t o0, int kq, int64_t k) const {
        return k + kq < k_hi ? o0 + static_cast<uint32_t>(k * 2) : kOutOfRange;
    }
    template <int S>
    __device__ __forceinline__ void issue(Stage<S>, int64_t k, int wave) const {
#pragma unroll
        for (int i = 0; i < 4; ++i) load_lds16(ra, off(oa[i], ka[i], k), stage_a<S>() + (wave + 4 * i) * 512);
#pragma unroll
        for (int i = 0; i < 4; ++i) load_lds16(rb, off(ob[i], kb[i], k), stage_b<S>() + (wave + 4 * i) * 512);
    }
    template <int S>
    __device__ __forceinline__ void read(Stage<S>, int ks, bf16x8 (&a)[4], bf16x8 (&b)[4]) const {
#pragma unroll
        for (int i = 0; i < 4; ++i)
            a[i] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(stage_a<S>() + offa[ks][i]));
#pragma unroll
        for (int j = 0; j < 4; ++j)
            b[j] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(stage_b<S>() + offb[ks][j]));
    }
};

// Four waves, one per SIMD, each owning a 128 x 128 block of a 256 x 256 output
// tile: TR selects the dW form (ColMajorOps4) or the dX form (RowMajorOps4, plain
// epilogues only: no addend, and the fp32 result or its bf16 copy, not both).
template <bool TR, int NST>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void k_gemm4(const GemmLaunch gl) {
    constexpr int MI = 4, NJ = 4, BN = 256;
    static_assert(NST == 4 || NST == 5, "stages");
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // tile and split of this workgroup: the same XCD-contiguous map and grouped
    // tile order as k_gemm
    const int nwg = static_cast<int>(gridDim.x);
    const int lin = static_cast<int>(blockIdx.x);
    const int xq = nwg / kXcds, xr = nwg % kXcds, xcd = lin % kXcds;
    const int logical = (xcd < xr ? xcd * (xq + 1) : xr * (xq + 1) + (xcd - xr) * xq) + lin / kXcds;
    const int tile_all = logical % gl.tiles, split = logical / gl.tiles;
    const int q = __builtin_amdgcn_readfirstlane(tile_all >= gl.tiles0 ? 1 : 0);
    const GemmArgs g = q ? gl.p[1] : gl.p[0];
    const int tile = tile_all - (q ? gl.tiles0 : 0);
    const int ncb = q ? gl.cb[1] : gl.cb[0];  // a select: an indexed kernel argument would not be uniform
    const int nrb = (q ? gl.tiles - gl.tiles0 : gl.tiles0) / ncb;
    const int grp = tile / (kGroupRows * ncb), first = grp * kGroupRows;
    const int gh = min(kGroupRows, nrb - first), within = tile - grp * kGroupRows * ncb;
    const int64_t r0 = static_cast<int64_t>(first + within % gh) * BM;
    const int64_t c0 = static_cast<int64_t>(within / gh) * BN;
    const int64_t k_lo = static_cast<int64_t>(split) * g.kper;
    const int64_t k_hi = min(g.Kr, k_lo + g.kper);
    const int wr = (wave >> 1) * 128;
    const int wc = (wave & 1) * 128;
    const int64_t nsteps = k_hi > k_lo ? (k_hi - k_lo + BK - 1) / BK : 0;

    std::conditional_t<TR, ColMajorOps4, RowMajorOps4> ops;
    ops.init(g, r0, c0, k_hi, wave, lane, wr, wc);
    f32x16 acc[MI][NJ];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
    typedef bf16x8 FA[MI];
    typedef bf16x8 FB[NJ];
    auto mm = [&](const FA& a, const FB& b) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < MI; ++i)
#pragma unroll
            for (int j = 0; j < NJ; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    };
    auto read_any = [&](int s, int ks, FA& a, FB& b) __attribute__((always_inline)) {
        switch (s) {
            case 0: ops.read(Stage<0>{}, ks, a, b); break;
            case 1: ops.read(Stage<1>{}, ks, a, b); break;
            case 2: ops.read(Stage<2>{}, ks, a, b); break;
            case 3: ops.read(Stage<3>{}, ks, a, b); break;
            default: ops.read(Stage<(NST > 4 ? 4 : 3)>{}, ks, a, b); break;
        }
    };
    constexpr int PER = 8;  // wave loads per stage
    // the first NST - 1 stages
    if (nsteps > 0) ops.issue(Stage<0>{}, k_lo, wave);
    if (nsteps > 1) ops.issue(Stage<1>{}, k_lo + BK, wave);
    if (nsteps > 2) ops.issue(Stage<2>{}, k_lo + 2 * BK, wave);
    if constexpr (NST == 5)
        if (nsteps > 3) ops.issue(Stage<3>{}, k_lo + 3 * BK, wave);
    const int64_t steady = nsteps >= NST - 1 ? nsteps - (NST - 1) : 0;
    if (steady > 0) wait_vm<PER * (NST - 2)>();
    else wait_vm<0>();
    ring_barrier();
    FA a0, a1;
    FB b0, b1;
    if (nsteps > 0) ops.read(Stage<0>{}, 0, a0, b0);
    // MFMAs interleaved with the fragment reads (and the stage loads) of the
    // other half step, one read or load between consecutive MFMAs, so that the
    // matrix pipe is not left idle while they issue
    auto interleave = [&](auto Loads) __attribute__((always_inline)) {
        constexpr int NL = decltype(Loads)::value;
#pragma unroll
        for (int k = 0; k < MI * NJ; ++k) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);      // one MFMA
            if (k < NL) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // one stage load
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);      // one fragment read
        }
    };
    auto step = [&](auto St, int64_t t) __attribute__((always_inline)) {
        constexpr int S = decltype(St)::value;
        ops.read(St, 1, a1, b1);
        mm(a0, b0);
        interleave(std::integral_constant<int, 0>{});
        wait_vm<PER * (NST - 3)>();  // step t+1's loads, every wave
        ring_barrier();
        ops.issue(Stage<(S + NST - 1) % NST>{}, k_lo + (t + NST - 1) * BK, wave);
        ops.read(Stage<(S + 1) % NST>{}, 0, a0, b0);
        mm(a1, b1);
        interleave(std::integral_constant<int, PER>{});
        __builtin_amdgcn_sched_barrier(0);
    };
    int64_t t = 0;
    auto ring = [&](int64_t t) __attribute__((always_inline)) {
        step(Stage<0>{}, t);
        step(Stage<1>{}, t + 1);
        step(Stage<2>{}, t + 2);
        step(Stage<3>{}, t + 3);
        if constexpr (NST == 5) step(Stage<(NST > 4 ? 4 : 3)>{}, t + 4);
    };
    // Four passes over the ring per loop iteration: at the loop head the compiler
    // no longer knows which stage each direct-to-LDS load in flight writes, and
    // waits for nearly all of them before the first fragment read (vmcnt(4), then
    // vmcnt(0)), where the explicit waits need only the next stage's; with the
    // body four rings long that drain comes once per 20 steps instead of 5.
    constexpr int kRings = 4;
    for (; t + kRings * NST <= steady; t += kRings * NST) {
#pragma unroll
        for (int u = 0; u < kRings; ++u) ring(t + u * NST);
    }
    for (; t + NST <= steady; t += NST) ring(t);
    const int64_t rem = steady - t;
    if (rem > 0) step(Stage<0>{}, t);
    if (rem > 1) step(Stage<1>{}, t + 1);
    if (rem > 2) step(Stage<2>{}, t + 2);
    if constexpr (NST == 5)
        if (rem > 3) step(Stage<3>{}, t + 3);
    if (steady > 0 && steady < nsteps) {
        wait_vm<0>();
        ring_barrier();
    }
    for (int64_t u = steady; u < nsteps; ++u) {
        const int s = static_cast<int>(u % NST);
        read_any(s, 1, a1, b1);
        mm(a0, b0);
        if (u + 1 < nsteps) read_any(s + 1 == NST ? 0 : s + 1, 0, a0, b0);
        mm(a1, b1);
    }

    float* dst = g.C + (g.direct ? 0 : static_cast<int64_t>(split) * g.R * g.Cc);
    const bool accum = g.direct && g.accum;
    const bool full = r0 + BM <= g.R && c0 + BN <= g.Cc;
    const int64_t ldc = g.direct ? g.ldc : g.Cc;
    auto store = [&](auto Ft, auto At) __attribute__((always_inline)) {
        store_tile<false, decltype(At)::value, true, false, decltype(Ft)::value>(
            acc, dst, ldc, nullptr, 0, nullptr, 0, g.R, g.Cc, r0 + wr, c0 + wc, lane);
    };
    if constexpr (!TR) {
        // the dX form's other plain epilogue: only the bf16 copy (no fp32 result)
        if (g.direct && g.out16) {
            if (full)
                store_tile<false, false, false, true, true>(acc, nullptr, 0, nullptr, 0, g.out16, g.ld16, g.R, g.Cc,
                                                            r0 + wr, c0 + wc, lane);
            else
                store_tile<false, false, false, true, false>(acc, nullptr, 0, nullptr, 0, g.out16, g.ld16, g.R, g.Cc,
                                                             r0 + wr, c0 + wc, lane);
            return;
        }
    }
    if (full) {
        if (accum) store(std::true_type{}, std::true_type{});
        else store(std::true_type{}, std::false_type{});
    } else {
        if (accum) store(std::false_type{}, std::true_type{});
        else store(std::false_type{}, std::false_type{});
    }
}

// Second stage of a split GEMM: result = sum over splits (in split order) +
// (add) (+ the existing C if accum), the same combination as the single-pass
// epilogue, written to C (if given) and/or as bf16 into out16 (row stride ld16).
// Four consecutive elements of a row per thread (the output width is a multiple
// of 8); the loads of up to eight splits are issued ahead of the in-order adds.
// One launch serves the products of one GEMM launch: workgroups [0, blocks0)
// reduce product 0, the rest product 1.
struct ReduceArgs {
    int64_t R, Cc;
    const float* part;  // [splits][R][Cc]
    float* dst;         // row stride ldc
    int accum;
    const float* add;   // row stride ldadd
    uint16_t* out16;
    int64_t ld16;
    int64_t ldc, ldadd;
};
struct ReduceLaunch {
    ReduceArgs p[2];
    unsigned blocks0;
    int splits;
};

__global__ __launch_bounds__(256) void k_splitk_reduce(const ReduceLaunch rl) {
    const int q = blockIdx.x >= rl.blocks0 ? 1 : 0;
    const ReduceArgs& a = rl.p[q];
    const int64_t blk = static_cast<int64_t>(blockIdx.x) - (q ? rl.blocks0 : 0);
    const int64_t RC = a.R * a.Cc;
    const int64_t i = (blk * 256 + threadIdx.x) * 4;
    if (i >= RC) return;
    const int splits = rl.splits;
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int q0 = 0; q0 < splits; q0 += 8) {
        float4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            v[u] = q0 + u < splits ? *reinterpret_cast<const float4*>(a.part + (q0 + u) * RC + i)
                                   : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            if (q0 + u < splits) {
                s.x += v[u].x;
                s.y += v[u].y;
                s.z += v[u].z;
                s.w += v[u].w;
            }
        }
    }
    const int64_t row = i / a.Cc, col = i - row * a.Cc;
    float4 e = a.add ? *reinterpret_cast<const float4*>(a.add + row * a.ldadd + col) : make_float4(0.f, 0.f, 0.f, 0.f);
    if (a.accum) {
        const float4 d = *reinterpret_cast<const float4*>(a.dst + row * a.ldc + col);
        e = make_float4(e.x + d.x, e.y + d.y, e.z + d.z, e.w + d.w);
    }
    const float4 val = make_float4(s.x + e.x, s.y + e.y, s.z + e.z, s.w + e.w);
    if (a.dst) *reinterpret_cast<float4*>(a.dst + row * a.ldc + col) = val;
    if (a.out16) {
        uint16_t* o = a.out16 + row * a.ld16 + col;
        o[0] = f2bf(val.x);
        o[1] = f2bf(val.y);
        o[2] = f2bf(val.z);
        o[3] = f2bf(val.w);
    }
}

inline int64_t cdiv64(int64_t a, int64_t b) { return (a + b - 1) / b; }

constexpr int kCUs = 256;
// Most workgroups of one launch (the grid is one-dimensional and its thread count
// must fit 32 bits).
constexpr int64_t kMaxWgs = (int64_t(1) << 23) - 1;

// Output-tile width and reduction splits for the outputs R_q x Cc_q of one launch
// (one or two products) with reduction Kr, from a simple time model: rounds of 256
// workgroups x the time of one workgroup's share (per 32-step stage at full
// load, measured: 0.57 us for 128 columns, 0.80 for 192, 0.84 for 256 on the
// four-wave kernel), plus the
// HBM time of writing and re-reading the split partials (4 TB/s).  256-column
// tiles (`wide`) for dW, and for dX when its epilogue is plain (no addend, and
// either the fp32 result or its bf16 copy: the four-wave kernel's registers hold
// no more).
struct Plan {
    int bn;
    int splits;
};

Plan plan_gemm(int np, const int64_t* R, const int64_t* Cc, int64_t Kr, bool allow_split, bool wide) {
    Plan best{192, 1};
    double best_us = 1e300;
    const int bns[3] = {192, 128, 256};
    const double step_us[3] = {0.80, 0.57, 0.84};
    double out = 0.0;  // output elements of all products
    for (int q = 0; q < np; ++q) out += static_cast<double>(R[q]) * static_cast<double>(Cc[q]);
    for (int b = 0; b < 3; ++b) {
        const int bn = bns[b];
        if (bn == 256 && !wide) continue;
        int64_t tiles = 0;
        for (int q = 0; q < np; ++q) tiles += cdiv64(R[q], BM) * cdiv64(Cc[q], bn);
        const int64_t iters = (Kr + BK - 1) / BK;
        for (int s = 1; s <= (allow_split ? 32 : 1); ++s) {
            if (s > 1 && iters / s < 8) break;
            const int64_t wgs = tiles * s;
            const double rounds = static_cast<double>((wgs + kCUs - 1) / kCUs);
            double us = rounds * step_us[b] * static_cast<double>((iters + s - 1) / s);
            if (s > 1) us += static_cast<double>(s) * out * 8.0 / 4e12 * 1e6;
            if (us < best_us * 0.999) {
                best_us = us;
                best = Plan{bn, s};
            }
        }
    }
    return best;
}
Plan plan_gemm(int64_t R, int64_t Cc, int64_t Kr, bool allow_split, bool wide) {
    return plan_gemm(1, &R, &Cc, Kr, allow_split, wide);
}

// 256-column tiles run on the four-wave kernel with kStages4 stages.
constexpr int kStages4 = 5;

template <bool TR, int BN>
void launch_tile(const GemmLaunch& gl, int splits, hipStream_t s) {
    if constexpr (BN == 256) {
        hipLaunchKernelGGL((k_gemm4<TR, kStages4>), dim3(static_cast<unsigned>(gl.tiles * splits)), dim3(256), 0, s,
                           gl);
    } else {
        hipLaunchKernelGGL((k_gemm<TR, BN>), dim3(static_cast<unsigned>(gl.tiles * splits)), dim3(512), 0, s, gl);
    }
}

// One launch over the np products g[0..np) (same reduction split) with the
// plan's tile width; false if the grid is too large.
template <bool TR>
bool launch_plan(const GemmArgs* g, int np, const Plan& pl, hipStream_t s) {
    GemmLaunch gl{};
    int64_t t[2] = {0, 0};
    for (int q = 0; q < np; ++q) {
        gl.p[q] = g[q];
        gl.cb[q] = static_cast<int>(cdiv64(g[q].Cc, pl.bn));
        t[q] = cdiv64(g[q].R, BM) * gl.cb[q];
    }
    if (np == 1) {
        gl.p[1] = g[0];
        gl.cb[1] = gl.cb[0];
    }
    if ((t[0] + t[1]) * pl.splits > kMaxWgs) return false;
    gl.tiles0 = static_cast<int>(t[0]);
    gl.tiles = static_cast<int>(t[0] + t[1]);
    if (pl.bn == 128) launch_tile<TR, 128>(gl, pl.splits, s);
    else if (pl.bn == 256) launch_tile<TR, 256>(gl, pl.splits, s);
    else launch_tile<TR, 192>(gl, pl.splits, s);
    return true;
}

// Split partials of the products of one plan (else none): product q's partials
// follow those of the products before it.
size_t split_workspace(const Plan& pl, int np, const int64_t* R, const int64_t* Cc) {
    if (pl.splits == 1) return 0;
    size_t total = 0;
    for (int q = 0; q < np; ++q) total += static_cast<size_t>(pl.splits) * R[q] * Cc[q] * sizeof(float);
    return total;
}
int64_t split_range(int64_t Kr, int splits) {
    const int64_t per = (Kr + splits - 1) / splits;
    return (per + BK - 1) / BK * BK;
}
// Second stage over the products g[0..np) (their C is the partials); fin[q] is
// product q's final epilogue.
void launch_reduce(const GemmArgs* g, const ReduceArgs* fin, int np, int splits, hipStream_t s) {
    ReduceLaunch rl{};
    unsigned nb[2] = {0, 0};
    for (int q = 0; q < np; ++q) {
        rl.p[q] = fin[q];
        rl.p[q].R = g[q].R;
        rl.p[q].Cc = g[q].Cc;
        rl.p[q].part = g[q].C;
        nb[q] = static_cast<unsigned>(cdiv64(g[q].R * g[q].Cc, 1024));
    }
    if (np == 1) rl.p[1] = rl.p[0];
    rl.blocks0 = nb[0];
    rl.splits = splits;
    hipLaunchKernelGGL(k_splitk_reduce, dim3(nb[0] + nb[1]), dim3(256), 0, s, rl);
}

// dW_q = X_q^T dZ_q for np products with the same reduction length M.
size_t dw_workspace(int np, const DwProduct* d, int64_t M) {
    int64_t R[2], Cc[2];
    for (int q = 0; q < np; ++q) {
        R[q] = d[q].K;
        Cc[q] = d[q].N;
    }
    return split_workspace(plan_gemm(np, R, Cc, M, true, true), np, R, Cc);
}

hipError_t launch_dw(int np, const DwProduct* d, int64_t M, void* ws, hipStream_t s, const char* timer = nullptr) {
    int64_t R[2], Cc[2];
    for (int q = 0; q < np; ++q) {
        R[q] = d[q].K;
        Cc[q] = d[q].N;
    }
    const Plan pl = plan_gemm(np, R, Cc, M, true, true);
    const bool direct = pl.splits == 1;
    GemmArgs g[2];
    ReduceArgs fin[2];
    float* part = static_cast<float*>(ws);
    for (int q = 0; q < np; ++q) {
        g[q] = GemmArgs{d[q].K, d[q].N, M, d[q].X, d[q].ldx, d[q].dZ, d[q].lddz, direct ? d[q].dW : part,
                        split_range(M, pl.splits), direct ? 1 : 0, d[q].accum ? 1 : 0, nullptr, nullptr, 0,
                        d[q].N, 0};
        fin[q] = ReduceArgs{0, 0, nullptr, d[q].dW, d[q].accum ? 1 : 0, nullptr, nullptr, 0, d[q].N, 0};
        if (!direct) part += static_cast<int64_t>(pl.splits) * d[q].K * d[q].N;
    }
    {
        SSMK_TIMED(timer ? timer : "gemm_dw", s);
        if (!launch_plan<true>(g, np, pl, s)) return hipErrorInvalidConfiguration;
    }
    if (!direct) {
        SSMK_TIMED("splitk_reduce", s);
        launch_reduce(g, fin, np, pl.splits, s);
    }
    return hipGetLastError();
}

}  // namespace

size_t gemm_dw_workspace(int64_t M, int64_t K, int64_t N) {
    const DwProduct d{K, N, nullptr, 0, nullptr, 0, nullptr, false};
    return dw_workspace(1, &d, M);
}

size_t gemm_dw2_workspace(int64_t M, const DwProduct& a, const DwProduct& b) {
    const DwProduct d[2] = {a, b};
    return dw_workspace(2, d, M);
}

size_t gemm_dx_workspace(int64_t M, int64_t K, int64_t N) {
    // either epilogue (the plan with 256-column tiles applies to plain ones)
    const size_t a = split_workspace(plan_gemm(M, K, N, true, false), 1, &M, &K);
    const size_t b = split_workspace(plan_gemm(M, K, N, true, true), 1, &M, &K);
    return a > b ? a : b;
}

hipError_t launch_gemm_dw(int64_t M, int64_t K, int64_t N, const uint16_t* X, int64_t ldx,
                          const uint16_t* dZ, int64_t lddz, float* dW, bool accum, void* ws,
                          hipStream_t s, const char* timer) {
    const DwProduct d{K, N, X, ldx, dZ, lddz, dW, accum};
    return launch_dw(1, &d, M, ws, s, timer);
}

hipError_t launch_gemm_dw2(int64_t M, const DwProduct& a, const DwProduct& b, void* ws, hipStream_t s) {
    const DwProduct d[2] = {a, b};
    return launch_dw(2, d, M, ws, s);
}

hipError_t launch_gemm_dx(int64_t M, int64_t K, int64_t N, const uint16_t* dZ, int64_t lddz,
                          const uint16_t* W, int64_t ldw, float* dX, bool accum, const float* add,
                          uint16_t* out16, int64_t ld16, void* ws, hipStream_t s, int64_t ldx, int64_t ldadd,
                          const char* timer) {
    if (ldx <= 0) ldx = K;
    if (ldadd <= 0) ldadd = K;
    // outputs with few tiles (narrow projections) split the reduction as dW does
    const Plan pl = plan_gemm(M, K, N, true, add == nullptr && (out16 == nullptr || dX == nullptr));
    const bool direct = pl.splits == 1;
    const GemmArgs g{M, K, N, dZ, lddz, W, ldw, direct ? dX : static_cast<float*>(ws), split_range(N, pl.splits),
                     direct ? 1 : 0, accum ? 1 : 0, add, out16, ld16, ldx, ldadd};
    {
        SSMK_TIMED(timer ? timer : "gemm_dx", s);
        if (!launch_plan<false>(&g, 1, pl, s)) return hipErrorInvalidConfiguration;
    }
    if (!direct) {
        SSMK_TIMED("splitk_reduce", s);
        const ReduceArgs fin{0, 0, nullptr, dX, accum ? 1 : 0, add, out16, ld16, ldx, ldadd};
        launch_reduce(&g, &fin, 1, pl.splits, s);
    }
    return hipGetLastError();
}

}  // namespace ssmk
