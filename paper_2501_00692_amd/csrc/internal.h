// internal.h -- launch interface between the C ABI (abi.cpp) and the HIP kernels.
// Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ssmk {

// Opt-in per-kernel timing (timing.cpp): while enabled, a TimedScope records a
// hipEvent on the launch stream before and after the kernel launched inside it.
bool timing_enabled();
class TimedScope {
  public:
    TimedScope(const char* name, hipStream_t s);
    ~TimedScope();
    TimedScope(const TimedScope&) = delete;
    TimedScope& operator=(const TimedScope&) = delete;

  private:
    bool on_;
    hipStream_t s_;
    size_t idx_ = 0;
};
#define SSMK_CAT2(a, b) a##b
#define SSMK_CAT(a, b) SSMK_CAT2(a, b)
#define SSMK_TIMED(name, s) ::ssmk::TimedScope SSMK_CAT(ssmk_timed_, __LINE__)(name, s)

// Waves per workgroup of the fused gradient kernel; each wave works on one
// 16-channel tile at a time.
constexpr int kGradWaves = 4;

// One scan problem: the selective diagonal layer of shape [b][T][D] x N states,
// split into nc = ceil(T / L) carry chunks of L steps.
struct ScanProblem {
    int64_t nb, T, D, N, L, nc;
    bool bf16;       // inputs are bf16 (else fp32)
    bool softplus;   // delta holds Delta_pre
    bool gate;       // SiLU output gate with z
    bool trunc;      // truncated estimator with window tbar (< T)
    bool ascalar;    // one decay rate per channel: A_log, dA_log are [D]
    bool bdelta;     // input term Delta * B * x
    int64_t tbar;
    int nsplit;      // channel splits of the fused kernel (dB/dC partials when > 1)
    int tps;         // 16-channel tiles per split (a multiple of kGradWaves unless one split)
    int nslice;      // slices of the dA_log reduction
    // inputs
    const void* x;
    const void* delta;
    const float* A_log;
    const void* B;
    const void* C;
    const float* h0;
    const void* z;
    const void* dy;
    // outputs
    void* y;
    float* h_last;
    float* dx;
    float* ddelta;
    float* dA_log;
    float* dB;
    float* dC;
    float* dz;
    float* dh0;
    // optional bf16 (round to nearest even) copies for the projection GEMMs:
    // ddelta -> dd16[row * ld_dd16 + d], dz -> dz16[row * ld_dz16 + d],
    // dB -> bc16[row * ld_bc16 + n], dC -> bc16[row * ld_bc16 + N + n], row = b*T + t
    uint16_t* dd16;
    int64_t ld_dd16;
    uint16_t* dz16;
    int64_t ld_dz16;
    uint16_t* bc16;
    int64_t ld_bc16;
    uint16_t* dx16;  // dx -> dx16[row * ld_dx16 + d] (with the copies; required with only16)
    int64_t ld_dx16;
    bool only16;    // with the copies: write no fp32 dx, ddelta and dz (only the bf16 copies)
    // workspace regions
    float* hbuf;    // [b][nc][N][D]
    float* hseg;    // [b][nc][L/seg][Dp][16]: state at each segment start from a zero chunk carry-in
    float* cseg;    // [b][nc][L/seg][Dp]: sum of Delta from the chunk start to each segment start
    int64_t Dp;     // channels rounded up to a multiple of 64
    int seg;        // segment length of the fused gradient kernel
    float* mbuf;    // [b][nc][N][D]
    double* sdel;   // [b][nc][D]
    double* psum;   // [b][nc+1][D]
    float* pB;      // [nsplit][b][T][N]
    float* pC;      // [nsplit][b][T][N]
    float* dAtmp;   // [nslice][N][D]
    float* sink;    // 1 KB that padding lanes store into (gradient only)
};

// Workspace layout shared by the size query and the launch.
struct ScanWorkspace {
    size_t off_hbuf, off_mbuf, off_hseg, off_cseg, off_sdel, off_psum, off_pB, off_pC, off_dAtmp, off_sink,
        total;
};

int64_t default_chunk();
// Segment length of the fused gradient kernel for chunk length L.
inline int grad_segment(int64_t) { return 8; }
inline int64_t padded_channels(int64_t D) { return (D + 63) / 64 * 64; }
bool chunk_supported(int64_t L);
void choose_split(int64_t nb, int64_t D, int64_t nc, int* nsplit, int* tiles_per_split);
int choose_nslice(int64_t nb, int64_t nc);
ScanWorkspace scan_workspace(int64_t nb, int64_t T, int64_t D, int64_t N, int64_t L, bool grad,
                             bool trunc);
void bind_workspace(ScanProblem& p, void* ws, const ScanWorkspace& w);

hipError_t launch_forward(const ScanProblem& p, hipStream_t s);
// The optional debug output da [b][T][D][N] of the gradient (da_debug.hip).
hipError_t launch_da_debug(const ScanProblem& p, float* da, hipStream_t s);

// Scratch of ssm_adjoint_grad_noalloc (noalloc.hip): a file-scope device array of
// kNoallocScratchBytes per GPU; noalloc_scratch returns the current device's
// address of it (looked up once per device with that device current).
constexpr size_t kNoallocScratchBytes = size_t(64) << 20;
hipError_t noalloc_scratch(void** ptr);
hipError_t launch_grad(const ScanProblem& p, hipStream_t s);

// The unstructured SSM of Table 1 (unstructured.hip): 16 states shared by P
// channels, per-step matrices A [b][T][16][16], B [b][T][16][P], C [b][T][P][16],
// fp32; chunks of L steps (16..256).
struct UnstructuredProblem {
    int64_t nb, T, P, L;
    bool trunc;
    int64_t tbar;
    const float *A, *B, *C, *x, *h0, *dy;
    float *dA, *dB, *dC, *dx, *dh0;
};
size_t unstructured_workspace(int64_t nb, int64_t T, int64_t L, bool trunc);
hipError_t launch_unstructured_grad(const UnstructuredProblem& u, void* ws, hipStream_t s);

// The layer's reassociated input-projection gradient (layer.hip): dW_in[:, D:2D] =
// G[:, D:2D] and the bf16 hi/lo split of G[:, 2D:2D+nx] into hi, lo [dm][nx].
hipError_t launch_layer_split(const float* G, int64_t ldg, int64_t dm, int64_t D, int64_t nx, float* dW_in,
                              int64_t ldw, uint16_t* hi, uint16_t* lo, hipStream_t s);

// Kernels of the K-layer residual stack (stack.hip).
hipError_t launch_rms_fwd(const float* y, uint16_t* u, float* rinv, int64_t M, int64_t D, hipStream_t s);
// g (+)= (du - u mean(du u)) / rms; accum = false overwrites g; g16 (the bf16 copy)
// may be NULL.
hipError_t launch_rms_bwd(const float* y, const float* rinv, const float* du, float* g, uint16_t* g16, int64_t M,
                          int64_t D, hipStream_t s, bool accum = true);
hipError_t launch_residual(const float* yin, const uint16_t* ytil, float* yout, int64_t n, hipStream_t s);
hipError_t launch_to_bf16(const float* x, uint16_t* y, int64_t n, hipStream_t s);
hipError_t launch_transpose16(const uint16_t* in, uint16_t* out, int64_t R, int64_t C, hipStream_t s);

// The language head's row step (head.hip): per row of fp32 logits [rows][V] (ldo)
// and int32 target, the cross-entropy loss and the bf16 logit gradient
// softmax - onehot [rows][V] (ldg).  V, ldo and ldg must be multiples of 4.
hipError_t launch_head_xent(const float* logits, int64_t ldo, const int32_t* targets, float* loss, uint16_t* G,
                            int64_t ldg, int64_t rows, int64_t V, hipStream_t s);

// The gradient by the explicit pair formulation (pairs.hip): workspace layout and
// launch; W is the window (tbar, or T for the full gradient).
struct PairsWorkspace {
    size_t off_hbuf, off_sdel, off_dl, off_g, off_mu, off_pB, off_pC, off_dAtmp, total;
};
PairsWorkspace pairs_workspace(int64_t nb, int64_t T, int64_t D, int64_t N, int64_t L);
hipError_t launch_grad_pairs(ScanProblem& p, void* ws, const PairsWorkspace& w, int64_t W, hipStream_t s);

// bf16 MFMA GEMMs (gemm.hip).
// dW[K][N] (+)= X^T dZ with X [M][K] (ldx), dZ [M][N] (lddz); `timer` names the
// launch in the per-kernel timing (default "gemm_dw").
size_t gemm_dw_workspace(int64_t M, int64_t K, int64_t N);
hipError_t launch_gemm_dw(int64_t M, int64_t K, int64_t N, const uint16_t* X, int64_t ldx,
                          const uint16_t* dZ, int64_t lddz, float* dW, bool accum, void* ws,
                          hipStream_t s, const char* timer = nullptr);
// Two weight gradients dW_q[K_q][N_q] (+)= X_q^T dZ_q over the same M rows in one
// launch (and one second-stage launch when the reduction is split): the tiles of
// both fill the GPU together.  ws holds gemm_dw2_workspace bytes.
struct DwProduct {
    int64_t K, N;
    const uint16_t* X;
    int64_t ldx;
    const uint16_t* dZ;
    int64_t lddz;
    float* dW;
    bool accum;
};
size_t gemm_dw2_workspace(int64_t M, const DwProduct& a, const DwProduct& b);
hipError_t launch_gemm_dw2(int64_t M, const DwProduct& a, const DwProduct& b, void* ws, hipStream_t s);
// dX[M][K] (+)= dZ W^T with dZ [M][N] (lddz), W [K][N] (ldw); optional fp32 addend
// add[M][K] (ld = K) and optional bf16 copy of the result into out16 (ld16); dX may
// be NULL when out16 is given (only the copy is written).  Narrow outputs split the
// reduction: ws holds gemm_dx_workspace(M, K, N) bytes (none otherwise).
size_t gemm_dx_workspace(int64_t M, int64_t K, int64_t N);
// ldx and ldadd are the row strides of dX and of the addend (0: K); `timer` names
// the launch in the per-kernel timing (default "gemm_dx").
hipError_t launch_gemm_dx(int64_t M, int64_t K, int64_t N, const uint16_t* dZ, int64_t lddz,
                          const uint16_t* W, int64_t ldw, float* dX, bool accum, const float* add,
                          uint16_t* out16, int64_t ld16, void* ws, hipStream_t s, int64_t ldx = 0,
                          int64_t ldadd = 0, const char* timer = nullptr);

}  // namespace ssmk
