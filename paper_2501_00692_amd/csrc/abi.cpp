// abi.cpp -- the extern "C" entry points declared in include/ssm_adjoint.h:
// argument validation (before anything is enqueued), workspace layout and
// dispatch to the HIP kernels.
#include "ssm_adjoint.h"

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <string>

#include "internal.h"

namespace {

thread_local std::string g_last_error;

ssm_status fail(ssm_status st, const char* fmt, ...) {
    char msg[512];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(msg, sizeof msg, fmt, ap);
    va_end(ap);
    g_last_error = msg;
    return st;
}

ssm_status hip_fail(hipError_t e, const char* where) {
    return fail(SSM_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned256(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 255u) == 0; }

constexpr int64_t kMaxGridYZ = 65535;
constexpr int64_t kMaxGridX = (int64_t(1) << 31) - 1;

// Shape checks shared by forward and gradient.  Fills L (chunk) and nc.
ssm_status check_desc(const ssm_desc* d, int64_t* L, int64_t* nc) {
    if (!d) return fail(SSM_ERR_NULL, "desc is NULL");
    if (d->batch < 1 || d->seqlen < 1 || d->channels < 1 || d->dstate < 1)
        return fail(SSM_ERR_SHAPE, "batch, seqlen, channels and dstate must be >= 1 (got %lld, %lld, %lld, %lld)",
                    (long long)d->batch, (long long)d->seqlen, (long long)d->channels,
                    (long long)d->dstate);
    if (d->dstate > 16) return fail(SSM_ERR_UNSUPPORTED, "dstate %lld > 16", (long long)d->dstate);
    if (d->in_dtype != SSM_F32 && d->in_dtype != SSM_BF16)
        return fail(SSM_ERR_DTYPE, "unknown in_dtype %d", (int)d->in_dtype);
    if (d->flags & ~(SSM_DELTA_SOFTPLUS | SSM_GATE_SILU | SSM_A_SCALAR | SSM_B_DELTA))
        return fail(SSM_ERR_SHAPE, "unknown flag bits 0x%x", (unsigned)d->flags);
    const int64_t l = d->chunk == 0 ? ssmk::default_chunk() : d->chunk;
    if (!ssmk::chunk_supported(l))
        return fail(SSM_ERR_UNSUPPORTED, "chunk %lld not in {16, 32, 64, 128, 256}", (long long)d->chunk);
    const int64_t n = (d->seqlen + l - 1) / l;
    if (n > kMaxGridYZ || d->batch > kMaxGridYZ / 2)
        return fail(SSM_ERR_UNSUPPORTED, "seqlen/chunk (%lld) or batch (%lld) exceeds the launch grid",
                    (long long)n, (long long)d->batch);
    // Index arithmetic is 64-bit, except the byte offsets within one chunk of
    // rows (L * D elements, below 2^31 bytes for D <= 2^20).
    if (d->batch * d->seqlen > (int64_t(1) << 40) || d->channels > (int64_t(1) << 20))
        return fail(SSM_ERR_SHAPE, "problem too large");
    *L = l;
    *nc = n;
    return SSM_OK;
}

ssm_status check_mode(const ssm_desc* d, int32_t mode, int64_t tbar, bool* trunc) {
    if (mode != SSM_FULL && mode != SSM_TRUNCATED)
        return fail(SSM_ERR_SHAPE, "unknown mode %d", (int)mode);
    *trunc = false;
    if (mode == SSM_TRUNCATED) {
        if (tbar < 1) return fail(SSM_ERR_SHAPE, "truncated mode needs tbar >= 1 (got %lld)", (long long)tbar);
        *trunc = tbar < d->seqlen;  // tbar >= T is the full gradient
    }
    return SSM_OK;
}

#define REQUIRE_PTR(p, name)                                                         \
    do {                                                                             \
        if (!(p)) return fail(SSM_ERR_NULL, "%s is NULL", name);                     \
        if (!aligned16(p)) return fail(SSM_ERR_ALIGN, "%s is not 16-byte aligned", name); \
    } while (0)
#define OPTIONAL_PTR(p, name)                                                        \
    do {                                                                             \
        if ((p) && !aligned16(p)) return fail(SSM_ERR_ALIGN, "%s is not 16-byte aligned", name); \
    } while (0)

ssm_status check_workspace(void* ws, size_t have, size_t need) {
    if (need == 0) return SSM_OK;
    if (!ws) return fail(SSM_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
    if (!aligned256(ws)) return fail(SSM_ERR_ALIGN, "workspace is not 256-byte aligned");
    if (have < need) return fail(SSM_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", have, need);
    return SSM_OK;
}

ssmk::ScanProblem make_problem(const ssm_desc* d, int64_t L, int64_t nc) {
    ssmk::ScanProblem p{};
    p.nb = d->batch;
    p.T = d->seqlen;
    p.D = d->channels;
    p.N = d->dstate;
    p.L = L;
    p.nc = nc;
    p.bf16 = d->in_dtype == SSM_BF16;
    p.softplus = (d->flags & SSM_DELTA_SOFTPLUS) != 0;
    p.gate = (d->flags & SSM_GATE_SILU) != 0;
    p.ascalar = (d->flags & SSM_A_SCALAR) != 0;
    p.bdelta = (d->flags & SSM_B_DELTA) != 0;
    return p;
}

// Workspace of the whole-layer call: the scan workspace, then the bf16 operands
// of the projection products, fp32 scan outputs that the caller did not supply,
// the reassociated input-projection gradient's G and its bf16 hi/lo parts
// (d_model < D only), and the GEMM workspace.
struct LayerWs {
    size_t scan_off, z_off, f32_off, g_off, hl_off, gemm_off, total;
    size_t scan_total;
};

size_t up256(size_t v) { return (v + 255) & ~size_t(255); }

// The input projection's gradient is reassociated when d_model < D:
// dW_in[:, :D] = u^T (dx + dZx W_x^T) = u^T dx + (u^T dZx) W_x^T, which replaces the
// M x (D+2N) x D product that forms dx_total by M x d_model x (D+2N) more columns
// of the weight-gradient launch and a d_model x (D+2N) x D product.
bool layer_reassoc(int64_t d_model, int64_t D) { return d_model < D; }

LayerWs layer_ws(const ssm_desc* d, int64_t L, bool trunc, int64_t d_model) {
    LayerWs w{};
    const int64_t M = d->batch * d->seqlen, D = d->channels, N = d->dstate;
    const int64_t nx = D + 2 * N, nz = 3 * D + 2 * N;
    const bool re = layer_reassoc(d_model, D);
    ssmk::ScanWorkspace sw = ssmk::scan_workspace(d->batch, d->seqlen, D, N, L, true, trunc);
    w.scan_total = sw.total;
    size_t off = 0;
    w.scan_off = off;
    off = up256(off + sw.total);
    // bf16 [M][3D+2N]: reassociated, Z = [dx | dz | dDelta_pre | dB | dC]; otherwise
    // dZx = [dDelta_pre | dB | dC] ([M][D+2N]) followed by [dx_total | dz] ([M][2D])
    w.z_off = off;
    off = up256(off + size_t(M) * nz * 2);
    w.f32_off = off;  // fp32 dx, ddelta, dz [M][D] and dB, dC [M][N]
    off = up256(off + size_t(M) * (3 * D + 2 * N) * 4);
    w.g_off = off;  // fp32 G [d_model][3D+2N]
    if (re) off = up256(off + size_t(d_model) * nz * 4);
    w.hl_off = off;  // bf16 hi, lo [d_model][D+2N]
    if (re) off = up256(off + size_t(d_model) * nx * 2 * 2);
    w.gemm_off = off;
    // the layer's GEMM launches run one after the other and share the region
    const ssmk::DwProduct dwx{D, nx, nullptr, 0, nullptr, 0, nullptr, false};
    const ssmk::DwProduct dwin{d_model, re ? nz : 2 * D, nullptr, 0, nullptr, 0, nullptr, false};
    size_t g = ssmk::gemm_dw2_workspace(M, dwx, dwin);
    for (size_t gi : {ssmk::gemm_dx_workspace(M, D, nx), ssmk::gemm_dx_workspace(M, d_model, 2 * D),
                      re ? ssmk::gemm_dx_workspace(d_model, D, nx) : size_t(0)})
        g = gi > g ? gi : g;
    off = up256(off + g);
    w.total = off;
    return w;
}

}  // namespace

extern "C" {

const char* ssm_last_error(void) { return g_last_error.c_str(); }

ssm_status ssm_adjoint_forward_workspace_size(const ssm_desc* desc, size_t* bytes) {
    int64_t L, nc;
    ssm_status st = check_desc(desc, &L, &nc);
    if (st) return st;
    if (!bytes) return fail(SSM_ERR_NULL, "bytes is NULL");
    *bytes = ssmk::scan_workspace(desc->batch, desc->seqlen, desc->channels, desc->dstate, L,
                                  false, false)
                 .total;
    return SSM_OK;
}

ssm_status ssm_adjoint_grad_workspace_size(const ssm_desc* desc, int32_t mode, int64_t tbar,
                                           size_t* bytes) {
    int64_t L, nc;
    ssm_status st = check_desc(desc, &L, &nc);
    if (st) return st;
    bool trunc;
    st = check_mode(desc, mode, tbar, &trunc);
    if (st) return st;
    if (!bytes) return fail(SSM_ERR_NULL, "bytes is NULL");
    *bytes = ssmk::scan_workspace(desc->batch, desc->seqlen, desc->channels, desc->dstate, L,
                                  true, trunc)
                 .total;
    return SSM_OK;
}

ssm_status ssm_adjoint_forward(const ssm_desc* desc, const void* x, const void* delta,
                               const float* A_log, const void* B, const void* C, const float* h0,
                               const void* z, void* y, float* h_last, void* workspace,
                               size_t workspace_bytes, void* stream) {
    int64_t L, nc;
    ssm_status st = check_desc(desc, &L, &nc);
    if (st) return st;
    REQUIRE_PTR(x, "x");
    REQUIRE_PTR(delta, "delta");
    REQUIRE_PTR(A_log, "A_log");
    REQUIRE_PTR(B, "B");
    REQUIRE_PTR(C, "C");
    REQUIRE_PTR(y, "y");
    OPTIONAL_PTR(h0, "h0");
    OPTIONAL_PTR(h_last, "h_last");
    const bool gate = (desc->flags & SSM_GATE_SILU) != 0;
    if (gate) REQUIRE_PTR(z, "z");
    else if (z) return fail(SSM_ERR_SHAPE, "z given without SSM_GATE_SILU");
    ssmk::ScanWorkspace w = ssmk::scan_workspace(desc->batch, desc->seqlen, desc->channels,
                                                 desc->dstate, L, false, false);
    st = check_workspace(workspace, workspace_bytes, w.total);
    if (st) return st;
    ssmk::ScanProblem p = make_problem(desc, L, nc);
    p.x = x;
    p.delta = delta;
    p.A_log = A_log;
    p.B = B;
    p.C = C;
    p.h0 = h0;
    p.z = z;
    p.y = y;
    p.h_last = h_last;
    ssmk::bind_workspace(p, workspace, w);
    p.mbuf = nullptr;
    hipError_t e = ssmk::launch_forward(p, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "ssm_adjoint_forward launch");
    return SSM_OK;
}

static ssm_status grad_validate(const ssm_desc* desc, int32_t mode, int64_t tbar, const void* x,
                                const void* delta, const float* A_log, const void* B,
                                const void* C, const float* h0, const void* z, const void* dy,
                                float* dx, float* ddelta, float* dA_log, float* dB, float* dC,
                                float* dz, float* dh0, int64_t* L, int64_t* nc, bool* trunc) {
    ssm_status st = check_desc(desc, L, nc);
    if (st) return st;
    st = check_mode(desc, mode, tbar, trunc);
    if (st) return st;
    REQUIRE_PTR(x, "x");
    REQUIRE_PTR(delta, "delta");
    REQUIRE_PTR(A_log, "A_log");
    REQUIRE_PTR(B, "B");
    REQUIRE_PTR(C, "C");
    REQUIRE_PTR(dy, "dy");
    REQUIRE_PTR(dx, "dx");
    REQUIRE_PTR(ddelta, "ddelta");
    REQUIRE_PTR(dA_log, "dA_log");
    REQUIRE_PTR(dB, "dB");
    REQUIRE_PTR(dC, "dC");
    OPTIONAL_PTR(h0, "h0");
    const bool gate = (desc->flags & SSM_GATE_SILU) != 0;
    if (gate) {
        REQUIRE_PTR(z, "z");
        REQUIRE_PTR(dz, "dz");
    } else if (z || dz) {
        return fail(SSM_ERR_SHAPE, "z/dz given without SSM_GATE_SILU");
    }
    OPTIONAL_PTR(dh0, "dh0");
    if (dh0 && mode == SSM_TRUNCATED && *trunc)
        return fail(SSM_ERR_UNSUPPORTED, "dh0 is defined for the full gradient only");
    return SSM_OK;
}

static void grad_bind(ssmk::ScanProblem& p, const void* x, const void* delta, const float* A_log,
                      const void* B, const void* C, const float* h0, const void* z, const void* dy,
                      float* dx, float* ddelta, float* dA_log, float* dB, float* dC, float* dz,
                      float* dh0) {
    p.x = x;
    p.delta = delta;
    p.A_log = A_log;
    p.B = B;
    p.C = C;
    p.h0 = h0;
    p.z = z;
    p.dy = dy;
    p.dx = dx;
    p.ddelta = ddelta;
    p.dA_log = dA_log;
    p.dB = dB;
    p.dC = dC;
    p.dz = dz;
    p.dh0 = dh0;
}

// Launch of a validated gradient call on a workspace laid out as `w`.
static ssm_status grad_launch(const ssm_desc* desc, int64_t L, int64_t nc, bool trunc, int64_t tbar,
                              const void* x, const void* delta, const float* A_log, const void* B,
                              const void* C, const float* h0, const void* z, const void* dy, float* dx,
                              float* ddelta, float* dA_log, float* dB, float* dC, float* dz, float* dh0,
                              float* da_debug, void* workspace, const ssmk::ScanWorkspace& w, void* stream,
                              const char* where) {
    ssmk::ScanProblem p = make_problem(desc, L, nc);
    p.trunc = trunc;
    p.tbar = trunc ? tbar : 0;
    ssmk::choose_split(p.nb, p.D, nc, &p.nsplit, &p.tps);
    p.nslice = ssmk::choose_nslice(p.nb, nc);
    grad_bind(p, x, delta, A_log, B, C, h0, z, dy, dx, ddelta, dA_log, dB, dC, dz, dh0);
    ssmk::bind_workspace(p, workspace, w);
    hipError_t e = ssmk::launch_grad(p, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, where);
    if (da_debug) {
        e = ssmk::launch_da_debug(p, da_debug, static_cast<hipStream_t>(stream));
        if (e != hipSuccess) return hip_fail(e, "da_debug launch");
    }
    return SSM_OK;
}

ssm_status ssm_adjoint_grad(const ssm_desc* desc, int32_t mode, int64_t tbar, const void* x,
                            const void* delta, const float* A_log, const void* B, const void* C,
                            const float* h0, const void* z, const void* dy, float* dx,
                            float* ddelta, float* dA_log, float* dB, float* dC, float* dz,
                            float* dh0, float* da_debug, void* workspace, size_t workspace_bytes, void* stream) {
    int64_t L, nc;
    bool trunc;
    ssm_status st = grad_validate(desc, mode, tbar, x, delta, A_log, B, C, h0, z, dy, dx, ddelta,
                                  dA_log, dB, dC, dz, dh0, &L, &nc, &trunc);
    if (st) return st;
    OPTIONAL_PTR(da_debug, "da_debug");
    ssmk::ScanWorkspace w = ssmk::scan_workspace(desc->batch, desc->seqlen, desc->channels,
                                                 desc->dstate, L, true, trunc);
    st = check_workspace(workspace, workspace_bytes, w.total);
    if (st) return st;
    return grad_launch(desc, L, nc, trunc, tbar, x, delta, A_log, B, C, h0, z, dy, dx, ddelta, dA_log, dB,
                       dC, dz, dh0, da_debug, workspace, w, stream, "ssm_adjoint_grad launch");
}

ssm_status ssm_adjoint_grad_noalloc(const ssm_desc* desc, int32_t mode, int64_t tbar, const void* x,
                                    const void* delta, const float* A_log, const void* B, const void* C,
                                    const float* h0, const void* z, const void* dy, float* dx,
                                    float* ddelta, float* dA_log, float* dB, float* dC, float* dz,
                                    float* dh0, float* da_debug, void* stream) {
    int64_t L, nc;
    bool trunc;
    ssm_status st = grad_validate(desc, mode, tbar, x, delta, A_log, B, C, h0, z, dy, dx, ddelta,
                                  dA_log, dB, dC, dz, dh0, &L, &nc, &trunc);
    if (st) return st;
    OPTIONAL_PTR(da_debug, "da_debug");
    ssmk::ScanWorkspace w = ssmk::scan_workspace(desc->batch, desc->seqlen, desc->channels,
                                                 desc->dstate, L, true, trunc);
    if (w.total > ssmk::kNoallocScratchBytes)
        return fail(SSM_ERR_WORKSPACE,
                    "this gradient needs %zu bytes of scratch; the no-allocation entry point has %zu "
                    "(use ssm_adjoint_grad with a workspace)",
                    w.total, ssmk::kNoallocScratchBytes);
    void* scratch = nullptr;
    hipError_t e = ssmk::noalloc_scratch(&scratch);
    if (e != hipSuccess) return hip_fail(e, "ssm_adjoint_grad_noalloc scratch");
    return grad_launch(desc, L, nc, trunc, tbar, x, delta, A_log, B, C, h0, z, dy, dx, ddelta, dA_log, dB,
                       dC, dz, dh0, da_debug, scratch, w, stream, "ssm_adjoint_grad_noalloc launch");
}

// Limits of the pair formulation: its channel blocks form a grid dimension, and
// its workspace holds the summed adjoint states of every (step, channel).
static ssm_status check_pairs(const ssm_desc* d) {
    if ((d->channels + 63) / 64 > kMaxGridYZ)
        return fail(SSM_ERR_UNSUPPORTED, "channels (%lld) exceed the pair kernel's launch grid",
                    (long long)d->channels);
    if (d->batch * d->seqlen * d->channels > (int64_t(1) << 40))
        return fail(SSM_ERR_UNSUPPORTED, "batch * seqlen * channels too large for the pair workspace");
    return SSM_OK;
}

ssm_status ssm_adjoint_grad_pairs_workspace_size(const ssm_desc* desc, int32_t mode, int64_t tbar,
                                                 size_t* bytes) {
    int64_t L, nc;
    ssm_status st = check_desc(desc, &L, &nc);
    if (st) return st;
    st = check_pairs(desc);
    if (st) return st;
    bool trunc;
    st = check_mode(desc, mode, tbar, &trunc);
    if (st) return st;
    if (!bytes) return fail(SSM_ERR_NULL, "bytes is NULL");
    *bytes = ssmk::pairs_workspace(desc->batch, desc->seqlen, desc->channels, desc->dstate, L).total;
    return SSM_OK;
}

ssm_status ssm_adjoint_grad_pairs(const ssm_desc* desc, int32_t mode, int64_t tbar, const void* x,
                                  const void* delta, const float* A_log, const void* B, const void* C,
                                  const float* h0, const void* z, const void* dy, float* dx,
                                  float* ddelta, float* dA_log, float* dB, float* dC, float* dz,
                                  float* dh0, float* da_debug, void* workspace, size_t workspace_bytes,
                                  void* stream) {
    int64_t L, nc;
    bool trunc;
    ssm_status st = grad_validate(desc, mode, tbar, x, delta, A_log, B, C, h0, z, dy, dx, ddelta,
                                  dA_log, dB, dC, dz, dh0, &L, &nc, &trunc);
    if (st) return st;
    OPTIONAL_PTR(da_debug, "da_debug");
    st = check_pairs(desc);
    if (st) return st;
    ssmk::PairsWorkspace w = ssmk::pairs_workspace(desc->batch, desc->seqlen, desc->channels,
                                                   desc->dstate, L);
    st = check_workspace(workspace, workspace_bytes, w.total);
    if (st) return st;
    ssmk::ScanProblem p = make_problem(desc, L, nc);
    p.trunc = trunc;
    p.tbar = trunc ? tbar : 0;
    grad_bind(p, x, delta, A_log, B, C, h0, z, dy, dx, ddelta, dA_log, dB, dC, dz, dh0);
    hipError_t e = ssmk::launch_grad_pairs(p, workspace, w, trunc ? tbar : desc->seqlen,
                                           static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "ssm_adjoint_grad_pairs launch");
    if (da_debug) {
        e = ssmk::launch_da_debug(p, da_debug, static_cast<hipStream_t>(stream));
        if (e != hipSuccess) return hip_fail(e, "da_debug launch");
    }
    return SSM_OK;
}

// The unstructured SSM of Table 1: 16 states, P channels (desc->channels), fp32.
static ssm_status check_unstructured(const ssm_desc* d, int32_t mode, int64_t tbar, int64_t* L, bool* trunc) {
    if (!d) return fail(SSM_ERR_NULL, "desc is NULL");
    if (d->batch < 1 || d->seqlen < 1 || d->channels < 1 || d->dstate < 1)
        return fail(SSM_ERR_SHAPE, "batch, seqlen, channels and dstate must be >= 1");
    if (d->dstate != 16) return fail(SSM_ERR_UNSUPPORTED, "the unstructured SSM takes dstate = 16 (got %lld)",
                                     (long long)d->dstate);
    if (d->channels % 16 || d->channels > 4096)
        return fail(SSM_ERR_UNSUPPORTED, "channels must be a multiple of 16, at most 4096 (got %lld)",
                    (long long)d->channels);
    if (d->in_dtype != SSM_F32) return fail(SSM_ERR_UNSUPPORTED, "the unstructured SSM takes fp32 tensors");
    if (d->flags) return fail(SSM_ERR_UNSUPPORTED, "no flags apply to the unstructured SSM");
    const int64_t l = d->chunk == 0 ? 64 : d->chunk;
    if (!ssmk::chunk_supported(l))
        return fail(SSM_ERR_UNSUPPORTED, "chunk %lld not in {16, 32, 64, 128, 256}", (long long)d->chunk);
    if (d->batch > kMaxGridYZ) return fail(SSM_ERR_UNSUPPORTED, "batch exceeds the launch grid");
    if (d->batch * d->seqlen > (int64_t(1) << 36)) return fail(SSM_ERR_SHAPE, "problem too large");
    if (mode != SSM_FULL && mode != SSM_TRUNCATED) return fail(SSM_ERR_SHAPE, "unknown mode %d", (int)mode);
    *trunc = false;
    if (mode == SSM_TRUNCATED) {
        if (tbar < 1) return fail(SSM_ERR_SHAPE, "truncated mode needs tbar >= 1 (got %lld)", (long long)tbar);
        *trunc = tbar < d->seqlen;
        // one workgroup per block of tbar steps
        if (*trunc && (d->seqlen + tbar - 1) / tbar > kMaxGridX)
            return fail(SSM_ERR_UNSUPPORTED, "seqlen / tbar exceeds the launch grid");
    }
    *L = l;
    return SSM_OK;
}

ssm_status ssm_unstructured_grad_workspace_size(const ssm_desc* desc, int32_t mode, int64_t tbar, size_t* bytes) {
    int64_t L;
    bool trunc;
    ssm_status st = check_unstructured(desc, mode, tbar, &L, &trunc);
    if (st) return st;
    if (!bytes) return fail(SSM_ERR_NULL, "bytes is NULL");
    *bytes = ssmk::unstructured_workspace(desc->batch, desc->seqlen, L, trunc);
    return SSM_OK;
}

ssm_status ssm_unstructured_grad(const ssm_desc* desc, int32_t mode, int64_t tbar, const float* A, const float* B,
                                 const float* C, const float* x, const float* h0, const float* dy, float* dA,
                                 float* dB, float* dC, float* dx, float* dh0, void* workspace,
                                 size_t workspace_bytes, void* stream) {
    int64_t L;
    bool trunc;
    ssm_status st = check_unstructured(desc, mode, tbar, &L, &trunc);
    if (st) return st;
    REQUIRE_PTR(A, "A");
    REQUIRE_PTR(B, "B");
    REQUIRE_PTR(C, "C");
    REQUIRE_PTR(x, "x");
    REQUIRE_PTR(dy, "dy");
    REQUIRE_PTR(dA, "dA");
    REQUIRE_PTR(dB, "dB");
    REQUIRE_PTR(dC, "dC");
    REQUIRE_PTR(dx, "dx");
    OPTIONAL_PTR(h0, "h0");
    OPTIONAL_PTR(dh0, "dh0");
    if (dh0 && trunc) return fail(SSM_ERR_UNSUPPORTED, "dh0 is defined for the full gradient only");
    st = check_workspace(workspace, workspace_bytes, ssmk::unstructured_workspace(desc->batch, desc->seqlen, L, trunc));
    if (st) return st;
    ssmk::UnstructuredProblem u{};
    u.nb = desc->batch;
    u.T = desc->seqlen;
    u.P = desc->channels;
    u.L = L;
    u.trunc = trunc;
    u.tbar = trunc ? tbar : 0;
    u.A = A;
    u.B = B;
    u.C = C;
    u.x = x;
    u.h0 = h0;
    u.dy = dy;
    u.dA = dA;
    u.dB = dB;
    u.dC = dC;
    u.dx = dx;
    u.dh0 = dh0;
    hipError_t e = ssmk::launch_unstructured_grad(u, workspace, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "ssm_unstructured_grad launch");
    return SSM_OK;
}

ssm_status ssm_proj_grad_workspace_size(int64_t M, int64_t K, int64_t Nout, uint32_t flags,
                                        size_t* bytes) {
    if (!bytes) return fail(SSM_ERR_NULL, "bytes is NULL");
    if (M < 1 || K < 1 || Nout < 1) return fail(SSM_ERR_SHAPE, "M, K, Nout must be >= 1");
    if (flags & ~(SSM_ACCUM_DW | SSM_ACCUM_DX)) return fail(SSM_ERR_SHAPE, "unknown flag bits");
    const size_t dw = ssmk::gemm_dw_workspace(M, K, Nout), dx = ssmk::gemm_dx_workspace(M, K, Nout);
    *bytes = dw > dx ? dw : dx;  // the two products run one after the other
    return SSM_OK;
}

constexpr int64_t kMaxLd = int64_t(1) << 21;

static ssm_status check_gemm_shape(int64_t M, int64_t K, int64_t Nout, int64_t ldx, int64_t lddz,
                                   int64_t ldw, bool need_w) {
    if (M < 1 || K < 1 || Nout < 1)
        return fail(SSM_ERR_SHAPE, "M, K, Nout must be >= 1 (got %lld, %lld, %lld)", (long long)M,
                    (long long)K, (long long)Nout);
    if (K % 8 || Nout % 8)
        return fail(SSM_ERR_UNSUPPORTED, "K and Nout must be multiples of 8 (got %lld, %lld)",
                    (long long)K, (long long)Nout);
    if (ldx < K || lddz < Nout || (need_w && ldw < Nout))
        return fail(SSM_ERR_SHAPE, "leading dimension smaller than the row length");
    if (ldx % 8 || lddz % 8 || (need_w && ldw % 8))
        return fail(SSM_ERR_ALIGN, "leading dimensions must be multiples of 8 elements");
    if (M > (int64_t(1) << 31) || K > (int64_t(1) << 20) || Nout > (int64_t(1) << 20))
        return fail(SSM_ERR_SHAPE, "GEMM too large");
    // the kernels address an operand tile (at most 256 rows) with 32-bit byte offsets
    if (ldx > kMaxLd || lddz > kMaxLd || (need_w && ldw > kMaxLd))
        return fail(SSM_ERR_SHAPE, "leading dimensions must be at most %lld elements", (long long)kMaxLd);
    return SSM_OK;
}

ssm_status ssm_proj_grad(int64_t M, int64_t K, int64_t Nout, const void* X, int64_t ldx,
                         const void* dZ, int64_t lddz, const void* W, int64_t ldw, float* dW,
                         float* dX, uint32_t flags, void* workspace, size_t workspace_bytes,
                         void* stream) {
    if (flags & ~(SSM_ACCUM_DW | SSM_ACCUM_DX)) return fail(SSM_ERR_SHAPE, "unknown flag bits");
    ssm_status st = check_gemm_shape(M, K, Nout, dW ? ldx : K, lddz, ldw, dX != nullptr);
    if (st) return st;
    REQUIRE_PTR(dZ, "dZ");
    if (dW) REQUIRE_PTR(X, "X");
    if (dX) REQUIRE_PTR(W, "W");
    OPTIONAL_PTR(dW, "dW");
    OPTIONAL_PTR(dX, "dX");
    {
        const size_t dw = dW ? ssmk::gemm_dw_workspace(M, K, Nout) : 0;
        const size_t dx = dX ? ssmk::gemm_dx_workspace(M, K, Nout) : 0;
        st = check_workspace(workspace, workspace_bytes, dw > dx ? dw : dx);
        if (st) return st;
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (dW) {
        hipError_t e = ssmk::launch_gemm_dw(M, K, Nout, static_cast<const uint16_t*>(X), ldx,
                                            static_cast<const uint16_t*>(dZ), lddz, dW,
                                            (flags & SSM_ACCUM_DW) != 0, workspace, s);
        if (e != hipSuccess) return hip_fail(e, "ssm_proj_grad dW launch");
    }
    if (dX) {
        hipError_t e = ssmk::launch_gemm_dx(M, K, Nout, static_cast<const uint16_t*>(dZ), lddz,
                                            static_cast<const uint16_t*>(W), ldw, dX,
                                            (flags & SSM_ACCUM_DX) != 0, nullptr, nullptr, 0, workspace, s);
        if (e != hipSuccess) return hip_fail(e, "ssm_proj_grad dX launch");
    }
    return SSM_OK;
}

ssm_status ssm_layer_grad_workspace_size(const ssm_desc* desc, int32_t mode, int64_t tbar,
                                         int64_t d_model, size_t* bytes) {
    int64_t L, nc;
    ssm_status st = check_desc(desc, &L, &nc);
    if (st) return st;
    bool trunc;
    st = check_mode(desc, mode, tbar, &trunc);
    if (st) return st;
    if (!bytes) return fail(SSM_ERR_NULL, "bytes is NULL");
    if (d_model < 1) return fail(SSM_ERR_SHAPE, "d_model must be >= 1");
    *bytes = layer_ws(desc, L, trunc, d_model).total;
    return SSM_OK;
}

ssm_status ssm_layer_grad(const ssm_desc* desc, int32_t mode, int64_t tbar, int64_t d_model,
                          const void* u, const void* x, const void* z, const void* delta_pre,
                          const void* B, const void* C, const void* W_x, const void* W_in,
                          const float* A_log, const void* dy, float* dW_in, float* dW_x,
                          float* dA_log, float* du, float* dx, float* ddelta, float* dB,
                          float* dC, float* dz, float* dx_total, void* workspace,
                          size_t workspace_bytes, void* stream) {
    int64_t L, nc;
    ssm_status st = check_desc(desc, &L, &nc);
    if (st) return st;
    if (desc->in_dtype != SSM_BF16)
        return fail(SSM_ERR_UNSUPPORTED, "the layer gradient takes bf16 activations");
    bool trunc;
    st = check_mode(desc, mode, tbar, &trunc);
    if (st) return st;
    if (d_model < 1) return fail(SSM_ERR_SHAPE, "d_model must be >= 1");
    const int64_t M = desc->batch * desc->seqlen, D = desc->channels, N = desc->dstate;
    st = check_gemm_shape(M, D, D + 2 * N, D, D + 2 * N, D + 2 * N, true);
    if (st) return st;
    st = check_gemm_shape(M, d_model, 2 * D, d_model, 2 * D, 2 * D, du != nullptr);
    if (st) return st;
    if (layer_reassoc(d_model, D)) {  // the shapes of G = u^T Z
        st = check_gemm_shape(M, d_model, 3 * D + 2 * N, d_model, 3 * D + 2 * N, 0, false);
        if (st) return st;
    }
    REQUIRE_PTR(u, "u");
    REQUIRE_PTR(W_x, "W_x");
    REQUIRE_PTR(dW_in, "dW_in");
    REQUIRE_PTR(dW_x, "dW_x");
    if (du) {
        REQUIRE_PTR(W_in, "W_in");
        OPTIONAL_PTR(du, "du");
    }
    OPTIONAL_PTR(dx_total, "dx_total");
    LayerWs w = layer_ws(desc, L, trunc, d_model);
    st = check_workspace(workspace, workspace_bytes, w.total);
    if (st) return st;
    char* ws = static_cast<char*>(workspace);
    float* f32 = reinterpret_cast<float*>(ws + w.f32_off);
    float* dx_ = dx ? dx : f32;
    float* dd_ = ddelta ? ddelta : f32 + M * D;
    float* dz_ = dz ? dz : f32 + 2 * M * D;
    float* dB_ = dB ? dB : f32 + 3 * M * D;
    float* dC_ = dC ? dC : f32 + 3 * M * D + M * N;

    ssm_desc sd = *desc;
    sd.flags = SSM_DELTA_SOFTPLUS | SSM_GATE_SILU | (desc->flags & (SSM_A_SCALAR | SSM_B_DELTA));
    bool trunc2;
    st = grad_validate(&sd, mode, tbar, x, delta_pre, A_log, B, C, nullptr, z, dy, dx_, dd_, dA_log,
                       dB_, dC_, dz_, nullptr, &L, &nc, &trunc2);
    if (st) return st;

    hipStream_t s = static_cast<hipStream_t>(stream);
    const bool re = layer_reassoc(d_model, D);
    const int64_t nx = D + 2 * N, nz = 3 * D + 2 * N;
    ssmk::ScanWorkspace sw = ssmk::scan_workspace(sd.batch, sd.seqlen, D, N, L, true, trunc);
    ssmk::ScanProblem p = make_problem(&sd, L, nc);
    p.trunc = trunc;
    p.tbar = trunc ? tbar : 0;
    ssmk::choose_split(p.nb, p.D, nc, &p.nsplit, &p.tps);
    p.nslice = ssmk::choose_nslice(p.nb, nc);
    grad_bind(p, x, delta_pre, A_log, B, C, nullptr, z, dy, dx_, dd_, dA_log, dB_, dC_, dz_, nullptr);
    ssmk::bind_workspace(p, ws + w.scan_off, sw);
    uint16_t* zb = reinterpret_cast<uint16_t*>(ws + w.z_off);
    void* gws = ws + w.gemm_off;
    const bool need_dxt = dx_total || du;  // dx_total = dx + dZx W_x^T is formed
    hipError_t e;
    if (re) {
        // the scan kernels write Z = [dx | dz | dDelta_pre | dB | dC] in bf16; fp32 dx,
        // dDelta_pre and dz only when the caller asks for one of them or for dx_total
        p.dx16 = zb;
        p.ld_dx16 = nz;
        p.dz16 = zb + D;
        p.ld_dz16 = nz;
        p.dd16 = zb + 2 * D;
        p.ld_dd16 = nz;
        p.bc16 = zb + 3 * D;
        p.ld_bc16 = nz;
        p.only16 = !dx && !ddelta && !dz && !need_dxt;
        e = ssmk::launch_grad(p, s);
        if (e != hipSuccess) return hip_fail(e, "ssm_layer_grad scan launch");
        // dW_x = x^T dZx and G = u^T Z in one launch
        float* G = reinterpret_cast<float*>(ws + w.g_off);
        const ssmk::DwProduct px{D, nx, static_cast<const uint16_t*>(x), D, zb + 2 * D, nz, dW_x, false};
        const ssmk::DwProduct pg{d_model, nz, static_cast<const uint16_t*>(u), d_model, zb, nz, G, false};
        e = ssmk::launch_gemm_dw2(M, px, pg, gws, s);
        if (e != hipSuccess) return hip_fail(e, "ssm_layer_grad dW_x / G launch");
        // dW_in[:, D:] = G[:, D:2D]; hi + lo = G[:, 2D:] = u^T dZx
        uint16_t* hi = reinterpret_cast<uint16_t*>(ws + w.hl_off);
        uint16_t* lo = hi + d_model * nx;
        e = ssmk::launch_layer_split(G, nz, d_model, D, nx, dW_in, 2 * D, hi, lo, s);
        if (e != hipSuccess) return hip_fail(e, "ssm_layer_grad split launch");
        // dW_in[:, :D] = G[:, :D] + lo W_x^T, then += hi W_x^T
        const uint16_t* Wx = static_cast<const uint16_t*>(W_x);
        e = ssmk::launch_gemm_dx(d_model, D, nx, lo, nx, Wx, nx, dW_in, false, G, nullptr, 0, gws, s, 2 * D, nz,
                                 "gemm_dwin_fix");
        if (e != hipSuccess) return hip_fail(e, "ssm_layer_grad dW_in launch");
        e = ssmk::launch_gemm_dx(d_model, D, nx, hi, nx, Wx, nx, dW_in, true, nullptr, nullptr, 0, gws, s, 2 * D,
                                 0, "gemm_dwin_fix");
        if (e != hipSuccess) return hip_fail(e, "ssm_layer_grad dW_in launch");
        if (need_dxt) {
            // dx_total = dx + dZx W_x^T; its bf16 copy replaces dx in Z, so that
            // Z[:, :2D] = [dx_total | dz] for du
            e = ssmk::launch_gemm_dx(M, D, nx, zb + 2 * D, nz, Wx, nx, dx_total, false, dx_, zb, nz, gws, s);
            if (e != hipSuccess) return hip_fail(e, "ssm_layer_grad dx_total launch");
        }
        if (du) {
            e = ssmk::launch_gemm_dx(M, d_model, 2 * D, zb, nz, static_cast<const uint16_t*>(W_in), 2 * D, du, false,
                                     nullptr, nullptr, 0, gws, s);
            if (e != hipSuccess) return hip_fail(e, "ssm_layer_grad du launch");
        }
        return SSM_OK;
    }
    // d_model >= D: dx_total first, then both weight gradients in one launch
    // (the scan kernels write dZx and the dz half of [dx_total | dz] in bf16, and dx
    // in fp32 as the dx_total product's addend)
    uint16_t* dzx = zb;
    uint16_t* dxz = zb + M * nx;
    p.dd16 = dzx;
    p.ld_dd16 = nx;
    p.bc16 = dzx + D;
    p.ld_bc16 = nx;
    p.dz16 = dxz + D;
    p.ld_dz16 = 2 * D;
    e = ssmk::launch_grad(p, s);
    if (e != hipSuccess) return hip_fail(e, "ssm_layer_grad scan launch");
    // dx_total = dx + dZx W_x^T, also packed into [dx_total | dz]
    // (the fp32 dx_total only when the caller asks for it)
    e = ssmk::launch_gemm_dx(M, D, nx, dzx, nx, static_cast<const uint16_t*>(W_x), nx, dx_total, false, dx_, dxz,
                             2 * D, gws, s);
    if (e != hipSuccess) return hip_fail(e, "ssm_layer_grad dx_total launch");
    // dW_x = x^T dZx and dW_in = u^T [dx_total | dz], in one launch
    const ssmk::DwProduct px{D, nx, static_cast<const uint16_t*>(x), D, dzx, nx, dW_x, false};
    const ssmk::DwProduct pin{d_model, 2 * D, static_cast<const uint16_t*>(u), d_model, dxz, 2 * D, dW_in, false};
    e = ssmk::launch_gemm_dw2(M, px, pin, gws, s);
    if (e != hipSuccess) return hip_fail(e, "ssm_layer_grad dW_x / dW_in launch");
    if (du) {
        e = ssmk::launch_gemm_dx(M, d_model, 2 * D, dxz, 2 * D, static_cast<const uint16_t*>(W_in),
                                 2 * D, du, false, nullptr, nullptr, 0, gws, s);
        if (e != hipSuccess) return hip_fail(e, "ssm_layer_grad du launch");
    }
    return SSM_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// K-layer residual stack (Sec. 3.2, Prop. 3, Alg. 1).
// ---------------------------------------------------------------------------
namespace {

constexpr int64_t kMaxStackLayers = 4096;

// Workspace of the stack: per layer the activations the forward stores (u, x,
// z, Delta_pre as bf16 [M][D], B, C as bf16 [M][N], 1/rms [M], the layer's
// fp32 input y for layers after the first, the transposed projections), then
// the shared buffers (the layer output, the running upstream and its bf16 copy,
// du, y_K when the caller does not take it, the scan and layer workspaces).
struct StackWs {
    size_t per_layer, off_u, off_x, off_z, off_dp, off_B, off_C, off_r, off_y, off_wi, off_wx;
    size_t off_ytil, off_g, off_g16, off_du, off_yk, off_fws, off_lws, off_gws, total;
    size_t fws_bytes, lws_bytes;
};

StackWs stack_ws(const ssm_desc* d, int64_t K, int64_t L, bool trunc) {
    StackWs w{};
    const int64_t M = d->batch * d->seqlen, D = d->channels, N = d->dstate;
    const size_t a16 = size_t(M) * D * 2, n16 = size_t(M) * N * 2, f32 = size_t(M) * D * 4;
    size_t o = 0;
    w.off_u = o; o = up256(o + a16);
    w.off_x = o; o = up256(o + a16);
    w.off_z = o; o = up256(o + a16);
    w.off_dp = o; o = up256(o + a16);
    w.off_B = o; o = up256(o + n16);
    w.off_C = o; o = up256(o + n16);
    w.off_r = o; o = up256(o + size_t(M) * 4);
    w.off_y = o; o = up256(o + f32);
    w.off_wi = o; o = up256(o + size_t(2 * D) * D * 2);
    w.off_wx = o; o = up256(o + size_t(D + 2 * N) * D * 2);
    w.per_layer = o;
    o = w.per_layer * size_t(K);
    w.off_ytil = o; o = up256(o + a16);
    w.off_g = o; o = up256(o + f32);
    w.off_g16 = o; o = up256(o + a16);
    w.off_du = o; o = up256(o + f32);
    w.off_yk = o; o = up256(o + f32);
    ssm_desc ld = *d;
    ld.flags = SSM_DELTA_SOFTPLUS | SSM_GATE_SILU;
    w.fws_bytes = ssmk::scan_workspace(ld.batch, ld.seqlen, D, N, L, false, false).total;
    w.off_fws = o; o = up256(o + w.fws_bytes);
    w.lws_bytes = layer_ws(&ld, L, trunc, D).total;
    w.off_lws = o; o = up256(o + w.lws_bytes);
    // split partials of the forward projections (the narrow B and C products)
    const size_t gx = ssmk::gemm_dx_workspace(M, D, D), gn = ssmk::gemm_dx_workspace(M, N, D);
    w.off_gws = o; o = up256(o + (gx > gn ? gx : gn));
    w.total = o;
    return w;
}

ssm_status check_stack(const ssm_desc* desc, int64_t K, int32_t grad, int32_t mode, int64_t tbar, int64_t* L,
                       bool* trunc) {
    int64_t nc;
    ssm_status st = check_desc(desc, L, &nc);
    if (st) return st;
    if (desc->in_dtype != SSM_BF16) return fail(SSM_ERR_UNSUPPORTED, "the stack takes bf16 activations");
    if (desc->flags != 0) return fail(SSM_ERR_UNSUPPORTED, "the stack's layers take no variant flags");
    if (K < 1 || K > kMaxStackLayers) return fail(SSM_ERR_SHAPE, "K must be in [1, %lld]", (long long)kMaxStackLayers);
    if (grad != SSM_STACK_ADJOINT && grad != SSM_STACK_EXACT && grad != SSM_STACK_FORWARD)
        return fail(SSM_ERR_SHAPE, "unknown gradient kind %d", grad);
    st = check_mode(desc, mode, tbar, trunc);
    if (st) return st;
    const int64_t M = desc->batch * desc->seqlen, D = desc->channels, N = desc->dstate;
    if (M >= (int64_t(1) << 31)) return fail(SSM_ERR_UNSUPPORTED, "batch * seqlen too large for the stack");
    if ((D + 31) / 32 > kMaxGridYZ) return fail(SSM_ERR_UNSUPPORTED, "channels too large for the stack");
    st = check_gemm_shape(M, D, D + 2 * N, D, D + 2 * N, D + 2 * N, true);
    if (st) return st;
    return check_gemm_shape(M, D, 2 * D, D, 2 * D, 2 * D, true);
}

}  // namespace

extern "C" {

ssm_status ssm_stack_grad_workspace_size(const ssm_desc* desc, int64_t K, int32_t grad, int32_t mode,
                                         int64_t tbar, size_t* bytes) {
    int64_t L;
    bool trunc;
    ssm_status st = check_stack(desc, K, grad, mode, tbar, &L, &trunc);
    if (st) return st;
    if (!bytes) return fail(SSM_ERR_NULL, "bytes is NULL");
    *bytes = stack_ws(desc, K, L, trunc).total;
    return SSM_OK;
}

ssm_status ssm_stack_grad(const ssm_desc* desc, int64_t K, int32_t grad, int32_t mode, int64_t tbar,
                          const float* y0, const void* const* W_in, const void* const* W_x,
                          const float* const* A_log, const float* gK, float* const* dW_in,
                          float* const* dW_x, float* const* dA_log, float* yK, void* workspace,
                          size_t workspace_bytes, void* stream) {
    int64_t L;
    bool trunc;
    ssm_status st = check_stack(desc, K, grad, mode, tbar, &L, &trunc);
    if (st) return st;
    const bool fwd_only = grad == SSM_STACK_FORWARD;
    REQUIRE_PTR(y0, "y0");
    if (fwd_only) {
        REQUIRE_PTR(yK, "yK");
    } else {
        REQUIRE_PTR(gK, "gK");
        OPTIONAL_PTR(yK, "yK");
    }
    if (!W_in || !W_x || !A_log || (!fwd_only && (!dW_in || !dW_x || !dA_log)))
        return fail(SSM_ERR_NULL, "a per-layer pointer array is NULL");
    for (int64_t k = 0; k < K; ++k) {
        REQUIRE_PTR(W_in[k], "W_in[k]");
        REQUIRE_PTR(W_x[k], "W_x[k]");
        REQUIRE_PTR(A_log[k], "A_log[k]");
        if (fwd_only) continue;
        REQUIRE_PTR(dW_in[k], "dW_in[k]");
        REQUIRE_PTR(dW_x[k], "dW_x[k]");
        REQUIRE_PTR(dA_log[k], "dA_log[k]");
    }
    const StackWs w = stack_ws(desc, K, L, trunc);
    st = check_workspace(workspace, workspace_bytes, w.total);
    if (st) return st;

    const int64_t M = desc->batch * desc->seqlen, D = desc->channels, N = desc->dstate;
    hipStream_t s = static_cast<hipStream_t>(stream);
    char* ws = static_cast<char*>(workspace);
    auto lay = [&](int64_t k, size_t off) { return ws + w.per_layer * size_t(k) + off; };
    auto u16 = [](char* p) { return reinterpret_cast<uint16_t*>(p); };
    auto f32 = [](char* p) { return reinterpret_cast<float*>(p); };
    uint16_t* ytil = u16(ws + w.off_ytil);
    float* g = f32(ws + w.off_g);
    uint16_t* g16 = u16(ws + w.off_g16);
    float* du = f32(ws + w.off_du);
    float* yout = yK ? yK : f32(ws + w.off_yk);
    ssm_desc ld = *desc;
    ld.flags = SSM_DELTA_SOFTPLUS | SSM_GATE_SILU;
    hipError_t e = hipSuccess;
#define STACK_HIP(call, what)                           \
    do {                                                \
        e = (call);                                     \
        if (e != hipSuccess) return hip_fail(e, what);  \
    } while (0)
#define STACK_SSM(call)            \
    do {                           \
        ssm_status r_ = (call);    \
        if (r_ != SSM_OK) return r_; \
    } while (0)

    // forward (Alg. 1): u = Norm(y), [x | z] = u W_in, [Delta_pre | B | C] = x W_x,
    // y += scan(...) * silu(z); every layer keeps its activations
    const float* ycur = y0;
    for (int64_t k = 0; k < K; ++k) {
        uint16_t* u = u16(lay(k, w.off_u));
        uint16_t* x = u16(lay(k, w.off_x));
        uint16_t* z = u16(lay(k, w.off_z));
        uint16_t* dp = u16(lay(k, w.off_dp));
        uint16_t* Bm = u16(lay(k, w.off_B));
        uint16_t* Cm = u16(lay(k, w.off_C));
        uint16_t* wi = u16(lay(k, w.off_wi));
        uint16_t* wx = u16(lay(k, w.off_wx));
        float* rinv = f32(lay(k, w.off_r));
        STACK_HIP(ssmk::launch_rms_fwd(ycur, u, rinv, M, D, s), "ssm_stack_grad norm");
        STACK_HIP(ssmk::launch_transpose16(static_cast<const uint16_t*>(W_in[k]), wi, D, 2 * D, s),
                  "ssm_stack_grad transpose");
        STACK_HIP(ssmk::launch_transpose16(static_cast<const uint16_t*>(W_x[k]), wx, D, D + 2 * N, s),
                  "ssm_stack_grad transpose");
        // out[M][c] = sum_j a[M][j] W^T[c][j]: the dX form of the projection GEMM
        void* gws = ws + w.off_gws;
        STACK_HIP(ssmk::launch_gemm_dx(M, D, D, u, D, wi, D, nullptr, false, nullptr, x, D, gws, s),
                  "ssm_stack_grad x");
        STACK_HIP(ssmk::launch_gemm_dx(M, D, D, u, D, wi + D * D, D, nullptr, false, nullptr, z, D, gws, s),
                  "ssm_stack_grad z");
        STACK_HIP(ssmk::launch_gemm_dx(M, D, D, x, D, wx, D, nullptr, false, nullptr, dp, D, gws, s),
                  "ssm_stack_grad Delta_pre");
        STACK_HIP(ssmk::launch_gemm_dx(M, N, D, x, D, wx + D * D, D, nullptr, false, nullptr, Bm, N, gws, s),
                  "ssm_stack_grad B");
        STACK_HIP(ssmk::launch_gemm_dx(M, N, D, x, D, wx + (D + N) * D, D, nullptr, false, nullptr, Cm, N, gws,
                                       s),
                  "ssm_stack_grad C");
        STACK_SSM(ssm_adjoint_forward(&ld, x, dp, A_log[k], Bm, Cm, nullptr, z, ytil, nullptr, ws + w.off_fws,
                                      w.fws_bytes, stream));
        float* ynext = k + 1 < K ? f32(lay(k + 1, w.off_y)) : yout;
        STACK_HIP(ssmk::launch_residual(ycur, ytil, ynext, M * D, s), "ssm_stack_grad residual");
        ycur = ynext;
    }

    if (fwd_only) return SSM_OK;
    // gradients: Prop. 3 (every layer under dL/dy_K) or backpropagation
    if (grad == SSM_STACK_EXACT)
        STACK_HIP(hipMemcpyAsync(g, gK, size_t(M) * D * 4, hipMemcpyDeviceToDevice, s), "ssm_stack_grad copy");
    STACK_HIP(ssmk::launch_to_bf16(gK, g16, M * D, s), "ssm_stack_grad upstream");
    for (int64_t k = K - 1; k >= 0; --k) {
        const bool back = grad == SSM_STACK_EXACT && k > 0;
        STACK_SSM(ssm_layer_grad(&ld, mode, tbar, D, lay(k, w.off_u), lay(k, w.off_x), lay(k, w.off_z),
                                 lay(k, w.off_dp), lay(k, w.off_B), lay(k, w.off_C), W_x[k], W_in[k], A_log[k], g16,
                                 dW_in[k], dW_x[k], dA_log[k], back ? du : nullptr, nullptr, nullptr, nullptr,
                                 nullptr, nullptr, nullptr, ws + w.off_lws, w.lws_bytes, stream));
        if (back)  // dL/dy_{k-1} = dL/dy_k + Norm'(y_{k-1})^T du_k
            STACK_HIP(ssmk::launch_rms_bwd(f32(lay(k, w.off_y)), f32(lay(k, w.off_r)), du, g, g16, M, D, s),
                      "ssm_stack_grad norm backward");
    }
#undef STACK_HIP
#undef STACK_SSM
    return SSM_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// The language head and its loss (Sec. 3.2, Alg. 1).
// ---------------------------------------------------------------------------
namespace {

constexpr size_t kHeadLogitBytes = size_t(4) << 30;  // fp32 logits of one row block

// Workspace of the head: per row block Norm(y) (bf16) and its transpose, 1/rms,
// Omega^T (bf16 [P][V]), the block's fp32 logits and bf16 logit gradients, dU
// (fp32), and the GEMM workspace shared by the block's three products.
struct HeadWs {
    int64_t rows;
    size_t off_u, off_ut, off_r, off_omt, off_logit, off_g, off_du, off_gws, total;
};

// Row blocks whose logits are computed by the weight-gradient GEMM form from
// Norm(y)^T: a multiple of 8 rows (the form's 16-byte operand pieces) and at most
// this many (the transpose's grid height).
constexpr int64_t kHeadMaxTransRows = int64_t(65535) * 32;
bool head_logits_dw(int64_t mb) { return mb % 8 == 0 && mb <= kHeadMaxTransRows; }

HeadWs head_ws(int64_t M, int64_t P, int64_t V, int64_t block_rows) {
    HeadWs w{};
    int64_t rows = block_rows ? block_rows : static_cast<int64_t>(kHeadLogitBytes / (size_t(V) * 4)) / 256 * 256;
    if (rows < 256) rows = 256;
    if (rows > M) rows = M;
    w.rows = rows;
    size_t o = 0;
    w.off_u = o; o = up256(o + size_t(rows) * P * 2);
    w.off_ut = o; o = up256(o + size_t(rows) * P * 2);
    w.off_r = o; o = up256(o + size_t(rows) * 4);
    w.off_omt = o; o = up256(o + size_t(P) * V * 2);
    w.off_logit = o; o = up256(o + size_t(rows) * V * 4);
    w.off_g = o; o = up256(o + size_t(rows) * V * 2);
    w.off_du = o; o = up256(o + size_t(rows) * P * 4);
    // a whole block and the last, shorter one (whose split may differ)
    size_t g = 0;
    for (int64_t mb : {rows, M % rows}) {
        if (mb == 0) continue;
        for (size_t gi : {ssmk::gemm_dx_workspace(mb, V, P), ssmk::gemm_dx_workspace(mb, P, V),
                          ssmk::gemm_dw_workspace(mb, V, P), ssmk::gemm_dw_workspace(P, mb, V)})
            g = gi > g ? gi : g;
    }
    w.off_gws = o; o = up256(o + g);
    w.total = o;
    return w;
}

ssm_status check_head(int64_t M, int64_t P, int64_t V, uint32_t flags, int64_t block_rows) {
    if (flags & ~SSM_HEAD_NORM) return fail(SSM_ERR_SHAPE, "unknown flag bits");
    if (M < 1 || P < 1 || V < 1) return fail(SSM_ERR_SHAPE, "M, P, V must be >= 1");
    if (M >= (int64_t(1) << 31)) return fail(SSM_ERR_SHAPE, "M must be below 2^31");
    if (block_rows < 0 || block_rows % 256 || block_rows >= (int64_t(1) << 31))
        return fail(SSM_ERR_SHAPE, "block_rows must be 0 or a positive multiple of 256 below 2^31");
    const int64_t rows = head_ws(M, P, V, block_rows).rows;
    ssm_status st = check_gemm_shape(rows, V, P, V, P, P, true);  // logits = u Omega^T
    if (st) return st;
    return check_gemm_shape(rows, P, V, P, V, V, true);            // dU = G Omega, dOmega = G^T u
}

}  // namespace

extern "C" {

ssm_status ssm_lm_head_grad_workspace_size(int64_t M, int64_t P, int64_t V, uint32_t flags, int64_t block_rows,
                                           size_t* bytes) {
    ssm_status st = check_head(M, P, V, flags, block_rows);
    if (st) return st;
    if (!bytes) return fail(SSM_ERR_NULL, "bytes is NULL");
    *bytes = head_ws(M, P, V, block_rows).total;
    return SSM_OK;
}

ssm_status ssm_lm_head_grad(int64_t M, int64_t P, int64_t V, uint32_t flags, int64_t block_rows, const float* y,
                            const void* omega, const int32_t* targets, float* loss, float* dy, float* domega,
                            void* workspace, size_t workspace_bytes, void* stream) {
    ssm_status st = check_head(M, P, V, flags, block_rows);
    if (st) return st;
    REQUIRE_PTR(y, "y");
    REQUIRE_PTR(omega, "omega");
    REQUIRE_PTR(targets, "targets");
    REQUIRE_PTR(loss, "loss");
    REQUIRE_PTR(dy, "dy");
    OPTIONAL_PTR(domega, "domega");
    const HeadWs w = head_ws(M, P, V, block_rows);
    st = check_workspace(workspace, workspace_bytes, w.total);
    if (st) return st;
    const bool norm = (flags & SSM_HEAD_NORM) != 0;
    hipStream_t s = static_cast<hipStream_t>(stream);
    char* ws = static_cast<char*>(workspace);
    uint16_t* u = reinterpret_cast<uint16_t*>(ws + w.off_u);
    uint16_t* ut = reinterpret_cast<uint16_t*>(ws + w.off_ut);
    float* rinv = reinterpret_cast<float*>(ws + w.off_r);
    uint16_t* omt = reinterpret_cast<uint16_t*>(ws + w.off_omt);
    float* logit = reinterpret_cast<float*>(ws + w.off_logit);
    uint16_t* G = reinterpret_cast<uint16_t*>(ws + w.off_g);
    float* du = reinterpret_cast<float*>(ws + w.off_du);
    void* gws = ws + w.off_gws;
    const uint16_t* om = static_cast<const uint16_t*>(omega);
    hipError_t e = ssmk::launch_transpose16(om, omt, V, P, s);
    if (e != hipSuccess) return hip_fail(e, "ssm_lm_head_grad transpose");
#define HEAD_HIP(call, what)                           \
    do {                                               \
        e = (call);                                    \
        if (e != hipSuccess) return hip_fail(e, what); \
    } while (0)
    for (int64_t m0 = 0; m0 < M; m0 += w.rows) {
        const int64_t mb = M - m0 < w.rows ? M - m0 : w.rows;
        const float* yb = y + m0 * P;
        float* dyb = dy + m0 * P;
        if (norm)
            HEAD_HIP(ssmk::launch_rms_fwd(yb, u, rinv, mb, P, s), "ssm_lm_head_grad norm");
        else
            HEAD_HIP(ssmk::launch_to_bf16(yb, u, mb * P, s), "ssm_lm_head_grad input");
        // logits [mb][V] = u Omega^T = (u^T)^T (Omega^T), the reduction over P.  The
        // weight-gradient form stages 32 whole rows of u^T and Omega^T per step, each
        // read as whole cache lines, where the dX form stages 64-byte pieces of 256
        // rows of u and Omega: 3.9 against 4.5 ms at 32,768 x 32,000 x 2,048, for a
        // transpose of u of about 0.1 ms.  Other block heights take the dX form.
        if (head_logits_dw(mb)) {
            HEAD_HIP(ssmk::launch_transpose16(u, ut, mb, P, s), "ssm_lm_head_grad transpose");
            HEAD_HIP(ssmk::launch_gemm_dw(P, mb, V, ut, mb, omt, V, logit, false, gws, s, "head_logits"),
                     "ssm_lm_head_grad logits");
        } else {
            HEAD_HIP(ssmk::launch_gemm_dx(mb, V, P, u, P, om, P, logit, false, nullptr, nullptr, 0, gws, s, 0, 0,
                                          "head_logits"),
                     "ssm_lm_head_grad logits");
        }
        HEAD_HIP(ssmk::launch_head_xent(logit, V, targets + m0, loss + m0, G, V, mb, V, s),
                 "ssm_lm_head_grad loss");
        // dU [mb][P] = G Omega = G (Omega^T)^T: the dX form with the reduction over V
        HEAD_HIP(ssmk::launch_gemm_dx(mb, P, V, G, V, omt, V, norm ? du : dyb, false, nullptr, nullptr, 0, gws, s,
                                      0, 0, "head_du"),
                 "ssm_lm_head_grad dU");
        if (norm) HEAD_HIP(ssmk::launch_rms_bwd(yb, rinv, du, dyb, nullptr, mb, P, s, false), "ssm_lm_head_grad dy");
        if (domega)  // dOmega [V][P] (+)= G^T u, the blocks added in order
            HEAD_HIP(ssmk::launch_gemm_dw(mb, V, P, G, V, u, P, domega, m0 > 0, gws, s), "ssm_lm_head_grad dOmega");
    }
#undef HEAD_HIP
    return SSM_OK;
}

}  // extern "C"
