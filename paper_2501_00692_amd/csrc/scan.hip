// scan.hip -- workspace layout of the scan kernels, the forward dispatch and
// the gradient dispatch to the per-(dtype, mode) translation units.
#include "scan_kernels.h"

namespace ssmk {
namespace {

template <typename TI>
hipError_t forward_dispatch(const ScanProblem& p, hipStream_t s) {
    const bool n16 = p.N == 16;
#define SSMK_FWD(SP, GT) \
    return n16 ? forward_impl<TI, SP, GT, true>(p, s) : forward_impl<TI, SP, GT, false>(p, s)
    if (p.softplus) {
        if (p.gate) SSMK_FWD(true, true);
        SSMK_FWD(true, false);
    }
    if (p.gate) SSMK_FWD(false, true);
    SSMK_FWD(false, false);
#undef SSMK_FWD
}

size_t align_up(size_t v) { return (v + 255) & ~static_cast<size_t>(255); }

}  // namespace

int64_t default_chunk() { return 128; }

bool chunk_supported(int64_t L) { return L == 16 || L == 32 || L == 64 || L == 128 || L == 256; }

void choose_split(int64_t nb, int64_t D, int64_t nc, int* nsplit, int* tiles_per_split) {
    // Workgroups of kGradWaves waves take tiles in groups of kGradWaves; aim at
    // one round of two workgroups per CU (256 CUs), every split with at least
    // one group.
    const int64_t target = 512;
    const int64_t ntile = (D + 15) / 16;
    const int64_t groups = (ntile + kGradWaves - 1) / kGradWaves;
    int64_t ns = (target + nb * nc - 1) / (nb * nc);
    if (ns < 1) ns = 1;
    if (ns > groups) ns = groups;
    const int64_t gps = (groups + ns - 1) / ns;
    *tiles_per_split = static_cast<int>(gps * kGradWaves);
    *nsplit = static_cast<int>((groups + gps - 1) / gps);
}

int choose_nslice(int64_t nb, int64_t nc) {
    int64_t nq = nb * nc;
    if (nq <= 256) return 1;  // one pass, in the same launch as the dB/dC sums
    int64_t s = nq / 16;
    if (s < 1) s = 1;
    if (s > 64) s = 64;
    return static_cast<int>(s);
}

ScanWorkspace scan_workspace(int64_t nb, int64_t T, int64_t D, int64_t N, int64_t L, bool grad,
                             bool trunc) {
    ScanWorkspace w{};
    const int64_t nc = (T + L - 1) / L;
    size_t off = 0;
    const size_t carry = static_cast<size_t>(nb * nc * N * D) * sizeof(float);
    w.off_hbuf = off;
    off = align_up(off + carry);
    w.off_mbuf = off;
    if (grad) off = align_up(off + carry);
    // segment-start states of every chunk (gradient only)
    const int64_t nseg = grad ? L / grad_segment(L) : 0;
    const int64_t Dp = padded_channels(D);
    w.off_hseg = off;
    off = align_up(off + static_cast<size_t>(nb * nc * nseg * Dp * 16) * sizeof(float));
    w.off_cseg = off;
    off = align_up(off + static_cast<size_t>(nb * nc * nseg * Dp) * sizeof(float));
    w.off_sdel = off;
    off = align_up(off + static_cast<size_t>(nb * nc * D) * sizeof(double));
    w.off_psum = off;
    if (grad && trunc) off = align_up(off + static_cast<size_t>(nb * (nc + 1) * D) * sizeof(double));
    w.off_pB = w.off_pC = w.off_dAtmp = off;
    if (grad) {
        int ns, tps;
        choose_split(nb, D, nc, &ns, &tps);
        if (ns > 1) {
            const size_t part = static_cast<size_t>(ns) * nb * T * N * sizeof(float);
            w.off_pB = off;
            off = align_up(off + part);
            w.off_pC = off;
            off = align_up(off + part);
        }
        w.off_dAtmp = off;
        off = align_up(off + static_cast<size_t>(choose_nslice(nb, nc)) * N * D * sizeof(float));
    }
    w.off_sink = off;
    if (grad) off = align_up(off + 1024);
    w.total = off;
    return w;
}

void bind_workspace(ScanProblem& p, void* ws, const ScanWorkspace& w) {
    char* b = static_cast<char*>(ws);
    p.hbuf = reinterpret_cast<float*>(b + w.off_hbuf);
    p.mbuf = w.off_mbuf != w.off_hseg ? reinterpret_cast<float*>(b + w.off_mbuf) : nullptr;
    p.hseg = w.off_hseg != w.off_cseg ? reinterpret_cast<float*>(b + w.off_hseg) : nullptr;
    p.cseg = w.off_cseg != w.off_sdel ? reinterpret_cast<float*>(b + w.off_cseg) : nullptr;
    p.Dp = padded_channels(p.D);
    p.seg = grad_segment(p.L);
    p.sdel = reinterpret_cast<double*>(b + w.off_sdel);
    p.psum = w.off_psum != w.off_pB ? reinterpret_cast<double*>(b + w.off_psum) : nullptr;
    p.pB = w.off_pB != w.off_pC ? reinterpret_cast<float*>(b + w.off_pB) : nullptr;
    p.pC = p.pB ? reinterpret_cast<float*>(b + w.off_pC) : nullptr;
    p.dAtmp = w.off_dAtmp != w.off_sink ? reinterpret_cast<float*>(b + w.off_dAtmp) : nullptr;
    p.sink = w.off_sink != w.total ? reinterpret_cast<float*>(b + w.off_sink) : nullptr;
}

hipError_t launch_forward(const ScanProblem& p, hipStream_t s) {
    return p.bf16 ? forward_dispatch<uint16_t>(p, s) : forward_dispatch<float>(p, s);
}

hipError_t launch_grad(const ScanProblem& p, hipStream_t s) {
    if (p.bf16) return p.trunc ? grad_bf16_trunc(p, s) : grad_bf16_full(p, s);
    return p.trunc ? grad_f32_trunc(p, s) : grad_f32_full(p, s);
}

}  // namespace ssmk
