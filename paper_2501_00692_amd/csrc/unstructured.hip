// unstructured.hip -- the adjoint gradient of the unstructured SSM of Table 1
// (gfx950): an N = 16 state shared by the P channels, with per-step matrices
//   h_t = A_t h_{t-1} + B_t x_t,   y_t = C_t h_t,
//   A_t [N][N], B_t [N][P], C_t [P][N] (fp32, row-major), L = sum <dy_t, y_t>.
// Outputs: dA_t = mu_t h_{t-1}^T, dB_t = mu_t x_t^T, dx_t = B_t^T mu_t,
// dC_t = dy_t h_t^T (never truncated), dh0 = A_0^T mu_0 (full mode), where mu is
// the state cotangent mu_t = C_t^T dy_t + A_{t+1}^T mu_{t+1} (Prop. 1, summed over
// the loss terms as in Prop. 2), or in truncated mode the windowed adjoint of
// Eq. "capped", mubar_i = sum_{t=i}^{i+tbar-1} (A_{i+1}^T ... A_t^T) C_t^T dy_t.
//
// The state is tiny (16 values per sequence), so the parallelism comes from
// time: the sequence is cut into chunks of L steps, one wave per chunk.
//   k_un_aggr  : per chunk, the transition product Phi_c = A_e ... A_s (16x16x16
//                products on fp32 MFMA), the local end state from zero, the
//                local adjoint aggregate sum_t (A_t ... A_s)^T v_t and the
//                readout cotangents v_t = C_t^T dy_t of every step;
//   k_un_carry : per sequence, the chunk carries H_{c+1} = Phi_c H_c + hloc_c
//                and M_{c-1} = Phi_c^T M_c + mloc_c, in order;
//   k_un_wpre, k_un_wsuf : truncated mode.  The windowed adjoint obeys
//                mubar_i = u_i + A_{i+1}^T mubar_{i+1} with u_i = v_i - w_i and
//                w_i = Phi(i, i+tbar)^T v_{i+tbar}, Phi(i, j) = A_j ... A_{i+1} (the
//                step that leaves the window is taken out as it leaves), so it is
//                the full gradient's recurrence with v replaced by u.  w_i splits
//                at the block boundary k (blocks of tbar steps, i < k <= i + tbar):
//                w_i = Phi(i, k)^T y_{i+tbar} with y_j = Phi(k, j)^T v_j; k_un_wpre
//                runs the prefix products Phi(k, j) of each block and writes y,
//                k_un_wsuf the suffix products Phi(i, k)^T and writes u = v - w
//                over v; both keep the 16 x 16 products in MFMA registers;
//   k_un_madj  : truncated mode, each chunk's adjoint aggregate of u (the full
//                mode forms it inside k_un_aggr from v);
//   k_un_grad  : per chunk, the states recomputed from the carry (kept in LDS),
//                then the reverse sweep (or the windowed adjoints) and the vjps.
//   k_un_proj  : per step, the two reductions over the P channels that the
//                sequential passes need: bx_t = B_t x_t and v_t = C_t^T dy_t
//                (fully parallel, ahead of the chunk passes, so that these walk
//                only A_t and two 16-vectors per step, loaded a step ahead).
// Lane layout of a wave: lane l = 16 q + i; i indexes a row of the 16 x 16
// matrices, q one of four quarters of the reduction (matrix columns 4q..4q+3,
// or a quarter of the P channels), summed across quarters with two xor
// shuffles.  Vectors of 16 are kept replicated in all four quarters.
#include "internal.h"

namespace ssmk {
namespace {

constexpr int UN = 16;  // state size

// Sum over the four quarters of the wave (lanes i, i+16, i+32, i+48).
__device__ __forceinline__ float qsum(float v) {
    v += __shfl_xor(v, 16);
    v += __shfl_xor(v, 32);
    return v;
}

struct UnArgs {
    int64_t nb, T, P, L, nc, tbar;
    int trunc;
    const float* A;   // [b][T][16][16]
    const float* B;   // [b][T][16][P]
    const float* C;   // [b][T][P][16]
    const float* x;   // [b][T][P]
    const float* h0;  // [b][16] or null
    const float* dy;  // [b][T][P]
    float* dA;
    float* dB;
    float* dC;
    float* dx;
    float* dh0;       // [b][16] or null (full mode)
    float* h_last;    // [b][16] or null
    // workspace
    float* phi;       // [b][nc][16][16]
    float* hc;        // [b][nc][16]: local end state, then the carry into the chunk
    float* mc;        // [b][nc][16]: local adjoint aggregate, then the carry from the right
    float* v;         // [b][T][16]: C_t^T dy_t
    float* y;         // [b][T][16]: y_j = Phi(k, j)^T v_j (truncated mode)
    float* bx;        // [b][T][16]: B_t x_t
};

// h[4q + r] from the lane that holds it (vectors of 16 are replicated in the
// four quarters; lane 4q + r of the first quarter has component 4q + r).
__device__ __forceinline__ float4 quarter_of(float h, int q) {
    return make_float4(__shfl(h, 4 * q), __shfl(h, 4 * q + 1), __shfl(h, 4 * q + 2), __shfl(h, 4 * q + 3));
}

// grid (ceil(T / 4), b), 64 threads: four steps per wave, one at a time.
// bx_t = B_t x_t: instruction j reads rows 4j..4j+3 of B_t (row 4j + g in lanes
// 16 g .. 16 g + 15, four channels per lane, 64 channels per pass), and each
// row's partial sums are added over its 16 lanes.  v_t = C_t^T dy_t: lane l reads
// C_t[p][4(l%4) .. +3] for p = l/4 + 16 k (64 lanes cover 16 rows of C_t per
// pass), weighted by dy_t[p], and the 16 lanes with the same l%4 are added.
// Reads of B_t and C_t are contiguous across the wave.
__global__ __launch_bounds__(64) void k_un_proj(const UnArgs a) {
    const int lane = threadIdx.x, g = lane >> 4, sub = lane & 15, cq = lane & 3;
    const int64_t bb = blockIdx.y, P = a.P;
    for (int w = 0; w < 4; ++w) {
        const int64_t t = static_cast<int64_t>(blockIdx.x) * 4 + w;
        if (t >= a.T) return;  // wave-uniform
        const int64_t row = bb * a.T + t;
        const float* Bt = a.B + row * UN * P;
        const float* xt = a.x + row * P;
        const float* Ct = a.C + row * P * UN;
        const float* dyt = a.dy + row * P;
        float sb[4] = {0.f, 0.f, 0.f, 0.f};
        for (int64_t p = 4 * sub; p < P; p += 64) {
            const float4 x4 = *reinterpret_cast<const float4*>(xt + p);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const float4 b4 = *reinterpret_cast<const float4*>(Bt + (4 * j + g) * P + p);
                sb[j] = fmaf(b4.x, x4.x, fmaf(b4.y, x4.y, fmaf(b4.z, x4.z, fmaf(b4.w, x4.w, sb[j]))));
            }
        }
        float sc[4] = {0.f, 0.f, 0.f, 0.f};
        for (int64_t pr = lane >> 2; pr < P; pr += 16) {
            const float4 c4 = *reinterpret_cast<const float4*>(Ct + pr * UN + 4 * cq);
            const float d = dyt[pr];
            sc[0] = fmaf(c4.x, d, sc[0]);
            sc[1] = fmaf(c4.y, d, sc[1]);
            sc[2] = fmaf(c4.z, d, sc[2]);
            sc[3] = fmaf(c4.w, d, sc[3]);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            for (int m = 1; m < 16; m <<= 1) sb[j] += __shfl_xor(sb[j], m);
            for (int m = 4; m < 64; m <<= 1) sc[j] += __shfl_xor(sc[j], m);
        }
        // lane 16 g + 0 holds bx rows 4j + g; lanes 0..3 hold v[4 cq + j]
        if (sub == 0) {
#pragma unroll
            for (int j = 0; j < 4; ++j) a.bx[row * UN + 4 * j + g] = sb[j];
        }
        if (lane < 4) {
#pragma unroll
            for (int j = 0; j < 4; ++j) a.v[row * UN + 4 * cq + j] = sc[j];
        }
    }
}

typedef float f4 __attribute__((ext_vector_type(4)));

// M X for a 16 x 16 matrix M and X in the MFMA output layout (lane 16 g + j holds
// X[4g + r][j] in component r): the four v_mfma_f32_16x16x4_f32 of the product
// each take, in lane 16 q + i, M[i][4q + kb] and X[4q + kb][i] (so instruction kb
// sums over the columns 4q + kb of M), and the latter is component kb of the
// lane's own X: the product needs no data movement and its result is again in
// the output layout.  m4 holds the lane's operand values of M (M[i][4q + kb], a
// float4 of row i; M[4q + kb][i] for M^T X, see vals_t), loaded ahead by the
// caller.
__device__ __forceinline__ f4 mul_vals(const float4 m4, f4 X) {
    f4 acc = {0.f, 0.f, 0.f, 0.f};
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(m4.x, X[0], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(m4.y, X[1], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(m4.z, X[2], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(m4.w, X[3], acc, 0, 0, 0);
    return acc;
}
// Lane 16 q + i's operand values of M^T X.
__device__ __forceinline__ float4 vals_t(const float* M, int i, int q) {
    return make_float4(M[(4 * q) * UN + i], M[(4 * q + 1) * UN + i], M[(4 * q + 2) * UN + i], M[(4 * q + 3) * UN + i]);
}
__device__ __forceinline__ f4 identity16(int i, int q) {
    f4 e;
    for (int r = 0; r < 4; ++r) e[r] = (4 * q + r == i) ? 1.f : 0.f;
    return e;
}

// grid (nc, b), 64 threads
__global__ __launch_bounds__(64) void k_un_aggr(const UnArgs a) {
    const int lane = threadIdx.x, i = lane & 15, q = lane >> 4;
    const int64_t c = blockIdx.x, bb = blockIdx.y;
    const int64_t s0 = c * a.L, s1 = min(s0 + a.L, a.T);
    // Phi in the MFMA output layout: lane (q, i) holds Phi[4q + r][i], r = 0..3
    f4 phi = identity16(i, q);
    float h = 0.f, m = 0.f;  // replicated: lane (q, i) holds h[i], m[i]
    // step t's A_t[i][4q..4q+3], bx_t[i] and v_t[4q..4q+3], loaded a step ahead
    // (the last step reloads its own)
    const int64_t r0 = bb * a.T + s0;
    float4 an = *reinterpret_cast<const float4*>(a.A + r0 * UN * UN + i * UN + 4 * q);
    float bn = a.bx[r0 * UN + i];
    float4 vn = *reinterpret_cast<const float4*>(a.v + r0 * UN + 4 * q);
    for (int64_t t = s0; t < s1; ++t) {
        const int64_t row = bb * a.T + t;
        const float4 a4 = an, v4 = vn;
        const float bxt = bn;
        const int64_t nx = t + 1 < s1 ? row + 1 : row;
        an = *reinterpret_cast<const float4*>(a.A + nx * UN * UN + i * UN + 4 * q);
        bn = a.bx[nx * UN + i];
        vn = *reinterpret_cast<const float4*>(a.v + nx * UN + 4 * q);
        // h <- A_t h + B_t x_t
        const float4 hq = quarter_of(h, q);
        h = qsum(a4.x * hq.x + a4.y * hq.y + a4.z * hq.z + a4.w * hq.w) + bxt;
        // Phi <- A_t Phi (operands in registers, see mul_vals)
        phi = mul_vals(a4, phi);
        if (!a.trunc) {
            // the adjoint aggregate m += Phi_t^T v_t; lane (q, j): sum_r Phi[4q + r][j] v[4q + r]
            m += qsum(phi[0] * v4.x + phi[1] * v4.y + phi[2] * v4.z + phi[3] * v4.w);
        }
    }
    const int64_t cb = bb * a.nc + c;
    for (int r = 0; r < 4; ++r) a.phi[cb * UN * UN + (4 * q + r) * UN + i] = phi[r];
    if (q == 0) {
        a.hc[cb * UN + i] = h;
        a.mc[cb * UN + i] = m;
    }
}

// grid (2 b), 64 threads: lanes (q, i) as above; workgroup 2 bb + dir walks
// sequence bb forwards (dir 0) or backwards (dir 1); each chunk's Phi and
// aggregate loaded a chunk ahead.
__global__ __launch_bounds__(64) void k_un_carry(const UnArgs a) {
    const int lane = threadIdx.x, i = lane & 15, q = lane >> 4;
    const int64_t bb = blockIdx.x >> 1;
    const int dir = blockIdx.x & 1;
    const int64_t nc = a.nc, c0 = bb * nc;
    if (dir == 1) {
        // M_{c-1} = Phi_c^T M_c + mloc_c  (lane (q, j): rows 4q..4q+3 of column j)
        float M = 0.f;
        const int64_t cl = c0 + nc - 1;
        float4 qn = vals_t(a.phi + cl * UN * UN, i, q);
        float mn = a.mc[cl * UN + i];
        for (int64_t c = nc - 1; c >= 0; --c) {
            const int64_t cb = c0 + c;
            const float4 p4 = qn;
            const float ml = mn;
            const int64_t nx = c > 0 ? cb - 1 : cb;
            qn = vals_t(a.phi + nx * UN * UN, i, q);
            mn = a.mc[nx * UN + i];
            const float4 mq = quarter_of(M, q);
            const float Mn = qsum(p4.x * mq.x + p4.y * mq.y + p4.z * mq.z + p4.w * mq.w) + ml;
            if (q == 0) a.mc[cb * UN + i] = M;  // the carry from the right into chunk c
            M = Mn;
        }
        if (a.dh0 && q == 0) a.dh0[bb * UN + i] = M;
        return;
    }
    float H = a.h0 ? a.h0[bb * UN + i] : 0.f;  // replicated
    // H_{c+1} = Phi_c H_c + hloc_c  (lane (q, i): columns 4q..4q+3 of row i)
    float4 pn = *reinterpret_cast<const float4*>(a.phi + c0 * UN * UN + i * UN + 4 * q);
    float hn = a.hc[c0 * UN + i];
    for (int64_t c = 0; c < nc; ++c) {
        const int64_t cb = c0 + c;
        const float4 p4 = pn;
        const float hl = hn;
        const int64_t nx = c + 1 < nc ? cb + 1 : cb;
        pn = *reinterpret_cast<const float4*>(a.phi + nx * UN * UN + i * UN + 4 * q);
        hn = a.hc[nx * UN + i];
        const float4 hq = quarter_of(H, q);
        const float Hn = qsum(p4.x * hq.x + p4.y * hq.y + p4.z * hq.z + p4.w * hq.w) + hl;
        if (q == 0) a.hc[cb * UN + i] = H;  // the carry into chunk c (hloc_c was read above)
        H = Hn;
    }
    if (a.h_last && q == 0) a.h_last[bb * UN + i] = H;
}

// grid (blocks - 1, b), 64 threads: block beta >= 1, steps [k, k + tbar) with
// k = beta tbar; Pre = Phi(k, j) = A_j ... A_{k+1} in registers (output layout),
// y_j = Pre^T v_j (lane (g, j'): sum_r Pre[4g + r][j'] v_j[4g + r], summed over g).
__global__ __launch_bounds__(64) void k_un_wpre(const UnArgs a) {
    const int lane = threadIdx.x, i = lane & 15, q = lane >> 4;
    const int64_t bb = blockIdx.y;
    const int64_t k = (static_cast<int64_t>(blockIdx.x) + 1) * a.tbar;
    if (k >= a.T) return;
    const int64_t k1 = min(k + a.tbar, a.T);
    f4 pre = identity16(i, q);
    // A_j's operand values and v_j of step j, loaded one step ahead (the last step
    // reloads its own; A_k is loaded and not used)
    const int64_t r0 = bb * a.T + k;
    float4 an = *reinterpret_cast<const float4*>(a.A + r0 * UN * UN + i * UN + 4 * q);
    float4 vn = *reinterpret_cast<const float4*>(a.v + r0 * UN + 4 * q);
    for (int64_t j = k; j < k1; ++j) {
        const int64_t row = bb * a.T + j;
        const float4 ac = an, v4 = vn;
        const int64_t nx = j + 1 < k1 ? row + 1 : row;
        an = *reinterpret_cast<const float4*>(a.A + nx * UN * UN + i * UN + 4 * q);
        vn = *reinterpret_cast<const float4*>(a.v + nx * UN + 4 * q);
        if (j > k) pre = mul_vals(ac, pre);
        const float y = qsum(pre[0] * v4.x + pre[1] * v4.y + pre[2] * v4.z + pre[3] * v4.w);
        if (q == 0) a.y[row * UN + i] = y;
    }
}

// Sum over the 16 lanes of each quarter of the wave.
__device__ __forceinline__ float sum16(float v) {
    v += __shfl_xor(v, 1);
    v += __shfl_xor(v, 2);
    v += __shfl_xor(v, 4);
    v += __shfl_xor(v, 8);
    return v;
}

// grid (blocks, b), 64 threads: block beta, steps [beta tbar, k) with k =
// (beta + 1) tbar < T; S = Phi(i, k)^T = A_{i+1}^T S(i + 1), S(k) = I, in registers
// (output layout: lane (g, n) holds S[4g + r][n]); w_i = S y_{i+tbar} (lane (g, n):
// S[4g + r][n] y[n], summed over n), and v_i -= w_i while i + tbar < T.
__global__ __launch_bounds__(64) void k_un_wsuf(const UnArgs a) {
    const int lane = threadIdx.x, i = lane & 15, q = lane >> 4;
    const int64_t bb = blockIdx.y;
    const int64_t k0 = static_cast<int64_t>(blockIdx.x) * a.tbar;
    const int64_t k = k0 + a.tbar;
    if (k >= a.T) return;
    f4 sm = identity16(i, q);
    // A_{t+1}'s operand values and y_{t+tbar} of the next step, loaded one step
    // ahead (clamped to valid rows; a y past the end is not used)
    const int64_t base = bb * a.T;
    float4 an = vals_t(a.A + (base + k) * UN * UN, i, q);
    float yv = a.y[(base + min(k - 1 + a.tbar, a.T - 1)) * UN + i];
    for (int64_t t = k - 1; t >= k0; --t) {
        const int64_t row = base + t;
        const float4 ac = an;
        const float yn = yv;
        const int64_t tn = t > k0 ? t - 1 : t;
        an = vals_t(a.A + (base + tn + 1) * UN * UN, i, q);
        yv = a.y[(base + min(tn + a.tbar, a.T - 1)) * UN + i];
        sm = mul_vals(ac, sm);
        if (t + a.tbar >= a.T) continue;  // wave-uniform
        float w[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) w[r] = sum16(sm[r] * yn);
        if (i < 4) {
            const float wr = i == 0 ? w[0] : i == 1 ? w[1] : i == 2 ? w[2] : w[3];
            a.v[row * UN + 4 * q + i] -= wr;
        }
    }
}

// grid (nc, b), 64 threads: the chunk's adjoint aggregate of u (v after
// k_un_wsuf), as k_un_aggr forms it from v in full mode: rho_e = u_e,
// rho_t = u_t + A_{t+1}^T rho_{t+1}, mloc = A_s^T rho_s.
__global__ __launch_bounds__(64) void k_un_madj(const UnArgs a) {
    __shared__ float sr[UN];
    const int lane = threadIdx.x, i = lane & 15, q = lane >> 4;
    const int64_t c = blockIdx.x, bb = blockIdx.y;
    const int64_t s0 = c * a.L, s1 = min(s0 + a.L, a.T);
    float carry = 0.f;  // A_{t+1}^T rho_{t+1} (replicated)
    for (int64_t t = s1 - 1; t >= s0; --t) {
        const int64_t row = bb * a.T + t;
        const float rho = a.v[row * UN + i] + carry;
        if (q == 0) sr[i] = rho;
        __syncthreads();
        const float* At = a.A + row * UN * UN;
        float part = 0.f;
        for (int r = 0; r < 4; ++r) part = fmaf(At[(4 * q + r) * UN + i], sr[4 * q + r], part);
        carry = qsum(part);
        __syncthreads();
    }
    if (q == 0) a.mc[(bb * a.nc + c) * UN + i] = carry;
}

// grid (nc, b), 64 threads; LDS holds the chunk's states h_{s-1} .. h_e.
template <int L>
__global__ __launch_bounds__(64) void k_un_grad(const UnArgs a) {
    __shared__ float shs[L + 1][UN];
    __shared__ float smu[L][UN];
    const int lane = threadIdx.x, i = lane & 15, q = lane >> 4;
    const int64_t c = blockIdx.x, bb = blockIdx.y;
    const int64_t s0 = c * L, s1 = min(s0 + L, a.T);
    const int64_t cb = bb * a.nc + c;
    const int64_t P = a.P;
    // the states h_{s-1} .. h_e into LDS (h in registers, replicated), with step
    // t's A_t[i][4q..4q+3] and bx_t[i] loaded a step ahead
    {
        float h = a.hc[cb * UN + i];
        if (q == 0) shs[0][i] = h;
        const int64_t r0 = bb * a.T + s0;
        float4 an = *reinterpret_cast<const float4*>(a.A + r0 * UN * UN + i * UN + 4 * q);
        float bn = a.bx[r0 * UN + i];
        for (int64_t t = s0; t < s1; ++t) {
            const int64_t row = bb * a.T + t;
            const float4 a4 = an;
            const float bxt = bn;
            const int64_t nx = t + 1 < s1 ? row + 1 : row;
            an = *reinterpret_cast<const float4*>(a.A + nx * UN * UN + i * UN + 4 * q);
            bn = a.bx[nx * UN + i];
            const float4 hq = quarter_of(h, q);
            h = qsum(a4.x * hq.x + a4.y * hq.y + a4.z * hq.z + a4.w * hq.w) + bxt;
            if (q == 0) shs[t - s0 + 1][i] = h;
        }
    }
    // the chunk's adjoints, sequential: mu_t = v_t + A_{t+1}^T mu_{t+1} (replicated,
    // exchanged by shuffles), into LDS; in truncated mode v holds u and the
    // recurrence gives the windowed adjoint.  v_t and step t's operand values of
    // A_t^T mu are loaded a step ahead.
    {
        float mun = a.mc[cb * UN + i];  // A_{t+1}^T mu_{t+1}
        const int64_t re = bb * a.T + s1 - 1;
        float vn = a.v[re * UN + i];
        float4 an = vals_t(a.A + re * UN * UN, i, q);
        for (int64_t t = s1 - 1; t >= s0; --t) {
            const int64_t row = bb * a.T + t;
            const float vt = vn;
            const float4 a4 = an;
            const int64_t nx = t > s0 ? row - 1 : row;
            vn = a.v[nx * UN + i];
            an = vals_t(a.A + nx * UN * UN, i, q);
            const float mu = vt + mun;
            if (q == 0) smu[t - s0][i] = mu;
            const float4 mq = quarter_of(mu, q);
            mun = qsum(a4.x * mq.x + a4.y * mq.y + a4.z * mq.z + a4.w * mq.w);
        }
    }
    __syncthreads();
    // the vjps of every step, independent of one another
    for (int64_t t = s0; t < s1; ++t) {
        const int64_t row = bb * a.T + t;
        const int k = static_cast<int>(t - s0);
        // dA_t[r][4(l%4) .. +3] = mu[r] h_{t-1}[..], r = l / 4
        {
            const int r = lane >> 2, c4 = (lane & 3) * 4;
            const float m = smu[k][r];
            const float4 hv = make_float4(shs[k][c4] * m, shs[k][c4 + 1] * m, shs[k][c4 + 2] * m,
                                          shs[k][c4 + 3] * m);
            *reinterpret_cast<float4*>(a.dA + row * UN * UN + r * UN + c4) = hv;
        }
        // dB_t[r][p] = mu[r] x_t[p]; dC_t[p][r] = dy_t[p] h_t[r]; four values per lane and pass
        const float* xt = a.x + row * P;
        const float* dyt = a.dy + row * P;
        for (int64_t e = 4 * lane; e < UN * P; e += 256) {
            const int64_t r = e / P, p = e % P;
            const float m = smu[k][r];
            const float4 x4 = *reinterpret_cast<const float4*>(xt + p);
            *reinterpret_cast<float4*>(a.dB + row * UN * P + e) = make_float4(m * x4.x, m * x4.y, m * x4.z, m * x4.w);
            const int64_t pc = e / UN, rc = e % UN;
            const float g = dyt[pc];
            *reinterpret_cast<float4*>(a.dC + row * P * UN + e) =
                make_float4(g * shs[k + 1][rc], g * shs[k + 1][rc + 1], g * shs[k + 1][rc + 2], g * shs[k + 1][rc + 3]);
        }
        // dx_t[p] = sum_r B_t[r][p] mu[r]
        const float* Bt = a.B + row * UN * P;
        for (int64_t p = lane; p < P; p += 64) {
            float sx = 0.f;
            for (int r = 0; r < UN; ++r) sx = fmaf(Bt[r * P + p], smu[k][r], sx);
            a.dx[row * P + p] = sx;
        }
    }
}

}  // namespace

size_t unstructured_workspace(int64_t nb, int64_t T, int64_t L, bool trunc) {
    const int64_t nc = (T + L - 1) / L;
    auto up = [](size_t v) { return (v + 255) & ~size_t(255); };
    size_t s = up(size_t(nb * nc) * UN * UN * 4) + 2 * up(size_t(nb * nc) * UN * 4) + 2 * up(size_t(nb * T) * UN * 4);
    if (trunc) s += up(size_t(nb * T) * UN * 4);
    return s;
}

hipError_t launch_unstructured_grad(const UnstructuredProblem& u, void* ws, hipStream_t s) {
    UnArgs a{};
    a.nb = u.nb;
    a.T = u.T;
    a.P = u.P;
    a.L = u.L;
    a.nc = (u.T + u.L - 1) / u.L;
    a.trunc = u.trunc ? 1 : 0;
    a.tbar = u.tbar;
    a.A = u.A;
    a.B = u.B;
    a.C = u.C;
    a.x = u.x;
    a.h0 = u.h0;
    a.dy = u.dy;
    a.dA = u.dA;
    a.dB = u.dB;
    a.dC = u.dC;
    a.dx = u.dx;
    a.dh0 = u.dh0;
    a.h_last = nullptr;
    auto up = [](size_t v) { return (v + 255) & ~size_t(255); };
    char* w = static_cast<char*>(ws);
    a.phi = reinterpret_cast<float*>(w);
    w += up(size_t(a.nb * a.nc) * UN * UN * 4);
    a.hc = reinterpret_cast<float*>(w);
    w += up(size_t(a.nb * a.nc) * UN * 4);
    a.mc = reinterpret_cast<float*>(w);
    w += up(size_t(a.nb * a.nc) * UN * 4);
    a.v = reinterpret_cast<float*>(w);
    w += up(size_t(a.nb * a.T) * UN * 4);
    a.bx = reinterpret_cast<float*>(w);
    w += up(size_t(a.nb * a.T) * UN * 4);
    a.y = u.trunc ? reinterpret_cast<float*>(w) : nullptr;
    const dim3 gc(static_cast<unsigned>(a.nc), static_cast<unsigned>(a.nb));
    {
        SSMK_TIMED("un_proj", s);
        hipLaunchKernelGGL(k_un_proj, dim3(static_cast<unsigned>((a.T + 3) / 4), static_cast<unsigned>(a.nb)),
                           dim3(64), 0, s, a);
    }
    {
        SSMK_TIMED("un_aggr", s);
        hipLaunchKernelGGL(k_un_aggr, gc, dim3(64), 0, s, a);
    }
    if (a.trunc) {
        const int64_t nblk = (a.T + a.tbar - 1) / a.tbar;  // at least 2 (tbar < T)
        {
            SSMK_TIMED("un_wpre", s);
            hipLaunchKernelGGL(k_un_wpre, dim3(static_cast<unsigned>(nblk - 1), static_cast<unsigned>(a.nb)),
                               dim3(64), 0, s, a);
        }
        {
            SSMK_TIMED("un_wsuf", s);
            hipLaunchKernelGGL(k_un_wsuf, dim3(static_cast<unsigned>(nblk), static_cast<unsigned>(a.nb)), dim3(64),
                               0, s, a);
        }
        SSMK_TIMED("un_madj", s);
        hipLaunchKernelGGL(k_un_madj, gc, dim3(64), 0, s, a);
    }
    {
        SSMK_TIMED("un_carry", s);
        hipLaunchKernelGGL(k_un_carry, dim3(static_cast<unsigned>(2 * a.nb)), dim3(64), 0, s, a);
    }
    SSMK_TIMED("un_grad", s);
    switch (a.L) {
        case 16: hipLaunchKernelGGL(k_un_grad<16>, gc, dim3(64), 0, s, a); break;
        case 32: hipLaunchKernelGGL(k_un_grad<32>, gc, dim3(64), 0, s, a); break;
        case 64: hipLaunchKernelGGL(k_un_grad<64>, gc, dim3(64), 0, s, a); break;
        case 128: hipLaunchKernelGGL(k_un_grad<128>, gc, dim3(64), 0, s, a); break;
        default: hipLaunchKernelGGL(k_un_grad<256>, gc, dim3(64), 0, s, a); break;
    }
    return hipGetLastError();
}

}  // namespace ssmk
