/*
 * oracle.c -- plain, slow, fp64 CPU oracle for the per-layer adjoint gradient
 * of a selective diagonal state-space layer ("Adjoint sharding for very long
 * context training of state space models", arXiv 2501.00692).
 *
 * TEST INFRASTRUCTURE ONLY. It is loaded by the test suite, by the smoke check
 * and by the benchmark's CPU-baseline leg, never by the product path, and it
 * shares no code, header, table or helper with the HIP library.
 *
 * The layer (Sec. 3.1, the five SSM steps, specialised to a diagonal,
 * input-dependent decay):
 *   a_t[d,n] = exp(-Delta_t[d] * exp(A_log[d,n]))          step 1, A^t = A(x^t)
 *   h_t[d,n] = a_t[d,n] h_{t-1}[d,n] + B_t[n] x_t[d]        step 4
 *   y_t[d]   = sum_n C_t[n] h_t[d,n]                        step 5
 * with h_0 a fixed constant (zero unless given).  Optional extras that the
 * layer workloads use: Delta = softplus(Delta_pre), and a SiLU output gate
 * out_t = y_t * silu(z_t).  The loss is L = sum_{b,t,d} dy_t[d] * out_t[d],
 * so dy is the upstream gradient dL/dout.
 *
 * The `flags` argument selects (bits):
 *   OR_SOFTPLUS  the delta input is Delta_pre and Delta = softplus(Delta_pre);
 *   OR_A_SCALAR  the "scalar SSM" row of Table 1: one decay per channel,
 *                A^t = a_t[d] I with a_t[d] = exp(-Delta_t[d] exp(A_log[d]));
 *                A_log and dA_log are [D];
 *   OR_B_DELTA   the input term scaled by the step size, B^t x^t -> Delta_t B_t x_t
 *                (the step-size-scaled input of selective SSM discretisations).
 *
 * Layouts (row-major, fp64): x, delta, z, dy, out, dx, ddelta, dz : [b][T][D];
 * B, C, dB, dC : [b][T][N]; A_log, dA_log : [D][N] (or [D]); h0, h_last, dh0 :
 * [b][D][N]; da : [b][T][D][N], the cotangent of the decay a_t[d,n] itself (the
 * diagonal of Prop. 2's vjp_A term before it is chained into Delta and A_log).
 * All gradient outputs are overwritten.
 *
 * Functions and the passages they follow:
 *   oracle_forward      Sec. 3.1 five steps (sequential loop over t).
 *   oracle_bptt         exact gradient by backpropagation through time, i.e.
 *                       the nested expansion of Sec. 3.3 evaluated from the
 *                       outermost step inwards (Prop. 1 recurrence for the
 *                       state cotangent).
 *   oracle_adjoint_sum  Prop. 2 (and Eq. "capped" for the truncated form)
 *                       taken literally: for every t, the adjoint states
 *                       lambda^{t,i} = C^t A^t ... A^{i+1} are formed for
 *                       i = t, t-1, ..., and each vjp_A / vjp_B / vjp_C term is
 *                       accumulated.  Cost O(T * Tbar) per channel.
 *   oracle_trunc_tail   the truncated estimator of Eq. "capped" rewritten with
 *                       the tail identity (derivation in the module header of
 *                       the Python wrapper); O(T) per channel, used where the
 *                       literal double sum is too slow.  Pinned against
 *                       oracle_adjoint_sum by the tests.
 *   oracle_proj_dw/dx   dW = X^T dZ and dX = dZ W^T by plain loops on sampled
 *                       entries (the chain rule through the input projections).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Channel blocks with private dB/dC accumulators: a fixed count, so the final
 * summation order (and hence every output bit) does not depend on the number
 * of threads. */
#define ORACLE_NBLK 16

enum { OR_SOFTPLUS = 1, OR_A_SCALAR = 2, OR_B_DELTA = 4 };

/* log of the decay rate of (channel d, state n). */
static double alog_at(const double* A_log, int flags, int64_t d, int64_t N, int64_t n) {
    return (flags & OR_A_SCALAR) ? A_log[d] : A_log[d * N + n];
}

static double softplus(double p) { return p > 0.0 ? p + log1p(exp(-p)) : log1p(exp(p)); }
static double sigmoid(double p) {
    if (p >= 0.0) return 1.0 / (1.0 + exp(-p));
    double e = exp(p);
    return e / (1.0 + e);
}

static void set_threads(int nthreads) {
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
}

int oracle_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------------------ */
/* Forward: Sec. 3.1 steps 1-5, one channel at a time, sequential in t.      */
/* ------------------------------------------------------------------------ */
int oracle_forward(int64_t nb, int64_t T, int64_t D, int64_t N,
                   const double* x, const double* delta, int flags,
                   const double* A_log, const double* B, const double* C,
                   const double* h0, const double* z,
                   double* out, double* h_last, int nthreads) {
    if (nb < 1 || T < 1 || D < 1 || N < 1) return -1;
    set_threads(nthreads);
#pragma omp parallel for schedule(dynamic)
    for (int64_t d = 0; d < D; ++d) {
        double* h = (double*)malloc((size_t)N * sizeof(double));
        for (int64_t bb = 0; bb < nb; ++bb) {
            for (int64_t n = 0; n < N; ++n) h[n] = h0 ? h0[(bb * D + d) * N + n] : 0.0;
            for (int64_t t = 0; t < T; ++t) {
                int64_t td = (bb * T + t) * D + d;
                double dl = (flags & OR_SOFTPLUS) ? softplus(delta[td]) : delta[td];
                double u = (flags & OR_B_DELTA) ? dl * x[td] : x[td];
                double y = 0.0;
                for (int64_t n = 0; n < N; ++n) {
                    double a = exp(-dl * exp(alog_at(A_log, flags, d, N, n)));
                    h[n] = a * h[n] + B[(bb * T + t) * N + n] * u;
                    y += C[(bb * T + t) * N + n] * h[n];
                }
                out[td] = z ? y * z[td] * sigmoid(z[td]) : y;
            }
            if (h_last)
                for (int64_t n = 0; n < N; ++n) h_last[(bb * D + d) * N + n] = h[n];
        }
        free(h);
    }
    return 0;
}

/* Shared by the three gradient routines: the forward of one channel with all
 * states kept (hs[0] = h_0, hs[t+1] = h_t), the decays a[t][n], the effective
 * step sizes, and the gated upstream g_t = dL/dy_t together with dz. */
typedef struct {
    double* hs;   /* (T+1) x N */
    double* a;    /* T x N */
    double* dl;   /* T, Delta_t */
    double* g;    /* T, dL/dy_t */
} chan_fwd;

static void chan_forward(int64_t bb, int64_t d, int64_t T, int64_t D, int64_t N,
                         const double* x, const double* delta, int flags,
                         const double* A_log, const double* B, const double* C,
                         const double* h0, const double* z, const double* dy,
                         chan_fwd* f, double* dz) {
    for (int64_t n = 0; n < N; ++n) f->hs[n] = h0 ? h0[(bb * D + d) * N + n] : 0.0;
    for (int64_t t = 0; t < T; ++t) {
        int64_t td = (bb * T + t) * D + d;
        f->dl[t] = (flags & OR_SOFTPLUS) ? softplus(delta[td]) : delta[td];
        double u = (flags & OR_B_DELTA) ? f->dl[t] * x[td] : x[td];
        double y = 0.0;
        for (int64_t n = 0; n < N; ++n) {
            double a = exp(-f->dl[t] * exp(alog_at(A_log, flags, d, N, n)));
            f->a[t * N + n] = a;
            f->hs[(t + 1) * N + n] = a * f->hs[t * N + n] + B[(bb * T + t) * N + n] * u;
            y += C[(bb * T + t) * N + n] * f->hs[(t + 1) * N + n];
        }
        if (z) {
            double s = sigmoid(z[td]);
            f->g[t] = dy[td] * z[td] * s;                        /* d out / d y = silu(z) */
            if (dz) dz[td] = dy[td] * y * s * (1.0 + z[td] * (1.0 - s)); /* silu'(z) */
        } else {
            f->g[t] = dy[td];
        }
    }
}

/* VJP of step i with respect to (a_i, b_i = B_i u_i), given the state
 * cotangent w[n] = dL/dh_i (or the part of it that is being accumulated):
 *   vjp_A: dL/da_i = w * h_{i-1}, chained through a = exp(-Delta e^{A_log});
 *   vjp_B: dL/db_i = w, chained through b = B_i u_i with u_i = x_i (or
 *          Delta_i x_i with OR_B_DELTA, which also reaches Delta).  */
static void step_vjp(int64_t bb, int64_t i, int64_t d, int64_t T, int64_t D, int64_t N, int flags,
                     const double* w, const chan_fwd* f, const double* x,
                     const double* A_log, const double* B,
                     double* dx, double* ddelta_raw, double* dA_log_row, double* dB_acc, double* da_out) {
    int64_t td = (bb * T + i) * D + d;
    double sc = (flags & OR_B_DELTA) ? f->dl[i] : 1.0;  /* d u / d x */
    double sdx = 0.0, sdd = 0.0;
    for (int64_t n = 0; n < N; ++n) {
        double ea = exp(alog_at(A_log, flags, d, N, n));
        double da = w[n] * f->hs[i * N + n];            /* h_{i-1} is hs[i] */
        if (da_out) da_out[td * N + n] += da;             /* the cotangent of a_i itself */
        double ai = f->a[i * N + n];
        sdd += da * ai * (-ea);                           /* d a / d Delta */
        dA_log_row[(flags & OR_A_SCALAR) ? 0 : n] += da * ai * (-f->dl[i] * ea); /* d a / d A_log */
        sdx += w[n] * B[(bb * T + i) * N + n];
        dB_acc[(bb * T + i) * N + n] += w[n] * x[td] * sc;
    }
    dx[td] += sdx * sc;
    ddelta_raw[td] += sdd + ((flags & OR_B_DELTA) ? sdx * x[td] : 0.0);  /* d u / d Delta = x */
}

static int grad_common_checks(int64_t nb, int64_t T, int64_t D, int64_t N) {
    return (nb < 1 || T < 1 || D < 1 || N < 1) ? -1 : 0;
}

/* Apply dDelta_pre = dDelta * sigmoid(Delta_pre) when the step size is a
 * softplus of the stored input. */
static void finish_softplus(int64_t nb, int64_t T, int64_t D, const double* delta,
                            int flags, double* ddelta) {
    if (!(flags & OR_SOFTPLUS)) return;
    for (int64_t k = 0; k < nb * T * D; ++k) ddelta[k] *= sigmoid(delta[k]);
}

/* Sum the per-block dB/dC accumulators in block order. */
static void reduce_blocks(double* out, double* const* blk, int64_t len) {
    for (int64_t k = 0; k < len; ++k) {
        double s = 0.0;
        for (int q = 0; q < ORACLE_NBLK; ++q) s += blk[q][k];
        out[k] = s;
    }
}

/* Mode selector for the shared driver below. */
enum { MODE_BPTT = 0, MODE_DOUBLESUM = 1, MODE_TAIL = 2 };

static int grad_driver(int mode, int64_t nb, int64_t T, int64_t D, int64_t N, int64_t tbar,
                       const double* x, const double* delta, int flags,
                       const double* A_log, const double* B, const double* C,
                       const double* h0, const double* z, const double* dy,
                       double* dx, double* ddelta, double* dA_log, double* dB, double* dC,
                       double* dz, double* dh0, double* da, int nthreads) {
    if (grad_common_checks(nb, T, D, N)) return -1;
    int full = (tbar <= 0 || tbar >= T);
    if (!full && dh0) return -2; /* dh0 is defined for the full gradient only */
    if (mode == MODE_BPTT && !full) return -3;
    set_threads(nthreads);

    memset(dx, 0, (size_t)(nb * T * D) * sizeof(double));
    memset(ddelta, 0, (size_t)(nb * T * D) * sizeof(double));
    const int64_t NA = (flags & OR_A_SCALAR) ? 1 : N;  /* decay rates per channel */
    memset(dA_log, 0, (size_t)(D * NA) * sizeof(double));
    if (dz) memset(dz, 0, (size_t)(nb * T * D) * sizeof(double));
    if (dh0) memset(dh0, 0, (size_t)(nb * D * N) * sizeof(double));
    if (da) memset(da, 0, (size_t)(nb * T * D * N) * sizeof(double));

    int64_t btn = nb * T * N;
    double* blkB[ORACLE_NBLK];
    double* blkC[ORACLE_NBLK];
    for (int q = 0; q < ORACLE_NBLK; ++q) {
        blkB[q] = (double*)calloc((size_t)btn, sizeof(double));
        blkC[q] = (double*)calloc((size_t)btn, sizeof(double));
        if (!blkB[q] || !blkC[q]) return -4;
    }
    int64_t per = (D + ORACLE_NBLK - 1) / ORACLE_NBLK;

#pragma omp parallel for schedule(dynamic, 1)
    for (int q = 0; q < ORACLE_NBLK; ++q) {
        chan_fwd f;
        f.hs = (double*)malloc((size_t)((T + 1) * N) * sizeof(double));
        f.a = (double*)malloc((size_t)(T * N) * sizeof(double));
        f.dl = (double*)malloc((size_t)T * sizeof(double));
        f.g = (double*)malloc((size_t)T * sizeof(double));
        double* w = (double*)malloc((size_t)N * sizeof(double));
        double* lam = (double*)malloc((size_t)N * sizeof(double));
        double* mu = (mode == MODE_TAIL) ? (double*)malloc((size_t)((T + 1) * N) * sizeof(double)) : NULL;
        double* wsum = (mode == MODE_TAIL) ? (double*)malloc((size_t)(T + 1) * sizeof(double)) : NULL;
        int64_t d_lo = q * per, d_hi = (q + 1) * per < D ? (q + 1) * per : D;
        for (int64_t d = d_lo; d < d_hi; ++d) {
            double* dA_row = dA_log + d * NA; /* one writer per channel */
            for (int64_t bb = 0; bb < nb; ++bb) {
                chan_forward(bb, d, T, D, N, x, delta, flags, A_log, B, C, h0, z, dy, &f, dz);
                /* vjp_C (never truncated): dL/dC_t[n] += g_t h_t[n]. */
                for (int64_t t = 0; t < T; ++t)
                    for (int64_t n = 0; n < N; ++n)
                        blkC[q][(bb * T + t) * N + n] += f.g[t] * f.hs[(t + 1) * N + n];

                if (mode == MODE_BPTT) {
                    /* Backward through the recurrence: lam = dL/dh_t arriving
                     * from step t+1 (that is a_{t+1} * dL/dh_{t+1}); the total
                     * state cotangent at t adds the readout's g_t C_t. */
                    for (int64_t n = 0; n < N; ++n) lam[n] = 0.0;
                    for (int64_t t = T - 1; t >= 0; --t) {
                        for (int64_t n = 0; n < N; ++n)
                            w[n] = f.g[t] * C[(bb * T + t) * N + n] + lam[n];
                        step_vjp(bb, t, d, T, D, N, flags, w, &f, x, A_log, B, dx, ddelta, dA_row, blkB[q], da);
                        for (int64_t n = 0; n < N; ++n) lam[n] = f.a[t * N + n] * w[n];
                    }
                    if (dh0)
                        for (int64_t n = 0; n < N; ++n) dh0[(bb * D + d) * N + n] = lam[n];
                } else if (mode == MODE_DOUBLESUM) {
                    /* Prop. 2 / Eq. "capped": for each loss term t, the
                     * adjoint states lambda^{t,i} for i = t down to the window
                     * edge, lambda^{t,t} = C^t, lambda^{t,i-1} = lambda^{t,i} A^i. */
                    for (int64_t t = 0; t < T; ++t) {
                        int64_t i_lo = full ? 0 : (t - tbar + 1 > 0 ? t - tbar + 1 : 0);
                        for (int64_t n = 0; n < N; ++n) lam[n] = C[(bb * T + t) * N + n];
                        for (int64_t i = t; i >= i_lo; --i) {
                            for (int64_t n = 0; n < N; ++n) w[n] = f.g[t] * lam[n];
                            step_vjp(bb, i, d, T, D, N, flags, w, &f, x, A_log, B, dx, ddelta, dA_row, blkB[q], da);
                            for (int64_t n = 0; n < N; ++n) lam[n] *= f.a[i * N + n];
                        }
                        /* Prop. 1's lambda^0 term: only the full gradient
                         * reaches the initial state. */
                        if (full && dh0)
                            for (int64_t n = 0; n < N; ++n)
                                dh0[(bb * D + d) * N + n] += f.g[t] * lam[n];
                    }
                } else {
                    /* Tail form: mu_i = sum_{t>=i} g_t lambda^{t,i} obeys
                     * mu_i = g_i C_i + a_{i+1} mu_{i+1}; the window of Eq.
                     * "capped" keeps t in [i, i+Tbar-1], which equals
                     * mu_i - P(i, i+Tbar) mu_{i+Tbar} with
                     * P(i, i+Tbar) = prod_{j=i+1}^{i+Tbar} a_j
                     *             = exp(-e^{A_log} * sum_{j=i+1}^{i+Tbar} Delta_j). */
                    for (int64_t n = 0; n < N; ++n) mu[T * N + n] = 0.0;
                    for (int64_t t = T - 1; t >= 0; --t)
                        for (int64_t n = 0; n < N; ++n)
                            mu[t * N + n] = f.g[t] * C[(bb * T + t) * N + n] +
                                            (t + 1 < T ? f.a[(t + 1) * N + n] * mu[(t + 1) * N + n] : 0.0);
                    /* prefix sums of Delta in fp64: wsum[k] = sum_{j<k} Delta_j */
                    wsum[0] = 0.0;
                    for (int64_t t = 0; t < T; ++t) wsum[t + 1] = wsum[t] + f.dl[t];
                    for (int64_t i = 0; i < T; ++i) {
                        for (int64_t n = 0; n < N; ++n) w[n] = mu[i * N + n];
                        if (!full && i + tbar < T) {
                            double win = wsum[i + tbar + 1] - wsum[i + 1];
                            for (int64_t n = 0; n < N; ++n) {
                                double P = exp(-exp(alog_at(A_log, flags, d, N, n)) * win);
                                w[n] -= P * mu[(i + tbar) * N + n];
                            }
                        }
                        step_vjp(bb, i, d, T, D, N, flags, w, &f, x, A_log, B, dx, ddelta, dA_row, blkB[q], da);
                    }
                    if (full && dh0)
                        for (int64_t n = 0; n < N; ++n)
                            dh0[(bb * D + d) * N + n] = f.a[n] * mu[n];
                }
            }
        }
        free(f.hs); free(f.a); free(f.dl); free(f.g); free(w); free(lam);
        free(mu); free(wsum);
    }
    reduce_blocks(dB, blkB, btn);
    reduce_blocks(dC, blkC, btn);
    for (int q = 0; q < ORACLE_NBLK; ++q) { free(blkB[q]); free(blkC[q]); }
    finish_softplus(nb, T, D, delta, flags, ddelta);
    return 0;
}

int oracle_bptt(int64_t nb, int64_t T, int64_t D, int64_t N,
                const double* x, const double* delta, int flags,
                const double* A_log, const double* B, const double* C,
                const double* h0, const double* z, const double* dy,
                double* dx, double* ddelta, double* dA_log, double* dB, double* dC,
                double* dz, double* dh0, double* da, int nthreads) {
    return grad_driver(MODE_BPTT, nb, T, D, N, 0, x, delta, flags, A_log, B, C, h0, z,
                       dy, dx, ddelta, dA_log, dB, dC, dz, dh0, da, nthreads);
}

int oracle_adjoint_sum(int64_t nb, int64_t T, int64_t D, int64_t N, int64_t tbar,
                       const double* x, const double* delta, int flags,
                       const double* A_log, const double* B, const double* C,
                       const double* h0, const double* z, const double* dy,
                       double* dx, double* ddelta, double* dA_log, double* dB, double* dC,
                       double* dz, double* dh0, double* da, int nthreads) {
    return grad_driver(MODE_DOUBLESUM, nb, T, D, N, tbar, x, delta, flags, A_log, B, C,
                       h0, z, dy, dx, ddelta, dA_log, dB, dC, dz, dh0, da, nthreads);
}

int oracle_trunc_tail(int64_t nb, int64_t T, int64_t D, int64_t N, int64_t tbar,
                      const double* x, const double* delta, int flags,
                      const double* A_log, const double* B, const double* C,
                      const double* h0, const double* z, const double* dy,
                      double* dx, double* ddelta, double* dA_log, double* dB, double* dC,
                      double* dz, double* dh0, double* da, int nthreads) {
    return grad_driver(MODE_TAIL, nb, T, D, N, tbar, x, delta, flags, A_log, B, C, h0,
                       z, dy, dx, ddelta, dA_log, dB, dC, dz, dh0, da, nthreads);
}

/* ------------------------------------------------------------------------ */
/* Projection gradients on sampled entries (bf16 operands, exact upcast).    */
/* ------------------------------------------------------------------------ */
static double bf16_to_f64(uint16_t v) {
    uint32_t u = (uint32_t)v << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* out[p] = sum_m X[m][kk[p]] * dZ[m][jj[p]]  (dW = X^T dZ). */
int oracle_proj_dw(int64_t M, int64_t K, int64_t Nout, const uint16_t* X, int64_t ldx,
                   const uint16_t* dZ, int64_t lddz, int64_t npairs, const int64_t* kk,
                   const int64_t* jj, double* out, int nthreads) {
    if (M < 1 || K < 1 || Nout < 1 || ldx < K || lddz < Nout) return -1;
    set_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 4)
    for (int64_t p = 0; p < npairs; ++p) {
        double s = 0.0;
        for (int64_t m = 0; m < M; ++m)
            s += bf16_to_f64(X[m * ldx + kk[p]]) * bf16_to_f64(dZ[m * lddz + jj[p]]);
        out[p] = s;
    }
    return 0;
}

/* out[r][k] = sum_j dZ[rows[r]][j] * W[k][j]  (dX = dZ W^T, W stored [K][Nout]). */
int oracle_proj_dx(int64_t M, int64_t K, int64_t Nout, const uint16_t* dZ, int64_t lddz,
                   const uint16_t* W, int64_t ldw, int64_t nrows, const int64_t* rows,
                   double* out, int nthreads) {
    if (M < 1 || K < 1 || Nout < 1 || lddz < Nout || ldw < Nout) return -1;
    set_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < nrows; ++r)
        for (int64_t k = 0; k < K; ++k) {
            double s = 0.0;
            for (int64_t j = 0; j < Nout; ++j)
                s += bf16_to_f64(dZ[rows[r] * lddz + j]) * bf16_to_f64(W[k * ldw + j]);
            out[r * K + k] = s;
        }
    return 0;
}
