/*
 * ssm_adjoint.h -- C ABI of the MI355X (gfx950) per-layer adjoint-gradient
 * library for a selective diagonal state-space layer.
 *
 * The operation ("Adjoint sharding for very long context training of state
 * space models", arXiv 2501.00692):
 *   Sec. 3.1 (the five SSM steps), specialised to a diagonal, input-dependent
 *   decay with D channels of N states each:
 *     a_t[d,n] = exp(-Delta_t[d] * exp(A_log[d,n]))
 *     h_t[d,n] = a_t[d,n] * h_{t-1}[d,n] + B_t[n] * x_t[d]      (h_{-1} = h0, or 0)
 *     y_t[d]   = sum_n C_t[n] * h_t[d,n]
 *   optional: Delta = softplus(Delta_pre) (SSM_DELTA_SOFTPLUS) and a SiLU output
 *   gate out_t = y_t * silu(z_t) (SSM_GATE_SILU).
 *   Variants (Table 1 and the input discretisation):
 *     SSM_A_SCALAR : the scalar-decay SSM, one decay per channel shared by its
 *                    states, a_t[d,n] = exp(-Delta_t[d] * exp(A_log[d]));
 *                    A_log and dA_log are [channels];
 *     SSM_B_DELTA  : the input term scaled by the step size,
 *                    h_t = a_t * h_{t-1} + Delta_t[d] * B_t[n] * x_t[d].
 *   Prop. 2 (one layer): the gradient of L = sum_{b,t,d} dy_t[d] * out_t[d]
 *   splits into vector-Jacobian products of the A, B and C maps weighted by the
 *   adjoint states lambda^{t,i} = C^t A^t ... A^{i+1}; summed over the loss terms
 *   t these are the adjoint mu_i = sum_{t>=i} g_t lambda^{t,i}.
 *   Eq. "capped" (Sec. 4.3): the truncated form keeps, for every t, only the
 *   steps i in [t+1-Tbar, t] in the A and B terms; the C term is never truncated.
 *
 * Conventions for every entry point:
 *   - Tensor pointers are DEVICE pointers owned by the caller.  The library
 *     never allocates or frees device memory; scratch comes from the caller's
 *     `workspace` (size from the matching *_workspace_size query, 256-byte
 *     aligned pointer).
 *   - Layouts are row-major and contiguous: x, delta, z, dy, y, dx, ddelta, dz
 *     are [batch][seqlen][channels]; B, C, dB, dC are [batch][seqlen][dstate];
 *     A_log and dA_log are [channels][dstate]; h0, h_last, dh0 are
 *     [batch][channels][dstate].
 *   - "in_dtype" tensors are fp32 or bf16 (bit pattern of the upper 16 bits of
 *     an fp32); every gradient output is fp32 and is overwritten.
 *   - Every call validates its arguments on the host first; on any error it
 *     returns a non-zero status, enqueues nothing and leaves the outputs
 *     untouched.  On success the work is enqueued on `stream` (a hipStream_t;
 *     NULL is the default stream) and the call returns without synchronising;
 *     asynchronous faults surface at the caller's next synchronisation.
 *   - Results are deterministic: fixed-order reductions, no float atomics.
 *   - ssm_last_error() returns a thread-local description of the last failure.
 */
#ifndef SSM_ADJOINT_H
#define SSM_ADJOINT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    SSM_OK = 0,
    SSM_ERR_NULL = 1,        /* a required pointer is NULL                      */
    SSM_ERR_SHAPE = 2,       /* a size is out of range or inconsistent           */
    SSM_ERR_DTYPE = 3,       /* unknown dtype code                               */
    SSM_ERR_UNSUPPORTED = 4, /* valid request the library does not implement      */
    SSM_ERR_WORKSPACE = 5,   /* workspace NULL or smaller than the query says    */
    SSM_ERR_ALIGN = 6,       /* a pointer is not aligned as documented           */
    SSM_ERR_HIP = 7          /* the HIP runtime reported an error at launch       */
} ssm_status;

typedef enum { SSM_F32 = 0, SSM_BF16 = 1 } ssm_dtype;
typedef enum { SSM_FULL = 0, SSM_TRUNCATED = 1 } ssm_mode;

/* ssm_desc.flags */
#define SSM_DELTA_SOFTPLUS 1u /* `delta` holds Delta_pre; Delta = softplus(Delta_pre),
                                 and `ddelta` is the gradient w.r.t. Delta_pre          */
#define SSM_GATE_SILU 2u      /* `z` present: out = y * silu(z); `dy` is dL/dout        */
#define SSM_A_SCALAR 4u       /* one decay rate per channel: A_log, dA_log are [D]      */
#define SSM_B_DELTA 8u        /* input term Delta * B * x (dDelta includes its path)    */

/* ssm_stack_grad gradient kinds */
#define SSM_STACK_ADJOINT 0   /* Prop. 3: every layer's vjps under dL/dy_K                 */
#define SSM_STACK_EXACT 1     /* backpropagation through the whole stack                   */
#define SSM_STACK_FORWARD 2   /* the forward only: y_K for the language head                */

/* ssm_proj_grad flags */
#define SSM_ACCUM_DW 1u       /* dW += X^T dZ instead of dW = X^T dZ                   */
#define SSM_ACCUM_DX 2u       /* dX += dZ W^T instead of dX = dZ W^T                   */

typedef struct {
    int64_t batch;    /* b >= 1; b * T at most 2^40                                  */
    int64_t seqlen;   /* T >= 1                                                     */
    int64_t channels; /* D >= 1, at most 2^20 (the paper's P for a diagonal layer)   */
    int64_t dstate;   /* N, 1..16                                                   */
    int64_t chunk;    /* L, time steps per carry chunk: 0 (default 128), or one of
                         16, 32, 64, 128, 256.  Results do not depend on it beyond
                         rounding.                                                  */
    int32_t in_dtype; /* ssm_dtype of x, delta, B, C, z, dy (and of y)              */
    uint32_t flags;   /* SSM_DELTA_SOFTPLUS | SSM_GATE_SILU | SSM_A_SCALAR | SSM_B_DELTA */
} ssm_desc;

/* Workspace bytes needed by ssm_adjoint_forward / ssm_adjoint_grad for `desc`
 * (and `mode`, `tbar`).  Returns SSM_OK and writes *bytes, or an error status. */
ssm_status ssm_adjoint_forward_workspace_size(const ssm_desc* desc, size_t* bytes);
ssm_status ssm_adjoint_grad_workspace_size(const ssm_desc* desc, int32_t mode, int64_t tbar,
                                           size_t* bytes);

/* Forward pass (Sec. 3.1 steps 4-5, with the state recomputed chunk by chunk and
 * never stored per step).
 *   x, delta, B, C : in_dtype inputs;  A_log : fp32 [D][N] ([D] with SSM_A_SCALAR);
 *   h0     : fp32 [b][D][N] initial state, or NULL for zero;
 *   z      : in_dtype gate input, required iff SSM_GATE_SILU;
 *   y      : in_dtype output [b][T][D] (y, or y * silu(z) with the gate);
 *   h_last : fp32 [b][D][N] final state, or NULL. */
ssm_status ssm_adjoint_forward(const ssm_desc* desc, const void* x, const void* delta,
                               const float* A_log, const void* B, const void* C, const float* h0,
                               const void* z, void* y, float* h_last, void* workspace,
                               size_t workspace_bytes, void* stream);

/* Per-layer adjoint gradient (Prop. 2; with mode SSM_TRUNCATED the estimator of
 * Eq. "capped" with window `tbar` >= 1, where tbar >= T is the full gradient).
 * Inputs as for the forward, plus dy (in_dtype [b][T][D]) = dL/dout.
 * Outputs (fp32, overwritten):
 *   dx     [b][T][D]  B-path cotangent summed over the state, sum_n mubar B_t[n]
 *   ddelta [b][T][D]  dL/dDelta, or dL/dDelta_pre with SSM_DELTA_SOFTPLUS
 *   dA_log [D][N] ([D] with SSM_A_SCALAR)
 *   dB, dC [b][T][N]  (dC is never truncated)
 *   dz     [b][T][D]  required iff SSM_GATE_SILU, else must be NULL
 *   dh0    [b][D][N]  dL/dh0, full mode only (must be NULL when truncating), or NULL.
 *   da_debug [b][T][D][N] or NULL: a debug output, the cotangent of each decay value,
 *          da_t[d,n] = mubar_t[d,n] h_{t-1}[d,n] (Prop. 2's vjp_A term before it is
 *          chained into Delta and A_log; mubar the full or the windowed adjoint).  It
 *          is computed by a separate, slow kernel (one thread per batch, channel and
 *          state walking the sequence) that runs only when the pointer is given. 
 * The truncated A- and B-path terms use the windowed adjoint
 * mubar_i = sum_{t=i}^{min(T-1, i+tbar-1)} g_t C_t P(i, t), P(i, j) = prod_{k=i+1}^{j} a_k,
 * computed by its own reverse recurrence mubar_i = g_i C_i + a_{i+1} mubar_{i+1}
 * - P(i, i+tbar) g_{i+tbar} C_{i+tbar}. */
ssm_status ssm_adjoint_grad(const ssm_desc* desc, int32_t mode, int64_t tbar, const void* x,
                            const void* delta, const float* A_log, const void* B, const void* C,
                            const float* h0, const void* z, const void* dy, float* dx,
                            float* ddelta, float* dA_log, float* dB, float* dC, float* dz,
                            float* dh0, float* da_debug, void* workspace, size_t workspace_bytes,
                            void* stream);

/* ssm_adjoint_grad without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  Arguments, outputs, results and error
 * behaviour are those of ssm_adjoint_grad (the same kernels, bit-identical
 * outputs); the scratch is a 64 MiB device array inside the library, one per
 * GPU, held from the first call on that GPU until the process ends.  The call
 * allocates nothing.  It returns SSM_ERR_WORKSPACE, before anything is
 * enqueued, when the problem needs more scratch than that (the workspace size
 * that ssm_adjoint_grad_workspace_size reports for the same arguments is what
 * it needs).  Every call on one GPU uses that GPU's single array: calls that
 * can overlap on one GPU (different streams, or host threads) race and must be
 * serialised by the caller; calls on one stream are ordered.  No part of the
 * scratch needs to start at zero. */
ssm_status ssm_adjoint_grad_noalloc(const ssm_desc* desc, int32_t mode, int64_t tbar, const void* x,
                                    const void* delta, const float* A_log, const void* B,
                                    const void* C, const float* h0, const void* z, const void* dy,
                                    float* dx, float* ddelta, float* dA_log, float* dB, float* dC,
                                    float* dz, float* dh0, float* da_debug, void* stream);

/* The same gradient as ssm_adjoint_grad (identical arguments, layouts, outputs
 * and error behaviour), evaluated by the explicit pair formulation of Prop. 2 and
 * Eq. "capped": for every step i and every loss term t in its window
 * (i <= t < i + tbar, all t >= i in full mode) the adjoint state
 * lambda^{t,i} = g_t C_t prod_{j=i+1}^{t} a_j is built as a running product (the
 * zeta products of Alg. 2) and its vector-Jacobian products are accumulated, as
 * in the paper's count of independent VJPs (Sec. 4.3): the work grows as
 * b (tbar T - tbar (tbar-1)/2) D N, or b T (T+1)/2 D N in full mode, instead of
 * b T D N for ssm_adjoint_grad.  dh0 (full mode) is the sum over the pairs
 * (t, -1).  Results agree with ssm_adjoint_grad up to fp32 rounding. */
ssm_status ssm_adjoint_grad_pairs_workspace_size(const ssm_desc* desc, int32_t mode, int64_t tbar,
                                                 size_t* bytes);
ssm_status ssm_adjoint_grad_pairs(const ssm_desc* desc, int32_t mode, int64_t tbar, const void* x,
                                  const void* delta, const float* A_log, const void* B, const void* C,
                                  const float* h0, const void* z, const void* dy, float* dx,
                                  float* ddelta, float* dA_log, float* dB, float* dC, float* dz,
                                  float* dh0, float* da_debug, void* workspace, size_t workspace_bytes,
                                  void* stream);

/* Adjoint gradient of the unstructured SSM of Table 1 (Sec. 4.5): the general
 * SSM of Sec. 3.1 with a 16-dimensional state shared by the P channels and
 * full per-step matrices (the outputs of the A, B, C networks, taken as given):
 *   h_t = A_t h_{t-1} + B_t x_t,   y_t = C_t h_t,   L = sum_{b,t} <dy_t, y_t>,
 *   A [b][T][16][16], B [b][T][16][P], C [b][T][P][16], x, dy [b][T][P] (fp32,
 *   row-major), h0 [b][16] or NULL (zero).
 * desc: batch, seqlen, channels = P (a multiple of 16, at most 4096), dstate = 16,
 * chunk (0: 64; 16..256), in_dtype SSM_F32, flags 0 (SSM_ERR_UNSUPPORTED otherwise).
 * Outputs (fp32, overwritten): dA_t = mu_t h_{t-1}^T [b][T][16][16], dB_t = mu_t x_t^T
 * [b][T][16][P], dC_t = dy_t h_t^T [b][T][P][16] (never truncated), dx_t = B_t^T mu_t
 * [b][T][P], dh0 = A_0^T mu_0 [b][16] (full mode only, or NULL); mu is the state
 * cotangent mu_t = C_t^T dy_t + A_{t+1}^T mu_{t+1}, or with SSM_TRUNCATED the
 * windowed adjoint of Eq. "capped", sum_{t=i}^{i+tbar-1} (A_{i+1}^T ... A_t^T) C_t^T dy_t.
 * The chunk transition products A_e ... A_s are 16x16x16 products on fp32 MFMA.
 * Tensor pointers 16-byte aligned; workspace from the size query. */
ssm_status ssm_unstructured_grad_workspace_size(const ssm_desc* desc, int32_t mode, int64_t tbar,
                                                size_t* bytes);
ssm_status ssm_unstructured_grad(const ssm_desc* desc, int32_t mode, int64_t tbar, const float* A,
                                 const float* B, const float* C, const float* x, const float* h0,
                                 const float* dy, float* dA, float* dB, float* dC, float* dx,
                                 float* dh0, void* workspace, size_t workspace_bytes, void* stream);

/* Projection gradients of a linear map Z = X W (Sec. 4.5: the A, B, C networks
 * are single-layer maps; the per-step vjps summed over t give these products):
 *   dW [K][Nout] (fp32)  = X^T dZ      (skipped if dW == NULL)
 *   dX [M][K]    (fp32)  = dZ W^T      (skipped if dX == NULL; needs W)
 * X: bf16 [M][K] with row stride ldx >= K; dZ: bf16 [M][Nout], stride lddz >= Nout;
 * W: bf16 [K][Nout], stride ldw >= Nout.  flags: SSM_ACCUM_DW / SSM_ACCUM_DX.
 * bf16 operands, fp32 accumulation (MFMA).  Strides are in elements, multiples of
 * 8 and at most 2^21; K and Nout multiples of 8 and at most 2^20; pointers 16-byte
 * aligned (SSM_ERR_SHAPE / SSM_ERR_UNSUPPORTED / SSM_ERR_ALIGN otherwise). */
ssm_status ssm_proj_grad_workspace_size(int64_t M, int64_t K, int64_t Nout, uint32_t flags,
                                        size_t* bytes);
ssm_status ssm_proj_grad(int64_t M, int64_t K, int64_t Nout, const void* X, int64_t ldx,
                         const void* dZ, int64_t lddz, const void* W, int64_t ldw, float* dW,
                         float* dX, uint32_t flags, void* workspace, size_t workspace_bytes,
                         void* stream);

/* Whole-layer gradient for a layer with input projections (bf16 activations):
 *   [x | z] = u W_in,   [Delta_pre | B | C] = x W_x,   Delta = softplus(Delta_pre),
 *   out = y * silu(z).
 * Given the stored activations u [M][d_model], x, z, delta_pre [M][D], B, C [M][N]
 * (M = b*T rows), the weights W_x [D][D+2N] and W_in [d_model][2D] (bf16), A_log and
 * the upstream dy = dL/dout, it computes the scan gradient (as ssm_adjoint_grad with
 * SSM_DELTA_SOFTPLUS | SSM_GATE_SILU; of desc->flags only SSM_A_SCALAR and
 * SSM_B_DELTA are used), then
 *   dZx = [dDelta_pre | dB | dC]            (bf16, internal)
 *   dW_x = x^T dZx                           fp32 [D][D+2N]
 *   dx_total = dx + dZx W_x^T                fp32 [M][D] (optional output)
 *   dW_in = u^T [dx_total | dz]              fp32 [d_model][2D]
 *   du = [dx_total | dz] W_in^T              fp32 [M][d_model] (optional; needs W_in)
 * The per-token scan gradients dx, ddelta, dB, dC, dz may be given (fp32 outputs)
 * or NULL (kept in the workspace).  dA_log, dW_x and dW_in are required. */
ssm_status ssm_layer_grad_workspace_size(const ssm_desc* desc, int32_t mode, int64_t tbar,
                                         int64_t d_model, size_t* bytes);
ssm_status ssm_layer_grad(const ssm_desc* desc, int32_t mode, int64_t tbar, int64_t d_model,
                          const void* u, const void* x, const void* z, const void* delta_pre,
                          const void* B, const void* C, const void* W_x, const void* W_in,
                          const float* A_log, const void* dy, float* dW_in, float* dW_x,
                          float* dA_log, float* du, float* dx, float* ddelta, float* dB,
                          float* dC, float* dz, float* dx_total, void* workspace,
                          size_t workspace_bytes, void* stream);

/* Measurement support (not part of the method).  While enabled, every kernel the
 * library launches is bracketed by two hipEvents recorded on its stream;
 * ssm_timing_summary waits for the recorded events, writes one line
 * "<kernel> <launches> <total_ms>" per kernel name into buf (NUL-terminated,
 * truncated to len; SSM_ERR_SHAPE if truncated, SSM_ERR_HIP if an event failed)
 * and clears the records.  Timing adds an event pair per launch and is meant for
 * profiling runs only.  Not thread-safe across concurrent profiling sessions. */
ssm_status ssm_timing_enable(int32_t on);
ssm_status ssm_timing_summary(char* buf, size_t len);

/* Thread-local, NUL-terminated description of the last non-OK status returned on
 * the calling thread ("" if none).  Owned by the library. */
const char* ssm_last_error(void);

/* Parameter gradients of a stack of K residual SSM layers (Sec. 3.2 and Alg. 1:
 * y_0 given; for k = 1..K:  u_k = Norm(y_{k-1}),  y_k = y_{k-1} + SSM_k(u_k)),
 * with L = sum g_K * y_K for a given upstream g_K = dL/dy_K (the language head
 * and the loss stay with the caller, as Alg. 1 computes them once and hands
 * dL/dy_K to every device).  Norm is the root-mean-square normalisation over
 * the channels, u = y / sqrt(mean(y^2) + 1e-6), without a learned scale.  SSM_k is
 * the selective layer of ssm_layer_grad with its projections
 * ([x | z] = u W_in, [Delta_pre | B | C] = x W_x, out = scan(...) * silu(z)),
 * channel count D equal to the residual width (the paper's SSM maps P to P).
 *   desc   : batch b, seqlen T, channels D (= residual width), dstate N, chunk;
 *            in_dtype must be SSM_BF16 (the stored activations u, x, z,
 *            Delta_pre, B, C and each layer's output are bf16, round to
 *            nearest even); flags must be 0.
 *   K      : number of layers, 1..4096;  grad : SSM_STACK_ADJOINT (Prop. 3: each
 *            layer's gradient taken with the upstream g_K and the layer's own
 *            input, independently of the other layers) or SSM_STACK_EXACT
 *            (backpropagation: layer k's upstream is dL/dy_k, including the paths
 *            through later layers) or SSM_STACK_FORWARD (the forward alone: yK is
 *            required, gK and the gradient arrays may be NULL and are not touched;
 *            Alg. 1 runs it, evaluates the language head on y_K with
 *            ssm_lm_head_grad, and passes that call's dy as gK to a gradient
 *            call);  mode/tbar : as for ssm_adjoint_grad.
 *   y0     : fp32 [b][T][D];  gK : fp32 [b][T][D] (passed to the layers in bf16);
 *   W_in, W_x, A_log : host arrays of K device pointers (bf16 [D][2D], bf16
 *            [D][D+2N], fp32 [D][N]);  dW_in, dW_x, dA_log : host arrays of K device
 *            pointers to the fp32 outputs (overwritten);
 *   yK     : fp32 [b][T][D] output of the forward, or NULL.
 * The forward runs first and keeps every layer's activations in the workspace
 * (about 12 b T D bytes per layer plus the transposed projections); the layer
 * gradients then reuse the ssm_layer_grad path.  Everything is validated before
 * anything is enqueued. */
ssm_status ssm_stack_grad_workspace_size(const ssm_desc* desc, int64_t K, int32_t grad, int32_t mode,
                                         int64_t tbar, size_t* bytes);
ssm_status ssm_stack_grad(const ssm_desc* desc, int64_t K, int32_t grad, int32_t mode, int64_t tbar,
                          const float* y0, const void* const* W_in, const void* const* W_x,
                          const float* const* A_log, const float* gK, float* const* dW_in,
                          float* const* dW_x, float* const* dA_log, float* yK, void* workspace,
                          size_t workspace_bytes, void* stream);

/* The language head of Sec. 3.2 with its loss, the first gradient step of Alg. 1:
 * the prediction o^t = Omega Norm(y^t) (SSM_HEAD_NORM; flags 0 gives
 * o^t = Omega y^t, as Alg. 1 writes it), the per-token cross-entropy
 * l^t = log sum_v exp(o^t_v) - o^t_{target_t} (the paper leaves l open), and
 * the gradients dy = dl/dy (the upstream g_K that ssm_stack_grad takes) and
 * dOmega.  Norm is the stack's root-mean-square normalisation.
 *   M rows (tokens), P width, V vocabulary: P and V multiples of 8, at most 2^20;
 *             M below 2^31.
 *   y       : fp32 [M][P];  omega : bf16 [V][P];
 *   targets : int32 [M]; a negative target marks a token without a loss (l = 0,
 *             no gradient), a target >= V gives l = NaN and no gradient;
 *   loss    : fp32 [M];  dy : fp32 [M][P];  domega : fp32 [V][P], or NULL to skip it.
 *   block_rows : rows per block (a multiple of 256), or 0 for as many as keep the
 *             block's fp32 logits within 4 GiB; the workspace (which also holds
 *             Omega^T in bf16) grows with it.  Norm(y) and the logit gradients enter the
 * products as bf16 (round to nearest even) with fp32 accumulation; the
 * normalisation's backward recomputes Norm(y) in fp32; dOmega adds the blocks in
 * order.  SSM_ERR_UNSUPPORTED for P or V not a multiple of 8. */
#define SSM_HEAD_NORM 1u
ssm_status ssm_lm_head_grad_workspace_size(int64_t M, int64_t P, int64_t V, uint32_t flags, int64_t block_rows,
                                           size_t* bytes);
ssm_status ssm_lm_head_grad(int64_t M, int64_t P, int64_t V, uint32_t flags, int64_t block_rows, const float* y,
                            const void* omega,
                            const int32_t* targets, float* loss, float* dy, float* domega, void* workspace,
                            size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SSM_ADJOINT_H */
