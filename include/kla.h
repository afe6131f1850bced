/*
 * kla.h -- C ABI of the Kalman Linear Attention (KLA) filter layer for MI355X (gfx950).
 *
 * The layer is the time-parallel information-form Kalman filter of Kalman
 * Linear Attention (Sec. 4.2 of the paper; Algorithm 1, eqs. kla-prec-mat and
 * kla-mean-mat in Appendix A).  Per batch b and head h, with key slots n < dk
 * and value channels d < dv, for t = 1..T:
 *
 *   rho_t[n] = 1 / (abar_t[n]^2 + pbar_t[n] * lam_{t-1}[n])      prior ratio (gate view of Thm 1)
 *   lam_t[n] = rho_t[n] * lam_{t-1}[n] + k_t[n]^2 * r_t            precision (Theorem 1)
 *   F_t[n]   = abar_t[n] * rho_t[n]                                forget gate (Theorem 2)
 *   H_t[n,d] = F_t[n] * H_{t-1}[n,d] + r_t * k_t[n] * v_t[d]        information state (Theorem 2)
 *   y_t[d]   = sum_n q_t[n] / lam_t[n] * H_t[n,d]                  posterior-mean readout (Alg. 1)
 *   yvar_t   = sum_n q_t[n]^2 / lam_t[n]                            readout variance (Alg. 1, optional)
 *
 * r_t = Lambda^v_t is one observation precision per (token, head), so the
 * precision lam and the gate F depend on the key slot only.
 *
 * Conventions shared by every entry point
 *   Layout   : all tensors contiguous row-major.  Per-token tensors are
 *              [B, T, H, width] (width dk for q, k, abar, pbar; dv for v, y, dy),
 *              r is [B, T, H], yvar is [B, T, H]; beliefs are lam [B, H, dk],
 *              eta = H [B, H, dk, dv].
 *   Memory   : every pointer is a device pointer owned by the caller.  The
 *              library never allocates, frees or synchronises (KLA_CHECK=1 aside);
 *              all work is
 *              enqueued asynchronously on `stream` (0 = the null stream).
 *              Inputs are read-only; outputs must not alias inputs (except the
 *              in-place belief of kla_decode_step).  Base pointers must be
 *              16-byte aligned.
 *   dtype    : q, k, v, abar, pbar, r, y, dy and the input gradients share
 *              `dtype` (fp32 or bf16).  Beliefs and yvar are fp32 at the
 *              boundary.  The arithmetic is fp32 for bf16 inputs and fp64 for
 *              fp32 inputs (their 1e-4 gradients need fp64 adjoint carries).
 *   Shapes   : B, H >= 1, T >= 0, dk and dv each in {16, 32, 64, 128}.
 *   Domain   : abar in (0, 1], pbar >= 0, r > 0, lam0 > 0, all finite.  Not
 *              checked unless the environment sets KLA_CHECK=1, in which case
 *              a validation kernel runs first and the call synchronises and
 *              returns KLA_ERR_NUMERIC on a violation.
 *   Range    : the chunked path (bf16 inputs, see kla_forward) walks Theorem
 *              1's precision update over 32-token chunks in homogeneous
 *              coordinates: per key slot it carries, from the chunk start to
 *              token t, A_t = prod abar and z_t = prod (abar^2 + pbar lam_{t-1})
 *              (so lam_t = x_t / z_t and the product of the forget gates of
 *              Theorem 2 is P_t = A_t / z_t) and forms q P_t / lam_t and
 *              r k / P_t.  A_t, z_t and lam_t z_t must stay inside fp32's normal
 *              range over every chunk: roughly, the geometric mean of abar over
 *              32 consecutive tokens above 0.066 and that of abar^2 + pbar lam
 *              below 16 (abar = 0.03 over a whole chunk is outside: A underflows).
 *              Outside that range y and the gradients are not finite.  fp32
 *              inputs with dk and dv in {16, 32} take the same chunk walk in
 *              fp64, whose range is far wider (the geometric mean of abar over
 *              32 tokens above about 1e-9; abar = 1e-12 over a chunk is
 *              outside).  Under KLA_CHECK=1 the walks of the chunked forward
 *              and backward record whether any of those products was not
 *              finite, and the call synchronises and returns KLA_ERR_RANGE.
 *              The token-recurrent path (fp32 inputs at dk or dv of 64 or 128)
 *              and the per-channel entry points have no such limit.
 *   Empty    : with T == 0 the per-token pointers may be NULL; the final
 *              belief is then the initial one and its gradients pass through.
 *   Errors   : return codes only; on any error nothing has been enqueued
 *              (except KLA_ERR_HIP, reported when a launch fails).
 *   Threads  : no global mutable state (except the per-GPU workspace of
 *              kla_backward_noalloc, see there); calls are thread-safe.  Results
 *              are bitwise reproducible for a given descriptor.
 */
#ifndef KLA_H
#define KLA_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { KLA_F32 = 0, KLA_BF16 = 1 } kla_dtype;

typedef enum {
    KLA_OK = 0,
    KLA_ERR_NULL = 1,       /* a required pointer is NULL                         */
    KLA_ERR_SHAPE = 2,      /* unsupported or inconsistent sizes                  */
    KLA_ERR_DTYPE = 3,      /* unknown dtype                                      */
    KLA_ERR_ALIGN = 4,      /* a pointer is not 16-byte aligned                   */
    KLA_ERR_WORKSPACE = 5,  /* workspace missing or smaller than required         */
    KLA_ERR_NUMERIC = 6,    /* KLA_CHECK=1 found an input outside the domain      */
    KLA_ERR_HIP = 7,        /* a HIP launch or runtime call failed                */
    KLA_ERR_RANGE = 8       /* KLA_CHECK=1: a chunk's gate products left the walk's range */
} kla_status;

/* Problem descriptor: batch, sequence length, heads, key width, value width, dtype. */
typedef struct {
    int32_t B, T, H, dk, dv;
    int32_t dtype; /* kla_dtype */
} kla_desc;

/* Bytes of device workspace kla_forward needs (0 is possible). */
size_t kla_forward_workspace(const kla_desc* desc);

/* Bytes of the optional saved context that kla_forward can fill for
 * kla_backward: the precision and information state at every chunk start, and
 * the precision walk's state after the chunk's first 16 tokens (chunked layout:
 * bf16 inputs with dk >= 32 and dv >= 32, the shapes whose backward is
 * chunked); the precision and information state at every chunk start in fp64
 * (fp32 inputs with dk and dv in {16, 32}, the chunked fp64 path); else the
 * precision after every token and the information state before every 64th
 * token (fp32; fp64 for fp32 inputs, whose token-recurrent kernels accumulate
 * in fp64).  Both calls pick the layout by the same rule, so a context from
 * kla_forward always fits kla_backward. */
size_t kla_saved_bytes(const kla_desc* desc);

/* Bytes of device workspace kla_backward needs when it is given a saved
 * context (`with_saved` != 0) or must recompute one (`with_saved` == 0). */
size_t kla_backward_workspace(const kla_desc* desc, int with_saved);

/*
 * kla_forward -- the filter over a whole sequence (Algorithm 1: Moebius scan of
 * the precision, linear scan of the information state, query readout).
 *
 *   q, k, abar, pbar  [B, T, H, dk]  dtype      v [B, T, H, dv] dtype   r [B, T, H] dtype
 *   lam0 [B, H, dk] fp32, eta0 [B, H, dk, dv] fp32: initial belief; NULL means
 *        lam0 = 1 and eta0 = 0 respectively.
 *   y    [B, T, H, dv] dtype  (required)
 *   yvar [B, T, H] fp32 or NULL
 *   lamT [B, H, dk] fp32, etaT [B, H, dk, dv] fp32: final belief, each may be NULL.
 *   saved: NULL, or kla_saved_bytes(desc) bytes that kla_backward may later
 *        consume with the same inputs.
 *   ws / ws_bytes: workspace of at least kla_forward_workspace(desc) bytes.
 */
kla_status kla_forward(const kla_desc* desc,
                       const void* q, const void* k, const void* v,
                       const void* abar, const void* pbar, const void* r,
                       const float* lam0, const float* eta0,
                       void* y, float* yvar, float* lamT, float* etaT,
                       void* saved, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * kla_backward -- exact gradient of kla_forward's y, yvar, lamT and etaT with
 * respect to every input.
 *
 *   q .. r, lam0, eta0: exactly the forward inputs (NULL beliefs as in forward).
 *   saved: the context a kla_forward call with these inputs filled, or NULL
 *          (then it is recomputed inside the workspace).
 *   dy [B, T, H, dv] dtype (required); dyvar [B, T, H] fp32, the upstream
 *          gradient of the readout variance (the Monte Carlo readout of the
 *          paper's appendix, eq. nmll, samples through it), NULL meaning zero;
 *          dlamT [B, H, dk] and detaT [B, H, dk, dv] fp32 upstream gradients of
 *          the final belief, NULL meaning zero.
 *   dq, dk, dabar, dpbar [B, T, H, dk], dv [B, T, H, dv], dr [B, T, H]: dtype, required.
 *   dlam0 [B, H, dk], deta0 [B, H, dk, dv]: fp32 or NULL.
 *   ws / ws_bytes: at least kla_backward_workspace(desc, saved != NULL) bytes.
 */
kla_status kla_backward(const kla_desc* desc,
                        const void* q, const void* k, const void* v,
                        const void* abar, const void* pbar, const void* r,
                        const float* lam0, const float* eta0, const void* saved,
                        const void* dy, const float* dyvar, const float* dlamT, const float* detaT,
                        void* dq, void* dk, void* dv, void* dabar, void* dpbar, void* dr,
                        float* dlam0, float* deta0,
                        void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * kla_backward_noalloc -- kla_backward for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation).  Arguments and results are those of kla_backward, minus the
 * workspace: the library keeps one workspace of KLA_NOALLOC_SCRATCH_BYTES per GPU
 * for the life of the process (a file-scope device array; nothing is allocated,
 * freed or synchronised per call).
 *
 *   saved: required (T > 0): the context is read, never recomputed here.
 *   Returns KLA_ERR_WORKSPACE when kla_backward_workspace(desc, 1) exceeds
 *   KLA_NOALLOC_SCRATCH_BYTES (64 MiB: the LM-layer shape B8 T2048 H16 d128 bf16
 *   needs 8 MiB, the state-tracking shape B64 T512 H4 d32 fp32 256 bytes).
 *   Calls that overlap on one GPU share its workspace and race: order them on one
 *   stream.  With KLA_CHECK=1 the call synchronises, which graph capture forbids.
 */
#define KLA_NOALLOC_SCRATCH_BYTES (64u << 20)
kla_status kla_backward_noalloc(const kla_desc* desc,
                                const void* q, const void* k, const void* v,
                                const void* abar, const void* pbar, const void* r,
                                const float* lam0, const float* eta0, const void* saved,
                                const void* dy, const float* dyvar, const float* dlamT, const float* detaT,
                                void* dq, void* dk, void* dv, void* dabar, void* dpbar, void* dr,
                                float* dlam0, float* deta0, hipStream_t stream);

/*
 * kla_decode_step -- one recurrent token for S independent sequences (the
 * O(1)-per-token inference form of the filter): the same update as above for a
 * single t, applied IN PLACE to the carried belief.
 *
 *   q, k, abar, pbar [S, H, dk] dtype   v [S, H, dv] dtype   r [S, H] dtype
 *   lam [S, H, dk] fp32 and eta [S, H, dk, dv] fp32: read then overwritten.
 *   y [S, H, dv] dtype (required); yvar [S, H] fp32 or NULL.
 */
kla_status kla_decode_step(int32_t S, int32_t H, int32_t dk, int32_t dv, int32_t dtype,
                           const void* q, const void* k, const void* v,
                           const void* abar, const void* pbar, const void* r,
                           float* lam, float* eta, void* y, float* yvar, hipStream_t stream);

/*
 * OU gates (Sec. 4.1, eq. discretisation; Algorithm 1's OU-Discretisation
 * steps).  The layer can take its decay and process noise from time-invariant
 * parameters of an Ornstein-Uhlenbeck prior instead of per-token tensors: for
 * head h and key slot n, mean reversion a > 0, diffusion scale p and step size
 * delta > 0 give, for every token of every sequence,
 *
 *   abar[h,n] = exp(-a delta),   pbar[h,n] = p^2 (1 - exp(-2 a delta)) / (2 a)
 *
 * (formed in fp64 on the device, then rounded to fp32).  a, p, delta are
 * [H, dk] fp32 device arrays; every other argument is as in the entry point of
 * the same name above.  The gate gradients, summed over (b, t), reach the
 * parameters by the chain rule: da, dp, ddelta are [H, dk] fp32, overwritten.
 * Domain under KLA_CHECK=1: a > 0, delta > 0, p finite (and the rest as above).
 */

/* Workspace of kla_backward_ou: kla_backward_workspace plus the per-part token
 * sums of the two gate gradients. */
size_t kla_backward_ou_workspace(const kla_desc* desc, int with_saved);

/* kla_forward with OU gates; its saved context serves kla_backward_ou. */
kla_status kla_forward_ou(const kla_desc* desc,
                          const void* q, const void* k, const void* v,
                          const float* a, const float* p, const float* delta, const void* r,
                          const float* lam0, const float* eta0,
                          void* y, float* yvar, float* lamT, float* etaT,
                          void* saved, void* ws, size_t ws_bytes, hipStream_t stream);

/* kla_backward with OU gates: dq, dk, dv, dr (dtype), dlam0, deta0 as there, and
 * the parameter gradients da, dp, ddelta [H, dk] fp32 (required).
 * ws_bytes >= kla_backward_ou_workspace(desc, saved != NULL). */
kla_status kla_backward_ou(const kla_desc* desc,
                           const void* q, const void* k, const void* v,
                           const float* a, const float* p, const float* delta, const void* r,
                           const float* lam0, const float* eta0, const void* saved,
                           const void* dy, const float* dyvar, const float* dlamT, const float* detaT,
                           void* dq, void* dk, void* dv, float* da, float* dp, float* ddelta, void* dr,
                           float* dlam0, float* deta0,
                           void* ws, size_t ws_bytes, hipStream_t stream);

/* kla_decode_step with OU gates (a, p, delta [H, dk] fp32, shared by the S
 * sequences). */
kla_status kla_decode_step_ou(int32_t S, int32_t H, int32_t dk, int32_t dv, int32_t dtype,
                              const void* q, const void* k, const void* v,
                              const float* a, const float* p, const float* delta, const void* r,
                              float* lam, float* eta, void* y, float* yvar, hipStream_t stream);

/*
 * Per-channel precision (Algorithm 1 with Lambda^v of shape (B, T, 1, D)): one
 * observation precision per value channel, r_t[d], so that the precision and
 * the forget gate are dk x dv arrays per head (eqs. kla-prec-mat and
 * kla-mean-mat elementwise):
 *
 *   rho_t[n,d] = 1 / (abar_t[n]^2 + pbar_t[n] lam_{t-1}[n,d])
 *   lam_t[n,d] = rho_t[n,d] lam_{t-1}[n,d] + k_t[n]^2 r_t[d]
 *   H_t[n,d]   = abar_t[n] rho_t[n,d] H_{t-1}[n,d] + k_t[n] r_t[d] v_t[d]
 *   y_t[d]     = sum_n q_t[n] H_t[n,d] / lam_t[n,d]
 *   yvar_t[d]  = sum_n q_t[n]^2 / lam_t[n,d]
 *
 * Shapes differ from the entry points above only in: r, dr, dyvar [B, T, H, dv]
 * (decode: r [S, H, dv]) in dtype (dyvar fp32); lam0, lamT, dlamT, dlam0 and
 * decode lam [.., H, dk, dv] fp32; yvar [B, T, H, dv] fp32 (decode: [S, H, dv]).
 * The saved context holds the belief every 8 tokens (kla_saved_pc_bytes);
 * forward workspace: kla_forward_workspace, backward: kla_backward_pc_workspace.
 * Every other convention is as above.
 */
size_t kla_saved_pc_bytes(const kla_desc* desc);
size_t kla_backward_pc_workspace(const kla_desc* desc, int with_saved);

kla_status kla_forward_pc(const kla_desc* desc,
                          const void* q, const void* k, const void* v,
                          const void* abar, const void* pbar, const void* r,
                          const float* lam0, const float* eta0,
                          void* y, float* yvar, float* lamT, float* etaT,
                          void* saved, void* ws, size_t ws_bytes, hipStream_t stream);

/* Exact gradient of kla_forward_pc's y, yvar, lamT and etaT (arguments as in
 * kla_backward, with the per-channel shapes above). */
kla_status kla_backward_pc(const kla_desc* desc,
                           const void* q, const void* k, const void* v,
                           const void* abar, const void* pbar, const void* r,
                           const float* lam0, const float* eta0, const void* saved,
                           const void* dy, const float* dyvar, const float* dlamT, const float* detaT,
                           void* dq, void* dk, void* dv, void* dabar, void* dpbar, void* dr,
                           float* dlam0, float* deta0,
                           void* ws, size_t ws_bytes, hipStream_t stream);

kla_status kla_decode_step_pc(int32_t S, int32_t H, int32_t dk, int32_t dv, int32_t dtype,
                              const void* q, const void* k, const void* v,
                              const void* abar, const void* pbar, const void* r,
                              float* lam, float* eta, void* y, float* yvar, hipStream_t stream);

/*
 * Gates per (key slot, value channel): Algorithm 1 as written, with the decay and
 * process noise of shape (N, D) per head, time-invariant, from OU parameters
 * A, P, Delta : (N, D) by the exact discretisation (Sec. 4.1, eq. discretisation),
 * together with the per-channel observation precision above:
 *
 *   abar[h,n,d] = exp(-a delta),  pbar[h,n,d] = p^2 (1 - exp(-2 a delta)) / (2 a)
 *   rho_t[n,d] = 1 / (abar[n,d]^2 + pbar[n,d] lam_{t-1}[n,d]),  lam_t = rho_t lam_{t-1} + k^2 r_t[d]
 *   H_t[n,d]   = abar[n,d] rho_t[n,d] H_{t-1}[n,d] + k_t[n] r_t[d] v_t[d],  readouts as above
 *
 * a, p, delta, da, dp, ddelta are [H, dk, dv] fp32 (formed in the arithmetic type
 * of the per-channel kernels: fp64 for fp32 inputs, fp32 for bf16); every other
 * argument is as in the per-channel entry point of the same name.  The parameter
 * gradients are the per-token gate gradients summed over (b, t) and taken through
 * the discretisation in fp64.  Domain under KLA_CHECK=1: a > 0, delta > 0, p finite.
 */
size_t kla_backward_pc_ou_workspace(const kla_desc* desc, int with_saved);

kla_status kla_forward_pc_ou(const kla_desc* desc,
                             const void* q, const void* k, const void* v,
                             const float* a, const float* p, const float* delta, const void* r,
                             const float* lam0, const float* eta0,
                             void* y, float* yvar, float* lamT, float* etaT,
                             void* saved, void* ws, size_t ws_bytes, hipStream_t stream);

kla_status kla_backward_pc_ou(const kla_desc* desc,
                              const void* q, const void* k, const void* v,
                              const float* a, const float* p, const float* delta, const void* r,
                              const float* lam0, const float* eta0, const void* saved,
                              const void* dy, const float* dyvar, const float* dlamT, const float* detaT,
                              void* dq, void* dk, void* dv, float* da, float* dp, float* ddelta, void* dr,
                              float* dlam0, float* deta0,
                              void* ws, size_t ws_bytes, hipStream_t stream);

kla_status kla_decode_step_pc_ou(int32_t S, int32_t H, int32_t dk, int32_t dv, int32_t dtype,
                                 const void* q, const void* k, const void* v,
                                 const float* a, const float* p, const float* delta, const void* r,
                                 float* lam, float* eta, void* y, float* yvar, hipStream_t stream);

/*
 * Block scaffolding around the layer (the Mamba-style block of Sec. 4.4 and
 * Appendix A): a causal depthwise 1D convolution of kernel size 4 fused with
 * SiLU, QK-norm, and the SiLU output gate.  The paper fixes no details beyond
 * that; the definitions implemented are:
 *
 *   conv:  u[b,t,c] = silu(bias[c] + sum_{j<4} w[c,j] x[b,t-3+j,c])   (x = 0 before t = 0;
 *          tap 3 is the current token)                      x, u [B, T, C] dtype; w [C, 4] fp32;
 *                                                           bias [C] fp32 or NULL
 *   norm:  out = x / sqrt(mean_row(x^2) + eps) * w           rows of n in {16, 32, 64, 128}
 *          (one head's q or k of one token), w [n] fp32 shared by the rows; rstd [rows] fp32
 *          receives 1 / sqrt(mean(x^2) + eps) for the backward (may be NULL in the forward)
 *   gate:  out = y * silu(z)                                 y, z, out [n] dtype
 *
 * silu(s) = s / (1 + exp(-s)).  C must be a multiple of 8 (bf16) or 4 (fp32),
 * as must the gate's n; pointers 16-byte aligned.  Weight gradients (dw,
 * dbias) are overwritten and summed over (b, t) or rows in a fixed order through
 * the workspace.  Every other convention of this header applies.
 */
size_t kla_conv_silu_workspace(int32_t B, int32_t T, int32_t C);
kla_status kla_conv_silu_forward(int32_t B, int32_t T, int32_t C, int32_t dtype, const void* x, const float* w,
                                 const float* bias, void* u, hipStream_t stream);
kla_status kla_conv_silu_backward(int32_t B, int32_t T, int32_t C, int32_t dtype, const void* x, const float* w,
                                  const float* bias, const void* du, void* dx, float* dw, float* dbias,
                                  void* ws, size_t ws_bytes, hipStream_t stream);

size_t kla_qk_norm_workspace(int32_t n);
kla_status kla_qk_norm_forward(int64_t rows, int32_t n, int32_t dtype, const void* x, const float* w, float eps,
                               void* out, float* rstd, hipStream_t stream);
kla_status kla_qk_norm_backward(int64_t rows, int32_t n, int32_t dtype, const void* x, const float* w,
                                const float* rstd, const void* dout, void* dx, float* dw,
                                void* ws, size_t ws_bytes, hipStream_t stream);

kla_status kla_gate_forward(int64_t n, int32_t dtype, const void* y, const void* z, void* out, hipStream_t stream);
kla_status kla_gate_backward(int64_t n, int32_t dtype, const void* y, const void* z, const void* dout,
                             void* dy, void* dz, hipStream_t stream);

/*
 * Monte Carlo readout of KLA+ (the log-marginal-likelihood training loss of the
 * paper's appendix, eqs. nmll_integral and nmll_logsumexp).  The readout of
 * channel d is Gaussian under the posterior, with mean ymu = y of kla_forward and
 * variance yvar (one per token and head, the slots being independent a
 * posteriori), so S draws are
 *
 *   ys[s, b, t, h, d] = ymu[b, t, h, d] + sqrt(yvar[b, t, h]) eps[s, b, t, h, d]
 *
 * with eps standard normal, drawn by the counter-based generator Philox4x64-10
 * (Salmon et al., "Parallel random numbers: as easy as 1, 2, 3", SC 2011) and the
 * Box-Muller transform: for the flat index e of [S, B, T, H, dv], Philox block
 * j = e / 8 (counter (j, 0, 0, 0), key (seed, 0)) gives four 64-bit words, i.e. eight
 * 32-bit halves u_0..u_7 (low half first); each pair gives
 * r = sqrt(-2 ln(((u_2p >> 8) + 1) 2^-24)), a = (u_2p+1 >> 8) 2^-23 and the normals
 * eps_2p = r cos(pi a), eps_2p+1 = r sin(pi a); element e takes eps_(e mod 8).  The
 * integer stream is exact; ln, sqrt, cos and sin are the GPU's hardware functions
 * (within a few ulp, or 2^-20 absolute for cos / sin), so eps agrees with the formula
 * to about 1e-6.  Nothing is stored between the draws and their backward, which
 * draws the same eps again.
 *
 * The decoder p(o | y) belongs to the model; the loss takes its log-probabilities
 * of the target tokens, logp [S, n] fp32, and returns per token
 *   nll[i] = -logsumexp_s(logp[s, i]) + log S        (cross-entropy when S = 1).
 *
 *   ymu, dymu [B, T, H, dv] and ys, dys [S, B, T, H, dv]: dtype; yvar, dyvar [B, T, H]
 *   fp32 (yvar > 0).  dv in {16, 32, 64, 128}.  The backward of the draws returns
 *   dymu = sum_s dys and dyvar = sum_{s,d} dys eps / (2 sqrt(yvar)); that of the loss
 *   dlogp[s, i] = -dnll[i] softmax_s(logp[., i]).  Every output is overwritten.
 */
kla_status kla_mc_sample(int32_t S, int32_t B, int32_t T, int32_t H, int32_t dv, int32_t dtype, uint64_t seed,
                         const void* ymu, const float* yvar, void* ys, hipStream_t stream);
kla_status kla_mc_sample_backward(int32_t S, int32_t B, int32_t T, int32_t H, int32_t dv, int32_t dtype,
                                  uint64_t seed, const float* yvar, const void* dys, void* dymu, float* dyvar,
                                  hipStream_t stream);
kla_status kla_mc_nll(int32_t S, int64_t n, const float* logp, float* nll, hipStream_t stream);
kla_status kla_mc_nll_backward(int32_t S, int64_t n, const float* logp, const float* dnll, float* dlogp,
                               hipStream_t stream);

/* Static, human-readable name of a status code. */
const char* kla_status_string(kla_status status);

#ifdef __cplusplus
}
#endif

#endif /* KLA_H */
