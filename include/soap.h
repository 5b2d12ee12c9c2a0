/*
 * soap.h — C ABI of the MI355X (gfx950) SOAP optimizer-step library.
 *
 * The library performs the per-weight-matrix SOAP update of "SOAP, Muon, and
 * Beyond: Pushing LLM Pretraining Scales" (Algorithm 2, KL-SOAP listing, with
 * the plain-EMA Kronecker factors of the Section 2 Shampoo primer, eigenbasis
 * refresh every step (F = 1, hyperparameter table of Section 5.4) and the
 * real-time refresh of Section 5.4.2).  One call of soap_step does, in order:
 *
 *   1. L <- b2 L + (1-b2) G G^T,   R <- b2 R + (1-b2) G^T G          (factor EMA)
 *   2. Q_L <- QR(L Q_L).Q,  Q_R <- QR(R Q_R).Q, diag(R-factor) >= 0  (refresh)
 *   3. M <- b1 M + (1-b1) G;  G' = Q_L^T G Q_R;  M' = Q_L^T M Q_R    (rotate in)
 *   4. V <- b2 V + (1-b2) G'^2;  N = (M'/c1) / (sqrt(V/c2) + eps)    (Adam)
 *   5. W <- (1 - lr wd) W - lr Q_L N Q_R^T                            (rotate out)
 *
 * with c1 = 1 - b1^t and c2 = 1 - b2^t (c1 = c2 = 1 under
 * SOAP_FLAG_NO_BIAS_CORRECTION).  M is the first moment in weight space; by
 * linearity and orthogonality of the Q this equals Algorithm 2's
 * eigenbasis-resident m when the basis is refreshed every step.  V is indexed
 * by (column of Q_L, column of Q_R).
 *
 * Conventions for every entry point:
 *  - All matrices are fp32, row-major and dense: the leading dimension is the
 *    number of columns.  A weight is m x n ("in" x "out" in Algorithm 2):
 *    param, grad, M, V are m x n; L, Q_L are m x m; R, Q_R are n x n.
 *    Batched tensors are contiguous [batch][rows][cols].
 *  - Matrix pointers are DEVICE pointers (hipMalloc or torch device memory),
 *    16-byte aligned.  The caller owns every buffer, including the workspace;
 *    the library never allocates or frees device memory.  It keeps no
 *    optimizer state between calls.  It does keep, until the process ends:
 *    the thread-local error string; per device, three internal streams of
 *    default priority (created on first use: the m x m factor's chain and
 *    the block factorizations of both QRs run on them, forked from and
 *    joined back into the caller's stream with events); per host thread and
 *    device, seven HIP events for the step's forks and joins, and per host
 *    thread a pool of up to 4096 events for those of the QR; per device, the
 *    result of one occupancy query (how many QR block workgroups the device
 *    holds at once); and, while soap_timing_enable(1) is in force, timing
 *    events.
 *  - Work is enqueued on `stream` (0 = the null stream) and the call returns
 *    without synchronising.  Validation happens on the host before anything is
 *    enqueued: on failure nothing is enqueued, a negative soap_status is
 *    returned and soap_last_error() describes it.  A HIP launch error is
 *    reported as SOAP_ERR_HIP; a device fault surfaces at the caller's next
 *    synchronisation.  NaN/Inf in the inputs propagate and are not checked.
 *  - Calls on different streams are safe when their buffers and workspaces are
 *    disjoint (several steps running at once may make a QR give up and keep
 *    its old basis: see soap_workspace_status).  No C++ exception crosses
 *    this boundary.
 *  - Every dimension must be in [1, SOAP_MAX_DIM].
 */
#ifndef SOAP_MI355X_H
#define SOAP_MI355X_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SOAP_OK = 0,
  SOAP_ERR_NULL = -1,       /* a required pointer is NULL                       */
  SOAP_ERR_SHAPE = -2,      /* batch/m/n outside [1, SOAP_MAX_DIM] or overflow   */
  SOAP_ERR_HPARAM = -3,     /* beta outside [0,1), eps/lr/wd negative or not finite,
                               step < 1, unknown flag bits                       */
  SOAP_ERR_WORKSPACE = -4,  /* workspace smaller than the *_workspace_bytes value */
  SOAP_ERR_ALIGN = -5,      /* a pointer is not 16-byte aligned                  */
  SOAP_ERR_ALIAS = -6,      /* grad overlaps a buffer the call writes, or two
                               written buffers overlap                           */
  SOAP_ERR_HIP = -7,        /* a HIP runtime call failed                         */
  SOAP_ERR_QR_GAVE_UP = -8  /* soap_workspace_status: a QR's bounded wait gave up  */
} soap_status;

/* Step flags (bitwise or):
 *  SOAP_FLAG_NO_BIAS_CORRECTION  c1 = c2 = 1 (Algorithm 2 as printed).
 *  SOAP_FLAG_SKIP_REFRESH        keep Q_L, Q_R: no power product, no QR this
 *                                step (Algorithm 2 refreshes when t mod F = 0;
 *                                the caller sets this flag on the other steps).
 *                                The factors and the Adam part are updated.
 *  SOAP_FLAG_STALE_REFRESH       refresh from the factors as they were before
 *                                this step's gradient was added: the lagging
 *                                preconditioner of Section 5.4.1, which the
 *                                real-time refresh of Section 5.4.2 replaces
 *                                (an ablation; no effect with SKIP_REFRESH). */
enum {
  SOAP_FLAG_NO_BIAS_CORRECTION = 1u << 0,
  SOAP_FLAG_SKIP_REFRESH = 1u << 1,
  SOAP_FLAG_STALE_REFRESH = 1u << 2
};

#define SOAP_MAX_DIM 16384

/* Bits of a step's status word (soap_workspace_status): the QR of the m x m
 * factor (or soap_qr_f32's matrix) / of the n x n factor gave up. */
enum { SOAP_STATUS_QR_L = 1u << 0, SOAP_STATUS_QR_R = 1u << 1 };

/* Bytes of device workspace soap_step / soap_step_batched need for `batch`
 * matrices of shape m x n (batch = 1 for soap_step).  Returns 0 for an invalid
 * shape.  The workspace holds the power products L Q_L and R Q_R, the QR
 * block reflectors and the rotation intermediates; its contents need not be
 * initialised and are garbage after the call. */
size_t soap_workspace_bytes(int64_t batch, int64_t m, int64_t n);

/* Initial optimizer state (the paper gives none; identity bases keep the
 * first power product nonsingular): L = R = Q_L = Q_R = I, M = V = 0, for
 * `batch` contiguous matrices.  Any of the six pointers may be NULL to skip
 * that tensor. */
int soap_init_state(int64_t batch, int64_t m, int64_t n, float *L, float *R, float *Q_L,
                    float *Q_R, float *M, float *V, hipStream_t stream);

/* One SOAP step on one m x n weight (Algorithm 2, F = 1).  `param`, L, R,
 * Q_L, Q_R, M, V are updated in place; `grad` is read only.  L and R are read
 * from their lower triangle and written fully symmetric.  `step` is the
 * 1-based t of this update.  beta1, beta2 in [0,1); eps, lr, weight_decay
 * finite and >= 0; flags is a combination of the SOAP_FLAG_* bits. */
int soap_step(float *param, const float *grad, float *L, float *R, float *Q_L, float *Q_R,
              float *M, float *V, int64_t m, int64_t n, float beta1, float beta2, float eps,
              float lr, float weight_decay, int64_t step, uint32_t flags, void *workspace,
              size_t workspace_bytes, hipStream_t stream);

/* soap_step on `batch` same-shape matrices in one call (e.g. the experts of an
 * MoE layer).  Every tensor is contiguous [batch][..][..] in the layout of
 * soap_step; the matrices are independent and share the hyperparameters. */
int soap_step_batched(int64_t batch, float *param, const float *grad, float *L, float *R,
                      float *Q_L, float *Q_R, float *M, float *V, int64_t m, int64_t n,
                      float beta1, float beta2, float eps, float lr, float weight_decay,
                      int64_t step, uint32_t flags, void *workspace, size_t workspace_bytes,
                      hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): soap_step
 * without a workspace argument.  The library's own scratch, a static device
 * array of SOAP_NOALLOC_MAX_WORKSPACE_BYTES per GPU (held until the process
 * ends), takes the workspace's place; the call allocates and frees nothing.
 * Shapes whose soap_workspace_bytes(1, m, n) exceed it are rejected with
 * SOAP_ERR_WORKSPACE (up to 2048 x 2048 fits).  Arguments, results and errors
 * otherwise as for soap_step.  Every call on one GPU shares that GPU's
 * scratch: calls that overlap on one GPU (different streams, or host threads
 * without ordering) race and must not be issued.  The step clears what it
 * needs cleared; the scratch keeps the last call's contents.  A QR give-up
 * keeps the basis as in soap_step, but its status word lives in the scratch
 * and is not readable through soap_workspace_status.  The first call on a
 * device and host thread creates the library's streams and events (host-side
 * objects, no device memory). */
#define SOAP_NOALLOC_MAX_WORKSPACE_BYTES ((size_t)256 << 20)
int soap_step_noalloc(float *param, const float *grad, float *L, float *R, float *Q_L,
                      float *Q_R, float *M, float *V, int64_t m, int64_t n, float beta1,
                      float beta2, float eps, float lr, float weight_decay, int64_t step,
                      uint32_t flags, hipStream_t stream);

/* ---- KL-SOAP (the variant the paper recommends: Sections 5.4.3 and 7) ----
 * One KL-SOAP step replaces step 1 of soap_step by the KL-Shampoo accumulation
 * of Algorithm 2.  With the bases and factors of the previous step:
 *
 *   lambda_L = diag(Q_L^T L Q_L),   lambda_R = diag(Q_R^T R Q_R)
 *   L <- bk L + (1-bk)/n  G Q_R diag(1/(lambda_R+eps)) Q_R^T G^T
 *   R <- bk R + (1-bk)/m  G^T Q_L diag(1/(lambda_L+eps)) Q_L^T G
 *
 * (bk = beta_kron; n = "out", m = "in").  Readings of Algorithm 2: bk
 * multiplies the old factor, as every EMA of the Section 2 primer does; the
 * exponent on (lambda + eps) is -1, the inverse that the KL-Shampoo rule of
 * Appendix A.3 uses; the estimates act in the basis that measured them, so
 * the weight is the other factor's inverse as that basis diagonalises it.
 * Steps 2-5 are those of soap_step; eps serves both the eigenvalue floor and
 * Adam (hyperparameter table of Section 5.4).  Arguments, layout, ownership
 * and errors as for soap_step, except that L and R must hold both triangles
 * on entry (the estimates read the whole stored factor; every step leaves
 * them symmetric); beta_kron must lie in [0, 1).  The workspace is larger
 * than soap_step's (one more m x n buffer and the estimates). */
size_t soap_kl_workspace_bytes(int64_t batch, int64_t m, int64_t n);
int soap_kl_step(float *param, const float *grad, float *L, float *R, float *Q_L, float *Q_R,
                 float *M, float *V, int64_t m, int64_t n, float beta1, float beta2,
                 float beta_kron, float eps, float lr, float weight_decay, int64_t step,
                 uint32_t flags, void *workspace, size_t workspace_bytes, hipStream_t stream);
int soap_kl_step_batched(int64_t batch, float *param, const float *grad, float *L, float *R,
                         float *Q_L, float *Q_R, float *M, float *V, int64_t m, int64_t n,
                         float beta1, float beta2, float beta_kron, float eps, float lr,
                         float weight_decay, int64_t step, uint32_t flags, void *workspace,
                         size_t workspace_bytes, hipStream_t stream);

/* ---- Muon (Algorithm 1, the paper's second optimizer) ----
 * One Muon step on an m x n weight ("in" x "out"):
 *
 *   M <- beta1 M + (1 - beta1) G
 *   X_0 = M / max(||M||_F, eps)
 *   for i = 1..n_iters:  A = X X^T,  B = b_i A + c_i A^2,  X <- a_i X + B X
 *   W <- (1 - lr wd) W - lr sqrt(max(m, n)) X_n
 *
 * The polynomial acts on singular values only, so the library forms the Gram
 * matrix on the smaller side (X^T X and X <- a X + X B when m > n); the
 * result is the same iterate.  coeffs is a HOST array of 3 n_iters floats
 * (a_1, b_1, c_1, a_2, ...): the paper uses the PolarExpress schedule with
 * n = 16 (hyperparameter table of Section 5.3) without printing it, so the
 * caller supplies the schedule.  param, grad, M are device pointers in the
 * layout of soap_step (grad read only, param and M updated); beta1 in [0, 1),
 * lr and weight_decay finite and >= 0, eps finite and > 0, n_iters in
 * [0, 1024].  flags 0: the products run in fp32 on the matrix cores.
 * flags SOAP_MUON_BF16: the Newton-Schulz iterations run in bfloat16, the
 * paper's precision for them (its discussion of orthogonalisation accuracy
 * in the conclusion): X_0, every A, B and X are bfloat16, each product
 * accumulated in fp32 on the bf16 matrix cores and rounded once to nearest
 * (ties to even); the momentum, the norm and the weight update stay fp32.
 * It needs m and n multiples of 8 (SOAP_ERR_SHAPE otherwise).
 * Ownership, streams and errors as for soap_step. */
enum { SOAP_MUON_BF16 = 1u << 0 };
size_t soap_muon_workspace_bytes(int64_t batch, int64_t m, int64_t n);
int soap_muon_step(float *param, const float *grad, float *M, int64_t m, int64_t n, float beta1,
                   float lr, float weight_decay, float eps, const float *coeffs, int64_t n_iters,
                   uint32_t flags, void *workspace, size_t workspace_bytes, hipStream_t stream);
int soap_muon_step_batched(int64_t batch, float *param, const float *grad, float *M, int64_t m,
                           int64_t n, float beta1, float lr, float weight_decay, float eps,
                           const float *coeffs, int64_t n_iters, uint32_t flags, void *workspace,
                           size_t workspace_bytes, hipStream_t stream);

/* Description of the last failure on the calling thread ("" after success).
 * Valid until the next call on the same thread. */
const char *soap_last_error(void);

/* Device-side outcome of the last step (soap_step, soap_kl_step and their
 * batched forms) or soap_qr_f32 call enqueued with `workspace`.
 *
 * The QR factors each 128-column block with one launch whose workgroups must
 * all be resident at once (they exchange partial sums through memory); the
 * library sizes these launches from an occupancy query, but other work on the
 * GPU (another process, communication kernels that wait for peers, concurrent
 * steps on other streams) can hold the compute units they need.  Their waits
 * are therefore bounded: if one gives up, that factor's factorization is
 * marked failed, its eigenbasis (Q_L or Q_R; soap_qr_f32's Q) is LEFT AS IT
 * WAS ON ENTRY, and the rest of the step runs with it, exactly as a step with
 * SOAP_FLAG_SKIP_REFRESH would for that side.  The step sets the bit of that
 * side in the status word at offset 0 of its workspace; every step clears the
 * word when it starts.
 *
 * This call waits for `stream` (a host synchronisation), reads the word into
 * *status (if not NULL) and returns SOAP_OK when it is 0, SOAP_ERR_QR_GAVE_UP
 * when a SOAP_STATUS_QR_* bit is set (soap_last_error() names the side), or
 * SOAP_ERR_WORKSPACE when it holds other bits (not such a workspace). */
int soap_workspace_status(const void *workspace, uint32_t *status, hipStream_t stream);

/* Byte offset, inside the workspace of soap_step / soap_step_batched /
 * soap_kl_step(_batched), of the eigenbasis update N = (M'/c1) /
 * (sqrt(V/c2) + eps) that the last step wrote there (fp32, [batch][m][n]);
 * valid once that step's stream has been synchronised and until the next call
 * with the workspace.  For diagnostics; 0 for an invalid shape. */
size_t soap_workspace_update_offset(int64_t batch, int64_t m, int64_t n);

/* TEST HOOK, not for production use.  Every later QR (of a step or of
 * soap_qr_f32) whose SOAP_STATUS_QR_* bit is in `mask` starts with the abort
 * flags of its resident block factorizations raised, so that each of their
 * bounded waits gives up at once and every kernel still exits normally: the
 * give-up path above, on demand.  mask = 0 restores normal operation.  Only
 * QRs that take the resident block path are affected (matrices whose
 * factorization runs in more than one workgroup per block; batches that the
 * library factors with its panel path have no waits).  Returns
 * SOAP_ERR_HPARAM for other bits. */
int soap_test_force_qr_give_up(uint32_t mask);

/* ---- stage entry points (used by the tests to check each kernel alone) ---- */

/* Eigenbasis refresh QR (Algorithm 2, "QR(.).Q"): A = Q Rf for one n x n
 * matrix, with diag(Rf) >= 0, by blocked Householder.  A is read only; Q (n x n)
 * receives the Q factor; Rf (n x n, may be NULL) the triangular factor with its
 * strict lower part zeroed.  If the factorization gives up (see
 * soap_workspace_status, bit SOAP_STATUS_QR_L) Q is left as it was on entry
 * and Rf is undefined. */
size_t soap_qr_workspace_bytes(int64_t n);
int soap_qr_f32(int64_t n, const float *A, float *Q, float *Rf, void *workspace,
                size_t workspace_bytes, hipStream_t stream);

/* The MFMA GEMM used for every product of the step:
 * C = alpha * op(A) op(B) + beta * C, op(X) = X or X^T (trans != 0),
 * op(A) M x K, op(B) K x N, row-major with leading dimensions lda, ldb, ldc.
 * When beta == 0, C is not read. */
int soap_gemm_f32(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K, float alpha,
                  const float *A, int64_t lda, const float *B, int64_t ldb, float beta,
                  float *C, int64_t ldc, hipStream_t stream);

/* Factor EMA (Section 2 primer): F <- beta F + (1 - beta) X X^T for X = G
 * (trans = 0, F is m x m) or X = G^T (trans = 1, F is n x n), G m x n.  Only
 * the lower triangle of X X^T is computed; F is written fully symmetric. */
int soap_factor_ema_f32(int trans, int64_t m, int64_t n, const float *G, float *F, float beta,
                        hipStream_t stream);

/* KL-Shampoo accumulation alone (step 1 of soap_kl_step) for one m x n
 * gradient G: L (m x m) and R (n x n) are read whole (both triangles; the
 * new term is added to the lower triangle) and written fully symmetric; Q_L,
 * Q_R (the previous step's bases) are read only.  lam_L (m floats) and lam_R (n floats), if not NULL, receive the
 * eigenvalue estimates diag(Q_L^T L Q_L), diag(Q_R^T R Q_R) of the factors
 * as they were on entry.  All pointers are device pointers; the workspace
 * (soap_kl_factors_workspace_bytes) is the caller's. */
size_t soap_kl_factors_workspace_bytes(int64_t m, int64_t n);
int soap_kl_factors_f32(int64_t m, int64_t n, const float *G, float *L, float *R,
                        const float *Q_L, const float *Q_R, float beta_kron, float eps,
                        float *lam_L, float *lam_R, void *workspace, size_t workspace_bytes,
                        hipStream_t stream);
/* ---- measurement ---- */

/* When enabled, every stage of soap_step / soap_step_batched records a pair
 * of HIP events on the call's stream.  soap_timing_collect synchronises on
 * them and adds their durations to per-stage totals; soap_timing_reset clears
 * the totals.  Stage ids are 0 .. soap_timing_num_stages()-1. */
int soap_timing_enable(int enable);
int soap_timing_num_stages(void);
const char *soap_timing_stage_name(int stage);
int soap_timing_collect(void);
int soap_timing_reset(void);
/* Totals since the last reset: milliseconds, launches, and the algorithmic
 * flops of those launches (one triangle for the factor EMA, 2 m n k for a
 * product, (4/3) n^3 + (4/3) n^3 for a QR with its explicit Q). */
int soap_timing_get(int stage, double *total_ms, int64_t *launches, double *flops);

#ifdef __cplusplus
}
#endif

#endif /* SOAP_MI355X_H */
