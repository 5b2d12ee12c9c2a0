// Internal declarations shared by the host orchestration and the kernel files
// of the SOAP library.  Nothing here is part of the public C ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <functional>

#include <cstddef>
#include <cstdint>

namespace soap {

// ----------------------------------------------------------------- GEMM
// op(A) is M x K, op(B) is K x N, C is M x N; all row-major.
//   trans_a = 0: op(A)[i][k] = A[i*lda + k]      trans_a = 1: op(A)[i][k] = A[k*lda + i]
//   trans_b = 0: op(B)[k][j] = B[k*ldb + j]      trans_b = 1: op(B)[k][j] = B[j*ldb + k]
// A batch of independent products is laid out with element strides sA, sB, sC.
struct GemmDesc {
  int trans_a = 0, trans_b = 0;
  int64_t M = 0, N = 0, K = 0;
  const float *A = nullptr;
  int64_t lda = 0, sA = 0;
  const float *B = nullptr;
  int64_t ldb = 0, sB = 0;
  float *C = nullptr;
  int64_t ldc = 0, sC = 0;
  float alpha = 1.f, beta = 0.f;
  int64_t batch = 1;
  // Split-K: when splitk > 1 the K range is cut into `splitk` slices whose
  // partial products go to `part` (batch * splitk * M * N floats) and are then
  // summed in a fixed order by a second kernel.
  int splitk = 1;
  float *part = nullptr;
  // With split-K: leave the partials in `part` for the caller to reduce
  // (C is not written).
  bool partials_only = false;
  // Distinct kernel symbol for profiling (0 = shared GEMM; 1, 2 = the power
  // products L Q_L and R Q_R), so that a trace can attribute time per stage.
  int tag = 0;
  // If > 0, at most this many workgroups (rounded down to a multiple of 8)
  // are launched and each loops over tiles: the product then holds only part
  // of the compute units, leaving the rest to concurrent work.
  int max_wg = 0;
  // If set, the product of batch entry b is not computed (C, and the split-K
  // partials, are left untouched) when skip[b * sSkip] != 0 at launch time.
  const unsigned *skip = nullptr;
  int64_t sSkip = 0;
};

// A split-K factor that gives at least ~2 workgroups per CU for a product with
// the given tile count and K, capped by the partial buffer `max_split`.
int choose_splitk(int64_t M, int64_t N, int64_t K, int64_t batch, int max_split);

// C = alpha op(A) op(B) + beta C (C not read when beta == 0).
hipError_t launch_gemm(const GemmDesc &d, hipStream_t s);

// Symmetric rank-k EMA on one triangle:  C <- beta C + alpha op(A) op(B) where
// op(A) op(B) is symmetric (op(B) = op(A)^T, or op(A) D op(A)^T with the
// diagonal scaling folded into B), only tiles on or below the diagonal are
// computed and each result is stored at (i,j) and (j,i).  C is read from its
// lower triangle.  max_wg caps it like a GEMM for the layouts (0, 1) and (1, 0).
hipError_t launch_syrk_ema(const GemmDesc &d, hipStream_t s);

// Fused second rotation + Adam in the eigenbasis.  op(A) (trans_a = 0,
// d.M = 2 m rows) holds T_G and T_M interleaved by rows: row 2i is row i of
// T_G, row 2i+1 row i of T_M.  With op(B) = Q_R one product gives
//   G' = T_G Q_R,  M' = T_M Q_R  (rows 2i, 2i+1 of the result), and the
// epilogue does  V <- b2 V + (1-b2) G'^2,  Nout = (M'/c1) / (sqrt(V/c2) + eps)
// on the m x n outputs, which use the leading dimension and batch stride of
// C in the descriptor.  d.M odd or trans_a != 0: hipErrorInvalidValue.
struct AdamEpi {
  float *V = nullptr;
  float *Nout = nullptr;
  float b2 = 0.f, c1 = 1.f, c2 = 1.f, eps = 0.f;
};
hipError_t launch_gemm_adam(const GemmDesc &d, const AdamEpi &e, hipStream_t s);

// ------------------------------------------------------- elementwise
// M <- b1 M + (1-b1) G over `count` floats.
hipError_t launch_momentum(float *M, const float *G, int64_t count, float b1, hipStream_t s);
// Fill `batch` row-major r x c matrices (element stride sbatch between them)
// with diag_value on the diagonal and 0 elsewhere.
hipError_t launch_fill_diag(float *X, int64_t batch, int64_t r, int64_t c, int64_t sbatch,
                            float diag_value, hipStream_t s);
// Zero `count` 32-bit words.
hipError_t launch_zero_u32(uint32_t *p, int64_t count, hipStream_t s);
// Copy `count` floats.
hipError_t launch_copy(float *dst, const float *src, int64_t count, hipStream_t s);

// ------------------------------------------------------------ KL factors
// lambda[b][k] = sum_i X[b][k][i] Q[b][i][k] for `batch` d x d row-major X, Q
// (element stride d*d): the diagonal of X Q, i.e. diag(Q^T F Q) when
// X = Q^T F.  `part` holds diag_partial_floats(batch, d) floats of partial sums.
int diag_chunks(int64_t batch, int64_t d);
size_t diag_partial_floats(int64_t batch, int64_t d);
hipError_t launch_diag_of_product(const float *X, const float *Q, int64_t batch, int64_t d,
                                  float *part, float *lam, hipStream_t s);
// Z = Y diag(1/(lambda+eps)) (by_row = 0; lambda has `cols` entries per
// matrix) or Z = diag(1/(lambda+eps)) Y (by_row = 1; `rows` entries), for
// `batch` contiguous rows x cols matrices.
hipError_t launch_kl_scale(const float *Y, float *Z, const float *lam, int64_t batch,
                           int64_t rows, int64_t cols, int by_row, float eps, hipStream_t s);

// ----------------------------------------------------------------- Muon
// X = M / max(||M||_F, eps) for `batch` contiguous matrices of `count` floats;
// `part` holds muon_norm_partial_bytes(batch) bytes, inv receives the batch
// factors 1 / max(||M||_F, eps).
size_t muon_norm_partial_bytes(int64_t batch);
hipError_t launch_muon_normalise(const float *M, float *X, int64_t batch, int64_t count,
                                 float eps, double *part, float *inv, hipStream_t s);
// W <- alpha W + beta X over `count` floats.
hipError_t launch_axpby(float *W, const float *X, int64_t count, float alpha, float beta,
                        hipStream_t s);
// inv[b] = 1 / max(||M_b||_F, eps) only (norm in double, fixed order).
hipError_t launch_muon_norm_inv(const float *M, int64_t batch, int64_t count, float eps,
                                double *part, float *inv, hipStream_t s);

// ---------------------------------------------------- bfloat16 products
// C = round_bf16(alpha * P Q^T + beta * D) for `batch` products (element
// strides sP, sQ, sD, sC, sCt), bfloat16 stored as uint16_t, row-major:
// P is M x K (rows k-contiguous, leading dimension ldp), Q is N x K, D and C
// are M x N.  D may be null (beta ignored).  syrk: M == N, P == Q, only the
// tiles on or below the diagonal are computed and C is written mirrored.
// Ct, if not null, receives C^T (N x M, leading dimension ldct).  Needs
// K, ldp, ldq multiples of 8, ldct a multiple of 4 and 16-byte aligned
// P, Q (else hipErrorInvalidValue).  The sum runs in fp32 on the matrix
// cores; C is rounded once, to nearest with ties to even.
struct BfGemmDesc {
  int64_t M = 0, N = 0, K = 0;
  const uint16_t *P = nullptr;
  int64_t ldp = 0, sP = 0;
  const uint16_t *Q = nullptr;
  int64_t ldq = 0, sQ = 0;
  const uint16_t *D = nullptr;
  int64_t ldd = 0, sD = 0;
  uint16_t *C = nullptr;
  int64_t ldc = 0, sC = 0;
  uint16_t *Ct = nullptr;
  int64_t ldct = 0, sCt = 0;
  float alpha = 1.f, beta = 0.f;
  int64_t batch = 1;
  bool syrk = false;
};
hipError_t launch_gemm_bf16_nt(const BfGemmDesc &d, hipStream_t s);
// Xo = round_bf16(inv[b] * S_b) (rows x cols; S_b read transposed, i.e. as a
// cols x rows fp32 matrix, when trans) and Xt = Xo^T, per batch entry b.
hipError_t launch_bf16_scale_both(const float *S, int64_t batch, int64_t rows, int64_t cols,
                                  bool trans, const float *inv, uint16_t *Xo, uint16_t *Xt,
                                  hipStream_t s);
// W <- alpha W + beta X over `count` values (X bfloat16).
hipError_t launch_axpby_bf16(float *W, const uint16_t *X, int64_t count, float alpha, float beta,
                             hipStream_t s);

// ----------------------------------------------------------------- QR
// Blocked Householder QR of `batch` n x n matrices A, each given TRANSPOSED:
// At = A^T row-major (element stride n*n between matrices).  At is overwritten
// by the factorization; the Q factor with non-negative diag(R) is written
// row-major to Q.  If Rf is non-null the triangular factor is written there
// (row-major, strict lower part zero).  Work is ordered on stream s; the
// block factorizations run on stream sp and the T matrices of block pairs on
// stream st (both joined back into s with events; st may equal sp).
// If q_free is not null, s waits for it before Q is first written (Q may
// still be read by work on other streams until then).  If at_mid is set it
// is called once, when the host loop over the outer blocks reaches block
// mid_frac * (number of outer blocks) (or at the end of the factorization),
// right after recording `mid` on s (if not null), so that the caller can
// enqueue work that waits for that event: the factorization's later blocks
// leave most of the GPU idle.
//
// Resident block factorizations wait for each other's partial sums with
// bounded waits.  If a wait gives up (the launch's workgroups could not all
// be resident, e.g. because other work held the compute units), the matrix's
// factorization is marked failed: `status_bit` is or-ed into *status (if
// status is not null), and Q (and Rf) of that matrix are left as they were
// on entry -- the Q formation is skipped for it.  qr_force_give_up(mask)
// makes every later call whose status_bit is in `mask` start with its
// matrices' abort flags raised (a test hook: every bounded wait then ends at
// once and the kernels exit normally).
//
// With `split`, the batch is two factors' matrices of the same order (batch
// = 2 half): Q is then a contiguous buffer of the whole batch that the call
// uses as its own, and at the end entries [0, half) are copied to QA and
// [half, 2 half) to QB; a failed entry is not copied and or-s bitA or bitB
// (by its half) into *status (status_bit is not used; Rf must be null).
struct QrSplitOut {
  float *QA;
  float *QB;
  int64_t half;
  unsigned bitA;
  unsigned bitB;
};
size_t qr_workspace_bytes(int64_t batch, int64_t n);
void qr_force_give_up(unsigned mask);
// Whether a call over `batch` matrices of order n runs the resident block
// factorization on the current device (else the slower panel path).
hipError_t qr_block_path(int64_t batch, int64_t n, bool *out);
hipError_t qr_factor_and_form_q(float *At, float *Q, float *Rf, int64_t batch, int64_t n,
                                void *ws, size_t ws_bytes, hipStream_t s, hipStream_t sp,
                                hipStream_t st, unsigned *status, unsigned status_bit,
                                hipEvent_t q_free = nullptr,
                                hipEvent_t mid = nullptr, float mid_frac = 0.5f,
                                const std::function<hipError_t()> &at_mid = {},
                                const QrSplitOut *split = nullptr);
// dst = src^T for one n x n row-major matrix.
hipError_t launch_transpose(float *dst, const float *src, int64_t n, hipStream_t s);

}  // namespace soap
