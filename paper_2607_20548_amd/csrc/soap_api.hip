// Host side of the SOAP C ABI: argument validation, workspace carving, the
// ordered sequence of kernel launches for one step, stage timing and the
// thread-local error string.  Everything is enqueued on the caller's stream;
// nothing here allocates device memory.
#include "soap.h"

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <vector>

#include "internal.h"

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

int ok() {
  g_err[0] = '\0';
  return SOAP_OK;
}

int hip_fail(hipError_t e, const char *where) {
  return fail(SOAP_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

bool dim_ok(int64_t d) { return d >= 1 && d <= SOAP_MAX_DIM; }
bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// ---------------------------------------------------------------- timing
enum Stage {
  ST_MOMENTUM = 0,
  ST_FACTOR_L,
  ST_FACTOR_R,
  ST_POWER_L,
  ST_POWER_R,
  ST_QR_L,
  ST_QR_R,
  ST_ROT_IN_L,
  ST_ROT_IN_R_ADAM,
  ST_ROT_OUT_L,
  ST_ROT_OUT_R_UPDATE,
  ST_KL_EIG_L,
  ST_KL_EIG_R,
  ST_KL_PROJ_L,
  ST_KL_PROJ_R,
  ST_KL_FACTOR_L,
  ST_KL_FACTOR_R,
  ST_KL_LOWRANK_L,
  ST_KL_LOWRANK_R,
  ST_MUON_NORMALISE,
  ST_MUON_NEWTON_SCHULZ,
  ST_MUON_UPDATE,
  ST_QR_LR,
  ST_COUNT
};

const char *kStageNames[ST_COUNT] = {
    "momentum_ema",     "factor_ema_L",    "factor_ema_R",  "power_L",
    "power_R",          "qr_L",            "qr_R",          "rotate_in_QLt",
    "rotate_in_QR_adam", "rotate_out_QL",  "rotate_out_QRt_update", "kl_eig_L",
    "kl_eig_R",         "kl_proj_L",       "kl_proj_R",     "kl_factor_L",
    "kl_factor_R",      "kl_lowrank_L",    "kl_lowrank_R",  "muon_normalise",
    "muon_newton_schulz", "muon_update", "qr_L_R"};

struct Pending {
  int stage;
  hipEvent_t a, b;
  double flops;
};

struct Timing {
  std::mutex mu;
  bool enabled = false;
  std::vector<Pending> pending;
  std::vector<hipEvent_t> free_events;
  double ms[ST_COUNT] = {};
  int64_t launches[ST_COUNT] = {};
  double flops[ST_COUNT] = {};
};

Timing &timing() {
  static Timing t;
  return t;
}

hipEvent_t take_event(Timing &t) {
  if (!t.free_events.empty()) {
    hipEvent_t e = t.free_events.back();
    t.free_events.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Records a pair of events around one stage when timing is enabled.
class StageScope {
 public:
  StageScope(int stage, double flops, hipStream_t s) : stage_(stage), flops_(flops), s_(s) {
    Timing &t = timing();
    std::lock_guard<std::mutex> g(t.mu);
    if (!t.enabled) return;
    a_ = take_event(t);
    b_ = take_event(t);
    if (a_ && b_ && hipEventRecord(a_, s_) == hipSuccess) active_ = true;
  }
  ~StageScope() {
    if (!active_) return;
    Timing &t = timing();
    std::lock_guard<std::mutex> g(t.mu);
    if (hipEventRecord(b_, s_) == hipSuccess) t.pending.push_back({stage_, a_, b_, flops_});
  }

 private:
  int stage_;
  double flops_;
  hipStream_t s_;
  hipEvent_t a_ = nullptr, b_ = nullptr;
  bool active_ = false;
};

// ------------------------------------------------------ auxiliary stream
// The L-side chain (factor EMA L, power product, QR of m x m) and the R-side
// chain are independent until the rotations; the L side runs on one
// auxiliary stream per device (default priority, created on first use) and is
// joined back with events, so its latency-bound QR panels overlap the R side.
// Streams per device: 0 = L side, 1 / 2 = block factorizations of the L- /
// R-side QR (look-ahead).  With the caller's stream that is four: HIP maps a
// process's streams onto a few hardware queues (four by default) and streams
// that share a queue run in submission order, so the step uses no more.
// The T matrices of block pairs go on streams with slack: the R side's on
// the L-side stream, the L side's on the L-side block stream.
constexpr int N_AUX = 3;
// Fraction of the R-side QR's outer blocks after which the rotations Q_L^T G,
// Q_L^T M start: the factorization's later blocks leave most compute units
// idle.
constexpr float kRotateInFrom = 0.5f;
// Fraction of the R-side QR's outer blocks after which the L side's QR starts
// when R is the larger factor.
constexpr float kLSideFrom = 0.35f;
// Workgroup cap of products that run beside the resident block kernels of
// the other side's QR: 160 of the 256 compute units, leaving about 12 per XCD.
constexpr int kSideWorkgroups = 160;
std::mutex g_aux_mu;
hipStream_t g_aux[64][N_AUX] = {};

hipError_t aux_stream(int which, hipStream_t *out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64 || which < 0 || which >= N_AUX) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> g(g_aux_mu);
  if (!g_aux[dev][which]) {
    e = hipStreamCreateWithFlags(&g_aux[dev][which], hipStreamNonBlocking);
    if (e != hipSuccess) return e;
  }
  *out = g_aux[dev][which];
  return hipSuccess;
}

// ------------------------------------------------------------- workspace
// The KL step adds one m x n buffer, the eigenvalue estimates and their
// partial sums; the QR workspaces stay last (each QR uses up to the next
// region, the R side up to the end).
// The status word of the step comes first (soap_workspace_status reads it at
// offset 0).
struct StepLayout {
  size_t st, al, ar, tg, tm, nb, kz, kw, laml, lamr, partl, partr, qrl, qrr, total;
};

StepLayout step_layout(int64_t batch, int64_t m, int64_t n, bool kl) {
  StepLayout L{};
  const size_t f = sizeof(float);
  size_t o = 0;
  L.st = o; o = align256(o + sizeof(uint32_t));
  L.al = o; o = align256(o + f * batch * m * m);
  L.ar = o; o = align256(o + f * batch * n * n);
  L.tg = o; o = align256(o + f * batch * m * n);   // T_G, T_M: adjacent, so that the
  L.tm = o; o = align256(o + f * batch * m * n);   // row-interleaved pair fits over both
  L.nb = o; o = align256(o + f * batch * m * n);
  if (kl) {
    L.kz = o; o = align256(o + f * batch * m * n);
    L.kw = o; o = align256(o + f * batch * m * n);
    L.laml = o; o = align256(o + f * batch * m);
    L.lamr = o; o = align256(o + f * batch * n);
    L.partl = o; o = align256(o + f * soap::diag_partial_floats(batch, m));
    L.partr = o; o = align256(o + f * soap::diag_partial_floats(batch, n));
  }
  L.qrl = o; o = align256(o + soap::qr_workspace_bytes(batch, m));
  L.qrr = o; o = align256(o + soap::qr_workspace_bytes(batch, n));
  L.total = o;
  return L;
}

// Workspace of the KL accumulation alone (soap_kl_factors_f32).
struct KlLayout {
  size_t xl, xr, yl, zl, yr, zr, laml, lamr, partl, partr, total;
};

KlLayout kl_layout(int64_t m, int64_t n) {
  KlLayout L{};
  const size_t f = sizeof(float);
  size_t o = 0;
  L.xl = o; o = align256(o + f * m * m);
  L.xr = o; o = align256(o + f * n * n);
  L.yl = o; o = align256(o + f * m * n);
  L.zl = o; o = align256(o + f * m * n);
  L.yr = o; o = align256(o + f * m * n);
  L.zr = o; o = align256(o + f * m * n);
  L.laml = o; o = align256(o + f * m);
  L.lamr = o; o = align256(o + f * n);
  L.partl = o; o = align256(o + f * soap::diag_partial_floats(1, m));
  L.partr = o; o = align256(o + f * soap::diag_partial_floats(1, n));
  L.total = o;
  return L;
}

// ------------------------------------------------- KL-Shampoo accumulation
// Buffers of the accumulation: X = Q^T F of each side (d x d), the projected
// gradients Y_L = Q_L^T G, Y_R = G Q_R and their inverse-eigenvalue-scaled
// copies Z (m x n), the estimates lambda and the diagonal's partial sums.
struct KlBufs {
  float *XL, *XR, *YL, *ZL, *YR, *ZR, *lamL, *lamR, *partL, *partR;
};

// Algorithm 2's KL-Shampoo accumulation, enqueued on two streams: the L side
// (sl) and the R side (s).  With the previous step's bases,
//   lambda_L = diag(Q_L^T L Q_L),   lambda_R = diag(Q_R^T R Q_R),
//   L <- bk L + (1-bk)/n  Y_R diag(1/(lambda_R+eps)) Y_R^T,   Y_R = G Q_R,
//   R <- bk R + (1-bk)/m  Y_L^T diag(1/(lambda_L+eps)) Y_L,   Y_L = Q_L^T G,
// i.e. each factor's new term weighs G by the other factor's inverse as its
// basis diagonalises it.  Cross-stream order: ev_lamr (s -> sl) carries
// lambda_R, ev_zl (sl -> s) carries Y_L and Z_L; ev_yr is recorded on sl once
// Q_R has been read, and the caller must make Q_R's writer wait for it.
// Returns the failing step's name in *where.
hipError_t kl_accumulate(int64_t batch, int64_t m, int64_t n, const float *G, float *L, float *R,
                         const float *QL, const float *QR, float bk, float eps, const KlBufs &b,
                         hipStream_t s, hipStream_t sl, hipEvent_t ev_lamr, hipEvent_t ev_zl,
                         hipEvent_t ev_yr, const char **where) {
  const int64_t mn = m * n, mm = m * m, nn = n * n;
  const double B = (double)batch, md = (double)m, nd = (double)n;
  hipError_t e;
  {  // X_L = Q_L^T L, lambda_L = diag(X_L Q_L)
    StageScope sc(ST_KL_EIG_L, B * 2.0 * md * md * md, sl);
    soap::GemmDesc d;
    d.trans_a = 1; d.trans_b = 0; d.M = m; d.N = m; d.K = m;
    d.A = QL; d.lda = m; d.sA = mm; d.B = L; d.ldb = m; d.sB = mm;
    d.C = b.XL; d.ldc = m; d.sC = mm; d.batch = batch; d.tag = 1;
    if ((e = soap::launch_gemm(d, sl)) != hipSuccess) { *where = "KL eigenvalues L"; return e; }
    if ((e = soap::launch_diag_of_product(b.XL, QL, batch, m, b.partL, b.lamL, sl)) != hipSuccess) {
      *where = "KL eigenvalues L"; return e;
    }
  }
  {  // Y_L = Q_L^T G, Z_L = diag(1/(lambda_L+eps)) Y_L
    StageScope sc(ST_KL_PROJ_L, B * 2.0 * md * md * nd, sl);
    soap::GemmDesc d;
    d.trans_a = 1; d.trans_b = 0; d.M = m; d.N = n; d.K = m;
    d.A = QL; d.lda = m; d.sA = mm; d.B = G; d.ldb = n; d.sB = mn;
    d.C = b.YL; d.ldc = n; d.sC = mn; d.batch = batch;
    if ((e = soap::launch_gemm(d, sl)) != hipSuccess) { *where = "KL projection L"; return e; }
    if ((e = soap::launch_kl_scale(b.YL, b.ZL, b.lamL, batch, m, n, 1, eps, sl)) != hipSuccess) {
      *where = "KL scaling L"; return e;
    }
  }
  if ((e = hipEventRecord(ev_zl, sl)) != hipSuccess) { *where = "KL event"; return e; }
  {  // X_R = Q_R^T R, lambda_R = diag(X_R Q_R)
    StageScope sc(ST_KL_EIG_R, B * 2.0 * nd * nd * nd, s);
    soap::GemmDesc d;
    d.trans_a = 1; d.trans_b = 0; d.M = n; d.N = n; d.K = n;
    d.A = QR; d.lda = n; d.sA = nn; d.B = R; d.ldb = n; d.sB = nn;
    d.C = b.XR; d.ldc = n; d.sC = nn; d.batch = batch; d.tag = 2;
    if ((e = soap::launch_gemm(d, s)) != hipSuccess) { *where = "KL eigenvalues R"; return e; }
    if ((e = soap::launch_diag_of_product(b.XR, QR, batch, n, b.partR, b.lamR, s)) != hipSuccess) {
      *where = "KL eigenvalues R"; return e;
    }
  }
  if ((e = hipEventRecord(ev_lamr, s)) != hipSuccess) { *where = "KL event"; return e; }
  if ((e = hipStreamWaitEvent(sl, ev_lamr, 0)) != hipSuccess) { *where = "KL event"; return e; }
  {  // Y_R = G Q_R, Z_R = Y_R diag(1/(lambda_R+eps))
    StageScope sc(ST_KL_PROJ_R, B * 2.0 * md * nd * nd, sl);
    soap::GemmDesc d;
    d.trans_a = 0; d.trans_b = 0; d.M = m; d.N = n; d.K = n;
    d.A = G; d.lda = n; d.sA = mn; d.B = QR; d.ldb = n; d.sB = nn;
    d.C = b.YR; d.ldc = n; d.sC = mn; d.batch = batch;
    if ((e = soap::launch_gemm(d, sl)) != hipSuccess) { *where = "KL projection R"; return e; }
    if ((e = hipEventRecord(ev_yr, sl)) != hipSuccess) { *where = "KL event"; return e; }
    if ((e = soap::launch_kl_scale(b.YR, b.ZR, b.lamR, batch, m, n, 0, eps, sl)) != hipSuccess) {
      *where = "KL scaling R"; return e;
    }
  }
  {  // L <- bk L + (1-bk)/n Y_R Z_R^T (lower triangle, mirrored)
    StageScope sc(ST_KL_FACTOR_L, B * md * (md + 1) * nd, sl);
    soap::GemmDesc d;
    d.trans_a = 0; d.trans_b = 1; d.M = m; d.N = m; d.K = n;
    d.A = b.YR; d.lda = n; d.sA = mn; d.B = b.ZR; d.ldb = n; d.sB = mn;
    d.C = L; d.ldc = m; d.sC = mm; d.alpha = (float)((1.0 - (double)bk) / nd); d.beta = bk;
    d.batch = batch;
    if ((e = soap::launch_syrk_ema(d, sl)) != hipSuccess) { *where = "KL factor L"; return e; }
  }
  if ((e = hipStreamWaitEvent(s, ev_zl, 0)) != hipSuccess) { *where = "KL event"; return e; }
  {  // R <- bk R + (1-bk)/m Y_L^T Z_L
    StageScope sc(ST_KL_FACTOR_R, B * nd * (nd + 1) * md, s);
    soap::GemmDesc d;
    d.trans_a = 1; d.trans_b = 0; d.M = n; d.N = n; d.K = m;
    d.A = b.YL; d.lda = n; d.sA = mn; d.B = b.ZL; d.ldb = n; d.sB = mn;
    d.C = R; d.ldc = n; d.sC = nn; d.alpha = (float)((1.0 - (double)bk) / md); d.beta = bk;
    d.batch = batch;
    if ((e = soap::launch_syrk_ema(d, s)) != hipSuccess) { *where = "KL factor R"; return e; }
  }
  return hipSuccess;
}

struct Range {
  const void *p;
  size_t bytes;
  const char *name;
};

bool overlap(const Range &x, const Range &y) {
  const char *a = static_cast<const char *>(x.p), *b = static_cast<const char *>(y.p);
  return a < b + y.bytes && b < a + x.bytes;
}

int check_hparams(float beta1, float beta2, float eps, float lr, float wd, int64_t step,
                  uint32_t flags) {
  if (!std::isfinite(beta1) || beta1 < 0.f || beta1 >= 1.f)
    return fail(SOAP_ERR_HPARAM, "beta1 = %g is outside [0, 1)", (double)beta1);
  if (!std::isfinite(beta2) || beta2 < 0.f || beta2 >= 1.f)
    return fail(SOAP_ERR_HPARAM, "beta2 = %g is outside [0, 1)", (double)beta2);
  if (!std::isfinite(eps) || eps < 0.f)
    return fail(SOAP_ERR_HPARAM, "eps = %g must be finite and >= 0", (double)eps);
  if (!std::isfinite(lr) || lr < 0.f)
    return fail(SOAP_ERR_HPARAM, "lr = %g must be finite and >= 0", (double)lr);
  if (!std::isfinite(wd) || wd < 0.f)
    return fail(SOAP_ERR_HPARAM, "weight_decay = %g must be finite and >= 0", (double)wd);
  if (step < 1) return fail(SOAP_ERR_HPARAM, "step = %lld must be >= 1", (long long)step);
  if (flags & ~uint32_t(SOAP_FLAG_NO_BIAS_CORRECTION | SOAP_FLAG_SKIP_REFRESH |
                        SOAP_FLAG_STALE_REFRESH))
    return fail(SOAP_ERR_HPARAM, "unknown flag bits 0x%x", flags);
  return SOAP_OK;
}

// The front of a KL-SOAP step: the KL-Shampoo accumulation of both factors
// and the transposed power products A_L^T = Q_L^T L_new, A_R^T = Q_R^T R_new
// that the QRs consume, with the previous step's bases throughout.  The
// product X = Q^T F_old of each side serves the eigenvalue estimates, and on
// a side whose dimension d exceeds twice the other (e) it also gives the power
// product without a second d^3 product, because the new term has rank e:
//   A_R^T = bk X_R + cR W_R^T Z_L,   W_R = Y_L Q_R   (4 d^2 e flops, not 2 d^3)
//   A_L^T = bk X_L + cL W_L Z_R^T,   W_L = Q_L^T Y_R
// with Y_L = Q_L^T G, Z_L = diag(1/(lambda_L+eps)) Y_L, Y_R = G Q_R,
// Z_R = Y_R diag(1/(lambda_R+eps)), cL = (1-bk)/n, cR = (1-bk)/m.
// Streams: the R side on s, the L side on sl.  sl produces Y_L, Z_L (and
// W_R) and records ev_a; s forms X_R, lambda_R, waits for ev_a, finishes
// A_R^T and records ev_power; sl then waits for ev_power (R-side work first:
// it is on the critical path), forms Y_R (recording ev_yr once the old Q_R is
// read), Z_R, L_new and A_L^T.  On the R-trick side the update of R itself is
// not needed before the QR and is left to the caller (*defer_r = true), who
// runs it later on sl with the L side's Y_L, Z_L.  Without a refresh
// (refresh = false) only the factors are updated; with a stale refresh the
// power products are the products X = Q^T F_old of the estimates.
struct KlStepBufs {
  float *AL, *AR, *YL, *ZL, *YR, *ZR, *W, *lamL, *lamR, *partL, *partR;
};

hipError_t kl_front(int64_t batch, int64_t m, int64_t n, const float *G, float *L, float *R,
                    const float *QL, const float *QR, float bk, float eps, const KlStepBufs &b,
                    hipStream_t s, hipStream_t sl, hipEvent_t ev_a, hipEvent_t ev_power,
                    hipEvent_t ev_yr, bool refresh, bool stale, bool *defer_r,
                    const char **where) {
  const int64_t mn = m * n, mm = m * m, nn = n * n;
  const double B = (double)batch, md = (double)m, nd = (double)n;
  // Without a refresh no power product is formed; a stale refresh uses
  // X = Q^T F_old itself, which the estimates leave in A_L, A_R.
  const bool fresh = refresh && !stale;
  const bool trick_r = fresh && n > 2 * m, trick_l = fresh && m > 2 * n;
  const float cL = (float)((1.0 - (double)bk) / nd), cR = (float)((1.0 - (double)bk) / md);
  hipError_t e;
  auto fail_at = [&](const char *w, hipError_t err) { *where = w; return err; };
  {  // X_L = Q_L^T L, lambda_L = diag(X_L Q_L)
    StageScope sc(ST_KL_EIG_L, B * 2.0 * md * md * md, sl);
    soap::GemmDesc d;
    d.trans_a = 1; d.trans_b = 0; d.M = m; d.N = m; d.K = m;
    d.A = QL; d.lda = m; d.sA = mm; d.B = L; d.ldb = m; d.sB = mm;
    d.C = b.AL; d.ldc = m; d.sC = mm; d.batch = batch; d.tag = 1;
    if ((e = soap::launch_gemm(d, sl)) != hipSuccess) return fail_at("KL eigenvalues L", e);
    if ((e = soap::launch_diag_of_product(b.AL, QL, batch, m, b.partL, b.lamL, sl)) != hipSuccess)
      return fail_at("KL eigenvalues L", e);
  }
  {  // Y_L = Q_L^T G, Z_L = diag(1/(lambda_L+eps)) Y_L
    StageScope sc(ST_KL_PROJ_L, B * 2.0 * md * md * nd, sl);
    soap::GemmDesc d;
    d.trans_a = 1; d.trans_b = 0; d.M = m; d.N = n; d.K = m;
    d.A = QL; d.lda = m; d.sA = mm; d.B = G; d.ldb = n; d.sB = mn;
    d.C = b.YL; d.ldc = n; d.sC = mn; d.batch = batch;
    if ((e = soap::launch_gemm(d, sl)) != hipSuccess) return fail_at("KL projection L", e);
    if ((e = soap::launch_kl_scale(b.YL, b.ZL, b.lamL, batch, m, n, 1, eps, sl)) != hipSuccess)
      return fail_at("KL scaling L", e);
  }
  if (trick_r) {  // W_R = Y_L Q_R
    StageScope sc(ST_KL_LOWRANK_R, B * 2.0 * md * nd * nd, sl);
    soap::GemmDesc d;
    d.trans_a = 0; d.trans_b = 0; d.M = m; d.N = n; d.K = n;
    d.A = b.YL; d.lda = n; d.sA = mn; d.B = QR; d.ldb = n; d.sB = nn;
    d.C = b.W; d.ldc = n; d.sC = mn; d.batch = batch;
    if ((e = soap::launch_gemm(d, sl)) != hipSuccess) return fail_at("KL low-rank R", e);
  }
  if ((e = hipEventRecord(ev_a, sl)) != hipSuccess) return fail_at("KL event", e);
  {  // X_R = Q_R^T R, lambda_R = diag(X_R Q_R)
    StageScope sc(ST_KL_EIG_R, B * 2.0 * nd * nd * nd, s);
    soap::GemmDesc d;
    d.trans_a = 1; d.trans_b = 0; d.M = n; d.N = n; d.K = n;
    d.A = QR; d.lda = n; d.sA = nn; d.B = R; d.ldb = n; d.sB = nn;
    d.C = b.AR; d.ldc = n; d.sC = nn; d.batch = batch; d.tag = 2;
    if ((e = soap::launch_gemm(d, s)) != hipSuccess) return fail_at("KL eigenvalues R", e);
    if ((e = soap::launch_diag_of_product(b.AR, QR, batch, n, b.partR, b.lamR, s)) != hipSuccess)
      return fail_at("KL eigenvalues R", e);
  }
  if ((e = hipStreamWaitEvent(s, ev_a, 0)) != hipSuccess) return fail_at("KL event", e);
  if (trick_r) {  // A_R^T = bk X_R + cR W_R^T Z_L
    StageScope sc(ST_KL_LOWRANK_R, B * 2.0 * nd * nd * md, s);
    soap::GemmDesc d;
    d.trans_a = 1; d.trans_b = 0; d.M = n; d.N = n; d.K = m;
    d.A = b.W; d.lda = n; d.sA = mn; d.B = b.ZL; d.ldb = n; d.sB = mn;
    d.C = b.AR; d.ldc = n; d.sC = nn; d.alpha = cR; d.beta = bk; d.batch = batch;
    if ((e = soap::launch_gemm(d, s)) != hipSuccess) return fail_at("KL low-rank R", e);
  } else {
    {  // R <- bk R + cR Y_L^T Z_L
      StageScope sc(ST_KL_FACTOR_R, B * nd * (nd + 1) * md, s);
      soap::GemmDesc d;
      d.trans_a = 1; d.trans_b = 0; d.M = n; d.N = n; d.K = m;
      d.A = b.YL; d.lda = n; d.sA = mn; d.B = b.ZL; d.ldb = n; d.sB = mn;
      d.C = R; d.ldc = n; d.sC = nn; d.alpha = cR; d.beta = bk; d.batch = batch;
      if ((e = soap::launch_syrk_ema(d, s)) != hipSuccess) return fail_at("KL factor R", e);
    }
    if (fresh) {  // A_R^T = Q_R^T R
      StageScope sc(ST_POWER_R, B * 2.0 * nd * nd * nd, s);
      soap::GemmDesc d;
      d.trans_a = 1; d.trans_b = 0; d.M = n; d.N = n; d.K = n;
      d.A = QR; d.lda = n; d.sA = nn; d.B = R; d.ldb = n; d.sB = nn;
      d.C = b.AR; d.ldc = n; d.sC = nn; d.batch = batch; d.tag = 2;
      if ((e = soap::launch_gemm(d, s)) != hipSuccess) return fail_at("power R", e);
    }
  }
  if ((e = hipEventRecord(ev_power, s)) != hipSuccess) return fail_at("KL event", e);
  if ((e = hipStreamWaitEvent(sl, ev_power, 0)) != hipSuccess) return fail_at("KL event", e);
  {  // Y_R = G Q_R, Z_R = Y_R diag(1/(lambda_R+eps))
    StageScope sc(ST_KL_PROJ_R, B * 2.0 * md * nd * nd, sl);
    soap::GemmDesc d;
    d.trans_a = 0; d.trans_b = 0; d.M = m; d.N = n; d.K = n;
    d.A = G; d.lda = n; d.sA = mn; d.B = QR; d.ldb = n; d.sB = nn;
    d.C = b.YR; d.ldc = n; d.sC = mn; d.batch = batch; d.max_wg = kSideWorkgroups;
    if ((e = soap::launch_gemm(d, sl)) != hipSuccess) return fail_at("KL projection R", e);
    if ((e = hipEventRecord(ev_yr, sl)) != hipSuccess) return fail_at("KL event", e);
    if ((e = soap::launch_kl_scale(b.YR, b.ZR, b.lamR, batch, m, n, 0, eps, sl)) != hipSuccess)
      return fail_at("KL scaling R", e);
  }
  if (trick_l) {  // W_L = Q_L^T Y_R
    StageScope sc(ST_KL_LOWRANK_L, B * 2.0 * md * md * nd, sl);
    soap::GemmDesc d;
    d.trans_a = 1; d.trans_b = 0; d.M = m; d.N = n; d.K = m;
    d.A = QL; d.lda = m; d.sA = mm; d.B = b.YR; d.ldb = n; d.sB = mn;
    d.C = b.W; d.ldc = n; d.sC = mn; d.batch = batch; d.max_wg = kSideWorkgroups;
    if ((e = soap::launch_gemm(d, sl)) != hipSuccess) return fail_at("KL low-rank L", e);
  }
  {  // L <- bk L + cL Y_R Z_R^T
    StageScope sc(ST_KL_FACTOR_L, B * md * (md + 1) * nd, sl);
    soap::GemmDesc d;
    d.trans_a = 0; d.trans_b = 1; d.M = m; d.N = m; d.K = n;
    d.A = b.YR; d.lda = n; d.sA = mn; d.B = b.ZR; d.ldb = n; d.sB = mn;
    d.C = L; d.ldc = m; d.sC = mm; d.alpha = cL; d.beta = bk; d.batch = batch;
    d.max_wg = kSideWorkgroups;
    if ((e = soap::launch_syrk_ema(d, sl)) != hipSuccess) return fail_at("KL factor L", e);
  }
  if (trick_l) {  // A_L^T = bk X_L + cL W_L Z_R^T
    StageScope sc(ST_KL_LOWRANK_L, B * 2.0 * md * md * nd, sl);
    soap::GemmDesc d;
    d.trans_a = 0; d.trans_b = 1; d.M = m; d.N = m; d.K = n;
    d.A = b.W; d.lda = n; d.sA = mn; d.B = b.ZR; d.ldb = n; d.sB = mn;
    d.C = b.AL; d.ldc = m; d.sC = mm; d.alpha = cL; d.beta = bk; d.batch = batch;
    d.max_wg = kSideWorkgroups;
    if ((e = soap::launch_gemm(d, sl)) != hipSuccess) return fail_at("KL low-rank L", e);
  } else if (fresh) {  // A_L^T = Q_L^T L
    StageScope sc(ST_POWER_L, B * 2.0 * md * md * md, sl);
    soap::GemmDesc d;
    d.trans_a = 1; d.trans_b = 0; d.M = m; d.N = m; d.K = m;
    d.A = QL; d.lda = m; d.sA = mm; d.B = L; d.ldb = m; d.sB = mm;
    d.C = b.AL; d.ldc = m; d.sC = mm; d.batch = batch; d.tag = 1; d.max_wg = kSideWorkgroups;
    if ((e = soap::launch_gemm(d, sl)) != hipSuccess) return fail_at("power L", e);
  }
  *defer_r = trick_r;
  return hipSuccess;
}

// The fork/join events of a step: seven per host thread and device, created
// on first use and kept until the process ends.  A step records each at most
// once and enqueues every wait on it before returning, so the next step may
// record it again (a wait captures the record current when it is enqueued).
struct StepEvents {
  static constexpr int kCount = 7;
  hipEvent_t *ev = nullptr;
  hipError_t create() {
    thread_local hipEvent_t pool[64][kCount] = {};
    int dev = 0;
    hipError_t r = hipGetDevice(&dev);
    if (r != hipSuccess) return r;
    if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    for (hipEvent_t &e : pool[dev])
      if (!e && (r = hipEventCreateWithFlags(&e, hipEventDisableTiming)) != hipSuccess) return r;
    ev = pool[dev];
    return hipSuccess;
  }
};

// One SOAP step (kl = false: factor EMA of the Section 2 primer) or KL-SOAP
// step (kl = true: KL-Shampoo accumulation with coefficient beta_kron).
int step_impl(int64_t batch, float *param, const float *grad, float *L, float *R, float *QL,
              float *QR, float *M, float *V, int64_t m, int64_t n, float beta1, float beta2,
              float eps, float lr, float wd, int64_t step, uint32_t flags, void *ws,
              size_t ws_bytes, hipStream_t s, bool kl, float beta_kron) {
  if (!dim_ok(batch) || !dim_ok(m) || !dim_ok(n))
    return fail(SOAP_ERR_SHAPE, "batch=%lld m=%lld n=%lld: each must be in [1, %d]",
                (long long)batch, (long long)m, (long long)n, SOAP_MAX_DIM);
  const Range bufs[] = {
      {param, sizeof(float) * batch * m * n, "param"}, {grad, sizeof(float) * batch * m * n, "grad"},
      {L, sizeof(float) * batch * m * m, "L"},         {R, sizeof(float) * batch * n * n, "R"},
      {QL, sizeof(float) * batch * m * m, "Q_L"},      {QR, sizeof(float) * batch * n * n, "Q_R"},
      {M, sizeof(float) * batch * m * n, "M"},         {V, sizeof(float) * batch * m * n, "V"},
      {ws, ws_bytes, "workspace"}};
  for (const Range &b : bufs)
    if (!b.p) return fail(SOAP_ERR_NULL, "%s is NULL", b.name);
  int rc = check_hparams(beta1, beta2, eps, lr, wd, step, flags);
  if (rc != SOAP_OK) return rc;
  if (kl && (!std::isfinite(beta_kron) || beta_kron < 0.f || beta_kron >= 1.f))
    return fail(SOAP_ERR_HPARAM, "beta_kron = %g is outside [0, 1)", (double)beta_kron);
  const StepLayout lay = step_layout(batch, m, n, kl);
  if (ws_bytes < lay.total)
    return fail(SOAP_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", ws_bytes, lay.total);
  for (const Range &b : bufs)
    if (!aligned16(b.p)) return fail(SOAP_ERR_ALIGN, "%s is not 16-byte aligned", b.name);
  const int nb = sizeof(bufs) / sizeof(bufs[0]);
  for (int i = 0; i < nb; ++i)
    for (int j = i + 1; j < nb; ++j)
      if (overlap(bufs[i], bufs[j]))
        return fail(SOAP_ERR_ALIAS, "%s overlaps %s", bufs[i].name, bufs[j].name);

  const bool bc = !(flags & SOAP_FLAG_NO_BIAS_CORRECTION);
  const bool refresh = !(flags & SOAP_FLAG_SKIP_REFRESH);
  const bool stale = (flags & SOAP_FLAG_STALE_REFRESH) != 0;
  const float c1 = bc ? (float)(1.0 - std::pow((double)beta1, (double)step)) : 1.f;
  const float c2 = bc ? (float)(1.0 - std::pow((double)beta2, (double)step)) : 1.f;

  char *w = static_cast<char *>(ws);
  uint32_t *status = reinterpret_cast<uint32_t *>(w + lay.st);
  float *AL = reinterpret_cast<float *>(w + lay.al);
  float *AR = reinterpret_cast<float *>(w + lay.ar);
  float *TG = reinterpret_cast<float *>(w + lay.tg);
  float *TM = reinterpret_cast<float *>(w + lay.tm);
  float *NN = reinterpret_cast<float *>(w + lay.nb);
  void *qws_l = w + lay.qrl;
  const size_t qws_l_bytes = lay.qrr - lay.qrl;
  void *qws_r = w + lay.qrr;
  const size_t qws_r_bytes = ws_bytes - lay.qrr;
  const int64_t mn = m * n, mm = m * m, nn = n * n;
  const double B = (double)batch, md = (double)m, nd = (double)n;
  hipError_t e;

  // The status word starts clear; a QR that gives up sets its side's bit.
  if ((e = soap::launch_zero_u32(status, 1, s)) != hipSuccess) return hip_fail(e, "status");
  {  // M <- b1 M + (1-b1) G (weight space)
    StageScope sc(ST_MOMENTUM, 0.0, s);
    if ((e = soap::launch_momentum(M, grad, batch * mn, beta1, s)) != hipSuccess)
      return hip_fail(e, "momentum");
  }
  // Fork: the L side on the auxiliary stream, the R side on the caller's.
  hipStream_t sl = nullptr, spl = nullptr, spr = nullptr;
  if ((e = aux_stream(0, &sl)) != hipSuccess || (e = aux_stream(1, &spl)) != hipSuccess ||
      (e = aux_stream(2, &spr)) != hipSuccess)
    return hip_fail(e, "auxiliary stream");
  StepEvents evs;
  if ((e = evs.create()) != hipSuccess) return hip_fail(e, "event");
  hipEvent_t ev_fork = evs.ev[0], ev_join = evs.ev[1], ev_power = evs.ev[2];
  hipEvent_t ev_a = evs.ev[3], ev_yr = evs.ev[4], ev_lside = evs.ev[5], ev_mid = evs.ev[6];
  if ((e = hipEventRecord(ev_fork, s)) != hipSuccess) return hip_fail(e, "fork record");
  if ((e = hipStreamWaitEvent(sl, ev_fork, 0)) != hipSuccess) return hip_fail(e, "fork wait");
  bool defer_r = false;
  if (kl) {
    // KL-Shampoo accumulation and power products.  Buffer reuse: Y_L, Z_L in
    // T_G, T_M (rewritten on the L stream by the rotation, after their last
    // reads), Y_R in N (written after the join).
    const KlStepBufs kb{AL, AR, TG, TM, NN,
                        reinterpret_cast<float *>(w + lay.kz), reinterpret_cast<float *>(w + lay.kw),
                        reinterpret_cast<float *>(w + lay.laml), reinterpret_cast<float *>(w + lay.lamr),
                        reinterpret_cast<float *>(w + lay.partl), reinterpret_cast<float *>(w + lay.partr)};
    const char *where = "";
    if ((e = kl_front(batch, m, n, grad, L, R, QL, QR, beta_kron, eps, kb, s, sl, ev_a,
                      ev_power, ev_yr, refresh, stale, &defer_r, &where)) != hipSuccess)
      return hip_fail(e, where);
  } else {
    auto factor_l = [&]() -> hipError_t {  // L <- b2 L + (1-b2) G G^T
      StageScope sc(ST_FACTOR_L, B * md * (md + 1) * nd, sl);
      soap::GemmDesc d;
      d.trans_a = 0; d.trans_b = 1; d.M = m; d.N = m; d.K = n;
      d.A = grad; d.lda = n; d.sA = mn; d.B = grad; d.ldb = n; d.sB = mn;
      d.C = L; d.ldc = m; d.sC = mm; d.alpha = 1.f - beta2; d.beta = beta2; d.batch = batch;
      return soap::launch_syrk_ema(d, sl);
    };
    // Power products, produced transposed for the QR: (L Q_L)^T = Q_L^T L
    // since L is symmetric (both triangles are stored).
    auto power_l = [&]() -> hipError_t {  // A_L^T = Q_L^T L
      StageScope sc(ST_POWER_L, B * 2.0 * md * md * md, sl);
      soap::GemmDesc d;
      d.trans_a = 1; d.trans_b = 0;
      d.M = m; d.N = m; d.K = m; d.A = QL; d.lda = m; d.sA = mm; d.B = L; d.ldb = m; d.sB = mm;
      d.C = AL; d.ldc = m; d.sC = mm; d.batch = batch; d.tag = 1;
      return soap::launch_gemm(d, sl);
    };
    auto factor_r = [&]() -> hipError_t {  // R <- b2 R + (1-b2) G^T G
      StageScope sc(ST_FACTOR_R, B * nd * (nd + 1) * md, s);
      soap::GemmDesc d;
      d.trans_a = 1; d.trans_b = 0; d.M = n; d.N = n; d.K = m;
      d.A = grad; d.lda = n; d.sA = mn; d.B = grad; d.ldb = n; d.sB = mn;
      d.C = R; d.ldc = n; d.sC = nn; d.alpha = 1.f - beta2; d.beta = beta2; d.batch = batch;
      return soap::launch_syrk_ema(d, s);
    };
    auto power_r = [&]() -> hipError_t {  // A_R^T = Q_R^T R
      StageScope sc(ST_POWER_R, B * 2.0 * nd * nd * nd, s);
      soap::GemmDesc d;
      d.trans_a = 1; d.trans_b = 0;
      d.M = n; d.N = n; d.K = n; d.A = QR; d.lda = n; d.sA = nn; d.B = R; d.ldb = n; d.sB = nn;
      d.C = AR; d.ldc = n; d.sC = nn; d.batch = batch; d.tag = 2;
      return soap::launch_gemm(d, s);
    };
    // A stale refresh takes the power products before the gradient enters
    // the factors; without a refresh there are none.
    if (refresh && stale) {
      if ((e = power_l()) != hipSuccess) return hip_fail(e, "power L");
      if ((e = factor_l()) != hipSuccess) return hip_fail(e, "factor EMA L");
      if ((e = power_r()) != hipSuccess) return hip_fail(e, "power R");
      if ((e = factor_r()) != hipSuccess) return hip_fail(e, "factor EMA R");
    } else {
      if ((e = factor_l()) != hipSuccess) return hip_fail(e, "factor EMA L");
      if (refresh && (e = power_l()) != hipSuccess) return hip_fail(e, "power L");
      if ((e = factor_r()) != hipSuccess) return hip_fail(e, "factor EMA R");
      if (refresh && (e = power_r()) != hipSuccess) return hip_fail(e, "power R");
    }
    // The L-side QR starts once the R-side power product is done: its
    // resident block kernels need free compute units, which that long
    // product holds.
    if ((e = hipEventRecord(ev_power, s)) != hipSuccess) return hip_fail(e, "power record");
    if ((e = hipStreamWaitEvent(sl, ev_power, 0)) != hipSuccess) return hip_fail(e, "power wait");
  }
  // The L side's QR, its KL factor update and the rotations Q_L^T G, Q_L^T M.
  // When R is the larger factor (n >= 2m) they are enqueued from inside the
  // R-side QR's host loop once it reaches a fraction of its outer blocks,
  // right after an event recorded there: the first part of the R-side
  // factorization has its far trailing updates on the critical path, its
  // later blocks leave most compute units idle.  (Waits on an event recorded
  // later in host order resolve late, hence the callback.)
  const bool late_l = refresh && n >= 2 * m;
  const char *side_where = nullptr;
  auto l_side = [&](bool after_mid) -> hipError_t {
    hipError_t r;
    if (after_mid && (r = hipStreamWaitEvent(sl, ev_mid, 0)) != hipSuccess) {
      side_where = "QR R mid wait";
      return r;
    }
    if (refresh) {  // Q_L = QR(A_L).Q
      StageScope sc(ST_QR_L, B * (8.0 / 3.0) * md * md * md, sl);
      if ((r = soap::qr_factor_and_form_q(AL, QL, nullptr, batch, m, qws_l, qws_l_bytes, sl, spl,
                                          spl, status, SOAP_STATUS_QR_L)) != hipSuccess) {
        side_where = "QR L";
        return r;
      }
    }
    if (defer_r) {  // R <- bk R + (1-bk)/m Y_L^T Z_L, beside the R-side QR
      StageScope sc(ST_KL_FACTOR_R, B * nd * (nd + 1) * md, sl);
      soap::GemmDesc d;
      d.trans_a = 1; d.trans_b = 0; d.M = n; d.N = n; d.K = m;
      d.A = TG; d.lda = n; d.sA = mn; d.B = TM; d.ldb = n; d.sB = mn;
      d.C = R; d.ldc = n; d.sC = nn; d.alpha = (float)((1.0 - (double)beta_kron) / md);
      d.beta = beta_kron; d.batch = batch; d.max_wg = kSideWorkgroups;
      if ((r = soap::launch_syrk_ema(d, sl)) != hipSuccess) { side_where = "KL factor R"; return r; }
    }
    if ((r = hipEventRecord(ev_lside, sl)) != hipSuccess) { side_where = "L side record"; return r; }
    return hipSuccess;
  };
  // T_G = Q_L^T G,  T_M = Q_L^T M on the L side's block stream (free once the
  // L-side QR is done), held back to the R-side factorization's second half;
  // beside a much larger R side they are capped to part of the GPU (its
  // block kernels need whole compute units free).
  auto rotate_in_l_products = [&](hipStream_t st, int max_wg) -> hipError_t {
    hipError_t r;
    StageScope sc(ST_ROT_IN_L, B * 4.0 * md * md * nd, st);
    soap::GemmDesc d;
    d.trans_a = 1; d.trans_b = 0; d.M = m; d.N = n; d.K = m;
    d.A = QL; d.lda = m; d.sA = mm; d.B = grad; d.ldb = n; d.sB = mn;
    // T_G and T_M interleaved by rows over the T_G and T_M buffers (adjacent,
    // 2 m n floats per matrix): row 2i = T_G row i, row 2i+1 = T_M row i.
    d.C = TG; d.ldc = 2 * n; d.sC = 2 * mn; d.batch = batch;
    d.max_wg = max_wg;
    if ((r = soap::launch_gemm(d, st)) != hipSuccess) { side_where = "rotate in G"; return r; }
    d.B = M; d.C = TG + n;
    if ((r = soap::launch_gemm(d, st)) != hipSuccess) { side_where = "rotate in M"; return r; }
    return hipSuccess;
  };
  auto rotate_in_l = [&](bool after_mid) -> hipError_t {
    hipError_t r;
    if ((r = hipStreamWaitEvent(spl, ev_lside, 0)) != hipSuccess) { side_where = "L side wait"; return r; }
    if (after_mid && (r = hipStreamWaitEvent(spl, ev_mid, 0)) != hipSuccess) {
      side_where = "QR R mid wait";
      return r;
    }
    // Capped only beside a much larger R-side factorization; otherwise the
    // two QRs are of similar size (or the L side is the larger) and this
    // product runs when the R side has no resident blocks left to starve.
    if ((r = rotate_in_l_products(spl, late_l ? kSideWorkgroups : 0)) != hipSuccess) return r;
    if ((r = hipEventRecord(ev_join, spl)) != hipSuccess) { side_where = "join record"; return r; }
    return hipSuccess;
  };
  // Square factors: both QRs as one call over the 2 x batch matrices A_L,
  // A_R (adjacent in the workspace).  Two factorizations side by side contend
  // for the compute units and double the launches of the block chain; one
  // call carries both in each launch (4096 x 4096, Q formed backwards: 14.6
  // ms for the pair against 13.2 ms for one alone).  Its Q's are formed in
  // T_G, T_M (adjacent, free until the rotation; up to order 4096 forwards,
  // while the factorization runs) and copied to Q_L, Q_R; the rotation
  // Q_L^T G then follows on the caller's stream.
  bool pair = false;
  if (refresh && !kl && m == n && AR == AL + batch * nn && TM == TG + batch * nn &&
      soap::qr_workspace_bytes(2 * batch, n) <= ws_bytes - lay.qrl) {
    if ((e = soap::qr_block_path(2 * batch, n, &pair)) != hipSuccess) return hip_fail(e, "QR path");
  }
  if (pair) {
    if ((e = hipEventRecord(ev_lside, sl)) != hipSuccess) return hip_fail(e, "L side record");
    if ((e = hipStreamWaitEvent(s, ev_lside, 0)) != hipSuccess) return hip_fail(e, "L side wait");
    {
      StageScope sc(ST_QR_LR, 2.0 * B * (8.0 / 3.0) * nd * nd * nd, s);
      const soap::QrSplitOut so{QL, QR, batch, SOAP_STATUS_QR_L, SOAP_STATUS_QR_R};
      if ((e = soap::qr_factor_and_form_q(AL, TG, nullptr, 2 * batch, n, qws_l, ws_bytes - lay.qrl,
                                          s, spr, sl, status, 0u, nullptr, nullptr, 0.5f, {},
                                          &so)) != hipSuccess)
        return hip_fail(e, "QR L and R");
    }
    if ((e = rotate_in_l_products(s, 0)) != hipSuccess) return hip_fail(e, side_where);
  } else {
    if (!late_l && (e = l_side(false)) != hipSuccess) return hip_fail(e, side_where);
    if (refresh) {  // Q_R = QR(A_R).Q; under KL, Q_R is written only after G Q_R has read it
      StageScope sc(ST_QR_R, B * (8.0 / 3.0) * nd * nd * nd, s);
      auto at_mid = [&]() -> hipError_t {
        hipError_t r;
        if (late_l && (r = l_side(true)) != hipSuccess) return r;
        return rotate_in_l(true);
      };
      if ((e = soap::qr_factor_and_form_q(AR, QR, nullptr, batch, n, qws_r, qws_r_bytes, s, spr, sl,
                                          status, SOAP_STATUS_QR_R, kl ? ev_yr : nullptr, ev_mid,
                                          late_l ? kLSideFrom : kRotateInFrom, at_mid)) != hipSuccess)
        return hip_fail(e, side_where ? side_where : "QR R");
    } else if ((e = rotate_in_l(false)) != hipSuccess) {
      return hip_fail(e, side_where);
    }
    if ((e = hipStreamWaitEvent(s, ev_join, 0)) != hipSuccess) return hip_fail(e, "join wait");
  }
  {  // G' = T_G Q_R, M' = T_M Q_R (one product over the interleaved rows), then Adam
    StageScope sc(ST_ROT_IN_R_ADAM, B * 4.0 * md * nd * nd, s);
    soap::GemmDesc d;
    d.M = 2 * m; d.N = n; d.K = n; d.A = TG; d.lda = n; d.sA = 2 * mn; d.B = QR; d.ldb = n;
    d.sB = nn; d.C = nullptr; d.ldc = n; d.sC = mn; d.batch = batch;
    soap::AdamEpi ae;
    ae.V = V; ae.Nout = NN; ae.b2 = beta2; ae.c1 = c1; ae.c2 = c2; ae.eps = eps;
    if ((e = soap::launch_gemm_adam(d, ae, s)) != hipSuccess) return hip_fail(e, "rotate in + Adam");
  }
  {  // T2 = Q_L N (into T_G, which is dead now)
    StageScope sc(ST_ROT_OUT_L, B * 2.0 * md * md * nd, s);
    soap::GemmDesc d;
    d.M = m; d.N = n; d.K = m; d.A = QL; d.lda = m; d.sA = mm; d.B = NN; d.ldb = n; d.sB = mn;
    d.C = TG; d.ldc = n; d.sC = mn; d.batch = batch;
    if ((e = soap::launch_gemm(d, s)) != hipSuccess) return hip_fail(e, "rotate out L");
  }
  {  // W <- (1 - lr wd) W - lr T2 Q_R^T
    StageScope sc(ST_ROT_OUT_R_UPDATE, B * 2.0 * md * nd * nd, s);
    soap::GemmDesc d;
    d.trans_a = 0; d.trans_b = 1; d.M = m; d.N = n; d.K = n;
    d.A = TG; d.lda = n; d.sA = mn; d.B = QR; d.ldb = n; d.sB = nn;
    d.C = param; d.ldc = n; d.sC = mn; d.alpha = -lr; d.beta = 1.f - lr * wd; d.batch = batch;
    if ((e = soap::launch_gemm(d, s)) != hipSuccess) return hip_fail(e, "rotate out R + update");
  }
  return ok();
}

// ------------------------------------------------------------------ Muon
struct MuonLayout {
  size_t x, xn, a, bm, part, inv, total;
};

MuonLayout muon_layout(int64_t batch, int64_t m, int64_t n) {
  MuonLayout L{};
  const size_t f = sizeof(float);
  const int64_t d = std::min(m, n);
  size_t o = 0;
  L.x = o; o = align256(o + f * batch * m * n);
  L.xn = o; o = align256(o + f * batch * m * n);
  L.a = o; o = align256(o + f * batch * d * d);
  L.bm = o; o = align256(o + f * batch * d * d);
  L.part = o; o = align256(o + soap::muon_norm_partial_bytes(batch));
  L.inv = o; o = align256(o + f * batch);
  L.total = o;
  return L;
}

constexpr int64_t kMuonMaxIters = 1024;

// Newton-Schulz in bfloat16 (SOAP_MUON_BF16), after the momentum update:
// X, A and B are bfloat16, each product accumulated in fp32 on the matrix
// cores and rounded once.  The iterate of the d x e problem (d = min(m, n))
// is kept in both layouts, X (d x e) and X^T (e x d), so that every product
// reads k-contiguous rows: A = X X^T and B = b A + c A A^T (A symmetric) as
// one-triangle products, X <- a X + B X as (B, X^T) with both layouts of the
// result written.  The workspace of the fp32 form holds these buffers.
int muon_ns_bf16(int64_t batch, float *param, const float *M, int64_t m, int64_t n, float lr,
                 float wd, float eps, const float *coeffs, int64_t iters, char *w,
                 const MuonLayout &lay, hipStream_t s) {
  const bool tall = m > n;
  const int64_t d = tall ? n : m, e2 = tall ? m : n;
  const int64_t mn = m * n, dd = d * d;
  uint16_t *X = reinterpret_cast<uint16_t *>(w + lay.x), *Xt = X + batch * mn;
  uint16_t *Y = reinterpret_cast<uint16_t *>(w + lay.xn), *Yt = Y + batch * mn;
  uint16_t *A = reinterpret_cast<uint16_t *>(w + lay.a), *B = A + batch * dd;
  float *inv = reinterpret_cast<float *>(w + lay.inv);
  const double Bt = (double)batch, dd_ = (double)d, ee = (double)e2;
  hipError_t e;
  {  // X_0 = round(M / max(||M||_F, eps)) as d x e (M^T when tall) and its transpose
    StageScope sc(ST_MUON_NORMALISE, 0.0, s);
    if ((e = soap::launch_muon_norm_inv(M, batch, mn, eps, reinterpret_cast<double *>(w + lay.part),
                                        inv, s)) != hipSuccess)
      return hip_fail(e, "normalise");
    if ((e = soap::launch_bf16_scale_both(M, batch, d, e2, tall, inv, X, Xt, s)) != hipSuccess)
      return hip_fail(e, "normalise (bf16)");
  }
  for (int64_t it = 0; it < iters; ++it) {
    const float a = coeffs[3 * it], b = coeffs[3 * it + 1], c = coeffs[3 * it + 2];
    StageScope sc(ST_MUON_NEWTON_SCHULZ,
                  Bt * (dd_ * (dd_ + 1) * ee + (c != 0.f ? 2.0 * dd_ * dd_ * dd_ : 0.0) +
                        2.0 * dd_ * dd_ * ee), s);
    soap::BfGemmDesc g;   // A = X X^T
    g.M = d; g.N = d; g.K = e2; g.P = X; g.ldp = e2; g.sP = mn; g.Q = X; g.ldq = e2; g.sQ = mn;
    g.C = A; g.ldc = d; g.sC = dd; g.batch = batch; g.syrk = true;
    if ((e = soap::launch_gemm_bf16_nt(g, s)) != hipSuccess) return hip_fail(e, "Newton-Schulz A (bf16)");
    const uint16_t *Bop = A;
    float alpha_b = b;
    if (c != 0.f) {       // B = b A + c A A^T
      soap::BfGemmDesc h;
      h.M = d; h.N = d; h.K = d; h.P = A; h.ldp = d; h.sP = dd; h.Q = A; h.ldq = d; h.sQ = dd;
      h.D = A; h.ldd = d; h.sD = dd; h.C = B; h.ldc = d; h.sC = dd;
      h.alpha = c; h.beta = b; h.batch = batch; h.syrk = true;
      if ((e = soap::launch_gemm_bf16_nt(h, s)) != hipSuccess) return hip_fail(e, "Newton-Schulz B (bf16)");
      Bop = B;
      alpha_b = 1.f;
    }
    soap::BfGemmDesc x;   // X <- a X + B X, both layouts
    x.M = d; x.N = e2; x.K = d; x.P = Bop; x.ldp = d; x.sP = dd; x.Q = Xt; x.ldq = d; x.sQ = mn;
    x.D = X; x.ldd = e2; x.sD = mn; x.C = Y; x.ldc = e2; x.sC = mn;
    x.Ct = Yt; x.ldct = d; x.sCt = mn; x.alpha = alpha_b; x.beta = a; x.batch = batch;
    if ((e = soap::launch_gemm_bf16_nt(x, s)) != hipSuccess) return hip_fail(e, "Newton-Schulz X (bf16)");
    std::swap(X, Y);
    std::swap(Xt, Yt);
  }
  {  // W <- (1 - lr wd) W - lr sqrt(max(m, n)) X_n, X_n in the m x n layout
    StageScope sc(ST_MUON_UPDATE, 0.0, s);
    const float scale = (float)std::sqrt((double)std::max(m, n));
    if ((e = soap::launch_axpby_bf16(param, tall ? Xt : X, batch * mn, 1.f - lr * wd, -lr * scale,
                                     s)) != hipSuccess)
      return hip_fail(e, "update");
  }
  return ok();
}

// One Muon step (Algorithm 1) on `batch` m x n matrices.  The Newton-Schulz
// polynomial acts on singular values only, so its Gram matrix is formed on
// the smaller side: A = X X^T (m x m) with X <- a X + B X when m <= n, and
// A = X^T X (n x n) with X <- a X + X B otherwise; both are Algorithm 1's
// iterate exactly (for the wide case the same steps applied to X^T).
int muon_impl(int64_t batch, float *param, const float *grad, float *M, int64_t m, int64_t n,
              float beta1, float lr, float wd, float eps, const float *coeffs, int64_t iters,
              uint32_t flags, void *ws, size_t ws_bytes, hipStream_t s) {
  if (!dim_ok(batch) || !dim_ok(m) || !dim_ok(n))
    return fail(SOAP_ERR_SHAPE, "batch=%lld m=%lld n=%lld: each must be in [1, %d]",
                (long long)batch, (long long)m, (long long)n, SOAP_MAX_DIM);
  if (iters < 0 || iters > kMuonMaxIters)
    return fail(SOAP_ERR_HPARAM, "n_iters = %lld is outside [0, %lld]", (long long)iters,
                (long long)kMuonMaxIters);
  const Range bufs[] = {{param, sizeof(float) * batch * m * n, "param"},
                        {grad, sizeof(float) * batch * m * n, "grad"},
                        {M, sizeof(float) * batch * m * n, "M"},
                        {ws, ws_bytes, "workspace"}};
  for (const Range &b : bufs)
    if (!b.p) return fail(SOAP_ERR_NULL, "%s is NULL", b.name);
  if (iters > 0 && !coeffs) return fail(SOAP_ERR_NULL, "coeffs is NULL");
  if (!std::isfinite(beta1) || beta1 < 0.f || beta1 >= 1.f)
    return fail(SOAP_ERR_HPARAM, "beta1 = %g is outside [0, 1)", (double)beta1);
  if (!std::isfinite(lr) || lr < 0.f)
    return fail(SOAP_ERR_HPARAM, "lr = %g must be finite and >= 0", (double)lr);
  if (!std::isfinite(wd) || wd < 0.f)
    return fail(SOAP_ERR_HPARAM, "weight_decay = %g must be finite and >= 0", (double)wd);
  if (!std::isfinite(eps) || eps <= 0.f)
    return fail(SOAP_ERR_HPARAM, "eps = %g must be finite and > 0", (double)eps);
  for (int64_t i = 0; i < 3 * iters; ++i)
    if (!std::isfinite(coeffs[i]))
      return fail(SOAP_ERR_HPARAM, "coefficient %lld is not finite", (long long)i);
  if ((flags & ~(uint32_t)SOAP_MUON_BF16) != 0)
    return fail(SOAP_ERR_HPARAM, "unknown flag bits 0x%x", flags);
  const bool bf16 = (flags & SOAP_MUON_BF16) != 0;
  if (bf16 && (m % 8 != 0 || n % 8 != 0))
    return fail(SOAP_ERR_SHAPE, "SOAP_MUON_BF16 needs m and n multiples of 8 (m=%lld n=%lld)",
                (long long)m, (long long)n);
  const MuonLayout lay = muon_layout(batch, m, n);
  if (ws_bytes < lay.total)
    return fail(SOAP_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", ws_bytes, lay.total);
  for (const Range &b : bufs)
    if (!aligned16(b.p)) return fail(SOAP_ERR_ALIGN, "%s is not 16-byte aligned", b.name);
  for (int i = 0; i < 4; ++i)
    for (int j = i + 1; j < 4; ++j)
      if (overlap(bufs[i], bufs[j]))
        return fail(SOAP_ERR_ALIAS, "%s overlaps %s", bufs[i].name, bufs[j].name);

  char *w = static_cast<char *>(ws);
  float *X = reinterpret_cast<float *>(w + lay.x);
  float *Xn = reinterpret_cast<float *>(w + lay.xn);
  float *A = reinterpret_cast<float *>(w + lay.a);
  float *Bm = reinterpret_cast<float *>(w + lay.bm);
  const bool tall = m > n;
  const int64_t d = tall ? n : m, e2 = tall ? m : n;
  const int64_t mn = m * n, dd = d * d;
  const double Bt = (double)batch, dd_ = (double)d, ee = (double)e2;
  hipError_t e;
  {  // M <- b1 M + (1-b1) G
    StageScope sc(ST_MOMENTUM, 0.0, s);
    if ((e = soap::launch_momentum(M, grad, batch * mn, beta1, s)) != hipSuccess)
      return hip_fail(e, "momentum");
  }
  if (bf16) return muon_ns_bf16(batch, param, M, m, n, lr, wd, eps, coeffs, iters, w, lay, s);
  {  // X_0 = M / max(||M||_F, eps)
    StageScope sc(ST_MUON_NORMALISE, 0.0, s);
    if ((e = soap::launch_muon_normalise(M, X, batch, mn, eps,
                                         reinterpret_cast<double *>(w + lay.part),
                                         reinterpret_cast<float *>(w + lay.inv), s)) != hipSuccess)
      return hip_fail(e, "normalise");
  }
  for (int64_t it = 0; it < iters; ++it) {
    const float a = coeffs[3 * it], b = coeffs[3 * it + 1], c = coeffs[3 * it + 2];
    StageScope sc(ST_MUON_NEWTON_SCHULZ,
                  Bt * (dd_ * (dd_ + 1) * ee + (c != 0.f ? 2.0 * dd_ * dd_ * dd_ : 0.0) +
                        2.0 * dd_ * dd_ * ee), s);
    {  // A = X X^T (wide) or X^T X (tall), one triangle mirrored
      soap::GemmDesc g;
      g.trans_a = tall ? 1 : 0; g.trans_b = tall ? 0 : 1;
      g.M = d; g.N = d; g.K = e2;
      g.A = X; g.lda = n; g.sA = mn; g.B = X; g.ldb = n; g.sB = mn;
      g.C = A; g.ldc = d; g.sC = dd; g.alpha = 1.f; g.beta = 0.f; g.batch = batch;
      if ((e = soap::launch_syrk_ema(g, s)) != hipSuccess) return hip_fail(e, "Newton-Schulz A");
    }
    const float *Bop = A;
    float alpha_b = b;
    if (c != 0.f) {  // B = b A + c A^2
      if ((e = soap::launch_copy(Bm, A, batch * dd, s)) != hipSuccess) return hip_fail(e, "copy");
      soap::GemmDesc g;
      g.M = d; g.N = d; g.K = d;
      g.A = A; g.lda = d; g.sA = dd; g.B = A; g.ldb = d; g.sB = dd;
      g.C = Bm; g.ldc = d; g.sC = dd; g.alpha = c; g.beta = b; g.batch = batch;
      if ((e = soap::launch_gemm(g, s)) != hipSuccess) return hip_fail(e, "Newton-Schulz B");
      Bop = Bm;
      alpha_b = 1.f;
    }
    // X <- a X + B X (wide) or a X + X B (tall)
    if ((e = soap::launch_copy(Xn, X, batch * mn, s)) != hipSuccess) return hip_fail(e, "copy");
    soap::GemmDesc g;
    g.M = m; g.N = n; g.K = d;
    if (tall) {
      g.A = X; g.lda = n; g.sA = mn; g.B = Bop; g.ldb = d; g.sB = dd;
    } else {
      g.A = Bop; g.lda = d; g.sA = dd; g.B = X; g.ldb = n; g.sB = mn;
    }
    g.C = Xn; g.ldc = n; g.sC = mn; g.alpha = alpha_b; g.beta = a; g.batch = batch;
    if ((e = soap::launch_gemm(g, s)) != hipSuccess) return hip_fail(e, "Newton-Schulz X");
    std::swap(X, Xn);
  }
  {  // W <- (1 - lr wd) W - lr sqrt(max(m, n)) X_n
    StageScope sc(ST_MUON_UPDATE, 0.0, s);
    const float scale = (float)std::sqrt((double)std::max(m, n));
    if ((e = soap::launch_axpby(param, X, batch * mn, 1.f - lr * wd, -lr * scale, s)) != hipSuccess)
      return hip_fail(e, "update");
  }
  return ok();
}

// ------------------------------------------------ no-allocation step
// Scratch of soap_step_noalloc in place of a caller workspace.  Each GPU that
// loads the library holds its own copy until the process ends.  The array's
// name is not a device address in host code: the address comes from
// hipGetSymbolAddress, once per device with that device current, and only
// that pointer is handed to the kernels.
constexpr size_t kScratchBytes = SOAP_NOALLOC_MAX_WORKSPACE_BYTES;
__device__ __align__(256) unsigned char scratch[kScratchBytes];
std::mutex g_scratch_mu;
void *g_scratch_ptr[64] = {};

hipError_t scratch_address(void **out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    if ((e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

extern "C" {

int soap_step_noalloc(float *param, const float *grad, float *L, float *R, float *Q_L, float *Q_R,
                      float *M, float *V, int64_t m, int64_t n, float beta1, float beta2,
                      float eps, float lr, float weight_decay, int64_t step, uint32_t flags,
                      hipStream_t stream) {
  // Checks that need no device come first (the step repeats them all).
  if (!dim_ok(m) || !dim_ok(n))
    return fail(SOAP_ERR_SHAPE, "m=%lld n=%lld: each must be in [1, %d]", (long long)m,
                (long long)n, SOAP_MAX_DIM);
  const size_t need = step_layout(1, m, n, false).total;
  if (need > kScratchBytes)
    return fail(SOAP_ERR_WORKSPACE,
                "a %lld x %lld step needs %zu bytes of scratch; soap_step_noalloc holds %zu "
                "(call soap_step with a workspace instead)",
                (long long)m, (long long)n, need, kScratchBytes);
  const void *ptrs[] = {param, grad, L, R, Q_L, Q_R, M, V};
  for (const void *p : ptrs)
    if (!p) return fail(SOAP_ERR_NULL, "a state or gradient pointer is NULL");
  int rc = check_hparams(beta1, beta2, eps, lr, weight_decay, step, flags);
  if (rc != SOAP_OK) return rc;
  void *ws = nullptr;
  hipError_t e = scratch_address(&ws);
  if (e != hipSuccess) return hip_fail(e, "scratch address");
  return step_impl(1, param, grad, L, R, Q_L, Q_R, M, V, m, n, beta1, beta2, eps, lr,
                   weight_decay, step, flags, ws, kScratchBytes, stream, false, 0.f);
}

size_t soap_workspace_bytes(int64_t batch, int64_t m, int64_t n) {
  if (!dim_ok(batch) || !dim_ok(m) || !dim_ok(n)) return 0;
  return step_layout(batch, m, n, false).total;
}

int soap_init_state(int64_t batch, int64_t m, int64_t n, float *L, float *R, float *Q_L,
                    float *Q_R, float *M, float *V, hipStream_t stream) {
  if (!dim_ok(batch) || !dim_ok(m) || !dim_ok(n))
    return fail(SOAP_ERR_SHAPE, "batch=%lld m=%lld n=%lld: each must be in [1, %d]",
                (long long)batch, (long long)m, (long long)n, SOAP_MAX_DIM);
  struct T { float *p; int64_t r, c; float d; const char *name; } ts[] = {
      {L, m, m, 1.f, "L"}, {R, n, n, 1.f, "R"}, {Q_L, m, m, 1.f, "Q_L"},
      {Q_R, n, n, 1.f, "Q_R"}, {M, m, n, 0.f, "M"}, {V, m, n, 0.f, "V"}};
  for (const T &t : ts)
    if (t.p && !aligned16(t.p)) return fail(SOAP_ERR_ALIGN, "%s is not 16-byte aligned", t.name);
  for (const T &t : ts) {
    if (!t.p) continue;
    hipError_t e = soap::launch_fill_diag(t.p, batch, t.r, t.c, t.r * t.c, t.d, stream);
    if (e != hipSuccess) return hip_fail(e, "init state");
  }
  return ok();
}

int soap_step(float *param, const float *grad, float *L, float *R, float *Q_L, float *Q_R,
              float *M, float *V, int64_t m, int64_t n, float beta1, float beta2, float eps,
              float lr, float weight_decay, int64_t step, uint32_t flags, void *workspace,
              size_t workspace_bytes, hipStream_t stream) {
  return step_impl(1, param, grad, L, R, Q_L, Q_R, M, V, m, n, beta1, beta2, eps, lr,
                   weight_decay, step, flags, workspace, workspace_bytes, stream, false, 0.f);
}

int soap_step_batched(int64_t batch, float *param, const float *grad, float *L, float *R,
                      float *Q_L, float *Q_R, float *M, float *V, int64_t m, int64_t n,
                      float beta1, float beta2, float eps, float lr, float weight_decay,
                      int64_t step, uint32_t flags, void *workspace, size_t workspace_bytes,
                      hipStream_t stream) {
  return step_impl(batch, param, grad, L, R, Q_L, Q_R, M, V, m, n, beta1, beta2, eps, lr,
                   weight_decay, step, flags, workspace, workspace_bytes, stream, false, 0.f);
}

size_t soap_workspace_update_offset(int64_t batch, int64_t m, int64_t n) {
  if (!dim_ok(batch) || !dim_ok(m) || !dim_ok(n)) return 0;
  return step_layout(batch, m, n, false).nb;
}

size_t soap_kl_workspace_bytes(int64_t batch, int64_t m, int64_t n) {
  if (!dim_ok(batch) || !dim_ok(m) || !dim_ok(n)) return 0;
  return step_layout(batch, m, n, true).total;
}

int soap_kl_step(float *param, const float *grad, float *L, float *R, float *Q_L, float *Q_R,
                 float *M, float *V, int64_t m, int64_t n, float beta1, float beta2,
                 float beta_kron, float eps, float lr, float weight_decay, int64_t step,
                 uint32_t flags, void *workspace, size_t workspace_bytes, hipStream_t stream) {
  return step_impl(1, param, grad, L, R, Q_L, Q_R, M, V, m, n, beta1, beta2, eps, lr,
                   weight_decay, step, flags, workspace, workspace_bytes, stream, true, beta_kron);
}

int soap_kl_step_batched(int64_t batch, float *param, const float *grad, float *L, float *R,
                         float *Q_L, float *Q_R, float *M, float *V, int64_t m, int64_t n,
                         float beta1, float beta2, float beta_kron, float eps, float lr,
                         float weight_decay, int64_t step, uint32_t flags, void *workspace,
                         size_t workspace_bytes, hipStream_t stream) {
  return step_impl(batch, param, grad, L, R, Q_L, Q_R, M, V, m, n, beta1, beta2, eps, lr,
                   weight_decay, step, flags, workspace, workspace_bytes, stream, true, beta_kron);
}

size_t soap_kl_factors_workspace_bytes(int64_t m, int64_t n) {
  if (!dim_ok(m) || !dim_ok(n)) return 0;
  return kl_layout(m, n).total;
}

int soap_kl_factors_f32(int64_t m, int64_t n, const float *G, float *L, float *R,
                        const float *Q_L, const float *Q_R, float beta_kron, float eps,
                        float *lam_L, float *lam_R, void *workspace, size_t workspace_bytes,
                        hipStream_t stream) {
  if (!dim_ok(m) || !dim_ok(n))
    return fail(SOAP_ERR_SHAPE, "m=%lld n=%lld: each must be in [1, %d]", (long long)m,
                (long long)n, SOAP_MAX_DIM);
  if (!std::isfinite(beta_kron) || beta_kron < 0.f || beta_kron >= 1.f)
    return fail(SOAP_ERR_HPARAM, "beta_kron = %g is outside [0, 1)", (double)beta_kron);
  if (!std::isfinite(eps) || eps < 0.f)
    return fail(SOAP_ERR_HPARAM, "eps = %g must be finite and >= 0", (double)eps);
  const Range bufs[] = {{G, sizeof(float) * m * n, "G"},     {L, sizeof(float) * m * m, "L"},
                        {R, sizeof(float) * n * n, "R"},     {Q_L, sizeof(float) * m * m, "Q_L"},
                        {Q_R, sizeof(float) * n * n, "Q_R"}, {workspace, workspace_bytes, "workspace"}};
  for (const Range &b : bufs)
    if (!b.p) return fail(SOAP_ERR_NULL, "%s is NULL", b.name);
  const KlLayout lay = kl_layout(m, n);
  if (workspace_bytes < lay.total)
    return fail(SOAP_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", workspace_bytes, lay.total);
  for (const Range &b : bufs)
    if (!aligned16(b.p)) return fail(SOAP_ERR_ALIGN, "%s is not 16-byte aligned", b.name);
  std::vector<Range> all(bufs, bufs + 6);
  if (lam_L) all.push_back({lam_L, sizeof(float) * m, "lam_L"});
  if (lam_R) all.push_back({lam_R, sizeof(float) * n, "lam_R"});
  for (size_t i = 0; i < all.size(); ++i)
    for (size_t j = i + 1; j < all.size(); ++j)
      if (overlap(all[i], all[j]))
        return fail(SOAP_ERR_ALIAS, "%s overlaps %s", all[i].name, all[j].name);
  char *w = static_cast<char *>(workspace);
  auto at = [&](size_t off) { return reinterpret_cast<float *>(w + off); };
  const KlBufs kb{at(lay.xl), at(lay.xr), at(lay.yl), at(lay.zl), at(lay.yr), at(lay.zr),
                  lam_L ? lam_L : at(lay.laml), lam_R ? lam_R : at(lay.lamr), at(lay.partl),
                  at(lay.partr)};
  StepEvents evs;
  hipError_t e = evs.create();
  if (e != hipSuccess) return hip_fail(e, "event");
  const char *where = "";
  // Both sides on the caller's stream: the events then order nothing new.
  if ((e = kl_accumulate(1, m, n, G, L, R, Q_L, Q_R, beta_kron, eps, kb, stream, stream,
                         evs.ev[0], evs.ev[1], evs.ev[2], &where)) != hipSuccess)
    return hip_fail(e, where);
  return ok();
}

const char *soap_last_error(void) { return g_err; }

int soap_workspace_status(const void *workspace, uint32_t *status, hipStream_t stream) {
  if (!workspace) return fail(SOAP_ERR_NULL, "workspace is NULL");
  uint32_t word = 0;
  hipError_t e = hipMemcpyAsync(&word, workspace, sizeof(word), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return hip_fail(e, "status read");
  if (status) *status = word;
  if (word & ~uint32_t(SOAP_STATUS_QR_L | SOAP_STATUS_QR_R))
    return fail(SOAP_ERR_WORKSPACE, "status word 0x%x has unknown bits: not a step or QR "
                "workspace, or it was overwritten", word);
  if (word)
    return fail(SOAP_ERR_QR_GAVE_UP,
                "the eigenbasis QR of %s gave up waiting for its resident workgroups (other "
                "work held the compute units); that basis was kept as it was",
                word == (SOAP_STATUS_QR_L | SOAP_STATUS_QR_R)
                    ? "both factors"
                    : (word & SOAP_STATUS_QR_L) ? "the m x m factor" : "the n x n factor");
  return ok();
}

int soap_test_force_qr_give_up(uint32_t mask) {
  if (mask & ~uint32_t(SOAP_STATUS_QR_L | SOAP_STATUS_QR_R))
    return fail(SOAP_ERR_HPARAM, "unknown QR bits 0x%x", mask);
  soap::qr_force_give_up(mask);
  return ok();
}

// Workspace of soap_qr_f32: the status word, A^T, the QR's own buffers.
size_t soap_qr_workspace_bytes(int64_t n) {
  if (!dim_ok(n)) return 0;
  return align256(sizeof(uint32_t)) + align256(sizeof(float) * n * n) +
         soap::qr_workspace_bytes(1, n);
}

int soap_qr_f32(int64_t n, const float *A, float *Q, float *Rf, void *workspace,
                size_t workspace_bytes, hipStream_t stream) {
  if (!dim_ok(n)) return fail(SOAP_ERR_SHAPE, "n=%lld must be in [1, %d]", (long long)n, SOAP_MAX_DIM);
  if (!A || !Q || !workspace) return fail(SOAP_ERR_NULL, "A, Q and workspace must be non-NULL");
  const size_t need = soap_qr_workspace_bytes(n);
  if (workspace_bytes < need)
    return fail(SOAP_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", workspace_bytes, need);
  if (!aligned16(A) || !aligned16(Q) || (Rf && !aligned16(Rf)) || !aligned16(workspace))
    return fail(SOAP_ERR_ALIGN, "pointers must be 16-byte aligned");
  const Range rs[] = {{A, sizeof(float) * n * n, "A"}, {Q, sizeof(float) * n * n, "Q"},
                      {Rf ? Rf : Q, Rf ? sizeof(float) * n * n : 0, "Rf"},
                      {workspace, workspace_bytes, "workspace"}};
  for (int i = 0; i < 4; ++i)
    for (int j = i + 1; j < 4; ++j)
      if (rs[i].bytes && rs[j].bytes && overlap(rs[i], rs[j]))
        return fail(SOAP_ERR_ALIAS, "%s overlaps %s", rs[i].name, rs[j].name);
  uint32_t *status = static_cast<uint32_t *>(workspace);
  const size_t head = align256(sizeof(uint32_t)) + align256(sizeof(float) * n * n);
  float *Aw = reinterpret_cast<float *>(static_cast<char *>(workspace) + align256(sizeof(uint32_t)));
  char *rest = static_cast<char *>(workspace) + head;
  hipError_t e = soap::launch_zero_u32(status, 1, stream);
  if (e == hipSuccess) e = soap::launch_transpose(Aw, A, n, stream);   // the QR factors A^T
  if (e == hipSuccess) {
    hipStream_t sp = nullptr, st = nullptr;
    if (e == hipSuccess) e = aux_stream(2, &sp);
    if (e == hipSuccess) e = aux_stream(1, &st);
    if (e == hipSuccess)
      e = soap::qr_factor_and_form_q(Aw, Q, Rf, 1, n, rest, workspace_bytes - head, stream, sp,
                                     st, status, SOAP_STATUS_QR_L);
  }
  if (e != hipSuccess) return hip_fail(e, "QR");
  return ok();
}

int soap_gemm_f32(int trans_a, int trans_b, int64_t M, int64_t N, int64_t K, float alpha,
                  const float *A, int64_t lda, const float *B, int64_t ldb, float beta, float *C,
                  int64_t ldc, hipStream_t stream) {
  if (M < 1 || N < 1 || K < 0 || M > (1 << 24) || N > (1 << 24) || K > (1 << 24))
    return fail(SOAP_ERR_SHAPE, "bad GEMM shape M=%lld N=%lld K=%lld", (long long)M,
                (long long)N, (long long)K);
  if (!A || !B || !C) return fail(SOAP_ERR_NULL, "A, B and C must be non-NULL");
  const int64_t ra = trans_a ? K : M, ca = trans_a ? M : K;
  const int64_t rb = trans_b ? N : K, cb = trans_b ? K : N;
  if (lda < std::max<int64_t>(1, ca) || ldb < std::max<int64_t>(1, cb) || ldc < N)
    return fail(SOAP_ERR_SHAPE, "leading dimension too small");
  (void)ra; (void)rb;
  soap::GemmDesc d;
  d.trans_a = trans_a ? 1 : 0; d.trans_b = trans_b ? 1 : 0;
  d.M = M; d.N = N; d.K = K; d.A = A; d.lda = lda; d.B = B; d.ldb = ldb;
  d.C = C; d.ldc = ldc; d.alpha = alpha; d.beta = beta;
  hipError_t e = soap::launch_gemm(d, stream);
  if (e != hipSuccess) return hip_fail(e, "GEMM");
  return ok();
}

int soap_factor_ema_f32(int trans, int64_t m, int64_t n, const float *G, float *F, float beta,
                        hipStream_t stream) {
  if (!dim_ok(m) || !dim_ok(n)) return fail(SOAP_ERR_SHAPE, "bad shape m=%lld n=%lld", (long long)m, (long long)n);
  if (!G || !F) return fail(SOAP_ERR_NULL, "G and F must be non-NULL");
  if (!std::isfinite(beta) || beta < 0.f || beta >= 1.f)
    return fail(SOAP_ERR_HPARAM, "beta = %g is outside [0, 1)", (double)beta);
  const int64_t d = trans ? n : m;
  const Range rg{G, sizeof(float) * m * n, "G"}, rf{F, sizeof(float) * d * d, "F"};
  if (overlap(rg, rf)) return fail(SOAP_ERR_ALIAS, "G overlaps F");
  soap::GemmDesc g;
  g.trans_a = trans ? 1 : 0; g.trans_b = trans ? 0 : 1;
  g.M = d; g.N = d; g.K = trans ? m : n;
  g.A = G; g.lda = n; g.B = G; g.ldb = n;
  g.C = F; g.ldc = d; g.alpha = 1.f - beta; g.beta = beta;
  hipError_t e = soap::launch_syrk_ema(g, stream);
  if (e != hipSuccess) return hip_fail(e, "factor EMA");
  return ok();
}

size_t soap_muon_workspace_bytes(int64_t batch, int64_t m, int64_t n) {
  if (!dim_ok(batch) || !dim_ok(m) || !dim_ok(n)) return 0;
  return muon_layout(batch, m, n).total;
}

int soap_muon_step(float *param, const float *grad, float *M, int64_t m, int64_t n, float beta1,
                   float lr, float weight_decay, float eps, const float *coeffs, int64_t n_iters,
                   uint32_t flags, void *workspace, size_t workspace_bytes, hipStream_t stream) {
  return muon_impl(1, param, grad, M, m, n, beta1, lr, weight_decay, eps, coeffs, n_iters, flags,
                   workspace, workspace_bytes, stream);
}

int soap_muon_step_batched(int64_t batch, float *param, const float *grad, float *M, int64_t m,
                           int64_t n, float beta1, float lr, float weight_decay, float eps,
                           const float *coeffs, int64_t n_iters, uint32_t flags, void *workspace,
                           size_t workspace_bytes, hipStream_t stream) {
  return muon_impl(batch, param, grad, M, m, n, beta1, lr, weight_decay, eps, coeffs, n_iters,
                   flags, workspace, workspace_bytes, stream);
}

int soap_timing_enable(int enable) {
  Timing &t = timing();
  std::lock_guard<std::mutex> g(t.mu);
  t.enabled = enable != 0;
  return SOAP_OK;
}

int soap_timing_num_stages(void) { return ST_COUNT; }

const char *soap_timing_stage_name(int stage) {
  return (stage >= 0 && stage < ST_COUNT) ? kStageNames[stage] : "";
}

int soap_timing_collect(void) {
  Timing &t = timing();
  std::lock_guard<std::mutex> g(t.mu);
  for (Pending &p : t.pending) {
    hipError_t e = hipEventSynchronize(p.b);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, p.a, p.b);
    if (e != hipSuccess) return hip_fail(e, "timing collect");
    t.ms[p.stage] += ms;
    t.launches[p.stage] += 1;
    t.flops[p.stage] += p.flops;
    t.free_events.push_back(p.a);
    t.free_events.push_back(p.b);
  }
  t.pending.clear();
  return ok();
}

int soap_timing_reset(void) {
  Timing &t = timing();
  std::lock_guard<std::mutex> g(t.mu);
  for (int i = 0; i < ST_COUNT; ++i) { t.ms[i] = 0; t.launches[i] = 0; t.flops[i] = 0; }
  return SOAP_OK;
}

int soap_timing_get(int stage, double *total_ms, int64_t *launches, double *flops) {
  if (stage < 0 || stage >= ST_COUNT) return fail(SOAP_ERR_SHAPE, "no stage %d", stage);
  Timing &t = timing();
  std::lock_guard<std::mutex> g(t.mu);
  if (total_ms) *total_ms = t.ms[stage];
  if (launches) *launches = t.launches[stage];
  if (flops) *flops = t.flops[stage];
  return SOAP_OK;
}

}  // extern "C"
