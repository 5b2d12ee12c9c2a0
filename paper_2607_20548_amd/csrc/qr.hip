// Blocked Householder QR with explicit Q, for the SOAP eigenbasis refresh
// (the paper's Algorithm 2 takes QR(L_t Q_L).Q and QR(R_t Q_R).Q every step).
//
// Structure:
//  * Outer blocks of NB = 128 columns.  After an outer block is factored, its
//    reflectors act on the trailing matrix through the compact-WY form
//    H_1 ... H_nb = I - Y T Y^T:  A_trail -= Y (T^T (Y^T A_trail)), three fp32
//    MFMA GEMMs (the first one split over K).  Look-ahead: the next block's
//    columns are updated first, then the next block is factored on a second
//    stream while the rest of the trailing matrix is updated.
//  * An outer block is factored by qr_block_kernel: one launch whose
//    workgroups keep the block in registers and sum the dot products of each
//    column grid-wide (see the comment above the kernel).  It needs all of
//    its workgroups resident; batches too large for that take the panel
//    path:
//  * Panel path: inner panels of width b in {16, 8, 4} are each factored by
//    ONE 512-thread workgroup that holds the whole panel (rows ci..n-1, b
//    columns) in registers (wave64 butterfly reductions, two barriers per
//    column); a row-split reduction then forms the panel's T block, the T
//    column and the update coefficients, and a row-parallel apply updates the
//    rest of the outer block.
//  * Q is formed backwards, Q[c:, c:] -= Y (T (Y^T Q[c:, c:])), starting from
//    diag(d).
//
// Reflector convention (as in LAPACK's larfg): for x = A[j:, j] with
// s = ||x[1:]||^2 and sigma = ||x||, v0 = x0 + sgn(x0) sigma (sgn(0) = +1),
// v = x / v0 (so v[0] = 1), beta = 2 v0^2 / (s + v0^2), and H x = -sgn(x0) sigma e_1.
// |v0| >= |x0| keeps every |v_i| <= 1 and beta in [1, 2], which keeps the
// compact-WY products well scaled in fp32.  (The opposite choice, which makes
// R's diagonal positive directly, produces Householder vectors of size
// 1e4..1e5 on the near-identity matrices L Q of SOAP and loses about two
// digits in the blocked form.)  s == 0 means the column is already
// triangular: H = I.  The diagonal of R then has signs d_j; the unique Q with
// non-negative diag(R) is Q_house diag(d), obtained by starting the backward
// accumulation of Q from diag(d) instead of I.
//
// Storage: the matrix is factored in transposed form, At = A^T row-major (so
// At[col * n + row] = A[row][col]).  A panel's columns are then contiguous
// rows of At and every panel load and store is coalesced; the compact-WY
// GEMMs take the transposition through their operand flags.  After factoring,
// At holds R above the outer-block diagonal blocks (transposed) and, inside
// every outer block, the explicit unit lower-trapezoidal Y (zeros above its
// diagonal, ones on it), which the GEMMs read directly.
#include "internal.h"

#include <algorithm>
#include <atomic>
#include <mutex>
#include <vector>

namespace soap {
namespace {

constexpr int NB = 128;            // outer block width
constexpr int PANEL_THREADS = 512;
constexpr int PANEL_WAVES = PANEL_THREADS / 64;
constexpr int RCH = 256;           // rows per workgroup in the inner reduction
constexpr int RED_THREADS = 1024;  // threads of the inner reduction
constexpr int APPLY_ROWS = 8;      // rows per workgroup in the inner apply
constexpr int MAX_B = 32;
constexpr int MAX_PANEL = 16;      // widest inner panel
constexpr int PART_STRIDE = MAX_B * NB;   // floats per partial block

// --------------------------------------------------------------- reductions
// Sum of NV values over the panel workgroup; the NV totals are left in tot
// (LDS) for every thread to read.  Each value is summed over the wave with
// xor shuffles (no lane-dependent selects: a transposed butterfly would need
// per-lane choices of which half to keep, which the compiler lowers to
// compare/select chains over the whole array), then across waves in LDS.
// red: [PANEL_WAVES][NV] in LDS.
template <int NV>
__device__ __forceinline__ void block_allreduce(float (&v)[NV], float *red, float *tot) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int mask = 32; mask >= 1; mask >>= 1)
#pragma unroll
    for (int i = 0; i < NV; ++i) v[i] += __shfl_xor(v[i], mask);
  if (lane == 0) {
#pragma unroll
    for (int i = 0; i < NV; ++i) red[wave * NV + i] = v[i];
  }
  __syncthreads();
  if (threadIdx.x < NV) {
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < PANEL_WAVES; ++w) s += red[w * NV + threadIdx.x];
    tot[threadIdx.x] = s;
  }
  __syncthreads();
}

// Copies a rows x cols block (row strides sld, dld) from global memory to LDS
// with NT threads, keeping 8 loads in flight per thread.
template <int NT>
__device__ __forceinline__ void stage_block(float *dst, int dld, const float *src, int sld,
                                            int rows, int cols) {
  const int total = rows * cols;
  for (int base = threadIdx.x; base < total; base += 8 * NT) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = base + u * NT;
      v[u] = (e < total) ? src[(e / cols) * sld + e % cols] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = base + u * NT;
      if (e < total) dst[(e / cols) * dld + e % cols] = v[u];
    }
  }
}

struct PanelParams {
  float *At;         // batch of transposed n x n matrices (At[col*n + row])
  int64_t sA;
  int n;
  int c;             // first column of the outer block
  int ci;            // first column of this panel
  int beff;          // panel width actually used (<= B)
  float *T;          // T of this outer block: NB x NB row-major, batch stride sT
  int64_t sT;
  float *Rf;         // optional triangular-factor output, row-major (batch stride sA)
  float *dsign;      // sign of each R diagonal entry, n per matrix
  float *beta;       // reflector coefficient of each column, n per matrix
};

// Factors A[ci:n, ci:ci+beff] in registers; writes Y back (zeros above the
// diagonal inside the outer block, ones on it), the reflector coefficients,
// the R-diagonal signs and, if requested, the R entries of these columns for
// rows c .. ci+beff-1.  Thread t owns rows ci + t + PANEL_THREADS*s.  (The
// panel's block of T is formed by the row-parallel reduction that follows.)
template <int B, int RPT>
__global__ __launch_bounds__(PANEL_THREADS) void qr_panel_kernel(PanelParams p) {
  static_assert(B * RPT <= 128, "panel must fit in 128 registers per thread");
  __shared__ float red[PANEL_WAVES * B];
  __shared__ float tot[B];
  __shared__ float piv[2][B];

  const int64_t bz = blockIdx.x;
  float *At = p.At + bz * p.sA;
  float *Rf = p.Rf ? p.Rf + bz * p.sA : nullptr;
  const int n = p.n, ci = p.ci, c = p.c, beff = p.beff;
  const int N = n - ci;
  const int t = threadIdx.x;
  const unsigned un = (unsigned)n;   // n*n < 2^31: 32-bit offsets within a matrix

  // R entries above this panel inside the outer block: rows c..ci-1.
  for (int e = t; e < (ci - c) * beff; e += PANEL_THREADS) {
    const int j = e / (ci - c), r = c + e % (ci - c);
    const unsigned off = (unsigned)(ci + j) * un + r;
    if (Rf) Rf[(unsigned)r * un + ci + j] = At[off];
    At[off] = 0.f;
  }

  float a[RPT][B];
#pragma unroll
  for (int s = 0; s < RPT; ++s) {
    const int lr = t + PANEL_THREADS * s;
#pragma unroll
    for (int j = 0; j < B; ++j)
      a[s][j] = (lr < N && j < beff) ? At[(unsigned)(ci + j) * un + ci + lr] : 0.f;
  }
  // Column loop, fully unrolled: j is a compile-time index, so every register
  // access is static and finished columns cost nothing.  The guard j < beff
  // is uniform across the workgroup.
#pragma unroll
  for (int j = 0; j < B; ++j) {
    if (j < beff) {
      float *pv = piv[j & 1];
      if (t == j) {
#pragma unroll
        for (int cc = 0; cc < B; ++cc)
          if (cc >= j) pv[cc] = a[0][cc];
      }
      float v[B];
#pragma unroll
      for (int cc = 0; cc < B; ++cc) v[cc] = 0.f;
#pragma unroll
      for (int s = 0; s < RPT; ++s) {
        const int lr = t + PANEL_THREADS * s;
        float x = 0.f;
#pragma unroll
        for (int cc = 0; cc < B; ++cc)
          if (cc == j) x = a[s][cc];
        const float y = (lr > j && lr < N) ? x : 0.f;
#pragma unroll
        for (int cc = 0; cc < B; ++cc)
          if (cc >= j) v[cc] += y * a[s][cc];
      }
      block_allreduce<B>(v, red, tot);
      const float x0 = pv[j];
      const float st = tot[j];
      float beta, inv_v0, rjj;
      if (st == 0.f) {          // already triangular: H = I
        inv_v0 = 0.f;
        beta = 0.f;
        rjj = x0;
      } else {
        const float sigma = sqrtf(x0 * x0 + st);
        const float v0 = (x0 >= 0.f) ? (x0 + sigma) : (x0 - sigma);
        beta = 2.f * v0 * v0 / (st + v0 * v0);
        inv_v0 = 1.f / v0;
        rjj = (x0 >= 0.f) ? -sigma : sigma;
      }
      float f[B];   // beta * v^T a_cc for the columns right of j
#pragma unroll
      for (int cc = 0; cc < B; ++cc)
        f[cc] = (cc > j) ? beta * (pv[cc] + tot[cc] * inv_v0) : 0.f;
#pragma unroll
      for (int s = 0; s < RPT; ++s) {
        const int lr = t + PANEL_THREADS * s;
        const bool live = (lr > j) && (lr < N);
        float x = 0.f;
#pragma unroll
        for (int cc = 0; cc < B; ++cc)
          if (cc == j) x = a[s][cc];
        const float y = live ? x * inv_v0 : 0.f;   // Householder vector entry
#pragma unroll
        for (int cc = 0; cc < B; ++cc) {
          if (cc > j) a[s][cc] -= f[cc] * y;
          if (cc == j) a[s][cc] = live ? y : a[s][cc];
        }
      }
      if (t == j) {
#pragma unroll
        for (int cc = 0; cc < B; ++cc) {
          if (cc > j) a[0][cc] -= f[cc];
          if (cc == j) a[0][cc] = rjj;
        }
      }
      if (t == 0) {
        p.beta[bz * n + ci + j] = beta;
        p.dsign[bz * n + ci + j] = (rjj < 0.f) ? -1.f : 1.f;
      }
    }
  }

  // Write Y (explicit zeros above its diagonal, ones on it) and the R entries.
#pragma unroll
  for (int s = 0; s < RPT; ++s) {
    const int lr = t + PANEL_THREADS * s;
    if (lr >= N) continue;
#pragma unroll
    for (int j = 0; j < B; ++j) {
      if (j < beff) {
        if (lr <= j && Rf) Rf[(unsigned)(ci + lr) * un + ci + j] = a[s][j];
        At[(unsigned)(ci + j) * un + ci + lr] = (lr > j) ? a[s][j] : (lr == j ? 1.f : 0.f);
      }
    }
  }
}

struct InnerParams {
  float *At;
  int64_t sA;
  int n, c, ci, b, cend;
  float *T;           // outer-block T, batch stride sT
  int64_t sT;
  const float *beta;  // reflector coefficients, n per matrix
  float *Wi;          // b x w output (T_p^T Y_p^T A_rest), batch stride sW
  int64_t sW;
  float *part;        // partial products, batch stride sP (P * PART_STRIDE)
  int64_t sP;
  unsigned *cnt;      // one arrival counter per matrix (zero between uses)
  int P;              // workgroups per matrix
};

constexpr int TS = RCH + 1;   // LDS column stride of the reduction tile (bank spread)

// One workgroup per RCH rows computes O = Y_p^T [Y_prev | Y_p | A_rest] over
// its rows (Y_p = this panel's reflectors, Y_prev = the earlier panels of the
// outer block, A_rest = the outer block's columns right of the panel).  The
// last workgroup to arrive (per matrix) sums the partials in workgroup order
// and forms, from G = Y_p^T Y_p, X = Y_prev^T Y_p and W = Y_p^T A_rest:
//   T_p (upper triangular):  T_p[j][j] = beta_j,
//                            T_p[0:j, j] = -beta_j T_p[0:j, 0:j] G[0:j, j]
//   the T column block:      T[0:off, off:off+b] = -T[0:off, 0:off] X T_p
//   the update coefficients: Wi = T_p^T W.
__global__ __launch_bounds__(RED_THREADS) void qr_inner_reduce_kernel(InnerParams p) {
  // Column-major tile of the outer block's rows r0..r0+RCH-1.  Once the
  // partials are written the last workgroup reuses it for the summed partials
  // (Os: b x NB), the Z block (Zs: NB x MAX_B) and T (Ts: NB x NB).
  __shared__ float tile[NB * TS];
  __shared__ int last;
  float *Os = tile;
  float *Zs = tile + MAX_B * NB;
  float *Ts = tile + 2 * MAX_B * NB;
  const int64_t bz = blockIdx.y;
  const int g = blockIdx.x;
  const float *At = p.At + bz * p.sA;
  const int n = p.n, c = p.c, ci = p.ci, b = p.b;
  const int ncol = p.cend - c;
  const int off = ci - c;
  const int w = p.cend - (ci + b);
  const int r0 = ci + g * RCH;
  const int rows = min(RCH, n - r0);
  const int t = threadIdx.x;

  // tile load: thread -> (row, group of 32 columns); 32 coalesced loads in
  // flight.  Rows past the end are zero-filled (they enter the contraction).
  {
    const int rr = t & (RCH - 1), cg = t / RCH;    // 4 column groups
    const float *src = At + (int64_t)(c + 32 * cg) * n + r0 + rr;
    float v[32];
#pragma unroll
    for (int u = 0; u < 32; ++u)
      v[u] = (rr < rows && 32 * cg + u < ncol) ? src[(int64_t)u * n] : 0.f;
#pragma unroll
    for (int u = 0; u < 32; ++u) tile[(32 * cg + u) * TS + rr] = v[u];
  }
  __syncthreads();

  // O[i][q] = sum_rows Y_p[row][i] * X[row][q] on the matrix cores: wave w < 8
  // owns the 16 x 16 block q in [16w, 16w+16) (i < 16 covers any panel width),
  // v_mfma_f32_16x16x4_f32 over the 256 rows.  The K order is permuted: at
  // step s, lane group g = lane/16 takes row 64 g + s, so each lane reads four
  // consecutive rows of its tile column with one 16-byte LDS read.
  const int lane = t & 63, wave = t >> 6;
  float *part = p.part + bz * p.sP + (int64_t)g * PART_STRIDE;
  if (wave < 8) {
    typedef float v4f __attribute__((ext_vector_type(4)));
    const int i = lane & 15, grp = lane >> 4;
    const int q = 16 * wave + i;
    // A operand: Y_p column i (zero beyond the panel width); B operand: column q
    const float *acol = tile + (off + (i < b ? i : 0)) * TS + 64 * grp;
    const float *bcol = tile + q * TS + 64 * grp;
    const float amask = (i < b) ? 1.f : 0.f;
    v4f acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
    for (int s4 = 0; s4 < 64; s4 += 4) {
      float a4[4], b4[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) { a4[u] = acol[s4 + u] * amask; b4[u] = bcol[s4 + u]; }
#pragma unroll
      for (int u = 0; u < 4; ++u) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[u], b4[u], acc, 0, 0, 0);
    }
    // accumulator r of lane l holds O[4*(l/16) + r][16*wave + l%16]
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int ii = 4 * grp + r;
      if (ii < b && q < ncol) part[ii * NB + q] = acc[r];
    }
  }
  __threadfence();
  __syncthreads();
  if (t == 0) {
    const unsigned prev = atomicAdd(p.cnt + bz, 1u);
    last = (prev == (unsigned)(p.P - 1));
  }
  __syncthreads();
  if (!last) return;
  __threadfence();

  float *T = p.T + bz * p.sT;
  const float *beta = p.beta + bz * p.n + ci;
  stage_block<RED_THREADS>(Ts, NB, T, NB, off, off);
  const float *pb = p.part + bz * p.sP;
  for (int e = t; e < b * ncol; e += RED_THREADS) {
    const int jj = e / ncol, qq = e - jj * ncol;
    const float *src = pb + jj * NB + qq;
    float s[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) s[u] = 0.f;
    for (int gg = 0; gg < p.P; gg += 16) {
#pragma unroll
      for (int u = 0; u < 16; ++u)
        if (gg + u < p.P) s[u] += src[(int64_t)(gg + u) * PART_STRIDE];
    }
    float tot16 = 0.f;
#pragma unroll
    for (int u = 0; u < 16; ++u) tot16 += s[u];
    Os[jj * NB + qq] = tot16;
  }
  __syncthreads();
  // T_p by wave 0: lane i keeps row i of T_p in registers; everything is
  // unrolled over the (at most 16) panel columns, so there is no barrier and
  // no dependent LDS round trip inside the recurrence.
  //   T_p[j][j] = beta_j,  T_p[i][j] = -beta_j sum_{l=i}^{j-1} T_p[i][l] G[l][j],
  // with G[l][j] = Os[l][off + j] (the panel's Gram matrix).
  if (t < 64) {
    const int i = t;
    float trow[MAX_PANEL];
#pragma unroll
    for (int j = 0; j < MAX_PANEL; ++j) {
      float val = 0.f;
      if (j < b) {
        const float bj = beta[j];
        float acc = 0.f;
#pragma unroll
        for (int l = 0; l < j; ++l)
          if (l >= i) acc += trow[l] * Os[l * NB + off + j];
        val = (i == j) ? bj : (i < j ? -bj * acc : 0.f);
      }
      trow[j] = val;
    }
    if (i < b) {
#pragma unroll
      for (int j = 0; j < MAX_PANEL; ++j)
        if (j < b) Ts[(off + i) * NB + off + j] = trow[j];
    }
  }
  __syncthreads();
  // rows off..off+b of T: zeros left of the diagonal block, then T_p
  for (int e = t; e < b * (off + b); e += RED_THREADS) {
    const int i = e / (off + b), jc = e % (off + b);
    T[(off + i) * NB + jc] = (jc < off) ? 0.f : Ts[(off + i) * NB + jc];
  }
  // Wi[jj][q] = sum_{l <= jj} T_p[l][jj] * W[l][q],  W[l][q] = Os[l][off + b + q]
  float *Wi = p.Wi + bz * p.sW;
  for (int e = t; e < b * w; e += RED_THREADS) {
    const int jj = e / w, qq = e - jj * w;
    float s = 0.f;
#pragma unroll
    for (int l = 0; l < MAX_PANEL; ++l)
      if (l <= jj) s += Ts[(off + l) * NB + off + jj] * Os[l * NB + off + b + qq];
    Wi[jj * w + qq] = s;
  }
  if (off > 0) {
    // Z[i][jj] = sum_{l <= jj} X[i][l] T_p[l][jj],  X[i][l] = Os[l][i]
    for (int e = t; e < off * b; e += RED_THREADS) {
      const int i = e / b, jj = e - i * b;
      float s = 0.f;
#pragma unroll
      for (int l = 0; l < MAX_PANEL; ++l)
        if (l <= jj) s += Os[l * NB + i] * Ts[(off + l) * NB + off + jj];
      Zs[i * MAX_B + jj] = s;
    }
    __syncthreads();
    // T[i][off + jj] = -sum_{l = i}^{off-1} T[i][l] Z[l][jj]
    for (int e = t; e < off * b; e += RED_THREADS) {
      const int i = e / b, jj = e - i * b;
      float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
      int l = i;
      for (; l + 4 <= off; l += 4) {
        s0 += Ts[i * NB + l + 0] * Zs[(l + 0) * MAX_B + jj];
        s1 += Ts[i * NB + l + 1] * Zs[(l + 1) * MAX_B + jj];
        s2 += Ts[i * NB + l + 2] * Zs[(l + 2) * MAX_B + jj];
        s3 += Ts[i * NB + l + 3] * Zs[(l + 3) * MAX_B + jj];
      }
      for (; l < off; ++l) s0 += Ts[i * NB + l] * Zs[l * MAX_B + jj];
      T[i * NB + off + jj] = -((s0 + s1) + (s2 + s3));
    }
  }
  if (t == 0) p.cnt[bz] = 0u;
}

struct ApplyParams {
  float *At;
  int64_t sA;
  int n, ci, b, w;
  const float *Wi;
  int64_t sW;
};

// A[r][ci+b+q] -= sum_l Y[r][l] Wi[l][q] for rows r >= ci; one thread per row
// so that every access to At (column-major A) is coalesced.
__global__ __launch_bounds__(256) void qr_inner_apply_kernel(ApplyParams p) {
  __shared__ float Ws[MAX_B * NB];
  const int64_t bz = blockIdx.y;
  float *At = p.At + bz * p.sA;
  const float *Wi = p.Wi + bz * p.sW;
  const int n = p.n, ci = p.ci, b = p.b, w = p.w;
  const int t = threadIdx.x;
  stage_block<256>(Ws, NB, Wi, w, b, w);
  __syncthreads();
  const int r = ci + blockIdx.x * 256 + t;
  if (r >= n) return;
  float y[MAX_B];
#pragma unroll
  for (int l = 0; l < MAX_B; ++l) y[l] = (l < b) ? At[(int64_t)(ci + l) * n + r] : 0.f;
  float *dst = At + (int64_t)(ci + b) * n + r;
  int q = 0;
  for (; q + 8 <= w; q += 8) {
    float cur[8], s[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) { cur[u] = dst[(int64_t)(q + u) * n]; s[u] = 0.f; }
#pragma unroll
    for (int l = 0; l < MAX_B; ++l)
#pragma unroll
      for (int u = 0; u < 8; ++u) s[u] += y[l] * Ws[l * NB + q + u];
#pragma unroll
    for (int u = 0; u < 8; ++u) dst[(int64_t)(q + u) * n] = cur[u] - s[u];
  }
  for (; q < w; ++q) {
    float s = 0.f;
#pragma unroll
    for (int l = 0; l < MAX_B; ++l) s += y[l] * Ws[l * NB + q];
    dst[(int64_t)q * n] -= s;
  }
}

// ------------------------------------------------ resident-block factorization
// One launch factors a whole outer block (rows c..n-1, nb <= NB columns) with
// the same reflectors as the panel path.  Workgroup g keeps rows
// c + g*BK_ROWS .. c + (g+1)*BK_ROWS - 1 of the block in registers: the eight
// lanes 8q..8q+7 of wave w own column k = 16q + w (so every wave keeps the
// same number of active columns as the factorization advances) and lane part
// holds the local rows 32 i + 4 part + e (i < BK_R/4, e < 4): 32 values per
// lane and four waves per SIMD to hide the latency of each round.  The columns
// are taken in rounds of up to BK_KMAX.  Per round (pivot columns j..j+K-1):
//   * the pivot columns are broadcast through LDS, pivot j+i with its rows up
//     to j+i cleared (its tail y_i), and every thread forms the partial dots
//     of its column with every tail;
//   * the partials are summed grid-wide in one hop through global memory:
//     each workgroup posts its partials, workgroup 0 also the column's values
//     in the diagonal rows j..j+K-1, and every workgroup reads back the P
//     partials of each dot of the columns it needs and sums them in one
//     fixed order, so that all of them hold bit-identical totals;
//   * from the totals of the pivot columns, every thread (rounds of up to
//     four columns) or wave 0 with one lane per pivot (more) forms the
//     round's reflectors (Gram recurrence below), and every thread applies
//     them to its own column as one combination of the tails.
// Workgroup 0 holds the block's diagonal rows: its broadcasts are zero at and
// above each pivot's diagonal row (so its dot products need no masks), and it
// keeps S = strict upper part of Y^T Y (from the same dot products), from
// which it forms T after the column loop,
//   T[k][k] = beta_k,  T[k][j] = -beta_j sum_{l=k}^{j-1} T[k][l] S[l][j]  (j > k),
// by blocks of 8 columns (the diagonal blocks by this recurrence, the others
// by T_IJ = -(sum_{K=I}^{J-1} T_IK S_KJ) T_JJ).
// The launch needs all of its workgroups resident at once; the host limits it
// to BK_MAX_WG workgroups and to what the device can hold at once (an
// occupancy query).  Waits are bounded: one that exceeds BK_SPIN_LIMIT polls
// raises a per-matrix abort flag, after which every wait returns at once and
// the block is written as NaN, so the kernel always ends.  A workgroup that
// saw the abort marks the matrix's factorization failed (the Q formation
// then leaves that matrix's Q as it was) and or-s the caller's status bit
// into its status word.
constexpr int BK_THREADS = 1024;
constexpr int BK_WAVES = BK_THREADS / 64;
constexpr int BK_PARTS = 8;                     // threads per column
constexpr int BK_R = 32;                        // rows per thread
constexpr int BK_ROWS = BK_PARTS * BK_R;        // rows per workgroup
// Blocks with few rows take half as many rows per thread (twice the
// workgroups): the work of each round halves while the exchange grows by P
// items per column (with four-column rounds, measured on the 4096 x 4096 and
// 24-layer steps: best up to 24 workgroups, 16 and 32 slightly slower, 40
// slower still).
constexpr int BK_R_SMALL = 16;
constexpr int BK_ROWS_SMALL = BK_PARTS * BK_R_SMALL;
constexpr int BK_SMALL_MAX_P = 24;
constexpr int BK_LI = 4 * BK_PARTS;             // local-row stride of a thread's register groups
constexpr int BK_MAX_P = 64;                    // workgroups per matrix (n <= 16384)
constexpr int BK_MAX_WG = 96;                   // workgroups per launch
constexpr unsigned BK_SPIN_LIMIT = 1u << 22;
constexpr int BK_TSTR = NB + 4;                 // LDS row stride of T and S (spreads banks)
constexpr int BK_KMAX = 8;                      // columns per round at most
// A round stops before pivot j+i (i > 0) when the reflectors j..j+i-1 leave
// less than this fraction of its squared norm (rows j+i.. after them against
// rows j.. before them): the sums that give its reflector would lose digits
// to cancellation.
constexpr float BK_TAU = 0.0625f;
// Exchange area per matrix, in 32-bit words: a header (the abort flag, the
// failed flag, and per slot area the words written there since it was last
// emptied), then two slot areas that the outer blocks use in turn.  A round
// of a block with P workgroups has a slot of its own, bk_col_words(P) items
// of NB columns each: [BK_KMAX][P] partials of the dots (pivot i, workgroup g
// is item i * P + g), then the BK_KMAX values of workgroup 0 in the diagonal
// rows; item e of column k at word e * NB + (k mod 8) * 16 + k / 8 (the
// columns of one wave are adjacent, so that one load by a wave touches few
// cache lines).  Every word is written at most once between two
// emptyings, over the empty pattern BK_EMPTY (a NaN that no post carries:
// posted NaNs are canonical), so a reader knows a value has arrived from its
// bits alone.  A block kernel empties, after its rounds, what the previous
// block wrote into the area that the next block uses.
constexpr int64_t BK_XABORT = 0;
constexpr int64_t BK_XFAILED = 1;
constexpr int64_t BK_XUSED = 2;                 // words 2, 3: written words of area 0, 1
constexpr int64_t BK_XHDR = 64;
constexpr unsigned BK_EMPTY = 0xFFFFFFFFu;
// Workgroups of the widest block launch for order n (the big-R kernel at
// block 0, or the small-R kernel where it is taken).
constexpr int64_t bk_max_p(int64_t n) {
  const int64_t big = (n + BK_ROWS - 1) / BK_ROWS;
  const int64_t sm = (n + BK_ROWS_SMALL - 1) / BK_ROWS_SMALL;
  const int64_t s2 = sm < BK_SMALL_MAX_P ? sm : BK_SMALL_MAX_P;
  return big > s2 ? big : s2;
}
__host__ __device__ constexpr int64_t bk_col_words(int64_t P) { return BK_KMAX * P + BK_KMAX; }
// words of one slot area: at most NB rounds per block
constexpr int64_t bk_area_words(int64_t n) { return (int64_t)NB * NB * bk_col_words(bk_max_p(n)); }
constexpr int64_t bk_xstride(int64_t n) { return BK_XHDR + 2 * bk_area_words(n); }

struct BlockParams {
  float *At;
  int64_t sA;
  int n, c, nb;
  float *T;                  // this block's T (NB x NB row-major), batch stride sT
  int64_t sT;
  float *Rf;                 // optional triangular-factor output (batch stride sA)
  float *dsign, *beta;       // n per matrix
  unsigned *xch;             // exchange area, xstride words per matrix
  int64_t xstride, area_words;
  int area;                  // slot area of this block (0 or 1)
  int P;                     // workgroups per matrix
  unsigned *status;          // caller's status word (or nullptr) ...
  unsigned status_bit;       // ... and the bit a give-up or-s into it
};

__device__ __forceinline__ void bk_put(unsigned *p, float v) {
  const unsigned w = (v != v) ? 0x7FC00000u : __float_as_uint(v);   // never BK_EMPTY
  __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ unsigned bk_get(const unsigned *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// One failed poll: counts it, raises the abort flag past the limit, and
// reports whether the wait must end (limit reached or abort seen).  Polls
// back off (s_sleep grows to about 0.2 us) so that waiting workgroups do not
// crowd out the stores they wait for.
__device__ __forceinline__ bool bk_give_up(unsigned &spins, unsigned *abort_flag) {
  ++spins;
  if (spins >= BK_SPIN_LIMIT) {
    __hip_atomic_store(abort_flag, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return true;
  }
  if ((spins & 63u) == 0u &&
      __hip_atomic_load(abort_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u)
    return true;
  if (spins < 4) __builtin_amdgcn_s_sleep(1);
  else if (spins < 16) __builtin_amdgcn_s_sleep(2);
  else __builtin_amdgcn_s_sleep(4);
  return false;
}

// Waits for the cnt <= H items at byte offsets off + 4 NB i (i < cnt) of the
// buffer r and, if xoff >= 0, the item at byte offset xoff, re-reading only
// those still empty; returns the sum of the first in index order and the
// value of x.  The loads take the cache policy of an agent-scope load (sc1,
// as the atomic loads above) through a buffer resource, so that one offset
// register and the instruction's offset field address every item.  All
// pending items are fetched at once (their loads issued before any is
// examined), so a poll costs about one memory latency however many items
// there are.  false: aborted.
constexpr int BK_LOAD_AGENT = 16;   // cache policy operand: sc1
constexpr int BK_RSRC_WORD3 = 0x00020000;   // buffer resource: raw 32-bit data
template <int H>
__device__ __forceinline__ bool bk_gather(__amdgpu_buffer_rsrc_t r, unsigned off, int cnt,
                                          int xoff, unsigned *abort_flag, float &sum, float &xv) {
  static_assert(H <= 32, "one pending bit per item");
  unsigned v[H];
  unsigned pending = cnt >= 32 ? 0xFFFFFFFFu : ((1u << cnt) - 1u);
  bool hx = xoff < 0;
  unsigned spins = 0;
  for (;;) {
    // a new offset value each poll as far as the compiler knows: the loads
    // are issued again, not kept from the previous poll
    asm volatile("" : "+v"(off));
    unsigned vx = 0;
    if (!hx) vx = __builtin_amdgcn_raw_buffer_load_b32(r, xoff + (int)(off & 0u), 0, BK_LOAD_AGENT);
#pragma unroll
    for (int i = 0; i < H; ++i)
      if (pending & (1u << i))
        v[i] = __builtin_amdgcn_raw_buffer_load_b32(r, (int)(off + (unsigned)(i * NB * 4)), 0,
                                                    BK_LOAD_AGENT);
    unsigned still = pending;
#pragma unroll
    for (int i = 0; i < H; ++i)
      if ((pending & (1u << i)) && v[i] != BK_EMPTY) still &= ~(1u << i);
    if (!hx && vx != BK_EMPTY) {
      xv = __uint_as_float(vx);
      hx = true;
    }
    pending = still;
    if (pending == 0u && hx) break;
    if (bk_give_up(spins, abort_flag)) return false;
  }
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < H; ++i)
    if (i < cnt) s += __uint_as_float(v[i]);
  sum = s;
  return true;
}

// Lane exchanges inside the 8 lanes of a column (lanes 8q..8q+7, one half of
// a DPP row) by DPP moves, which take no LDS round trip: bk_sum2, bk_sum4 and
// bk_sum8 leave in every lane the sum over its aligned group of 2, 4 and 8
// lanes.  Additions are commutative, so every lane of a group holds a
// bit-identical result.
template <int CTRL>
__device__ __forceinline__ float bk_mov(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, false));
}
constexpr int DPP_XOR1 = 0xB1;         // quad_perm [1, 0, 3, 2]
constexpr int DPP_XOR2 = 0x4E;         // quad_perm [2, 3, 0, 1]
constexpr int DPP_HALF_MIRROR = 0x141; // lane i <- lane 7 - i within 8 lanes
__device__ __forceinline__ float bk_sum2(float v) { return v + bk_mov<DPP_XOR1>(v); }
__device__ __forceinline__ float bk_sum4(float v) {
  v = bk_sum2(v);
  return v + bk_mov<DPP_XOR2>(v);
}
__device__ __forceinline__ float bk_sum8(float v) {
  v = bk_sum4(v);
  return v + bk_mov<DPP_HALF_MIRROR>(v);
}

// a[idx / 4][idx % 4] = v for a wave-uniform or lane-varying idx < 4 NQ (a
// compare per candidate register instead of a select chain over the rows).
template <int NQ, int NI>
__device__ __forceinline__ void bk_reg_set(float (&a)[NI][4], int idx, float v) {
#pragma unroll
  for (int q = 0; q < 4 * NQ; ++q)
    if (q == idx) a[q >> 2][q & 3] = v;
}

// Householder reflector of a column with diagonal value x0 and tail sum of
// squares st (the larfg convention above): beta, 1 / v0 and the R diagonal.
// st == 0: the column is already triangular, H = I.
__device__ __forceinline__ void bk_reflector(float x0, float st, float &bet, float &inv_v0,
                                             float &rjj) {
  if (st == 0.f) {
    bet = 0.f;
    inv_v0 = 0.f;
    rjj = x0;
  } else {
    // hardware square root and reciprocals (1 ulp each): beta is formed from
    // v0 as computed, so the reflector stays orthogonal to rounding
    const float sigma = __builtin_amdgcn_sqrtf(x0 * x0 + st);
    const float v0 = (x0 >= 0.f) ? (x0 + sigma) : (x0 - sigma);
    bet = 2.f * v0 * v0 * __builtin_amdgcn_rcpf(st + v0 * v0);
    inv_v0 = __builtin_amdgcn_rcpf(v0);
    rjj = (x0 >= 0.f) ? -sigma : sigma;
  }
}

// Columns per round of the block kernels: up to eight with 16 rows per
// thread (BK_R_SMALL) and with 32 rows per thread for launches of at most
// BK_MID_MAX_P workgroups (the gather then holds one dot's P partials per
// lane), four for the wider 32-row launches (two lanes per dot).
constexpr int BK_K_BIG = 4;
constexpr int BK_K_MID = 8;
constexpr int BK_MID_MAX_P = 16;
constexpr int BK_K_SMALL = 8;
// Parameters of one reflector of a round of more than four columns, as the
// column loop reads them (an LDS row of bk_prm_words(K) floats): beta, 1/v0,
// R diagonal, (unused), gamma_i[l], c_i[l], p_l[i] (l < K).
constexpr int bk_prm_words(int K) { return 4 + 3 * K; }

template <int R, int KM>
__global__ __launch_bounds__(BK_THREADS) void qr_block_kernel(BlockParams p) {
  static_assert(KM >= 1 && KM <= BK_KMAX, "columns per round");
  constexpr int NI = R / 4;
  constexpr int RS = BK_PARTS * R;
  // Items per lane of a gather: the P partials of one dot over 8 / K' lanes
  // (K' = columns of the round rounded up to a power of two), at most H
  // (registers): eight-column rounds hold one dot's P partials per lane
  // (launched for at most BK_MID_MAX_P or BK_SMALL_MAX_P workgroups), and
  // launches of the four-column 32-row kernel with more than 56 workgroups
  // (orders past 14336) take two columns per round.
  constexpr int KP2 = KM > 4 ? 8 : (KM > 2 ? 4 : KM);
  constexpr int H = R == BK_R ? (KM > 4 ? BK_MID_MAX_P : 28) : (BK_SMALL_MAX_P * KP2 + 7) / 8;
  // rounds of more than four columns form their reflectors in wave 0, one
  // lane per pivot, and leave them in LDS for every column
  constexpr bool LANE_PIVOTS = KM > 4;
  constexpr int PRM = bk_prm_words(KM);
  // register groups i that can hold one of the diagonal rows 0..NB-1 of
  // workgroup 0 (local row BK_LI i + 4 part + e < NB); only these need masks
  constexpr int NIM = (NB / BK_LI < NI) ? NB / BK_LI : NI;
  // One LDS block, the small arrays that every round reads first (their
  // addresses then fit the 16-bit offset of an LDS instruction).
  struct Lds {
    float pv[2][KM][2 * KM];            // pivot totals: dots, diagonal-row values
    float prm[LANE_PIVOTS ? KM : 1][PRM];   // the round's reflectors
    float bs[NB];                       // beta_j (workgroup 0)
    float px[2][KM][RS];                // pivot tails, by round parity
    float Ss[NB * BK_TSTR];             // S (workgroup 0), row-major
    float Ts[NB * BK_TSTR];             // T (workgroup 0), row-major
    int prm_taken;                      // reflectors the round takes
  };
  static_assert(sizeof(float) * (2 * 2 * KM * KM + (LANE_PIVOTS ? KM : 1) * PRM + NB) % 16 == 0,
                "16-byte aligned LDS arrays");
  __shared__ __align__(16) Lds lds;
  auto &pv = lds.pv;
  auto &prm = lds.prm;
  auto &bs = lds.bs;
  auto &px = lds.px;
  float *const Ss = lds.Ss;
  float *const Ts = lds.Ts;
  int &prm_taken = lds.prm_taken;

  const int g = blockIdx.x;
  const int64_t bz = blockIdx.y;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6, part = t & (BK_PARTS - 1);
  const int k = BK_WAVES * (lane / BK_PARTS) + wave;
  const int n = p.n, c = p.c, nb = p.nb, P = p.P;
  const unsigned un = (unsigned)n;     // n*n < 2^31
  float *At = p.At + bz * p.sA;
  const int r0 = c + g * RS;
  const bool w0 = (g == 0);
  const bool col = k < nb;
  unsigned *X = p.xch + bz * p.xstride;
  unsigned *abort_flag = X + BK_XABORT;
  unsigned *slots = X + BK_XHDR + p.area * p.area_words;   // this block's rounds
  const int64_t cw = (int64_t)KM * P + KM;          // items per column and round
  const int64_t pk = (int64_t)(wave * (64 / BK_PARTS) + lane / BK_PARTS);   // position of column k
  const int lbase = lane & ~(BK_PARTS - 1);

  float a[NI][4];
  {
    const float *src = At + (unsigned)(c + (col ? k : 0)) * un;
#pragma unroll
    for (int i = 0; i < NI; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = r0 + BK_LI * i + 4 * part + e;
        a[i][e] = (col && row < n) ? src[row] : 0.f;
      }
  }
  bool alive = true;
  const bool want_r = p.Rf != nullptr;   // the triangular factor is an output
  // Workgroup 0 keeps a copy of its diagonal rows (local rows < NB) in Ts,
  // unused until T is formed after the loop: Ts[k][row], rewritten after
  // every round, so the values of the diagonal rows of each column are LDS
  // reads (not a selection among the registers).
  auto save_diag_rows = [&]() {
    if (w0 && col) {
#pragma unroll
      for (int i = 0; i < NIM; ++i)
        *reinterpret_cast<float4 *>(Ts + k * BK_TSTR + BK_LI * i + 4 * part) =
            make_float4(a[i][0], a[i][1], a[i][2], a[i][3]);
    }
  };
  save_diag_rows();

  // Round at column j with K pivots p_0..p_{K-1} (columns j..j+K-1); rows are
  // counted from j (row s is row j+s).  A column a enters the round with its
  // diagonal-row values A[s] (s < K) and its dots with the tails,
  //   D[i] = sum_{s > i} a[s] p_i[s].
  // After reflectors 0..i-1 a column is a - sum_{l<i} g_l y_l on every row
  // past i-1 (each tail y_l covers them), so the reflectors act on the
  // coefficients g alone: with Phi_i(u, w) = sum_{s > i} u[s] w[s],
  //   Phi_i(p_l, a) = D[l] - sum_{s=l+1}^{i} p_l[s] A[s]          (l < i),
  //   a_i = A[i] - sum_{l<i} g_l p_l[i]        (its value in row i),
  //   v_i^T a = a_i + (1/v0_i) (D[i] - sum_l gamma_i[l] Phi_i(p_l, a)
  //                                   - sum_l g_l c_i[l]),
  // where gamma_i are the coefficients of pivot i when its reflector is
  // formed and c_i[l] = Phi_i(current pivot i, p_l).  Reflector i is applied
  // as f = beta_i v_i^T a, g_i = f / v0_i, g_l -= g_i gamma_i[l].  The pivot
  // columns' own totals give the reflectors (the same recurrence run on them,
  // with the pivot's squared tail Phi_i(pivot i, pivot i)); a round stops
  // before a pivot whose norm the earlier reflectors have mostly removed
  // (BK_TAU).  Every workgroup forms the same rounds from the same totals
  // with the same arithmetic.  Rows 0..taken-1 are R rows afterwards; the
  // combination leaves them inexact, and nothing but the triangular-factor
  // output reads them (later dots, broadcasts and diagonal-row values start
  // below them), which sets them from the recurrence.
  int j = 0;
  int round = 0;
  for (; j < nb; ++round) {
    const int par = round & 1;
    // columns this round: the most (a power of two up to KM) whose partials
    // fit H items per lane of a gather
    int kcap = KM;
#pragma unroll
    for (int q = 0; q < 3; ++q)
      if (kcap > 1 && (P * kcap + 7) / 8 > H) kcap >>= 1;
    const int kr = min(kcap, nb - j);
    const int rho = k - j;                          // this column's index in the round
    if (rho >= 0 && rho < kr) {
      float *dst = px[par][rho];
#pragma unroll
      for (int i = 0; i < NI; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int lr = BK_LI * i + 4 * part + e;
          dst[lr] = (w0 && i < NIM && lr <= k) ? 0.f : a[i][e];
        }
    }
    __syncthreads();
    float D[KM], A[KM];
#pragma unroll
    for (int q = 0; q < KM; ++q) D[q] = A[q] = 0.f;
    if (col) {
#pragma unroll
      for (int q = 0; q < KM; ++q) {
        if (q < kr) {
          const float *y = px[par][q];
          float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int i = 0; i < NI; ++i)
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[e] += a[i][e] * y[BK_LI * i + 4 * part + e];
          D[q] = (acc[0] + acc[1]) + (acc[2] + acc[3]);
        }
      }
      if (w0) {
#pragma unroll
        for (int s = 0; s < KM; ++s)
          if (s < kr) A[s] = Ts[k * BK_TSTR + j + s];
      }
    }
#pragma unroll
    for (int q = 0; q < KM; ++q)
      if (q < kr) D[q] = bk_sum8(D[q]);
    if (P > 1) {
      // Lane part < K posts its column's partial of dot `part`; lanes 4..7 of
      // workgroup 0 the diagonal-row values.  Then each dot's P partials are
      // read by 8/K' lanes (K' = K rounded up to a power of two), ceil(P K'/8)
      // contiguous items each, summed in index order and then over the lanes
      // of the dot in a fixed tree; lanes part < K also fetch the diagonal-row
      // value `part` from workgroup 0.
      unsigned *sl = slots + (int64_t)round * NB * cw;        // this round's slot
      unsigned *cb = sl + pk;                                  // item e at cb[e * NB]
      if (col) {
        float mine = D[0];
#pragma unroll
        for (int q = 1; q < KM; ++q)
          if (part == q) mine = D[q];
        if (part < kr) bk_put(cb + ((int64_t)part * P + g) * NB, mine);
        if (KM > 4 && w0 && part < kr) {
          float tv = A[0];
#pragma unroll
          for (int s = 1; s < KM; ++s)
            if (part == s) tv = A[s];
          bk_put(cb + ((int64_t)KM * P + part) * NB, tv);
        }
        if (KM <= 4 && w0 && part >= 4 && part - 4 < kr) {
          float tv = A[0];
#pragma unroll
          for (int s = 1; s < KM; ++s)
            if (part - 4 == s) tv = A[s];
          bk_put(cb + ((int64_t)KM * P + (part - 4)) * NB, tv);
        }
      }
      if (col && (w0 || k >= j)) {
        const int lg = (kr == 1) ? 3 : ((kr == 2) ? 2 : (kr <= 4 ? 1 : 0));   // log2 lanes per dot
        const int q = part >> lg, h = part & ((1 << lg) - 1);
        const int hn = (P + (1 << lg) - 1) >> lg;
        const int g0 = h * hn;
        const int cnt = (q < kr) ? max(0, min(P - g0, hn)) : 0;
        // (the column position is formed again from the thread index each
        // round: kept across the loop, its offsets would go to scratch)
        int tq = t;
        asm volatile("" : "+v"(tq));
        const int pkq = (tq >> 6) * (64 / BK_PARTS) + (tq & 63) / BK_PARTS;
        const int xoff = (!w0 && part < kr) ? ((KM * P + part) * NB + pkq) * 4 : -1;
        const __amdgpu_buffer_rsrc_t rs =
            __builtin_amdgcn_make_buffer_rsrc(sl, (short)0, (int)(NB * cw * 4), BK_RSRC_WORD3);
        float ssum = 0.f, xval = 0.f;
        if (alive)
          alive = bk_gather<H>(rs, (unsigned)(((q * P + g0) * NB + pkq) * 4), cnt, xoff, abort_flag,
                               ssum, xval);
        float s = ssum;
        if (lg == 1) s = bk_sum2(s);
        else if (lg == 2) s = bk_sum4(s);
        else if (lg == 3) s = bk_sum8(s);
#pragma unroll
        for (int qq = 0; qq < KM; ++qq)
          if (qq < kr) D[qq] = __shfl(s, lbase + (qq << lg));
        if (!w0) {
#pragma unroll
          for (int ss = 0; ss < KM; ++ss)
            if (ss < kr) A[ss] = __shfl(xval, lbase + ss);
        }
      }
    }
    if (rho >= 0 && rho < kr && part == 0) {
#pragma unroll
      for (int q = 0; q < KM; ++q) {
        pv[par][rho][q] = D[q];
        pv[par][rho][KM + q] = A[q];
      }
    }
    __syncthreads();
    if constexpr (LANE_PIVOTS) {
      // Wave 0 forms the round's reflectors from the pivots' totals, lane m
      // holding pivot m's row of ph, pt and gm (the quantities of the
      // per-thread form below); each step reads the values it needs from
      // other lanes as wave-uniform scalars and leaves, in prm[i], what the
      // column loop needs of reflector i.  Every workgroup runs the same
      // instructions on the same totals.
      if (wave == 0) {
        float phr[KM], ptr[KM], gmr[KM];
        {
          const int mm = lane < KM ? lane : 0;
          float row[2 * KM];
#pragma unroll
          for (int q = 0; q < 2 * KM; q += 4)
            *reinterpret_cast<float4 *>(&row[q]) = *reinterpret_cast<const float4 *>(&pv[par][mm][q]);
#pragma unroll
          for (int l = 0; l < KM; ++l) {
            phr[l] = row[l];
            ptr[l] = row[KM + l];
            gmr[l] = 0.f;
          }
        }
        auto rdl = [](float v, int l) {
          return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
        };
        int tk = kr;
#pragma unroll
        for (int i = 0; i < KM; ++i) {
          if (i < tk) {
            float spt[KM], sgi[KM], src[KM];
#pragma unroll
            for (int l = 0; l < i; ++l) spt[l] = rdl(ptr[i], l);   // p_l[i]
            // row i leaves the tails Phi(p_l, .), l < i
#pragma unroll
            for (int l = 0; l < i; ++l) phr[l] -= spt[l] * ptr[i];
            // the lane's pivot in row i after reflectors 0..i-1 (x0 in lane i)
            float cur = ptr[i];
#pragma unroll
            for (int l = 0; l < i; ++l) cur -= gmr[l] * spt[l];
#pragma unroll
            for (int l = 0; l < i; ++l) sgi[l] = rdl(gmr[l], i);   // gamma_i[l]
            float tt = phr[i];
#pragma unroll
            for (int l = 0; l < i; ++l) tt -= sgi[l] * phr[l];
#pragma unroll
            for (int l = 0; l < i; ++l) src[l] = rdl(tt, l);       // c_i[l]
            // Phi_i(current pivot i, lane's pivot) (the squared tail in lane i)
            float phv = tt;
#pragma unroll
            for (int l = 0; l < i; ++l) phv -= gmr[l] * src[l];
            float ref = phr[i];
#pragma unroll
            for (int q = 0; q <= i; ++q) ref += ptr[q] * ptr[q];
            const float x0 = rdl(cur, i), st = rdl(phv, i), rf = rdl(ref, i);
            if (i > 0 && !(st >= 0.f && x0 * x0 + st >= BK_TAU * rf)) {
              tk = i;
            } else {
              float bet, iv0, rjj;
              bk_reflector(x0, st, bet, iv0, rjj);
              float *pr = prm[i];
              if (lane == i) {
                pr[0] = bet;
                pr[1] = iv0;
                pr[2] = rjj;
#pragma unroll
                for (int l = 0; l < i; ++l) pr[4 + l] = gmr[l];
              }
              if (lane < i) {
                pr[4 + KM + lane] = tt;
                pr[4 + 2 * KM + lane] = ptr[i];
              }
              if (lane > i && lane < KM) {
                const float qf = bet * (cur + iv0 * phv) * iv0;
#pragma unroll
                for (int l = 0; l < i; ++l) gmr[l] -= qf * sgi[l];
                gmr[i] = qf;
              }
            }
          }
        }
        if (lane == 0) prm_taken = tk;
      }
      __syncthreads();
      const int taken = __builtin_amdgcn_readfirstlane(prm_taken);
      float iv0_own = 1.f, rj_own = 0.f;
      if (rho >= 0 && rho < taken) {
        iv0_own = prm[rho][1];
        rj_own = prm[rho][2];
      }
      if (col && (rho >= 0 || w0)) {
        // as below, with reflector i's quantities read from prm[i]
        float gc[KM], Rr[KM], phi[KM];
#pragma unroll
        for (int q = 0; q < KM; ++q) {
          gc[q] = Rr[q] = 0.f;
          phi[q] = D[q];
        }
#pragma unroll
        for (int i = 0; i < KM; ++i) {
          if (i < taken) {
            const float *pr = prm[i];
            const float bet = pr[0], iv0 = pr[1];
            const float Ai = A[i];
            float cur = Ai;
#pragma unroll
            for (int l = 0; l < i; ++l) {
              const float pli = pr[4 + 2 * KM + l];
              phi[l] -= pli * Ai;
              cur -= gc[l] * pli;
            }
            float phv = phi[i];
#pragma unroll
            for (int l = 0; l < i; ++l) phv -= pr[4 + l] * phi[l] + gc[l] * pr[4 + KM + l];
            const float hv = cur + iv0 * phv;
            if (rho > i) {
              const float f = bet * hv;
              Rr[i] = cur - f;
              const float qf = f * iv0;
#pragma unroll
              for (int l = 0; l < i; ++l) gc[l] -= qf * pr[4 + l];
              gc[i] = qf;
            } else if (rho < i && w0 && part == 0) {
              Ss[k * BK_TSTR + j + i] = hv * iv0_own;
            }
          }
        }
        if (rho >= 0) {
          // a -= sum_l g_l y_l (a consumed pivot: its own coefficients, then
          // scaled by 1/v0 into its reflector's vector)
#pragma unroll
          for (int l = 0; l < KM; ++l)
            if (l < taken) {
              const float *y = px[par][l];
              const float gl = gc[l];
#pragma unroll
              for (int i = 0; i < NI; ++i)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                  a[i][e] = fmaf(-gl, y[BK_LI * i + 4 * part + e], a[i][e]);
            }
          if (rho < taken) {
            // (with the triangular-factor output, workgroup 0's R rows above
            // the pivot's diagonal row keep their values)
            const bool keep_r = w0 && want_r;
#pragma unroll
            for (int i = 0; i < NI; ++i)
#pragma unroll
              for (int e = 0; e < 4; ++e)
                if (!keep_r || i >= NIM || BK_LI * i + 4 * part + e > k) a[i][e] *= iv0_own;
          }
          if (w0 && want_r) {
            // R rows j..: R[j+s][k] = Rr[s] for the reflectors applied to this
            // column, and the R diagonal for a consumed pivot
            const int nl = rho < taken ? rho : taken;
#pragma unroll
            for (int s = 0; s < KM; ++s) {
              const int row = j + s;
              if (s < nl && part == ((row >> 2) & (BK_PARTS - 1)))
                bk_reg_set<NIM>(a, (row / BK_LI) * 4 + (row & 3), Rr[s]);
            }
            if (rho < taken && part == ((k >> 2) & (BK_PARTS - 1)))
              bk_reg_set<NIM>(a, (k / BK_LI) * 4 + (k & 3), rj_own);
          }
        }
      }
      if (w0 && t == 0) {
#pragma unroll
        for (int i = 0; i < KM; ++i)
          if (i < taken) {
            bs[j + i] = prm[i][0];
            p.beta[bz * n + c + j + i] = prm[i][0];
            p.dsign[bz * n + c + j + i] = (prm[i][2] < 0.f) ? -1.f : 1.f;
          }
      }
      if (j + taken < nb) save_diag_rows();
      j += taken;
    } else {
      // The round's reflectors from the pivots' totals, formed alike in every
      // thread (registers only): pt[m][s] = p_m[s], ph[m][l] = Phi_i(p_l, p_m),
      // gm[m][l] = coefficients of pivot m (l < m); per step i: beta rb[i],
      // 1/v0 rv[i], R diagonal rr[i], gamma_i = gm[i][l] and c_i = rc[i][l].
      float pt[KM][KM], rb[KM], rv[KM], rr[KM], gm[KM][KM], rc[KM][KM];
      int taken = kr;
      {
        // (rows and columns past kr hold stale values: no step below reads them
        // into a value it keeps, since every step i < taken <= kr reads only
        // indices below i or its own row)
        float ph[KM][KM];
#pragma unroll
        for (int m = 0; m < KM; ++m) {
          rb[m] = rv[m] = rr[m] = 0.f;
          float row[8];
          *reinterpret_cast<float4 *>(&row[0]) = *reinterpret_cast<const float4 *>(&pv[par][m][0]);
          *reinterpret_cast<float4 *>(&row[4]) = *reinterpret_cast<const float4 *>(&pv[par][m][4]);
#pragma unroll
          for (int l = 0; l < KM; ++l) {
            ph[m][l] = row[l];
            pt[m][l] = row[KM + l];
            gm[m][l] = rc[m][l] = 0.f;
          }
        }
#pragma unroll
        for (int i = 0; i < KM; ++i) {
          if (i < taken) {
            // row i leaves the tails Phi(p_l, .), l < i
#pragma unroll
            for (int m = 0; m < KM; ++m)
#pragma unroll
              for (int l = 0; l < i; ++l) ph[m][l] -= pt[l][i] * pt[m][i];
            float x0 = pt[i][i];
#pragma unroll
            for (int l = 0; l < i; ++l) {
              x0 -= gm[i][l] * pt[l][i];
              float v = ph[l][i];
#pragma unroll
              for (int l2 = 0; l2 < i; ++l2) v -= gm[i][l2] * ph[l][l2];
              rc[i][l] = v;
            }
            float st = ph[i][i];
#pragma unroll
            for (int l = 0; l < i; ++l) st -= gm[i][l] * (ph[i][l] + rc[i][l]);
            float ref = ph[i][i];
#pragma unroll
            for (int s = 0; s <= i; ++s) ref += pt[i][s] * pt[i][s];
            // (every lane holds the same totals: the decision is read from lane 0
            // so that the round's bounds stay wave-uniform scalars)
            const bool ok =
                __builtin_amdgcn_readfirstlane((i == 0 || (st >= 0.f && x0 * x0 + st >= BK_TAU * ref))
                                                   ? 1
                                                   : 0) != 0;
            if (!ok) {
              taken = i;
            } else {
              bk_reflector(x0, st, rb[i], rv[i], rr[i]);
              const float bet = rb[i], iv0 = rv[i];
#pragma unroll
              for (int m = i + 1; m < KM; ++m) {
                float cur = pt[m][i];
                float phv = ph[m][i];
#pragma unroll
                for (int l = 0; l < i; ++l) {
                  cur -= gm[m][l] * pt[l][i];
                  phv -= gm[i][l] * ph[m][l] + gm[m][l] * rc[i][l];
                }
                const float qf = bet * (cur + iv0 * phv) * iv0;
#pragma unroll
                for (int l = 0; l < i; ++l) gm[m][l] -= qf * gm[i][l];
                gm[m][i] = qf;
              }
            }
          }
        }
      }
      // this column's 1/v0 and R diagonal if it is a pivot the round takes
      float iv0_own = 1.f, rj_own = 0.f;
#pragma unroll
      for (int m = 0; m < KM; ++m)
        if (rho == m && m < taken) {
          iv0_own = rv[m];
          rj_own = rr[m];
        }
      if (col && (rho >= 0 || w0)) {
        // This column's coefficients, its R entries in rows j.. (Rr) and, for
        // the reflectors past it, S = y_k^T v (stored and consumed columns).
        float gc[KM], Rr[KM];
#pragma unroll
        for (int q = 0; q < KM; ++q) gc[q] = Rr[q] = 0.f;
        float phi[KM];
#pragma unroll
        for (int q = 0; q < KM; ++q) phi[q] = D[q];
#pragma unroll
        for (int i = 0; i < KM; ++i) {
          if (i < taken) {
            const float Ai = A[i];
            float cur = Ai;
#pragma unroll
            for (int l = 0; l < i; ++l) {
              phi[l] -= pt[l][i] * Ai;
              cur -= gc[l] * pt[l][i];
            }
            float phv = phi[i];
#pragma unroll
            for (int l = 0; l < i; ++l) phv -= gm[i][l] * phi[l] + gc[l] * rc[i][l];
            const float hv = cur + rv[i] * phv;
            if (rho > i) {
              const float f = rb[i] * hv;
              Rr[i] = cur - f;
              const float qf = f * rv[i];
#pragma unroll
              for (int l = 0; l < i; ++l) gc[l] -= qf * gm[i][l];
              gc[i] = qf;
            } else if (rho < i && w0 && part == 0) {
              Ss[k * BK_TSTR + j + i] = hv * iv0_own;
            }
          }
        }
        if (rho >= 0) {
          // a -= sum_l g_l y_l (a consumed pivot: its own coefficients, then
          // scaled by 1/v0 into its reflector's vector)
#pragma unroll
          for (int l = 0; l < KM; ++l)
            if (l < taken) {
              const float *y = px[par][l];
              const float gl = gc[l];
#pragma unroll
              for (int i = 0; i < NI; ++i)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                  a[i][e] = fmaf(-gl, y[BK_LI * i + 4 * part + e], a[i][e]);
            }
          if (rho < taken) {
            // (with the triangular-factor output, workgroup 0's R rows above
            // the pivot's diagonal row keep their values)
            const bool keep_r = w0 && want_r;
#pragma unroll
            for (int i = 0; i < NI; ++i)
#pragma unroll
              for (int e = 0; e < 4; ++e)
                if (!keep_r || i >= NIM || BK_LI * i + 4 * part + e > k) a[i][e] *= iv0_own;
          }
          if (w0 && want_r) {
            // R rows j..: R[j+s][k] = Rr[s] for the reflectors applied to this
            // column, and the R diagonal for a consumed pivot
            const int nl = rho < taken ? rho : taken;
#pragma unroll
            for (int s = 0; s < KM; ++s) {
              const int row = j + s;
              if (s < nl && part == ((row >> 2) & (BK_PARTS - 1)))
                bk_reg_set<NIM>(a, (row / BK_LI) * 4 + (row & 3), Rr[s]);
            }
            if (rho < taken && part == ((k >> 2) & (BK_PARTS - 1)))
              bk_reg_set<NIM>(a, (k / BK_LI) * 4 + (k & 3), rj_own);
          }
        }
      }
      if (w0 && t == 0) {
#pragma unroll
        for (int i = 0; i < KM; ++i)
          if (i < taken) {
            bs[j + i] = rb[i];
            p.beta[bz * n + c + j + i] = rb[i];
            p.dsign[bz * n + c + j + i] = (rr[i] < 0.f) ? -1.f : 1.f;
          }
      }
      // (not after the last round: T's formation clears Ts right after the
      // loop, with no barrier in between)
      if (j + taken < nb) save_diag_rows();
      j += taken;
    }
  }
  // Write Y (zeros above its diagonal, ones on it) and the R entries of the
  // block's diagonal rows.  An aborted exchange poisons the block.
  const bool bad =
      P > 1 && __hip_atomic_load(abort_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u;
  if (bad && t == 0) {   // the factorization of this matrix failed: no Q is formed from it
    __hip_atomic_store(X + BK_XFAILED, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (p.status)
      __hip_atomic_fetch_or(p.status, p.status_bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  const float nan = __builtin_nanf("");
  if (col) {
    float *dst = At + (unsigned)(c + k) * un;
    float *Rf = p.Rf ? p.Rf + bz * p.sA : nullptr;
#pragma unroll
    for (int i = 0; i < NI; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int lr = BK_LI * i + 4 * part + e;
        const int row = r0 + lr;
        if (row < n) {
          float v = a[i][e];
          if (w0 && lr <= k) {
            if (Rf) Rf[(unsigned)row * un + c + k] = bad ? nan : v;
            v = (lr == k) ? 1.f : 0.f;
          }
          dst[row] = bad ? nan : v;
        }
      }
  }
  {
    // The words this block wrote, for the emptying after the next block;
    // then what the previous block wrote into the other area (which the next
    // block uses) back to the empty pattern.
    if (w0 && t == 0)
      __hip_atomic_store(X + BK_XUSED + p.area, P > 1 ? (unsigned)(round * NB * cw) : 0u,
                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int64_t used = (int64_t)__hip_atomic_load(X + BK_XUSED + (1 - p.area), __ATOMIC_RELAXED,
                                                    __HIP_MEMORY_SCOPE_AGENT);
    uint4 *nx = reinterpret_cast<uint4 *>(X + BK_XHDR + (1 - p.area) * p.area_words);
    const uint4 e4 = make_uint4(BK_EMPTY, BK_EMPTY, BK_EMPTY, BK_EMPTY);
    for (int64_t i = (int64_t)g * BK_THREADS + t; i < used / 4; i += (int64_t)P * BK_THREADS)
      nx[i] = e4;
  }
  if (!w0) return;
  // T by blocks of 8 columns: first every diagonal block T_JJ (rows of one
  // block are independent recurrences of at most 8 steps), then, row by row,
  //   T_IJ = -(sum_{K=I}^{J-1} T_IK S_KJ) T_JJ  for J > I.
  // Row k belongs to the eight lanes of column k; they exchange values only
  // through shuffles and their own row of Ts, so no barrier is needed after
  // the diagonal blocks.
  for (int e = t; e < NB * BK_TSTR; e += BK_THREADS) Ts[e] = 0.f;
  __syncthreads();
  float *trow = Ts + k * BK_TSTR;
  const int J0 = k >> 3;
  if (col) {
    const int jend = min(nb, 8 * J0 + 8);
    for (int j = k; j < jend; ++j) {
      float s = 0.f;
      for (int l = k + part; l < j; l += BK_PARTS) s += trow[l] * Ss[l * BK_TSTR + j];
#pragma unroll
      for (int msk = 1; msk < BK_PARTS; msk <<= 1) s += __shfl_xor(s, msk);
      __builtin_amdgcn_wave_barrier();
      if (part == 0) trow[j] = (j == k) ? bs[j] : -bs[j] * s;
      __builtin_amdgcn_wave_barrier();
    }
  }
  __syncthreads();
  if (col) {
    const int lead = lane & ~(BK_PARTS - 1);
    for (int J = J0 + 1; 8 * J < nb; ++J) {
      // X[c] = sum_{l=k}^{8J-1} T[k][l] S[l][8J+c]; lane part forms c = part
      const int c0 = 8 * J + part;
      float x0a = 0.f, x0b = 0.f;
      int l = k;
      for (; l + 1 < 8 * J; l += 2) {
        x0a += trow[l] * Ss[l * BK_TSTR + c0];
        x0b += trow[l + 1] * Ss[(l + 1) * BK_TSTR + c0];
      }
      if (l < 8 * J) x0a += trow[l] * Ss[l * BK_TSTR + c0];
      // columns past nb of S were never written: keep them out of X
      const float xa = (c0 < nb) ? x0a + x0b : 0.f;
      // T[k][8J+q] = -sum_c X[c] T_JJ[c][q],  X[c] from lane lead + c
      float r0 = 0.f;
#pragma unroll
      for (int cc = 0; cc < 8; ++cc) {
        const float xc = __shfl(xa, lead + cc);
        r0 += xc * Ts[(8 * J + cc) * BK_TSTR + 8 * J + part];
      }
      __builtin_amdgcn_wave_barrier();
      if (c0 < nb) trow[c0] = -r0;
      __builtin_amdgcn_wave_barrier();
    }
  }
  __syncthreads();
  float *T = p.T + bz * p.sT;
  for (int e = t; e < NB * NB; e += BK_THREADS)
    T[e] = bad ? nan : Ts[(e / NB) * BK_TSTR + e % NB];
}

// Final triangular factor: entries of an earlier outer block than their column
// come from At, except the squares of full pairs (rows of block 2p, columns
// of block 2p+1, p < np), which the factorization moved to Rf already scaled;
// entries inside an outer block were stored by the panels; every row i is
// then scaled by d_i so that diag(R) >= 0.  Strict lower part = 0.
__global__ __launch_bounds__(256) void qr_extract_r_kernel(const float *At, float *Rf,
                                                           const float *dsign, int n,
                                                           int64_t sA, int np) {
  const int64_t bz = blockIdx.y;
  const float *Ab = At + bz * sA;
  float *Rb = Rf + bz * sA;
  const float *d = dsign + bz * n;
  const int64_t nn = (int64_t)n * n;
  for (int64_t e = blockIdx.x * 256 + threadIdx.x; e < nn; e += (int64_t)gridDim.x * 256) {
    const int i = (int)(e / n), j = (int)(e % n);
    const int bi = i / NB, bj = j / NB;
    if (i > j) Rb[e] = 0.f;
    else if ((bi & 1) == 0 && bj == bi + 1 && bi / 2 < np) continue;   // moved already
    else Rb[e] = d[i] * ((bi < bj) ? Ab[(int64_t)j * n + i] : Rb[e]);
  }
}

// Full pair p = (blocks a, b = a + 1) once both are factored: the R entries
// of block b's columns in block a's rows (At[c_b + j][c_a + i], i, j < NB)
// are final; they move to Rf (scaled by d of their row) when it is wanted,
// and are cleared in At, so that rows c_a..c_a+2NB of At from column c_a on
// hold the pair's unit lower-trapezoidal Y for the rank-2NB updates.
__global__ __launch_bounds__(256) void qr_clear_pair_square_kernel(float *At, int64_t sA,
                                                                   float *Rf,
                                                                   const float *dsign, int n,
                                                                   int ca) {
  const int64_t bz = blockIdx.y;
  float *Ab = At + bz * sA;
  const int cb = ca + NB;
  for (int e = blockIdx.x * 256 + threadIdx.x; e < NB * NB; e += gridDim.x * 256) {
    const int j = e / NB, i = e % NB;   // column cb + j, row ca + i
    float *src = Ab + (int64_t)(cb + j) * n + ca + i;
    if (Rf) Rf[bz * sA + (int64_t)(ca + i) * n + cb + j] = dsign[bz * n + ca + i] * *src;
    *src = 0.f;
  }
}

// Zeroes, in At, the entries of each column above its outer block's rows
// (At[j][i] for i < NB floor(j / NB)): R entries, no longer needed once R has
// been extracted.  Y then has explicit zeros above every block, so two
// consecutive blocks form one unit lower-trapezoidal Y of 2 NB columns.
__global__ __launch_bounds__(256) void qr_zero_above_blocks_kernel(float *At, int n, int64_t sA) {
  float *A = At + (int64_t)blockIdx.y * sA;
  const int64_t nn = (int64_t)n * n;
  for (int64_t e = blockIdx.x * 256 + threadIdx.x; e < nn; e += (int64_t)gridDim.x * 256) {
    const int j = (int)(e / n), i = (int)(e - (int64_t)j * n);
    if (i < (j / NB) * NB) A[e] = 0.f;
  }
}

// T of a pair of consecutive full blocks a, b (2 NB x 2 NB, row-major):
//   [[T_a, T_ab], [0, T_b]]; T_ab was written in place by the caller.
__global__ __launch_bounds__(256) void qr_assemble_pair_t_kernel(float *TP, int64_t sTP,
                                                                 const float *Ta, const float *Tb,
                                                                 int64_t sT, int w, int ldab) {
  // TP is 2w x 2w (row-major); Ta, Tb are w x w with leading dimension ldab.
  float *P = TP + (int64_t)blockIdx.y * sTP;
  const float *A = Ta + (int64_t)blockIdx.y * sT, *B = Tb + (int64_t)blockIdx.y * sT;
  for (int e = blockIdx.x * 256 + threadIdx.x; e < 4 * w * w; e += gridDim.x * 256) {
    const int r = e / (2 * w), c = e % (2 * w);
    if (r < w && c < w) P[e] = A[r * ldab + c];
    else if (r >= w && c < w) P[e] = 0.f;
    else if (r >= w) P[e] = B[(r - w) * ldab + (c - w)];
  }
}

// Trailing update, second product: W2 = T^T W with W = sum_s part[s] (the S
// split-K partials of W = Y^T A_trail, each nb x Nt row-major, summed in slice
// order) and T the block's nb x nb upper-triangular factor (row-major, leading
// dimension NB).  One workgroup per 8 columns of W2: it sums its columns of
// the partials into LDS, stages T, and forms its 8 columns of T^T W (k in
// increasing order).  Replaces a reduction pass and a latency-bound GEMM with
// K = nb on the factorization's critical path.
template <int CW>
__global__ __launch_bounds__(256) void qr_reduce_tt_kernel(const float *__restrict__ part,
                                                                int S, int nb, int Nt,
                                                                const float *__restrict__ T,
                                                                int64_t sT, float *__restrict__ W2,
                                                                int64_t sW) {
  // CW columns per workgroup; EPT entries per thread, loaded SB slices at a
  // time (32 loads in flight per thread)
  constexpr int EPT = NB * CW / 256, SB = 32 / EPT;
  __shared__ float Ts[NB][NB + 1];
  __shared__ float Ws[NB][CW];
  const int64_t bz = blockIdx.y;
  const int t = threadIdx.x;
  const int j0 = blockIdx.x * CW;
  const float *Tb = T + bz * sT;
  if (nb == NB && (reinterpret_cast<uintptr_t>(Tb) & 15u) == 0) {   // 16 float4 per thread
    const float4 *T4 = reinterpret_cast<const float4 *>(Tb);
    float4 tv[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) tv[q] = T4[t + 256 * q];
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int e4 = t + 256 * q, k = e4 / (NB / 4), i = 4 * (e4 % (NB / 4));
      Ts[k][i] = tv[q].x; Ts[k][i + 1] = tv[q].y; Ts[k][i + 2] = tv[q].z; Ts[k][i + 3] = tv[q].w;
    }
  } else {
    for (int e = t; e < NB * NB; e += 256) {
      const int k = e / NB, i = e % NB;
      Ts[k][i] = (k < nb && i < nb) ? Tb[k * NB + i] : 0.f;
    }
  }
  const int64_t slice = (int64_t)nb * Nt;
  const float *pb = part + bz * S * slice;
  // EPT entries per thread, slices summed in order, SB at a time so that
  // their load latencies overlap.
  float acc[EPT];
  int64_t off[EPT];
  bool ok[EPT];
#pragma unroll
  for (int q = 0; q < EPT; ++q) {
    const int e = t + 256 * q, k = e / CW, j = j0 + (e % CW);
    acc[q] = 0.f;
    ok[q] = k < nb && j < Nt;
    off[q] = ok[q] ? (int64_t)k * Nt + j : 0;
  }
  for (int s0 = 0; s0 < S; s0 += SB) {
    float v[SB][EPT];
#pragma unroll
    for (int u = 0; u < SB; ++u)
#pragma unroll
      for (int q = 0; q < EPT; ++q)
        v[u][q] = (s0 + u < S && ok[q]) ? pb[(int64_t)(s0 + u) * slice + off[q]] : 0.f;
#pragma unroll
    for (int u = 0; u < SB; ++u)
#pragma unroll
      for (int q = 0; q < EPT; ++q) acc[q] += v[u][q];
  }
#pragma unroll
  for (int q = 0; q < EPT; ++q) {
    const int e = t + 256 * q;
    Ws[e / CW][e % CW] = acc[q];
  }
  __syncthreads();
  float *Wb = W2 + bz * sW;
  for (int e = t; e < NB * CW; e += 256) {
    const int i = e / CW, c = e % CW, j = j0 + c;
    if (i >= nb || j >= Nt) continue;
    float a = 0.f;
    for (int k = 0; k < nb; ++k) a += Ts[k][i] * Ws[k][c];
    Wb[(int64_t)i * Nt + j] = a;
  }
}

// Q <- diag(d) for each matrix of the batch.
__global__ __launch_bounds__(256) void qr_init_q_kernel(float *Q, const float *dsign, int n,
                                                        int64_t sA, const unsigned *skip,
                                                        int64_t sSkip) {
  const int64_t bz = blockIdx.y;
  if (skip && skip[bz * sSkip] != 0u) return;   // failed factorization: Q is kept
  float *Qb = Q + bz * sA;
  const float *d = dsign + bz * n;
  const int64_t nn = (int64_t)n * n;
  for (int64_t e = blockIdx.x * 256 + threadIdx.x; e < nn; e += (int64_t)gridDim.x * 256) {
    const int i = (int)(e / n), j = (int)(e % n);
    Qb[e] = (i == j) ? d[i] : 0.f;
  }
}

// Q of entry bz of a call over two factors' matrices (contiguous, n x n each)
// to its owner: Q_A + bz nn for bz < half, Q_B + (bz - half) nn after, with
// column j scaled by dsign[bz n + j] (the signs that make diag(R) >= 0).  An
// entry whose factorization failed is not copied (its destination keeps the
// Q it held) and its half's bit is or-ed into *status.
__global__ __launch_bounds__(256) void qr_scatter_q_kernel(const float *Qs, float *QA, float *QB,
                                                           int64_t half, int n,
                                                           const float *dsign,
                                                           const unsigned *skip, int64_t sSkip,
                                                           unsigned *status, unsigned bitA,
                                                           unsigned bitB) {
  const int64_t bz = blockIdx.y;
  if (skip && skip[bz * sSkip] != 0u) {
    if (status && blockIdx.x == 0 && threadIdx.x == 0)
      __hip_atomic_fetch_or(status, bz < half ? bitA : bitB, __ATOMIC_RELAXED,
                            __HIP_MEMORY_SCOPE_AGENT);
    return;
  }
  const int64_t nn = (int64_t)n * n;
  const float *src = Qs + bz * nn;
  const float *d = dsign ? dsign + bz * n : nullptr;
  float *dst = bz < half ? QA + bz * nn : QB + (bz - half) * nn;
  const int64_t stride = (int64_t)gridDim.x * 256;
  if ((n & 3) == 0) {   // every entry starts 16-byte aligned; four columns of one row
    const float4 *s4 = reinterpret_cast<const float4 *>(src);
    float4 *d4 = reinterpret_cast<float4 *>(dst);
    for (int64_t e = blockIdx.x * 256 + threadIdx.x; e < nn / 4; e += stride) {
      float4 v = s4[e];
      if (d) {
        const int j = (int)((4 * e) % n);
        v.x *= d[j]; v.y *= d[j + 1]; v.z *= d[j + 2]; v.w *= d[j + 3];
      }
      d4[e] = v;
    }
  } else {
    for (int64_t e = blockIdx.x * 256 + threadIdx.x; e < nn; e += stride)
      dst[e] = d ? src[e] * d[e % n] : src[e];
  }
}

// Q = I for every matrix of the batch (n x n, batch stride sA).
__global__ __launch_bounds__(256) void qr_identity_kernel(float *Q, int n, int64_t sA) {
  float *Qb = Q + (int64_t)blockIdx.y * sA;
  const int64_t nn = (int64_t)n * n;
  for (int64_t e = blockIdx.x * 256 + threadIdx.x; e < nn; e += (int64_t)gridDim.x * 256)
    Qb[e] = (e / n == e % n) ? 1.f : 0.f;
}

// The first w columns of W = Y^T Q[c:, c:] for a group of w reflectors
// starting at column c, while rows and columns c..c+w-1 of Q still hold
// diag(d): W[i][j] = Y[j][i] d[c+j] = At[c+i][c+j] d[c+j] (i, j < w).
// W has leading dimension ldw and batch stride sW.
__global__ __launch_bounds__(256) void qr_q_head_kernel(float *W, int64_t ldw, int64_t sW,
                                                        const float *At, int64_t sA,
                                                        const float *dsign, int n, int64_t c,
                                                        int w, const unsigned *skip,
                                                        int64_t sSkip) {
  const int64_t bz = blockIdx.y;
  if (skip && skip[bz * sSkip] != 0u) return;
  float *Wb = W + bz * sW;
  const float *Ab = At + bz * sA + c * n + c;
  const float *d = dsign + bz * n + c;
  const int64_t ww = (int64_t)w * w;
  for (int64_t e = blockIdx.x * 256 + threadIdx.x; e < ww; e += (int64_t)gridDim.x * 256) {
    const int64_t i = e / w, j = e % w;
    Wb[i * ldw + j] = Ab[i * n + j] * d[j];
  }
}

// Raises the abort flag of each of `batch` exchange areas (the forced
// give-up of qr_force_give_up).
__global__ __launch_bounds__(64) void qr_raise_abort_kernel(unsigned *xch, int64_t xstride,
                                                            int64_t batch) {
  for (int64_t b = blockIdx.x * 64 + threadIdx.x; b < batch; b += (int64_t)gridDim.x * 64)
    __hip_atomic_store(xch + b * xstride + BK_XABORT, 1u, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}

// Exchange areas at the start of a call: header words zero, area 0 (the
// first block's) empty, and area 1 marked as written throughout, so that the
// first block empties all of it for the second.
__global__ __launch_bounds__(256) void qr_xch_init_kernel(unsigned *xch, int64_t xstride,
                                                          int64_t area_words) {
  unsigned *X = xch + (int64_t)blockIdx.y * xstride;
  const int64_t cnt = BK_XHDR + area_words;
  for (int64_t i = blockIdx.x * 256 + threadIdx.x; i < cnt; i += (int64_t)gridDim.x * 256)
    X[i] = (i < BK_XHDR) ? (i == BK_XUSED + 1 ? (unsigned)area_words : 0u) : BK_EMPTY;
}

// dst = src^T for one n x n matrix, through 32 x 32 LDS tiles.
__global__ __launch_bounds__(256) void transpose_kernel(float *dst, const float *src, int n) {
  __shared__ float tile[32][33];
  const int bx = blockIdx.x * 32, by = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int k = ty; k < 32; k += 8) {
    const int r = by + k, cc = bx + tx;
    if (r < n && cc < n) tile[k][tx] = src[(int64_t)r * n + cc];
  }
  __syncthreads();
  for (int k = ty; k < 32; k += 8) {
    const int r = bx + k, cc = by + tx;
    if (r < n && cc < n) dst[(int64_t)r * n + cc] = tile[tx][k];
  }
}

// ------------------------------------------------------------ host driver
struct QrLayout {
  int64_t n, nob;
  bool block;          // outer blocks factored by qr_block_kernel (else the panel path)
  size_t t_off, w_off, w2_off, sk_off, part_off, wi_off, d_off, b_off, cnt_off, x_off, total;
  size_t tp_off, sx_off, skp_off, skp2_off, tq_off, sq_off, to_off, so_off, wn_off, skn_off;
  size_t fv_off;
  int64_t sT, sWbuf, sSk, sPart, sWi;
  int64_t sFv;         // the forward Q formation's V = Q Y and V T (n x 2 NB each)
  int64_t sWn, sSkn;   // the near update's own W, W2 (NB x NB each) and split-K partials
  int64_t np;          // pairs of full outer blocks
  int64_t nq;          // quads (pairs of full pairs)
  int64_t no;          // octs (pairs of full quads), for n >= OCT_MIN_N
  int64_t sTP, sSx, sSkp, sTQ, sSq, sTO, sSo;
};

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

constexpr int MAX_SPLIT = 8;
// From this size on, Q is formed by rank-1024 updates (octs of blocks): the
// longer K brings the update near the long-K products' rate, which outweighs
// the coarser trapezoid (1.5 w / n more flops than the block-level count).
constexpr int64_t OCT_MIN_N = 8192;
// Shortest K slice of the near update's first product (its split-K slices
// run side by side: shorter slices, more workgroups, less latency).
constexpr int64_t NEAR_MIN_K = 64;

QrLayout qr_layout(int64_t batch, int64_t n) {
  QrLayout L{};
  L.n = n;
  L.nob = (n + NB - 1) / NB;
  const int64_t P = (n + RCH - 1) / RCH;
  L.sT = L.nob * NB * NB;
  L.np = (n / NB) / 2;
  L.nq = L.np / 2;
  L.no = (n >= OCT_MIN_N) ? L.nq / 2 : 0;
  L.sWbuf = (int64_t)(L.no > 0 ? 8 : 4) * NB * n;
  // Split-K partials: MAX_SPLIT slices of 2 NB x n for the trailing updates,
  // four of 8 NB x n for the rank-1024 Q-formation products.
  L.sSk = (int64_t)(L.no > 0 ? 32 * NB : MAX_SPLIT * 2 * NB) * n;
  L.sTP = L.np * 4 * NB * NB;
  L.sSx = L.np * 2 * NB * NB;
  L.sSkp = (int64_t)64 * NB * NB;
  L.sWn = (int64_t)2 * NB * NB;
  L.sSkn = std::max<int64_t>(1, std::min<int64_t>(64, n / NEAR_MIN_K)) * NB * NB;
  L.sTQ = L.nq * 16 * NB * NB;
  L.sSq = L.nq * 8 * NB * NB;
  L.sTO = L.no * 64 * NB * NB;
  L.sSo = L.no * 32 * NB * NB;
  L.sPart = P * PART_STRIDE;
  L.sWi = (int64_t)MAX_B * NB;
  L.sFv = (int64_t)4 * NB * n;
  size_t o = 0;
  L.t_off = o;    o = align256(o + sizeof(float) * batch * L.sT);
  L.w_off = o;    o = align256(o + sizeof(float) * batch * L.sWbuf);
  L.w2_off = o;   o = align256(o + sizeof(float) * batch * L.sWbuf);
  L.sk_off = o;   o = align256(o + sizeof(float) * batch * L.sSk);
  L.part_off = o; o = align256(o + sizeof(float) * batch * L.sPart);
  L.wi_off = o;   o = align256(o + sizeof(float) * batch * L.sWi);
  L.d_off = o;    o = align256(o + sizeof(float) * batch * n);
  L.b_off = o;    o = align256(o + sizeof(float) * batch * n);
  L.cnt_off = o;  o = align256(o + sizeof(unsigned) * batch);
  L.tp_off = o;   o = align256(o + sizeof(float) * batch * L.sTP);
  L.sx_off = o;   o = align256(o + sizeof(float) * batch * L.sSx);
  L.skp_off = o;  o = align256(o + sizeof(float) * batch * L.sSkp);
  L.skp2_off = o; o = align256(o + sizeof(float) * batch * L.sSkp);
  L.tq_off = o;   o = align256(o + sizeof(float) * batch * L.sTQ);
  L.sq_off = o;   o = align256(o + sizeof(float) * batch * L.sSq);
  L.to_off = o;   o = align256(o + sizeof(float) * batch * L.sTO);
  L.so_off = o;   o = align256(o + sizeof(float) * batch * L.sSo);
  L.wn_off = o;   o = align256(o + sizeof(float) * batch * L.sWn);
  L.skn_off = o;  o = align256(o + sizeof(float) * batch * L.sSkn);
  L.fv_off = o;   o = align256(o + sizeof(float) * batch * L.sFv);
  // The resident-block path needs every workgroup of a launch resident at
  // once: at most BK_MAX_WG workgroups (two such launches, one per factor,
  // may run together on the 256 compute units).
  const int64_t P0 = (n + BK_ROWS - 1) / BK_ROWS;
  L.block = P0 <= BK_MAX_P && P0 * batch <= BK_MAX_WG;
  L.x_off = o;
  if (L.block) o = align256(o + sizeof(unsigned) * batch * bk_xstride(n));
  L.total = o;
  return L;
}

template <int B, int RPT>
hipError_t launch_panel(const PanelParams &pp, int64_t batch, hipStream_t s) {
  hipLaunchKernelGGL((qr_panel_kernel<B, RPT>), dim3((unsigned)batch), dim3(PANEL_THREADS), 0, s,
                     pp);
  return hipGetLastError();
}

// Panel width for `rows` remaining rows: the widest b with b * ceil(rows/512) <= 128.
int panel_width(int64_t rows) {
  if (rows <= 4096) return 16;
  if (rows <= 8192) return 8;
  return 4;
}

}  // namespace

size_t qr_workspace_bytes(int64_t batch, int64_t n) { return qr_layout(batch, n).total; }

hipError_t launch_transpose(float *dst, const float *src, int64_t n, hipStream_t s) {
  const unsigned g = (unsigned)((n + 31) / 32);
  hipLaunchKernelGGL(transpose_kernel, dim3(g, g), dim3(256), 0, s, dst, src, (int)n);
  return hipGetLastError();
}

#define SOAP_TRY(x)                         \
  do {                                      \
    hipError_t e_ = (x);                    \
    if (e_ != hipSuccess) return e_;        \
  } while (0)

namespace {

// Event pool for the fork/join of the look-ahead, one per host thread.  An
// event is re-recorded only after the waits on its previous record have
// been enqueued (waits capture the record current at the time of the call),
// and the cursor cycles through many events before any reuse.
struct EventPool {
  std::vector<hipEvent_t> ev;
  size_t next = 0;
  hipError_t get(hipEvent_t *out) {
    constexpr size_t CAP = 4096;
    if (ev.size() < CAP && next >= ev.size()) {
      hipEvent_t e = nullptr;
      hipError_t err = hipEventCreateWithFlags(&e, hipEventDisableTiming);
      if (err != hipSuccess) return err;
      ev.push_back(e);
    }
    *out = ev[next % ev.size()];
    next = (next + 1) % CAP;
    return hipSuccess;
  }
};

thread_local EventPool t_events;

struct QrCtx {
  float *At, *Q, *Rf;
  int64_t batch, n, sA;
  int ni;
  QrLayout L;
  int cap_small;             // workgroups a small-R block launch may use
  const unsigned *skip;      // per-matrix failed flags (stride sSkip words), or nullptr
  int64_t sSkip;
  unsigned *status;
  unsigned status_bit;
  float *Tb, *Wb, *W2, *Sk, *Pt, *Wi, *dsign, *betas;
  unsigned *cnt;
  unsigned *xch;
  float *TP, *Sx, *Skp, *TQ, *Sq, *TO, *So;
  float *Wn, *Skn;
  float *Skp2;     // split-K partials of the pair T's (the merges use Skp)
  float *Fv;       // V and V T of the forward Q formation
};

hipError_t panel_phase(const QrCtx &x, int64_t ob, hipStream_t s);

// Split-K for a latency-critical product with a single tile row/column
// (M, N <= NB, e.g. the near update's W = Y^T A_next): up to 64 slices of at
// least min_k of K each, within the partial buffer of cap_floats floats.
int narrow_split(int64_t M, int64_t N, int64_t K, int64_t batch, int64_t cap_floats,
                 int64_t min_k = 256) {
  int64_t s = std::min<int64_t>(64, K / min_k);
  s = std::min<int64_t>(s, cap_floats / std::max<int64_t>(1, M * N * batch));
  return (int)std::max<int64_t>(1, s);
}

// Workgroups of block ob's resident-block launch and whether it takes the
// small-R kernel.
int block_launch_p(const QrCtx &x, int64_t ob, bool *small) {
  const int64_t c = ob * NB;
  const int Ps = (int)((x.n - c + BK_ROWS_SMALL - 1) / BK_ROWS_SMALL);
  *small = Ps <= BK_SMALL_MAX_P && Ps * x.batch <= x.cap_small;
  return *small ? Ps : (int)((x.n - c + BK_ROWS - 1) / BK_ROWS);
}

// Factors outer block ob on stream s (resident-block kernel or panel path).
hipError_t factor_block(const QrCtx &x, int64_t ob, hipStream_t s) {
  if (!x.L.block) return panel_phase(x, ob, s);
  const int c = (int)(ob * NB);
  const int nb = (int)std::min<int64_t>(NB, x.n - c);
  bool small = false;
  const int P = block_launch_p(x, ob, &small);
  BlockParams bp{x.At, x.sA, x.ni, c, nb, x.Tb + ob * NB * NB, x.L.sT, x.Rf, x.dsign, x.betas,
                 x.xch, bk_xstride(x.n), bk_area_words(x.n), (int)(ob & 1), P,
                 x.status, x.status_bit};
  const dim3 grid((unsigned)P, (unsigned)x.batch);
  if (small)
    hipLaunchKernelGGL((qr_block_kernel<BK_R_SMALL, BK_K_SMALL>), grid, dim3(BK_THREADS), 0, s, bp);
  else if (P <= BK_MID_MAX_P)
    hipLaunchKernelGGL((qr_block_kernel<BK_R, BK_K_MID>), grid, dim3(BK_THREADS), 0, s, bp);
  else
    hipLaunchKernelGGL((qr_block_kernel<BK_R, BK_K_BIG>), grid, dim3(BK_THREADS), 0, s, bp);
  return hipGetLastError();
}

// Factors the columns of outer block ob (inner panels, their row-parallel
// reductions and applies) on stream s.
hipError_t panel_phase(const QrCtx &x, int64_t ob, hipStream_t s) {
  const int n = x.ni;
  const int c = (int)(ob * NB);
  const int cend = (int)std::min<int64_t>(x.n, c + NB);
  float *Tob = x.Tb + ob * NB * NB;
  for (int ci = c; ci < cend;) {
    const int64_t rows = x.n - ci;
    const int B = panel_width(rows);
    const int beff = std::min(B, cend - ci);
    PanelParams pp{x.At, x.sA, n, c, ci, beff, Tob, x.L.sT, x.Rf, x.dsign, x.betas};
    switch (B) {
      case 16: SOAP_TRY((launch_panel<16, 8>(pp, x.batch, s))); break;
      case 8: SOAP_TRY((launch_panel<8, 16>(pp, x.batch, s))); break;
      default: SOAP_TRY((launch_panel<4, 32>(pp, x.batch, s))); break;
    }
    const int w = cend - (ci + beff);
    {
      const int P = (int)((rows + RCH - 1) / RCH);
      InnerParams ip{x.At, x.sA, n, c, ci, beff, cend, Tob, x.L.sT, x.betas, x.Wi, x.L.sWi, x.Pt,
                     x.L.sPart, x.cnt, P};
      hipLaunchKernelGGL(qr_inner_reduce_kernel, dim3(P, (unsigned)x.batch), dim3(RED_THREADS), 0,
                         s, ip);
      SOAP_TRY(hipGetLastError());
    }
    if (w > 0) {
      ApplyParams ap{x.At, x.sA, n, ci, beff, w, x.Wi, x.L.sWi};
      const unsigned gx = (unsigned)((rows + 255) / 256);
      hipLaunchKernelGGL(qr_inner_apply_kernel, dim3(gx, (unsigned)x.batch), dim3(256), 0, s, ap);
      SOAP_TRY(hipGetLastError());
    }
    ci += beff;
  }
  return hipSuccess;
}

// Applies outer block ob's reflectors to the columns [j0, j1) of A (rows c..n):
// A[c:, j0:j1] -= Y (T^T (Y^T A[c:, j0:j1])), on stream s.
hipError_t trailing_update(const QrCtx &x, int64_t ob, int64_t j0, int64_t j1, hipStream_t s,
                           bool near) {
  const int64_t n = x.n;
  const int64_t c = ob * NB;
  const int64_t nb = std::min<int64_t>(n, c + NB) - c, Kr = n - c, Nt = j1 - j0;
  if (Nt <= 0) return hipSuccess;
  float *Tob = x.Tb + ob * NB * NB;
  // The near update runs beside the others on its own stream: its own
  // buffers.  Only narrow updates (at most NB columns) go there.
  float *Wb = near ? x.Wn : x.Wb, *W2 = near ? x.Wn + NB * NB : x.W2;
  float *Sk = near ? x.Skn : x.Sk;
  const int64_t sW = near ? x.L.sWn : x.L.sWbuf;
  const int64_t skcap = x.batch * (near ? x.L.sSkn : x.L.sSk);
  if (near && Nt > NB) return hipErrorInvalidValue;
  // W = Y^T A[c:n, j0:j1]:  W[i][j] = sum_k At[c+i][c+k] At[j0+j][c+k]
  GemmDesc g1;
  g1.trans_a = 0; g1.trans_b = 1; g1.M = nb; g1.N = Nt; g1.K = Kr;
  g1.A = x.At + c * n + c; g1.lda = n; g1.sA = x.sA;
  g1.B = x.At + j0 * n + c; g1.ldb = n; g1.sB = x.sA;
  g1.C = Wb; g1.ldc = Nt; g1.sC = sW; g1.batch = x.batch;
  g1.splitk = (Nt <= NB) ? narrow_split(nb, Nt, Kr, x.batch, skcap, near ? NEAR_MIN_K : 256)
                          : choose_splitk(nb, Nt, Kr, x.batch, MAX_SPLIT);
  g1.part = Sk;
  // split products sum their slices and form T^T W in one pass (the near
  // update is on the critical path, and so are the far updates of the first
  // half of a large factorization)
  const bool fused = g1.splitk > 1;
  g1.partials_only = fused;
  SOAP_TRY(launch_gemm(g1, s));
  if (fused) {   // W2 = T^T (sum of the partials) in one pass
    // many slices (the near update's): two columns per workgroup, so that
    // each thread's loads are in flight together
    if (g1.splitk > 8)
      hipLaunchKernelGGL(qr_reduce_tt_kernel<2>, dim3((unsigned)((Nt + 1) / 2), (unsigned)x.batch),
                         dim3(256), 0, s, Sk, g1.splitk, (int)nb, (int)Nt, Tob, x.L.sT, W2, sW);
    else
      hipLaunchKernelGGL(qr_reduce_tt_kernel<8>, dim3((unsigned)((Nt + 7) / 8), (unsigned)x.batch),
                         dim3(256), 0, s, Sk, g1.splitk, (int)nb, (int)Nt, Tob, x.L.sT, W2, sW);
    SOAP_TRY(hipGetLastError());
  }
  // W2 = T^T W
  GemmDesc g2;
  g2.trans_a = 1; g2.trans_b = 0; g2.M = nb; g2.N = Nt; g2.K = nb;
  g2.A = Tob; g2.lda = NB; g2.sA = x.L.sT;
  g2.B = Wb; g2.ldb = Nt; g2.sB = sW;
  g2.C = W2; g2.ldc = Nt; g2.sC = sW; g2.batch = x.batch;
  if (!fused) SOAP_TRY(launch_gemm(g2, s));
  // At[j0+j][c+k] -= sum_i W2[i][j] Y[k][i]
  GemmDesc g3;
  g3.trans_a = 1; g3.trans_b = 0; g3.M = Nt; g3.N = Kr; g3.K = nb;
  g3.A = W2; g3.lda = Nt; g3.sA = sW;
  g3.B = x.At + c * n + c; g3.ldb = n; g3.sB = x.sA;
  g3.C = x.At + j0 * n + c; g3.ldc = n; g3.sC = x.sA;
  g3.alpha = -1.f; g3.beta = 1.f; g3.batch = x.batch;
  return launch_gemm(g3, s);
}

// Trailing update of columns j0..n-1 by full pair p (blocks 2p, 2p+1) at
// once, with the pair's T (2NB x 2NB): W = Y^T A[c:n, j0:n] (K = n - c),
// W2 = T^T W, A[c:n, j0:n] -= Y W2 (K = 2NB), c = 2p NB.  Needs the pair's
// square cleared (Y unit lower trapezoidal over rows c.. of the 2NB rows of
// At) and T_p formed.  Rank 2NB: half the passes over the trailing matrix
// of two rank-NB updates, at a higher matrix-core rate.
hipError_t far_update_pair(const QrCtx &x, int64_t p, int64_t j0, hipStream_t s) {
  const int64_t n = x.n, c = 2 * p * NB, w = 2 * NB, Kr = n - c, Nt = n - j0;
  if (Nt <= 0) return hipSuccess;
  const float *Tp = x.TP + p * 4 * NB * NB;
  GemmDesc g1;  // W[i][j] = sum_k At[c+i][c+k] At[j0+j][c+k]
  g1.trans_a = 0; g1.trans_b = 1; g1.M = w; g1.N = Nt; g1.K = Kr;
  g1.A = x.At + c * n + c; g1.lda = n; g1.sA = x.sA;
  g1.B = x.At + j0 * n + c; g1.ldb = n; g1.sB = x.sA;
  g1.C = x.Wb; g1.ldc = Nt; g1.sC = x.L.sWbuf; g1.batch = x.batch;
  g1.splitk = choose_splitk(w, Nt, Kr, x.batch, MAX_SPLIT);
  g1.part = x.Sk;
  SOAP_TRY(launch_gemm(g1, s));
  GemmDesc g2;  // W2 = T^T W
  g2.trans_a = 1; g2.trans_b = 0; g2.M = w; g2.N = Nt; g2.K = w;
  g2.A = Tp; g2.lda = w; g2.sA = x.L.sTP;
  g2.B = x.Wb; g2.ldb = Nt; g2.sB = x.L.sWbuf;
  g2.C = x.W2; g2.ldc = Nt; g2.sC = x.L.sWbuf; g2.batch = x.batch;
  SOAP_TRY(launch_gemm(g2, s));
  GemmDesc g3;  // At[j0+j][c+k] -= sum_i W2[i][j] Y[k][i]
  g3.trans_a = 1; g3.trans_b = 0; g3.M = Nt; g3.N = Kr; g3.K = w;
  g3.A = x.W2; g3.lda = Nt; g3.sA = x.L.sWbuf;
  g3.B = x.At + c * n + c; g3.ldb = n; g3.sB = x.sA;
  g3.C = x.At + j0 * n + c; g3.ldc = n; g3.sC = x.sA;
  g3.alpha = -1.f; g3.beta = 1.f; g3.batch = x.batch;
  return launch_gemm(g3, s);
}

// T of pair p (full blocks a = 2p, b = 2p+1), on stream st (the stream
// that then applies the pair's far update):
//   S = Y_a^T Y_b over rows >= c_b (where Y_b is nonzero), X = T_a S,
//   T_ab = -X T_b into the top-right block of the pair's T, then the
//   diagonal blocks.  Reads only At rows of the two blocks at columns >= c_b
//   and their T, which the concurrent updates and factorizations do not
//   touch.  Its split-K partials are its own (the merges run beside it).
hipError_t pair_t(const QrCtx &x, int64_t p, hipStream_t st) {
  const int64_t n = x.n, ca = 2 * p * NB, cb = ca + NB;
  float *S = x.Sx + p * 2 * NB * NB, *X = S + NB * NB;
  const float *Ta = x.Tb + (2 * p) * NB * NB, *Tbk = Ta + NB * NB;
  float *TP = x.TP + p * 4 * NB * NB;
  GemmDesc gs;  // S[i][j] = sum_r At[ca+i][r] At[cb+j][r], r in [cb, n)
  gs.trans_a = 0; gs.trans_b = 1; gs.M = NB; gs.N = NB; gs.K = n - cb;
  gs.A = x.At + ca * n + cb; gs.lda = n; gs.sA = x.sA;
  gs.B = x.At + cb * n + cb; gs.ldb = n; gs.sB = x.sA;
  gs.C = S; gs.ldc = NB; gs.sC = x.L.sSx; gs.batch = x.batch;
  gs.splitk = narrow_split(NB, NB, n - cb, x.batch, x.batch * x.L.sSkp);
  gs.part = x.Skp2;
  SOAP_TRY(launch_gemm(gs, st));
  GemmDesc gx;  // X = T_a S
  gx.M = NB; gx.N = NB; gx.K = NB;
  gx.A = Ta; gx.lda = NB; gx.sA = x.L.sT;
  gx.B = S; gx.ldb = NB; gx.sB = x.L.sSx;
  gx.C = X; gx.ldc = NB; gx.sC = x.L.sSx; gx.batch = x.batch;
  SOAP_TRY(launch_gemm(gx, st));
  GemmDesc gt;  // T_ab = -X T_b
  gt.M = NB; gt.N = NB; gt.K = NB;
  gt.A = X; gt.lda = NB; gt.sA = x.L.sSx;
  gt.B = Tbk; gt.ldb = NB; gt.sB = x.L.sT;
  gt.C = TP + NB; gt.ldc = 2 * NB; gt.sC = x.L.sTP; gt.alpha = -1.f; gt.batch = x.batch;
  SOAP_TRY(launch_gemm(gt, st));
  hipLaunchKernelGGL(qr_assemble_pair_t_kernel, dim3(64, (unsigned)x.batch), dim3(256), 0, st, TP,
                     x.L.sTP, Ta, Tbk, x.L.sT, NB, NB);
  return hipGetLastError();
}

// T of group g at level lv (lv = 2: quads, pairs of full pairs; lv = 3:
// octs, pairs of full quads), on stream st, from the T's of its halves a, b
// (level lv - 1, hw = NB 2^(lv-1) reflectors each): S = Y_a^T Y_b,
// X = T_a S, T_ab = -X T_b, then the diagonal blocks.  The blocks of Y_b
// after its first still hold R entries above their diagonal blocks (the
// factorization is running), so S is formed block by block of Y_b, each over
// the rows where that block's reflectors live.  Reads only At rows of the
// group at columns >= c_b, which the concurrent trailing update does not
// touch.
hipError_t merge_t(const QrCtx &x, int lv, int64_t g, hipStream_t st) {
  const int64_t n = x.n, hw = (int64_t)NB << (lv - 1), W = 2 * hw;
  const int64_t ca = g * W, cb = ca + hw;
  float *Tlo = lv == 2 ? x.TP : x.TQ, *Thi = lv == 2 ? x.TQ : x.TO;
  float *Sg = lv == 2 ? x.Sq : x.So;
  const int64_t sLo = lv == 2 ? x.L.sTP : x.L.sTQ, sHi = lv == 2 ? x.L.sTQ : x.L.sTO;
  const int64_t sS = lv == 2 ? x.L.sSq : x.L.sSo;
  float *S = Sg + g * 2 * hw * hw, *X = S + hw * hw;
  const float *Ta = Tlo + (2 * g) * hw * hw, *Tbg = Ta + hw * hw;
  float *TG = Thi + g * W * W;
  for (int64_t j = 0; j < hw / NB; ++j) {   // S[:, j NB : (j+1) NB]
    const int64_t cr = cb + j * NB;
    GemmDesc gs;  // S[i][jj] = sum_r At[ca+i][r] At[cr+jj][r], r in [cr, n)
    gs.trans_a = 0; gs.trans_b = 1; gs.M = hw; gs.N = NB; gs.K = n - cr;
    gs.A = x.At + ca * n + cr; gs.lda = n; gs.sA = x.sA;
    gs.B = x.At + cr * n + cr; gs.ldb = n; gs.sB = x.sA;
    gs.C = S + j * NB; gs.ldc = hw; gs.sC = sS; gs.batch = x.batch;
    gs.splitk = narrow_split(hw, NB, n - cr, x.batch, x.batch * x.L.sSkp);
    gs.part = x.Skp;
    SOAP_TRY(launch_gemm(gs, st));
  }
  GemmDesc gx;  // X = T_a S
  gx.M = hw; gx.N = hw; gx.K = hw;
  gx.A = Ta; gx.lda = hw; gx.sA = sLo;
  gx.B = S; gx.ldb = hw; gx.sB = sS;
  gx.C = X; gx.ldc = hw; gx.sC = sS; gx.batch = x.batch;
  SOAP_TRY(launch_gemm(gx, st));
  GemmDesc gt;  // T_ab = -X T_b
  gt.M = hw; gt.N = hw; gt.K = hw;
  gt.A = X; gt.lda = hw; gt.sA = sS;
  gt.B = Tbg; gt.ldb = hw; gt.sB = sLo;
  gt.C = TG + hw; gt.ldc = W; gt.sC = sHi; gt.alpha = -1.f; gt.batch = x.batch;
  SOAP_TRY(launch_gemm(gt, st));
  hipLaunchKernelGGL(qr_assemble_pair_t_kernel, dim3(64, (unsigned)x.batch), dim3(256), 0, st, TG,
                     sHi, Ta, Tbg, sLo, (int)hw, (int)hw);
  return hipGetLastError();
}

// Q[c:, c:] -= Y (T (Y^T Q[c:, c:])) for the w reflectors stored in At rows
// c..c+w-1 (zero above row c + their index) with T (w x w, leading dimension
// ldt, batch stride sT).  The groups are applied from the last to the first,
// so rows and columns c..c+w-1 of Q still hold diag(d) here: the first w
// columns of W = Y^T Q[c:, c:] are Y's top w x w block scaled by d, and the
// rest is a product over the trailing Kr - w rows and columns only.
hipError_t q_update(const QrCtx &x, int64_t c, int64_t w, const float *T, int64_t ldt,
                    int64_t sT, hipStream_t s) {
  const int64_t n = x.n, Kr = n - c, Kt = Kr - w;
  {
    const unsigned gx = (unsigned)std::min<int64_t>((w * w + 255) / 256, 1024);
    hipLaunchKernelGGL(qr_q_head_kernel, dim3(gx, (unsigned)x.batch), dim3(256), 0, s, x.Wb, Kr,
                       x.L.sWbuf, x.At, x.sA, x.dsign, x.ni, c, (int)w, x.skip, x.sSkip);
    SOAP_TRY(hipGetLastError());
  }
  // W[:, w:] = Y[w:, :]^T Q[c+w:, c+w:]:  op(A)[i][k] = At[c+i][c+w+k]
  // (nothing for the last group, whose Kr is w)
  if (Kt > 0) {
    GemmDesc g1;
    g1.trans_a = 0; g1.trans_b = 0; g1.M = w; g1.N = Kt; g1.K = Kt;
    g1.A = x.At + c * n + c + w; g1.lda = n; g1.sA = x.sA;
    g1.B = x.Q + (c + w) * n + c + w; g1.ldb = n; g1.sB = x.sA;
    g1.C = x.Wb + w; g1.ldc = Kr; g1.sC = x.L.sWbuf; g1.batch = x.batch;
    // A few hundred tiles of long K (the rank-1024 groups) leave a last,
    // mostly empty round of workgroups: K slices of a quarter or half the
    // length (as many as the partial buffer holds) balance it.
    const int g1max = (int)(x.L.sSk / n / std::max<int64_t>(w, 2 * NB));
    g1.splitk = choose_splitk(w, Kt, Kt, x.batch, g1max);
    if (g1.splitk == 1 && g1max >= 4 && Kt >= 8192) g1.splitk = 4;
    else if (g1.splitk == 1 && g1max >= 2 && Kt >= 4096) g1.splitk = 2;
    g1.part = x.Sk;
    g1.skip = x.skip; g1.sSkip = x.sSkip;
    SOAP_TRY(launch_gemm(g1, s));
  }
  GemmDesc g2;  // W2 = T W
  g2.trans_a = 0; g2.trans_b = 0; g2.M = w; g2.N = Kr; g2.K = w;
  g2.A = T; g2.lda = ldt; g2.sA = sT;
  g2.B = x.Wb; g2.ldb = Kr; g2.sB = x.L.sWbuf;
  g2.C = x.W2; g2.ldc = Kr; g2.sC = x.L.sWbuf; g2.batch = x.batch;
  g2.skip = x.skip; g2.sSkip = x.sSkip;
  SOAP_TRY(launch_gemm(g2, s));
  GemmDesc g3;  // Q[c:n, c:n] -= Y W2:  op(A)[k][i] = Y[k][i] = At[c+i][c+k]
  g3.trans_a = 1; g3.trans_b = 0; g3.M = Kr; g3.N = Kr; g3.K = w;
  g3.A = x.At + c * n + c; g3.lda = n; g3.sA = x.sA;
  g3.B = x.W2; g3.ldb = Kr; g3.sB = x.L.sWbuf;
  g3.C = x.Q + c * n + c; g3.ldc = n; g3.sC = x.sA;
  g3.alpha = -1.f; g3.beta = 1.f; g3.batch = x.batch;
  g3.skip = x.skip; g3.sSkip = x.sSkip;
  return launch_gemm(g3, s);
}

// Forward Q formation: Q[:, c:] -= ((Q[:, c:] Y) T) Y^T for the w
// reflectors stored in At rows c..c+w-1 (explicit: zero before their pivot,
// one on it), i.e. Q <- Q (I - Y T Y^T).  Applied group after group from
// the first on, it accumulates Q = H_1 H_2 ... (the column signs follow at
// the copy out).  Every row of Q takes part (2 n^3 flops in all, against
// (4/3) n^3 backwards), but each group's update can run as soon as its T
// exists, beside the factorization; capped to `max_wg` workgroups so that
// whole compute units stay free for the block kernels.
hipError_t q_forward_update(const QrCtx &x, int64_t c, int64_t w, const float *T, int64_t ldt,
                            int64_t sT, int max_wg, hipStream_t s) {
  const int64_t n = x.n, Kr = n - c;
  float *V = x.Fv, *V2 = x.Fv + 2 * NB * n;
  GemmDesc g1;  // V = Q[:, c:] Y:  op(B)[k][j] = Y[k][j] = At[c+j][c+k]
  g1.trans_a = 0; g1.trans_b = 1; g1.M = n; g1.N = w; g1.K = Kr;
  g1.A = x.Q + c; g1.lda = n; g1.sA = x.sA;
  g1.B = x.At + c * n + c; g1.ldb = n; g1.sB = x.sA;
  g1.C = V; g1.ldc = w; g1.sC = x.L.sFv; g1.batch = x.batch;
  g1.skip = x.skip; g1.sSkip = x.sSkip; g1.max_wg = max_wg;
  SOAP_TRY(launch_gemm(g1, s));
  GemmDesc g2;  // V2 = V T
  g2.M = n; g2.N = w; g2.K = w;
  g2.A = V; g2.lda = w; g2.sA = x.L.sFv;
  g2.B = T; g2.ldb = ldt; g2.sB = sT;
  g2.C = V2; g2.ldc = w; g2.sC = x.L.sFv; g2.batch = x.batch;
  g2.skip = x.skip; g2.sSkip = x.sSkip; g2.max_wg = max_wg;
  SOAP_TRY(launch_gemm(g2, s));
  GemmDesc g3;  // Q[:, c:] -= V2 Y^T:  B = Y^T = At rows c..c+w-1 from column c
  g3.M = n; g3.N = Kr; g3.K = w;
  g3.A = V2; g3.lda = w; g3.sA = x.L.sFv;
  g3.B = x.At + c * n + c; g3.ldb = n; g3.sB = x.sA;
  g3.C = x.Q + c; g3.ldc = n; g3.sC = x.sA;
  g3.alpha = -1.f; g3.beta = 1.f; g3.batch = x.batch;
  g3.skip = x.skip; g3.sSkip = x.sSkip; g3.max_wg = max_wg;
  return launch_gemm(g3, s);
}

// Workgroups of a forward Q update running beside the factorization.
constexpr int FWD_MAX_WG = 160;
// Largest order whose paired QR forms Q forwards: the block chain leaves
// the device mostly idle up to here (a square 2048 step 7.8 -> 7.3 ms, 4096
// 25.3 -> 23.9 ms); from 6144 on its far updates already fill it and the
// extra flops slow the chain (6144: 60.8 -> 63.7 ms, 8192: 123 -> 135 ms).
constexpr int64_t FWD_MAX_N = 4096;

std::atomic<unsigned> g_force_give_up{0};

// Workgroups of one block-kernel launch (R rows per thread) that the current
// device holds at once, halved: the two factors' QRs of a step may run
// together.  Asked once per device and kernel.
int resident_cap(bool small, hipError_t *err) {
  static std::mutex mu;
  static int cap[64][2] = {};
  int dev = 0;
  if ((*err = hipGetDevice(&dev)) != hipSuccess) return 0;
  if (dev < 0 || dev >= 64) {
    *err = hipErrorInvalidDevice;
    return 0;
  }
  std::lock_guard<std::mutex> g(mu);
  int &c = cap[dev][small ? 1 : 0];
  if (c == 0) {
    int per_cu = 0, per_cu_mid = 0, cus = 0;
    if (small) {
      *err = hipOccupancyMaxActiveBlocksPerMultiprocessor(
          &per_cu, qr_block_kernel<BK_R_SMALL, BK_K_SMALL>, BK_THREADS, 0);
    } else {
      // (the 32-row launches take one of two kernels: the smaller count)
      *err = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, qr_block_kernel<BK_R, BK_K_BIG>,
                                                          BK_THREADS, 0);
      if (*err == hipSuccess)
        *err = hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &per_cu_mid, qr_block_kernel<BK_R, BK_K_MID>, BK_THREADS, 0);
      per_cu = std::min(per_cu, per_cu_mid);
    }
    if (*err != hipSuccess) return 0;
    if ((*err = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) !=
        hipSuccess)
      return 0;
    c = std::max(1, per_cu * cus / 2);
  }
  return c;
}

}  // namespace

void qr_force_give_up(unsigned mask) { g_force_give_up.store(mask); }

hipError_t qr_block_path(int64_t batch, int64_t n, bool *out) {
  *out = qr_layout(batch, n).block;
  if (!*out) return hipSuccess;
  hipError_t err = hipSuccess;
  const int cap_big = resident_cap(false, &err);
  if (err != hipSuccess) return err;
  const int64_t P0 = (n + BK_ROWS - 1) / BK_ROWS;
  *out = P0 * batch <= std::min(BK_MAX_WG, cap_big);
  return hipSuccess;
}

hipError_t qr_factor_and_form_q(float *At, float *Q, float *Rf, int64_t batch, int64_t n,
                                void *ws, size_t ws_bytes, hipStream_t s, hipStream_t sp,
                                hipStream_t st, unsigned *status, unsigned status_bit,
                                hipEvent_t q_free, hipEvent_t mid, float mid_frac,
                                const std::function<hipError_t()> &at_mid,
                                const QrSplitOut *split) {
  QrCtx x;
  x.L = qr_layout(batch, n);
  if (ws_bytes < x.L.total) return hipErrorInvalidValue;
  if (split && (Rf || batch != 2 * split->half || !split->QA || !split->QB))
    return hipErrorInvalidValue;
  x.cap_small = BK_MAX_WG;
  if (x.L.block) {   // resident blocks only where the device holds them all at once
    SOAP_TRY(qr_block_path(batch, n, &x.L.block));
    hipError_t err = hipSuccess;
    const int cap_small = resident_cap(true, &err);
    if (err != hipSuccess) return err;
    x.cap_small = std::min(BK_MAX_WG, cap_small);
  }
  // (with two destinations the scatter of the Q's reports failures per half)
  x.status = split ? nullptr : status;
  x.status_bit = split ? 0u : status_bit;
  char *base = static_cast<char *>(ws);
  x.At = At; x.Q = Q; x.Rf = Rf; x.batch = batch; x.n = n; x.sA = n * n; x.ni = (int)n;
  x.Tb = reinterpret_cast<float *>(base + x.L.t_off);
  x.Wb = reinterpret_cast<float *>(base + x.L.w_off);
  x.W2 = reinterpret_cast<float *>(base + x.L.w2_off);
  x.Sk = reinterpret_cast<float *>(base + x.L.sk_off);
  x.Pt = reinterpret_cast<float *>(base + x.L.part_off);
  x.Wi = reinterpret_cast<float *>(base + x.L.wi_off);
  x.dsign = reinterpret_cast<float *>(base + x.L.d_off);
  x.betas = reinterpret_cast<float *>(base + x.L.b_off);
  x.cnt = reinterpret_cast<unsigned *>(base + x.L.cnt_off);
  x.xch = reinterpret_cast<unsigned *>(base + x.L.x_off);
  x.TP = reinterpret_cast<float *>(base + x.L.tp_off);
  x.Sx = reinterpret_cast<float *>(base + x.L.sx_off);
  x.Skp = reinterpret_cast<float *>(base + x.L.skp_off);
  x.Skp2 = reinterpret_cast<float *>(base + x.L.skp2_off);
  x.TQ = reinterpret_cast<float *>(base + x.L.tq_off);
  x.Sq = reinterpret_cast<float *>(base + x.L.sq_off);
  x.TO = reinterpret_cast<float *>(base + x.L.to_off);
  x.So = reinterpret_cast<float *>(base + x.L.so_off);
  x.Wn = reinterpret_cast<float *>(base + x.L.wn_off);
  x.Skn = reinterpret_cast<float *>(base + x.L.skn_off);
  x.Fv = reinterpret_cast<float *>(base + x.L.fv_off);
  const int64_t nob = x.L.nob, np = x.L.np;
  // With two destinations Q is the call's own buffer and, up to order
  // FWD_MAX_N, is written as the factorization runs: formed forwards, group
  // by group beside it (a failed matrix's partial Q is never copied out).
  const bool fwd = split != nullptr && n <= FWD_MAX_N;

  SOAP_TRY(launch_zero_u32(x.cnt, batch, s));
  x.skip = nullptr;
  x.sSkip = 0;
  if (x.L.block) {  // header clear, area 0 empty, area 1 emptied by the first block
    const int64_t xs = bk_xstride(n), aw = bk_area_words(n);
    const unsigned gx = (unsigned)std::min<int64_t>((BK_XHDR + aw + 255) / 256, 1024);
    hipLaunchKernelGGL(qr_xch_init_kernel, dim3(gx, (unsigned)batch), dim3(256), 0, s, x.xch, xs,
                       aw);
    SOAP_TRY(hipGetLastError());
    x.skip = x.xch + BK_XFAILED;
    x.sSkip = xs;
    for (int h = 0; h < (split ? 2 : 1); ++h) {
      const unsigned bit = split ? (h ? split->bitB : split->bitA) : status_bit;
      const int64_t cnt = split ? split->half : batch;
      if (g_force_give_up.load() & bit) {
        hipLaunchKernelGGL(qr_raise_abort_kernel,
                           dim3((unsigned)std::min<int64_t>((cnt + 63) / 64, 1024)), dim3(64), 0,
                           s, x.xch + h * cnt * xs, xs, cnt);
        SOAP_TRY(hipGetLastError());
      }
    }
  }

  // Look-ahead of depth two.  The block stream sp carries the critical
  // chain: block ob+1's columns updated by block ob (the "near" update),
  // then block ob+1 factored.  Stream s applies the rest of block ob's
  // trailing update once block ob is factored: block by block to the
  // columns of blocks ob+2 and (ob even) ob+3, which the next near updates
  // wait for; the columns past those by pairs of blocks: once block 2p+1 is
  // factored, the pair's T is formed and the pair updates every column from
  // block 2p+4 on at once (rank 2NB), while blocks 2p+2 and 2p+3 are
  // factored.  The quad and oct T's of the Q formation follow on st.
  hipEvent_t ev;
  SOAP_TRY(t_events.get(&ev));
  SOAP_TRY(hipEventRecord(ev, s));
  SOAP_TRY(hipStreamWaitEvent(sp, ev, 0));
  if (fwd) {   // Q = I on the stream of the forward updates
    SOAP_TRY(hipStreamWaitEvent(st, ev, 0));
    const unsigned gx = (unsigned)std::min<int64_t>((n * n + 255) / 256, 2048);
    hipLaunchKernelGGL(qr_identity_kernel, dim3(gx, (unsigned)batch), dim3(256), 0, st, Q, x.ni,
                       x.sA);
    SOAP_TRY(hipGetLastError());
  }
  SOAP_TRY(factor_block(x, 0, sp));
  hipEvent_t ev_f;                                // block ob factored (on sp)
  SOAP_TRY(t_events.get(&ev_f));
  SOAP_TRY(hipEventRecord(ev_f, sp));
  hipEvent_t ev_a = nullptr;                      // block ob+1's columns current (on s)
  const int64_t mid_ob = (int64_t)(mid_frac * (float)nob);
  bool mid_done = (mid == nullptr && !at_mid);
  auto col0 = [&](int64_t b) { return std::min<int64_t>(n, b * NB); };
  for (int64_t ob = 0; ob < nob; ++ob) {
    if (!mid_done && ob >= mid_ob) {
      if (mid) SOAP_TRY(hipEventRecord(mid, s));
      if (at_mid) SOAP_TRY(at_mid());
      mid_done = true;
    }
    hipEvent_t ev_next = nullptr;
    if (ob + 1 < nob) {
      if (ev_a) SOAP_TRY(hipStreamWaitEvent(sp, ev_a, 0));
      SOAP_TRY(trailing_update(x, ob, col0(ob + 1), col0(ob + 2), sp, true));  // near
      SOAP_TRY(factor_block(x, ob + 1, sp));
      SOAP_TRY(t_events.get(&ev_next));
      SOAP_TRY(hipEventRecord(ev_next, sp));
    }
    SOAP_TRY(hipStreamWaitEvent(s, ev_f, 0));                   // block ob factored
    ev_a = nullptr;
    if (ob + 2 < nob) {                                         // block ob+2's columns
      SOAP_TRY(trailing_update(x, ob, col0(ob + 2), col0(ob + 3), s, false));
      SOAP_TRY(t_events.get(&ev_a));
      SOAP_TRY(hipEventRecord(ev_a, s));
    }
    if (ob % 2 == 0) {
      if (ob + 3 < nob)                                         // block ob+3's columns
        SOAP_TRY(trailing_update(x, ob, col0(ob + 3), col0(ob + 4), s, false));
    } else if (ob / 2 < np) {                                   // pair (ob-1, ob) complete
      const int64_t p = ob / 2;
      hipLaunchKernelGGL(qr_clear_pair_square_kernel, dim3(64, (unsigned)batch), dim3(256), 0, s,
                         x.At, x.sA, x.Rf, x.dsign, x.ni, (int)((ob - 1) * NB));
      SOAP_TRY(hipGetLastError());
      SOAP_TRY(pair_t(x, p, s));
      if (fwd) {                                           // Q <- Q (I - Y_p T_p Y_p^T)
        SOAP_TRY(t_events.get(&ev));
        SOAP_TRY(hipEventRecord(ev, s));
        SOAP_TRY(hipStreamWaitEvent(st, ev, 0));
        SOAP_TRY(q_forward_update(x, 2 * p * NB, 2 * NB, x.TP + p * 4 * NB * NB, 2 * NB, x.L.sTP,
                                  FWD_MAX_WG, st));
      } else if (p % 2 == 1 && p / 2 < x.L.nq) {           // quad (p-1, p) complete
        SOAP_TRY(t_events.get(&ev));
        SOAP_TRY(hipEventRecord(ev, s));
        SOAP_TRY(hipStreamWaitEvent(st, ev, 0));
        const int64_t q = p / 2;
        SOAP_TRY(merge_t(x, 2, q, st));
        if (q % 2 == 1 && q / 2 < x.L.no) SOAP_TRY(merge_t(x, 3, q / 2, st));   // oct (q-1, q)
      }
      if (ob + 3 < nob) SOAP_TRY(far_update_pair(x, p, col0(ob + 3), s));   // blocks ob+3..
    } else if (ob + 3 < nob) {
      return hipErrorInvalidValue;   // unreachable: unpaired blocks have no columns past ob+2
    }
    if (ev_next) ev_f = ev_next;
  }
  if (!mid_done) {
    if (mid) SOAP_TRY(hipEventRecord(mid, s));
    if (at_mid) SOAP_TRY(at_mid());
  }
  if (np > 0 || fwd) {                                          // pair T's (or Q) done
    SOAP_TRY(t_events.get(&ev));
    SOAP_TRY(hipEventRecord(ev, st));
    SOAP_TRY(hipStreamWaitEvent(s, ev, 0));
  }
  if (Rf) {
    const int64_t nn = n * n;
    const unsigned gx = (unsigned)std::min<int64_t>((nn + 255) / 256, 2048);
    hipLaunchKernelGGL(qr_extract_r_kernel, dim3(gx, (unsigned)batch), dim3(256), 0, s, At, Rf,
                       x.dsign, x.ni, x.sA, (int)np);
    SOAP_TRY(hipGetLastError());
  }
  if (fwd) {   // the blocks past the last full pair, forwards
    for (int64_t ob = 2 * np; ob < nob; ++ob) {
      const int64_t c = ob * NB;
      SOAP_TRY(q_forward_update(x, c, std::min<int64_t>(n, c + NB) - c, x.Tb + ob * NB * NB, NB,
                                x.L.sT, 0, s));
    }
  } else {
    if (np > 0) {   // R is no longer needed: clear it above the block rows of every column
      const unsigned gx = (unsigned)std::min<int64_t>((n * n + 255) / 256, 2048);
      hipLaunchKernelGGL(qr_zero_above_blocks_kernel, dim3(gx, (unsigned)batch), dim3(256), 0, s,
                         At, x.ni, x.sA);
      SOAP_TRY(hipGetLastError());
    }

    // Explicit Q (row-major), accumulated backwards from diag(d).
    if (q_free) SOAP_TRY(hipStreamWaitEvent(s, q_free, 0));
    {
      const unsigned gx = (unsigned)std::min<int64_t>((n * n + 255) / 256, 2048);
      hipLaunchKernelGGL(qr_init_q_kernel, dim3(gx, (unsigned)batch), dim3(256), 0, s, Q, x.dsign,
                         x.ni, x.sA, x.skip, x.sSkip);
      SOAP_TRY(hipGetLastError());
    }
    // Backwards: the blocks past the last full pair one by one, then the
    // pairs, quads and octs past the last full group of the next size as
    // rank-2NB, 4NB and 8NB updates (longer K per product: the update runs
    // nearer the matrix cores' rate than with rank 256).
    const int64_t nq = x.L.nq, no = x.L.no;
    for (int64_t ob = nob - 1; ob >= 2 * np; --ob) {
      const int64_t c = ob * NB;
      SOAP_TRY(q_update(x, c, std::min<int64_t>(n, c + NB) - c, x.Tb + ob * NB * NB, NB, x.L.sT, s));
    }
    for (int64_t p = np - 1; p >= 2 * nq; --p)
      SOAP_TRY(q_update(x, 2 * p * NB, 2 * NB, x.TP + p * 4 * NB * NB, 2 * NB, x.L.sTP, s));
    for (int64_t q = nq - 1; q >= 2 * no; --q)
      SOAP_TRY(q_update(x, 4 * q * NB, 4 * NB, x.TQ + q * 16 * NB * NB, 4 * NB, x.L.sTQ, s));
    for (int64_t o8 = no - 1; o8 >= 0; --o8)
      SOAP_TRY(q_update(x, 8 * o8 * NB, 8 * NB, x.TO + o8 * 64 * NB * NB, 8 * NB, x.L.sTO, s));
  }
  if (split) {
    const unsigned gx = (unsigned)std::min<int64_t>((n * n / 4 + 255) / 256, 1024);
    hipLaunchKernelGGL(qr_scatter_q_kernel, dim3(std::max(gx, 1u), (unsigned)batch), dim3(256), 0,
                       s, Q, split->QA, split->QB, split->half, x.ni, fwd ? x.dsign : nullptr,
                       x.skip, x.sSkip, status, split->bitA, split->bitB);
    SOAP_TRY(hipGetLastError());
  }
  return hipSuccess;
}

}  // namespace soap
