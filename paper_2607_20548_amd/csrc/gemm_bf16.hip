// bfloat16 products of the Muon Newton-Schulz iteration on the CDNA4 matrix
// cores (v_mfma_f32_32x32x16_bf16): C = round_bf16(alpha * P Q^T + beta * D)
// with P (M x K), Q (N x K) and D, C (M x N) bfloat16, row-major, every row
// k-contiguous.  The sum is accumulated in fp32 and rounded to bfloat16 once
// (nearest, ties to even), after the epilogue's linear combination.
//
// Tiling: a 256-thread workgroup (4 wave64s, 2 x 2) computes a 128 x 128 tile;
// each wave owns 64 x 64 as 2 x 2 MFMA 32x32 accumulators.  K advances in
// slabs of 64 staged through double-buffered LDS as [x][k] rows padded to 72
// bfloat16 (144 bytes, so that the 16-byte reads of 16 consecutive lanes fall
// in distinct banks); at MFMA step q a lane (row xl, half h) feeds the 8
// values k = 16 q + 8 h .. +7 of its row, the same k for both operands.
// Global loads are 16 bytes (8 bfloat16) at addresses clamped into the
// operand; rows past the operand only reach outputs that are never written,
// and k past K is zeroed at the LDS store of the last slab.
//
// SYRK mode launches only the tiles on or below the diagonal and mirrors
// each stored value, so C is bitwise symmetric (for P = Q).  A second output
// Ct = C^T is optional (the iterate is kept in both layouts so that every
// product reads k-contiguous rows).
#include "internal.h"

#include <algorithm>

namespace soap {
namespace {

typedef float v16f __attribute__((ext_vector_type(16)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

constexpr int TB = 128;          // tile rows and columns
constexpr int KB = 64;           // K slab (bfloat16 values)
constexpr int LDK = KB + 8;      // LDS row stride in bfloat16
constexpr int NTH = 256;
constexpr int TILE_U16 = TB * LDK;

enum { BMODE_GENERAL = 0, BMODE_SYRK = 1 };

struct BfParams {
  int M, N, K;
  const uint16_t *P; int64_t ldp, sP;
  const uint16_t *Q; int64_t ldq, sQ;
  const uint16_t *D; int64_t ldd, sD;
  uint16_t *C; int64_t ldc, sC;
  uint16_t *Ct; int64_t ldct, sCt;
  float alpha, beta;
  int tiles_m, tiles_n, ntiles;
};

__device__ __forceinline__ uint16_t to_bf16(float f) {   // nearest, ties to even
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu) != 0u)
    return (uint16_t)((u >> 16) | 0x0040u);                  // NaN stays a (quiet) NaN
  return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}
__device__ __forceinline__ float from_bf16(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// One operand slab: 128 rows x 64 k as 1024 chunks of 8 values, four per
// thread (chunk = tid + 256 s: row chunk >> 3, k offset 8 (chunk & 7)).
struct Slab {
  uint4 r[4];
  __device__ __forceinline__ void load(const uint16_t *__restrict__ base, int64_t ld, int x0,
                                       int k0, int X, int K, int tid) {
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int c = tid + NTH * s;
      const int x = min(x0 + (c >> 3), X - 1);
      const int k = min(k0 + 8 * (c & 7), K - 8);
      r[s] = *reinterpret_cast<const uint4 *>(base + (int64_t)x * ld + k);
    }
  }
  // kvalid: k-values of this slab inside K (KB except in the last slab).
  __device__ __forceinline__ void store(uint16_t *lds, int tid, int kvalid) {
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int c = tid + NTH * s;
      if (8 * (c & 7) >= kvalid) r[s] = make_uint4(0u, 0u, 0u, 0u);   // K % 8 == 0
      *reinterpret_cast<uint4 *>(lds + (c >> 3) * LDK + 8 * (c & 7)) = r[s];
    }
  }
};

template <int MODE>
__device__ __forceinline__ void bf_tile_coords(const BfParams &p, int t, int &tm, int &tn) {
  const int nt = p.ntiles;
  if ((nt & 7) == 0) t = (t & 7) * (nt >> 3) + (t >> 3);   // contiguous run per XCD
  if (MODE == BMODE_SYRK) {
    int r = (int)((sqrtf(8.f * (float)t + 1.f) - 1.f) * 0.5f);
    while ((r + 1) * (r + 2) / 2 <= t) ++r;
    while (r * (r + 1) / 2 > t) --r;
    tm = r;
    tn = t - r * (r + 1) / 2;
  } else {
    const int per_group = 8 * p.tiles_n;
    const int group = t / per_group;
    const int first_m = group * 8;
    const int gsz = min(p.tiles_m - first_m, 8);
    const int in_group = t - group * per_group;
    tm = first_m + in_group % gsz;
    tn = in_group / gsz;
  }
}

template <int MODE>
__global__ __launch_bounds__(NTH, 2) void gemm_bf16_nt(BfParams p) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[2 * 2 * TILE_U16];
  int tm, tn;
  bf_tile_coords<MODE>(p, blockIdx.x, tm, tn);
  const int64_t bz = blockIdx.z;
  const uint16_t *P = p.P + bz * p.sP;
  const uint16_t *Q = p.Q + bz * p.sQ;
  const int m0 = tm * TB, n0 = tn * TB;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int xl = lane & 31, h = lane >> 5;

  v16f acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  auto buf = [&](int stage, int which) { return lds + (stage * 2 + which) * TILE_U16; };
  const int nk = (p.K + KB - 1) / KB;
  Slab sa, sb;
  if (nk > 0) {
    sa.load(P, p.ldp, m0, 0, p.M, p.K, tid);
    sb.load(Q, p.ldq, n0, 0, p.N, p.K, tid);
    const int kv = min(KB, p.K);
    sa.store(buf(0, 0), tid, kv);
    sb.store(buf(0, 1), tid, kv);
  }
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) {
      sa.load(P, p.ldp, m0, (kt + 1) * KB, p.M, p.K, tid);
      sb.load(Q, p.ldq, n0, (kt + 1) * KB, p.N, p.K, tid);
    }
    const uint16_t *la = buf(cur, 0), *lb = buf(cur, 1);
#pragma unroll
    for (int q = 0; q < KB / 16; ++q) {
      v8bf fa[2], fb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        fa[i] = __builtin_bit_cast(
            v8bf, *reinterpret_cast<const uint4 *>(la + (wm * 64 + 32 * i + xl) * LDK + 16 * q + 8 * h));
#pragma unroll
      for (int j = 0; j < 2; ++j)
        fb[j] = __builtin_bit_cast(
            v8bf, *reinterpret_cast<const uint4 *>(lb + (wn * 64 + 32 * j + xl) * LDK + 16 * q + 8 * h));
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
    if (more) {
      const int kv = min(KB, p.K - (kt + 1) * KB);
      sa.store(buf(cur ^ 1, 0), tid, kv);
      sb.store(buf(cur ^ 1, 1), tid, kv);
    }
    __syncthreads();
  }

  // Epilogue.  Accumulator register r of block (i, j) holds
  // C[row0 + 8 (r/4) + 4 h + r%4][col0 + xl].
  uint16_t *C = p.C + bz * p.sC;
  const uint16_t *D = p.D ? p.D + bz * p.sD : nullptr;
  uint16_t *Ct = p.Ct ? p.Ct + bz * p.sCt : nullptr;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = n0 + wn * 64 + 32 * j + xl;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int rowb = m0 + wm * 64 + 32 * i + 8 * g + 4 * h;
        uint16_t v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int row = rowb + e;
          float x = p.alpha * acc[i][j][4 * g + e];
          if (D && row < p.M && col < p.N) x += p.beta * from_bf16(D[(int64_t)row * p.ldd + col]);
          v[e] = to_bf16(x);
        }
        if (col >= p.N) continue;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int row = rowb + e;
          if (row >= p.M) continue;
          if (MODE == BMODE_SYRK && row < col) continue;   // the mirror is written by its owner
          C[(int64_t)row * p.ldc + col] = v[e];
          if (MODE == BMODE_SYRK && row != col) C[(int64_t)col * p.ldc + row] = v[e];
        }
        if (Ct) {   // Ct[col][rowb .. rowb+3]: one 8-byte store when all four rows exist
          uint16_t *dst = Ct + (int64_t)col * p.ldct + rowb;
          if (rowb + 3 < p.M) {
            *reinterpret_cast<uint2 *>(dst) =
                make_uint2((uint32_t)v[0] | ((uint32_t)v[1] << 16), (uint32_t)v[2] | ((uint32_t)v[3] << 16));
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (rowb + e < p.M) dst[e] = v[e];
          }
        }
      }
    }
}

// X_0 in both layouts: Xo = round_bf16(inv * S) (rows x cols) and Xt = Xo^T,
// through 32 x 32 LDS tiles; S is fp32 (transposed on input when trans).
__global__ __launch_bounds__(256) void bf16_scale_both_kernel(const float *__restrict__ S,
                                                              int rows, int cols, int trans,
                                                              const float *__restrict__ inv,
                                                              uint16_t *__restrict__ Xo,
                                                              uint16_t *__restrict__ Xt) {
  __shared__ uint16_t tile[32][34];
  const int64_t bz = blockIdx.z;
  const int64_t rc = (int64_t)rows * cols;
  const float *Sb = S + bz * rc;
  uint16_t *Xob = Xo + bz * rc, *Xtb = Xt + bz * rc;
  const float sc = inv[bz];
  const int r0 = blockIdx.y * 32, c0 = blockIdx.x * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int k = ty; k < 32; k += 8) {
    const int r = r0 + k, c = c0 + tx;
    if (r < rows && c < cols) {
      // element (r, c) of the (possibly transposed) source
      const float s = trans ? Sb[(int64_t)c * rows + r] : Sb[(int64_t)r * cols + c];
      const uint16_t b = to_bf16(s * sc);
      Xob[(int64_t)r * cols + c] = b;
      tile[k][tx] = b;
    }
  }
  __syncthreads();
  for (int k = ty; k < 32; k += 8) {
    const int c = c0 + k, r = r0 + tx;
    if (r < rows && c < cols) Xtb[(int64_t)c * rows + r] = tile[tx][k];
  }
}

// W <- alpha W + beta X (X bfloat16).
__global__ __launch_bounds__(256) void axpby_bf16_kernel(float *__restrict__ W,
                                                         const uint16_t *__restrict__ X, int64_t n,
                                                         float alpha, float beta) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    W[i] = alpha * W[i] + beta * from_bf16(X[i]);
}

}  // namespace

hipError_t launch_gemm_bf16_nt(const BfGemmDesc &d, hipStream_t s) {
  if (d.M <= 0 || d.N <= 0 || d.batch <= 0) return hipSuccess;
  if (d.K % 8 != 0 || d.ldp % 8 != 0 || d.ldq % 8 != 0 || (d.Ct && d.ldct % 4 != 0))
    return hipErrorInvalidValue;
  BfParams p;
  p.M = (int)d.M; p.N = (int)d.N; p.K = (int)d.K;
  p.P = d.P; p.ldp = d.ldp; p.sP = d.sP;
  p.Q = d.Q; p.ldq = d.ldq; p.sQ = d.sQ;
  p.D = d.D; p.ldd = d.ldd; p.sD = d.sD;
  p.C = d.C; p.ldc = d.ldc; p.sC = d.sC;
  p.Ct = d.Ct; p.ldct = d.ldct; p.sCt = d.sCt;
  p.alpha = d.alpha; p.beta = d.beta;
  p.tiles_m = (p.M + TB - 1) / TB;
  p.tiles_n = (p.N + TB - 1) / TB;
  if (d.syrk) {
    if (p.M != p.N) return hipErrorInvalidValue;
    p.ntiles = p.tiles_m * (p.tiles_m + 1) / 2;
    hipLaunchKernelGGL(gemm_bf16_nt<BMODE_SYRK>, dim3(p.ntiles, 1, (unsigned)d.batch), dim3(NTH),
                       0, s, p);
  } else {
    p.ntiles = p.tiles_m * p.tiles_n;
    hipLaunchKernelGGL(gemm_bf16_nt<BMODE_GENERAL>, dim3(p.ntiles, 1, (unsigned)d.batch),
                       dim3(NTH), 0, s, p);
  }
  return hipGetLastError();
}

hipError_t launch_bf16_scale_both(const float *S, int64_t batch, int64_t rows, int64_t cols,
                                  bool trans, const float *inv, uint16_t *Xo, uint16_t *Xt,
                                  hipStream_t s) {
  if (batch <= 0 || rows <= 0 || cols <= 0) return hipSuccess;
  hipLaunchKernelGGL(bf16_scale_both_kernel,
                     dim3((unsigned)((cols + 31) / 32), (unsigned)((rows + 31) / 32), (unsigned)batch),
                     dim3(256), 0, s, S, (int)rows, (int)cols, trans ? 1 : 0, inv, Xo, Xt);
  return hipGetLastError();
}

hipError_t launch_axpby_bf16(float *W, const uint16_t *X, int64_t count, float alpha, float beta,
                             hipStream_t s) {
  if (count <= 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((count + 255) / 256, 2048);
  hipLaunchKernelGGL(axpby_bf16_kernel, dim3((unsigned)blocks), dim3(256), 0, s, W, X, count, alpha,
                     beta);
  return hipGetLastError();
}

}  // namespace soap
