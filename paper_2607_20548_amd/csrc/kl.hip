// Kernels of the KL-Shampoo factor accumulation (Algorithm 2, KL-SOAP):
//   * the eigenvalue estimates lambda = diag(Q^T F Q) of a factor in the
//     previous step's basis, read off the product X = Q^T F that the power
//     product kernel already forms: lambda[k] = sum_i X[k][i] Q[i][k];
//   * the inverse-eigenvalue scaling Z = Y diag(1/(lambda+eps)) (columns) or
//     Z = diag(1/(lambda+eps)) Y (rows) of the projected gradient.
// Both are HBM-bound streams next to the products around them.
#include "internal.h"

namespace soap {
namespace {

constexpr int DG_TILE = 64;     // k and i extent of one tile
constexpr int DG_THREADS = 256;
constexpr int DG_TARGET_BLOCKS = 2048;

// One workgroup owns 64 consecutive k and a chunk of i.  Each 64 x 64 tile of
// X (rows k, columns i) and of Q (rows i, columns k) is read with coalesced
// row loads into LDS; a thread then sums X[k][i] Q[i][k] over 16 of the
// tile's i.  The partial of every (chunk, k) is stored and summed in chunk
// order by diag_finish_kernel, so the result does not depend on timing.
__global__ __launch_bounds__(DG_THREADS) void diag_partial_kernel(
    const float *__restrict__ X, const float *__restrict__ Q, int64_t d, int64_t sbatch,
    int64_t rows_per_chunk, float *__restrict__ part) {
  __shared__ float xs[DG_TILE][DG_TILE + 1];
  __shared__ float qs[DG_TILE][DG_TILE + 1];
  __shared__ float red[4][DG_TILE];
  const int64_t b = blockIdx.z;
  const float *Xb = X + b * sbatch;
  const float *Qb = Q + b * sbatch;
  const int64_t k0 = (int64_t)blockIdx.x * DG_TILE;
  const int64_t ibeg = (int64_t)blockIdx.y * rows_per_chunk;
  const int64_t iend = min(d, ibeg + rows_per_chunk);
  const int t = threadIdx.x;
  const int col = t & 63, r4 = t >> 6;
  const int kk = t & 63, q = t >> 6;
  float acc = 0.f;
  for (int64_t i0 = ibeg; i0 < iend; i0 += DG_TILE) {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int r = 4 * e + r4;
      const int64_t xr = k0 + r, xc = i0 + col;   // X[k][i]
      xs[r][col] = (xr < d && xc < iend) ? Xb[xr * d + xc] : 0.f;
      const int64_t qr = i0 + r, qc = k0 + col;   // Q[i][k]
      qs[r][col] = (qr < iend && qc < d) ? Qb[qr * d + qc] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int i = 16 * q + e;
      acc += xs[kk][i] * qs[i][kk];
    }
    __syncthreads();
  }
  red[q][kk] = acc;
  __syncthreads();
  if (t < DG_TILE && k0 + t < d) {
    const float s = ((red[0][t] + red[1][t]) + red[2][t]) + red[3][t];
    part[(b * gridDim.y + blockIdx.y) * d + k0 + t] = s;
  }
}

__global__ __launch_bounds__(256) void diag_finish_kernel(const float *__restrict__ part,
                                                          int nchunk, int64_t d,
                                                          float *__restrict__ lam) {
  const int64_t b = blockIdx.y;
  const int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (k >= d) return;
  const float *p = part + b * nchunk * d + k;
  float s = 0.f;
  for (int c = 0; c < nchunk; ++c) s += p[(int64_t)c * d];
  lam[b * d + k] = s;
}

// Z = Y scaled by 1/(lambda + eps): by column index (by_row = 0, lambda has
// `cols` entries per matrix) or by row index (by_row = 1, `rows` entries).
__global__ __launch_bounds__(256) void kl_scale_vec4(const float4 *__restrict__ Y,
                                                     float4 *__restrict__ Z,
                                                     const float *__restrict__ lam,
                                                     int64_t rows, int64_t cols, int by_row,
                                                     float eps) {
  const int64_t b = blockIdx.y;
  const int64_t n4 = rows * cols / 4;
  const float4 *Yb = Y + b * n4;
  float4 *Zb = Z + b * n4;
  const float *lb = lam + b * (by_row ? rows : cols);
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4;
       i += (int64_t)gridDim.x * 256) {
    const int64_t e = 4 * i;
    const int64_t row = e / cols, c0 = e - row * cols;
    float4 y = Yb[i];
    if (by_row) {
      const float r = 1.f / (lb[row] + eps);
      y.x *= r; y.y *= r; y.z *= r; y.w *= r;
    } else {
      y.x *= 1.f / (lb[c0] + eps);
      y.y *= 1.f / (lb[c0 + 1] + eps);
      y.z *= 1.f / (lb[c0 + 2] + eps);
      y.w *= 1.f / (lb[c0 + 3] + eps);
    }
    Zb[i] = y;
  }
}

__global__ __launch_bounds__(256) void kl_scale_scalar(const float *__restrict__ Y,
                                                       float *__restrict__ Z,
                                                       const float *__restrict__ lam,
                                                       int64_t rows, int64_t cols, int by_row,
                                                       float eps) {
  const int64_t b = blockIdx.y;
  const int64_t n = rows * cols;
  const float *Yb = Y + b * n;
  float *Zb = Z + b * n;
  const float *lb = lam + b * (by_row ? rows : cols);
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < n;
       e += (int64_t)gridDim.x * 256) {
    const int64_t row = e / cols, c = e - row * cols;
    Zb[e] = Yb[e] * (1.f / (lb[by_row ? row : c] + eps));
  }
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

int diag_chunks(int64_t batch, int64_t d) {
  const int64_t kb = (d + DG_TILE - 1) / DG_TILE;
  int64_t c = (DG_TARGET_BLOCKS + kb * batch - 1) / (kb * batch);
  if (c > kb) c = kb;
  if (c < 1) c = 1;
  return (int)c;
}

size_t diag_partial_floats(int64_t batch, int64_t d) {
  return (size_t)diag_chunks(batch, d) * (size_t)batch * (size_t)d;
}

hipError_t launch_diag_of_product(const float *X, const float *Q, int64_t batch, int64_t d,
                                  float *part, float *lam, hipStream_t s) {
  if (batch <= 0 || d <= 0) return hipSuccess;
  const int nchunk = diag_chunks(batch, d);
  const int64_t tiles = (d + DG_TILE - 1) / DG_TILE;
  const int64_t rows_per_chunk = ((tiles + nchunk - 1) / nchunk) * DG_TILE;
  const int used = (int)((d + rows_per_chunk - 1) / rows_per_chunk);  // chunks with rows
  hipLaunchKernelGGL(diag_partial_kernel, dim3((unsigned)tiles, (unsigned)used, (unsigned)batch),
                     dim3(DG_THREADS), 0, s, X, Q, d, d * d, rows_per_chunk, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(diag_finish_kernel, dim3((unsigned)((d + 255) / 256), (unsigned)batch),
                     dim3(256), 0, s, part, used, d, lam);
  return hipGetLastError();
}

hipError_t launch_kl_scale(const float *Y, float *Z, const float *lam, int64_t batch,
                           int64_t rows, int64_t cols, int by_row, float eps, hipStream_t s) {
  if (batch <= 0 || rows <= 0 || cols <= 0) return hipSuccess;
  const int64_t n = rows * cols;
  const bool vec = cols % 4 == 0 && aligned16(Y) && aligned16(Z);
  const int64_t items = vec ? n / 4 : n;
  int64_t bx = (items + 255) / 256;
  const int64_t cap = std::max<int64_t>(1, 2048 / batch);
  if (bx > cap) bx = cap;
  if (vec)
    hipLaunchKernelGGL(kl_scale_vec4, dim3((unsigned)bx, (unsigned)batch), dim3(256), 0, s,
                       reinterpret_cast<const float4 *>(Y), reinterpret_cast<float4 *>(Z), lam,
                       rows, cols, by_row, eps);
  else
    hipLaunchKernelGGL(kl_scale_scalar, dim3((unsigned)bx, (unsigned)batch), dim3(256), 0, s, Y,
                       Z, lam, rows, cols, by_row, eps);
  return hipGetLastError();
}

}  // namespace soap
