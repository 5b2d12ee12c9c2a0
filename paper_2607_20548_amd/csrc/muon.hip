// Streaming kernels of the Muon step (Algorithm 1): the Frobenius norm of
// the momentum, the normalisation X_0 = M / max(||M||_F, eps) and the final
// weight update W <- (1 - lr wd) W - lr sqrt(max(in, out)) X_n.  The Newton-
// Schulz products themselves are GEMMs.  All are HBM-bound.
#include "internal.h"

namespace soap {
namespace {

constexpr int NR_THREADS = 256;
constexpr int NR_BLOCKS = 1024;  // partial sums per matrix (fixed: the order is fixed)

// Sum of squares of each matrix's `count` floats: block j of matrix b covers
// a fixed contiguous range (a multiple of 4 floats, read as float4 when the
// matrix is 16-byte aligned), accumulates in double, and reduces in a fixed
// tree; norm_finish adds the NR_BLOCKS partials in index order.
__global__ __launch_bounds__(NR_THREADS) void norm_partial(const float *__restrict__ X,
                                                          int64_t count, double *__restrict__ part) {
  __shared__ double red[NR_THREADS];
  const int64_t b = blockIdx.y;
  const float *Xb = X + b * count;
  const int64_t per = 4 * ((count + 4 * NR_BLOCKS - 1) / (4 * NR_BLOCKS));
  const int64_t beg = blockIdx.x * per, end = min(count, beg + per);
  double acc = 0.0;
  if ((reinterpret_cast<uintptr_t>(Xb) & 15u) == 0 && end - beg == per) {
    const float4 *X4 = reinterpret_cast<const float4 *>(Xb + beg);
    for (int64_t i = threadIdx.x; i < per / 4; i += NR_THREADS) {
      const float4 v = X4[i];
      acc += (double)v.x * v.x + (double)v.y * v.y + (double)v.z * v.z + (double)v.w * v.w;
    }
  } else {
    for (int64_t i = beg + threadIdx.x; i < end; i += NR_THREADS) {
      const double v = Xb[i];
      acc += v * v;
    }
  }
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int s = NR_THREADS / 2; s > 0; s >>= 1) {
    if (threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) part[b * NR_BLOCKS + blockIdx.x] = red[0];
}

// inv[b] = 1 / max(sqrt(sum of squares), eps)
__global__ __launch_bounds__(64) void norm_finish(const double *__restrict__ part, int64_t batch,
                                                  float eps, float *__restrict__ inv) {
  const int64_t b = (int64_t)blockIdx.x * 64 + threadIdx.x;
  if (b >= batch) return;
  double s = 0.0;
  for (int j = 0; j < NR_BLOCKS; ++j) s += part[b * NR_BLOCKS + j];
  const double nrm = sqrt(s);
  inv[b] = (float)(1.0 / (nrm > (double)eps ? nrm : (double)eps));
}

__global__ __launch_bounds__(256) void scale_by_inv(const float *__restrict__ M,
                                                    float *__restrict__ X,
                                                    const float *__restrict__ inv, int64_t count) {
  const int64_t b = blockIdx.y;
  const float r = inv[b];
  const float *Mb = M + b * count;
  float *Xb = X + b * count;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count;
       i += (int64_t)gridDim.x * 256)
    Xb[i] = Mb[i] * r;
}

__global__ __launch_bounds__(256) void axpby_kernel(float *__restrict__ W,
                                                    const float *__restrict__ X, int64_t n,
                                                    float alpha, float beta) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * 256)
    W[i] = alpha * W[i] + beta * X[i];
}

unsigned grid_for(int64_t items, int64_t batch) {
  int64_t bx = (items + 255) / 256;
  const int64_t cap = std::max<int64_t>(1, 2048 / batch);
  if (bx > cap) bx = cap;
  return (unsigned)bx;
}

}  // namespace

size_t muon_norm_partial_bytes(int64_t batch) { return sizeof(double) * NR_BLOCKS * batch; }

hipError_t launch_muon_normalise(const float *M, float *X, int64_t batch, int64_t count,
                                 float eps, double *part, float *inv, hipStream_t s) {
  if (batch <= 0 || count <= 0) return hipSuccess;
  hipLaunchKernelGGL(norm_partial, dim3(NR_BLOCKS, (unsigned)batch), dim3(NR_THREADS), 0, s, M,
                     count, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(norm_finish, dim3((unsigned)((batch + 63) / 64)), dim3(64), 0, s, part,
                     batch, eps, inv);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(scale_by_inv, dim3(grid_for(count, batch), (unsigned)batch), dim3(256), 0, s,
                     M, X, inv, count);
  return hipGetLastError();
}

hipError_t launch_muon_norm_inv(const float *M, int64_t batch, int64_t count, float eps,
                                double *part, float *inv, hipStream_t s) {
  if (batch <= 0 || count <= 0) return hipSuccess;
  hipLaunchKernelGGL(norm_partial, dim3(NR_BLOCKS, (unsigned)batch), dim3(NR_THREADS), 0, s, M,
                     count, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(norm_finish, dim3((unsigned)((batch + 63) / 64)), dim3(64), 0, s, part,
                     batch, eps, inv);
  return hipGetLastError();
}

hipError_t launch_axpby(float *W, const float *X, int64_t count, float alpha, float beta,
                        hipStream_t s) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(axpby_kernel, dim3(grid_for(count, 1)), dim3(256), 0, s, W, X, count, alpha,
                     beta);
  return hipGetLastError();
}

}  // namespace soap
