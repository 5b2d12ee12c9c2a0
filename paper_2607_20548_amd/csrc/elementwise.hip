// Streaming kernels of the SOAP step: the weight-space first-moment EMA and the
// fills used to initialise state.  They are HBM-bound; each thread handles
// 16-byte vectors when the pointers allow it, and the grid is capped at a few
// workgroups per CU with a grid-stride loop.
#include "internal.h"

namespace soap {
namespace {

constexpr int EW_THREADS = 256;

unsigned ew_blocks(int64_t work_items) {
  int64_t b = (work_items + EW_THREADS - 1) / EW_THREADS;
  const int64_t cap = 256 * 8;  // 256 CUs, 8 workgroups each
  if (b > cap) b = cap;
  if (b < 1) b = 1;
  return (unsigned)b;
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

__global__ __launch_bounds__(EW_THREADS) void momentum_vec4(float4 *__restrict__ M,
                                                            const float4 *__restrict__ G,
                                                            int64_t n4, float b1) {
  const float a = 1.f - b1;
  for (int64_t i = blockIdx.x * (int64_t)EW_THREADS + threadIdx.x; i < n4;
       i += (int64_t)gridDim.x * EW_THREADS) {
    float4 m = M[i];
    const float4 g = G[i];
    m.x = b1 * m.x + a * g.x;
    m.y = b1 * m.y + a * g.y;
    m.z = b1 * m.z + a * g.z;
    m.w = b1 * m.w + a * g.w;
    M[i] = m;
  }
}

__global__ __launch_bounds__(EW_THREADS) void momentum_scalar(float *__restrict__ M,
                                                              const float *__restrict__ G,
                                                              int64_t n, float b1) {
  const float a = 1.f - b1;
  for (int64_t i = blockIdx.x * (int64_t)EW_THREADS + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * EW_THREADS)
    M[i] = b1 * M[i] + a * G[i];
}

__global__ __launch_bounds__(EW_THREADS) void fill_diag_kernel(float *X, int64_t r, int64_t c,
                                                               int64_t sbatch, float dv) {
  float *Xb = X + blockIdx.y * sbatch;
  const int64_t total = r * c;
  for (int64_t i = blockIdx.x * (int64_t)EW_THREADS + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * EW_THREADS) {
    const int64_t row = i / c, col = i - row * c;
    Xb[i] = (row == col) ? dv : 0.f;
  }
}

__global__ __launch_bounds__(EW_THREADS) void zero_u32_kernel(uint32_t *p, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)EW_THREADS + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * EW_THREADS)
    p[i] = 0u;
}

__global__ __launch_bounds__(EW_THREADS) void copy_kernel(float *__restrict__ d,
                                                          const float *__restrict__ s,
                                                          int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)EW_THREADS + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * EW_THREADS)
    d[i] = s[i];
}

}  // namespace

hipError_t launch_momentum(float *M, const float *G, int64_t count, float b1, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  if (count % 4 == 0 && aligned16(M) && aligned16(G)) {
    const int64_t n4 = count / 4;
    hipLaunchKernelGGL(momentum_vec4, dim3(ew_blocks(n4)), dim3(EW_THREADS), 0, s,
                       reinterpret_cast<float4 *>(M), reinterpret_cast<const float4 *>(G), n4, b1);
  } else {
    hipLaunchKernelGGL(momentum_scalar, dim3(ew_blocks(count)), dim3(EW_THREADS), 0, s, M, G,
                       count, b1);
  }
  return hipGetLastError();
}

hipError_t launch_fill_diag(float *X, int64_t batch, int64_t r, int64_t c, int64_t sbatch,
                            float diag_value, hipStream_t s) {
  if (batch <= 0 || r <= 0 || c <= 0) return hipSuccess;
  unsigned bx = ew_blocks(r * c);
  if (bx * batch > 65536 && bx > 1) bx = (unsigned)std::max<int64_t>(1, 65536 / batch);
  hipLaunchKernelGGL(fill_diag_kernel, dim3(bx, (unsigned)batch), dim3(EW_THREADS), 0, s, X, r,
                     c, sbatch, diag_value);
  return hipGetLastError();
}

hipError_t launch_zero_u32(uint32_t *p, int64_t count, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(zero_u32_kernel, dim3(ew_blocks(count)), dim3(EW_THREADS), 0, s, p, count);
  return hipGetLastError();
}

hipError_t launch_copy(float *dst, const float *src, int64_t count, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(copy_kernel, dim3(ew_blocks(count)), dim3(EW_THREADS), 0, s, dst, src,
                     count);
  return hipGetLastError();
}

}  // namespace soap
