// RMSNorm (the normalisation in front of each MLP block of a decoder stack)
// and the weight transpose that produces the neuron-major layout.
#include "device.hpp"
#include "internal.hpp"

namespace cats {

// One block per row: sum of squares with a fixed-order tree, then scale.
__global__ __launch_bounds__(256) void k_rmsnorm(const float* __restrict__ x, float* __restrict__ xn,
                                                 int d, float eps) {
  __shared__ float red[256];
  const int t = threadIdx.x;
  const float* xr = x + (size_t)blockIdx.x * d;
  float* outr = xn + (size_t)blockIdx.x * d;
  float ss = 0.f;
  for (int i = t; i < d; i += 256) ss = fmaf(xr[i], xr[i], ss);
  red[t] = ss;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (t < o) red[t] += red[t + o];
    __syncthreads();
  }
  const float inv = 1.0f / sqrtf(red[0] / (float)d + eps);
  for (int i = t; i < d; i += 256) outr[i] = xr[i] * inv;
}

hipError_t launch_rmsnorm(const float* x, float* xn, int B, int d, float eps, hipStream_t s) {
  KernelTimer timer("rmsnorm", s);
  hipExtLaunchKernelGGL(k_rmsnorm, dim3(B), dim3(256), 0, s, timer.start(), timer.stop(), 0, x, xn, d,
                        eps);
  return hipGetLastError();
}

// out[c * rows + r] = in[r * cols + c] through a padded 32 x 32 LDS tile.
template <typename E>
__global__ __launch_bounds__(256) void k_transpose(const E* __restrict__ in, E* __restrict__ out,
                                                   int rows, int cols) {
  __shared__ E tile[32][33];
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  const int c0 = blockIdx.x * 32, r0 = blockIdx.y * 32;
  for (int k = ty; k < 32; k += 8) {
    const int r = r0 + k, c = c0 + tx;
    if (r < rows && c < cols) tile[k][tx] = in[(size_t)r * cols + c];
  }
  __syncthreads();
  for (int k = ty; k < 32; k += 8) {
    const int c = c0 + k, r = r0 + tx;
    if (c < cols && r < rows) out[(size_t)c * rows + r] = tile[tx][k];
  }
}

hipError_t launch_transpose(const void* in, void* out, int rows, int cols, int elem_bytes,
                            hipStream_t s) {
  const dim3 grid((cols + 31) / 32, (rows + 31) / 32);
  KernelTimer timer("transpose", s);
  if (elem_bytes == 2)
    hipExtLaunchKernelGGL(k_transpose<uint16_t>, grid, dim3(256), 0, s, timer.start(), timer.stop(), 0,
                          static_cast<const uint16_t*>(in), static_cast<uint16_t*>(out), rows, cols);
  else
    hipExtLaunchKernelGGL(k_transpose<uint32_t>, grid, dim3(256), 0, s, timer.start(), timer.stop(), 0,
                          static_cast<const uint32_t*>(in), static_cast<uint32_t*>(out), rows, cols);
  return hipGetLastError();
}

}  // namespace cats
