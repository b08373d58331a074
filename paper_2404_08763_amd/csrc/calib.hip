// Cutoff calibration (Section 4.1, Eq. 3).
//
// 1. k_calib_acts: the activations the cutoff is a percentile of,
//    a[n, j] = |SiLU(x_n . W_gate[:, j])|, for N calibration vectors: a
//    batched gate product (an N x d by d x m contraction) tiled through LDS,
//    with |SiLU| applied in the epilogue.
// 2. Radix select: t = the r-th smallest |a|, which is
//    min{t' : F(t') >= k} for the empirical CDF F when r = ceil(k n).
//    Non-negative fp32 values order like their bit patterns read as
//    unsigned integers, so four passes over 8-bit digits (most significant
//    first) narrow the candidate set to the exact value.  Each pass builds a
//    256-bin histogram of the digit among keys matching the prefix found so
//    far (LDS counters, then integer atomics into one global histogram:
//    order-independent and exact), and a one-block kernel picks the bin
//    holding rank r.
#include "device.hpp"
#include "internal.hpp"

namespace cats {

constexpr int kCalibTM = 64;  // calibration vectors per tile
constexpr int kCalibTN = 64;  // neurons per tile
constexpr int kCalibTK = 16;  // reduction depth per LDS stage

template <typename WT>
__device__ __forceinline__ void load4_widen(const typename wtraits<WT>::elem* p, float* f);

template <>
__device__ __forceinline__ void load4_widen<wbf16>(const uint16_t* p, float* f) {
  const uint2 v = *reinterpret_cast<const uint2*>(p);
  f[0] = __uint_as_float(v.x << 16);
  f[1] = __uint_as_float(v.x & 0xffff0000u);
  f[2] = __uint_as_float(v.y << 16);
  f[3] = __uint_as_float(v.y & 0xffff0000u);
}

template <>
__device__ __forceinline__ void load4_widen<wf32>(const float* p, float* f) {
  const f32x4 v = *reinterpret_cast<const f32x4*>(p);
  f[0] = v.x;
  f[1] = v.y;
  f[2] = v.z;
  f[3] = v.w;
}

template <typename WT>
__global__ __launch_bounds__(256) void k_calib_acts(const float* __restrict__ X,
                                                    const typename wtraits<WT>::elem* __restrict__ Wt,
                                                    int N, int d, int m, float* __restrict__ out) {
  __shared__ __attribute__((aligned(16))) float Xs[kCalibTK][kCalibTM + 4];
  __shared__ __attribute__((aligned(16))) float Ws[kCalibTK][kCalibTN + 4];
  const int tid = threadIdx.x;
  const int tr = tid >> 4, tc = tid & 15;            // 4x4 outputs per thread
  const int lrow = tid >> 2, lk = (tid & 3) * 4;     // loader: 4 consecutive k of one row
  const int n0 = blockIdx.y * kCalibTM, j0 = blockIdx.x * kCalibTN;
  float acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int k = 0; k < 4; ++k) acc[i][k] = 0.f;

  for (int k0 = 0; k0 < d; k0 += kCalibTK) {
    {
      const int n = n0 + lrow, k = k0 + lk;
      f32x4 v = {0.f, 0.f, 0.f, 0.f};
      if (n < N && k < d) v = *reinterpret_cast<const f32x4*>(X + (size_t)n * d + k);
      Xs[lk + 0][lrow] = v.x;
      Xs[lk + 1][lrow] = v.y;
      Xs[lk + 2][lrow] = v.z;
      Xs[lk + 3][lrow] = v.w;
    }
    {
      const int j = j0 + lrow, k = k0 + lk;
      float f[4] = {0.f, 0.f, 0.f, 0.f};
      if (j < m && k < d) load4_widen<WT>(Wt + (size_t)j * d + k, f);
#pragma unroll
      for (int e = 0; e < 4; ++e) Ws[lk + e][lrow] = f[e];
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kCalibTK; ++kk) {
      const f32x4 av = *reinterpret_cast<const f32x4*>(&Xs[kk][tr * 4]);
      const f32x4 bv = *reinterpret_cast<const f32x4*>(&Ws[kk][tc * 4]);
      const float ar[4] = {av.x, av.y, av.z, av.w};
      const float br[4] = {bv.x, bv.y, bv.z, bv.w};
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int k = 0; k < 4; ++k) acc[i][k] = fmaf(ar[i], br[k], acc[i][k]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int n = n0 + tr * 4 + i;
    if (n >= N) continue;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int j = j0 + tc * 4 + k;
      if (j < m) out[(size_t)n * m + j] = fabsf(silu(acc[i][k]));
    }
  }
}

hipError_t launch_calib_acts(int wdtype_bf16, const float* x, const void* wg_t, int N, int d,
                             int m, float* acts, hipStream_t s) {
  const dim3 grid((m + kCalibTN - 1) / kCalibTN, (N + kCalibTM - 1) / kCalibTM);
  KernelTimer timer("calib_acts", s);
  if (wdtype_bf16)
    hipExtLaunchKernelGGL(k_calib_acts<wbf16>, grid, dim3(256), 0, s, timer.start(), timer.stop(), 0,
                          x, static_cast<const uint16_t*>(wg_t), N, d, m, acts);
  else
    hipExtLaunchKernelGGL(k_calib_acts<wf32>, grid, dim3(256), 0, s, timer.start(), timer.stop(), 0,
                          x, static_cast<const float*>(wg_t), N, d, m, acts);
  return hipGetLastError();
}

// scratch layout: [0, 256) histogram, [256] selected prefix, [257..258]
// remaining rank (low, high word).
constexpr int kRadixPrefix = 256;
constexpr int kRadixRankLo = 257;
constexpr int kRadixRankHi = 258;

__global__ __launch_bounds__(256) void k_radix_init(uint32_t* sc, uint64_t r) {
  const int t = threadIdx.x;
  sc[t] = 0u;
  if (t == 0) {
    sc[kRadixPrefix] = 0u;
    sc[kRadixRankLo] = (uint32_t)r;
    sc[kRadixRankHi] = (uint32_t)(r >> 32);
  }
}

__global__ __launch_bounds__(256) void k_radix_hist(const float* __restrict__ a, int64_t n,
                                                    uint32_t* __restrict__ sc, int pass) {
  __shared__ uint32_t lh[256];
  lh[threadIdx.x] = 0u;
  __syncthreads();
  const int shift = 24 - 8 * pass;
  const uint32_t prefix = sc[kRadixPrefix];
  const uint32_t himask = pass == 0 ? 0u : (0xffffffffu << (32 - 8 * pass));
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const uint32_t key = __float_as_uint(a[i]) & 0x7fffffffu;  // bits of |a|
    if ((key & himask) == prefix) atomicAdd(&lh[(key >> shift) & 0xffu], 1u);
  }
  __syncthreads();
  const uint32_t c = lh[threadIdx.x];
  if (c) atomicAdd(&sc[threadIdx.x], c);
}

__global__ __launch_bounds__(256) void k_radix_pick(uint32_t* sc, int pass) {
  __shared__ uint64_t cum[256];
  const int t = threadIdx.x;
  const uint64_t r = (uint64_t)sc[kRadixRankLo] | ((uint64_t)sc[kRadixRankHi] << 32);
  const uint32_t c = sc[t];
  cum[t] = c;
  __syncthreads();
  for (int o = 1; o < 256; o <<= 1) {  // inclusive scan of the bin counts
    const uint64_t v = t >= o ? cum[t - o] : 0ull;
    __syncthreads();
    cum[t] += v;
    __syncthreads();
  }
  const uint64_t before = cum[t] - c;
  if (before < r && r <= cum[t]) {  // exactly one bin holds rank r
    sc[kRadixPrefix] |= (uint32_t)t << (24 - 8 * pass);
    const uint64_t nr = r - before;
    sc[kRadixRankLo] = (uint32_t)nr;
    sc[kRadixRankHi] = (uint32_t)(nr >> 32);
  }
  sc[t] = 0u;  // histogram cleared for the next pass
}

hipError_t launch_radix_select(const float* a, int64_t n, int64_t r, uint32_t* scratch,
                               hipStream_t s) {
  int64_t blocks = (n + 256 * 16 - 1) / (256 * 16);
  if (blocks > 2048) blocks = 2048;
  if (blocks < 1) blocks = 1;
  {
    KernelTimer timer("radix_init", s);
    hipExtLaunchKernelGGL(k_radix_init, dim3(1), dim3(256), 0, s, timer.start(), timer.stop(), 0,
                          scratch, (uint64_t)r);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  for (int pass = 0; pass < 4; ++pass) {
    {
      KernelTimer timer("radix_hist", s);
      hipExtLaunchKernelGGL(k_radix_hist, dim3((unsigned)blocks), dim3(256), 0, s, timer.start(),
                            timer.stop(), 0, a, n, scratch, pass);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    {
      KernelTimer timer("radix_pick", s);
      hipExtLaunchKernelGGL(k_radix_pick, dim3(1), dim3(256), 0, s, timer.start(), timer.stop(), 0,
                            scratch, pass);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace cats
