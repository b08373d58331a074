// Cutoff calibration (Section 4.1, Eq. 3).
//
// 1. The activations the cutoff is a percentile of,
//    a[n, j] = |SiLU(x_n . W_gate[:, j])|, for N calibration vectors: a
//    batched gate product (an N x d by d x m contraction) tiled through LDS,
//    with |SiLU| applied in the epilogue; on the matrix cores for bf16
//    weights (k_calib_acts_mfma), on the vector ALUs for fp32 weights
//    (k_calib_acts).
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

// bf16 weights: the same contraction on the matrix cores.  A block owns
// 256 neurons x 128 calibration vectors; its eight waves own 64 x 64 each,
// 4 x 4 MFMA tiles of 16 x 16 (A: 16 neurons x 32 k of W_gate^T, bf16 as
// stored; B: 32 k x 16 vectors of x as bf16 hi + lo, two products per tile
// and step into one fp32 accumulator).  The reduction runs through LDS 64 k
// at a time; the next stage's global loads are in flight while a stage is
// multiplied.  |SiLU| is applied to each accumulator in the epilogue.
constexpr int kCmM = 256;            // neurons per block (128 x 128 took 0.81 ms at C2, 256 x 128 0.68)
constexpr int kCmN = 128;            // calibration vectors per block
constexpr int kCmK = 64;             // reduction depth per LDS stage
constexpr int kCmPitch = kCmK + 8;   // bf16 per LDS row (16 B pad: rows 4 banks apart)
constexpr int kCmThreads = 512;
constexpr int kCmWLoads = kCmM * kCmK * 2 / (16 * kCmThreads);  // 16-byte W loads per thread and stage
constexpr int kCmXLoads = kCmN * kCmK * 4 / (16 * kCmThreads);  // 16-byte x loads per thread and stage

static_assert(kCmN == 128 && (kCmM / 64) * (kCmN / 64) * kWaveSize == kCmThreads,
              "waves form a (kCmM / 64) x 2 grid of 64 x 64 tiles");

typedef __bf16 cm_bf16x8 __attribute__((ext_vector_type(8)));

__global__ __launch_bounds__(kCmThreads) void k_calib_acts_mfma(const float* __restrict__ X,
                                                               const uint16_t* __restrict__ Wt, int N, int d,
                                                               int m, float* __restrict__ out) {
  __shared__ __attribute__((aligned(16))) uint16_t s_w[kCmM][kCmPitch];
  __shared__ __attribute__((aligned(16))) uint16_t s_xh[kCmN][kCmPitch];
  __shared__ __attribute__((aligned(16))) uint16_t s_xl[kCmN][kCmPitch];
  const int tid = threadIdx.x, lane = tid & (kWaveSize - 1);
  const int w = tid / kWaveSize, wm = w >> 1, wn = w & 1;  // 4 x 2 waves of 64 x 64
  const int r16 = lane & 15, kb = lane >> 4;
  const int j0 = blockIdx.x * kCmM, v0 = blockIdx.y * kCmN;
  const int rows_w = min(kCmM, m - j0), rows_x = min(kCmN, N - v0);
  // per-block resources: at most 256 rows of W (<= 4 MB) and 128 of x (<= 4 MB)
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(Wt + (size_t)j0 * d, (uint32_t)(rows_w * d * 2));
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(X + (size_t)v0 * d, (uint32_t)(rows_x * d * 4));

  // loader coordinates: W, eight 16-byte pieces per 64-k row; x, sixteen
  // float4 per 64-k row
  auto w_off = [&](int q, int k0) -> uint32_t {
    const int row = q * (kCmThreads / 8) + (tid >> 3), k = k0 + 8 * (tid & 7);
    return (row < rows_w && k < d) ? (uint32_t)(row * d + k) * 2u : kOOB;
  };
  auto x_off = [&](int q, int k0) -> uint32_t {
    const int row = q * (kCmThreads / 16) + (tid >> 4), k = k0 + 4 * (tid & 15);
    return (row < rows_x && k < d) ? (uint32_t)(row * d + k) * 4u : kOOB;
  };
  u32x4 pw[kCmWLoads], px[kCmXLoads];
  auto fetch = [&](int k0) {
#pragma unroll
    for (int q = 0; q < kCmWLoads; ++q) pw[q] = ld_buf16(rw, w_off(q, k0));
#pragma unroll
    for (int q = 0; q < kCmXLoads; ++q) px[q] = ld_buf16(rx, x_off(q, k0));
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  fetch(0);
  for (int k0 = 0; k0 < d; k0 += kCmK) {
    __syncthreads();  // the previous stage's operand reads are done
#pragma unroll
    for (int q = 0; q < kCmWLoads; ++q)
      *reinterpret_cast<u32x4*>(&s_w[q * (kCmThreads / 8) + (tid >> 3)][8 * (tid & 7)]) = pw[q];
#pragma unroll
    for (int q = 0; q < kCmXLoads; ++q) {
      uint32_t h[4], l[4];
      const uint32_t f[4] = {px[q].x, px[q].y, px[q].z, px[q].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        h[e] = bf16_bits(__uint_as_float(f[e]));
        l[e] = bf16_bits(__uint_as_float(f[e]) - __uint_as_float(h[e] << 16));
      }
      const int row = q * (kCmThreads / 16) + (tid >> 4), c = 4 * (tid & 15);
      *reinterpret_cast<uint2*>(&s_xh[row][c]) = uint2{h[0] | (h[1] << 16), h[2] | (h[3] << 16)};
      *reinterpret_cast<uint2*>(&s_xl[row][c]) = uint2{l[0] | (l[1] << 16), l[2] | (l[3] << 16)};
    }
    __syncthreads();
    if (k0 + kCmK < d) fetch(k0 + kCmK);
#pragma unroll
    for (int ks = 0; ks < kCmK / 32; ++ks) {
      const int kc = 32 * ks + 8 * kb;
      cm_bf16x8 av[4], bh[4], bl[4];
#pragma unroll
      for (int a = 0; a < 4; ++a)
        av[a] = *reinterpret_cast<const cm_bf16x8*>(&s_w[64 * wm + 16 * a + r16][kc]);
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        bh[b] = *reinterpret_cast<const cm_bf16x8*>(&s_xh[64 * wn + 16 * b + r16][kc]);
        bl[b] = *reinterpret_cast<const cm_bf16x8*>(&s_xl[64 * wn + 16 * b + r16][kc]);
      }
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[a], bh[b], acc[a][b], 0, 0, 0);
          acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[a], bl[b], acc[a][b], 0, 0, 0);
        }
    }
  }

  // D[i][j] sits in lane j + 16 (i / 4), register i % 4: neuron i, vector j
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const int v = v0 + 64 * wn + 16 * b + r16;
    if (v >= N) continue;
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      const int j = j0 + 64 * wm + 16 * a + 4 * kb;
      const float r[4] = {acc[a][b].x, acc[a][b].y, acc[a][b].z, acc[a][b].w};
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (j + e < m) out[(size_t)v * m + j + e] = fabsf(silu(r[e]));
    }
  }
}

hipError_t launch_calib_acts(int wdtype_bf16, const float* x, const void* wg_t, int N, int d,
                             int m, float* acts, hipStream_t s) {
  KernelTimer timer("calib_acts", s);
  if (wdtype_bf16) {
    const dim3 grid((m + kCmM - 1) / kCmM, (N + kCmN - 1) / kCmN);
    hipExtLaunchKernelGGL(k_calib_acts_mfma, grid, dim3(kCmThreads), 0, s, timer.start(), timer.stop(), 0, x,
                          static_cast<const uint16_t*>(wg_t), N, d, m, acts);
  } else {
    const dim3 grid((m + kCalibTN - 1) / kCalibTN, (N + kCalibTM - 1) / kCalibTM);
    hipExtLaunchKernelGGL(k_calib_acts<wf32>, grid, dim3(256), 0, s, timer.start(), timer.stop(), 0,
                          x, static_cast<const float*>(wg_t), N, d, m, acts);
  }
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
