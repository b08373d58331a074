// Per-token top-k variant of CATS (future work in the appendix comparing
// target and actual sparsity: the target enforced at inference for every
// token instead of one calibrated t).  Row b keeps the neurons with
// |v_bj| >= t_b, t_b = the r-th smallest of its own m values |v_b.| (Eq. 3
// over one token), so every row keeps at least m - r + 1 neurons.
//
// k_gate_v (gate_v.hip): the gate activations v = SiLU(x W_gate) of up to
// 8 rows in one pass over W_gate.
// k_row_select: one block per row, the exact r-th smallest |v| by three
// radix passes over the fp32 bit patterns (LDS histogram, keys in registers).
// The fused kernel then runs with v and t_b given (VIN): no W_gate row is
// read a second time.
#include "device.hpp"
#include "internal.hpp"

namespace cats {

// One block per row: t[b] = the r-th smallest |v[b, :]| (1-indexed), exact.
// Non-negative fp32 values order like their bit patterns (bit 31 is 0), so
// the pattern is fixed digit by digit, most significant first: bits 30..20,
// 19..10, 9..0.  Each pass histograms the digit over the keys that match the
// digits fixed so far; the bin holding the remaining rank becomes the next
// digit.  The row's keys stay in registers across the passes (KPT per
// thread; padding keys have bit 31 set and never match), and one wave finds
// the bin by a prefix sum over its lanes.  r = 0 gives t = 0.
constexpr int kSelThreads = 1024;

template <int SHIFT, int BITS, int KPT>
__device__ __forceinline__ void select_pass(const uint32_t (&key)[KPT], uint32_t* hist, uint32_t& prefix,
                                            uint32_t& hi_mask, int& rem, uint32_t* s_state) {
  constexpr int NB = 1 << BITS;
  constexpr int BPL = NB / kWaveSize;  // bins per lane in the scan
  const int tid = threadIdx.x;
  for (int q = tid; q < NB; q += kSelThreads) hist[q] = 0u;
  __syncthreads();
#pragma unroll
  for (int k = 0; k < KPT; ++k)
    if ((key[k] & hi_mask) == prefix) atomicAdd(&hist[(key[k] >> SHIFT) & (NB - 1)], 1u);
  __syncthreads();
  if (tid < kWaveSize) {
    uint32_t h[BPL];
    uint32_t sum = 0;
#pragma unroll
    for (int q = 0; q < BPL; q += 4) {
      const uint4 v = *reinterpret_cast<const uint4*>(hist + tid * BPL + q);
      h[q] = v.x;
      h[q + 1] = v.y;
      h[q + 2] = v.z;
      h[q + 3] = v.w;
      sum += v.x + v.y + v.z + v.w;
    }
    uint32_t incl = sum;
#pragma unroll
    for (int o = 1; o < kWaveSize; o <<= 1) {
      const uint32_t u = (uint32_t)__shfl_up((int)incl, o);
      if (tid >= o) incl += u;
    }
    // lowest lane whose running count reaches the rank (one exists: the
    // matching keys number at least rem)
    const uint64_t hit = __ballot(incl >= (uint32_t)rem);
    const int lane = hit ? __builtin_ctzll(hit) : kWaveSize - 1;
    if (tid == lane) {
      uint32_t cum = incl - sum;
      int bin = BPL - 1;
#pragma unroll
      for (int q = 0; q < BPL; ++q) {
        if (cum + h[q] >= (uint32_t)rem) {
          bin = q;
          break;
        }
        cum += h[q];
      }
      s_state[0] = prefix | ((uint32_t)(lane * BPL + bin) << SHIFT);
      s_state[1] = (uint32_t)rem - cum;
    }
  }
  __syncthreads();
  prefix = s_state[0];
  rem = (int)s_state[1];
  hi_mask |= (uint32_t)(NB - 1) << SHIFT;
}

template <int KPT>
__global__ __launch_bounds__(kSelThreads) void k_row_select(const float* __restrict__ v, int m, int r,
                                                            float* __restrict__ t) {
  __shared__ __attribute__((aligned(16))) uint32_t hist[2048];
  __shared__ uint32_t s_state[2];
  const int tid = threadIdx.x;
  if (r <= 0) {
    if (tid == 0) t[blockIdx.x] = 0.f;
    return;
  }
  const float* vr = v + (size_t)blockIdx.x * m;
  uint32_t key[KPT];
#pragma unroll
  for (int k = 0; k < KPT; ++k) {
    const int i = tid + k * kSelThreads;
    key[k] = i < m ? __float_as_uint(fabsf(vr[i])) : 0xffffffffu;
  }
  uint32_t prefix = 0u, hi_mask = 0x80000000u;
  int rem = r;
  select_pass<20, 11>(key, hist, prefix, hi_mask, rem, s_state);
  select_pass<10, 10>(key, hist, prefix, hi_mask, rem, s_state);
  select_pass<0, 10>(key, hist, prefix, hi_mask, rem, s_state);
  if (tid == 0) t[blockIdx.x] = __uint_as_float(prefix);
}

hipError_t launch_row_select(const float* v, int B, int m, int64_t r, float* t, hipStream_t s) {
  if (B < 1 || m < 1 || m > 64 * kSelThreads || r > m) return hipErrorInvalidValue;
  KernelTimer timer("row_select", s);
  const dim3 grid(B), block(kSelThreads);
  const int ri = (int)(r < 0 ? 0 : r);
  if (m <= 4 * kSelThreads)
    hipExtLaunchKernelGGL(k_row_select<4>, grid, block, 0, s, timer.start(), timer.stop(), 0, v, m, ri, t);
  else if (m <= 16 * kSelThreads)
    hipExtLaunchKernelGGL(k_row_select<16>, grid, block, 0, s, timer.start(), timer.stop(), 0, v, m, ri, t);
  else
    hipExtLaunchKernelGGL(k_row_select<64>, grid, block, 0, s, timer.start(), timer.stop(), 0, v, m, ri, t);
  return hipGetLastError();
}

}  // namespace cats
