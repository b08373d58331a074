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
// For a single row of up to kGateSelMaxM neurons the gate kernel's last
// block does this select itself and k_row_select is not launched.
// The fused kernel then runs with v and t_b given (VIN): no W_gate row is
// read a second time.
#include "device.hpp"
#include "internal.hpp"
#include "topk_select.hpp"

namespace cats {

// One block per row: t[b] = the r-th smallest |v[b, :]| (1-indexed), exact
// (topk_select.hpp).  r = 0 gives t = 0.
constexpr int kSelThreads = 1024;

template <int KPT>
__global__ __launch_bounds__(kSelThreads) void k_row_select(const float* __restrict__ v, int m, int r,
                                                            float* __restrict__ t) {
  __shared__ __attribute__((aligned(16))) uint32_t hist[kSelHistBins];
  __shared__ uint32_t s_state[4];
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
  const float tb = select_rank<kSelThreads, KPT>(key, r, hist, s_state);
  if (tid == 0) t[blockIdx.x] = tb;
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
