// Second kernel of the MLP pass: sums the fused kernel's per-block partial
// y in a fixed order (plus the residual), and, when asked for, turns the
// blocks' ordered union segments into each row's ascending active-neuron
// list (the compressed index list of the Appendix D kernel algorithm).
#include "device.hpp"
#include "internal.hpp"

namespace cats {

constexpr int kReduceThreads = 256;
constexpr int kReduceCols4 = 8;                             // float4 columns per block
constexpr int kReduceSubs = kReduceThreads / kReduceCols4;  // partial subsets per block
constexpr int kReducePer = kFusedBlocks / kReduceSubs;      // partials per thread
static_assert(kFusedBlocks % kReduceSubs == 0, "partials must split evenly over the subsets");

__global__ __launch_bounds__(kReduceThreads) void k_mlp_reduce(ReduceArgs a) {
  const int tid = threadIdx.x;
  const int d4 = a.d >> 2;
  const int ncb = (d4 + kReduceCols4 - 1) / kReduceCols4;
  const int nred = a.B * ncb;

  if ((int)blockIdx.x < nred) {
    // y[b, c] = residual[b, c] + sum over sub (ascending) of (sum over
    // g = sub + 32 k, ascending k, of partial[g, b, c]); a fixed order, so
    // deterministic.  All loads of a thread are issued before the first add.
    __shared__ f32x4 red[kReduceSubs][kReduceCols4];
    const int b = blockIdx.x / ncb, cb = blockIdx.x - b * ncb;
    const int cl = tid % kReduceCols4;
    const int c4 = cb * kReduceCols4 + cl;
    const int sub = tid / kReduceCols4;
    const __amdgpu_buffer_rsrc_t rp =
        make_rsrc(a.partial, (uint32_t)((size_t)a.G * a.B * a.d * sizeof(float)));
    u32x4 v[kReducePer];
#pragma unroll
    for (int k = 0; k < kReducePer; ++k) {
      const int g = sub + k * kReduceSubs;
      const bool ok = g < a.G && c4 < d4;
      v[k] = ld_buf16(rp, ok ? (uint32_t)((((size_t)g * a.B + b) * a.d + (size_t)c4 * 4) * sizeof(float)) : kOOB);
    }
    f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = 0; k < kReducePer; ++k) {
      f32x4 f = {__uint_as_float(v[k].x), __uint_as_float(v[k].y), __uint_as_float(v[k].z),
                 __uint_as_float(v[k].w)};
      s += f;
    }
    red[sub][cl] = s;
    __syncthreads();
    if (sub == 0 && c4 < d4) {
      f32x4 tot = red[0][cl];
#pragma unroll
      for (int k = 1; k < kReduceSubs; ++k) tot += red[k][cl];
      if (a.residual) tot = reinterpret_cast<const f32x4*>(a.residual + (size_t)b * a.d)[c4] + tot;
      reinterpret_cast<f32x4*>(a.y + (size_t)b * a.d)[c4] = tot;
    }
    return;
  }

  // Finalize the active lists of row b: segment g (one per fused block)
  // starts at its block's first neuron and is ascending; segments are in
  // neuron order, so concatenating the entries whose row bit b is set gives
  // the ascending list.
  __shared__ int offs[kFusedBlocks + 1];
  const int b = blockIdx.x - nred;
  for (int g = tid; g < a.G; g += kReduceThreads) {
    const int base = (int)(((int64_t)g * a.m) / a.G);
    const int sc = a.seg_cnt[g];
    int mine = 0;
    for (int e = 0; e < sc; ++e) mine += (int)((a.seg_mask[base + e] >> b) & 1u);
    offs[g] = mine;
  }
  __syncthreads();
  if (tid == 0) {  // exclusive scan over the segment counts
    int run = 0;
    for (int k = 0; k < a.G; ++k) {
      const int c = offs[k];
      offs[k] = run;
      run += c;
    }
    offs[a.G] = run;
  }
  __syncthreads();
  for (int g = tid; g < a.G; g += kReduceThreads) {
    const int base = (int)(((int64_t)g * a.m) / a.G);
    const int sc = a.seg_cnt[g];
    int pos = offs[g];
    for (int e = 0; e < sc; ++e) {
      if ((a.seg_mask[base + e] >> b) & 1u) {
        const size_t o = (size_t)b * a.m + pos;
        if (a.active_idx) a.active_idx[o] = a.seg_j[base + e];
        if (a.active_v) a.active_v[o] = a.seg_v[(size_t)b * a.m + base + e];
        if (a.active_h) a.active_h[o] = a.seg_h[(size_t)b * a.m + base + e];
        ++pos;
      }
    }
  }
  if (tid == 0 && a.active_cnt) a.active_cnt[b] = offs[a.G];
}

hipError_t launch_reduce(const ReduceArgs& a, hipStream_t s) {
  const int d4 = a.d >> 2;
  const int ncb = (d4 + kReduceCols4 - 1) / kReduceCols4;
  const int grid = a.B * ncb + (a.aux ? a.B : 0);
  KernelTimer timer("k_mlp_reduce", s);
  hipExtLaunchKernelGGL(k_mlp_reduce, dim3(grid), dim3(kReduceThreads), 0, s, timer.start(), timer.stop(), 0,
                        a);
  return hipGetLastError();
}

}  // namespace cats
