// Second kernel of the MLP pass: sums the fused kernel's per-block partial
// y in a fixed order (plus the residual), and, when asked for, turns the
// blocks' ordered union segments into each row's ascending active-neuron
// list (the compressed index list of the Appendix D kernel algorithm).
#include "device.hpp"
#include "internal.hpp"

namespace cats {

// Eight waves, eight consecutive float4 columns: a block reads whole
// 128-byte lines of every partial row, so no line is fetched by two blocks
// (consecutive blocks run on different XCDs, whose L2s do not share lines).
constexpr int kReduceThreads = 512;
constexpr int kReduceWaves = kReduceThreads / kWaveSize;    // float4 columns per block
constexpr int kReducePer = kFusedBlocks / kWaveSize;        // partials per lane
static_assert(kFusedBlocks % kWaveSize == 0, "partials must split evenly over the lanes");

__global__ __launch_bounds__(kReduceThreads) void k_mlp_reduce(ReduceArgs a) {
  const int tid = threadIdx.x;
  const int lane = tid & (kWaveSize - 1);
  const int d4 = a.d >> 2;
  const int ncb = (d4 + kReduceWaves - 1) / kReduceWaves;
  const int nred = a.sum_y ? a.B * ncb : 0;

  if ((int)blockIdx.x < nred) {
    // One wave per float4 column c of row b:
    //   y[b, c] = residual[b, c] + wave_sum over lanes of
    //             (sum over k ascending of partial[lane + 64 k, b, c])
    // a fixed order (the wave sum's tree is fixed), so deterministic.  All
    // loads, the residual's included, are issued before the first add, and
    // no LDS or barrier is involved: the kernel costs one memory latency.
    const int b = blockIdx.x / ncb, cb = blockIdx.x - b * ncb;
    const int c4 = __builtin_amdgcn_readfirstlane(cb * kReduceWaves + tid / kWaveSize);
    if (c4 >= d4) return;  // whole wave
    const __amdgpu_buffer_rsrc_t rp =
        make_rsrc(a.partial, (uint32_t)((size_t)a.G * a.B * a.d * sizeof(float)));
    u32x4 v[kReducePer];
#pragma unroll
    for (int k = 0; k < kReducePer; ++k) {
      const int g = lane + k * kWaveSize;
      v[k] = ld_buf16(rp, g < a.G ? (uint32_t)((((size_t)g * a.B + b) * a.d + (size_t)c4 * 4) * sizeof(float)) : kOOB);
    }
    u32x4 rv = {0u, 0u, 0u, 0u};
    if (a.residual) {
      const __amdgpu_buffer_rsrc_t rr = make_rsrc(a.residual + (size_t)b * a.d, (uint32_t)(a.d * sizeof(float)));
      rv = ld_buf16(rr, (uint32_t)c4 * 16u);
    }
    float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
#pragma unroll
    for (int k = 0; k < kReducePer; ++k) {
      s0 += __uint_as_float(v[k].x);
      s1 += __uint_as_float(v[k].y);
      s2 += __uint_as_float(v[k].z);
      s3 += __uint_as_float(v[k].w);
    }
    f32x4 tot = {wave_sum(s0), wave_sum(s1), wave_sum(s2), wave_sum(s3)};
    if (lane == 0) {
      if (a.residual) {
        const f32x4 r = {__uint_as_float(rv.x), __uint_as_float(rv.y), __uint_as_float(rv.z), __uint_as_float(rv.w)};
        tot = r + tot;
      }
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
  for (int g = tid; g < a.Gseg; g += kReduceThreads) {
    const int base = (int)(((int64_t)g * a.m) / a.Gseg);
    const int sc = a.seg_cnt[g];
    int mine = 0;
    for (int e = 0; e < sc; ++e) mine += (int)((a.seg_mask[base + e] >> b) & 1u);
    offs[g] = mine;
  }
  __syncthreads();
  if (tid == 0) {  // exclusive scan over the segment counts
    int run = 0;
    for (int k = 0; k < a.Gseg; ++k) {
      const int c = offs[k];
      offs[k] = run;
      run += c;
    }
    offs[a.Gseg] = run;
  }
  __syncthreads();
  for (int g = tid; g < a.Gseg; g += kReduceThreads) {
    const int base = (int)(((int64_t)g * a.m) / a.Gseg);
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
  if (tid == 0 && a.active_cnt) a.active_cnt[b] = offs[a.Gseg];
}

hipError_t launch_reduce(const ReduceArgs& a, hipStream_t s) {
  const int d4 = a.d >> 2;
  const int ncb = (d4 + kReduceWaves - 1) / kReduceWaves;
  const int grid = (a.sum_y ? a.B * ncb : 0) + (a.aux ? a.B : 0);
  if (grid == 0) return hipSuccess;
  KernelTimer timer("k_mlp_reduce", s);
  hipExtLaunchKernelGGL(k_mlp_reduce, dim3(grid), dim3(kReduceThreads), 0, s, timer.start(), timer.stop(), 0,
                        a);
  return hipGetLastError();
}

}  // namespace cats
