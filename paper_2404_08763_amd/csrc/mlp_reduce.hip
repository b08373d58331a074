// Second kernel of the MLP pass: sums the fused kernel's per-block partial
// y in a fixed order (plus the residual), and, when asked for, turns the
// blocks' ordered union segments into each row's ascending active-neuron
// list (the compressed index list of the Appendix D kernel algorithm).
#include "device.hpp"
#include "internal.hpp"
#include "scan.hpp"

namespace cats {

// Eight waves, eight consecutive float4 columns: a block reads whole
// 128-byte lines of every partial row, so no line is fetched by two blocks
// (consecutive blocks run on different XCDs, whose L2s do not share lines).
constexpr int kReduceThreads = 512;
constexpr int kReduceWaves = kReduceThreads / kWaveSize;    // float4 columns per block
constexpr int kReducePer = kFusedBlocks / kWaveSize;        // partials per lane
static_assert(kFusedBlocks % kWaveSize == 0, "partials must split evenly over the lanes");
// List finalize: entries per thread per pass, and one count per wave and
// entry slot, which one wave scans.
constexpr int kFinPer = 8;
constexpr int kFinPass = kFinPer * kReduceThreads;
constexpr int kFinCounts = kFinPer * kReduceWaves;
static_assert(kFinCounts == kWaveSize, "one wave scans a pass's counts");
// Blocks per row: ranges of about kFinRange entries (one compaction pass of
// kFinPass covers a range); the count before a range reads kFinCountPer
// masks per thread at a time.
constexpr int kFinRange = 2048;
constexpr int kFinCountPer = 32;
constexpr int kFinCountPass = kFinCountPer * kReduceThreads;
__host__ __device__ constexpr int fin_blocks(int m) { return m > kFinRange ? (m + kFinRange - 1) / kFinRange : 1; }

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

  // Finalize the active lists.  Segment g (one per block of the producing
  // kernel) covers entries [floor(g m / Gseg), floor((g + 1) m / Gseg)) of
  // the segment arrays; its first seg_cnt[g] entries name the block's
  // union-active neurons in ascending order with their row masks, and the
  // producer zeroes the masks of the rest.  Segments are in neuron order, so
  // row b's list is the entries with bit b set, taken in order: an ordered
  // stream compaction.  A row's entries are split into fin_blocks(m) ranges,
  // one block each.  A block first counts the row's list entries before its
  // range (masks only, a pass's loads all in flight, one block sum), then
  // compacts its own range from that offset: kFinPer entries per thread at
  // a stride of the block (coalesced), a ballot counting each wave's 64
  // entries of a pass and one wave scanning the pass's 64 counts in entry
  // order.  No block waits for another.
  __shared__ int s_off[kFinCounts + 1];
  const int m = a.m;
  const int nfb = fin_blocks(m);
  const int fi = blockIdx.x - nred;
  const int b = fi / nfb, part = fi - b * nfb;
  const int p_lo = (int)(((int64_t)part * m) / nfb), p_hi = (int)(((int64_t)(part + 1) * m) / nfb);
  const int w = tid / kWaveSize;
  const uint32_t mb = (uint32_t)m * 4u;
  const __amdgpu_buffer_rsrc_t rm = make_rsrc(a.seg_mask, mb);
  const __amdgpu_buffer_rsrc_t rj = make_rsrc(a.active_idx ? a.seg_j : nullptr, a.active_idx ? mb : 0u);
  const __amdgpu_buffer_rsrc_t rv =
      make_rsrc(a.active_v ? a.seg_v + (size_t)b * m : nullptr, a.active_v ? mb : 0u);
  const __amdgpu_buffer_rsrc_t rh =
      make_rsrc(a.active_h ? a.seg_h + (size_t)b * m : nullptr, a.active_h ? mb : 0u);
  const uint64_t below = (1ull << lane) - 1ull;
  auto listed = [&](uint32_t mk) -> bool { return (mk >> b) & 1u; };

  int run = 0;  // list entries of row b before the current pass
  {
    int cnt = 0;
    for (int p0 = 0; p0 < p_lo; p0 += kFinCountPass) {
      uint32_t mk[kFinCountPer];
#pragma unroll
      for (int k = 0; k < kFinCountPer; ++k) {
        const int p = p0 + k * kReduceThreads + tid;
        mk[k] = __builtin_amdgcn_raw_buffer_load_b32(rm, p < p_lo ? (uint32_t)p * 4u : kOOB, 0, 0);
      }
#pragma unroll
      for (int k = 0; k < kFinCountPer; ++k) {
        const int p = p0 + k * kReduceThreads + tid;
        cnt += (p < p_lo && listed(mk[k])) ? 1 : 0;
      }
    }
    const int wcnt = (int)wave_incl_scan((uint32_t)cnt);  // the last lane holds the wave's count
    if (lane == kWaveSize - 1) s_off[w] = wcnt;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kReduceWaves; ++k) run += s_off[k];
    __syncthreads();  // s_off is rewritten below
  }

  struct Pass {
    uint32_t mk[kFinPer], jv[kFinPer], vv[kFinPer], hv[kFinPer];
  };
  auto load = [&](Pass& f, int p0) {  // entries past the range read as zero, no traffic
#pragma unroll
    for (int k = 0; k < kFinPer; ++k) {
      const int p = p0 + k * kReduceThreads + tid;
      const uint32_t off = p < p_hi ? (uint32_t)p * 4u : kOOB;
      f.mk[k] = __builtin_amdgcn_raw_buffer_load_b32(rm, off, 0, 0);
      f.jv[k] = __builtin_amdgcn_raw_buffer_load_b32(rj, off, 0, 0);
      f.vv[k] = __builtin_amdgcn_raw_buffer_load_b32(rv, off, 0, 0);
      f.hv[k] = __builtin_amdgcn_raw_buffer_load_b32(rh, off, 0, 0);
    }
  };
  auto compact = [&](const Pass& f, int p0) {
    uint64_t bal[kFinPer];
#pragma unroll
    for (int k = 0; k < kFinPer; ++k) {
      const int p = p0 + k * kReduceThreads + tid;
      bal[k] = __ballot(p < p_hi && listed(f.mk[k]));
      if (lane == 0) s_off[k * kReduceWaves + w] = __popcll(bal[k]);
    }
    __syncthreads();
    if (w == 0) {  // exclusive scan of the 64 counts, entry order = (k, w)
      const int c = s_off[lane];
      const int incl = (int)wave_incl_scan((uint32_t)c);
      s_off[lane] = incl - c;
      if (lane == kWaveSize - 1) s_off[kFinCounts] = incl;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kFinPer; ++k) {
      if ((bal[k] >> lane) & 1ull) {
        const size_t o = (size_t)b * m + run + s_off[k * kReduceWaves + w] + __popcll(bal[k] & below);
        if (a.active_idx) a.active_idx[o] = (int)f.jv[k];
        if (a.active_v) a.active_v[o] = __uint_as_float(f.vv[k]);
        if (a.active_h) a.active_h[o] = __uint_as_float(f.hv[k]);
      }
    }
    run += s_off[kFinCounts];
    __syncthreads();  // s_off is rewritten by the next pass
  };
  // The next pass's loads are in flight while a pass is compacted.
  Pass fa, fb;
  load(fa, p_lo);
  for (int p0 = p_lo; p0 < p_hi; p0 += 2 * kFinPass) {
    load(fb, p0 + kFinPass);
    compact(fa, p0);
    if (p0 + kFinPass < p_hi) {
      load(fa, p0 + 2 * kFinPass);
      compact(fb, p0 + kFinPass);
    }
  }
  if (tid == 0 && a.active_cnt && part == nfb - 1) a.active_cnt[b] = run;
}

hipError_t launch_reduce(const ReduceArgs& a, hipStream_t s) {
  const int d4 = a.d >> 2;
  const int ncb = (d4 + kReduceWaves - 1) / kReduceWaves;
  const int grid = (a.sum_y ? a.B * ncb : 0) + (a.aux ? a.B * fin_blocks(a.m) : 0);
  if (grid == 0) return hipSuccess;
  KernelTimer timer("k_mlp_reduce", s);
  hipExtLaunchKernelGGL(k_mlp_reduce, dim3(grid), dim3(kReduceThreads), 0, s, timer.start(), timer.stop(), 0,
                        a);
  return hipGetLastError();
}

}  // namespace cats
