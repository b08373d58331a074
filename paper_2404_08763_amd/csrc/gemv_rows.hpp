// Building blocks of the neuron-row GEMV kernels outside the fused kernel
// (gate activations, and the separate up and down kernels): the block's
// neuron range, staging x in LDS, one weight row's dot products with the
// staged rows, and the ordered compaction of a block's active neurons.
//
// A weight row of d elements is NCH chunks of 64 lanes x 16 bytes; lane l
// holds elements c * CH + l * VEC .. + VEC - 1 of chunk c.
#pragma once

#include "device.hpp"
#include "internal.hpp"

namespace cats {

// Neurons [n0, n0 + nb) of block blk out of G (the fused kernel's split).
struct NeuronRange {
  int n0, nb;
};
__device__ __forceinline__ NeuronRange neuron_range(int blk, int G, int m) {
  const int n0 = (int)(((int64_t)blk * m) / G);
  return {n0, (int)(((int64_t)(blk + 1) * m) / G) - n0};
}

template <typename WT, int NCH>
struct RowGeom {
  typedef typename wtraits<WT>::elem E;
  static constexpr int VEC = wtraits<WT>::VEC;
  static constexpr int CH = kWaveSize * VEC;
  static constexpr int DP = NCH * CH;  // padded row length in LDS
};

// Per-lane byte offsets of the NCH chunks inside a row; kOOB past d.
template <typename WT, int NCH>
__device__ __forceinline__ void lane_offsets(int lane, int d, uint32_t (&off)[NCH]) {
  typedef RowGeom<WT, NCH> R;
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int col = c * R::CH + lane * R::VEC;
    off[c] = (col < d) ? (uint32_t)col * sizeof(typename R::E) : kOOB;
  }
}

template <int NCH>
__device__ __forceinline__ void load_row16(u32x4 (&buf)[NCH], __amdgpu_buffer_rsrc_t r, uint32_t base,
                                           const uint32_t (&off)[NCH]) {
#pragma unroll
  for (int c = 0; c < NCH; ++c) buf[c] = ld_buf16_stream(r, base + off[c]);
}

// Stage B rows of x [B x d] into xs [BT x DP] (zeros past B and d) with all
// NT threads of the block.  `first` runs between issuing the x loads and
// writing them to LDS (the caller issues its first weight row there).  The
// caller synchronises afterwards.
template <int DP, int BT, int NT, typename F>
__device__ __forceinline__ void stage_x(float* xs, const float* x, int B, int d, F&& first) {
  const int tid = threadIdx.x;
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, (uint32_t)(B * d * sizeof(float)));
  constexpr int NV = BT * DP / 4;
  constexpr int PER = (NV + NT - 1) / NT;
  u32x4 xv[PER];
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int i4 = tid + k * NT;
    const int b = (i4 * 4) / DP, c = (i4 * 4) - b * DP;
    const bool ok = (NV % NT == 0 || i4 < NV) && b < B && c < d;
    xv[k] = ld_buf16(rx, ok ? (uint32_t)((b * d + c) * sizeof(float)) : kOOB);
  }
  first();
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int i4 = tid + k * NT;
    if (NV % NT == 0 || i4 < NV) *reinterpret_cast<u32x4*>(xs + i4 * 4) = xv[k];
  }
}

// out[b] = sum over the row of w * x_b (b < B), summed over the wave in a
// fixed order; every lane gets the result.
template <typename WT, int NCH, int BT>
__device__ __forceinline__ void row_dots(const u32x4 (&buf)[NCH], const float* xs, int lane, int B,
                                         float (&out)[BT]) {
  typedef RowGeom<WT, NCH> R;
  float acc[BT];
#pragma unroll
  for (int b = 0; b < BT; ++b) acc[b] = 0.f;
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int col = c * R::CH + lane * R::VEC;
    float wf[R::VEC];
    widen<WT>(buf[c], wf);
#pragma unroll
    for (int b = 0; b < BT; ++b) {
      if (b < B) {
        const float* xp = xs + b * R::DP + col;
#pragma unroll
        for (int e4 = 0; e4 < R::VEC; e4 += 4) {
          const f32x4 xv = *reinterpret_cast<const f32x4*>(xp + e4);
          acc[b] = fmaf(wf[e4 + 0], xv.x, acc[b]);
          acc[b] = fmaf(wf[e4 + 1], xv.y, acc[b]);
          acc[b] = fmaf(wf[e4 + 2], xv.z, acc[b]);
          acc[b] = fmaf(wf[e4 + 3], xv.w, acc[b]);
        }
      }
    }
  }
#pragma unroll
  for (int b = 0; b < BT; ++b) out[b] = (b < B) ? wave_sum(acc[b]) : 0.f;
}

// Ordered compaction of the block's local neurons [0, nb) whose row mask in
// l_mask is non-zero: writes seg_j[n0 + pos] = n0 + loc and seg_mask, in
// ascending loc, and returns the count (uniform).  No atomics: a ballot and
// popcount per wave, wave offsets through w_cnt [W + 1] in LDS.  Every
// thread of the block must call it.
template <int W>
__device__ __forceinline__ int compact_block(const uint32_t* l_mask, int nb, int n0, int* seg_j,
                                             uint32_t* seg_mask, int* w_cnt) {
  constexpr int NT = W * kWaveSize;
  const int tid = threadIdx.x;
  const int lane = tid & (kWaveSize - 1);
  const int w = tid / kWaveSize;
  int base = 0;
  for (int p = 0; p * NT < nb; ++p) {
    const int loc = p * NT + tid;
    const uint32_t mk = loc < nb ? l_mask[loc] : 0u;
    const uint64_t bal = __ballot(mk != 0u);
    if (lane == 0) w_cnt[w] = __popcll(bal);
    __syncthreads();
    if (tid == 0) {
      int run = 0;
      for (int k = 0; k < W; ++k) {
        const int c = w_cnt[k];
        w_cnt[k] = run;
        run += c;
      }
      w_cnt[W] = run;
    }
    __syncthreads();
    if (mk) {
      const int pos = base + w_cnt[w] + __popcll(bal & ((1ull << lane) - 1ull));
      seg_j[n0 + pos] = n0 + loc;
      seg_mask[n0 + pos] = mk;
    }
    base += w_cnt[W];
    __syncthreads();
  }
  return base;
}

}  // namespace cats
