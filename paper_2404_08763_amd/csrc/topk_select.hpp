// The exact r-th smallest of one row's |v| (1-indexed), for the per-token
// top-k variant (the cutoff of Eq. 3 taken over one token's m activations).
//
// Non-negative fp32 values order like their bit patterns (bit 31 is 0), so
// the pattern is fixed digit by digit, most significant first: bits 30..20,
// 19..10, 9..0.  Each pass histograms the digit over the keys that match the
// digits fixed so far; the bin holding the remaining rank becomes the next
// digit.  The row's keys stay in registers across the passes (KPT per
// thread of the NT-thread block; padding keys have bit 31 set and never
// match), and one wave finds the bin by a prefix sum over its lanes (DPP,
// scan.hpp).
#pragma once

#include "device.hpp"
#include "scan.hpp"

namespace cats {

constexpr int kSelHistBins = 2048;  // LDS words a select needs for its histogram

template <int NT, int SHIFT, int BITS, int KPT>
__device__ __forceinline__ void select_pass(const uint32_t (&key)[KPT], uint32_t* hist, uint32_t& prefix,
                                            uint32_t& hi_mask, int& rem, uint32_t* s_state) {
  constexpr int NB = 1 << BITS;
  constexpr int BPL = NB / kWaveSize;  // bins per lane in the scan
  static_assert(NB <= kSelHistBins, "histogram larger than its LDS");
  const int tid = threadIdx.x;
  for (int q = tid; q < NB; q += NT) hist[q] = 0u;
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
    const uint32_t incl = wave_incl_scan(sum);
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
      s_state[2] = h[bin];  // keys that share the new prefix
    }
  }
  __syncthreads();
  prefix = s_state[0];
  rem = (int)s_state[1];
  hi_mask |= (uint32_t)(NB - 1) << SHIFT;
}

// The r-th smallest key of the block's keys (r >= 1 and at most the number
// of real keys), as an fp32 value; every thread of the block takes part.
// s_state holds 4 words.  When the first two digits leave a single key with
// their prefix, that key is the answer and the third pass is skipped.
template <int NT, int KPT>
__device__ __forceinline__ float select_rank(const uint32_t (&key)[KPT], int r, uint32_t* hist, uint32_t* s_state) {
  uint32_t prefix = 0u, hi_mask = 0x80000000u;
  int rem = r;
  select_pass<NT, 20, 11>(key, hist, prefix, hi_mask, rem, s_state);
  select_pass<NT, 10, 10>(key, hist, prefix, hi_mask, rem, s_state);
  if (s_state[2] == 1u) {
#pragma unroll
    for (int k = 0; k < KPT; ++k)
      if ((key[k] & hi_mask) == prefix) s_state[3] = key[k];
    __syncthreads();
    return __uint_as_float(s_state[3]);
  }
  select_pass<NT, 0, 10>(key, hist, prefix, hi_mask, rem, s_state);
  return __uint_as_float(prefix);
}

}  // namespace cats
