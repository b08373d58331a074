// Per-token top-k variant of CATS (future work in the appendix comparing
// target and actual sparsity: the target enforced at inference for every
// token instead of one calibrated t).  Row b keeps the neurons with
// |v_bj| >= t_b, t_b = the r-th smallest of its own m values |v_b.| (Eq. 3
// over one token), so every row keeps at least m - r + 1 neurons.
//
// k_gate_v: the gate activations v = SiLU(x W_gate) of up to 8 rows, one
// pass over W_gate with the fused kernel's layout (a block's neurons walked
// by its waves, the next row in flight while one is reduced).
// k_row_select: one block per row, the exact r-th smallest |v| by three
// radix passes over the fp32 bit patterns (LDS histogram, keys in registers).
// The fused kernel then runs with v and t_b given (VIN): no W_gate row is
// read a second time.
#include "device.hpp"
#include "internal.hpp"

namespace cats {

struct GateVArgs {
  const void* wg;  // [m x d]
  const float* x;  // [B x d]
  int B, d, m;
  float* v;        // [B x m]
};

template <typename WT, int NCH, int BT>
__global__ __launch_bounds__(kFusedWaves* kWaveSize) void k_gate_v(GateVArgs a) {
  typedef typename wtraits<WT>::elem E;
  constexpr int VEC = wtraits<WT>::VEC;
  constexpr int CH = kWaveSize * VEC;
  constexpr int DP = NCH * CH;
  constexpr int W = kFusedWaves;
  constexpr int NT = W * kWaveSize;
  __shared__ __attribute__((aligned(16))) float xs[BT * DP];

  const int tid = threadIdx.x;
  const int lane = tid & (kWaveSize - 1);
  const int w = __builtin_amdgcn_readfirstlane(tid / kWaveSize);
  const int B = a.B, d = a.d, m = a.m;
  const uint32_t row_bytes = (uint32_t)d * sizeof(E);
  const __amdgpu_buffer_rsrc_t rg = make_rsrc(a.wg, (uint32_t)((uint64_t)m * row_bytes));
  const int G = gridDim.x, blk = blockIdx.x;
  const int n0 = (int)(((int64_t)blk * m) / G);
  const int nb = (int)(((int64_t)(blk + 1) * m) / G) - n0;
  const int ni = nb > w ? (nb - w + W - 1) / W : 0;

  uint32_t lane_off[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int col = c * CH + lane * VEC;
    lane_off[c] = (col < d) ? (uint32_t)col * sizeof(E) : kOOB;
  }
  auto load_row = [&](u32x4(&buf)[NCH], bool valid, int j) {
    const uint32_t base = valid ? (uint32_t)j * row_bytes : kOOB;
#pragma unroll
    for (int c = 0; c < NCH; ++c) buf[c] = ld_buf16_stream(rg, base + lane_off[c]);
  };
  u32x4 gA[NCH], gB[NCH];
  {
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(a.x, (uint32_t)(B * d * sizeof(float)));
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
    load_row(gA, 0 < ni, n0 + w);
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int i4 = tid + k * NT;
      if (NV % NT == 0 || i4 < NV) *reinterpret_cast<u32x4*>(xs + i4 * 4) = xv[k];
    }
  }
  __syncthreads();

  auto step = [&](int i, const u32x4(&cur)[NCH], u32x4(&nxt)[NCH]) {
    load_row(nxt, i + 1 < ni, n0 + w + (i + 1) * W);
    float acc[BT];
#pragma unroll
    for (int b = 0; b < BT; ++b) acc[b] = 0.f;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int col = c * CH + lane * VEC;
      float wf[VEC];
      widen<WT>(cur[c], wf);
#pragma unroll
      for (int b = 0; b < BT; ++b) {
        if (b < B) {
          const float* xp = xs + b * DP + col;
#pragma unroll
          for (int e4 = 0; e4 < VEC; e4 += 4) {
            const f32x4 xv = *reinterpret_cast<const f32x4*>(xp + e4);
            acc[b] = fmaf(wf[e4 + 0], xv.x, acc[b]);
            acc[b] = fmaf(wf[e4 + 1], xv.y, acc[b]);
            acc[b] = fmaf(wf[e4 + 2], xv.z, acc[b]);
            acc[b] = fmaf(wf[e4 + 3], xv.w, acc[b]);
          }
        }
      }
    }
    const int j = n0 + w + i * W;
#pragma unroll
    for (int b = 0; b < BT; ++b) {
      if (b < B) {
        const float g = wave_sum(acc[b]);
        if (lane == 0 && i < ni) a.v[(size_t)b * m + j] = silu(g);
      }
    }
  };
  for (int i = 0; i < ni; i += 2) {
    step(i, gA, gB);
    if (i + 1 < ni) step(i + 1, gB, gA);
  }
}

template <typename WT, int NCH>
static hipError_t launch_gate_v_nch(int bt, const GateVArgs& a, int G, hipStream_t s) {
  constexpr int DP = NCH * kWaveSize * wtraits<WT>::VEC;
  const dim3 grid(G), block(kFusedWaves * kWaveSize);
  KernelTimer timer("gate_v", s);
  switch (bt) {
    case 1: hipExtLaunchKernelGGL((k_gate_v<WT, NCH, 1>), grid, block, 0, s, timer.start(), timer.stop(), 0, a); break;
    case 2: hipExtLaunchKernelGGL((k_gate_v<WT, NCH, 2>), grid, block, 0, s, timer.start(), timer.stop(), 0, a); break;
    case 4:
      if constexpr (4 * DP * 4 <= kXLdsBytes) {
        hipExtLaunchKernelGGL((k_gate_v<WT, NCH, 4>), grid, block, 0, s, timer.start(), timer.stop(), 0, a);
        break;
      }
      return hipErrorInvalidValue;
    case 8:
      if constexpr (8 * DP * 4 <= kXLdsBytes) {
        hipExtLaunchKernelGGL((k_gate_v<WT, NCH, 8>), grid, block, 0, s, timer.start(), timer.stop(), 0, a);
        break;
      }
      return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename WT>
static hipError_t launch_gate_v_t(int nch, int bt, const GateVArgs& a, int G, hipStream_t s) {
  switch (nch) {
    case 1: return launch_gate_v_nch<WT, 1>(bt, a, G, s);
    case 2: return launch_gate_v_nch<WT, 2>(bt, a, G, s);
    case 4: return launch_gate_v_nch<WT, 4>(bt, a, G, s);
    case 8: return launch_gate_v_nch<WT, 8>(bt, a, G, s);
    case 10: return launch_gate_v_nch<WT, 10>(bt, a, G, s);
    case 16: return launch_gate_v_nch<WT, 16>(bt, a, G, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gate_v(int wdtype_bf16, int nch, int bt, const float* x, const void* wg, int B, int d, int m,
                         float* v, int G, hipStream_t s) {
  GateVArgs a;
  a.wg = wg;
  a.x = x;
  a.B = B;
  a.d = d;
  a.m = m;
  a.v = v;
  return wdtype_bf16 ? launch_gate_v_t<wbf16>(nch, bt, a, G, s) : launch_gate_v_t<wf32>(nch, bt, a, G, s);
}

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
