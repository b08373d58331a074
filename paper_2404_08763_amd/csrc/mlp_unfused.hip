// The CATS MLP in the paper's own kernel structure (Section 4.3 and
// Appendix D): a gate pass (gate_v.hip), then an up-projection kernel and a
// down-projection kernel that each find their rows on their own, then the
// fixed-order sum of the per-block partials (mlp_reduce.hip).  Two ways of
// finding the rows, the ablation of Appendix D:
//  - mask (the algorithm without atomic operations): every neuron of the
//    block's range is visited and its rows are loaded under the mask
//    |v_j| >= t; a masked row is an out-of-range buffer load that reads as
//    zero and moves no data, and contributes zero;
//  - index: only the neurons of the block's ordered active list (written by
//    the gate pass) are visited, with unpredicated loads.
// Both compute Algorithm 1 of Section 4.3 exactly as the fused kernel does:
// h_j = v_j (x . W_up[:, j]) for active j, y = sum_j h_j W_down[j, :].
// The intermediate h (the listing's x_1) goes through memory between the two
// kernels, which the fused kernel avoids.
#include "gemv_rows.hpp"

namespace cats {

// Up-projection: h = v * (x W_up) on the active neurons.  Mask mode writes
// h[b, j] for every neuron of the range (zero where row b masks j); index
// mode writes h[b, n0 + e] for list entry e.
template <typename WT, int NCH, int BT, bool IDX>
__global__ __launch_bounds__(kFusedWaves* kWaveSize) void k_unfused_up(UnfusedArgs a) {
  typedef RowGeom<WT, NCH> R;
  constexpr int W = kFusedWaves;
  constexpr int NT = W * kWaveSize;
  static_assert(kFusedMaxNeurons / W <= kWaveSize, "a wave's entries must fit one per lane");
  __shared__ __attribute__((aligned(16))) float xs[BT * R::DP];

  const int tid = threadIdx.x;
  const int lane = tid & (kWaveSize - 1);
  const int w = __builtin_amdgcn_readfirstlane(tid / kWaveSize);
  const int B = a.B, d = a.d, m = a.m;
  const uint32_t row_bytes = (uint32_t)d * sizeof(typename R::E);
  const __amdgpu_buffer_rsrc_t ru = make_rsrc(a.wu, (uint32_t)((uint64_t)m * row_bytes));
  const NeuronRange nr = neuron_range(blockIdx.x, gridDim.x, m);
  const int cnt = IDX ? __builtin_amdgcn_readfirstlane(a.seg_cnt[blockIdx.x]) : nr.nb;
  const int ni = cnt > w ? (cnt - w + W - 1) / W : 0;  // this wave's entries w, w + W, ...

  // Lane l holds entry w + l W: its neuron, v per row and row mask.
  int lj = 0;
  uint32_t lmask = 0;
  float lv[BT];
#pragma unroll
  for (int b = 0; b < BT; ++b) lv[b] = 0.f;
  if (lane < ni) {
    const int e = w + lane * W;
    lj = IDX ? a.seg_j[nr.n0 + e] : nr.n0 + e;
#pragma unroll
    for (int b = 0; b < BT; ++b) {
      if (b < B) {
        lv[b] = a.v[(size_t)b * m + lj];
        lmask |= (uint32_t)!(fabsf(lv[b]) < a.t) << b;
      }
    }
  }
  auto entry_base = [&](int i) -> uint32_t {
    const int j = __shfl(lj, i);
    const uint32_t mk = (uint32_t)__shfl((int)lmask, i);
    return (i < ni && mk != 0u) ? (uint32_t)j * row_bytes : kOOB;
  };

  uint32_t off[NCH];
  lane_offsets<WT, NCH>(lane, d, off);
  u32x4 uA[NCH], uB[NCH];
  stage_x<R::DP, BT, NT>(xs, a.x, B, d, [&] { load_row16<NCH>(uA, ru, entry_base(0), off); });
  __syncthreads();

  auto step = [&](int i, const u32x4(&cur)[NCH], u32x4(&nxt)[NCH]) {
    load_row16<NCH>(nxt, ru, entry_base(i + 1), off);
    float u[BT];
    row_dots<WT, NCH, BT>(cur, xs, lane, B, u);
    const int j = __shfl(lj, i);
    const uint32_t mk = (uint32_t)__shfl((int)lmask, i);
    const int pos = IDX ? nr.n0 + w + i * W : j;
#pragma unroll
    for (int b = 0; b < BT; ++b) {
      if (b < B) {
        const float v = __shfl(lv[b], i);
        const float h = ((mk >> b) & 1u) ? v * u[b] : 0.f;
        if (lane == 0) a.h[(size_t)b * m + pos] = h;
      }
    }
  };
  for (int i = 0; i < ni; i += 2) {
    step(i, uA, uB);
    if (i + 1 < ni) step(i + 1, uB, uA);
  }
}

// Down-projection into the block's partial y: the rows of the block's
// visited neurons split by columns over the waves (each wave owns chunks
// w, w + W, ... of every row and needs no cross-wave sum), eight rows per
// wave load, double-buffered.
template <typename WT, int NCH, int BT, bool IDX>
__global__ __launch_bounds__(kFusedWaves* kWaveSize) void k_unfused_down(UnfusedArgs a) {
  typedef RowGeom<WT, NCH> R;
  typedef typename R::E E;
  constexpr int VEC = R::VEC;
  constexpr int CH = R::CH;
  constexpr int W = kFusedWaves;
  constexpr int NT = W * kWaveSize;
  constexpr int QMAX = (NCH + W - 1) / W;
  constexpr int RB = QMAX >= 4 ? 2 : 8 / QMAX;
  __shared__ int l_j[kFusedMaxNeurons];           // row to load, -1 when masked
  __shared__ float l_h[kFusedMaxNeurons][BT];

  const int tid = threadIdx.x;
  const int lane = tid & (kWaveSize - 1);
  const int w = __builtin_amdgcn_readfirstlane(tid / kWaveSize);
  const int B = a.B, d = a.d, m = a.m;
  const uint32_t row_bytes = (uint32_t)d * sizeof(E);
  const __amdgpu_buffer_rsrc_t rd = make_rsrc(a.wd, (uint32_t)((uint64_t)m * row_bytes));
  const NeuronRange nr = neuron_range(blockIdx.x, gridDim.x, m);
  const int cnt = IDX ? __builtin_amdgcn_readfirstlane(a.seg_cnt[blockIdx.x]) : nr.nb;

  for (int e = tid; e < cnt; e += NT) {
    int j, pos;
    bool act = true;
    if constexpr (IDX) {
      j = a.seg_j[nr.n0 + e];
      pos = nr.n0 + e;
    } else {
      j = nr.n0 + e;
      pos = j;
      act = false;
      for (int b = 0; b < B; ++b) act = act || !(fabsf(a.v[(size_t)b * m + j]) < a.t);
    }
    l_j[e] = act ? j : -1;
#pragma unroll
    for (int b = 0; b < BT; ++b) l_h[e][b] = (b < B) ? a.h[(size_t)b * m + pos] : 0.f;
  }
  __syncthreads();

  uint32_t down_off[QMAX];
#pragma unroll
  for (int qq = 0; qq < QMAX; ++qq) {
    const int c = w + qq * W;
    const int col = c * CH + lane * VEC;
    down_off[qq] = (c < NCH && col < d) ? (uint32_t)col * sizeof(E) : kOOB;
  }
  float acc[BT][QMAX][VEC];
#pragma unroll
  for (int b = 0; b < BT; ++b)
#pragma unroll
    for (int q = 0; q < QMAX; ++q)
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc[b][q][e] = 0.f;

  auto load_batch = [&](u32x4(&buf)[RB][QMAX], int e0) {
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      const int e = e0 + r;
      const int j = e < cnt ? l_j[e] : -1;
      const uint32_t base = j >= 0 ? (uint32_t)j * row_bytes : kOOB;
#pragma unroll
      for (int qq = 0; qq < QMAX; ++qq) buf[r][qq] = ld_buf16_stream(rd, base + down_off[qq]);
    }
  };
  auto accum_batch = [&](const u32x4(&buf)[RB][QMAX], int e0) {
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      const int e = e0 + r;
      if (e < cnt) {
        float hb[BT];
#pragma unroll
        for (int b = 0; b < BT; ++b) hb[b] = l_h[e][b];
#pragma unroll
        for (int qq = 0; qq < QMAX; ++qq) {
          if (w + qq * W < NCH) {
            float wf[VEC];
            widen<WT>(buf[r][qq], wf);
#pragma unroll
            for (int b = 0; b < BT; ++b) {
              if (b < B) {
#pragma unroll
                for (int k = 0; k < VEC; ++k) acc[b][qq][k] = fmaf(hb[b], wf[k], acc[b][qq][k]);
              }
            }
          }
        }
      }
    }
  };
  {
    u32x4 dA[RB][QMAX], dB[RB][QMAX];
    load_batch(dA, 0);
    for (int e0 = 0; e0 < cnt; e0 += 2 * RB) {
      load_batch(dB, e0 + RB);
      accum_batch(dA, e0);
      load_batch(dA, e0 + 2 * RB);
      accum_batch(dB, e0 + RB);
    }
  }

  float* part = a.partial + (size_t)blockIdx.x * B * d;
#pragma unroll
  for (int b = 0; b < BT; ++b) {
    if (b < B) {
#pragma unroll
      for (int qq = 0; qq < QMAX; ++qq) {
        const int c = w + qq * W;
        const int col = c * CH + lane * VEC;
        if (c < NCH && col < d) {
#pragma unroll
          for (int e4 = 0; e4 < VEC; e4 += 4) {
            f32x4 o = {acc[b][qq][e4], acc[b][qq][e4 + 1], acc[b][qq][e4 + 2], acc[b][qq][e4 + 3]};
            *reinterpret_cast<f32x4*>(part + (size_t)b * d + col + e4) = o;
          }
        }
      }
    }
  }
}

template <typename WT, int NCH, bool IDX, bool UP>
static hipError_t launch_unfused_nch(int bt, const UnfusedArgs& a, int G, hipStream_t s) {
  constexpr int DP = RowGeom<WT, NCH>::DP;
  const dim3 grid(G), block(kFusedWaves * kWaveSize);
  KernelTimer timer(UP ? (IDX ? "unfused_up_index" : "unfused_up_mask")
                       : (IDX ? "unfused_down_index" : "unfused_down_mask"), s);
#define CATS_UNFUSED_LAUNCH(BTV)                                                                     \
  do {                                                                                               \
    if constexpr (UP)                                                                                \
      hipExtLaunchKernelGGL((k_unfused_up<WT, NCH, BTV, IDX>), grid, block, 0, s, timer.start(),    \
                            timer.stop(), 0, a);                                                     \
    else                                                                                             \
      hipExtLaunchKernelGGL((k_unfused_down<WT, NCH, BTV, IDX>), grid, block, 0, s, timer.start(),  \
                            timer.stop(), 0, a);                                                     \
  } while (0)
  switch (bt) {
    case 1: CATS_UNFUSED_LAUNCH(1); break;
    case 2: CATS_UNFUSED_LAUNCH(2); break;
    case 4:
      if constexpr (4 * DP * 4 <= kXLdsBytes) {
        CATS_UNFUSED_LAUNCH(4);
        break;
      }
      return hipErrorInvalidValue;
    case 8:
      if constexpr (8 * DP * 4 <= kXLdsBytes) {
        CATS_UNFUSED_LAUNCH(8);
        break;
      }
      return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
#undef CATS_UNFUSED_LAUNCH
  return hipGetLastError();
}

template <typename WT, bool IDX, bool UP>
static hipError_t launch_unfused_t(int nch, int bt, const UnfusedArgs& a, int G, hipStream_t s) {
  switch (nch) {
    case 1: return launch_unfused_nch<WT, 1, IDX, UP>(bt, a, G, s);
    case 2: return launch_unfused_nch<WT, 2, IDX, UP>(bt, a, G, s);
    case 4: return launch_unfused_nch<WT, 4, IDX, UP>(bt, a, G, s);
    case 8: return launch_unfused_nch<WT, 8, IDX, UP>(bt, a, G, s);
    case 10: return launch_unfused_nch<WT, 10, IDX, UP>(bt, a, G, s);
    case 16: return launch_unfused_nch<WT, 16, IDX, UP>(bt, a, G, s);
    default: return hipErrorInvalidValue;
  }
}

template <bool UP>
static hipError_t launch_unfused(int wdtype_bf16, int nch, int bt, bool index, const UnfusedArgs& a, int G,
                                 hipStream_t s) {
  if (wdtype_bf16)
    return index ? launch_unfused_t<wbf16, true, UP>(nch, bt, a, G, s)
                 : launch_unfused_t<wbf16, false, UP>(nch, bt, a, G, s);
  return index ? launch_unfused_t<wf32, true, UP>(nch, bt, a, G, s)
               : launch_unfused_t<wf32, false, UP>(nch, bt, a, G, s);
}

hipError_t launch_unfused_up(int wdtype_bf16, int nch, int bt, bool index, const UnfusedArgs& a, int G,
                             hipStream_t s) {
  return launch_unfused<true>(wdtype_bf16, nch, bt, index, a, G, s);
}

hipError_t launch_unfused_down(int wdtype_bf16, int nch, int bt, bool index, const UnfusedArgs& a, int G,
                               hipStream_t s) {
  return launch_unfused<false>(wdtype_bf16, nch, bt, index, a, G, s);
}

}  // namespace cats
