// Gate activations on their own: v = SiLU(x W_gate) for up to 8 rows in one
// pass over W_gate (Eq. 1's gate product and Eq. 2), written to memory.
// Used where the gate is a separate step: the per-token top-k variant
// (the cutoffs need every activation of a row first) and the unfused
// kernels of the Appendix D structure.  With SEG the kernel also applies
// the CATS_t mask (Eq. 4, 5) and writes each block's ordered list of the
// neurons active in some row: the index list of the Appendix D algorithm
// that builds one, compacted per block without atomics.
//
// A block owns the fused kernel's neuron range; wave w walks neurons
// n0 + w, n0 + w + W, ... with the next row in flight while one is reduced.
//
// With SEL (one row, m up to kGateSelMaxM) the kernel also fixes the row's
// top-k cutoff: every block writes its v with device-coherent stores and
// takes a ticket (ticket.hpp); the last block to arrive reads the whole row
// back and selects its r-th smallest |v| (topk_select.hpp), so no separate
// select launch is needed.  No block waits for another.
#include "gemv_rows.hpp"
#include "ticket.hpp"
#include "topk_select.hpp"

namespace cats {

template <typename WT, int NCH, int BT, bool SEG, bool SEL>
__global__ __launch_bounds__(kFusedWaves* kWaveSize) void k_gate_v(GateVArgs a) {
  typedef RowGeom<WT, NCH> R;
  constexpr int W = kFusedWaves;
  constexpr int NT = W * kWaveSize;
  static_assert(!SEL || (BT == 1 && !SEG), "the in-kernel select takes one row");
  __shared__ __attribute__((aligned(16))) float xs[BT * R::DP];
  __shared__ uint32_t l_mask[SEG ? kFusedMaxNeurons : 1];
  __shared__ int w_cnt[W + 1];
  __shared__ __attribute__((aligned(16))) uint32_t hist[SEL ? kSelHistBins : 1];
  __shared__ float l_vs[SEL ? kFusedMaxNeurons : 1];  // the block's v, stored in one burst at the end
  __shared__ uint32_t s_state[4];
  __shared__ int s_last;

  const int tid = threadIdx.x;
  // (with SEL the ticket word is read now, so that arriving costs one atomic)
  unsigned long long peek = 0ull;
  if constexpr (SEL) {
    if (tid == 0) peek = ticket_peek(a.ticket);
  }
  const int lane = tid & (kWaveSize - 1);
  const int w = __builtin_amdgcn_readfirstlane(tid / kWaveSize);
  const int B = a.B, d = a.d, m = a.m;
  const uint32_t row_bytes = (uint32_t)d * sizeof(typename R::E);
  const __amdgpu_buffer_rsrc_t rg = make_rsrc(a.wg, (uint32_t)((uint64_t)m * row_bytes));
  const NeuronRange nr = neuron_range(blockIdx.x, gridDim.x, m);
  const int ni = nr.nb > w ? (nr.nb - w + W - 1) / W : 0;

  uint32_t off[NCH];
  lane_offsets<WT, NCH>(lane, d, off);
  auto row_base = [&](bool valid, int j) -> uint32_t { return valid ? (uint32_t)j * row_bytes : kOOB; };
  u32x4 gA[NCH], gB[NCH];
  stage_x<R::DP, BT, NT>(xs, a.x, B, d, [&] { load_row16<NCH>(gA, rg, row_base(0 < ni, nr.n0 + w), off); });
  __syncthreads();

  auto step = [&](int i, const u32x4(&cur)[NCH], u32x4(&nxt)[NCH]) {
    load_row16<NCH>(nxt, rg, row_base(i + 1 < ni, nr.n0 + w + (i + 1) * W), off);
    float g[BT];
    row_dots<WT, NCH, BT>(cur, xs, lane, B, g);
    const int j = nr.n0 + w + i * W;
    uint32_t mask = 0;
#pragma unroll
    for (int b = 0; b < BT; ++b) {
      if (b < B) {
        const float v = silu(g[b]);
        if (lane == 0 && i < ni) {
          if constexpr (SEL)
            l_vs[w + i * W] = v;
          else
            a.v[(size_t)b * m + j] = v;
        }
        mask |= (uint32_t)!(fabsf(v) < a.t) << b;
      }
    }
    if constexpr (SEG) {
      if (lane == 0 && i < ni) l_mask[w + i * W] = mask;
    }
  };
  for (int i = 0; i < ni; i += 2) {
    step(i, gA, gB);
    if (i + 1 < ni) step(i + 1, gB, gA);
  }
  if constexpr (SEG) {
    __syncthreads();
    const int cnt = compact_block<W>(l_mask, nr.nb, nr.n0, a.seg_j, a.seg_mask, w_cnt);
    if (tid == 0) a.seg_cnt[blockIdx.x] = cnt;
  }
  if constexpr (SEL) {
    // the block's v as consecutive device-coherent stores (whole lines)
    __syncthreads();
    for (int q = tid; q < nr.nb; q += NT)
      __hip_atomic_store(a.v + nr.n0 + q, l_vs[q], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __builtin_amdgcn_s_waitcnt(0);  // this thread's v stores have completed
    __syncthreads();
    if (tid == 0) s_last = take_ticket(a.ticket, a.epoch, gridDim.x, peek);
    __syncthreads();
    if (!s_last) return;
    // the last block: every block's v is in memory
    if (a.rank <= 0) {
      if (tid == 0) a.t_out[0] = 0.f;
      return;
    }
    // device-coherent loads, all in flight at once (out of range past m)
    const __amdgpu_buffer_rsrc_t rv = make_rsrc(a.v, (uint32_t)m * 4u);
    uint32_t key[kGateSelKeys];
#pragma unroll
    for (int k = 0; k < kGateSelKeys; ++k) {
      const int i = tid + k * NT;
      key[k] = __builtin_amdgcn_raw_buffer_load_b32(rv, i < m ? (int)((uint32_t)i * 4u) : (int)kOOB, 0, kCachePolicySc1);
    }
#pragma unroll
    for (int k = 0; k < kGateSelKeys; ++k)
      key[k] = tid + k * NT < m ? (key[k] & 0x7fffffffu) : 0xffffffffu;  // |v| as bits; padding never matches
    const float tb = select_rank<NT, kGateSelKeys>(key, a.rank, hist, s_state);
    if (tid == 0) a.t_out[0] = tb;
  }
}

template <typename WT, int NCH, bool SEG>
static hipError_t launch_gate_v_nch(int bt, const GateVArgs& a, int G, hipStream_t s) {
  constexpr int DP = RowGeom<WT, NCH>::DP;
  const dim3 grid(G), block(kFusedWaves * kWaveSize);
  KernelTimer timer(SEG ? "gate_v_list" : "gate_v", s);
  switch (bt) {
    case 1: hipExtLaunchKernelGGL((k_gate_v<WT, NCH, 1, SEG, false>), grid, block, 0, s, timer.start(), timer.stop(), 0, a); break;
    case 2: hipExtLaunchKernelGGL((k_gate_v<WT, NCH, 2, SEG, false>), grid, block, 0, s, timer.start(), timer.stop(), 0, a); break;
    case 4:
      if constexpr (4 * DP * 4 <= kXLdsBytes) {
        hipExtLaunchKernelGGL((k_gate_v<WT, NCH, 4, SEG, false>), grid, block, 0, s, timer.start(), timer.stop(), 0, a);
        break;
      }
      return hipErrorInvalidValue;
    case 8:
      if constexpr (8 * DP * 4 <= kXLdsBytes) {
        hipExtLaunchKernelGGL((k_gate_v<WT, NCH, 8, SEG, false>), grid, block, 0, s, timer.start(), timer.stop(), 0, a);
        break;
      }
      return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename WT, bool SEG>
static hipError_t launch_gate_v_t(int nch, int bt, const GateVArgs& a, int G, hipStream_t s) {
  switch (nch) {
    case 1: return launch_gate_v_nch<WT, 1, SEG>(bt, a, G, s);
    case 2: return launch_gate_v_nch<WT, 2, SEG>(bt, a, G, s);
    case 4: return launch_gate_v_nch<WT, 4, SEG>(bt, a, G, s);
    case 8: return launch_gate_v_nch<WT, 8, SEG>(bt, a, G, s);
    case 10: return launch_gate_v_nch<WT, 10, SEG>(bt, a, G, s);
    case 16: return launch_gate_v_nch<WT, 16, SEG>(bt, a, G, s);
    default: return hipErrorInvalidValue;
  }
}

template <typename WT>
static hipError_t launch_gate_v_sel_t(int nch, const GateVArgs& a, int G, hipStream_t s) {
  const dim3 grid(G), block(kFusedWaves * kWaveSize);
  KernelTimer timer("gate_v_select", s);
  switch (nch) {
#define CATS_SEL(N)                                                                                  \
  case N:                                                                                            \
    hipExtLaunchKernelGGL((k_gate_v<WT, N, 1, false, true>), grid, block, 0, s, timer.start(),        \
                          timer.stop(), 0, a);                                                       \
    break;
    CATS_SEL(1)
    CATS_SEL(2)
    CATS_SEL(4)
    CATS_SEL(8)
    CATS_SEL(10)
    CATS_SEL(16)
#undef CATS_SEL
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_gate_v_select(int wdtype_bf16, int nch, const GateVArgs& a, int G, hipStream_t s) {
  if (a.B != 1 || a.m > kGateSelMaxM) return hipErrorInvalidValue;
  return wdtype_bf16 ? launch_gate_v_sel_t<wbf16>(nch, a, G, s) : launch_gate_v_sel_t<wf32>(nch, a, G, s);
}

hipError_t launch_gate_v(int wdtype_bf16, int nch, int bt, bool seg, const GateVArgs& a, int G, hipStream_t s) {
  if (wdtype_bf16)
    return seg ? launch_gate_v_t<wbf16, true>(nch, bt, a, G, s) : launch_gate_v_t<wbf16, false>(nch, bt, a, G, s);
  return seg ? launch_gate_v_t<wf32, true>(nch, bt, a, G, s) : launch_gate_v_t<wf32, false>(nch, bt, a, G, s);
}

}  // namespace cats
