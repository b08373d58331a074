// Fused CATS MLP kernel: gate GEMV -> SiLU -> CATS_t mask -> gathered
// up-projection times v -> ordered compaction -> neuron-major
// down-projection into per-block partial sums, in one pass over the weights.
//
// Method (Eq. 1, Eq. 2, Eq. 5 and the "MLP using CATS" algorithm of
// Section 4.3 / Appendix D):
//   v_j = SiLU(x . W_gate[:, j]);  neuron j is active when |v_j| >= t
//   h_j = v_j * (x . W_up[:, j])            only for active j
//   y  += h_j * W_down[j, :]                only for active j
//
// Design (batch 1 is memory-bound; one weight element feeds one FMA):
//  - Weights are neuron-major [m x d]; a row is streamed as NCH chunks of
//    64 lanes x 16 bytes, so every load instruction covers one contiguous
//    KiB.  An inactive neuron costs exactly its gate row; an active one
//    adds its up row and its down row, nothing else.
//  - Every weight load is a buffer load issued on every path; the row of a
//    masked neuron gets an out-of-range offset and reads as zero without
//    moving data (the paper's masked loads with other=0, done by the
//    address unit).  With no load inside a data-dependent branch the
//    compiler counts outstanding loads exactly and prefetches stay in
//    flight.
//  - A block owns a contiguous range of neurons.  Phase 1 needs no barrier:
//    each wave walks its neurons (j = n0 + w, n0 + w + W, ...) in a private
//    pipeline: the gate row of the next neuron is in flight while the
//    current one is reduced, and the up row of an active neuron is consumed
//    one neuron later, so loads always have a neuron's worth of work to
//    hide behind.  h_j lands in LDS.
//  - Phase 2 compacts the block's active neurons in order (ballot +
//    popcount per wave, wave offsets in LDS): the ascending index list of
//    the Appendix D algorithm, built without atomics.
//  - Phase 3 splits every active W_down row by columns over the waves, so
//    each wave keeps d/W accumulators per batch row and no cross-wave
//    reduction is needed; rows are loaded eight at a time, double-buffered.
//  - Each block writes one partial y; a second kernel sums the partials in
//    a fixed order, so results are deterministic run to run.
#pragma once

#include "device.hpp"
#include "internal.hpp"

namespace cats {

// VIN: the gate activations v (and one threshold per row) come precomputed
// (the per-token top-k variant); no W_gate row is read.
template <typename WT, int NCH, int BT, bool DENSE, bool AUX, bool VIN>
__global__ __launch_bounds__(fused_waves(NCH, BT, VIN)* kWaveSize) void k_mlp_fused(FusedArgs a) {
  typedef typename wtraits<WT>::elem E;
  constexpr int VEC = wtraits<WT>::VEC;
  constexpr int CH = kWaveSize * VEC;  // elements per chunk
  constexpr int DP = NCH * CH;         // padded row length in LDS
  constexpr int W = fused_waves(NCH, BT, VIN);
  constexpr int NT = W * kWaveSize;
  constexpr int QMAX = (NCH + W - 1) / W;  // down-stage chunks per wave
  constexpr int RB = QMAX >= 4 ? 2 : 8 / QMAX;  // down rows per batch
  constexpr int NBMAX = kFusedMaxNeurons;  // neurons per block

  __shared__ __attribute__((aligned(16))) float xs[BT * DP];
  __shared__ float l_h[NBMAX][BT];   // h of each local neuron (0 where masked)
  __shared__ float l_v[(AUX || VIN) ? NBMAX : 1][BT];  // v of each local neuron (VIN: as given)
  __shared__ uint32_t l_mask[NBMAX];  // row mask of each local neuron
  __shared__ int c_j[NBMAX];          // compacted: neuron index
  __shared__ float c_h[NBMAX][BT];    // compacted: h per batch row
  __shared__ int w_cnt[W + 1];

  const int tid = threadIdx.x;
  const int lane = tid & (kWaveSize - 1);
  // wave index as a scalar, so per-wave loop bounds are uniform branches
  const int w = __builtin_amdgcn_readfirstlane(tid / kWaveSize);
  const int B = a.B, d = a.d, m = a.m;
  const float t = a.t;
  // per-row cutoffs of the top-k variant (every row uses t otherwise)
  float trow[BT];
#pragma unroll
  for (int b = 0; b < BT; ++b) trow[b] = (VIN && b < B) ? a.vin_t[b] : t;
  const uint32_t row_bytes = (uint32_t)d * sizeof(E);
  const uint32_t mat_bytes = (uint32_t)((uint64_t)m * row_bytes);
  const __amdgpu_buffer_rsrc_t rg = make_rsrc(a.wg, mat_bytes);
  const __amdgpu_buffer_rsrc_t ru = make_rsrc(a.wu, mat_bytes);
  const __amdgpu_buffer_rsrc_t rd = make_rsrc(a.wd, mat_bytes);

  const int G = gridDim.x;
  const int blk = blockIdx.x;
  const int n0 = (int)(((int64_t)blk * m) / G);
  const int nb = (int)(((int64_t)(blk + 1) * m) / G) - n0;  // neurons of this block
  const int ni = nb > w ? (nb - w + W - 1) / W : 0;          // neurons of this wave

  // Per-lane byte offset of chunk c inside a row; kOOB past the row end.
  uint32_t lane_off[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int col = c * CH + lane * VEC;
    lane_off[c] = (col < d) ? (uint32_t)col * sizeof(E) : kOOB;
  }

  auto row_base = [&](bool valid, int j) -> uint32_t { return valid ? (uint32_t)j * row_bytes : kOOB; };

  auto load_row = [&](u32x4(&buf)[NCH], __amdgpu_buffer_rsrc_t r, uint32_t base) {
#pragma unroll
    for (int c = 0; c < NCH; ++c) buf[c] = ld_buf16_stream(r, base + lane_off[c]);
  };

  // Per-row factor on every gate and up dot product: 1, or the RMSNorm
  // scale 1/sqrt(mean(x^2) + eps) when the block is normalised in front
  // (x W scaled after the sum equals (x scaled) W up to rounding).
  float xscale[BT];
#pragma unroll
  for (int b = 0; b < BT; ++b) xscale[b] = 1.f;

  // Dot products of one weight row with the B staged x rows, wave-summed.
  auto row_dot = [&](const u32x4(&buf)[NCH], float(&out)[BT]) {
    float acc[BT];
#pragma unroll
    for (int b = 0; b < BT; ++b) acc[b] = 0.f;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int col = c * CH + lane * VEC;
      float wf[VEC];
      widen<WT>(buf[c], wf);
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
#pragma unroll
    for (int b = 0; b < BT; ++b) out[b] = (b < B) ? wave_sum(acc[b]) * xscale[b] : 0.f;
  };

  // Dot products of two weight rows (a gate row and the previous neuron's
  // up row) with the staged x rows in one pass, so each x value is read
  // from LDS once for both; each accumulator sums in row_dot's order, so the
  // results are row_dot's bits.
  auto row_dot2 = [&](const u32x4(&bufa)[NCH], const u32x4(&bufb)[NCH], float(&outa)[BT], float(&outb)[BT]) {
    float acca[BT], accb[BT];
#pragma unroll
    for (int b = 0; b < BT; ++b) acca[b] = accb[b] = 0.f;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int col = c * CH + lane * VEC;
      float wa[VEC], wb[VEC];
      widen<WT>(bufa[c], wa);
      widen<WT>(bufb[c], wb);
#pragma unroll
      for (int b = 0; b < BT; ++b) {
        if (b < B) {
          const float* xp = xs + b * DP + col;
#pragma unroll
          for (int e4 = 0; e4 < VEC; e4 += 4) {
            const f32x4 xv = *reinterpret_cast<const f32x4*>(xp + e4);
            acca[b] = fmaf(wa[e4 + 0], xv.x, acca[b]);
            acca[b] = fmaf(wa[e4 + 1], xv.y, acca[b]);
            acca[b] = fmaf(wa[e4 + 2], xv.z, acca[b]);
            acca[b] = fmaf(wa[e4 + 3], xv.w, acca[b]);
            accb[b] = fmaf(wb[e4 + 0], xv.x, accb[b]);
            accb[b] = fmaf(wb[e4 + 1], xv.y, accb[b]);
            accb[b] = fmaf(wb[e4 + 2], xv.z, accb[b]);
            accb[b] = fmaf(wb[e4 + 3], xv.w, accb[b]);
          }
        }
      }
    }
#pragma unroll
    for (int b = 0; b < BT; ++b) {
      outa[b] = (b < B) ? wave_sum(acca[b]) * xscale[b] : 0.f;
      outb[b] = (b < B) ? wave_sum(accb[b]) * xscale[b] : 0.f;
    }
  };

  // ---- stage x (rows past B and columns past d read as zero); its loads
  // go out first so the first gate row can stay in flight while x is
  // written to LDS
  u32x4 gA[NCH], gB[NCH], uA[NCH], uB[NCH];
  {
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(a.x, (uint32_t)(B * d * sizeof(float)));
    constexpr int NV = BT * DP / 4;  // float4 slots in LDS
    constexpr int PER = (NV + NT - 1) / NT;
    u32x4 xv[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int i4 = tid + k * NT;
      const int b = (i4 * 4) / DP, c = (i4 * 4) - b * DP;
      const bool ok = (NV % NT == 0 || i4 < NV) && b < B && c < d;
      xv[k] = ld_buf16(rx, ok ? (uint32_t)((b * d + c) * sizeof(float)) : kOOB);
    }
    if constexpr (!VIN) load_row(gA, rg, row_base(0 < ni, n0 + w));
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int i4 = tid + k * NT;
      if (NV % NT == 0 || i4 < NV) *reinterpret_cast<u32x4*>(xs + i4 * 4) = xv[k];
    }
    // VIN: the block's v values go to LDS with x, so a neuron's mask (and
    // with it the decision to load its up row) does not wait for a load of
    // its own v
    if constexpr (VIN) {
      for (int b = 0; b < B; ++b)
        for (int loc = tid; loc < nb; loc += NT) l_v[loc][b] = a.vin[(size_t)b * m + n0 + loc];
    }
  }
  __syncthreads();

  // ---- optional RMSNorm prologue (unit gain): wave b sums row b's squares
  // in a fixed order, so every block derives the same scale bit for bit.
  // It runs while the first gate row is still in flight.
  if (a.norm) {
    __shared__ float l_scale[BT];
    for (int b = w; b < B; b += W) {
      float ss = 0.f;
      for (int c = lane * 4; c < DP; c += kWaveSize * 4) {
        const f32x4 xv = *reinterpret_cast<const f32x4*>(xs + b * DP + c);
        ss = fmaf(xv.x, xv.x, ss);
        ss = fmaf(xv.y, xv.y, ss);
        ss = fmaf(xv.z, xv.z, ss);
        ss = fmaf(xv.w, xv.w, ss);
      }
      ss = wave_sum(ss);
      if (lane == 0) l_scale[b] = 1.f / sqrtf(ss / (float)d + a.eps);
    }
    __syncthreads();
#pragma unroll
    for (int b = 0; b < BT; ++b) xscale[b] = (b < B) ? l_scale[b] : 1.f;
  }

  // ---- phase 1: per-wave pipeline over this wave's neurons
  uint32_t pmask = 0;  // row mask of the previous neuron (its up row is in flight)
  float pv[BT];
#pragma unroll
  for (int b = 0; b < BT; ++b) pv[b] = 0.f;

  // With several rows (and the gate computed here) the gate dot of neuron
  // i and the up dot of neuron i - 1 share one pass over x: at 2..8 rows the
  // LDS reads of the staged rows, not the weight stream, set the pace.
  constexpr bool kPaired = BT > 1 && !VIN;
  // iteration i: prefetch gate(i+1) into gnxt; gate(i) -> mask, issue
  // up(i); finish up(i-1).
  auto iter = [&](int i, u32x4(&gcur)[NCH], u32x4(&gnxt)[NCH], u32x4(&ucur)[NCH],
                  u32x4(&uprev)[NCH]) {
    if constexpr (!VIN) load_row(gnxt, rg, row_base(i + 1 < ni, n0 + w + (i + 1) * W));
    uint32_t mask = 0;
    float v[BT], up2[BT];
#pragma unroll
    for (int b = 0; b < BT; ++b) v[b] = 0.f;
    if constexpr (kPaired) {
      // both buffers are consumed on every path (a missing neuron's rows read
      // as zeros), which keeps the count of loads in flight exact
      float g[BT];
      row_dot2(gcur, uprev, g, up2);
      if (i < ni) {
#pragma unroll
        for (int b = 0; b < BT; ++b)
          if (b < B) v[b] = silu(g[b]);
      }
    }
    if (i < ni) {
      if constexpr (VIN) {
#pragma unroll
        for (int b = 0; b < BT; ++b)
          if (b < B) v[b] = l_v[w + i * W][b];
      } else if constexpr (!kPaired) {
        float g[BT];
        row_dot(gcur, g);
#pragma unroll
        for (int b = 0; b < BT; ++b)
          if (b < B) v[b] = silu(g[b]);
      }
#pragma unroll
      for (int b = 0; b < BT; ++b) {
        if (b < B) {
          const bool keep = DENSE || !(fabsf(v[b]) < trow[b]);
          mask |= (uint32_t)keep << b;
        }
      }
    }
    load_row(ucur, ru, row_base(mask != 0u, n0 + w + i * W));
    if (i >= 1 && i - 1 < ni) {
      const int loc = w + (i - 1) * W;
      // Every up buffer is consumed on every path, a masked neuron's too
      // (its row reads as zeros), which keeps the compiler's count of loads
      // in flight exact across the loop.  With several rows the dot runs on
      // the zeros; with one row (the mask is then wave-uniform) a masked
      // neuron only waits for its dataless load and skips the dot.
      float h[BT], u[BT];
      if constexpr (kPaired) {
#pragma unroll
        for (int b = 0; b < BT; ++b) u[b] = up2[b];
      } else if (BT == 1 && uniform_u32(pmask) == 0u) {
#pragma unroll
        for (int c = 0; c < NCH; ++c) asm volatile("" ::"v"(uprev[c]));
#pragma unroll
        for (int b = 0; b < BT; ++b) u[b] = 0.f;
      } else {
        row_dot(uprev, u);
      }
#pragma unroll
      for (int b = 0; b < BT; ++b) h[b] = ((pmask >> b) & 1u) ? pv[b] * u[b] : 0.f;
      if (lane == 0) {
        l_mask[loc] = pmask;
#pragma unroll
        for (int b = 0; b < BT; ++b) {
          l_h[loc][b] = h[b];
          if constexpr (AUX) l_v[loc][b] = pv[b];
        }
      }
    }
    pmask = mask;
#pragma unroll
    for (int b = 0; b < BT; ++b) pv[b] = v[b];
  };
  // Two neurons per trip so buffers alternate without copies (a copy would
  // wait for the load it copies).
  for (int i = 0; i <= ni; i += 2) {
    iter(i, gA, gB, uA, uB);
    if (i + 1 <= ni) iter(i + 1, gB, gA, uB, uA);
  }
  __syncthreads();

  // ---- phase 2: ordered compaction of the block's active neurons
  int nact = 0;
  {
    const int WPASS = (nb + NT - 1) / NT;
    int base = 0;
    for (int p = 0; p < WPASS; ++p) {
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
        c_j[pos] = n0 + loc;
#pragma unroll
        for (int b = 0; b < BT; ++b) c_h[pos][b] = l_h[loc][b];
        if constexpr (AUX) {
          const size_t o = (size_t)n0 + pos;
          a.seg_j[o] = n0 + loc;
          a.seg_mask[o] = mk;
          for (int b = 0; b < B; ++b) {
            a.seg_v[(size_t)b * m + o] = l_v[loc][b];
            a.seg_h[(size_t)b * m + o] = l_h[loc][b];
          }
        }
      }
      base += w_cnt[W];
      __syncthreads();
    }
    nact = base;
  }
  if constexpr (AUX) {
    if (tid == 0) a.seg_cnt[blk] = nact;
    // the rest of the block's segment names no neuron: zero row masks, so a
    // list entry is exactly an entry with its row's bit set
    for (int i = nact + tid; i < nb; i += NT) a.seg_mask[n0 + i] = 0u;
  }

  // ---- phase 3: down-projection, columns split over the waves
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
      const uint32_t base = row_base(e < nact, c_j[e < nact ? e : 0]);
#pragma unroll
      for (int qq = 0; qq < QMAX; ++qq) buf[r][qq] = ld_buf16_stream(rd, base + down_off[qq]);
    }
  };
  auto accum_batch = [&](const u32x4(&buf)[RB][QMAX], int e0) {
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      const int e = e0 + r;
      if (e < nact) {
        float hb[BT];
#pragma unroll
        for (int b = 0; b < BT; ++b) hb[b] = c_h[e][b];
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
    for (int e0 = 0; e0 < nact; e0 += 2 * RB) {
      load_batch(dB, e0 + RB);
      accum_batch(dA, e0);
      load_batch(dA, e0 + 2 * RB);
      accum_batch(dB, e0 + RB);
    }
  }

  // This block's partial y (columns owned by this wave).
  float* part = a.partial + (size_t)blk * B * d;
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

// Launch one instantiation; NCH and the batch tile are compile-time, so the
// host picks them from d and B (see fused_nch / fused_bt_max).
template <typename WT, bool DENSE, bool AUX, bool VIN, int NCH>
hipError_t launch_fused_nch(int bt, const FusedArgs& a, int G, hipStream_t s) {
  constexpr int DP = NCH * kWaveSize * wtraits<WT>::VEC;
  const dim3 grid(G), block(fused_waves(NCH, bt, VIN) * kWaveSize);
  KernelTimer timer(VIN ? "mlp_fused_topk" : (DENSE ? "mlp_fused_dense" : "mlp_fused_cats"), s);
  switch (bt) {
    case 1: hipExtLaunchKernelGGL((k_mlp_fused<WT, NCH, 1, DENSE, AUX, VIN>), grid, block, 0, s, timer.start(), timer.stop(), 0, a); break;
    case 2: hipExtLaunchKernelGGL((k_mlp_fused<WT, NCH, 2, DENSE, AUX, VIN>), grid, block, 0, s, timer.start(), timer.stop(), 0, a); break;
    case 4:
      if constexpr (4 * DP * 4 <= kXLdsBytes) {
        hipExtLaunchKernelGGL((k_mlp_fused<WT, NCH, 4, DENSE, AUX, VIN>), grid, block, 0, s, timer.start(), timer.stop(), 0, a);
        break;
      }
      return hipErrorInvalidValue;
    case 8:
      if constexpr (8 * DP * 4 <= kXLdsBytes) {
        hipExtLaunchKernelGGL((k_mlp_fused<WT, NCH, 8, DENSE, AUX, VIN>), grid, block, 0, s, timer.start(), timer.stop(), 0, a);
        break;
      }
      return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename WT, bool DENSE, bool AUX, bool VIN = false>
hipError_t launch_fused_t(int nch, int bt, const FusedArgs& a, int G, hipStream_t s) {
  switch (nch) {
    case 1: return launch_fused_nch<WT, DENSE, AUX, VIN, 1>(bt, a, G, s);
    case 2: return launch_fused_nch<WT, DENSE, AUX, VIN, 2>(bt, a, G, s);
    case 4: return launch_fused_nch<WT, DENSE, AUX, VIN, 4>(bt, a, G, s);
    case 8: return launch_fused_nch<WT, DENSE, AUX, VIN, 8>(bt, a, G, s);
    case 10: return launch_fused_nch<WT, DENSE, AUX, VIN, 10>(bt, a, G, s);
    case 16: return launch_fused_nch<WT, DENSE, AUX, VIN, 16>(bt, a, G, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace cats
