// Batched CATS MLP for 5..16 rows with bf16 weights: the gate and up
// projections are dense contractions [B x d] . [d x m] and run on the matrix
// cores; the down-projection is split by column tiles so that few partial
// sums of y are written.
//
// Method (Eq. 1, 2 and 5 with one mask per row, as Eq. 5 is elementwise):
//   v_bj = SiLU(x_b . W_gate[:, j]);  (b, j) active when |v_bj| >= t
//   h_bj = v_bj * (x_b . W_up[:, j])  for active (b, j), else 0
//   y_b  = residual_b + sum_j h_bj W_down[j, :]
// Only the rows of W_up and W_down in the union of the rows' active sets
// are read (the union is what a batch must stream; the paper's kernels take
// one mask, batch 1).
//
// Kernel 1 (k_mlp_gateup_mfma): a block owns a contiguous neuron range in
// tiles of 16 neurons.  Each of its 16 waves owns one sixteenth of the columns
// of d and keeps its slice of x in registers as the B operand of
// v_mfma_f32_16x16x32_bf16 (x = hi + lo, both bf16: the two products carry
// 16 bits of x's 24-bit mantissa, relative error below 2^-16 per term, with
// fp32 accumulation).  The waves' partial dot products meet in LDS and are
// summed in wave order.  Gate tiles come first, then the up tiles of the
// neurons some row keeps; the next tile's weight loads are in flight while a
// tile is multiplied.  The block writes its union-active neurons in
// ascending order with their row masks and h (the segment lists the
// finalize step of k_mlp_reduce turns into per-row active lists).
//
// Kernel 2 (k_mlp_down_cols): block (column tile, neuron group) accumulates
// h_b W_down[j, cols] over the group's union-active rows, four rows per
// wave load (a quad of lanes per column chunk), and writes one partial y per
// neuron group; k_mlp_reduce sums the groups in order.
#include "device.hpp"
#include "internal.hpp"

namespace cats {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kBW = kBatchedWaves;
constexpr int kBThreads = kBW * kWaveSize;
constexpr int kGW = kGateUpWaves;
constexpr int kGThreads = kGW * kWaveSize;
constexpr int kBTileN = 16;  // neurons per MFMA tile (and batch columns)

// bf16 bit pattern nearest to f (ties to even); NaN stays a quiet NaN.
__device__ __forceinline__ uint32_t bf16_bits(float f) {
  const uint32_t u = __float_as_uint(f);
  const uint32_t rne = (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
  return ((u & 0x7fffffffu) > 0x7f800000u) ? ((u >> 16) | 0x40u) : rne;
}

__device__ __forceinline__ bf16x8 as_bf16x8(const u32x4& v) { return __builtin_bit_cast(bf16x8, v); }

// Split 8 fp32 values into bf16 hi and lo parts, packed two per word
// (element 2i in the low half of word i, the order of a 16-byte bf16 load).
// Also adds the squares of the 8 values to ss (for the RMSNorm scale).
__device__ __forceinline__ void split8(const u32x4& a, const u32x4& b, bf16x8& hi, bf16x8& lo, float& ss) {
  const float f[8] = {__uint_as_float(a.x), __uint_as_float(a.y), __uint_as_float(a.z), __uint_as_float(a.w),
                      __uint_as_float(b.x), __uint_as_float(b.y), __uint_as_float(b.z), __uint_as_float(b.w)};
  uint32_t h[8], l[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    ss = fmaf(f[e], f[e], ss);
    h[e] = bf16_bits(f[e]);
    l[e] = bf16_bits(f[e] - __uint_as_float(h[e] << 16));
  }
  const u32x4 hv = {h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
  const u32x4 lv = {l[0] | (l[1] << 16), l[2] | (l[3] << 16), l[4] | (l[5] << 16), l[6] | (l[7] << 16)};
  hi = as_bf16x8(hv);
  lo = as_bf16x8(lv);
}

// KS: MFMA k-steps (32 columns each) per wave; the kernel covers
// d = kGW * 32 * KS columns exactly, so no column needs a bounds check.
template <int KS, bool DENSE, bool AUX>
__global__ __launch_bounds__(kGThreads) void k_mlp_gateup_mfma(BatchedArgs a) {
  constexpr int KW = 32 * KS;  // columns per wave
  constexpr int NBMAX = kFusedMaxNeurons;

  __shared__ f32x4 red[kGW * kWaveSize];        // the waves' partial tiles
  __shared__ float l_v[NBMAX][kBTileN];         // v of each local neuron and row
  __shared__ float l_h[NBMAX][kBTileN];         // h (0 where the row masks it)
  __shared__ uint32_t l_mask[NBMAX];            // bit b: row b keeps the neuron
  __shared__ int w_cnt[kGW + 1];
  __shared__ float l_ss[kGW][kBTileN];          // the waves' sums of squares per row
  __shared__ float l_scale[kBTileN];            // per-row factor on every dot product

  const int tid = threadIdx.x;
  const int lane = tid & (kWaveSize - 1);
  const int w = __builtin_amdgcn_readfirstlane(tid / kWaveSize);
  const int B = a.B, d = a.d, m = a.m;
  const float t = a.t;
  const int G = gridDim.x, blk = blockIdx.x;
  const int n0 = (int)(((int64_t)blk * m) / G);
  const int nb = (int)(((int64_t)(blk + 1) * m) / G) - n0;
  const int T = (nb + kBTileN - 1) / kBTileN;  // tiles
  const int nops = 2 * T;                      // gate tiles, then up tiles

  const uint32_t row_bytes = (uint32_t)d * 2u;
  const uint32_t mat_bytes = (uint32_t)((uint64_t)m * row_bytes);
  const __amdgpu_buffer_rsrc_t rg = make_rsrc(a.wg, mat_bytes);
  const __amdgpu_buffer_rsrc_t ru = make_rsrc(a.wu, mat_bytes);

  for (int i = tid; i < nb; i += kGThreads) l_mask[i] = 0u;

  // This lane's operand coordinates: A row (neuron in tile) = lane % 16,
  // B column (batch row) = lane % 16, and 8 consecutive k at 8 * (lane / 16)
  // within each 32-column step.
  const int r16 = lane & 15;
  const int kb = lane >> 4;
  const int cw0 = w * KW + kb * 8;

  const uint32_t colb = (uint32_t)cw0 * 2u;  // this lane's byte offset in a weight row
  __syncthreads();  // l_mask cleared

  // Row base of this lane's neuron in operation `op` (kOOB where the row is
  // not read: past the block's neurons, past the last operation, or an up
  // row no batch row keeps).
  auto row_of = [&](int op) -> uint32_t {
    const bool up = op >= T;
    const int i = (up ? op - T : op) * kBTileN + r16;
    bool ok = op < nops && i < nb;
    if (!DENSE && up && ok) ok = l_mask[i] != 0u;
    return ok ? (uint32_t)(n0 + i) * row_bytes : kOOB;
  };

  // ---- x slice of this wave as hi/lo bf16 fragments (rows past B are
  // zero), loaded through a window of XWIN steps so that only the window's
  // fp32 values are live next to the fragments
  bf16x8 xh[KS], xl[KS];
  float ss = 0.f;  // sum of squares of this lane's x values (row r16)
  {
    constexpr int XWIN = KS < 8 ? KS : 8;
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(a.x, (uint32_t)(B * d * sizeof(float)));
    const uint32_t xrow = r16 < B ? (uint32_t)(r16 * d + cw0) * 4u : kOOB;
    u32x4 wa[XWIN], wb[XWIN];
#pragma unroll
    for (int s = 0; s < XWIN; ++s) {
      wa[s] = ld_buf16(rx, xrow + s * 128u);
      wb[s] = ld_buf16(rx, xrow + s * 128u + 16u);
    }
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      split8(wa[s % XWIN], wb[s % XWIN], xh[s], xl[s], ss);
      if (s + XWIN < KS) {
        wa[s % XWIN] = ld_buf16(rx, xrow + (s + XWIN) * 128u);
        wb[s % XWIN] = ld_buf16(rx, xrow + (s + XWIN) * 128u + 16u);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  // Per-row factor on the gate and up dot products: 1, or the RMSNorm scale
  // 1/sqrt(mean(x^2) + eps) when the block is normalised in front (the sum
  // of squares in a fixed order: lane, then the four lanes of a row in
  // ascending order, then the waves in order).
  if (a.norm) {
    float s4 = ss + __shfl_xor(ss, 16);
    s4 = s4 + __shfl_xor(s4, 32);
    if (lane < kBTileN) l_ss[w][lane] = s4;
    __syncthreads();
    if (tid < kBTileN) {
      float tot = 0.f;
#pragma unroll
      for (int ww = 0; ww < kGW; ++ww) tot += l_ss[ww][tid];
      l_scale[tid] = 1.f / sqrtf(tot / (float)d + a.eps);
    }
  } else if (tid < kBTileN) {
    l_scale[tid] = 1.f;
  }
  // The first gate tile's weights go out only now: issued before the x
  // fragments are built, they would sit in registers the fragments need,
  // and the compiler parks them elsewhere one load round trip at a time.
  u32x4 buf[KS];
  {
    const uint32_t rb = row_of(0);
#pragma unroll
    for (int s = 0; s < KS; ++s) buf[s] = ld_buf16_stream(rg, rb + colb + s * 64u);
  }
  __syncthreads();

  for (int op = 0; op < nops; ++op) {
    // The up tile of neuron tile i needs tile i's masks, known once gate
    // tile i is reduced; with a single tile that is after this operation.
    const bool defer = (T == 1 && op == 0);
    const uint32_t rbn = defer ? kOOB : row_of(op + 1);
    const __amdgpu_buffer_rsrc_t rn = (op + 1 < T) ? rg : ru;
    // Four independent accumulators (hi and lo products of even and odd
    // steps) keep the matrix core pipelined instead of waiting on one chain;
    // they are added in a fixed order at the end.  A step's buffer is
    // refilled one step later, once its products have read it.
    f32x4 ah0 = {0.f, 0.f, 0.f, 0.f}, ah1 = ah0, al0 = ah0, al1 = ah0;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const bf16x8 av = as_bf16x8(buf[s]);
      if (s & 1) {
        ah1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, xh[s], ah1, 0, 0, 0);
        al1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, xl[s], al1, 0, 0, 0);
      } else {
        ah0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, xh[s], ah0, 0, 0, 0);
        al0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, xl[s], al0, 0, 0, 0);
      }
      if (s >= 1) buf[s - 1] = ld_buf16_stream(rn, rbn + colb + (s - 1) * 64u);
      __builtin_amdgcn_sched_barrier(0);
    }
    buf[KS - 1] = ld_buf16_stream(rn, rbn + colb + (KS - 1) * 64u);
    const f32x4 acc = (ah0 + ah1) + (al0 + al1);
    red[w * kWaveSize + lane] = acc;
    __syncthreads();
    if (tid < kBTileN * kBTileN) {
      // D[i][j] sits in lane j + 16 (i / 4), register i % 4
      const int i = tid >> 4, jb = tid & 15;
      const int src = jb + 16 * (i >> 2), reg = i & 3;
      float sum = 0.f;
#pragma unroll
      for (int ww = 0; ww < kGW; ++ww) sum += red[ww * kWaveSize + src][reg];
      sum *= l_scale[jb];
      const bool up = op >= T;
      const int li = (up ? op - T : op) * kBTileN + i;
      if (li < nb && jb < B) {
        if (!up) {
          const float v = silu(sum);
          l_v[li][jb] = v;
          if (DENSE || !(fabsf(v) < t)) atomicOr(&l_mask[li], 1u << jb);
        } else {
          l_h[li][jb] = ((l_mask[li] >> jb) & 1u) ? l_v[li][jb] * sum : 0.f;
        }
      }
    }
    __syncthreads();
    if (defer) {
      const uint32_t rb = row_of(1);
#pragma unroll
      for (int s = 0; s < KS; ++s) buf[s] = ld_buf16_stream(ru, rb + colb + s * 64u);
    }
  }

  // ---- ordered compaction of the block's union-active neurons
  int base = 0;
  for (int p = 0; p * kGThreads < nb; ++p) {
    const int loc = p * kGThreads + tid;
    const uint32_t mk = loc < nb ? l_mask[loc] : 0u;
    const uint64_t bal = __ballot(mk != 0u);
    if (lane == 0) w_cnt[w] = __popcll(bal);
    __syncthreads();
    if (tid == 0) {
      int run = 0;
      for (int k = 0; k < kGW; ++k) {
        const int c = w_cnt[k];
        w_cnt[k] = run;
        run += c;
      }
      w_cnt[kGW] = run;
    }
    __syncthreads();
    if (mk) {
      const int pos = base + w_cnt[w] + __popcll(bal & ((1ull << lane) - 1ull));
      const size_t o = (size_t)n0 + pos;
      a.seg_j[o] = n0 + loc;
      a.seg_mask[o] = mk;
      for (int b = 0; b < B; ++b) {
        a.seg_h[(size_t)b * m + o] = l_h[loc][b];
        if constexpr (AUX) a.seg_v[(size_t)b * m + o] = l_v[loc][b];
      }
    }
    base += w_cnt[kGW];
    __syncthreads();
  }
  if (tid == 0) a.seg_cnt[blk] = base;
}

// Down-projection by column tiles.  Block (ct, q): columns
// [ct * kDownCols, +kDownCols), rows = the union-active neurons of K1 blocks
// [q G / NG, (q+1) G / NG) in ascending order.  Wave w owns 128 columns:
// lane = 4 * chunk + r, chunk = 8 columns, r = one of four rows loaded
// together; the quad's four row sums are added at the end (fixed order).
template <int BT>
__global__ __launch_bounds__(kBThreads) void k_mlp_down_cols(DownArgs a) {
  constexpr int RCH = kDownRowChunk;  // rows staged in LDS at a time
  constexpr int PD = 4;               // row quads in flight per lane
  __shared__ int s_j[RCH];
  __shared__ __attribute__((aligned(16))) float s_h[RCH][BT];
  __shared__ int s_pre[kFusedBlocks + 1];

  const int tid = threadIdx.x;
  const int lane = tid & (kWaveSize - 1);
  const int w = __builtin_amdgcn_readfirstlane(tid / kWaveSize);
  const int B = a.B, d = a.d, m = a.m, G = a.G, NG = a.NG;
  const int ct = blockIdx.x % a.CT, q = blockIdx.x / a.CT;
  const int g0 = (int)(((int64_t)q * G) / NG), g1 = (int)(((int64_t)(q + 1) * G) / NG);
  const int r = lane & 3, chunk = lane >> 2;
  const int col = ct * kDownCols + w * 128 + chunk * 8;
  const uint32_t colb = col < d ? (uint32_t)col * 2u : kOOB;
  const uint32_t row_bytes = (uint32_t)d * 2u;
  const __amdgpu_buffer_rsrc_t rd = make_rsrc(a.wd, (uint32_t)((uint64_t)m * row_bytes));

  // row offsets of the group's K1 blocks
  if (tid == 0) {
    int run = 0;
    for (int g = g0; g < g1; ++g) {
      s_pre[g - g0] = run;
      run += a.seg_cnt[g];
    }
    s_pre[g1 - g0] = run;
  }
  __syncthreads();
  const int R = s_pre[g1 - g0];

  float acc[BT][8];
#pragma unroll
  for (int b = 0; b < BT; ++b)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[b][e] = 0.f;

  for (int c0 = 0; c0 < R; c0 += RCH) {
    const int nr = min(RCH, R - c0);
    for (int e = tid; e < nr; e += kBThreads) {
      // row c0 + e lives in the segment of the K1 block whose range holds it
      const int re = c0 + e;
      int gi = 0;
      while (s_pre[gi + 1] <= re) ++gi;
      const size_t o = (size_t)(((int64_t)(g0 + gi) * m) / G) + (re - s_pre[gi]);
      s_j[e] = a.seg_j[o];
#pragma unroll
      for (int b = 0; b < BT; ++b) s_h[e][b] = b < B ? a.seg_h[(size_t)b * m + o] : 0.f;
    }
    __syncthreads();
    const int nq = (nr + 3) >> 2;  // row quads
    auto ld = [&](int qd) -> u32x4 {
      const int e = qd * 4 + r;
      return ld_buf16_stream(rd, (qd < nq && e < nr) ? (uint32_t)s_j[e] * row_bytes + colb : kOOB);
    };
    auto fma_row = [&](const u32x4& v, int qd) {
      const int e = qd * 4 + r;
      if (qd < nq && e < nr) {
        float wf[8];
        widen<wbf16>(v, wf);
        float hv[BT];
#pragma unroll
        for (int b4 = 0; b4 < BT; b4 += 4) {
          const f32x4 h4 = *reinterpret_cast<const f32x4*>(&s_h[e][b4]);
          hv[b4] = h4.x;
          hv[b4 + 1] = h4.y;
          hv[b4 + 2] = h4.z;
          hv[b4 + 3] = h4.w;
        }
#pragma unroll
        for (int b = 0; b < BT; ++b)
#pragma unroll
          for (int k = 0; k < 8; ++k) acc[b][k] = fmaf(hv[b], wf[k], acc[b][k]);
      }
    };
    u32x4 pb[PD];
#pragma unroll
    for (int p = 0; p < PD; ++p) pb[p] = ld(p);
    for (int qd = 0; qd < nq; qd += PD) {
#pragma unroll
      for (int p = 0; p < PD; ++p) {
        const u32x4 v = pb[p];
        pb[p] = ld(qd + p + PD);
        fma_row(v, qd + p);
        // one row quad at a time: its h values and products are not hoisted
        // next to the next quad's
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    __syncthreads();  // s_j / s_h are rewritten by the next chunk
  }

  // sum the quad's four rows (lanes 4 chunk + 0..3), then lane r == 0
  // writes this group's partial y for its 8 columns
  float* part = a.partial + (size_t)q * B * d;
#pragma unroll
  for (int b = 0; b < BT; ++b) {
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      float v = acc[b][k];
      v += dpp_f32<0xb1>(v);  // quad_perm [1,0,3,2]
      v += dpp_f32<0x4e>(v);  // quad_perm [2,3,0,1]
      acc[b][k] = v;
    }
  }
  if (r == 0 && col < d) {
#pragma unroll
    for (int b = 0; b < BT; ++b) {
      if (b < B) {
        f32x4 o0 = {acc[b][0], acc[b][1], acc[b][2], acc[b][3]};
        f32x4 o1 = {acc[b][4], acc[b][5], acc[b][6], acc[b][7]};
        *reinterpret_cast<f32x4*>(part + (size_t)b * d + col) = o0;
        *reinterpret_cast<f32x4*>(part + (size_t)b * d + col + 4) = o1;
      }
    }
  }
}

template <bool DENSE, bool AUX>
static hipError_t launch_gateup_t(int ks, const BatchedArgs& a, int G, hipStream_t s) {
  const dim3 grid(G), block(kGThreads);
  KernelTimer timer(DENSE ? "mlp_gateup_dense" : "mlp_gateup_cats", s);
  switch (ks) {
#define CATS_KS(K)                                                                                   \
  case K:                                                                                            \
    hipExtLaunchKernelGGL((k_mlp_gateup_mfma<K, DENSE, AUX>), grid, block, 0, s, timer.start(),       \
                          timer.stop(), 0, a);                                                       \
    break;
    CATS_KS(1)
    CATS_KS(2)
    CATS_KS(4)
    CATS_KS(6)
    CATS_KS(8)
#undef CATS_KS
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

int batched_ks(int d) {
  if (d % (kGW * 32) != 0) return 0;
  const int ks = d / (kGW * 32);
  // instantiated widths; wider rows do not fit the register-resident x slice
  return (ks == 1 || ks == 2 || ks == 4 || ks == 6 || ks == 8) ? ks : 0;
}

hipError_t launch_gateup(bool dense, bool aux, const BatchedArgs& a, int G, hipStream_t s) {
  const int ks = batched_ks(a.d);
  if (dense) return launch_gateup_t<true, false>(ks, a, G, s);
  return aux ? launch_gateup_t<false, true>(ks, a, G, s) : launch_gateup_t<false, false>(ks, a, G, s);
}

hipError_t launch_down_cols(const DownArgs& a, hipStream_t s) {
  const dim3 grid(a.CT * a.NG), block(kBThreads);
  KernelTimer timer("mlp_down_cols", s);
  if (a.B <= 4)
    hipExtLaunchKernelGGL(k_mlp_down_cols<4>, grid, block, 0, s, timer.start(), timer.stop(), 0, a);
  else if (a.B <= 8)
    hipExtLaunchKernelGGL(k_mlp_down_cols<8>, grid, block, 0, s, timer.start(), timer.stop(), 0, a);
  else
    hipExtLaunchKernelGGL(k_mlp_down_cols<16>, grid, block, 0, s, timer.start(), timer.stop(), 0, a);
  return hipGetLastError();
}

}  // namespace cats
