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
// Kernel 2 (k_mlp_down_mfma): block (column tile, neuron group) accumulates
// h_b W_down[j, cols] over the group's union-active rows on the matrix
// cores and writes one partial y per neuron group; k_mlp_reduce sums the
// groups in order.
#include "device.hpp"
#include "internal.hpp"

namespace cats {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short v4i16 __attribute__((ext_vector_type(4)));

constexpr int kBW = kBatchedWaves;
constexpr int kBThreads = kBW * kWaveSize;
constexpr int kGW = kGateUpWaves;
constexpr int kGThreads = kGW * kWaveSize;
constexpr int kBTileN = 16;  // neurons per MFMA tile (and batch columns)

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

// Weight steps a wave keeps in flight: a whole tile up to eight steps; at
// ten (d = 5120) the x slice and a whole tile would take 120 of the 128
// registers a wave has at four waves per SIMD, so the loads run five steps
// ahead, with the lo fragments of steps 6..9 kept in LDS (XLR below).
template <int KS>
constexpr int gateup_window() { return KS <= 8 ? KS : 5; }

// KS: MFMA k-steps (32 columns each) per wave; the kernel covers
// d = kGW * 32 * KS columns exactly, so no column needs a bounds check.
template <int KS, bool DENSE, bool AUX>
__global__ __launch_bounds__(kGThreads) void k_mlp_gateup_mfma(BatchedArgs a) {
  constexpr int KW = 32 * KS;  // columns per wave
  constexpr int WIN = gateup_window<KS>();
  static_assert(KS % WIN == 0, "a tile's steps must fill the window evenly");
  constexpr int NBMAX = kFusedMaxNeurons;

  __shared__ f32x4 red[kGW * kWaveSize];        // the waves' partial tiles
  __shared__ float l_v[NBMAX][kBTileN];         // v of each local neuron and row
  __shared__ float l_h[NBMAX][kBTileN];         // h (0 where the row masks it)
  __shared__ uint32_t l_mask[NBMAX];            // bit b: row b keeps the neuron
  __shared__ int w_cnt[kGW + 1];
  __shared__ float l_ss[kGW][kBTileN];          // the waves' sums of squares per row
  __shared__ float l_scale[kBTileN];            // per-row factor on every dot product
  // x-lo fragments of the steps from XLR on live in LDS, one slot per
  // thread and step (read back by the same thread, so no barrier is needed)
  constexpr int XLR = KS <= 8 ? KS : 6;
  __shared__ bf16x8 l_xl[(KS - XLR) > 0 ? (KS - XLR) * kGThreads : 1];

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
      if (s >= XLR) l_xl[(s - XLR) * kGThreads + tid] = xl[s];
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
  // Weight loads here are ordinary cached loads, not the non-temporal ones of
  // the other weight streams: one load instruction reads 64 bytes of each
  // of 16 rows, half of a 128-byte line, and the line's other half comes
  // with the next step; with the non-temporal hint the line was often gone
  // before its second half was asked for (the kernel then read 21% more
  // than the weights at d = 5120, and the layer ran 4-8% slower).
  // The first gate tile's weights go out only now: issued before the x
  // fragments are built, they would sit in registers the fragments need,
  // and the compiler parks them elsewhere one load round trip at a time.
  // buf[s % WIN] holds step s of the current tile; the loads stream over
  // (tile, step) pairs WIN steps ahead of the products, into the next tile
  // once the current one's steps are all out.
  u32x4 buf[WIN];
  uint32_t rbc = row_of(0);  // row base of the current operation
  {
#pragma unroll
    for (int s = 0; s < WIN; ++s) buf[s] = ld_buf16(rg, rbc + colb + s * 64u);
  }
  __syncthreads();

  for (int op = 0; op < nops; ++op) {
    // The up tile of neuron tile i needs tile i's masks, known once gate
    // tile i is reduced; with a single tile that is after this operation.
    const bool defer = (T == 1 && op == 0);
    const uint32_t rbn = defer ? kOOB : row_of(op + 1);
    const __amdgpu_buffer_rsrc_t rc = op < T ? rg : ru;
    const __amdgpu_buffer_rsrc_t rn = (op + 1 < T) ? rg : ru;
    // the load WIN steps after step f - WIN: step f of this tile, or step
    // f - KS of the next
    auto ld_ahead = [&](int f) -> u32x4 {
      return f < KS ? ld_buf16(rc, rbc + colb + f * 64u)
                    : ld_buf16(rn, rbn + colb + (f - KS) * 64u);
    };
    // Four independent accumulators (hi and lo products of even and odd
    // steps) keep the matrix core pipelined instead of waiting on one chain;
    // they are added in a fixed order at the end.  A step's buffer is
    // refilled one step later, once its products have read it.
    f32x4 ah0 = {0.f, 0.f, 0.f, 0.f}, ah1 = ah0, al0 = ah0, al1 = ah0;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const bf16x8 av = as_bf16x8(buf[s % WIN]);
      if (s & 1) {
        ah1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, xh[s], ah1, 0, 0, 0);
        al1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, s < XLR ? xl[s] : l_xl[(s - XLR) * kGThreads + tid], al1, 0, 0, 0);
      } else {
        ah0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, xh[s], ah0, 0, 0, 0);
        al0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, s < XLR ? xl[s] : l_xl[(s - XLR) * kGThreads + tid], al0, 0, 0, 0);
      }
      if (s >= 1) buf[(s - 1) % WIN] = ld_ahead(s - 1 + WIN);
      __builtin_amdgcn_sched_barrier(0);
    }
    buf[(KS - 1) % WIN] = ld_ahead(KS - 1 + WIN);
    rbc = rbn;
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
      rbc = row_of(1);
#pragma unroll
      for (int s = 0; s < WIN; ++s) buf[s] = ld_buf16(ru, rbc + colb + s * 64u);
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
  // the rest of the block's segment names no neuron: zero row masks, so a
  // list entry is exactly an entry with its row's bit set
  for (int i = base + tid; i < nb; i += kGThreads) a.seg_mask[n0 + i] = 0u;
}

// Down-projection on the matrix cores (5..16 rows). Block (ct, q) owns
// columns [ct * kDownCols, +kDownCols) and the union-active rows of neuron
// group q; wave w owns 128 of the columns, eight MFMA tiles of 16. The
// contraction runs over neurons:
//  D[c][b] += sum_k W_down[j_k][c] * h[b][j_k]
// with A[c][k] = W_down[j_k][c] (16 columns x 32 rows) and B[k][b] =
// h[b][j_k] (32 rows x 16 batch rows). A lane's A operand is eight rows of
// one column, which W_down's row-major layout does not hold contiguously, so
// each wave streams its 32-row x 128-column slice of a step into its own LDS
// region (one 256-byte run per row) and reads the operand back column-wise
// with gfx950's transposing LDS reads. h enters as bf16 hi + lo (as x does in
// the gate/up kernel: 16 of its 24 mantissa bits, products exact, fp32
// accumulation), staged per block as [batch row][staged row].
constexpr int kDmRows = 32;                 // rows per k-step
constexpr int kDmChunk = 256;               // rows staged per block at a time
constexpr int kDmPitch = 128 * 2 + 8;       // LDS bytes per row of a wave's slice (8 pad: q groups 16 banks apart)
constexpr int kDmHPitch = kDmChunk + 8;     // bf16 elements per batch row of the staged h

__global__ __launch_bounds__(kBThreads) void k_mlp_down_mfma(DownArgs a) {
  __shared__ __attribute__((aligned(16))) int s_j[kDmChunk];
  __shared__ __attribute__((aligned(16))) uint16_t s_hh[kBTileN * kDmHPitch];
  __shared__ __attribute__((aligned(16))) uint16_t s_hl[kBTileN * kDmHPitch];
  __shared__ __attribute__((aligned(16))) uint8_t s_w[kBW * kDmRows * kDmPitch];
  __shared__ int s_pre[kFusedBlocks + 1];

  const int tid = threadIdx.x;
  const int lane = tid & (kWaveSize - 1);
  const int w = __builtin_amdgcn_readfirstlane(tid / kWaveSize);
  const int B = a.B, d = a.d, m = a.m, G = a.G, NG = a.NG;
  const int ct = blockIdx.x % a.CT, q = blockIdx.x / a.CT;
  const int g0 = (int)(((int64_t)q * G) / NG), g1 = (int)(((int64_t)(q + 1) * G) / NG);
  const int col0 = ct * kDownCols + w * 128;  // this wave's first column
  const uint32_t row_bytes = (uint32_t)d * 2u;
  const __amdgpu_buffer_rsrc_t rd = make_rsrc(a.wd, (uint32_t)((uint64_t)m * row_bytes));
  uint8_t* wreg = s_w + (size_t)w * kDmRows * kDmPitch;
  const __amdgpu_buffer_rsrc_t rh = make_rsrc(a.seg_h, (uint32_t)((size_t)B * m * sizeof(float)));

  // streaming a step: load p (0..7) covers rows 4p + lane / 16, 16 bytes
  // (8 columns) per lane, one 256-byte run per row
  const int lr = lane >> 4, lc = lane & 15;
  const int lcol = col0 + lc * 8;
  const uint32_t lcolb = lcol < d ? (uint32_t)lcol * 2u : kOOB;
  // operands: A lane = column i + 16 kq, B lane = batch row jb + 16 kq;
  // both hold the eight rows 8 kq .. 8 kq + 7 of the step
  const int oi = lane & 15, kq = lane >> 4;

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

  f32x4 acch[8], accl[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    acch[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    accl[t] = acch[t];
  }

  for (int c0 = 0; c0 < R; c0 += kDmChunk) {
    const int nr = min(kDmChunk, R - c0);
    const int nsteps = (nr + kDmRows - 1) / kDmRows;
    // stage the chunk's rows: index, and h as bf16 hi / lo by batch row
    // (rows past nr and batch rows past B are zero).  A row's sixteen h
    // loads are unconditional buffer loads (out of range where absent), so
    // they are all in flight at once.
    for (int e = tid; e < nsteps * kDmRows; e += kBThreads) {
      int jrow = -1;
      uint32_t o = 0;
      if (e < nr) {
        const int re = c0 + e;
        int gi = 0;
        while (s_pre[gi + 1] <= re) ++gi;
        o = (uint32_t)(((int64_t)(g0 + gi) * m) / G) + (uint32_t)(re - s_pre[gi]);
        jrow = a.seg_j[o];
      }
      s_j[e] = jrow;
      uint32_t hb[kBTileN];
#pragma unroll
      for (int b = 0; b < kBTileN; ++b)
        hb[b] = __builtin_amdgcn_raw_buffer_load_b32(rh, (jrow >= 0 && b < B) ? ((uint32_t)b * m + o) * 4u : kOOB, 0, 0);
#pragma unroll
      for (int b = 0; b < kBTileN; ++b) {
        const float h = __uint_as_float(hb[b]);
        const uint32_t hi = bf16_bits(h);
        const uint32_t lo = bf16_bits(h - __uint_as_float(hi << 16));
        s_hh[b * kDmHPitch + e] = (uint16_t)hi;
        s_hl[b * kDmHPitch + e] = (uint16_t)lo;
      }
    }
    __syncthreads();

    // a lane's rows of a step are 8 lr .. 8 lr + 7 (load p takes row
    // 8 lr + p), so their indices come from LDS in two 16-byte reads
    auto load_step = [&](u32x4(&buf)[8], int st) {
      int jr[8];
      if (st < nsteps) {
        const int4 ja = *reinterpret_cast<const int4*>(s_j + st * kDmRows + 8 * lr);
        const int4 jb = *reinterpret_cast<const int4*>(s_j + st * kDmRows + 8 * lr + 4);
        jr[0] = ja.x; jr[1] = ja.y; jr[2] = ja.z; jr[3] = ja.w;
        jr[4] = jb.x; jr[5] = jb.y; jr[6] = jb.z; jr[7] = jb.w;
      } else {
#pragma unroll
        for (int p = 0; p < 8; ++p) jr[p] = -1;
      }
#pragma unroll
      for (int p = 0; p < 8; ++p)
        buf[p] = ld_buf16_stream(rd, jr[p] >= 0 ? (uint32_t)jr[p] * row_bytes + lcolb : kOOB);
    };
    // this wave's slice of a step into its LDS region (the previous step's
    // reads by this wave come first: LDS operations of a wave run in order)
    auto write_step = [&](const u32x4(&buf)[8]) {
#pragma unroll
      for (int p = 0; p < 8; ++p) {
        uint8_t* dst = wreg + (8 * lr + p) * kDmPitch + lc * 16;
        reinterpret_cast<uint2*>(dst)[0] = uint2{buf[p].x, buf[p].y};
        reinterpret_cast<uint2*>(dst)[1] = uint2{buf[p].z, buf[p].w};
      }
    };
    auto compute_step = [&](int st) {
      const int e0 = st * kDmRows + 8 * kq;
      const u32x4 bh = *reinterpret_cast<const u32x4*>(s_hh + oi * kDmHPitch + e0);
      const u32x4 bl = *reinterpret_cast<const u32x4*>(s_hl + oi * kDmHPitch + e0);
      const bf16x8 bhv = as_bf16x8(bh), blv = as_bf16x8(bl);
      // A operand by transposing reads: in each 16-lane group, lane r
      // names four consecutive 16-bit values (row 8 kq + r / 4, columns
      // 4 (r % 4) .. + 3 of the tile) and lane i receives value i % 4 of the
      // rows named by lanes i / 4 + 4 k, k = 0..3: column i of four
      // consecutive rows.  Two reads give the eight rows of a step's half.
      const int ar = 8 * kq + (oi >> 2);
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const uint8_t* src = wreg + ar * kDmPitch + (t * 16 + 4 * (oi & 3)) * 2;
        const v4i16 r0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16*)src);
        const v4i16 r1 =
            __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16*)(src + 4 * kDmPitch));
        const uint2 w0 = __builtin_bit_cast(uint2, r0), w1 = __builtin_bit_cast(uint2, r1);
        const bf16x8 av = as_bf16x8(u32x4{w0.x, w0.y, w1.x, w1.y});
        acch[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bhv, acch[t], 0, 0, 0);
        accl[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, blv, accl[t], 0, 0, 0);
      }
    };
    u32x4 rA[8], rB[8];
    load_step(rA, 0);
    load_step(rB, 1);
    for (int st = 0; st < nsteps; st += 2) {
      write_step(rA);
      load_step(rA, st + 2);
      compute_step(st);
      if (st + 1 < nsteps) {
        write_step(rB);
        load_step(rB, st + 3);
        compute_step(st + 1);
      }
    }
    __syncthreads();  // s_j / s_hh / s_hl are rewritten by the next chunk
  }

  // D[i][j] sits in lane j + 16 (i / 4), register i % 4: batch row
  // jb = lane % 16, columns 4 (lane / 16) .. + 3 of each tile
  const int jb = lane & 15, c4 = (lane >> 4) * 4;
  if (jb < B) {
    float* part = a.partial + ((size_t)q * B + jb) * d;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const int c = col0 + t * 16 + c4;
      if (c < d) *reinterpret_cast<f32x4*>(part + c) = acch[t] + accl[t];
    }
  }
}

hipError_t launch_down_mfma(const DownArgs& a, hipStream_t s) {
  const dim3 grid(a.CT * a.NG), block(kBThreads);
  KernelTimer timer("mlp_down_mfma", s);
  hipExtLaunchKernelGGL(k_mlp_down_mfma, grid, block, 0, s, timer.start(), timer.stop(), 0, a);
  return hipGetLastError();
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
    CATS_KS(10)
#undef CATS_KS
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

int batched_ks(int d) {
  if (d % (kGW * 32) != 0) return 0;
  const int ks = d / (kGW * 32);
  // instantiated widths; wider rows do not fit the register-resident x slice
  return (ks == 1 || ks == 2 || ks == 4 || ks == 6 || ks == 8 || ks == 10) ? ks : 0;
}

hipError_t launch_gateup(bool dense, bool aux, const BatchedArgs& a, int G, hipStream_t s) {
  const int ks = batched_ks(a.d);
  if (dense) return launch_gateup_t<true, false>(ks, a, G, s);
  return aux ? launch_gateup_t<false, true>(ks, a, G, s) : launch_gateup_t<false, false>(ks, a, G, s);
}



}  // namespace cats
