// CATS on the input of a linear layer (Appendix B wraps each attention
// block's input in CATS_t, so its Q/K/V projections take a sparse input):
//   y_b = residual_b + CATS_t(x_b) W,  CATS_t(z) = z where |z| >= t, else 0
// with W [d x n] channel-major (row i = input channel i, n contiguous
// weights).  Only the rows of the channels some batch row keeps are read.
//
// One kernel.  Block (ct, q) owns output columns [32 ct, 32 ct + 32) and
// input-channel group q of NG.  It compacts the group's kept channels in
// LDS (ascending; each row's mask bit; the kept value, 0 for a row that
// drops the channel), then its 8 waves stream the kept rows' 64-byte column
// slices, sixteen rows per wave load (four lanes per row, 8 columns each),
// and meet in LDS.  A round of compaction covers up to 4096 channels (one
// round for a 4096-wide input up to 4 rows).  Wide outputs (n >= 4096 or so) give enough column tiles
// for one group (NG = 1): y is written directly and consecutive column tiles
// run on one XCD, so its L2 serves both halves of each 128-byte line.
// Narrower outputs split the channels into NG > 1 groups: the blocks of a
// column tile leave device-coherent partial sums and take a ticket; the
// last of them adds the NG partials in group order (deterministic), adds
// the residual and writes y.  No block waits for another: the ticket (ticket.hpp) is a count in a
// word tagged with the call's epoch, so leftovers of earlier calls in the
// workspace never count.
#include "device.hpp"
#include "internal.hpp"
#include "scan.hpp"
#include "ticket.hpp"

namespace cats {

constexpr int kSW = 8;
constexpr int kSThreads = kSW * kWaveSize;

// Channels compacted per round (the LDS holds their indices and values):
// the whole input of a 4096-wide layer in one round up to 4 rows.
template <int BT> struct SparseChunk { static constexpr int value = BT <= 4 ? 4096 : (BT <= 8 ? 2048 : 1024); };

template <int BT>
__global__ __launch_bounds__(kSThreads) void k_sparse_input(SparseInputArgs a) {
  constexpr int CHUNK = SparseChunk<BT>::value;
  constexpr int CPT = CHUNK / kSThreads;  // consecutive channels per thread
  __shared__ int s_j[CHUNK];
  __shared__ __attribute__((aligned(16))) float s_h[CHUNK][BT];
  __shared__ __attribute__((aligned(16))) float red[kSW][BT][kSparseCols];
  __shared__ int w_tot[kSW];
  __shared__ int s_last;

  const int tid = threadIdx.x;
  const int lane = tid & (kWaveSize - 1);
  const int w = __builtin_amdgcn_readfirstlane(tid / kWaveSize);
  const int B = a.B, d = a.d, n = a.n, NG = a.NG, CT = a.CT;
  // Block b runs on XCD b mod 8: with one group and CT a multiple of 8,
  // XCD x takes the consecutive column tiles [x CT/8, (x+1) CT/8).
  int ct, q;
  if (NG == 1 && CT % 8 == 0) {
    ct = (blockIdx.x % 8) * (CT / 8) + blockIdx.x / 8;
    q = 0;
  } else {
    ct = blockIdx.x % CT;
    q = blockIdx.x / CT;
  }
  // (the ticket word is read now, so that arriving costs one atomic)
  const unsigned long long peek = (NG > 1 && tid == 0) ? ticket_peek(a.tickets + ct) : 0ull;
  const int c0 = (int)(((int64_t)q * d) / NG), c1 = (int)(((int64_t)(q + 1) * d) / NG);
  // A wave load covers RPL rows of the block's columns: LPR consecutive
  // lanes per row, 8 columns (16 bytes) each.
  constexpr int LPR = kSparseCols / 8;
  constexpr int RPL = kWaveSize / LPR;
  const int r = lane / LPR, chunk = lane % LPR;
  const int col = ct * kSparseCols + chunk * 8;
  const uint32_t colb = col < n ? (uint32_t)col * 2u : kOOB;
  const uint32_t row_bytes = (uint32_t)n * 2u;
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(a.w, (uint32_t)((uint64_t)d * row_bytes));
  const bool seg_writer = a.aux && ct == 0;

  float acc[BT][8];
#pragma unroll
  for (int bq = 0; bq < BT; ++bq)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[bq][e] = 0.f;

  int seg_base = 0;  // kept channels of this group before the current round
  for (int cb = c0; cb < c1; cb += CHUNK) {
    const int nc = min(CHUNK, c1 - cb);
    // ---- ordered compaction of channels [cb, cb + nc): thread t takes
    // the CPT consecutive channels from cb + CPT t, all its x values are
    // loaded at once, and one scan (within the wave, then over the waves)
    // places its kept channels
    const int cl0 = tid * CPT;
    float xv[CPT][BT];
#pragma unroll
    for (int u = 0; u < CPT; ++u)
#pragma unroll
      for (int bq = 0; bq < BT; ++bq)
        xv[u][bq] = (bq < B && cl0 + u < nc) ? a.x[(size_t)bq * d + cb + cl0 + u] : 0.f;
    uint32_t mk[CPT];
    int mine = 0;
#pragma unroll
    for (int u = 0; u < CPT; ++u) {
      mk[u] = 0;
#pragma unroll
      for (int bq = 0; bq < BT; ++bq)
        if (bq < B && cl0 + u < nc && !(fabsf(xv[u][bq]) < a.t)) mk[u] |= 1u << bq;
      mine += mk[u] != 0u;
    }
    const int incl = (int)wave_incl_scan((uint32_t)mine);  // inclusive scan over the wave's lanes
    if (lane == kWaveSize - 1) w_tot[w] = incl;
    __syncthreads();
    int pos = incl - mine;
    int kept = 0;
    for (int k = 0; k < kSW; ++k) {
      const int tk = w_tot[k];
      if (k < w) pos += tk;
      kept += tk;
    }
#pragma unroll
    for (int u = 0; u < CPT; ++u) {
      if (mk[u]) {
        s_j[pos] = cb + cl0 + u;
#pragma unroll
        for (int bq = 0; bq < BT; ++bq) s_h[pos][bq] = ((mk[u] >> bq) & 1u) ? xv[u][bq] : 0.f;
        if (seg_writer) {
          const size_t o = (size_t)c0 + seg_base + pos;
          a.seg_j[o] = cb + cl0 + u;
          a.seg_mask[o] = mk[u];
          for (int bq = 0; bq < B; ++bq) {
            const float v = ((mk[u] >> bq) & 1u) ? xv[u][bq] : 0.f;
            a.seg_h[(size_t)bq * d + o] = v;
            a.seg_v[(size_t)bq * d + o] = v;
          }
        }
        ++pos;
      }
    }
    __syncthreads();

    // ---- stream the kept rows: wave w takes row groups (RPL rows each)
    // w, w + 8, ...
    const int nq = (kept + RPL - 1) / RPL;
    auto ld = [&](int qd) -> u32x4 {
      const int e = qd * RPL + r;
      return ld_buf16_stream(rw, (qd < nq && e < kept) ? (uint32_t)s_j[e] * row_bytes + colb : kOOB);
    };
    auto fma_row = [&](const u32x4& v, int qd) {
      const int e = qd * RPL + r;
      if (qd < nq && e < kept) {
        float wf[8];
        widen<wbf16>(v, wf);
        if constexpr (BT == 1) {
          const float hv = s_h[e][0];
#pragma unroll
          for (int k = 0; k < 8; ++k) acc[0][k] = fmaf(hv, wf[k], acc[0][k]);
        } else {
#pragma unroll
          for (int b4 = 0; b4 < BT; b4 += 4) {
            const f32x4 h4 = *reinterpret_cast<const f32x4*>(&s_h[e][b4]);
            const float hv[4] = {h4.x, h4.y, h4.z, h4.w};
#pragma unroll
            for (int bb = 0; bb < 4; ++bb)
#pragma unroll
              for (int k = 0; k < 8; ++k) acc[b4 + bb][k] = fmaf(hv[bb], wf[k], acc[b4 + bb][k]);
          }
        }
      }
    };
    // row groups in flight per wave: as many as the registers allow, since
    // a block streams its rows in few round trips
    constexpr int PD = BT <= 4 ? 12 : (BT <= 8 ? 8 : 4);
    u32x4 pb[PD];
#pragma unroll
    for (int p = 0; p < PD; ++p) pb[p] = ld(w + p * kSW);
    for (int qd = w; qd < nq; qd += PD * kSW) {
#pragma unroll
      for (int p = 0; p < PD; ++p) {
        const u32x4 v = pb[p];
        pb[p] = ld(qd + (p + PD) * kSW);
        fma_row(v, qd + p * kSW);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    seg_base += kept;
    __syncthreads();  // s_j / s_h are rewritten by the next round
  }
  if (seg_writer) {
    // the rest of the group's segment holds no channel: zero row masks, so
    // a list entry is exactly an entry with its row's bit set
    for (int e = c0 + seg_base + tid; e < c1; e += kSThreads) a.seg_mask[e] = 0u;
    if (tid == 0) a.seg_cnt[q] = seg_base;
  }

  // ---- the wave's RPL rows (lanes LPR r + chunk: rotations within each
  // row of 16 lanes for strides below 16, swaps across rows above), then
  // the waves, in a fixed order
#pragma unroll
  for (int b = 0; b < BT; ++b)
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      float v = acc[b][k];
      if constexpr (LPR <= 4) v += dpp_f32<0x124>(v);  // row_ror:4
      if constexpr (LPR <= 8) v += dpp_f32<0x128>(v);  // row_ror:8
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      acc[b][k] = v;
    }
  if (r == 0) {
#pragma unroll
    for (int b = 0; b < BT; ++b) {
      *reinterpret_cast<f32x4*>(&red[w][b][chunk * 8]) = f32x4{acc[b][0], acc[b][1], acc[b][2], acc[b][3]};
      *reinterpret_cast<f32x4*>(&red[w][b][chunk * 8 + 4]) = f32x4{acc[b][4], acc[b][5], acc[b][6], acc[b][7]};
    }
  }
  __syncthreads();

  // item (b, c4): batch row b, float4 column c4 of this block's 128 columns
  constexpr int C4 = kSparseCols / 4;
  const int ib = tid / C4, ic4 = tid % C4;
  const int ocol = ct * kSparseCols + ic4 * 4;
  const bool item = ib < B && ocol < n;
  f32x4 sum = {0.f, 0.f, 0.f, 0.f};
  if (item) {
#pragma unroll
    for (int ww = 0; ww < kSW; ++ww) sum += *reinterpret_cast<const f32x4*>(&red[ww][ib][ic4 * 4]);
  }
  auto finish = [&](f32x4 s) {
    if (a.residual) s = *reinterpret_cast<const f32x4*>(a.residual + (size_t)ib * n + ocol) + s;
    *reinterpret_cast<f32x4*>(a.y + (size_t)ib * n + ocol) = s;
  };
  if (NG == 1) {
    if (item) finish(sum);
    return;
  }

  // ---- partial of this group, then the ticket of the column tile
  const __amdgpu_buffer_rsrc_t rp = make_rsrc(a.partial, (uint32_t)((size_t)NG * B * n * sizeof(float)));
  if (item) {
    const u32x4 o = {__float_as_uint(sum.x), __float_as_uint(sum.y), __float_as_uint(sum.z), __float_as_uint(sum.w)};
    st_buf16_coherent(rp, (uint32_t)((((size_t)q * B + ib) * n + ocol) * sizeof(float)), o);
  }
  __builtin_amdgcn_s_waitcnt(0);  // this thread's partial store has completed
  __syncthreads();
  if (tid == 0) s_last = take_ticket(a.tickets + ct, a.epoch, (uint32_t)NG, peek);
  __syncthreads();
  if (!s_last || !item) return;
  // the last block of the tile: every group's partial, in group order
  f32x4 tot = {0.f, 0.f, 0.f, 0.f};
  for (int g0 = 0; g0 < NG; g0 += 8) {
    u32x4 v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k)
      v[k] = ld_buf16_coherent(rp, g0 + k < NG ? (uint32_t)((((size_t)(g0 + k) * B + ib) * n + ocol) * sizeof(float)) : kOOB);
#pragma unroll
    for (int k = 0; k < 8; ++k)
      if (g0 + k < NG) tot += f32x4{__uint_as_float(v[k].x), __uint_as_float(v[k].y), __uint_as_float(v[k].z), __uint_as_float(v[k].w)};
  }
  finish(tot);
}

hipError_t launch_sparse_input(const SparseInputArgs& a, hipStream_t s) {
  const dim3 grid(a.CT * a.NG), block(kSThreads);
  KernelTimer timer("sparse_input", s);
  if (a.B == 1)
    hipExtLaunchKernelGGL(k_sparse_input<1>, grid, block, 0, s, timer.start(), timer.stop(), 0, a);
  else if (a.B <= 4)
    hipExtLaunchKernelGGL(k_sparse_input<4>, grid, block, 0, s, timer.start(), timer.stop(), 0, a);
  else if (a.B <= 8)
    hipExtLaunchKernelGGL(k_sparse_input<8>, grid, block, 0, s, timer.start(), timer.stop(), 0, a);
  else
    hipExtLaunchKernelGGL(k_sparse_input<16>, grid, block, 0, s, timer.start(), timer.stop(), 0, a);
  return hipGetLastError();
}

}  // namespace cats
