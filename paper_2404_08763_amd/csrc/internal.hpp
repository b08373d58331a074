// Host-side interface between the C ABI (cats_api.cpp) and the kernel
// translation units.  Every launcher assumes its arguments were validated.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "fused_params.hpp"

namespace cats {

// Batched path (bf16 weights, kBatchedMinRows..16 rows): gate and up on
// the matrix cores, then the down-projection by column tiles.  Below 5 rows
// the fused kernel is faster (one pass of its vector-ALU dot products over
// the staged rows); from 5 rows its dot products cost more than the
// matrix-core path, and above 8 it would need a second pass over the weights.
#ifndef CATS_BATCHED_MIN_ROWS
#define CATS_BATCHED_MIN_ROWS 5
#endif
constexpr int kBatchedMinRows = CATS_BATCHED_MIN_ROWS;
constexpr int kBatchedWaves = 8;   // the down-projection kernel's waves per block
// Waves of the gate/up kernel: each holds 1/16 of x's columns as matrix-core
// operands, so at d = 4096 the operands and a tile of weights in flight fit
// the 128 registers a wave has at four waves per SIMD.
constexpr int kGateUpWaves = 16;
constexpr int kDownCols = kBatchedWaves * 128;  // columns of a down-projection block
constexpr int kDownRowChunk = 1024;             // rows a down block stages in LDS at once

struct BatchedArgs {
  const void* wg;      // [m x d] W_gate^T (bf16)
  const void* wu;      // [m x d] W_up^T
  const float* x;      // [B x d]
  int B, d, m;
  float t;
  int norm;            // RMSNorm x (unit gain) before the block
  float eps;           // its epsilon
  int* seg_j;          // [m] union-active neurons, per block from its first neuron
  uint32_t* seg_mask;  // [m] their row masks
  float* seg_v;        // [B x m] (aux only)
  float* seg_h;        // [B x m]
  int* seg_cnt;        // [G]
};

struct DownArgs {
  const void* wd;      // [m x d] W_down (bf16)
  float* partial;      // [NG x B x d]
  const int* seg_j;
  const float* seg_h;
  const int* seg_cnt;
  int B, d, m;
  int G;               // blocks of the gate/up kernel (segments)
  int NG;              // neuron groups (partials)
  int CT;              // column tiles
};

// Rows of one call (the C ABI's CATS_MAX_BATCH).
constexpr int kMaxRows = 16;

// CATS on a layer's input (k_sparse_input): output columns per block (a
// 256-byte slice of each weight row; 32 and 64 are also valid).
constexpr int kSparseCols = 128;

struct SparseInputArgs {
  const void* w;            // [d x n] bf16, row i = input channel i
  const float* x;           // [B x d]
  const float* residual;    // [B x n] or null
  float* y;                 // [B x n]
  int B, d, n;
  float t;
  int NG, CT;               // input-channel groups, column tiles
  float* partial;           // [NG x B x n] (NG > 1)
  unsigned long long* tickets;  // [CT] epoch-tagged arrival counts
  uint32_t epoch;           // this call's tag (never 0)
  int aux;                  // blocks of column tile 0 write the segments
  int* seg_j;               // [d] kept channels, per group from its first channel
  uint32_t* seg_mask;       // [d]
  float* seg_v;             // [B x d]
  float* seg_h;             // [B x d]
  int* seg_cnt;             // [NG]
};

struct ReduceArgs {
  const float* partial;  // [G x B x d]
  int G, B, d, m;
  int Gseg;              // segments of the active lists (blocks of the first kernel)
  int sum_y;             // 0: only the active lists (y is already written)
  const float* residual;  // [B x d] or null
  float* y;               // [B x d]
  // aux (finalize) part; all null when not requested
  int aux;
  const int* seg_j;
  const uint32_t* seg_mask;
  const float* seg_v;
  const float* seg_h;
  const int* seg_cnt;
  int* active_idx;
  int* active_cnt;
  float* active_v;
  float* active_h;
};

// Instantiated chunk counts per row (NCH); a row of d elements uses the
// smallest instantiated NCH >= ceil(d / chunk).
int fused_nch(int wdtype_bf16, int d);
// Largest batch tile (1, 2, 4 or 8) whose x rows fit the LDS budget.
int fused_bt_max(int wdtype_bf16, int nch);
// Blocks of the fused kernel: block g owns neurons [g*m/G, (g+1)*m/G).
int fused_grid(int m);

// Fused-kernel launchers per weight type and variant (cats, cats with the
// active-list segments, dense).
hipError_t launch_fused_bf16_cats(int nch, int bt, const FusedArgs& a, int G, hipStream_t s);
hipError_t launch_fused_bf16_cats_aux(int nch, int bt, const FusedArgs& a, int G, hipStream_t s);
hipError_t launch_fused_bf16_dense(int nch, int bt, const FusedArgs& a, int G, hipStream_t s);
hipError_t launch_fused_f32_cats(int nch, int bt, const FusedArgs& a, int G, hipStream_t s);
hipError_t launch_fused_f32_cats_aux(int nch, int bt, const FusedArgs& a, int G, hipStream_t s);
hipError_t launch_fused_f32_dense(int nch, int bt, const FusedArgs& a, int G, hipStream_t s);
hipError_t launch_reduce(const ReduceArgs& a, hipStream_t s);

// Top-k variant: gate activations of B <= 8 rows into v [B x m], the per-row
// cutoffs (rank r of |v| within each row) into t [B], then the fused kernel
// reading v and t (no W_gate row).
struct GateVArgs {
  const void* wg;      // [m x d] W_gate^T
  const float* x;      // [B x d]
  int B, d, m;
  float* v;            // [B x m] SiLU(x W_gate)
  float t;             // with the list: the CATS threshold
  int* seg_j;          // with the list: [m] per block, its active neurons ascending
  uint32_t* seg_mask;  // [m] their row masks
  int* seg_cnt;        // [G]
  // with the in-kernel select (one row): the cutoff rank r (0 gives t = 0),
  // where t goes, and the epoch-tagged arrival count of the blocks
  int rank;
  float* t_out;
  unsigned long long* ticket;
  uint32_t epoch;
};
// The in-kernel select holds the row's keys in registers: kGateSelKeys per
// thread of a gate block, so rows of up to kGateSelMaxM neurons.
constexpr int kGateSelKeys = 32;
constexpr int kGateSelMaxM = kGateSelKeys * kFusedWaves * 64;  // 64-lane waves
hipError_t launch_gate_v(int wdtype_bf16, int nch, int bt, bool seg, const GateVArgs& a, int G, hipStream_t s);
hipError_t launch_gate_v_select(int wdtype_bf16, int nch, const GateVArgs& a, int G, hipStream_t s);
hipError_t launch_row_select(const float* v, int B, int m, int64_t r, float* t, hipStream_t s);
hipError_t launch_fused_bf16_topk(int nch, int bt, bool aux, const FusedArgs& a, int G, hipStream_t s);
hipError_t launch_fused_f32_topk(int nch, int bt, bool aux, const FusedArgs& a, int G, hipStream_t s);

// The MLP in separate up and down kernels (the paper's structure), rows
// found by the mask or by the gate pass's per-block index lists.
struct UnfusedArgs {
  const void* wu;       // [m x d] W_up^T
  const void* wd;       // [m x d] W_down
  const float* x;       // [B x d]
  const float* v;       // [B x m] gate activations
  float t;
  int B, d, m;
  const int* seg_j;     // index mode: per-block active lists (gate pass)
  const int* seg_cnt;   // [G]
  float* h;             // [B x m] v * (x W_up): at j (mask) or at the list position (index)
  float* partial;       // [G x B x d]
};
hipError_t launch_unfused_up(int wdtype_bf16, int nch, int bt, bool index, const UnfusedArgs& a, int G,
                             hipStream_t s);
hipError_t launch_unfused_down(int wdtype_bf16, int nch, int bt, bool index, const UnfusedArgs& a, int G,
                               hipStream_t s);

// k-steps of the batched gate/up kernel for width d (0: no instantiation
// covers d exactly; those widths use the fused kernel).
int batched_ks(int d);
hipError_t launch_gateup(bool dense, bool aux, const BatchedArgs& a, int G, hipStream_t s);
hipError_t launch_down_mfma(const DownArgs& a, hipStream_t s);
hipError_t launch_sparse_input(const SparseInputArgs& a, hipStream_t s);

hipError_t launch_calib_acts(int wdtype_bf16, const float* x, const void* wg_t, int N, int d,
                             int m, float* acts, hipStream_t s);
// Radix select of the r-th smallest |a| (1-indexed) over n fp32 values;
// `scratch` holds 260 words.  The selected bit pattern ends in scratch[256].
hipError_t launch_radix_select(const float* a, int64_t n, int64_t r, uint32_t* scratch,
                               hipStream_t s);

hipError_t launch_rmsnorm(const float* x, float* xn, int B, int d, float eps, hipStream_t s);
constexpr uint64_t kStreamReadMaxBytes = 1ull << 30;
// Plain read of bytes (a multiple of 16, at most kStreamReadMaxBytes) at buf by
// blocks x 256 threads with inflight (4, 8, 16) 16-byte loads per lane.
hipError_t launch_stream_read(const void* buf, uint32_t bytes, int blocks, int inflight, bool runs, uint32_t* sink,
                              hipStream_t s);
hipError_t launch_transpose(const void* in, void* out, int rows, int cols, int elem_bytes,
                            hipStream_t s);

// Optional per-kernel timing (cats_timer_*): while the timer is enabled a
// KernelTimer hands out a pair of HIP events that the launch (through
// hipExtLaunchKernelGGL) records at the kernel's own start and end; both
// are null otherwise.
class KernelTimer {
 public:
  KernelTimer(const char* name, hipStream_t s);
  hipEvent_t start() const { return a_; }
  hipEvent_t stop() const { return b_; }

 private:
  hipEvent_t a_ = nullptr, b_ = nullptr;
};

}  // namespace cats
