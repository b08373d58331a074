// Geometry and arguments of the fused MLP kernel (k_mlp_fused), kept apart
// from the other launch interfaces: everything the fused kernel's code
// depends on besides its own source and device.hpp lives here.
#pragma once

#include <stdint.h>

namespace cats {

// Geometry of the fused MLP kernel (build-time tunables): waves per block
// and the number of blocks, one or two per compute unit of an MI355X.
#ifndef CATS_FUSED_WAVES
#define CATS_FUSED_WAVES 8
#endif
#ifndef CATS_FUSED_BLOCKS
#define CATS_FUSED_BLOCKS 256
#endif
constexpr int kFusedWaves = CATS_FUSED_WAVES;
// Waves of a fused-kernel block for rows of nch 16-byte chunks per lane and
// a tile of bt batch rows.  One wave per SIMD when there is one row (each
// wave then walks twice the neurons, so the per-block imbalance of the last
// wave is half a neuron's share smaller) and at 16 chunks (bf16 rows of up
// to 8192, whose four row buffers alone need 256 registers: a wave gets the
// whole register file of its SIMD); two per SIMD otherwise, where the dot
// products over several staged rows need a second wave to hide their
// LDS reads, and when the gate activations are given (vin: no gate rows
// stream, so a wave has fewer loads in flight and two per SIMD keep more).
constexpr int fused_waves(int nch, int bt, bool vin) {
  return ((bt == 1 && !vin) || nch >= 16) ? 4 : kFusedWaves;
}
constexpr int kFusedBlocks = CATS_FUSED_BLOCKS;
// Neurons a fused-kernel block may own (its LDS lists are this long); with
// kFusedBlocks blocks this bounds m.
constexpr int kFusedMaxNeurons = 65536 / kFusedBlocks;
constexpr int kMaxNeurons = kFusedBlocks * kFusedMaxNeurons;
// LDS bytes the fused kernel may spend on the staged x rows.
constexpr int kXLdsBytes = 128 * 1024;

// Elements per 64-lane chunk of a weight row (16 bytes per lane).
inline int chunk_elems(int wdtype_bf16) { return wdtype_bf16 ? 512 : 256; }

struct FusedArgs {
  const void* wg;      // [m x d] W_gate^T
  const void* wu;      // [m x d] W_up^T
  const void* wd;      // [m x d] W_down
  const float* x;      // [B x d]
  int B, d, m;
  float t;
  int norm;            // RMSNorm x (unit gain) before the block
  float eps;           // its epsilon
  const float* vin;    // top-k variant: v [B x m] computed beforehand
  const float* vin_t;  // and one cutoff per row [B]
  float* partial;      // [G x B x d]
  int aux;             // write the union segments for the aux outputs
  int* seg_j;          // [m]
  uint32_t* seg_mask;  // [m] bit b = active in row b
  float* seg_v;        // [B x m]
  float* seg_h;        // [B x m]
  int* seg_cnt;        // [G]
};

}  // namespace cats
