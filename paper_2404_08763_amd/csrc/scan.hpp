// Inclusive prefix sum over the 64 lanes of a wave without LDS permutes:
// Hillis-Steele steps by DPP row shifts of 1, 2, 4 and 8 lanes within each
// row of 16 (lanes shifted in from outside the row read 0), then the last
// lane of row 0 is added to row 1 and of row 2 to row 3 (row_bcast:15),
// and the last lane of row 1 to rows 2 and 3 (row_bcast:31).  Integer
// addition, so the result does not depend on the order.  All lanes active.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cats {

__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xf, 0xf, true);   // row_shr:1
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xf, 0xf, true);   // row_shr:2
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xf, 0xf, true);   // row_shr:4
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xf, 0xf, true);   // row_shr:8
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xa, 0xf, false);  // row_bcast:15
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return v;
}

}  // namespace cats
