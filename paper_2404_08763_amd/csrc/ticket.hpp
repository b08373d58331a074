// Arrival tickets for "the last block finishes" without any block waiting.
//
// A ticket is a 64-bit word in the caller's workspace: the high 32 bits tag
// the call (a host epoch, never 0), the low 32 bits count the blocks of that
// call that have arrived.  The workspace may hold anything when a call
// starts (garbage, another call's leftovers).  Each block reads the word
// when it starts (ticket_peek), long before it arrives, so that arriving
// costs one atomic: with this call's tag it adds itself; with another tag it
// installs this call's tag with a count of one by compare-and-swap, and if
// another block installed it first it adds itself instead.  A stale word is
// never added to, so each block counts exactly once and no block retries
// more than once.  The last block (count == n) leaves the word at a zero
// count under the next epoch's tag, so a call that directly follows on the
// same workspace finds its own tag at once.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cats {

// The word as a block starts (one thread per block).
__device__ __forceinline__ unsigned long long ticket_peek(const unsigned long long* word) {
  return __hip_atomic_load(word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Called by one thread per block with its peek; true for the block that
// arrives last.
__device__ __forceinline__ bool take_ticket(unsigned long long* word, uint32_t epoch, uint32_t n,
                                            unsigned long long cur) {
  const unsigned long long tag = (unsigned long long)epoch << 32;
  unsigned long long got;
  for (;;) {
    if ((cur >> 32) == (unsigned long long)epoch) {
      got = __hip_atomic_fetch_add(word, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + 1ull;
      break;
    }
    if (__hip_atomic_compare_exchange_strong(word, &cur, tag | 1ull, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT)) {
      got = tag | 1ull;
      break;
    }
    // cur now holds what beat the swap: this call's tag (then add), or in
    // principle another stale value (then try to install again)
  }
  const bool last = (uint32_t)(got & 0xffffffffull) == n;
  if (last) {
    const uint32_t next = epoch == 0xffffffffu ? 1u : epoch + 1u;
    __hip_atomic_store(word, (unsigned long long)next << 32, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  return last;
}

}  // namespace cats
