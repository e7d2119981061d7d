// Device helpers shared by the greedy and the non-greedy tree acceptance:
// the pointer-jumping state of one node packed into a 32-bit word, and a
// wave-wide unsigned maximum.  Pointer jumping over the parent links finds,
// for every node at once, its depth and whether every node on its root path
// passed its test, in O(log depth) rounds.
#pragma once
#include <hip/hip_runtime.h>

#include "tv_plan.h"

namespace tv {

// state word: jump target (bits 0-10), path length to it (bits 11-22), and
// bit 23 set when every node on that stretch passed
constexpr unsigned int kJmpMask = 0x7FFu, kDepShift = 11, kDepMask = 0xFFFu, kOkBit = 1u << 23;
static_assert(kMaxNodes - 1 <= (int)kJmpMask && kMaxNodes - 1 <= (int)kDepMask, "state word fields");

__device__ __forceinline__ unsigned int pack_state(unsigned int jmp, unsigned int dep, bool ok) {
  return jmp | (dep << kDepShift) | (ok ? kOkBit : 0u);
}

// One jumping round for node i: read its state and its target's (either
// the previous round's words or, where the caller updates in place, the
// target's newer word: both are consistent), return the combined state.
__device__ __forceinline__ unsigned int jump_state(const unsigned int* sc, int i) {
  const unsigned int wi = sc[i];
  const unsigned int wj = sc[wi & kJmpMask];
  const unsigned int dep = ((wi >> kDepShift) & kDepMask) + ((wj >> kDepShift) & kDepMask);
  return pack_state(wj & kJmpMask, dep, (wi & wj & kOkBit) != 0);
}

// The deepest node that passed, lowest index on ties, as a sortable key
// depth << 16 | (0xFFFF - i) (0 when it did not pass).
__device__ __forceinline__ unsigned int deepest_key(unsigned int w, int i) {
  return (w & kOkBit) ? (((w >> kDepShift) & kDepMask) << 16) | (0xFFFFu - (unsigned int)i) : 0u;
}

__device__ __forceinline__ unsigned int wave_max_u32(unsigned int k) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const unsigned int other = __shfl_xor(k, o);
    k = other > k ? other : k;
  }
  return k;
}

}  // namespace tv
