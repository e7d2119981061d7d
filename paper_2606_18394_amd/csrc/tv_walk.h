// Device helpers shared by the greedy and the non-greedy tree acceptance:
// the pointer-jumping state of one node packed into a 32-bit word, and
// wave-wide unsigned maxima on DPP exchanges.  Pointer jumping over the parent links finds,
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

// One DPP exchange of a 32-bit value (all rows and banks enabled).
template <int CTRL>
__device__ __forceinline__ unsigned dpp_u32(unsigned x) {
  return (unsigned)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xF, 0xF, false);
}
// A row broadcast into the rows of ROWMASK; the other rows keep x.
template <int CTRL, int ROWMASK>
__device__ __forceinline__ unsigned dpp_bcast_u32(unsigned x) {
  return (unsigned)__builtin_amdgcn_update_dpp((int)x, (int)x, CTRL, ROWMASK, 0xF, false);
}

// Wave-wide maximum, returned as a wave-uniform value: DPP steps inside each
// row of 16 lanes (lane ^ 1, lane ^ 2, then the mirrored quads and halves),
// then row 1 takes row 0's maximum and row 3 row 2's, and rows 2 and 3 take
// row 1's (the two row broadcasts): lane 63 holds the wave's.  No step goes
// through the LDS crossbar.
__device__ __forceinline__ unsigned int wave_max_u32(unsigned int x) {
  x = max(x, dpp_u32<0xB1>(x));
  x = max(x, dpp_u32<0x4E>(x));
  x = max(x, dpp_u32<0x141>(x));
  x = max(x, dpp_u32<0x140>(x));
  x = max(x, dpp_bcast_u32<0x142, 0xA>(x));
  x = max(x, dpp_bcast_u32<0x143, 0xC>(x));
  return __builtin_amdgcn_readlane(x, 63);
}

}  // namespace tv
