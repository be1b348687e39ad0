// Wave-wide selection on 64-bit keys, shared by the few-row projection and
// the merge kernel.
//
// A (score, index) pair becomes one 64-bit key whose unsigned order is the
// order used everywhere in the library: higher score first, equal scores
// the lower index first.  The score is mapped to an order-preserving
// integer (-0 taken as +0, as the float comparison does) above the
// complement of the index.  The largest key of a wave is found without a
// branch: DPP maxima within each row of 16 lanes, the four row results read
// out and combined on the scalar unit, first for the high words, then for
// the low words of the lanes that hold the largest high word.
#pragma once

#include "kb_common.hpp"

namespace kb {

__device__ __forceinline__ uint64_t key_of(float score, int index) {
  const uint32_t u = (uint32_t)__float_as_int(score + 0.f);
  const uint32_t o = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((uint64_t)o << 32) | (uint32_t)~(uint32_t)index;
}
// key_of(-inf, INT_MAX): the empty entry, below every pair with a non-NaN score
constexpr uint64_t kEmptyKey = ((uint64_t)0x007FFFFFu << 32) | 0x80000000u;
__device__ __forceinline__ float key_score(uint64_t key) {
  const uint32_t o = (uint32_t)(key >> 32);
  return __int_as_float((int)((o & 0x80000000u) ? (o & 0x7fffffffu) : ~o));
}
__device__ __forceinline__ int key_index(uint64_t key) { return (int)~(uint32_t)key; }

__device__ __forceinline__ uint64_t readlane64(uint64_t v, int l) {
  const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)v, l);
  const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l);
  return ((uint64_t)hi << 32) | lo;
}

// DPP lane patterns within a row of 16 lanes: quad xor 1, quad xor 2,
// half-row mirror, row mirror (every lane has a source in each)
constexpr int kDppQXor1 = 0xB1, kDppQXor2 = 0x4E, kDppRowHalfMirror = 0x141, kDppRowMirror = 0x140;
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}

// wave-wide unsigned maximum; 0 is the identity, so the moves need no bound control
__device__ __forceinline__ uint32_t wave_umax(uint32_t v) {
  v = max(v, dpp_u32<kDppQXor1>(v));
  v = max(v, dpp_u32<kDppQXor2>(v));
  v = max(v, dpp_u32<kDppRowHalfMirror>(v));
  v = max(v, dpp_u32<kDppRowMirror>(v));
  const uint32_t a0 = __builtin_amdgcn_readlane((int)v, 0), a1 = __builtin_amdgcn_readlane((int)v, 16);
  const uint32_t a2 = __builtin_amdgcn_readlane((int)v, 32), a3 = __builtin_amdgcn_readlane((int)v, 48);
  return max(max(a0, a1), max(a2, a3));
}

// the wave's largest 64-bit key; every lane gets it
__device__ __forceinline__ uint64_t wave_max64(uint64_t v) {
  const uint32_t hi = (uint32_t)(v >> 32);
  const uint32_t mh = wave_umax(hi);
  const uint32_t ml = wave_umax(hi == mh ? (uint32_t)v : 0u);
  return ((uint64_t)mh << 32) | ml;
}

}  // namespace kb
