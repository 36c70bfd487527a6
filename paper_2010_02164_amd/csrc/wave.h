// Cross-lane combines within one 64-lane wave without going through LDS
// (gfx950). A full combine takes six stages; stage s pairs each lane with
// one partner so that after stages 0..s every lane holds the combination of
// 2^(s+1) lanes:
//   0: lane ^ 1            (DPP quad_perm [1,0,3,2])
//   1: lane ^ 2            (DPP quad_perm [2,3,0,1])
//   2: 7 - lane within 8   (DPP row_half_mirror)
//   3: 15 - lane within 16 (DPP row_mirror)
//   4: rows 0 <-> 1, 2 <-> 3 of 16 lanes (v_permlane16_swap)
//   5: lanes 0-31 <-> 32-63             (v_permlane32_swap)
// Stages 0-3 hand each lane its partner's value; stages 4-5 hand both lanes
// of a pair the same two values (first: the even row / low half, second:
// the odd row / high half), so a combine that is symmetric in its operands
// gives identical results in every lane.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sb {

template <int S>
__device__ __forceinline__ uint32_t dpp_partner(uint32_t x) {
  static_assert(S >= 0 && S <= 3, "DPP stages are 0..3");
  constexpr int ctrl = S == 0 ? 0xB1 : S == 1 ? 0x4E : S == 2 ? 0x141 : 0x140;
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, ctrl, 0xF, 0xF, false);
}

// Stages 4 (rows) and 5 (halves): the pair's two values, even/low first.
template <int S>
__device__ __forceinline__ void swap_pair(uint32_t x, uint32_t &first, uint32_t &second) {
  static_assert(S == 4 || S == 5, "swap stages are 4 and 5");
  if constexpr (S == 4) {
    const auto p = __builtin_amdgcn_permlane16_swap(x, x, false, false);
    first = p[0];
    second = p[1];
  } else {
    const auto p = __builtin_amdgcn_permlane32_swap(x, x, false, false);
    first = p[0];
    second = p[1];
  }
}

// Stage S applied to a 64-bit value: (own-or-first, partner-or-second).
template <int S>
__device__ __forceinline__ void stage64(unsigned long long x, unsigned long long &a, unsigned long long &b) {
  const uint32_t lo = (uint32_t)x, hi = (uint32_t)(x >> 32);
  if constexpr (S <= 3) {
    a = x;
    b = ((unsigned long long)dpp_partner<S>(hi) << 32) | dpp_partner<S>(lo);
  } else {
    uint32_t l0, l1, h0, h1;
    swap_pair<S>(lo, l0, l1);
    swap_pair<S>(hi, h0, h1);
    a = ((unsigned long long)h0 << 32) | l0;
    b = ((unsigned long long)h1 << 32) | l1;
  }
}

template <int S>
__device__ __forceinline__ void stage32(uint32_t x, uint32_t &a, uint32_t &b) {
  if constexpr (S <= 3) {
    a = x;
    b = dpp_partner<S>(x);
  } else {
    swap_pair<S>(x, a, b);
  }
}

}  // namespace sb
