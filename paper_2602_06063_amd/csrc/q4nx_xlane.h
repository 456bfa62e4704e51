// Cross-lane exchanges for gfx950 that stay in the VALU: lane l receives the
// value lane l ^ M holds.  The generic shuffle goes through the LDS crossbar
// (ds_bpermute: an LDS instruction and its wait per step); these use DPP and
// gfx950's permlane swaps instead, and are the same permutations, so every
// sum built from them is unchanged bit for bit.
//   M = 1, 2: DPP quad permutations [1,0,3,2] and [2,3,0,1];
//   M = 4:    DPP row shifts by 4 (left for lanes with bit 2 clear, right
//             for the others);
//   M = 8:    DPP rotation of each 16-lane row by 8;
//   M = 16:   v_permlane16_swap (odd and even rows of 16 exchanged);
//   M = 32:   v_permlane32_swap (the two halves of the wave exchanged).
// Every lane of the wave must be active (the kernels call these with full
// execution masks).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace q4nx {

__device__ __forceinline__ int lane_id() {
  return (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
}

template <int M>
__device__ __forceinline__ int xor_lane_bits(int x) {
  static_assert(M == 1 || M == 2 || M == 4 || M == 8 || M == 16 || M == 32, "lane mask");
  if constexpr (M == 1) {
    return __builtin_amdgcn_update_dpp(0, x, 0xB1, 0xF, 0xF, false);
  } else if constexpr (M == 2) {
    return __builtin_amdgcn_update_dpp(0, x, 0x4E, 0xF, 0xF, false);
  } else if constexpr (M == 4) {
    const int up = __builtin_amdgcn_update_dpp(0, x, 0x104, 0xF, 0xF, false);    // row_shl:4
    const int down = __builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, false);  // row_shr:4
    return (lane_id() & 4) ? down : up;
  } else if constexpr (M == 8) {
    return __builtin_amdgcn_update_dpp(0, x, 0x128, 0xF, 0xF, false);            // row_ror:8
  } else if constexpr (M == 16) {
    const auto p = __builtin_amdgcn_permlane16_swap((unsigned)x, (unsigned)x, false, false);
    return (int)(((lane_id() >> 4) & 1) ? p[0] : p[1]);
  } else {
    const auto p = __builtin_amdgcn_permlane32_swap((unsigned)x, (unsigned)x, false, false);
    return (int)((lane_id() >> 5) ? p[0] : p[1]);
  }
}

template <int M>
__device__ __forceinline__ float xor_lane(float v) {
  return __builtin_bit_cast(float, xor_lane_bits<M>(__builtin_bit_cast(int, v)));
}

}  // namespace q4nx
