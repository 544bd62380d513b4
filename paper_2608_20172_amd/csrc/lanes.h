// Lane-group reductions on the vector ALU's data-parallel-primitive (DPP) lane
// moves. __shfl_xor lowers to ds_bpermute, which goes through the LDS crossbar
// and competes with the LDS traffic of the kernels that reduce inside their
// inner loops; a DPP move is a modifier on an ordinary vector instruction.
#pragma once
#include <hip/hip_runtime.h>

namespace rel {

template <int CTRL>
__device__ __forceinline__ float dpp_move(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}

// Sum over each aligned group of G lanes (G = 2, 4, 8 or 16). Every lane of a
// group ends with the same bits (each step adds two equal partial sums in
// either order). Every lane of the wave must be active.
template <int G>
__device__ __forceinline__ float group_sum(float x) {
  static_assert(G == 2 || G == 4 || G == 8 || G == 16, "DPP groups stay inside a row of 16 lanes");
  x += dpp_move<0xB1>(x);                          // quad_perm [1,0,3,2]: lane ^ 1
  if constexpr (G >= 4) x += dpp_move<0x4E>(x);   // quad_perm [2,3,0,1]: lane ^ 2
  if constexpr (G >= 8) x += dpp_move<0x141>(x);  // row_half_mirror: lane i <-> 7 - i of its 8
  if constexpr (G >= 16) x += dpp_move<0x140>(x); // row_mirror: lane i <-> 15 - i of its 16
  return x;
}

// Sum over each aligned group of G lanes, G a power of two up to 64: DPP
// within rows of 16 lanes, then lane exchanges across rows.
template <int G>
__device__ __forceinline__ float lane_group_sum(float x) {
  if constexpr (G == 1) {
    return x;
  } else if constexpr (G <= 16) {
    return group_sum<G>(x);
  } else {
    x = group_sum<16>(x);
    x += __shfl_xor(x, 16, 64);
    if constexpr (G == 64) x += __shfl_xor(x, 32, 64);
    return x;
  }
}

}  // namespace rel
