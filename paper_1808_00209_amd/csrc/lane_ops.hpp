// Cross-lane ORs of a wave's packed words without the LDS: gfx950's
// v_permlane16/32_swap and DPP quad permutes run on the vector ALU, where a
// __shfl_xor becomes a ds_bpermute round trip through the LDS unit.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bnn {

// x of this lane OR x of lane ^ 32.  v_permlane32_swap exchanges one half of
// the wave between its two operands; with both operands equal to x, every
// lane of (x | first result | second result) holds x | x[lane ^ 32],
// whichever halves the instruction exchanges.
__device__ __forceinline__ uint32_t or_xor32(uint32_t x) {
  const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  return x | r[0] | r[1];
}

// x of this lane OR x of lane ^ 16 (v_permlane16_swap, as above per 32 lanes).
__device__ __forceinline__ uint32_t or_xor16(uint32_t x) {
  const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  return x | r[0] | r[1];
}

// OR over the 4 lanes of each quad (lanes 4k .. 4k + 3): DPP quad_perm
// [1,0,3,2] (lane ^ 1), then [2,3,0,1] (lane ^ 2).
__device__ __forceinline__ uint32_t or_quad(uint32_t x) {
  x |= static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0xB1, 0xF, 0xF, false));
  x |= static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x4E, 0xF, 0xF, false));
  return x;
}

}  // namespace bnn
