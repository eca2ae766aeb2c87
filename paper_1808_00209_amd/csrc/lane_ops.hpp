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

// Row r of a wave is lanes 16 r .. 16 r + 15.  v_permlane16_swap(a, b)
// exchanges the odd rows of a with the even rows of b; v_permlane32_swap(a, b)
// exchanges rows 2-3 of a with rows 0-1 of b.  For four words w0..w3 whose
// rows each hold disjoint bits of one value per lane column, row q of the
// result holds w_q ORed over its four rows (lane 16 q + c: column c).
// Three swaps serve four words, where or_xor16 / or_xor32 take two per word.
__device__ __forceinline__ uint32_t or_rows4(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3) {
  const auto a = __builtin_amdgcn_permlane16_swap(w0, w1, false, false);
  const auto b = __builtin_amdgcn_permlane16_swap(w2, w3, false, false);
  // Rows of x01: w0 (rows 0|1), w1 (rows 0|1), w0 (rows 2|3), w1 (rows 2|3).
  const uint32_t x01 = a[0] | a[1];
  const uint32_t x23 = b[0] | b[1];
  const auto c = __builtin_amdgcn_permlane32_swap(x01, x23, false, false);
  return c[0] | c[1];
}

// OR over the 4 lanes of each quad (lanes 4k .. 4k + 3): DPP quad_perm
// [1,0,3,2] (lane ^ 1), then [2,3,0,1] (lane ^ 2).
__device__ __forceinline__ uint32_t or_quad(uint32_t x) {
  x |= static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0xB1, 0xF, 0xF, false));
  x |= static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x4E, 0xF, 0xF, false));
  return x;
}

}  // namespace bnn
