// Packed +-1 words as fp4 (E2M1) matrix-core operands, shared by the binary
// conv kernels: a value of the method is exactly +-1.0 in E2M1, and a word of
// 32 values becomes the 4 registers of one lane's 32-value share of a
// v_mfma_scale_f32_32x32x64_f8f6f4 operand.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bnn {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v16f __attribute__((ext_vector_type(16)));


// One packed word -> four fp4 registers: register r, nibble n encodes bit
// 4n + r of the word (1 -> 0xA = -1.0, 0 -> 0x2 = +1.0).  Each register is
// one shift and one v_and_or_b32 (mask in an SGPR, fill constant in a VGPR:
// this VOP3 form takes no literal operands on gfx950).
__device__ __forceinline__ uint32_t and_or(uint32_t x, uint32_t smask, uint32_t vfill) {
  uint32_t d;
  asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(d) : "v"(x), "s"(smask), "v"(vfill));
  return d;
}

__device__ __forceinline__ v8i expand_fp4(uint32_t w, uint32_t smask, uint32_t vfill) {
  v8i x;
  x[0] = static_cast<int>(and_or(w << 3, smask, vfill));
  x[1] = static_cast<int>(and_or(w << 2, smask, vfill));
  x[2] = static_cast<int>(and_or(w << 1, smask, vfill));
  x[3] = static_cast<int>(and_or(w, smask, vfill));
  x[4] = x[5] = x[6] = x[7] = 0;
  return x;
}

// Two words at once: the pair (w1:w0) is shifted as one 64-bit value
// (v_lshlrev_b64 runs at full rate), 3 shifts + 8 v_and_or_b32 for two words
// instead of 3 + 3 + 8.  The bits w0 pushes into w1's low end land at
// positions 0..2, outside the 0x88888888 mask.
__device__ __forceinline__ uint64_t shl64(uint64_t x, int s) {
  uint64_t d;
  asm("v_lshlrev_b64 %0, %1, %2" : "=v"(d) : "i"(s), "v"(x));
  return d;
}

__device__ __forceinline__ void expand_pair(uint32_t w0, uint32_t w1, uint32_t smask,
                                            uint32_t vfill, v8i& x0, v8i& x1) {
  const uint64_t p = (static_cast<uint64_t>(w1) << 32) | w0;
  const uint64_t s1 = shl64(p, 1), s2 = shl64(p, 2), s3 = shl64(p, 3);
  x0[0] = static_cast<int>(and_or(static_cast<uint32_t>(s3), smask, vfill));
  x0[1] = static_cast<int>(and_or(static_cast<uint32_t>(s2), smask, vfill));
  x0[2] = static_cast<int>(and_or(static_cast<uint32_t>(s1), smask, vfill));
  x0[3] = static_cast<int>(and_or(w0, smask, vfill));
  x1[0] = static_cast<int>(and_or(static_cast<uint32_t>(s3 >> 32), smask, vfill));
  x1[1] = static_cast<int>(and_or(static_cast<uint32_t>(s2 >> 32), smask, vfill));
  x1[2] = static_cast<int>(and_or(static_cast<uint32_t>(s1 >> 32), smask, vfill));
  x1[3] = static_cast<int>(and_or(w1, smask, vfill));
  x0[4] = x0[5] = x0[6] = x0[7] = 0;
  x1[4] = x1[5] = x1[6] = x1[7] = 0;
}

// An activation word as the B operand against prepared weights (the
// operand form of prepare_weights_kernel).  Register r < 3 keeps bits 4n + r
// of the word where they are, so nibble n is the E2M1 value 0 (bit 0) or
// 2^(r-1) (bit 1: 0.5, 1.0, 2.0), one v_and_b32 each; register 3 is the +-1
// form of expand_fp4 (bit 1 -> -1.0).  The prepared weights hold +-4, +-2,
// +-1 in registers 0, 1, 2 (bit 1 -> +) and -1/+1 in register 3 (bit 1 ->
// -1), so with a the activation bit and s(b) = 2b - 1 every product is
// 2 a s(w) = s(a) s(w) + s(w) in registers 0-2 and s(a) s(w) in register 3:
// a window's sum comes out S + B_f, B_f = sum of s(w) over the positions of
// registers 0-2, a constant of the filter that the epilogue takes off.
// Four VALU instructions per word, against 5.5 for expand_pair.
__device__ __forceinline__ v8i act_operand(uint32_t x, uint32_t smask, uint32_t vfill) {
  v8i r;
  r[0] = static_cast<int>(x & 0x11111111u);
  r[1] = static_cast<int>(x & 0x22222222u);
  r[2] = static_cast<int>(x & 0x44444444u);
  r[3] = static_cast<int>(and_or(x, smask, vfill));
  r[4] = r[5] = r[6] = r[7] = 0;
  return r;
}

// Expands VW consecutive words (VW = 1, 2 or 4) into VW operands.
template <int VW>
__device__ __forceinline__ void expand_words(const uint32_t (&w)[VW], uint32_t smask,
                                             uint32_t vfill, v8i (&x)[VW]) {
  if constexpr (VW == 1) {
    x[0] = expand_fp4(w[0], smask, vfill);
  } else {
#pragma unroll
    for (int v = 0; v < VW; v += 2) expand_pair(w[v], w[v + 1], smask, vfill, x[v], x[v + 1]);
  }
}

}  // namespace bnn
