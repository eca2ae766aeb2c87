// fp32 image values on the bf16 matrix cores, and fp32 thresholds that
// compare exactly with an integer threshold.  Shared by the real-valued
// first-layer kernels (fconv.hip, fconv_bconv.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bnn {

typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

// x as the exact sum of three bf16 values: x's significand cut into three
// pieces of (at most) 8 significant bits, each truncated toward zero, so each
// part carries x's sign.  The parts are returned as fp32 bit patterns whose
// low 16 bits are zero (a bf16 value is the high half of its fp32 pattern).
//   p0 = x with the low 16 bits of its pattern cleared;
//   r1 = x - p0: exact (p0 <= x < 2 p0 in magnitude, same sign), at most 16
//        significant bits left;
//   p1 = r1 cleared likewise, r2 = r1 - p1 exact, at most 8 significant bits,
//        so r2's pattern already has zero low bits when r2 is a normal fp32.
// x = p0 + p1 + p2 holds exactly, each part a normal bf16 or zero, for
// finite x with |x| >= 2^-103 or x == 0 (then the last part's lowest bit is at
// least 2^-126).  Smaller magnitudes may lose up to |x| when the matrix core
// flushes a subnormal part.  A non-finite x gives non-finite parts.
struct Split3 {
  uint32_t p0, p1, p2;
};

__device__ __forceinline__ Split3 split3(float x) {
  const uint32_t h0 = __float_as_uint(x) & 0xFFFF0000u;
  const float r1 = x - __uint_as_float(h0);
  const uint32_t h1 = __float_as_uint(r1) & 0xFFFF0000u;
  const float r2 = r1 - __uint_as_float(h1);
  return Split3{h0, h1, __float_as_uint(r2) & 0xFFFF0000u};
}

// The bf16 half of a part pattern.
__device__ __forceinline__ uint16_t bf16_bits(uint32_t p) { return static_cast<uint16_t>(p >> 16); }

// Eight bf16 values from their 16-bit patterns.
__device__ __forceinline__ v8bf bf16x8(const uint16_t (&v)[8]) {
  typedef uint32_t v4u __attribute__((ext_vector_type(4)));
  v4u r;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    r[i] = static_cast<uint32_t>(v[2 * i]) | (static_cast<uint32_t>(v[2 * i + 1]) << 16);
  return __builtin_bit_cast(v8bf, r);
}

// bf16 +1.0, -1.0 and 0.0 (operands of the +-1 weights; 0 past the window).
constexpr uint16_t kBf16One = 0x3F80u, kBf16MinusOne = 0xBF80u, kBf16Zero = 0u;

// The smallest fp32 value t' >= t (t' = -0.0 for t = 0).  For every fp32 s
// that is not NaN, s >= t  <=>  s >= t', and the sign bit of the rounded
// difference s - t' is clear exactly when s >= t (a difference of two fp32
// values rounds to zero only when they are equal, and -0.0 as t' turns s =
// -0.0 into s - t' = +0.0).
__device__ __forceinline__ float thr_ceil_f32(int32_t t) {
  if (t == 0) return -0.0f;
  const double d = static_cast<double>(t);
  float f = static_cast<float>(d);  // nearest; |f| >= 1
  if (static_cast<double>(f) < d) f = __uint_as_float(__float_as_uint(f) + (f > 0.0f ? 1u : ~0u));
  return f;
}

}  // namespace bnn
