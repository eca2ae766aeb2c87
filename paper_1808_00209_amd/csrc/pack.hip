// Sign-to-bits packing (Eq. 1 and Eq. 2 of the paper with B = 32; input
// thresholding sign(X + T) of Sec. II-C).  Value i of a group of 32 goes to
// bit 31 - i, bit = ((x + offset) > 0) computed in fp32, tail bits 0.
//
// HBM-bound: 4 bytes read per value, 1/8 byte written.  Two mappings:
//  * D >= 32: one lane per value, 32 lanes per output word, so a wave reads
//    256 contiguous bytes; the word comes from a wave ballot, bit-reversed
//    so that lane 0 of the half-wave lands in bit 31.
//  * D < 32 (one word per row, e.g. RGB input with D = 3): one lane per row,
//    reading its D values; consecutive lanes read consecutive rows.
#include "kernels.hpp"

namespace bnn {
namespace {

constexpr int kBlock = 256;

__global__ __launch_bounds__(kBlock) void pack_ballot_kernel(
    const float* __restrict__ x, const float* __restrict__ offset,
    uint32_t rows, uint32_t D, uint32_t Dw, uint32_t* __restrict__ out) {
  const uint32_t total_words = rows * Dw;
  const uint32_t word = blockIdx.x * (kBlock / 32) + threadIdx.x / 32;
  const uint32_t slot = threadIdx.x & 31;
  bool bit = false;
  if (word < total_words) {
    const uint32_t r = word / Dw;
    const uint32_t d = (word - r * Dw) * 32 + slot;
    if (d < D) {
      float v = x[static_cast<uint64_t>(r) * D + d];
      if (offset) v = v + offset[d];
      bit = v > 0.0f;
    }
  }
  const uint64_t m = __ballot(bit);
  const uint32_t half = (threadIdx.x & 32) ? static_cast<uint32_t>(m >> 32)
                                           : static_cast<uint32_t>(m);
  if (slot == 0 && word < total_words) out[word] = __brev(half);
}

__global__ __launch_bounds__(kBlock) void pack_rows_kernel(
    const float* __restrict__ x, const float* __restrict__ offset,
    uint64_t rows, uint32_t D, uint32_t* __restrict__ out) {
  const uint64_t r = static_cast<uint64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (r >= rows) return;
  const float* xr = x + r * D;
  uint32_t v = 0;
  for (uint32_t d = 0; d < D; ++d) {
    float t = xr[d];
    if (offset) t = t + offset[d];
    v |= static_cast<uint32_t>(t > 0.0f) << (31 - d);
  }
  out[r] = v;
}

}  // namespace

hipError_t launch_pack_bits(const float* x, const float* offset, int64_t rows,
                            int64_t D, uint32_t* out, hipStream_t s) {
  if (D < 32) {
    const uint64_t blocks = (static_cast<uint64_t>(rows) + kBlock - 1) / kBlock;
    pack_rows_kernel<<<dim3(static_cast<uint32_t>(blocks)), dim3(kBlock), 0, s>>>(
        x, offset, static_cast<uint64_t>(rows), static_cast<uint32_t>(D), out);
  } else {
    const int64_t Dw = words_of(D);
    const int64_t words = rows * Dw;
    const int64_t blocks = (words + kBlock / 32 - 1) / (kBlock / 32);
    pack_ballot_kernel<<<dim3(static_cast<uint32_t>(blocks)), dim3(kBlock), 0, s>>>(
        x, offset, static_cast<uint32_t>(rows), static_cast<uint32_t>(D),
        static_cast<uint32_t>(Dw), out);
  }
  return hipGetLastError();
}

}  // namespace bnn
