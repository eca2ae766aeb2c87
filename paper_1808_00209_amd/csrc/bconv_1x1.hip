// Binary 1x1 conv with short windows (Eq. 4 with a single tap, K = C = 64,
// 128 or 256 bits) on the fp4 matrix cores, for large pixel counts.
//
// With K <= 256 a 32 x 32 output tile is only 1..4 MFMA k-steps deep, so in
// the general conv kernel a wave spends more on its pixel operands, its
// set-up and its epilogue than on the matrix cores.  Here a wave keeps the
// fp4 operands of its 64 pixels in registers, expanded once, and walks all
// filters in chunks of 64: per chunk it expands only the chunk's weights
// (prefetched one chunk ahead), runs 4 KS MFMAs and puts the chunk's two
// output words per pixel into the wave's LDS copy of its 64 output rows.  At
// the end the wave writes those rows out whole: consecutive lanes store
// consecutive 8-byte pieces of adjacent rows, where storing each word
// straight from its lane touched 64 rows per instruction, 4 bytes each (the
// stores then took about 40 % of the kernel).  The block's thresholds (as
// 0.5 - thr, the accumulators' start value) and flip words are staged in LDS
// once.
#include <stdint.h>

#include "fp4_expand.hpp"
#include "kernels.hpp"

namespace bnn {
namespace {

constexpr int kPix = 256;   // pixels per block: 4 waves x 64
constexpr int kMaxF = 1024;  // LDS: output rows 34 KB + thresholds 4 KB at F = 1024

struct B1Args {
  const uint32_t* in;    // [M, Cw]
  const uint32_t* w;     // [F, Cw]
  const int32_t* thr;    // [F]
  const uint32_t* flip;  // [Fw] or null
  uint32_t* bits;        // [M, Fw]
  int32_t M, F, Fw, K;
};

// KS consecutive words of a row: one 128-, 64- or 32-bit load.
template <int KS>
__device__ __forceinline__ void load_words(const uint32_t* p, uint32_t (&v)[KS]) {
  if constexpr (KS == 4) {
    const uint4 t = *reinterpret_cast<const uint4*>(p);
    v[0] = t.x;
    v[1] = t.y;
    v[2] = t.z;
    v[3] = t.w;
  } else if constexpr (KS == 2) {
    const uint2 t = *reinterpret_cast<const uint2*>(p);
    v[0] = t.x;
    v[1] = t.y;
  } else {
    v[0] = p[0];
  }
}

// KS = k-steps of 64 bits = Cw / 2.  Lane (h, c) feeds words h KS .. h KS +
// KS - 1 of its operand row, in both operands (the same permutation of the
// window's bit positions on both sides leaves every dot product unchanged):
// k-step s pairs word s of lane half 0 with word KS + s of lane half 1.
template <int KS>
__global__ __launch_bounds__(256) void bconv1x1_kernel(B1Args a) {
  constexpr int CW = 2 * KS;
  __shared__ float thl[kMaxF];
  __shared__ uint32_t nfl[kMaxF / 32];
  // The wave's output rows: 64 rows of Fw words at stride Fw + 2 (8-byte
  // aligned; an odd half-stride spreads a column over the banks).
  extern __shared__ uint32_t ostage[];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int h = lane >> 5, c = lane & 31;
  const int p0 = blockIdx.x * kPix + wave * 64;
  const int os = a.Fw + 2;
  uint32_t* orow = ostage + wave * 64 * os;

  // Pixel words and the first chunk's weight words, then the thresholds
  // (clamped to [-K-1, K+1], which keeps every comparison since |S| <= K).
  uint32_t xw[2][KS];
  bool pv[2];
#pragma unroll
  for (int tp = 0; tp < 2; ++tp) {
    const int p = p0 + 32 * tp + c;
    pv[tp] = p < a.M;
    load_words<KS>(a.in + static_cast<size_t>(pv[tp] ? p : a.M - 1) * CW + h * KS, xw[tp]);
  }
  uint32_t wa[2][KS], wb[2][KS];
#pragma unroll
  for (int tf = 0; tf < 2; ++tf)
    load_words<KS>(a.w + static_cast<size_t>(32 * tf + c) * CW + h * KS, wa[tf]);
  for (int f = threadIdx.x; f < a.F; f += 256)
    thl[f] = 0.5f - static_cast<float>(min(max(a.thr[f], -a.K - 1), a.K + 1));
  for (int i = threadIdx.x; i < a.Fw; i += 256) nfl[i] = ~(a.flip ? a.flip[i] : 0u);

  const uint32_t smask = __builtin_amdgcn_readfirstlane(0x88888888u);
  uint32_t vfill;
  asm("v_mov_b32 %0, 0x22222222" : "=v"(vfill));
  v8i B[2][KS];
#pragma unroll
  for (int tp = 0; tp < 2; ++tp) expand_words<KS>(xw[tp], smask, vfill, B[tp]);
  __syncthreads();

  // One chunk of 64 filters: expand its weights, prefetch the next chunk's,
  // MFMAs from 0.5 - thr, then the sign bits.  Register e of lane (h, c)
  // ends as S - thr + 0.5 of filter f0 + 32 tf + 8 (e / 4) + 4 h + e % 4 at
  // pixel c of tile tp; its sign bit is the complement of the output bit.
  // One v_permlane32_swap of the two filter tiles' words leaves lane half h
  // with the whole word of tile h.
  const int nch = a.F / 64;
  auto chunk = [&](int ch, const uint32_t (&cw)[2][KS], uint32_t (&nw)[2][KS]) {
    const int f0 = 64 * ch;
    v8i A[2][KS];
#pragma unroll
    for (int tf = 0; tf < 2; ++tf) expand_words<KS>(cw[tf], smask, vfill, A[tf]);
    if (ch + 1 < nch) {
#pragma unroll
      for (int tf = 0; tf < 2; ++tf)
        load_words<KS>(a.w + static_cast<size_t>(f0 + 64 + 32 * tf + c) * CW + h * KS, nw[tf]);
    }
    v16f acc[2][2];
#pragma unroll
    for (int tf = 0; tf < 2; ++tf) {
      v16f t;
#pragma unroll
      for (int e = 0; e < 16; ++e) t[e] = thl[f0 + 32 * tf + 8 * (e >> 2) + 4 * h + (e & 3)];
      acc[tf][0] = t;
      acc[tf][1] = t;
    }
#pragma unroll
    for (int s = 0; s < KS; ++s)
#pragma unroll
      for (int tf = 0; tf < 2; ++tf)
#pragma unroll
        for (int tp = 0; tp < 2; ++tp)
          acc[tf][tp] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
              A[tf][s], B[tp][s], acc[tf][tp], 4, 4, 0, 127, 0, 127);
    const uint32_t fx = nfl[f0 / 32 + h];
#pragma unroll
    for (int tp = 0; tp < 2; ++tp) {
      uint32_t wd[2];
#pragma unroll
      for (int tf = 0; tf < 2; ++tf) {
        wd[tf] = 0u;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          uint32_t nib = 0u;
#pragma unroll
          for (int r = 0; r < 4; ++r)
            nib = __builtin_amdgcn_alignbit(nib, __float_as_uint(acc[tf][tp][4 * g + r]), 31);
          wd[tf] |= nib << (28 - 8 * g - 4 * h);
        }
      }
      const auto sw = __builtin_amdgcn_permlane32_swap(wd[0], wd[1], false, false);
      orow[(32 * tp + c) * os + f0 / 32 + h] = (sw[0] | sw[1]) ^ fx;
    }
  };
  // Two chunks per trip, so the two weight register sets keep fixed names.
  for (int ch = 0; ch < nch; ch += 2) {
    chunk(ch, wa, wb);
    if (ch + 1 < nch) chunk(ch + 1, wb, wa);
  }
  __syncthreads();

  // Rows out: hw = Fw / 2 pieces of 8 bytes per row, rpi whole rows per
  // store instruction (lanes past rpi * hw idle), rows p0 .. p0 + 63 being
  // adjacent in memory.
  const int hw = a.Fw / 2;
  const int rpi = 64 / hw;
  const int r0 = lane / hw, q = lane - r0 * hw;
  if (r0 < rpi) {
    for (int r = r0; r < 64; r += rpi) {
      if (p0 + r >= a.M) break;
      const uint2 v = *reinterpret_cast<const uint2*>(&orow[r * os + 2 * q]);
      *reinterpret_cast<uint2*>(&a.bits[static_cast<size_t>(p0 + r) * a.Fw + 2 * q]) = v;
    }
  }
}

}  // namespace

bool bconv1x1_supported(const ConvGeom& g, bool sums) {
  const int64_t M = static_cast<int64_t>(g.N) * g.H * g.W;
  // C = 64, 128 or 256: 1, 2 or 4 k-steps, the instantiated variants (the
  // launcher maps Cw = 2 / 4 / 8 onto them and nothing else).
  return !sums && g.KH == 1 && g.KW == 1 && g.pad == 0 && g.pool == 0 &&
         (g.C == 64 || g.C == 128 || g.C == 256) && g.F % 64 == 0 && g.F <= kMaxF && M >= 256 * kPix &&
         M * g.Fw < (int64_t{1} << 31);
}

hipError_t launch_bconv1x1(const ConvGeom& g, const uint32_t* in, const uint32_t* w,
                           const int32_t* thr, const uint32_t* flip, uint32_t* bits,
                           hipStream_t s) {
  B1Args a;
  a.in = in;
  a.w = w;
  a.thr = thr;
  a.flip = flip;
  a.bits = bits;
  a.M = static_cast<int32_t>(static_cast<int64_t>(g.N) * g.H * g.W);
  a.F = g.F;
  a.Fw = g.Fw;
  a.K = g.C;
  const unsigned blocks = static_cast<unsigned>((a.M + kPix - 1) / kPix);
  const size_t lds = static_cast<size_t>(4 * 64) * (g.Fw + 2) * sizeof(uint32_t);
  switch (g.Cw) {
    case 2: bconv1x1_kernel<1><<<blocks, 256, lds, s>>>(a); break;
    case 4: bconv1x1_kernel<2><<<blocks, 256, lds, s>>>(a); break;
    case 8: bconv1x1_kernel<4><<<blocks, 256, lds, s>>>(a); break;
    default: return hipErrorInvalidValue;  // not reachable: bconv1x1_supported
  }
  return hipGetLastError();
}

}  // namespace bnn
