// First binary conv over a real-valued image that is binarized on the fly.
//
// The image is thresholded per channel, bit = (x + T_c) > 0 (the input
// binarization of §II-C), and convolved with packed +-1 filters, pad -1.
// When a whole window of KH x KW x C values fits in one 32-bit word
// (KH*KW*C <= 32; the 3x3x3 RGB layer has 27), the window itself is packed:
// this is the paper's patch packing (Algorithm 1) with B = KH*KW*C bits per
// word instead of one word per tap.  Each dot product of Eq. 4 is then a
// single XOR + popcount, against KH*KW of them (one per tap, 3 valid bits
// each) in the channel-packed layout.
//
// A block covers an 8 x 32 tile of output pixels, one per thread.  Its
// threads first threshold the input tile plus halo into C-bit codes in LDS
// (taps outside the image stay 0, the -1 pad value), then each builds its
// pixel's patch word from LDS.  The filters are turned into patch words the
// same way, once per block, together with a per-filter bias b = -q - 1 where
// q = floor((K - thr) / 2): then S >= thr <=> popcount(a ^ w) <= q <=>
// popcount(a ^ w) + b < 0, so v_bcnt with accumulate yields the output bit
// in its sign, and v_alignbit shifts it into the output word: three vector
// instructions per (pixel, filter).  2x2 OR-pooling uses quad shuffles as in
// the other binary kernels.
#include "kernels.hpp"

namespace bnn {
namespace {

constexpr int kTH = 8, kTW = 32;  // output tile rows x columns (256 threads)
constexpr int kFB = 256;          // filters staged in LDS per round
constexpr int kMaxTile = (kTH + 31) * (kTW + 31);  // KH * KW <= 32

struct PatchArgs {
  const float* x;
  const float* offset;
  const uint32_t* w;
  const int32_t* thr;
  const uint32_t* flip;
  int32_t* sums;
  uint32_t* bits;
  int32_t N, H, W, C, F, Fw, KH, KW, pad, Ho, Wo;
  int32_t P;           // KH * KW * C, bits per patch word
  int32_t tiles_x;     // tiles per output row
  int32_t tiles_y;     // tiles per output column
};

template <bool POOL, bool SUMS, bool BITS>
__global__ __launch_bounds__(256) void bconv_patch_kernel(PatchArgs a) {
  __shared__ uint32_t tile[kMaxTile];
  __shared__ uint32_t wpat[kFB];
  __shared__ int32_t wbias[kFB];

  const int t = threadIdx.x;
  int b = blockIdx.x;
  const int bx = b % a.tiles_x;
  b /= a.tiles_x;
  const int by = b % a.tiles_y;
  const int n = b / a.tiles_y;
  const int i0 = by * kTH, j0 = bx * kTW;

  // Threshold the input tile (plus halo) into C-bit codes, channel 0 in the
  // code's highest bit.
  const int TR = kTH + a.KH - 1, TC = kTW + a.KW - 1;
  for (int e = t; e < TR * TC; e += 256) {
    const int r = e / TC, cc = e - r * TC;
    const int gi = i0 - a.pad + r, gj = j0 - a.pad + cc;
    uint32_t code = 0;
    if (gi >= 0 && gi < a.H && gj >= 0 && gj < a.W) {
      const float* px = a.x + ((static_cast<size_t>(n) * a.H + gi) * a.W + gj) * a.C;
      for (int c = 0; c < a.C; ++c) {
        const float v = px[c] + (a.offset ? a.offset[c] : 0.0f);
        code |= static_cast<uint32_t>(v > 0.0f) << (a.C - 1 - c);
      }
    }
    tile[e] = code;
  }

  // This thread's output pixel; with pooling, lanes 4q..4q+3 are one window.
  int oy, ox;
  if constexpr (POOL) {
    const int win = t >> 2, q = t & 3;
    oy = 2 * (win / (kTW / 2)) + (q >> 1);
    ox = 2 * (win % (kTW / 2)) + (q & 1);
  } else {
    oy = t / kTW;
    ox = t % kTW;
  }
  const int i = i0 + oy, j = j0 + ox;
  const bool valid = i < a.Ho && j < a.Wo;
  __syncthreads();

  // Patch word: tap s = kh * KW + kw holds bits 31 - s*C ... 32 - (s+1)*C.
  uint32_t patch = 0;
  for (int kh = 0; kh < a.KH; ++kh)
    for (int kw = 0; kw < a.KW; ++kw) {
      const int s = kh * a.KW + kw;
      patch |= tile[(oy + kh) * TC + (ox + kw)] << (32 - (s + 1) * a.C);
    }

  const int Wp = POOL ? a.Wo / 2 : a.Wo;
  const int Hp = POOL ? a.Ho / 2 : a.Ho;
  for (int f0 = 0; f0 < a.F; f0 += kFB) {
    const int nf = min(kFB, a.F - f0);
    __syncthreads();  // previous round's filters are no longer read
    if (t < kFB) {
      uint32_t wp = 0;
      int32_t bias = 0;
      if (t < nf) {
        const int f = f0 + t;
        const uint32_t* wf = a.w + static_cast<size_t>(f) * a.KH * a.KW;  // one word per tap
        for (int s = 0; s < a.KH * a.KW; ++s)
          wp |= (wf[s] >> (32 - a.C)) << (32 - (s + 1) * a.C);
        if constexpr (BITS) {
          // q = floor((K - thr) / 2), clamped to [-1, K]
          const int64_t d = static_cast<int64_t>(a.P) - a.thr[f];
          int64_t q = d >= 0 ? d / 2 : -((1 - d) / 2);
          q = q < -1 ? -1 : (q > a.P ? a.P : q);
          bias = static_cast<int32_t>(-q - 1);
        }
      }
      wpat[t] = wp;
      wbias[t] = bias;
    }
    __syncthreads();

    for (int g = 0; g < nf; g += 32) {
      const int fw = (f0 + g) >> 5;
      if constexpr (SUMS) {
        if (valid) {
          int32_t* sp = a.sums + ((static_cast<size_t>(n) * a.Ho + i) * a.Wo + j) * a.F + f0 + g;
          const int m = min(32, nf - g);
          for (int k = 0; k < m; ++k)
            sp[k] = a.P - 2 * static_cast<int32_t>(__builtin_popcount(patch ^ wpat[g + k]));
        }
      }
      if constexpr (BITS) {
        uint32_t word = 0;
#pragma unroll
        for (int k = 0; k < 32; ++k) {
          const uint32_t d = static_cast<uint32_t>(__builtin_popcount(patch ^ wpat[g + k])) +
                             static_cast<uint32_t>(wbias[g + k]);
          word = __builtin_amdgcn_alignbit(word, d, 31);
        }
        if (a.flip) word ^= a.flip[fw];
        if (fw == a.Fw - 1) word &= tail_mask(a.F);
        if constexpr (POOL) {
          word |= __shfl_xor(word, 1);
          word |= __shfl_xor(word, 2);
          if ((t & 3) == 0 && (i >> 1) < Hp && (j >> 1) < Wp)
            a.bits[((static_cast<size_t>(n) * Hp + (i >> 1)) * Wp + (j >> 1)) * a.Fw + fw] = word;
        } else {
          if (valid) a.bits[((static_cast<size_t>(n) * a.Ho + i) * a.Wo + j) * a.Fw + fw] = word;
        }
      }
    }
  }
}

template <bool POOL>
hipError_t launch_pool(const PatchArgs& a, dim3 grid, hipStream_t s) {
  if (a.sums && a.bits)
    bconv_patch_kernel<POOL, true, true><<<grid, 256, 0, s>>>(a);
  else if (a.sums)
    bconv_patch_kernel<POOL, true, false><<<grid, 256, 0, s>>>(a);
  else
    bconv_patch_kernel<POOL, false, true><<<grid, 256, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace

bool bconv_patch_supported(const ConvGeom& g) {
  return int64_t{g.KH} * g.KW * g.C <= 32;
}

hipError_t launch_bconv_patch(const ConvGeom& g, const float* x, const float* offset,
                              const uint32_t* w, const int32_t* thr, const uint32_t* flip,
                              int32_t* sums, uint32_t* bits, hipStream_t s) {
  PatchArgs a;
  a.x = x;
  a.offset = offset;
  a.w = w;
  a.thr = thr;
  a.flip = flip;
  a.sums = sums;
  a.bits = bits;
  a.N = g.N;
  a.H = g.H;
  a.W = g.W;
  a.C = g.C;
  a.F = g.F;
  a.Fw = g.Fw;
  a.KH = g.KH;
  a.KW = g.KW;
  a.pad = g.pad;
  a.Ho = g.Ho;
  a.Wo = g.Wo;
  a.P = g.KH * g.KW * g.C;
  a.tiles_x = (g.Wo + kTW - 1) / kTW;
  a.tiles_y = (g.Ho + kTH - 1) / kTH;
  const dim3 grid(static_cast<unsigned>(int64_t{g.N} * a.tiles_x * a.tiles_y));
  return g.pool == 2 ? launch_pool<true>(a, grid, s) : launch_pool<false>(a, grid, s);
}

}  // namespace bnn
