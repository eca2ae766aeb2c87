// Real-valued first layer with packed +-1 weights (the paper's BCNN without
// input binarization, Table I / Table III): Eq. 3 with fp32 image values and
// +-1 weights, pad value 0.0, fp32 sums, then the threshold / flip / OR-pool
// epilogue shared with the binary conv.
//
// Lane = output pixel, wave = 64 pixels x 32 filters (one output word per
// lane), pooled windows on lane quads as in the binary conv.  Each image
// value is loaded once per lane and added to or subtracted from the 32 filter
// sums according to the (wave-uniform) weight bits: one sign flip and one add
// per multiply-accumulate.
#include "kernels.hpp"

namespace bnn {
namespace {

struct FconvArgs {
  const float* in;
  const uint32_t* w;
  const int32_t* thr;
  const uint32_t* flip;
  float* sums;
  uint32_t* bits;
  int32_t N, H, W, C, Cw, F, Fw, KH, KW, pad, Ho, Wo, Hp, Wp;
  int32_t fstride;  // words per filter, KH*KW*Cw
  int32_t items;
};

template <bool POOL, bool FULL>
__global__ __launch_bounds__(256) void fconv_binw_kernel(FconvArgs a) {
  const int lane = threadIdx.x & 63;
  const int fg = blockIdx.y * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (fg >= a.Fw) return;  // wave-uniform, no barrier in this kernel
  const int nf = FULL ? 32 : min(32, a.F - fg * 32);

  int n, i, j, item;
  bool valid;
  if constexpr (POOL) {
    item = blockIdx.x * 16 + (lane >> 2);
    valid = item < a.items;
    const int p = valid ? item : 0;
    const int jp = p % a.Wp;
    const int t = p / a.Wp;
    const int ip = t % a.Hp;
    n = t / a.Hp;
    i = 2 * ip + ((lane >> 1) & 1);
    j = 2 * jp + (lane & 1);
  } else {
    item = blockIdx.x * 64 + lane;
    valid = item < a.items;
    const int m = valid ? item : 0;
    j = m % a.Wo;
    const int t = m / a.Wo;
    i = t % a.Ho;
    n = t / a.Ho;
  }

  float acc[32];
#pragma unroll
  for (int f = 0; f < 32; ++f) acc[f] = 0.0f;
  const uint32_t* wg = a.w + static_cast<size_t>(fg) * 32 * a.fstride;
  for (int kh = 0; kh < a.KH; ++kh) {
    const int hi = i + kh - a.pad;
    for (int kw = 0; kw < a.KW; ++kw) {
      const int wi = j + kw - a.pad;
      const bool inside = valid && static_cast<unsigned>(hi) < static_cast<unsigned>(a.H) &&
                          static_cast<unsigned>(wi) < static_cast<unsigned>(a.W);
      const float* xp = a.in + (static_cast<size_t>(n * a.H + hi) * a.W + wi) * a.C;
      const uint32_t* wt = wg + (kh * a.KW + kw) * a.Cw;
      for (int c = 0; c < a.C; ++c) {
        const float x = inside ? xp[c] : 0.0f;
        const uint32_t xb = __float_as_uint(x);
        const int cw = c >> 5;
        const int sh = 31 - (c & 31);
#pragma unroll
        for (int f = 0; f < 32; ++f) {
          if (FULL || f < nf) {
            // weight bit 1 -> +x, bit 0 -> -x (flip the fp32 sign bit)
            const uint32_t sgn = ((~wt[f * a.fstride + cw] >> sh) & 1u) << 31;
            acc[f] += __uint_as_float(xb ^ sgn);
          }
        }
      }
    }
  }

  if (a.sums && valid) {
    float* sp = a.sums + (static_cast<size_t>(n * a.Ho + i) * a.Wo + j) * a.F + fg * 32;
#pragma unroll
    for (int f = 0; f < 32; ++f)
      if (FULL || f < nf) sp[f] = acc[f];
  }
  if (a.bits) {
    const int32_t* th = a.thr + fg * 32;
    uint32_t word = 0;
#pragma unroll
    for (int f = 0; f < 32; ++f)
      if (FULL || f < nf)
        word |= static_cast<uint32_t>(acc[f] >= static_cast<float>(th[f])) << (31 - f);
    if (a.flip) word ^= a.flip[fg];
    if (!FULL && nf < 32) word &= ~0u << (32 - nf);
    if constexpr (POOL) {
      word |= __shfl_xor(word, 1);
      word |= __shfl_xor(word, 2);
      if ((lane & 3) == 0 && valid) a.bits[static_cast<size_t>(item) * a.Fw + fg] = word;
    } else {
      if (valid) a.bits[static_cast<size_t>(item) * a.Fw + fg] = word;
    }
  }
}

hipError_t run_fconv(const ConvGeom& g, bool pool, const float* in,
                     const uint32_t* w, const int32_t* thr,
                     const uint32_t* flip, float* sums, uint32_t* bits,
                     hipStream_t s) {
  FconvArgs a;
  a.in = in;
  a.w = w;
  a.thr = thr;
  a.flip = flip;
  a.sums = sums;
  a.bits = bits;
  a.N = g.N;
  a.H = g.H;
  a.W = g.W;
  a.C = g.C;
  a.Cw = g.Cw;
  a.F = g.F;
  a.Fw = g.Fw;
  a.KH = g.KH;
  a.KW = g.KW;
  a.pad = g.pad;
  a.Ho = g.Ho;
  a.Wo = g.Wo;
  a.Hp = g.Hp;
  a.Wp = g.Wp;
  a.fstride = g.KH * g.KW * g.Cw;
  a.items = pool ? g.N * g.Hp * g.Wp : g.N * g.Ho * g.Wo;
  const int per_block = pool ? 16 : 64;
  const int wpb = g.Fw < 4 ? g.Fw : 4;
  dim3 grid(static_cast<unsigned>((a.items + per_block - 1) / per_block),
            static_cast<unsigned>((g.Fw + wpb - 1) / wpb));
  dim3 block(64 * wpb);
  const bool full = (g.F & 31) == 0;
  if (pool && full)
    fconv_binw_kernel<true, true><<<grid, block, 0, s>>>(a);
  else if (pool)
    fconv_binw_kernel<true, false><<<grid, block, 0, s>>>(a);
  else if (full)
    fconv_binw_kernel<false, true><<<grid, block, 0, s>>>(a);
  else
    fconv_binw_kernel<false, false><<<grid, block, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_fconv_binw(const ConvGeom& g, const float* in,
                             const uint32_t* w, const int32_t* thr,
                             const uint32_t* flip, float* sums,
                             uint32_t* bits, hipStream_t s) {
  if (g.pool == 2 && sums && ((g.Ho & 1) || (g.Wo & 1))) {
    hipError_t e = run_fconv(g, false, in, w, thr, flip, sums, nullptr, s);
    if (e != hipSuccess || !bits) return e;
    return run_fconv(g, true, in, w, thr, flip, nullptr, bits, s);
  }
  return run_fconv(g, g.pool == 2, in, w, thr, flip, sums, bits, s);
}

}  // namespace bnn
