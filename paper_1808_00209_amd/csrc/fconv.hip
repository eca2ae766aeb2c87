// Real-valued first layer with packed +-1 weights (the paper's BCNN without
// input binarization, Table I / Table III): Eq. 3 with fp32 image values and
// +-1 weights, pad value 0.0, fp32 sums, then the threshold / flip / OR-pool
// epilogue shared with the binary conv.  Every product with a +-1 weight is
// exact (the matrix-core path splits x into three bf16 parts), so a sum
// differs from the exact one only by fp32 rounding in the accumulation; the
// comparison S >= thr with the integer threshold is exact (thr_ceil_f32).
//
// Lane = output pixel, wave = 64 pixels x 32 filters (one output word per
// lane), pooled windows on lane quads as in the binary conv.  Each image
// value is loaded once per lane and added to or subtracted from the 32 filter
// sums according to the (wave-uniform) weight bits: one sign flip and one add
// per multiply-accumulate.

#include "fp32_split.hpp"
#include "kernels.hpp"
#include "lane_ops.hpp"

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
        word |= static_cast<uint32_t>(acc[f] >= thr_ceil_f32(th[f])) << (31 - f);
    if (a.flip) word ^= a.flip[fg];
    if (!FULL && nf < 32) word &= ~0u << (32 - nf);
    if constexpr (POOL) {
      word = or_quad(word);
      if ((lane & 3) == 0 && valid) a.bits[static_cast<size_t>(item) * a.Fw + fg] = word;
    } else {
      if (valid) a.bits[static_cast<size_t>(item) * a.Fw + fg] = word;
    }
  }
}

// Fast path for few input channels (RGB): lane = filter, so each lane keeps
// its own KH*KW*C weights as +-1.0 floats in registers, and the image values
// of the wave's pixels are wave-uniform (scalar loads).  Every multiply-
// accumulate is then one v_fmac_f32 with an SGPR operand.  A wave covers 64
// filters x a 2x8 tile of output pixels; the 64 threshold bits of a pixel
// come from one ballot (two output words), and 2x2 pooling ORs the ballots
// of the window's four pixels.
typedef __attribute__((address_space(4))) const float cf32;

constexpr int kTileH = 2;
constexpr int kTileW = 8;

// acc[q] += sum over kw, c of x[q + kw][c] * w[kw][c] for one kernel row.
template <int C, int KW>
__device__ __forceinline__ void row_fma(float (&acc)[kTileW], const float (&xs)[kTileW + KW - 1][C],
                                        const float* w) {
#pragma unroll
  for (int kw = 0; kw < KW; ++kw)
#pragma unroll
    for (int c = 0; c < C; ++c)
#pragma unroll
      for (int q = 0; q < kTileW; ++q) acc[q] = __builtin_fmaf(xs[q + kw][c], w[kw * C + c], acc[q]);
}

template <int C, int KH, int KW, bool POOL>
__global__ __launch_bounds__(256) void fconv_lanef_kernel(FconvArgs a) {
  const int lane = threadIdx.x & 63;
  const int fg = blockIdx.y * (blockDim.x >> 6) + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (fg * 64 >= a.F) return;  // wave-uniform, no barrier in this kernel
  const int f = fg * 64 + lane;
  const bool fvalid = f < a.F;

  // This lane's weights as +-1.0 (bit 1 -> +1).
  float wv[KH * KW * C];
  {
    const uint32_t* wr = a.w + static_cast<size_t>(fvalid ? f : 0) * a.fstride;
#pragma unroll
    for (int t = 0; t < KH * KW; ++t) {
#pragma unroll
      for (int c = 0; c < C; ++c) {
        const uint32_t word = wr[t * a.Cw + (c >> 5)];
        wv[t * C + c] = ((word >> (31 - (c & 31))) & 1u) ? 1.0f : -1.0f;
      }
    }
  }
  const float th = thr_ceil_f32(fvalid && a.thr ? a.thr[f] : 0);

  // Output tile.
  const int tiles_w = (a.Wo + kTileW - 1) / kTileW;
  const int tiles_h = (a.Ho + kTileH - 1) / kTileH;
  int b = blockIdx.x;
  const int tw = b % tiles_w;
  b /= tiles_w;
  const int tt = b % tiles_h;
  const int n = b / tiles_h;
  const int i0 = tt * kTileH;
  const int j0 = tw * kTileW;
  cf32* img = (cf32*)(a.in) + static_cast<size_t>(n) * a.H * a.W * C;

  uint64_t mask[kTileH][kTileW];
#pragma unroll
  for (int r = 0; r < kTileH; ++r) {
    const int i = i0 + r;
    float acc[kTileW];
#pragma unroll
    for (int q = 0; q < kTileW; ++q) acc[q] = 0.0f;
#pragma unroll
    for (int kh = 0; kh < KH; ++kh) {
      const int hi = i + kh - a.pad;
      if (hi < 0 || hi >= a.H || i >= a.Ho) continue;  // uniform
      cf32* row = img + static_cast<size_t>(hi) * a.W * C;
      const int cfirst = j0 - a.pad;
      // The multiply-accumulates sit inside each branch so that the image
      // values stay in SGPRs (no merge of the two paths into VGPRs).
      if (cfirst >= 0 && cfirst + kTileW + KW - 1 <= a.W) {
        // Interior: one contiguous run of (kTileW + KW - 1) * C values.
        cf32* seg = row + cfirst * C;
        float xs[kTileW + KW - 1][C];
#pragma unroll
        for (int q = 0; q < kTileW + KW - 1; ++q)
#pragma unroll
          for (int c = 0; c < C; ++c) xs[q][c] = seg[q * C + c];
        row_fma<C, KW>(acc, xs, wv + kh * KW * C);
      } else {
        // Image border: columns outside [0, W) read as 0.0 (the pad value).
        float xs[kTileW + KW - 1][C];
#pragma unroll
        for (int q = 0; q < kTileW + KW - 1; ++q) {
          const int col = cfirst + q;
          const bool ok = col >= 0 && col < a.W;
          const int cl = min(max(col, 0), a.W - 1);
#pragma unroll
          for (int c = 0; c < C; ++c) {
            const float v = row[cl * C + c];
            xs[q][c] = ok ? v : 0.0f;
          }
        }
        row_fma<C, KW>(acc, xs, wv + kh * KW * C);
      }
    }
#pragma unroll
    for (int q = 0; q < kTileW; ++q) {
      const int j = j0 + q;
      const bool pix = i < a.Ho && j < a.Wo;
      if (a.sums && pix && fvalid)
        a.sums[(static_cast<size_t>(n * a.Ho + i) * a.Wo + j) * a.F + f] = acc[q];
      mask[r][q] = __ballot(fvalid && acc[q] >= th);
    }
  }
  if (!a.bits) return;
  // Two output words per pixel: filters 64 fg + 0..31 and + 32..63.
  const int w0 = 2 * fg;
  const uint32_t fl0 = a.flip ? a.flip[w0] : 0u;
  const uint32_t fl1 = (a.flip && w0 + 1 < a.Fw) ? a.flip[w0 + 1] : 0u;
  const uint32_t tm0 = (w0 == a.Fw - 1) ? tail_mask(a.F) : ~0u;
  const uint32_t tm1 = (w0 + 1 == a.Fw - 1) ? tail_mask(a.F) : ~0u;
  if constexpr (POOL) {
#pragma unroll
    for (int q = 0; q < kTileW; q += 2) {
      const int ip = i0 / 2, jp = (j0 + q) / 2;
      if (ip >= a.Hp || jp >= a.Wp) continue;
      uint32_t lo = 0, hi = 0;
#pragma unroll
      for (int r = 0; r < 2; ++r)
#pragma unroll
        for (int d = 0; d < 2; ++d) {
          lo |= __brev(static_cast<uint32_t>(mask[r][q + d])) ^ fl0;
          hi |= __brev(static_cast<uint32_t>(mask[r][q + d] >> 32)) ^ fl1;
        }
      uint32_t* op = a.bits + (static_cast<size_t>(n * a.Hp + ip) * a.Wp + jp) * a.Fw + w0;
      if (lane == 0) op[0] = lo & tm0;
      if (lane == 1 && w0 + 1 < a.Fw) op[1] = hi & tm1;
    }
  } else {
#pragma unroll
    for (int r = 0; r < kTileH; ++r)
#pragma unroll
      for (int q = 0; q < kTileW; ++q) {
        const int i = i0 + r, j = j0 + q;
        if (i >= a.Ho || j >= a.Wo) continue;
        const uint32_t lo = (__brev(static_cast<uint32_t>(mask[r][q])) ^ fl0) & tm0;
        const uint32_t hi = (__brev(static_cast<uint32_t>(mask[r][q] >> 32)) ^ fl1) & tm1;
        uint32_t* op = a.bits + (static_cast<size_t>(n * a.Ho + i) * a.Wo + j) * a.Fw + w0;
        if (lane == 0) op[0] = lo;
        if (lane == 1 && w0 + 1 < a.Fw) op[1] = hi;
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

// Matrix-core path for few input channels: the block stages a zero-padded
// (8 + KH - 1) x (32 + KW - 1) x C input tile in LDS (the pad value 0.0 comes
// for free), splits every staged value x exactly into three bf16 parts
// (split3), and v_mfma_f32_16x16x32_bf16 multiplies them by the +-1 weights
// into fp32 accumulators: every product is exact and only the fp32 additions
// round.  For inputs on the 2^-16 grid whose window sums of |x| stay below
// 2^8 every partial sum is a multiple of 2^-16 below 2^8, so the sums are
// exact in any order.
// Block = 4 waves = an 8 x 32 tile of output pixels (4 x 16 2x2 windows when
// pooling) x FG groups of 64 filters; the result layout and epilogue follow
// the binary matrix-core kernel (lane: one pixel, four filters).  The +-1
// weight operands of the FG groups are built once per block into LDS by all
// its threads (their global loads overlap the input tile's), and every wave
// reads them with one ds_read_b128 per operand; the bf16 parts of each
// pixel window are built once and reused by every filter group.
constexpr int kMfTileH = 8;
constexpr int kMfTileW = 32;

typedef float v4f __attribute__((ext_vector_type(4)));

template <int C, int KH, int KW, bool POOL, bool FULL, int FG>
__global__ __launch_bounds__(256) void fconv_mfma_kernel(FconvArgs a) {
  constexpr int K = KH * KW * C;
  constexpr int KC = (K + 31) / 32;  // k-chunks of 32
  constexpr int LW = kMfTileW + KW - 1;
  constexpr int LH = kMfTileH + KH - 1;
  __shared__ float tile[LH * LW * C];
  __shared__ v8bf wop[FG][KC][4][64];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int q = lane >> 4, c = lane & 15;
  const int tiles_w = (a.Wo + kMfTileW - 1) / kMfTileW;
  const int tiles_h = (a.Ho + kMfTileH - 1) / kMfTileH;
  int b = blockIdx.x;
  const int tw = b % tiles_w;
  b /= tiles_w;
  const int th_ = b % tiles_h;
  const int n = b / tiles_h;
  const int i0 = th_ * kMfTileH, j0 = tw * kMfTileW;
  const int fb = blockIdx.y * 64 * FG;

  // Weight operands: thread t builds, for each group g and k-chunk kc, the
  // A operand of filter tile tf = t / 64 for lane (q', c') = t % 64: row
  // filter fb + 64 g + 16 tf + c', the 8 k values 32 kc + 8 q' + e, as +-1
  // (0 past K or F).
  {
    const int tf = threadIdx.x >> 6, qq = (threadIdx.x >> 4) & 3, cc = threadIdx.x & 15;
#pragma unroll
    for (int g = 0; g < FG; ++g)
#pragma unroll
    for (int kc = 0; kc < KC; ++kc) {
      const int f = fb + 64 * g + 16 * tf + cc;
      uint16_t op[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int k = 32 * kc + 8 * qq + e;
        const int tap = k / C, ch = k - (k / C) * C;
        const bool ok = k < K && (FULL || f < a.F);
        // unconditional load from a clamped (valid) address, then select
        const uint32_t word = a.w[static_cast<size_t>(ok ? f : 0) * a.fstride +
                                  (ok ? tap * a.Cw + (ch >> 5) : 0)];
        const bool one = (word >> (31 - (ch & 31))) & 1u;
        op[e] = ok ? (one ? kBf16One : kBf16MinusOne) : kBf16Zero;
      }
      wop[g][kc][tf][threadIdx.x & 63] = bf16x8(op);
    }
  }

  // The block's thresholds and flip words go to LDS with the input tile, so
  // their loads overlap it rather than following the MFMAs.
  __shared__ float thl[FG * 64];
  __shared__ uint32_t fll[FG * 2];
  if (a.bits && threadIdx.x < FG * 64) {
    const int f = fb + static_cast<int>(threadIdx.x);
    thl[threadIdx.x] = thr_ceil_f32((FULL || f < a.F) ? a.thr[f] : 0);
  }
  if (threadIdx.x < FG * 2) {
    const int wi = fb / 32 + static_cast<int>(threadIdx.x);
    fll[threadIdx.x] = (a.flip && wi < a.Fw) ? a.flip[wi] : 0u;
  }

  // Stage the input tile (zero outside the image).
  for (int e = threadIdx.x; e < LH * LW * C; e += 256) {
    const int ch = e % C;
    const int t = e / C;
    const int col = t % LW, row = t / LW;
    const int hi = i0 + row - a.pad, wi = j0 + col - a.pad;
    float v = 0.0f;
    if (hi >= 0 && hi < a.H && wi >= 0 && wi < a.W)
      v = a.in[((static_cast<size_t>(n) * a.H + hi) * a.W + wi) * C + ch];
    tile[e] = v;
  }

  // LDS offset of this lane's 8 k values relative to a pixel's window origin.
  int rel[KC][8];
#pragma unroll
  for (int kc = 0; kc < KC; ++kc)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int k = 32 * kc + 8 * q + e;
      const int tap = k / C, ch = k - (k / C) * C;
      const int kh = tap / KW, kw = tap - (tap / KW) * KW;
      rel[kc][e] = k < K ? (kh * LW + kw) * C + ch : -1;
    }
  __syncthreads();

  // This wave's 4 pixel tiles of 16: position of lane c's pixel in the block tile.
  int pr[4], pc[4];
#pragma unroll
  for (int tp = 0; tp < 4; ++tp) {
    if constexpr (POOL) {
      const int win = wave * 16 + tp * 4 + (c >> 2);  // 4 x 16 windows
      pr[tp] = 2 * (win / 16) + ((c >> 1) & 1);
      pc[tp] = 2 * (win % 16) + (c & 1);
    } else {
      pr[tp] = 2 * wave + (tp >> 1);
      pc[tp] = 16 * (tp & 1) + c;
    }
  }
  // bf16 parts of the 4 pixel windows (B operands), shared by all groups.
  v8bf xp[3][KC][4];
#pragma unroll
  for (int tp = 0; tp < 4; ++tp) {
    const int pbase = (pr[tp] * LW + pc[tp]) * C;
#pragma unroll
    for (int kc = 0; kc < KC; ++kc) {
      uint16_t p0[8], p1[8], p2[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float xv = tile[pbase + max(rel[kc][e], 0)];
        const Split3 sp = split3(rel[kc][e] >= 0 ? xv : 0.0f);
        p0[e] = bf16_bits(sp.p0);
        p1[e] = bf16_bits(sp.p1);
        p2[e] = bf16_bits(sp.p2);
      }
      xp[0][kc][tp] = bf16x8(p0);
      xp[1][kc][tp] = bf16x8(p1);
      xp[2][kc][tp] = bf16x8(p2);
    }
  }

#pragma unroll
  for (int g = 0; g < FG; ++g) {
    const int f0 = fb + 64 * g;
    if (!FULL && f0 >= a.F) break;  // block-uniform
    v4f acc[4][4];
#pragma unroll
    for (int tf = 0; tf < 4; ++tf)
#pragma unroll
      for (int tp = 0; tp < 4; ++tp) acc[tf][tp] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kc = 0; kc < KC; ++kc) {
      v8bf wa[4];
#pragma unroll
      for (int tf = 0; tf < 4; ++tf) wa[tf] = wop[g][kc][tf][lane];
#pragma unroll
      for (int pt = 0; pt < 3; ++pt)
#pragma unroll
        for (int tf = 0; tf < 4; ++tf)
#pragma unroll
          for (int tp = 0; tp < 4; ++tp)
            acc[tf][tp] =
                __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa[tf], xp[pt][kc][tp], acc[tf][tp], 0, 0, 0);
    }

    // Epilogue: lane (q, c) holds pixel c of each tile and filters 16 tf + 4 q + r.
    const int nf = FULL ? 64 : min(64, a.F - f0);
#pragma unroll
    for (int tp = 0; tp < 4; ++tp) {
      const int i = i0 + pr[tp], j = j0 + pc[tp];
      const bool pix = i < a.Ho && j < a.Wo;
      if (a.sums && pix) {
        float* sp = a.sums + (static_cast<size_t>(n * a.Ho + i) * a.Wo + j) * a.F + f0 + 4 * q;
#pragma unroll
        for (int tf = 0; tf < 4; ++tf)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (FULL || tf * 16 + 4 * q + r < nf) sp[tf * 16 + r] = acc[tf][tp][r];
      }
    }
    if (!a.bits) continue;
    float thf[4][4];
#pragma unroll
    for (int tf = 0; tf < 4; ++tf)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int fl = tf * 16 + 4 * q + r;
        thf[tf][r] = thl[64 * g + fl];
      }
    const int w0 = f0 / 32;
#pragma unroll
    for (int tp = 0; tp < 4; ++tp) {
      uint32_t word[2] = {0u, 0u};
#pragma unroll
      for (int tf = 0; tf < 4; ++tf)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int fl = tf * 16 + 4 * q + r;
          const bool on = acc[tf][tp][r] >= thf[tf][r] && (FULL || fl < nf);
          word[tf >> 1] |= static_cast<uint32_t>(on) << (31 - (16 * (tf & 1) + 4 * q + r));
        }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        word[h] = or_xor32(or_xor16(word[h]));
        if (FULL || w0 + h < a.Fw) {
          word[h] ^= fll[2 * g + h];
          if (!FULL && w0 + h == a.Fw - 1) word[h] &= tail_mask(a.F);
        }
        if constexpr (POOL) {
          word[h] = or_quad(word[h]);
        }
      }
      const int i = i0 + pr[tp], j = j0 + pc[tp];
      if constexpr (POOL) {
        const int ip = i >> 1, jp = j >> 1;
        if (q == 0 && (c & 3) == 0 && ip < a.Hp && jp < a.Wp) {
          uint32_t* op = a.bits + (static_cast<size_t>(n * a.Hp + ip) * a.Wp + jp) * a.Fw + w0;
          if (FULL)
            *reinterpret_cast<uint2*>(op) = make_uint2(word[0], word[1]);
          else {
            op[0] = word[0];
            if (w0 + 1 < a.Fw) op[1] = word[1];
          }
        }
      } else {
        if (q == 0 && i < a.Ho && j < a.Wo) {
          uint32_t* op = a.bits + (static_cast<size_t>(n * a.Ho + i) * a.Wo + j) * a.Fw + w0;
          if (FULL)
            *reinterpret_cast<uint2*>(op) = make_uint2(word[0], word[1]);
          else {
            op[0] = word[0];
            if (w0 + 1 < a.Fw) op[1] = word[1];
          }
        }
      }
    }
  }
}

template <int C>
hipError_t run_fmfma(const ConvGeom& g, bool pool, const float* in, const uint32_t* w,
                     const int32_t* thr, const uint32_t* flip, float* sums, uint32_t* bits,
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
  a.items = 0;
  const unsigned tiles = static_cast<unsigned>(g.N) * ((g.Ho + kMfTileH - 1) / kMfTileH) *
                         ((g.Wo + kMfTileW - 1) / kMfTileW);
  // Filter groups of 64 per block: 2 (the input tile and the bf16 parts
  // then serve 128 filters) only for grids that still have >= 4096 waves;
  // on smaller grids the extra parallelism of one group per block wins.
  const int fg =
      (g.F >= 128 && static_cast<int64_t>(tiles) * ((g.F + 127) / 128) * 4 >= 4096) ? 2 : 1;
  const bool full = g.F % 64 == 0;
  dim3 grid(tiles, static_cast<unsigned>((g.F + 64 * fg - 1) / (64 * fg)));
  if (fg == 2) {
    if (pool && full)
      fconv_mfma_kernel<C, 3, 3, true, true, 2><<<grid, dim3(256), 0, s>>>(a);
    else if (pool)
      fconv_mfma_kernel<C, 3, 3, true, false, 2><<<grid, dim3(256), 0, s>>>(a);
    else if (full)
      fconv_mfma_kernel<C, 3, 3, false, true, 2><<<grid, dim3(256), 0, s>>>(a);
    else
      fconv_mfma_kernel<C, 3, 3, false, false, 2><<<grid, dim3(256), 0, s>>>(a);
  } else {
    if (pool && full)
      fconv_mfma_kernel<C, 3, 3, true, true, 1><<<grid, dim3(256), 0, s>>>(a);
    else if (pool)
      fconv_mfma_kernel<C, 3, 3, true, false, 1><<<grid, dim3(256), 0, s>>>(a);
    else if (full)
      fconv_mfma_kernel<C, 3, 3, false, true, 1><<<grid, dim3(256), 0, s>>>(a);
    else
      fconv_mfma_kernel<C, 3, 3, false, false, 1><<<grid, dim3(256), 0, s>>>(a);
  }
  return hipGetLastError();
}

template <int C>
hipError_t run_lanef(const ConvGeom& g, bool pool, const float* in, const uint32_t* w,
                     const int32_t* thr, const uint32_t* flip, float* sums, uint32_t* bits,
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
  a.items = 0;
  const int fgroups = (g.F + 63) / 64;
  const int wpb = fgroups < 4 ? fgroups : 4;
  const unsigned tiles = static_cast<unsigned>(g.N) * ((g.Ho + kTileH - 1) / kTileH) *
                         ((g.Wo + kTileW - 1) / kTileW);
  dim3 grid(tiles, static_cast<unsigned>((fgroups + wpb - 1) / wpb));
  if (pool)
    fconv_lanef_kernel<C, 3, 3, true><<<grid, dim3(64 * wpb), 0, s>>>(a);
  else
    fconv_lanef_kernel<C, 3, 3, false><<<grid, dim3(64 * wpb), 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_fconv_binw(const ConvGeom& g, const float* in,
                             const uint32_t* w, const int32_t* thr,
                             const uint32_t* flip, float* sums,
                             uint32_t* bits, hipStream_t s) {
  // Few channels and a 3x3 kernel: the lane-per-filter kernel (its 2x8 pixel
  // tiles sit on even coordinates, so 2x2 windows never straddle tiles).
  if (g.KH == 3 && g.KW == 3 && g.C <= 4) {
    const bool pool = g.pool == 2;
    if (options().algo != BNN_ALGO_VALU) {
      // The matrix-core kernel's 8 x 32 pixel tiles sit on even coordinates.
      switch (g.C) {
        case 1: return run_fmfma<1>(g, pool, in, w, thr, flip, sums, bits, s);
        case 2: return run_fmfma<2>(g, pool, in, w, thr, flip, sums, bits, s);
        case 3: return run_fmfma<3>(g, pool, in, w, thr, flip, sums, bits, s);
        default: return run_fmfma<4>(g, pool, in, w, thr, flip, sums, bits, s);
      }
    }
    switch (g.C) {
      case 1: return run_lanef<1>(g, pool, in, w, thr, flip, sums, bits, s);
      case 2: return run_lanef<2>(g, pool, in, w, thr, flip, sums, bits, s);
      case 3: return run_lanef<3>(g, pool, in, w, thr, flip, sums, bits, s);
      default: return run_lanef<4>(g, pool, in, w, thr, flip, sums, bits, s);
    }
  }
  if (g.pool == 2 && sums && ((g.Ho & 1) || (g.Wo & 1))) {
    hipError_t e = run_fconv(g, false, in, w, thr, flip, sums, nullptr, s);
    if (e != hipSuccess || !bits) return e;
    return run_fconv(g, true, in, w, thr, flip, nullptr, bits, s);
  }
  return run_fconv(g, g.pool == 2, in, w, thr, flip, sums, bits, s);
}

}  // namespace bnn
