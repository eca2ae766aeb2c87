// The real-valued first layer (Eq. 3: fp32 image, +-1 weights, pad 0.0) and
// the binary conv after it (Eq. 4 on the first layer's output bits) in one
// launch, for the BCNN without input binarization (Table I): the first
// layer's output never goes to global memory.
//
// A block owns a TH x 32 tile of the second layer's output pixels of one
// image (TH = 8, or 4 on small grids; TH / 2 x 16 2x2 windows when it pools)
// and all of its filters (64 or 128; TH / 2 waves per 64 filters).
//   1. It stages the input tile the first layer needs for the (TH + 2) x
//      (32 + 2) pixels of the second layer's windows (halo of one pixel),
//      zero outside the image, with every value split once into three bf16
//      parts, x = p0 + p1 + p2 exactly (split3), plus both layers'
//      thresholds and the first layer's +-1 weight operands.  All global
//      loads are issued before the first LDS store.
//   2. All waves compute the first layer's outputs on that (TH + 2) x 34 tile with
//      v_mfma_f32_16x16x32_bf16 on the three parts (exact products, fp32
//      accumulation; exact sums in any order for inputs on the 2^-16 grid
//      whose window sums of |x| stay below 2^8), take
//      the sign bits of S - thr, OR the four lane rows' parts of the words
//      together (lane row q then holds word q of its pixel), flip, and store
//      each word in LDS already expanded to its fp4 operand.  Pixels outside
//      the first layer's output get the pad word 0 (-1) of the second conv.
//   3. Each wave takes 64 pixels (16 windows) x 64 filters of the second
//      layer on the fp4 matrix cores: activation operands straight from LDS
//      (no bounds tests: the halo holds the padding), weight words from
//      global memory, accumulators started at 0.5 - thr (the output bit is
//      the complement of the sign), OR-pool on lane quads and the packed
//      store.

#include <type_traits>

#include "fp32_split.hpp"
#include "fp4_expand.hpp"
#include "kernels.hpp"
#include "lane_ops.hpp"

namespace bnn {
namespace {

constexpr int kTW = 32;         // second-layer output tile width (height TH = 8 or 4)
constexpr int kAW = kTW + 2;    // first-layer tile width (second layer's windows)
constexpr int kIW = kAW + 2;    // input tile width (first layer's windows)

struct FbArgs {
  const float* in;
  const uint32_t* w0;
  const int32_t* thr0;
  const uint32_t* flip0;
  const uint32_t* w1;
  const int32_t* thr1;
  const uint32_t* flip1;
  uint32_t* bits;
  int32_t N, H, W;              // input image
  int32_t pad0, Ho0, Wo0;       // first layer
  int32_t pad1, Ho1, Wo1;       // second layer (before pooling)
  int32_t Hp, Wp;               // stored output (pooled dims when pooling)
  int32_t K1;                   // bits per second-layer window, 9 * F0
  int32_t w1_bytes;
  const int32_t* corr1;         // prepared w1 (PREP1): per-filter offsets B_f
  int32_t tiles_w, tiles_h;
  const float* offset;          // NPART = 1: per-channel thresholds T (or NULL)
};

constexpr uint32_t kRsrcWord3 = 0x00020000;
constexpr int64_t kCUs = 256;  // compute units of the chip

// PREP1: w1 holds the second layer's weights in the prepared operand form
// (bnn_prepare_weights: 16-byte entries [F1 / 32][9][F0 / 32][32], then the
// offsets corr1), so the second layer loads its A operands whole, and the
// first layer stores its bits as act_operand instead of expand_fp4 operands.
// TH: rows of the second layer's output tile, 8, or 4 on grids too small to
// fill the chip (half the workgroups' work each, for 1.25 times the
// first-layer work per output row).
// NPART = 3: the first layer is the real-valued one (fp32 input split into
// three bf16 parts, pad 0.0).  NPART = 1: the first layer is a binary conv
// over the input thresholded per channel (bit = x + T_c > 0, Sec. II-C), each
// value +-1.0 in bf16 and the pad -1, exactly the binary conv
// bnn_bconv2d_input computes with the same thresholds and flips.
template <int TH, int C0, int F0, int NFH, bool POOL, bool PREP1, int NPART>
__global__ __launch_bounds__(256 * NFH) void fconv_bconv_kernel(FbArgs a) {
  constexpr int kTH = TH;
  constexpr int kAH = kTH + 2;                // first-layer tile rows
  constexpr int kIH = kAH + 2;                // input tile rows
  constexpr int kAPix = kAH * kAW;            // 340 (TH = 8), 204 (TH = 4)
  constexpr int kATiles = (kAPix + 15) / 16;  // 16-pixel tiles of the first layer
  constexpr int PG = TH / 2;                  // 64-pixel groups of the second layer
  constexpr int NW2 = PG * NFH;               // second-layer waves
  // With 4-row tiles (small grids) the block has twice as many waves as the
  // second layer uses: the staging and the first layer spread over all of
  // them, the extra ones then stop.
  constexpr int NW = TH == 4 ? 2 * NW2 : NW2;  // waves
  constexpr int NT = 64 * NW;                 // threads
  constexpr int K0 = 9 * C0;
  constexpr int KC0 = (K0 + 31) / 32;  // first-layer k-chunks of 32
  constexpr int FT0 = F0 / 16;         // first-layer filter tiles of 16
  constexpr int CW1 = F0 / 32;         // words per first-layer output pixel
  constexpr int VW = CW1 % 4 == 0 ? 2 : 1;  // words per lane and k-step pair
  constexpr int NCH = CW1 / (2 * VW);       // chunks per tap
  constexpr int F1 = 64 * NFH;
  constexpr int FW1 = F1 / 32;

  constexpr int NX = kIH * kIW * C0;  // input values of the tile
  constexpr int XIT = NPART == 3 ? (NX + NT - 1) / NT : 1;
  constexpr int NPIX = kIH * kIW;     // input pixels of the tile
  constexpr int XIP = NPART == 1 ? (NPIX + NT - 1) / NT : 1;
  static_assert(NPART == 3 || K0 <= 32, "a thresholded window fits one word");

  // NPART = 3: the input tile as three bf16 parts and the first layer's
  // operands for v_mfma_f32_16x16x32_bf16.  NPART = 1: each input pixel's
  // C0 threshold bits (xcode) and each filter's K0 weight bits (wp0), for
  // v_mfma_scale_f32_32x32x64_f8f6f4 on +-1 fp4 operands.
  __shared__ uint16_t xs[NPART == 3 ? 3 : 1][NPART == 3 ? NX : 1];
  __shared__ v8bf wop[NPART == 3 ? FT0 : 1][KC0][64];
  __shared__ uint32_t xcode[NPART == 1 ? NPIX : 1];
  __shared__ uint32_t wp0[NPART == 1 ? F0 : 1];
  // First-layer output bits, each word already expanded to its fp4 operand:
  // word wi of tile pixel (r, c) at r RSX + c PSX + wi.  The spare entry per
  // pixel and the row stride (= 4 mod 8 entries) spread the 16-byte reads of
  // 8 neighbouring lanes (2 rows x 4 columns) over distinct banks.
  constexpr int PSX = CW1 + 1;
  constexpr int RSX = kAW * PSX + ((4 - (kAW * PSX) % 8) + 8) % 8;
  __shared__ v4i actx[kAH * RSX];
  __shared__ __attribute__((aligned(16))) float th0[F0];
  __shared__ uint32_t fl0[CW1];
  __shared__ float th1[F1];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int b = blockIdx.x;
  const int tw = b % a.tiles_w;
  b /= a.tiles_w;
  const int tht = b % a.tiles_h;
  const int n = b / a.tiles_h;
  const int i0 = tht * kTH, j0 = tw * kTW;  // second-layer output origin
  const int r0 = i0 - a.pad1, c0 = j0 - a.pad1;  // first-layer tile origin
  const int y0 = r0 - a.pad0, x0 = c0 - a.pad0;  // input tile origin

  // 1. Staging.  Every global load of the stage is issued before the first
  // LDS store, so the block waits for one memory round trip.
  // (Addresses clamped into the image, so the loads need no branch and all
  // issue back to back; values outside the image are replaced afterwards.)
  float xv[XIT];
  bool xin[XIT];
  float pxv[XIP][C0];
  bool pin[XIP];
  if constexpr (NPART == 3) {
#pragma unroll
    for (int i = 0; i < XIT; ++i) {
      const int e = tid + i * NT;
      const int ch = e % C0, t = e / C0;
      const int col = t % kIW, row = t / kIW;
      const int y = y0 + row, x = x0 + col;
      xin[i] = e < NX && y >= 0 && y < a.H && x >= 0 && x < a.W;
      const int yc = min(max(y, 0), a.H - 1), xc = min(max(x, 0), a.W - 1);
      xv[i] = a.in[((static_cast<size_t>(n) * a.H + yc) * a.W + xc) * C0 + ch];
    }
  } else {
    // whole pixels per thread (their C0 values make one code)
#pragma unroll
    for (int i = 0; i < XIP; ++i) {
      const int q = tid + i * NT;
      const int col = q % kIW, row = q / kIW;
      const int y = y0 + row, x = x0 + col;
      pin[i] = q < NPIX && y >= 0 && y < a.H && x >= 0 && x < a.W;
      const int yc = min(max(y, 0), a.H - 1), xc = min(max(x, 0), a.W - 1);
      const size_t base = ((static_cast<size_t>(n) * a.H + yc) * a.W + xc) * C0;
#pragma unroll
      for (int ch = 0; ch < C0; ++ch) pxv[i][ch] = a.in[base + ch];
    }
  }
  // NPART = 1: the per-channel thresholds (one uniform load each).
  float off[C0];
#pragma unroll
  for (int ch = 0; ch < C0; ++ch) off[ch] = 0.0f;
  if (NPART == 1 && a.offset) {
#pragma unroll
    for (int ch = 0; ch < C0; ++ch) off[ch] = a.offset[ch];
  }
  // First-layer weights: the 9 words of the filter of each A-operand entry
  // this thread builds (indices clamped, so the loads need no branch).
  constexpr int NOP = FT0 * KC0 * 64;
  constexpr int WIT = NPART == 3 ? (NOP + NT - 1) / NT : 1;
  uint32_t w0v[WIT][9];
#pragma unroll
  for (int i = 0; i < WIT; ++i) {
    const int e = min(tid + i * NT, NOP - 1);
    const int f = NPART == 3 ? 16 * ((e >> 6) / KC0) + (e & 15) : min(tid, F0 - 1);
#pragma unroll
    for (int t = 0; t < 9; ++t) w0v[i][t] = a.w0[f * 9 + t];
  }
  const int32_t thr0v = a.thr0[min(tid, F0 - 1)];
  const int32_t thr1v = a.thr1[min(tid, F1 - 1)];
  const int32_t corr1v = PREP1 ? a.corr1[min(tid, F1 - 1)] : 0;
  const uint32_t fl0v = a.flip0 ? a.flip0[min(tid, CW1 - 1)] : 0u;

  // First-layer A operands: row = filter 16 ft + (l % 16), 8 k values
  // 32 kc + 8 (l / 16) + j as +-1 (0 past K0).  The filter's K0 = 9 C0 weight
  // bits are gathered first, k = C0 tap + ch at bit K0 - 1 - k.
  using KBits = typename std::conditional<(K0 <= 32), uint32_t, uint64_t>::type;
#pragma unroll
  for (int i = 0; i < WIT; ++i) {
    const int e = tid + i * NT;
    if (NPART == 3 && e < NOP) {
      const int l = e & 63, kc = (e >> 6) % KC0, ft = (e >> 6) / KC0;
      const int q = l >> 4;
      KBits bits = 0;
#pragma unroll
      for (int t = 0; t < 9; ++t) bits = (bits << C0) | static_cast<KBits>(w0v[i][t] >> (32 - C0));
      uint16_t op[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int k = 32 * kc + 8 * q + j;
        const bool ok = k < K0;
        const bool one = (bits >> (ok ? K0 - 1 - k : 0)) & 1u;
        op[j] = ok ? (one ? kBf16One : kBf16MinusOne) : kBf16Zero;
      }
      wop[ft][kc][l] = bf16x8(op);
    }
  }
  // NPART = 1: filter tid's K0 weight bits, element k = C0 tap + ch at bit
  // 31 - k (the unused low bits 0).
  if (NPART == 1 && tid < F0) {
    uint32_t pw = 0u;
#pragma unroll
    for (int t = 0; t < 9; ++t) pw |= (w0v[0][t] >> (32 - C0)) << (32 - (t + 1) * C0);
    wp0[tid] = pw;
  }
  // First-layer thresholds as the smallest fp32 value >= thr (-0.0 for a
  // zero threshold): the sign bit of S - th0 is then clear exactly when
  // S >= thr, for every fp32 sum S (thr_ceil_f32).
  // Binary first layer (NPART = 1): integer sums |S| <= K0, so the
  // accumulators can start at 0.5 - thr (thr clamped to [-K0-1, K0+1]) and
  // their sign bit is that of S - thr + 0.5, exact in fp32, with no
  // subtraction after the MFMAs.
  if (tid < F0)
    th0[tid] = NPART == 3 ? thr_ceil_f32(thr0v)
                          : 0.5f - static_cast<float>(min(max(thr0v, -K0 - 1), K0 + 1));
  if (tid < CW1) fl0[tid] = fl0v;
  // Second-layer start values 0.5 - thr (thr clamped to [-K1-1, K1+1], which
  // keeps every comparison since |S| <= K1); with prepared weights the sums
  // come out B_f too high, so the start value is 0.5 - thr - B_f.
  if (tid < F1)
    th1[tid] = 0.5f - static_cast<float>(min(max(thr1v, -a.K1 - 1), a.K1 + 1) + corr1v);
  // Each input value split once into its three bf16 parts, or each input
  // pixel thresholded into its code: bit C0 - 1 - ch = (x_ch + T_ch > 0);
  // outside the image the code is 0, the pad -1.
  if constexpr (NPART == 3) {
#pragma unroll
    for (int i = 0; i < XIT; ++i) {
      const int e = tid + i * NT;
      if (e < NX) {
        const Split3 sp = split3(xin[i] ? xv[i] : 0.0f);
        xs[0][e] = bf16_bits(sp.p0);
        xs[1][e] = bf16_bits(sp.p1);
        xs[2][e] = bf16_bits(sp.p2);
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < XIP; ++i) {
      const int q = tid + i * NT;
      uint32_t code = 0u;
#pragma unroll
      for (int ch = 0; ch < C0; ++ch)
        code |= static_cast<uint32_t>(pin[i] && pxv[i][ch] + off[ch] > 0.0f) << (C0 - 1 - ch);
      if (q < NPIX) xcode[q] = code;
    }
  }
  __syncthreads();

  const uint32_t smask = __builtin_amdgcn_readfirstlane(0x88888888u);
  uint32_t vfill;
  asm("v_mov_b32 %0, 0x22222222" : "=v"(vfill));

  // 2. First layer on the (TH + 2) x 34 tile: lane (q, c) = (l / 16, l % 16) holds
  // pixel c of a 16-pixel tile and filters 16 ft + 4 q + r (r = 0..3).
  if constexpr (NPART == 3) {
    const int q = lane >> 4, c = lane & 15;
    // Offsets of this lane's k values from the window's first input value;
    // k >= K0 reuses offset 0 (its weight is 0).
    int koff[KC0][8];
#pragma unroll
    for (int kc = 0; kc < KC0; ++kc)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int k = 32 * kc + 8 * q + j;
        const int tap = k / C0, ch = k - tap * C0;
        const int kh = tap / 3, kw = tap - kh * 3;
        koff[kc][j] = k < K0 ? (kh * kIW + kw) * C0 + ch : 0;
      }
    v8bf wa[FT0][KC0];
#pragma unroll
    for (int ft = 0; ft < FT0; ++ft)
#pragma unroll
      for (int kc = 0; kc < KC0; ++kc) wa[ft][kc] = wop[ft][kc][lane];
    v4f thv[2 * CW1];
#pragma unroll
    for (int ft = 0; ft < 2 * CW1; ++ft)
      thv[ft] = *reinterpret_cast<const v4f*>(&th0[16 * ft + 4 * q]);
    // After the row reduction lane (q, c) holds word q % CW1 of pixel c.
    const uint32_t nfl = ~fl0[q % CW1];

    for (int pt = wave; pt < kATiles; pt += NW) {
      const int p = 16 * pt + c;
      const bool pv = p < kAPix;
      const int pp = pv ? p : 0;
      const int lr = pp / kAW, lc = pp - (pp / kAW) * kAW;
      const int base = (lr * kIW + lc) * C0;
      v8bf xp[NPART][KC0];
#pragma unroll
      for (int pt = 0; pt < NPART; ++pt)
#pragma unroll
        for (int kc = 0; kc < KC0; ++kc) {
          uint16_t v[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) v[j] = xs[pt][base + koff[kc][j]];
          xp[pt][kc] = bf16x8(v);
        }
      const int rr = r0 + lr, cc = c0 + lc;
      const bool inside = pv && rr >= 0 && rr < a.Ho0 && cc >= 0 && cc < a.Wo0;
      // All filter tiles' products of one part before the next part's, so
      // no MFMA waits on the one before it.
      v4f acc[2 * CW1];
#pragma unroll
      for (int ft = 0; ft < 2 * CW1; ++ft)
        acc[ft] = NPART == 3 ? v4f{0.f, 0.f, 0.f, 0.f} : thv[ft];
#pragma unroll
      for (int kc = 0; kc < KC0; ++kc)
#pragma unroll
        for (int pt = 0; pt < NPART; ++pt)
#pragma unroll
          for (int ft = 0; ft < 2 * CW1; ++ft)
            acc[ft] =
                __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa[ft][kc], xp[pt][kc], acc[ft], 0, 0, 0);
      // Sign bits of S - thr, filter fl of word wi at bit 31 - fl.
      uint32_t sg[CW1];
#pragma unroll
      for (int wi = 0; wi < CW1; ++wi) {
        sg[wi] = 0u;
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          const int ft = 2 * wi + hf;
          uint32_t nib = 0u;
#pragma unroll
          for (int r = 0; r < 4; ++r)
            nib = __builtin_amdgcn_alignbit(
                nib, __float_as_uint(NPART == 3 ? acc[ft][r] - thv[ft][r] : acc[ft][r]), 31);
          sg[wi] |= nib << (28 - 16 * hf - 4 * q);
        }
      }
      uint32_t rows;
      if constexpr (CW1 == 4)
        rows = or_rows4(sg[0], sg[1], sg[2], sg[3]);
      else
        rows = or_rows4(sg[0], sg[1], sg[0], sg[1]);
      // Output bit = (S >= thr) xor flip = sign xor ~flip.
      const uint32_t word = inside ? rows ^ nfl : 0u;
      if (q < CW1 && pv) {
        const v8i x = PREP1 ? act_operand(word, smask, vfill) : expand_fp4(word, smask, vfill);
        actx[lr * RSX + lc * PSX + q] = v4i{x[0], x[1], x[2], x[3]};
      }
    }
  } else {
    // NPART = 1, 32 pixels per round on the fp4 matrix cores: lane (h, c)
    // holds pixel c and, as operands, K half h of the window (h = 0: the
    // K0 <= 32 bits, k = C0 tap + ch at bit 31 - k, as +-1 fp4; h = 1:
    // zeros) and of filter 32 tf + c.  Result register e of lane (h, c):
    // filter 32 tf + 8 (e / 4) + 4 h + e % 4 at pixel c.  Positions past K0
    // are 0.0 in the weights, so their products vanish.
    const int h = lane >> 5, c = lane & 31;
    constexpr int kATiles32 = (kAPix + 31) / 32;
    v8i wa1[CW1];
#pragma unroll
    for (int tf = 0; tf < CW1; ++tf) {
      const v8i x = expand_fp4(wp0[32 * tf + c], smask, vfill);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        // nibble n of register r is bit 4 n + r: clear the bits below 32 - K0
        uint32_t m = 0xFFFFFFFFu;
#pragma unroll
        for (int bb = r; bb < 32 - K0; bb += 4) m &= ~(0xFu << (4 * (bb / 4)));
        wa1[tf][r] = h ? 0 : static_cast<int>(static_cast<uint32_t>(x[r]) & m);
      }
#pragma unroll
      for (int r = 4; r < 8; ++r) wa1[tf][r] = 0;
    }
    // After the lane-half exchange, lane half h holds the word of tile h
    // (and of tile 2 + h when CW1 = 4).
    const uint32_t nfl0 = ~fl0[h];
    const uint32_t nfl1 = ~fl0[CW1 == 4 ? 2 + h : h];
    for (int pt = wave; pt < kATiles32; pt += NW) {
      const int p = 32 * pt + c;
      const bool pv = p < kAPix;
      const int pp = pv ? p : 0;
      const int lr = pp / kAW, lc = pp - (pp / kAW) * kAW;
      uint32_t patch = 0u;
#pragma unroll
      for (int kh = 0; kh < 3; ++kh)
#pragma unroll
        for (int kw = 0; kw < 3; ++kw)
          patch |= xcode[(lr + kh) * kIW + lc + kw] << (32 - (3 * kh + kw + 1) * C0);
      v8i B = expand_fp4(patch, smask, vfill);
#pragma unroll
      for (int r = 0; r < 4; ++r) B[r] = h ? 0 : B[r];
      uint32_t wd[CW1];
#pragma unroll
      for (int tf = 0; tf < CW1; ++tf) {
        v16f t;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const v4f q4 = *reinterpret_cast<const v4f*>(&th0[32 * tf + 8 * g + 4 * h]);
#pragma unroll
          for (int r = 0; r < 4; ++r) t[4 * g + r] = q4[r];
        }
        const v16f acc =
            __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(wa1[tf], B, t, 4, 4, 0, 127, 0, 127);
        // sign bits of S - thr + 0.5: filter 8 g + 4 h + r at bit 31 - 8 g - 4 h - r
        wd[tf] = 0u;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          uint32_t nib = 0u;
#pragma unroll
          for (int r = 0; r < 4; ++r)
            nib = __builtin_amdgcn_alignbit(nib, __float_as_uint(acc[4 * g + r]), 31);
          wd[tf] |= nib << (28 - 8 * g - 4 * h);
        }
      }
      const auto s01 = __builtin_amdgcn_permlane32_swap(wd[0], wd[1], false, false);
      uint32_t wlo = s01[0] | s01[1], whi = 0u;
      if constexpr (CW1 == 4) {
        const auto s23 = __builtin_amdgcn_permlane32_swap(wd[2], wd[3], false, false);
        whi = s23[0] | s23[1];
      }
      const int rr = r0 + lr, cc = c0 + lc;
      const bool inside = pv && rr >= 0 && rr < a.Ho0 && cc >= 0 && cc < a.Wo0;
      // Output bit = (S >= thr) xor flip = sign xor ~flip.
      if (pv) {
        const uint32_t w0w = inside ? wlo ^ nfl0 : 0u;
        const v8i x0 = PREP1 ? act_operand(w0w, smask, vfill) : expand_fp4(w0w, smask, vfill);
        actx[lr * RSX + lc * PSX + h] = v4i{x0[0], x0[1], x0[2], x0[3]};
        if constexpr (CW1 == 4) {
          const uint32_t w1w = inside ? whi ^ nfl1 : 0u;
          const v8i x1 =
              PREP1 ? act_operand(w1w, smask, vfill) : expand_fp4(w1w, smask, vfill);
          actx[lr * RSX + lc * PSX + 2 + h] = v4i{x1[0], x1[1], x1[2], x1[3]};
        }
      }
    }
  }
  __syncthreads();

  // 3. Second layer: wave = pixel group pg (64 pixels) x filter half fh.
  if (wave >= NW2) return;  // (no barrier follows)
  const int pg = wave % PG, fh = wave / PG;
  const int h = lane >> 5, c = lane & 31;
  const int f0 = 64 * fh;
  int pr[2], pc[2], abase[2];
#pragma unroll
  for (int tp = 0; tp < 2; ++tp) {
    const int m = 32 * tp + c;
    if constexpr (POOL) {
      pr[tp] = 2 * pg + ((m >> 1) & 1);
      pc[tp] = 2 * (m >> 2) + (m & 1);
    } else {
      pr[tp] = 2 * pg + tp;
      pc[tp] = c;
    }
    abase[tp] = pr[tp] * RSX + pc[tp] * PSX + h * VW;
  }
  v16f acc[2][2];
#pragma unroll
  for (int tf = 0; tf < 2; ++tf) {
    v16f t;
#pragma unroll
    for (int e = 0; e < 16; ++e) t[e] = th1[f0 + 32 * tf + 8 * (e >> 2) + 4 * h + (e & 3)];
    acc[tf][0] = t;
    acc[tf][1] = t;
  }
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint32_t*>(a.w1), 0, a.w1_bytes, kRsrcWord3);
  using WReg = typename std::conditional<PREP1, v4i, uint32_t>::type;
  uint32_t woff[2];
#pragma unroll
  for (int tf = 0; tf < 2; ++tf)
    woff[tf] = PREP1 ? static_cast<uint32_t>((((f0 / 32 + tf) * 9 * CW1 + h * VW) * 32 + c) * 16)
                     : static_cast<uint32_t>(((f0 + 32 * tf + c) * 9 * CW1 + h * VW) * 4);

  auto load_w = [&](int it, WReg (&ww)[2][VW]) {
    const int tap = it / NCH, cc = (it - tap * NCH) * 2 * VW;
    if constexpr (PREP1) {
      const uint32_t so = static_cast<uint32_t>((tap * CW1 + cc) * 512);
#pragma unroll
      for (int tf = 0; tf < 2; ++tf)
#pragma unroll
        for (int v = 0; v < VW; ++v)
          ww[tf][v] = __builtin_bit_cast(
              v4i, __builtin_amdgcn_raw_buffer_load_b128(rw, woff[tf] + 512 * v, so, 0));
      return;
    }
    const uint32_t so = static_cast<uint32_t>((tap * CW1 + cc) * 4);
#pragma unroll
    for (int tf = 0; tf < 2; ++tf) {
      if constexpr (VW == 2) {
        typedef unsigned int u2 __attribute__((ext_vector_type(2)));
        const u2 t = __builtin_amdgcn_raw_buffer_load_b64(rw, woff[tf], so, 0);
        ww[tf][0] = t[0];
        ww[tf][1] = t[1];
      } else {
        ww[tf][0] = __builtin_amdgcn_raw_buffer_load_b32(rw, woff[tf], so, 0);
      }
    }
  };
  constexpr int ITERS = 9 * NCH;
  WReg wr[2][2][VW];
  load_w(0, wr[0]);
#pragma unroll
  for (int it = 0; it < ITERS; ++it) {
    const int cur = it & 1;
    if (it + 1 < ITERS) load_w(it + 1, wr[cur ^ 1]);
    const int tap = it / NCH, cc = (it - tap * NCH) * 2 * VW;
    const int kh = tap / 3, kw = tap - kh * 3;
    const int ao = kh * RSX + kw * PSX + cc;
    v8i A[2][VW], B[2][VW];
#pragma unroll
    for (int tp = 0; tp < 2; ++tp)
#pragma unroll
      for (int v = 0; v < VW; ++v) {
        const v4i t = actx[abase[tp] + ao + v];
        B[tp][v] = v8i{t[0], t[1], t[2], t[3], 0, 0, 0, 0};
      }
#pragma unroll
    for (int tf = 0; tf < 2; ++tf) {
      if constexpr (PREP1) {
#pragma unroll
        for (int v = 0; v < VW; ++v)
          A[tf][v] = v8i{wr[cur][tf][v][0], wr[cur][tf][v][1], wr[cur][tf][v][2],
                         wr[cur][tf][v][3], 0, 0, 0, 0};
      } else {
        expand_words<VW>(wr[cur][tf], smask, vfill, A[tf]);
      }
    }
#pragma unroll
    for (int v = 0; v < VW; ++v)
#pragma unroll
      for (int tf = 0; tf < 2; ++tf)
#pragma unroll
        for (int tp = 0; tp < 2; ++tp)
          acc[tf][tp] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
              A[tf][v], B[tp][v], acc[tf][tp], 4, 4, 0, 127, 0, 127);
  }

  // Epilogue: register e of lane (h, c) holds S - thr + 0.5 of filter
  // f0 + 32 tf + 8 (e / 4) + 4 h + e % 4 at pixel c of tile tp; its sign bit
  // is the complement of the output bit.  Both lane halves hold bits of each
  // filter tile's word; one v_permlane32_swap of the two tiles' words leaves
  // lane half h with the whole word of filter tile h.
  const uint32_t fxh = ~(a.flip1 ? a.flip1[f0 / 32 + h] : 0u);
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
    uint32_t word = (sw[0] | sw[1]) ^ fxh;
    if constexpr (POOL) {
      word = or_quad(word);
      const int ip = (i0 >> 1) + pg, jp = (j0 >> 1) + ((32 * tp + c) >> 2);
      if ((c & 3) == 0 && ip < a.Hp && jp < a.Wp)
        a.bits[(static_cast<size_t>(n * a.Hp + ip) * a.Wp + jp) * FW1 + f0 / 32 + h] = word;
    } else {
      const int i = i0 + pr[tp], j = j0 + pc[tp];
      if (i < a.Ho1 && j < a.Wo1)
        a.bits[(static_cast<size_t>(n * a.Ho1 + i) * a.Wo1 + j) * FW1 + f0 / 32 + h] = word;
    }
  }
}

template <int TH, int C0, int F0, bool PREP1, int NPART>
hipError_t launch_th(const FbArgs& a, int f1, bool pool, unsigned blocks, hipStream_t s) {
  if (f1 == 128) {
    if (pool)
      fconv_bconv_kernel<TH, C0, F0, 2, true, PREP1, NPART><<<blocks, 512, 0, s>>>(a);
    else
      fconv_bconv_kernel<TH, C0, F0, 2, false, PREP1, NPART><<<blocks, 512, 0, s>>>(a);
  } else {
    if (pool)
      fconv_bconv_kernel<TH, C0, F0, 1, true, PREP1, NPART><<<blocks, 256, 0, s>>>(a);
    else
      fconv_bconv_kernel<TH, C0, F0, 1, false, PREP1, NPART><<<blocks, 256, 0, s>>>(a);
  }
  return hipGetLastError();
}

template <int C0, int F0, bool PREP1, int NPART>
hipError_t launch_c0f0(const FbArgs& a, int th, int f1, bool pool, unsigned blocks,
                       hipStream_t s) {
  return th == 8 ? launch_th<8, C0, F0, PREP1, NPART>(a, f1, pool, blocks, s)
                 : launch_th<4, C0, F0, PREP1, NPART>(a, f1, pool, blocks, s);
}

template <int C0, int NPART>
hipError_t launch_c0(const FbArgs& a, int th, int f0, int f1, bool pool, unsigned blocks,
                     hipStream_t s) {
  if (a.corr1)
    return f0 == 128 ? launch_c0f0<C0, 128, true, NPART>(a, th, f1, pool, blocks, s)
                     : launch_c0f0<C0, 64, true, NPART>(a, th, f1, pool, blocks, s);
  return f0 == 128 ? launch_c0f0<C0, 128, false, NPART>(a, th, f1, pool, blocks, s)
                   : launch_c0f0<C0, 64, false, NPART>(a, th, f1, pool, blocks, s);
}

// Kernel arguments and grid shared by both first-layer forms; returns the
// tile height and the block count.
void fill_args(FbArgs& a, const ConvGeom& g0, const ConvGeom& g1, const float* in,
               const float* offset, const uint32_t* w0, const int32_t* thr0,
               const uint32_t* flip0, const uint32_t* w1, const void* w1prep,
               const int32_t* thr1, const uint32_t* flip1, uint32_t* bits, int& th,
               unsigned& blocks) {
  a.in = in;
  a.offset = offset;
  a.w0 = w0;
  a.thr0 = thr0;
  a.flip0 = flip0;
  // 8-row tiles, or 4-row tiles (blocks of twice the waves for the staging
  // and the first layer) where those still fit one workgroup per compute
  // unit: CIFAR L0 + L1 at batch 1 / 32 take 6.2 / 7.0 us with 4-row tiles
  // against 8.0 / 8.8 us with 8-row ones, at batch 48 / 64 11.0 / 11.3
  // against 9.2 / 9.5 us.  Prepared second-layer weights only with 8-row
  // tiles: on the small grids the 4x larger operands come from beyond L2
  // and the packed words are faster (batch 1 / 16: 7.25 / 7.70 us packed
  // against 7.77 / 8.11 prepared, measured with 4-row tiles of the block's
  // own waves only; batch 32 / 64 with 8-row tiles: 8.98 / 9.74 packed,
  // 8.70 / 9.36 prepared).
  const int64_t tiles8 =
      int64_t{g0.N} * ((g1.Wo + kTW - 1) / kTW) * ((g1.Ho + 7) / 8);
  th = 2 * tiles8 <= kCUs ? 4 : 8;
  if (th == 4) w1prep = nullptr;
  a.w1 = w1prep ? static_cast<const uint32_t*>(w1prep) : w1;
  a.thr1 = thr1;
  a.flip1 = flip1;
  a.bits = bits;
  a.N = g0.N;
  a.H = g0.H;
  a.W = g0.W;
  a.pad0 = g0.pad;
  a.Ho0 = g0.Ho;
  a.Wo0 = g0.Wo;
  a.pad1 = g1.pad;
  a.Ho1 = g1.Ho;
  a.Wo1 = g1.Wo;
  a.Hp = g1.Hp;
  a.Wp = g1.Wp;
  a.K1 = 9 * g1.C;
  a.w1_bytes = static_cast<int32_t>(static_cast<int64_t>(g1.F) * 9 * g1.Cw * 4);
  a.corr1 = nullptr;
  if (w1prep) {  // F1 and F0 are multiples of 64: entries [F1 / 32][9][F0 / 32][32]
    a.w1_bytes = g1.F * 9 * g1.Cw * 16;
    a.corr1 = reinterpret_cast<const int32_t*>(static_cast<const char*>(w1prep) + a.w1_bytes);
  }
  a.tiles_w = (g1.Wo + kTW - 1) / kTW;
  a.tiles_h = (g1.Ho + th - 1) / th;
  blocks = static_cast<unsigned>(g0.N) * a.tiles_w * a.tiles_h;
}

}  // namespace

bool fconv_bconv_supported(const ConvGeom& g0, const ConvGeom& g1) {
  return g0.KH == 3 && g0.KW == 3 && g0.C >= 1 && g0.C <= 4 && g0.pool == 0 &&
         (g0.pad == 0 || g0.pad == 1) && (g0.F == 64 || g0.F == 128) &&
         g1.KH == 3 && g1.KW == 3 && g1.C == g0.F && (g1.pad == 0 || g1.pad == 1) &&
         (g1.F == 64 || g1.F == 128) && (g1.pool == 0 || g1.pool == 2) &&
         g1.N == g0.N && g1.H == g0.Ho && g1.W == g0.Wo && g1.Ho >= 1 && g1.Wo >= 1 &&
         static_cast<int64_t>(g0.N) * g0.H * g0.W * g0.C < (int64_t{1} << 31);
}

bool input_bconv_bconv_supported(int mode, const ConvGeom& g0, const ConvGeom& g1) {
  return mode == BNN_INPUT_THRESHOLD && g0.C == 3 && fconv_bconv_supported(g0, g1);
}

hipError_t launch_fconv_bconv(const ConvGeom& g0, const ConvGeom& g1, const float* in,
                              const uint32_t* w0, const int32_t* thr0, const uint32_t* flip0,
                              const uint32_t* w1, const void* w1prep, const int32_t* thr1,
                              const uint32_t* flip1, uint32_t* bits, hipStream_t s) {
  FbArgs a;
  int th;
  unsigned blocks;
  fill_args(a, g0, g1, in, nullptr, w0, thr0, flip0, w1, w1prep, thr1, flip1, bits, th, blocks);
  const bool pool = g1.pool == 2;
  switch (g0.C) {
    case 1: return launch_c0<1, 3>(a, th, g0.F, g1.F, pool, blocks, s);
    case 2: return launch_c0<2, 3>(a, th, g0.F, g1.F, pool, blocks, s);
    case 3: return launch_c0<3, 3>(a, th, g0.F, g1.F, pool, blocks, s);
    default: return launch_c0<4, 3>(a, th, g0.F, g1.F, pool, blocks, s);
  }
}

hipError_t launch_input_bconv_bconv(const ConvGeom& g0, const ConvGeom& g1, const float* in,
                                    const float* offset, const uint32_t* w0,
                                    const int32_t* thr0, const uint32_t* flip0,
                                    const uint32_t* w1, const void* w1prep,
                                    const int32_t* thr1, const uint32_t* flip1,
                                    uint32_t* bits, hipStream_t s) {
  FbArgs a;
  int th;
  unsigned blocks;
  fill_args(a, g0, g1, in, offset, w0, thr0, flip0, w1, w1prep, thr1, flip1, bits, th, blocks);
  return launch_c0<3, 1>(a, th, g0.F, g1.F, g1.pool == 2, blocks, s);
}

}  // namespace bnn
