// Input binarization (Sec. II-C) and the first binary conv over a
// real-valued image binarized on the fly.
//
// Three binarizations of an fp32 NHWC image, each giving C <= 32 bits per
// pixel (channel 0 in the highest bit of the pixel's code):
//   THRESHOLD  C channels, bit = (x + T_c) > 0                (RGB thresholding)
//   GRAY       1 channel,  bit = (gray + T_0) > 0             (grayscale thresholding)
//   LBP        3 channels from the grayscale image: neighbours at radius 1
//              numbered clockwise from the top-left, channels = neighbours
//              0, 3, 6 (offsets (-1,-1), (0,+1), (+1,-1)), bit = neighbour's
//              gray > centre's, neighbours outside the image never exceed.
// gray = (0.299 R + 0.587 G) + 0.114 B in fp32 with each product rounded (the
// BT.601 luma; the paper names no conversion).
//
// The conv packs each output pixel's whole binarized window into P = KH*KW*C
// bits (the patch packing of Algorithm 1 with B = P bits instead of one word
// per tap), in PW = ceil(P / 32) <= 4 words, so a dot product of Eq. 4 is PW
// XOR + popcounts (one for the 3x3 RGB layer, P = 27) instead of one per tap.
//
// A block covers an 8 x 32 tile of output pixels, one per thread.  Its
// threads first binarize the input tile plus halo into codes in LDS (taps
// outside the image stay 0, the -1 pad value), then each builds its pixel's
// patch words from LDS.  The filters are turned into patch words the same
// way, once per block, together with a per-filter bias b = -q - 1 where
// q = floor((K - thr) / 2): S >= thr <=> popcount(a ^ w) <= q <=>
// popcount(a ^ w) + b < 0, so v_bcnt with accumulate leaves the output bit in
// the sign, and v_alignbit shifts it into the output word.  2x2 OR-pooling
// uses quad shuffles as in the other binary kernels.
#include "bnn.h"
#include "kernels.hpp"
#include "lane_ops.hpp"

namespace bnn {
namespace {

constexpr int kTH = 8, kTW = 32;                   // output tile (256 threads)
constexpr int kFB = 256;                           // filters staged per round
constexpr int kMaxTile = (kTH + 31) * (kTW + 31);  // KH, KW <= 32

struct BinArgs {
  const float* x;
  const float* offset;
  int32_t mode, N, H, W, Cin, C;
};

__device__ __forceinline__ float gray_of(const float* px) {
  const float r = 0.299f * px[0];
  const float g = 0.587f * px[1];
  const float b = 0.114f * px[2];
  const float rg = r + g;
  return rg + b;
}

// Binarized code of input pixel (n, i, j), which must lie inside the image.
__device__ uint32_t pixel_code(const BinArgs& a, int n, int i, int j) {
  const float* px = a.x + ((static_cast<size_t>(n) * a.H + i) * a.W + j) * a.Cin;
  if (a.mode == BNN_INPUT_THRESHOLD) {
    uint32_t code = 0;
    for (int c = 0; c < a.Cin; ++c) {
      const float v = px[c] + (a.offset ? a.offset[c] : 0.0f);
      code |= static_cast<uint32_t>(v > 0.0f) << (a.Cin - 1 - c);
    }
    return code;
  }
  const float g = gray_of(px);
  if (a.mode == BNN_INPUT_GRAY) return (g + (a.offset ? a.offset[0] : 0.0f)) > 0.0f ? 1u : 0u;
  // LBP: channel ch compares neighbour (i + dr, j + dc) with the centre.
  uint32_t code = 0;
#pragma unroll
  for (int ch = 0; ch < 3; ++ch) {
    const int ni = i + (ch == 0 ? -1 : ch == 1 ? 0 : 1);
    const int nj = j + (ch == 1 ? 1 : -1);
    uint32_t bit = 0;
    if (ni >= 0 && ni < a.H && nj >= 0 && nj < a.W) {
      const float* pn = a.x + ((static_cast<size_t>(n) * a.H + ni) * a.W + nj) * a.Cin;
      bit = gray_of(pn) > g ? 1u : 0u;
    }
    code |= bit << (2 - ch);
  }
  return code;
}

// One thread per pixel: the code, MSB-aligned, as the pixel's packed word.
__global__ __launch_bounds__(256) void binarize_kernel(BinArgs a, uint32_t* out) {
  const int64_t p = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t total = static_cast<int64_t>(a.N) * a.H * a.W;
  if (p >= total) return;
  const int j = static_cast<int>(p % a.W);
  const int64_t t = p / a.W;
  const int i = static_cast<int>(t % a.H);
  const int n = static_cast<int>(t / a.H);
  out[p] = pixel_code(a, n, i, j) << (32 - a.C);
}

struct PatchArgs {
  BinArgs in;
  const uint32_t* w;
  const int32_t* thr;
  const uint32_t* flip;
  int32_t* sums;
  uint32_t* bits;
  int32_t F, Fw, KH, KW, pad, Ho, Wo;
  int32_t P;        // KH * KW * C, bits per window
  int32_t tiles_x;  // tiles per output row
  int32_t tiles_y;  // tiles per output column
};

// ORs a code of C bits into a 128-bit big-endian patch (element 0 = bit 127)
// at elements e0 .. e0 + C - 1.
__device__ __forceinline__ void put_bits(uint64_t& hi, uint64_t& lo, uint32_t code, int e0, int C) {
  const int shift = 128 - e0 - C;
  if (shift >= 64) {
    hi |= static_cast<uint64_t>(code) << (shift - 64);
  } else {
    lo |= static_cast<uint64_t>(code) << shift;
    if (shift + C > 64) hi |= static_cast<uint64_t>(code) >> (64 - shift);
  }
}

template <int PW>
__device__ __forceinline__ void split_words(uint32_t (&pw)[PW], uint64_t hi, uint64_t lo) {
  const uint32_t all[4] = {static_cast<uint32_t>(hi >> 32), static_cast<uint32_t>(hi),
                           static_cast<uint32_t>(lo >> 32), static_cast<uint32_t>(lo)};
#pragma unroll
  for (int q = 0; q < PW; ++q) pw[q] = all[q];
}

template <int PW, bool POOL, bool SUMS, bool BITS>
__global__ __launch_bounds__(256) void bconv_patch_kernel(PatchArgs a) {
  __shared__ uint32_t tile[kMaxTile];
  __shared__ uint32_t wpat[kFB * PW];
  __shared__ int32_t wbias[kFB];
  __shared__ uint32_t wflip[kFB / 32];

  const int t = threadIdx.x;
  const int C = a.in.C;
  int b = blockIdx.x;
  const int bx = b % a.tiles_x;
  b /= a.tiles_x;
  const int by = b % a.tiles_y;
  const int n = b / a.tiles_y;
  const int i0 = by * kTH, j0 = bx * kTW;

  // Filter round f0 .. f0 + nf - 1 as patch words and biases in LDS (thread
  // t takes filter f0 + t).
  auto stage_filters = [&](int f0, int nf) {
    uint32_t wp[PW];
#pragma unroll
    for (int q = 0; q < PW; ++q) wp[q] = 0;
    int32_t bias = 0;
    if (t < nf) {
      const int f = f0 + t;
      const uint32_t* wf = a.w + static_cast<size_t>(f) * a.KH * a.KW;  // one word per tap
      uint64_t hi = 0, lo = 0;
      for (int s = 0; s < a.KH * a.KW; ++s) {
        const uint32_t code = wf[s] >> (32 - C);
        if constexpr (PW == 1)
          wp[0] |= code << (32 - (s + 1) * C);
        else
          put_bits(hi, lo, code, s * C, C);
      }
      if constexpr (PW > 1) split_words(wp, hi, lo);
      if constexpr (BITS) {
        // q = floor((K - thr) / 2), clamped to [-1, K]
        const int64_t d = static_cast<int64_t>(a.P) - a.thr[f];
        int64_t q = d >= 0 ? d / 2 : -((1 - d) / 2);
        q = q < -1 ? -1 : (q > a.P ? a.P : q);
        bias = static_cast<int32_t>(-q - 1);
      }
    }
#pragma unroll
    for (int q = 0; q < PW; ++q) wpat[t * PW + q] = wp[q];
    wbias[t] = bias;
    // the round's flip words (read once here rather than after each word's
    // popcounts, where the load's round trip would stall the wave)
    if (t < kFB / 32) wflip[t] = a.flip && 32 * t < nf ? a.flip[(f0 >> 5) + t] : 0u;
  };

  // Binarize the input tile plus halo, and stage the first filter round.
  // With at most 64 filters, wave 0 stages them while waves 1-3 binarize the
  // tile, so the two chains of global loads overlap.
  const int TR = kTH + a.KH - 1, TC = kTW + a.KW - 1;
  const int nf0 = min(kFB, a.F);
  const bool split = nf0 <= 64;
  if (split && t < 64) {
    stage_filters(0, nf0);
  } else {
    const int e0 = split ? t - 64 : t, step = split ? 192 : 256;
    for (int e = e0; e < TR * TC; e += step) {
      const int r = e / TC, cc = e - r * TC;
      const int gi = i0 - a.pad + r, gj = j0 - a.pad + cc;
      tile[e] = (gi >= 0 && gi < a.in.H && gj >= 0 && gj < a.in.W)
                    ? pixel_code(a.in, n, gi, gj)
                    : 0u;
    }
    if (!split) stage_filters(0, nf0);
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

  // Patch words: tap s = kh * KW + kw holds window elements s*C .. s*C+C-1,
  // element e at bit 31 - e % 32 of word e / 32.
  uint32_t patch[PW];
  if constexpr (PW == 1) {
    uint32_t p = 0;
    for (int kh = 0; kh < a.KH; ++kh)
      for (int kw = 0; kw < a.KW; ++kw) {
        const int s = kh * a.KW + kw;
        p |= tile[(oy + kh) * TC + (ox + kw)] << (32 - (s + 1) * C);
      }
    patch[0] = p;
  } else {
    uint64_t hi = 0, lo = 0;
    for (int kh = 0; kh < a.KH; ++kh)
      for (int kw = 0; kw < a.KW; ++kw)
        put_bits(hi, lo, tile[(oy + kh) * TC + (ox + kw)], (kh * a.KW + kw) * C, C);
    split_words(patch, hi, lo);
  }

  const int Wp = POOL ? a.Wo / 2 : a.Wo;
  const int Hp = POOL ? a.Ho / 2 : a.Ho;
  for (int f0 = 0; f0 < a.F; f0 += kFB) {
    const int nf = min(kFB, a.F - f0);
    if (f0 > 0) {
      __syncthreads();  // the previous round's filters are no longer read
      stage_filters(f0, nf);
      __syncthreads();
    }
    for (int g = 0; g < nf; g += 32) {
      const int fw = (f0 + g) >> 5;
      if constexpr (SUMS) {
        if (valid) {
          int32_t* sp = a.sums + ((static_cast<size_t>(n) * a.Ho + i) * a.Wo + j) * a.F + f0 + g;
          const int m = min(32, nf - g);
          for (int k = 0; k < m; ++k) {
            int32_t cnt = 0;
#pragma unroll
            for (int q = 0; q < PW; ++q) cnt += __builtin_popcount(patch[q] ^ wpat[(g + k) * PW + q]);
            sp[k] = a.P - 2 * cnt;
          }
        }
      }
      if constexpr (BITS) {
        uint32_t word = 0;
#pragma unroll
        for (int k = 0; k < 32; ++k) {
          uint32_t d = static_cast<uint32_t>(wbias[g + k]);
#pragma unroll
          for (int q = 0; q < PW; ++q)
            d += static_cast<uint32_t>(__builtin_popcount(patch[q] ^ wpat[(g + k) * PW + q]));
          word = __builtin_amdgcn_alignbit(word, d, 31);
        }
        word ^= wflip[g >> 5];
        if (fw == a.Fw - 1) word &= tail_mask(a.F);
        if constexpr (POOL) {
          word = or_quad(word);
          if ((t & 3) == 0 && (i >> 1) < Hp && (j >> 1) < Wp)
            a.bits[((static_cast<size_t>(n) * Hp + (i >> 1)) * Wp + (j >> 1)) * a.Fw + fw] = word;
        } else {
          if (valid) a.bits[((static_cast<size_t>(n) * a.Ho + i) * a.Wo + j) * a.Fw + fw] = word;
        }
      }
    }
  }
}

// Row-stream variant for bits-only output and a compile-time window whose
// rows fit a word (KW * C <= 32 bits) and whose rows pack into at most 3
// patch words.  The input tile is turned into one bit stream per tile row
// (the codes of its TC pixels, MSB first), each 64-element stretch by one
// wave ballot: with RGB thresholding straight from the image, whose tile row
// is TC * C consecutive floats, otherwise from the pixel codes staged in LDS.
// A window row of KW taps is then KW * C consecutive stream bits, which one
// funnel shift extracts, and the KH rows go to fixed slots of the patch words
// (RPW rows per word, the unused bits 0 in patches and filters alike, so the
// popcounts do not change).  This replaces the per-tap assembly of the
// general kernel, whose shifts and loop control cost as much as the
// XOR-popcounts themselves.
// popcount(x) + acc as one v_bcnt_u32_b32 (the compiler otherwise sums two or
// three popcounts with a separate v_add3, one more instruction per filter).
__device__ __forceinline__ uint32_t bcnt_acc(uint32_t x, uint32_t acc) {
  uint32_t d;
  asm("v_bcnt_u32_b32 %0, %1, %2" : "=v"(d) : "v"(x), "v"(acc));
  return d;
}

template <int KH, int KW, int C, bool POOL>
__global__ __launch_bounds__(256) void bconv_patch_rows_kernel(PatchArgs a) {
  constexpr int SW = KW * C;                   // bits per window row
  constexpr int RPW = 32 / SW;                 // window rows per patch word
  constexpr int PW = (KH + RPW - 1) / RPW;     // patch words
  constexpr int TR = kTH + KH - 1, TC = kTW + KW - 1;
  constexpr int E = TC * C;                    // stream bits per tile row
  constexpr int NW = (E + 31) / 32;            // stream words per tile row
  constexpr int RL = NW + 2;                   // stored: pad word, NW words, pad word
  constexpr int CH = (E + 63) / 64;            // ballots per tile row
  constexpr int JOBS = TR * CH;
  constexpr int JPW = (JOBS + 2) / 3;          // ballots per wave (3 or 4 waves)
  static_assert(SW <= 32 && PW <= 3, "window rows must fit the patch layout");
  __shared__ uint32_t stream[TR * RL];
  __shared__ uint32_t codes[C == 0 ? 1 : TR * TC];
  __shared__ float gt[C == 3 ? (TR + 2) * (TC + 2) : 1];  // LBP: grays with a ring
  __shared__ uint4 wsh[kFB];                   // patch words and bias per filter
  __shared__ uint32_t wflip[kFB / 32];

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  int b = blockIdx.x;
  const int bx = b % a.tiles_x;
  b /= a.tiles_x;
  const int by = b % a.tiles_y;
  const int n = b / a.tiles_y;
  const int i0 = by * kTH, j0 = bx * kTW;

  auto stage_filters = [&](int f0, int nf) {
    uint32_t pw[3] = {0u, 0u, 0u};
    int32_t bias = 0;
    if (t < nf) {
      const int f = f0 + t;
      const uint32_t* wf = a.w + static_cast<size_t>(f) * (KH * KW);  // one word per tap
#pragma unroll
      for (int kh = 0; kh < KH; ++kh) {
        uint32_t seg = 0;
#pragma unroll
        for (int kw = 0; kw < KW; ++kw) seg = (seg << C) | (wf[kh * KW + kw] >> (32 - C));
        pw[kh / RPW] |= seg << (32 - (kh % RPW + 1) * SW);
      }
      const int64_t d = static_cast<int64_t>(a.P) - a.thr[f];
      int64_t q = d >= 0 ? d / 2 : -((1 - d) / 2);
      q = q < -1 ? -1 : (q > a.P ? a.P : q);
      bias = static_cast<int32_t>(-q - 1);
    }
    wsh[t] = make_uint4(pw[0], pw[1], pw[2], static_cast<uint32_t>(bias));
    if (t < kFB / 32) wflip[t] = a.flip && 32 * t < nf ? a.flip[(f0 >> 5) + t] : 0u;
  };

  // Stream words of tile row r, 64 elements from element 64 q on: stored
  // at 1 + 2q and 2 + 2q (bit i of the ballot is element 64 q + i, which
  // goes to bit 31 - i % 32); the pad words around a row stay 0.
  auto put_ballot = [&](int r, int q, uint64_t bal) {
    const uint32_t lo = __builtin_bitreverse32(static_cast<uint32_t>(bal));
    const uint32_t hi = __builtin_bitreverse32(static_cast<uint32_t>(bal >> 32));
    uint32_t* row = stream + r * RL;
    if (lane < 2) row[1 + 2 * q + lane] = lane ? hi : lo;
    if (q == 0 && lane == 2) row[0] = 0u;
    if constexpr (NW % 2 == 0)
      if (q == CH - 1 && lane == 3) row[RL - 1] = 0u;
  };

  const int nf0 = min(kFB, a.F);
  const bool split = nf0 <= 64;  // wave 0 stages the filters meanwhile
  const int gi0 = i0 - a.pad, gj0 = j0 - a.pad;
  if (a.in.mode == BNN_INPUT_THRESHOLD) {
    if (split && wave == 0) {
      stage_filters(0, nf0);
    } else {
      const int wv = split ? wave - 1 : wave, nw = split ? 3 : 4;
      // Per 64-element stretch q of a tile row, fixed for the lane: its
      // element's offset in an image row, whether that column lies inside
      // the image, and its channel's threshold offset.  A job then only
      // picks its row (uniform) and stretch.
      int eo[CH];
      bool cok[CH];
      float oq[CH];
#pragma unroll
      for (int q = 0; q < CH; ++q) {
        const int e = q * 64 + lane, px = e / C, ch = e - px * C, gj = gj0 + px;
        cok[q] = e < E && gj >= 0 && gj < a.in.W;
        eo[q] = gj * C + ch;
        float o = 0.0f;
        if (a.in.offset) {
#pragma unroll
          for (int c = 0; c < C; ++c) o = ch == c ? a.in.offset[c] : o;
        }
        oq[q] = o;
      }
      // All of this wave's loads first, then the ballots.
      float v[JPW];
      bool in[JPW];
#pragma unroll
      for (int k = 0; k < JPW; ++k) {
        const int jb = wv + k * nw;
        const int r = jb / CH, q = jb - r * CH, gi = gi0 + r;
        const bool rok = jb < JOBS && gi >= 0 && gi < a.in.H;
        int o = eo[0];
        bool ok = cok[0];
#pragma unroll
        for (int qq = 1; qq < CH; ++qq)
          if (q == qq) o = eo[qq], ok = cok[qq];
        const float* rowp = a.in.x + (static_cast<size_t>(n) * a.in.H + (rok ? gi : 0)) *
                                         static_cast<size_t>(a.in.W) * C;
        in[k] = rok && ok;
        v[k] = in[k] ? rowp[o] : 0.0f;
      }
#pragma unroll
      for (int k = 0; k < JPW; ++k) {
        const int jb = wv + k * nw;
        if (jb < JOBS) {
          const int r = jb / CH, q = jb - r * CH;
          float o = oq[0];
#pragma unroll
          for (int qq = 1; qq < CH; ++qq)
            if (q == qq) o = oq[qq];
          put_ballot(r, q, __builtin_amdgcn_ballot_w64(in[k] && v[k] + o > 0.0f));
        }
      }
      if (!split) stage_filters(0, nf0);
    }
    __syncthreads();
  } else if (C == 3 && a.in.mode == BNN_INPUT_LBP) {
    // LBP: the grays of the tile plus a one-pixel ring first (NaN outside
    // the image, so such a neighbour never exceeds and a pixel outside the
    // image gets code 0, the pad), then each code from four grays in LDS,
    // rather than 12 global loads per pixel.
    constexpr int GC = TC + 2;
    if (split && wave == 0) {
      stage_filters(0, nf0);
    } else {
      const int e0 = split ? t - 64 : t, step = split ? 192 : 256;
      for (int e = e0; e < (TR + 2) * GC; e += step) {
        const int r = e / GC, cc = e - r * GC;
        const int gi = gi0 - 1 + r, gj = gj0 - 1 + cc;
        gt[e] = (gi >= 0 && gi < a.in.H && gj >= 0 && gj < a.in.W)
                    ? gray_of(a.in.x + ((static_cast<size_t>(n) * a.in.H + gi) * a.in.W + gj) *
                                           a.in.Cin)
                    : __builtin_nanf("");
      }
      if (!split) stage_filters(0, nf0);
    }
    __syncthreads();
    for (int e = t; e < TR * TC; e += 256) {
      const int r = e / TC, cc = e - r * TC;
      const float* gc = gt + (r + 1) * GC + cc + 1;  // the pixel's gray
      const float g = gc[0];
      codes[e] = (gc[-GC - 1] > g ? 4u : 0u) | (gc[1] > g ? 2u : 0u) | (gc[GC - 1] > g ? 1u : 0u);
    }
    __syncthreads();
    for (int jb = wave; jb < JOBS; jb += 4) {
      const int r = jb / CH, q = jb - r * CH;
      const int e = q * 64 + lane;
      const int px = e / C, ch = e - px * C;
      const bool bit = e < E && ((codes[r * TC + min(px, TC - 1)] >> (C - 1 - ch)) & 1u);
      put_ballot(r, q, __builtin_amdgcn_ballot_w64(bit));
    }
    __syncthreads();
  } else {
    if (split && wave == 0) {
      stage_filters(0, nf0);
    } else {
      const int e0 = split ? t - 64 : t, step = split ? 192 : 256;
      for (int e = e0; e < TR * TC; e += step) {
        const int r = e / TC, cc = e - r * TC;
        const int gi = gi0 + r, gj = gj0 + cc;
        codes[e] = (gi >= 0 && gi < a.in.H && gj >= 0 && gj < a.in.W)
                       ? pixel_code(a.in, n, gi, gj)
                       : 0u;
      }
      if (!split) stage_filters(0, nf0);
    }
    __syncthreads();
    for (int jb = wave; jb < JOBS; jb += 4) {
      const int r = jb / CH, q = jb - r * CH;
      const int e = q * 64 + lane;
      const int px = e / C, ch = e - px * C;
      const bool bit = e < E && ((codes[r * TC + min(px, TC - 1)] >> (C - 1 - ch)) & 1u);
      put_ballot(r, q, __builtin_amdgcn_ballot_w64(bit));
    }
    __syncthreads();
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

  // Window row kh is stream bits ox*C .. ox*C + SW - 1 of tile row oy + kh:
  // the top SW bits of alignbit(word, next word, 32 - bit offset), or of the
  // word itself (alignbit by 0 of the pad or previous word and it) when the
  // offset is 0.
  const int p = ox * C, bo = p & 31;
  const int base = (p >> 5) + (bo ? 1 : 0);
  const uint32_t sh = static_cast<uint32_t>(32 - bo) & 31u;
  uint32_t patch[PW];
#pragma unroll
  for (int q = 0; q < PW; ++q) patch[q] = 0u;
#pragma unroll
  for (int kh = 0; kh < KH; ++kh) {
    const uint32_t* row = stream + (oy + kh) * RL + base;
    const uint32_t seg = __builtin_amdgcn_alignbit(row[0], row[1], sh);
    constexpr uint32_t top = SW == 32 ? ~0u : ~(~0u >> SW);
    const int k = kh % RPW;
    patch[kh / RPW] |= (seg >> (k * SW)) & (top >> (k * SW));
  }

  const int Wp = POOL ? a.Wo / 2 : a.Wo;
  const int Hp = POOL ? a.Ho / 2 : a.Ho;
  for (int f0 = 0; f0 < a.F; f0 += kFB) {
    const int nf = min(kFB, a.F - f0);
    if (f0 > 0) {
      __syncthreads();  // the previous round's filters are no longer read
      stage_filters(f0, nf);
      __syncthreads();
    }
    for (int g = 0; g < nf; g += 32) {
      const int fw = (f0 + g) >> 5;
      uint32_t word = 0;
#pragma unroll
      for (int k = 0; k < 32; ++k) {
        const uint4 wk = wsh[g + k];
        uint32_t d = PW == 1 ? wk.w + static_cast<uint32_t>(__builtin_popcount(patch[0] ^ wk.x))
                             : bcnt_acc(patch[0] ^ wk.x, wk.w);
        if constexpr (PW > 1) d = bcnt_acc(patch[1] ^ wk.y, d);
        if constexpr (PW > 2) d = bcnt_acc(patch[2] ^ wk.z, d);
        word = __builtin_amdgcn_alignbit(word, d, 31);
      }
      word ^= wflip[g >> 5];
      if (fw == a.Fw - 1) word &= tail_mask(a.F);
      if constexpr (POOL) {
        word = or_quad(word);
        if ((t & 3) == 0 && (i >> 1) < Hp && (j >> 1) < Wp)
          a.bits[((static_cast<size_t>(n) * Hp + (i >> 1)) * Wp + (j >> 1)) * a.Fw + fw] = word;
      } else {
        if (i < a.Ho && j < a.Wo)
          a.bits[((static_cast<size_t>(n) * a.Ho + i) * a.Wo + j) * a.Fw + fw] = word;
      }
    }
  }
}

template <int KH, int KW, int C>
void launch_rows(const PatchArgs& a, bool pool, dim3 grid, hipStream_t s) {
  if (pool)
    bconv_patch_rows_kernel<KH, KW, C, true><<<grid, 256, 0, s>>>(a);
  else
    bconv_patch_rows_kernel<KH, KW, C, false><<<grid, 256, 0, s>>>(a);
}

// The row-stream kernel's instantiated windows (bits only).
bool try_launch_rows(const PatchArgs& a, bool pool, dim3 grid, hipStream_t s) {
  if (a.sums || !a.bits) return false;
  const int C = a.in.C;
  if (a.KH == 5 && a.KW == 5 && C == 3) launch_rows<5, 5, 3>(a, pool, grid, s);
  else if (a.KH == 5 && a.KW == 5 && C == 1) launch_rows<5, 5, 1>(a, pool, grid, s);
  else if (a.KH == 3 && a.KW == 3 && C == 3) launch_rows<3, 3, 3>(a, pool, grid, s);
  else if (a.KH == 3 && a.KW == 3 && C == 1) launch_rows<3, 3, 1>(a, pool, grid, s);
  else return false;
  return true;
}

template <int PW, bool POOL>
void launch_out(const PatchArgs& a, dim3 grid, hipStream_t s) {
  if (a.sums && a.bits)
    bconv_patch_kernel<PW, POOL, true, true><<<grid, 256, 0, s>>>(a);
  else if (a.sums)
    bconv_patch_kernel<PW, POOL, true, false><<<grid, 256, 0, s>>>(a);
  else
    bconv_patch_kernel<PW, POOL, false, true><<<grid, 256, 0, s>>>(a);
}

template <int PW>
void launch_pw(const PatchArgs& a, bool pool, dim3 grid, hipStream_t s) {
  if (pool)
    launch_out<PW, true>(a, grid, s);
  else
    launch_out<PW, false>(a, grid, s);
}

}  // namespace

int input_channels_of(int mode, int cin) {
  return mode == BNN_INPUT_GRAY ? 1 : mode == BNN_INPUT_LBP ? 3 : cin;
}

bool bconv_patch_supported(const ConvGeom& g) {
  return g.C <= 32 && g.KH <= 32 && g.KW <= 32 && int64_t{g.KH} * g.KW * g.C <= 128;
}

hipError_t launch_binarize(int mode, const float* x, const float* offset, int32_t N, int32_t H,
                           int32_t W, int32_t Cin, uint32_t* out, hipStream_t s) {
  BinArgs a{x, offset, mode, N, H, W, Cin, input_channels_of(mode, Cin)};
  const int64_t total = int64_t{N} * H * W;
  binarize_kernel<<<dim3(static_cast<unsigned>((total + 255) / 256)), 256, 0, s>>>(a, out);
  return hipGetLastError();
}

hipError_t launch_bconv_patch(const ConvGeom& g, int mode, const float* x, const float* offset,
                              const uint32_t* w, const int32_t* thr, const uint32_t* flip,
                              int32_t* sums, uint32_t* bits, hipStream_t s) {
  PatchArgs a;
  a.in = BinArgs{x, offset, mode, g.N, g.H, g.W, mode == BNN_INPUT_THRESHOLD ? g.C : 3, g.C};
  a.w = w;
  a.thr = thr;
  a.flip = flip;
  a.sums = sums;
  a.bits = bits;
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
  const bool pool = g.pool == 2;
  if (try_launch_rows(a, pool, grid, s)) return hipGetLastError();
  switch ((a.P + 31) / 32) {
    case 1: launch_pw<1>(a, pool, grid, s); break;
    case 2: launch_pw<2>(a, pool, grid, s); break;
    case 3: launch_pw<3>(a, pool, grid, s); break;
    default: launch_pw<4>(a, pool, grid, s); break;
  }
  return hipGetLastError();
}

}  // namespace bnn
