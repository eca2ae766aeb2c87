// Binary convolution on the gfx950 matrix cores.
//
// A +-1 value is exactly representable in the 4-bit E2M1 float format, and a
// dot product of K such values is an integer |S| <= K < 2^24, exact in the
// fp32 accumulator.  So the XOR-popcount dot product of Eq. 4 can equally be
// computed by v_mfma_scale_f32_16x16x128_f8f6f4 with both operands in fp4:
// 16x16x128 multiply-accumulates per instruction, against 32 bit-MACs per
// v_xor + v_bcnt pair on the vector ALU.  Each packed word is expanded to four
// fp4 registers (one nibble per bit) right before use; the expansion is the
// same for weights and activations, so the order of the 32 values inside the
// MFMA's k dimension does not matter, and a sign-swapped encoding (bit 1 ->
// -1.0, bit 0 -> +1.0) on both sides leaves every product unchanged.  A pad
// tap is the word 0, i.e. -1 in the method's encoding, as in the VALU kernel.
//
// Operand roles: A (16 rows) = weights of 16 filters, B (16 columns) =
// activations of 16 output pixels; lane l supplies row / column l % 16 and
// the l / 16-th quarter of the 128 k values.  The result tile holds, in lane
// l, register r, the sum for filter 4*(l/16) + r and pixel l % 16.  A wave
// computes 64 (or 32) filters x 64 pixels (4 (or 2) x 4 tiles); with pooling,
// the 16 pixels of a tile are four 2x2 windows so that a window sits in 4
// adjacent lanes.
//
// Requirements (bconv_mfma_supported): stride 1, C a multiple of 128, F a
// multiple of 32, at most 32 taps.
#include <stdlib.h>

#include "kernels.hpp"

namespace bnn {
namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

struct MfmaArgs {
  const uint32_t* in;
  const uint32_t* w;
  const int32_t* thr;
  const uint32_t* flip;
  int32_t* sums;
  uint32_t* bits;
  int32_t N, H, W, Cw, F, Fw, KH, KW, pad, Ho, Wo, Hp, Wp;
  int32_t fstride;  // words per filter, KH*KW*Cw
  int32_t items;    // output pixels covered (N*Ho*Wo, or 4*N*Hp*Wp when pooling)
  int32_t K;        // valid bits per window, KH*KW*C
  int32_t in_bytes; // size of the input buffer (raw-buffer range)
  int32_t w_bytes;  // size of the weight buffer
};

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

// Raw buffer loads: an offset at or beyond the buffer's size returns zeros,
// which is how taps outside the image read the pad word 0 without a branch
// (every load is unconditional, so the loop can keep loads in flight).
constexpr uint32_t kOutOfRange = 0x80000000u;
constexpr int kRsrcWord3 = 0x00020000;

template <int VW>
__device__ __forceinline__ void buf_load(uint32_t (&v)[VW], __amdgpu_buffer_rsrc_t r, uint32_t voff,
                                         uint32_t soff) {
  if constexpr (VW == 2) {
    typedef unsigned int u2 __attribute__((ext_vector_type(2)));
    const u2 t = __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0);
    v[0] = t[0];
    v[1] = t[1];
  } else {
    v[0] = __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0);
  }
}

// Template parameters:
//   VW   words each lane loads per operand row and iteration (1, 2 or 4).  One
//        MFMA k-step covers 4 words (one per lane quarter), so an iteration
//        (a chunk of 4*VW words of one tap) feeds VW k-steps.
//   POOL pixels ordered as 2x2 windows (4 adjacent lanes per window).
//   TF   16-filter tiles per wave (2: one output word, 4: two).
//   KS   1: the 4 waves of a block take 4 consecutive 64-pixel tiles;
//        >1: the KS waves of a block share one tile and split the iterations,
//        adding their partial sums in LDS (for grids too small to fill the
//        chip).
//   PD   iterations whose loads are in flight at once (software pipeline).
template <int VW, bool POOL, int TF, int KS, int PD>
__global__ __launch_bounds__(512) void bconv_mfma_kernel(MfmaArgs a) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int q = lane >> 4;   // k quarter (operands) / row group (result)
  const int c = lane & 15;   // operand row / column within a 16-tile
  const int p0 = (KS == 1 ? blockIdx.x * 4 + wave : blockIdx.x) * 64;
  const int f0 = blockIdx.y * (16 * TF);
  const int nchunk = a.Cw / (4 * VW);
  const int iters = a.KH * a.KW * nchunk;
  int it0 = 0, it1 = iters;
  if constexpr (KS > 1) {
    const int per = (iters + KS - 1) / KS;
    it0 = min(iters, wave * per);
    it1 = min(iters, it0 + per);
  }

  // Pixels this lane loads for (one per pixel tile): word offset of the
  // pixel in the input, and which of the KH*KW taps fall inside the image.
  int pbase[4], pn[4], pi[4], pj[4];
  uint32_t tapmask[4];
  bool pv[4];
#pragma unroll
  for (int tp = 0; tp < 4; ++tp) {
    const int item = p0 + tp * 16 + c;
    pv[tp] = item < a.items;
    const int m = pv[tp] ? item : 0;
    if constexpr (POOL) {
      const int win = m >> 2;
      const int jp = win % a.Wp;
      const int t = win / a.Wp;
      const int ip = t % a.Hp;
      pn[tp] = t / a.Hp;
      pi[tp] = 2 * ip + ((m >> 1) & 1);
      pj[tp] = 2 * jp + (m & 1);
    } else {
      pj[tp] = m % a.Wo;
      const int t = m / a.Wo;
      pi[tp] = t % a.Ho;
      pn[tp] = t / a.Ho;
    }
    pbase[tp] = (((pn[tp] * a.H + pi[tp]) * a.W + pj[tp]) * a.Cw + q * VW) * 4;
    uint32_t mk = 0;
    for (int kh = 0; kh < a.KH; ++kh)
      for (int kw = 0; kw < a.KW; ++kw) {
        const int hi = pi[tp] + kh - a.pad, wi = pj[tp] + kw - a.pad;
        const bool ok = pv[tp] && static_cast<unsigned>(hi) < static_cast<unsigned>(a.H) &&
                        static_cast<unsigned>(wi) < static_cast<unsigned>(a.W);
        mk |= static_cast<uint32_t>(ok) << (kh * a.KW + kw);
      }
    tapmask[tp] = mk;
  }

  v4f acc[TF][4];
#pragma unroll
  for (int tf = 0; tf < TF; ++tf)
#pragma unroll
    for (int tp = 0; tp < 4; ++tp) acc[tf][tp] = v4f{0.f, 0.f, 0.f, 0.f};

  // Buffer resources; per-lane byte offsets of the weight rows and pixels.
  const __amdgpu_buffer_rsrc_t rin = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint32_t*>(a.in), 0, a.in_bytes, kRsrcWord3);
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint32_t*>(a.w), 0, a.w_bytes, kRsrcWord3);
  uint32_t woff[TF];
#pragma unroll
  for (int tf = 0; tf < TF; ++tf)
    woff[tf] = static_cast<uint32_t>(((f0 + tf * 16 + c) * a.fstride + q * VW) * 4);
  const uint32_t smask = __builtin_amdgcn_readfirstlane(0x88888888u);
  uint32_t vfill;
  asm("v_mov_b32 %0, 0x22222222" : "=v"(vfill));

  // Loads of iteration `it` (clamped into range so that every load is
  // unconditional; the clamped repeats at the end are never used).
  auto load_it = [&](int it, uint32_t (&ww)[TF][VW], uint32_t (&aw)[4][VW]) {
    const int tap = it / nchunk;
    const int cc = (it - tap * nchunk) * 4 * VW;
    const int kh = tap / a.KW;
    const int kw = tap - kh * a.KW;
    const uint32_t wsoff = static_cast<uint32_t>((tap * a.Cw + cc) * 4);
#pragma unroll
    for (int tf = 0; tf < TF; ++tf) buf_load<VW>(ww[tf], rw, woff[tf], wsoff);
    const int dshift = (((kh - a.pad) * a.W + (kw - a.pad)) * a.Cw + cc) * 4;
    const uint32_t bit = 1u << tap;
#pragma unroll
    for (int tp = 0; tp < 4; ++tp) {
      const uint32_t off = (tapmask[tp] & bit) ? static_cast<uint32_t>(pbase[tp] + dshift)
                                               : kOutOfRange;
      buf_load<VW>(aw[tp], rin, off, 0u);
    }
  };
  auto compute = [&](const uint32_t (&ww)[TF][VW], const uint32_t (&aw)[4][VW]) {
#pragma unroll
    for (int v = 0; v < VW; ++v) {
      v8i A[TF], B[4];
#pragma unroll
      for (int tf = 0; tf < TF; ++tf) A[tf] = expand_fp4(ww[tf][v], smask, vfill);
#pragma unroll
      for (int tp = 0; tp < 4; ++tp) B[tp] = expand_fp4(aw[tp][v], smask, vfill);
#pragma unroll
      for (int tf = 0; tf < TF; ++tf)
#pragma unroll
        for (int tp = 0; tp < 4; ++tp)
          acc[tf][tp] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(
              A[tf], B[tp], acc[tf][tp], 4, 4, 0, 127, 0, 127);
    }
  };

  // A ring of PD register sets: the loads of PD iterations are in flight at
  // once, so a wave waits for memory about once per PD iterations (each
  // dependent round trip to L2 / HBM costs far more than one iteration of
  // MFMAs).  Loads past the end are clamped to the last iteration and unused.
  if (it0 < it1) {
    uint32_t wr[PD][TF][VW], xr[PD][4][VW];
#pragma unroll
    for (int s = 0; s < PD; ++s) load_it(min(it0 + s, it1 - 1), wr[s], xr[s]);
    __builtin_amdgcn_sched_barrier(0);
    for (int it = it0; it < it1; it += PD) {
#pragma unroll
      for (int s = 0; s < PD; ++s) {
        if (it + s < it1) compute(wr[s], xr[s]);
        __builtin_amdgcn_sched_barrier(0);
        load_it(min(it + s + PD, it1 - 1), wr[s], xr[s]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }

  if constexpr (KS > 1) {
    __shared__ v4f part[KS - 1][TF][4][64];
    if (wave > 0) {
#pragma unroll
      for (int tf = 0; tf < TF; ++tf)
#pragma unroll
        for (int tp = 0; tp < 4; ++tp) part[wave - 1][tf][tp][lane] = acc[tf][tp];
    }
    __syncthreads();
    if (wave > 0) return;
#pragma unroll
    for (int w = 0; w < KS - 1; ++w)
#pragma unroll
      for (int tf = 0; tf < TF; ++tf)
#pragma unroll
        for (int tp = 0; tp < 4; ++tp) acc[tf][tp] += part[w][tf][tp][lane];
  }

  // Epilogue.  Lane (q, c) holds, for pixel tile tp, the sums of pixel c and
  // filters f0 + 16 tf + 4 q + r (r = 0..3).
  if (a.sums) {
#pragma unroll
    for (int tp = 0; tp < 4; ++tp) {
      if (!pv[tp]) continue;
      int32_t* sp = a.sums + (static_cast<size_t>(pn[tp] * a.Ho + pi[tp]) * a.Wo + pj[tp]) * a.F +
                    f0 + 4 * q;
#pragma unroll
      for (int tf = 0; tf < TF; ++tf) {
        int4 t;
        t.x = static_cast<int>(acc[tf][tp][0]);
        t.y = static_cast<int>(acc[tf][tp][1]);
        t.z = static_cast<int>(acc[tf][tp][2]);
        t.w = static_cast<int>(acc[tf][tp][3]);
        *reinterpret_cast<int4*>(sp + tf * 16) = t;
      }
    }
  }
  if (a.bits) {
    // Threshold minus one half: S >= thr  <=>  (thr - 0.5) - S < 0 for
    // integer S, so the sign bit of that difference is the output bit.
    // Thresholds are clamped to [-K-1, K+1] first (|S| <= K, so this keeps
    // every comparison) to stay exact in fp32 for any int32 threshold.
    constexpr int NW = TF / 2;  // output words per pixel in this wave
    float th[TF][4];
#pragma unroll
    for (int tf = 0; tf < TF; ++tf)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = a.thr[f0 + tf * 16 + 4 * q + r];
        th[tf][r] = static_cast<float>(min(max(t, -a.K - 1), a.K + 1)) - 0.5f;
      }
    uint32_t fl[NW];
#pragma unroll
    for (int h = 0; h < NW; ++h) fl[h] = a.flip ? a.flip[f0 / 32 + h] : 0u;
#pragma unroll
    for (int tp = 0; tp < 4; ++tp) {
      uint32_t word[NW];
#pragma unroll
      for (int h = 0; h < NW; ++h) word[h] = 0u;
#pragma unroll
      for (int tf = 0; tf < TF; ++tf) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float d = th[tf][r] - acc[tf][tp][r];
          const uint32_t sgn = __float_as_uint(d) >> 31;
          // filter 16 (tf % 2) + 4 q + r of output word tf / 2 -> bit 31 - that
          word[tf >> 1] |= sgn << (31 - (16 * (tf & 1) + 4 * q + r));
        }
      }
#pragma unroll
      for (int h = 0; h < NW; ++h) {
        word[h] |= __shfl_xor(word[h], 16);
        word[h] |= __shfl_xor(word[h], 32);
        word[h] ^= fl[h];
        if constexpr (POOL) {
          word[h] |= __shfl_xor(word[h], 1);
          word[h] |= __shfl_xor(word[h], 2);
        }
      }
      const int item = p0 + tp * 16 + c;
      const bool writer = POOL ? (q == 0 && (c & 3) == 0 && pv[tp]) : (q == 0 && pv[tp]);
      if (writer) {
        uint32_t* op = a.bits + static_cast<size_t>(POOL ? (item >> 2) : item) * a.Fw + f0 / 32;
        if constexpr (NW == 2)
          *reinterpret_cast<uint2*>(op) = make_uint2(word[0], word[1]);
        else
          *op = word[0];
      }
    }
  }
}

template <int VW, bool POOL, int PD>
hipError_t launch_cfg(const MfmaArgs& a, int tf, int ks, hipStream_t s) {
  const unsigned fy = static_cast<unsigned>(a.F / (16 * tf));
  const unsigned tiles = static_cast<unsigned>((a.items + 63) / 64);
  if (ks == 1) {
    dim3 grid((tiles + 3) / 4, fy), block(256);
    if (tf == 4)
      bconv_mfma_kernel<VW, POOL, 4, 1, PD><<<grid, block, 0, s>>>(a);
    else
      bconv_mfma_kernel<VW, POOL, 2, 1, PD><<<grid, block, 0, s>>>(a);
  } else {
    dim3 grid(tiles, fy), block(64 * ks);
    if (ks == 2)
      bconv_mfma_kernel<VW, POOL, 2, 2, PD><<<grid, block, 0, s>>>(a);
    else if (ks == 4)
      bconv_mfma_kernel<VW, POOL, 2, 4, PD><<<grid, block, 0, s>>>(a);
    else
      bconv_mfma_kernel<VW, POOL, 2, 8, PD><<<grid, block, 0, s>>>(a);
  }
  return hipGetLastError();
}

int env_int(const char* name, int dflt) {
  const char* e = getenv(name);
  return e ? atoi(e) : dflt;
}

hipError_t run_mfma(const ConvGeom& g, bool pool, const uint32_t* in, const uint32_t* w,
                    const int32_t* thr, const uint32_t* flip, int32_t* sums, uint32_t* bits,
                    hipStream_t s) {
  MfmaArgs a;
  a.in = in;
  a.w = w;
  a.thr = thr;
  a.flip = flip;
  a.sums = sums;
  a.bits = bits;
  a.N = g.N;
  a.H = g.H;
  a.W = g.W;
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
  a.items = pool ? 4 * g.N * g.Hp * g.Wp : g.N * g.Ho * g.Wo;
  a.K = g.KH * g.KW * g.C;
  a.in_bytes = static_cast<int32_t>(static_cast<int64_t>(g.N) * g.H * g.W * g.Cw * 4);
  a.w_bytes = static_cast<int32_t>(static_cast<int64_t>(g.F) * a.fstride * 4);
  // VW = 4 (128-bit loads) doubles the prefetched words and spills with the
  // 64x64 wave tile, so loads stay at 64 bits.
  const int vw = (g.Cw % 8 == 0) ? 2 : 1;
  const int iters = g.KH * g.KW * (g.Cw / (4 * vw));

  // Tile shape and K split (measured on MI355X): 64-filter wave tiles down to
  // ~1 wave per SIMD (1024 waves), then 32-filter tiles, then a K split.
  const int64_t tiles = (a.items + 63) / 64;
  int tf = 4, ks = 1;
  if (g.F % 64 != 0 || tiles * (g.F / 64) < 1024) {
    tf = 2;
    const int64_t base = tiles * (g.F / 32);
    while (ks < 8 && base * ks < 1024 && iters >= 4 * ks) ks *= 2;
  }
  // Tuning overrides (pipeline depth, filter tiles per wave, K split).
  int pd = env_int("BNN_MFMA_PD", 2);
  tf = env_int("BNN_MFMA_TF", tf);
  ks = env_int("BNN_MFMA_KS", ks);
  if (g.F % (16 * tf) != 0 || (ks > 1 && tf != 2)) tf = 2;
#define BNN_CFG(V, PDV)                                                         \
  if (vw == V && pd == PDV)                                                     \
    return pool ? launch_cfg<V, true, PDV>(a, tf, ks, s)                        \
                : launch_cfg<V, false, PDV>(a, tf, ks, s);
  BNN_CFG(2, 2)
  BNN_CFG(2, 4)
  BNN_CFG(1, 2)
  BNN_CFG(1, 4)
  BNN_CFG(1, 8)
#undef BNN_CFG
  if (vw == 2) return pool ? launch_cfg<2, true, 2>(a, tf, ks, s) : launch_cfg<2, false, 2>(a, tf, ks, s);
  return pool ? launch_cfg<1, true, 2>(a, tf, ks, s) : launch_cfg<1, false, 2>(a, tf, ks, s);
  return hipErrorInvalidValue;
}

}  // namespace

bool bconv_mfma_supported(const ConvGeom& g) {
  // C a multiple of 128 (whole words, 4 words per k-step), F a multiple of
  // 32 (whole output words), at most 32 taps (per-lane tap masks), and inputs
  // and weights under 2 GiB (32-bit byte offsets of the raw buffer loads).
  return (g.C % 32) == 0 && (g.Cw % 4) == 0 && (g.F % 32) == 0 && g.KH * g.KW <= 32 &&
         static_cast<int64_t>(g.N) * g.H * g.W * g.Cw < (int64_t{1} << 29) &&
         static_cast<int64_t>(g.F) * g.KH * g.KW * g.Cw < (int64_t{1} << 29);
}

hipError_t launch_bconv_mfma(const ConvGeom& g, const uint32_t* in, const uint32_t* w,
                             const int32_t* thr, const uint32_t* flip, int32_t* sums,
                             uint32_t* bits, hipStream_t s) {
  if (g.pool == 2 && sums && ((g.Ho & 1) || (g.Wo & 1))) {
    hipError_t e = run_mfma(g, false, in, w, thr, flip, sums, nullptr, s);
    if (e != hipSuccess || !bits) return e;
    return run_mfma(g, true, in, w, thr, flip, nullptr, bits, s);
  }
  return run_mfma(g, g.pool == 2, in, w, thr, flip, sums, bits, s);
}

}  // namespace bnn
