// Binary convolution on the gfx950 matrix cores.
//
// A +-1 value is exactly representable in the 4-bit E2M1 float format, and a
// dot product of K such values is an integer |S| <= K, exact in the fp32
// accumulator for the K < 2^22 taken here.  So the XOR-popcount dot product
// of Eq. 4 can equally be computed by v_mfma_scale_f32_32x32x64_f8f6f4 with
// both operands in fp4:
// 32x32x64 multiply-accumulates per instruction (the fastest fp4 shape on
// MI355X), against 32 bit-MACs per v_xor + v_bcnt pair on the vector ALU.
// Each packed word is expanded to four fp4 registers (one nibble per bit)
// right before use; the expansion is the same for weights and activations,
// so the order of the 32 values inside the MFMA's k dimension does not
// matter, and a sign-swapped encoding (bit 1 -> -1.0, bit 0 -> +1.0) on both
// sides leaves every product unchanged.  A pad tap is the word 0, i.e. -1 in
// the method's encoding, as in the VALU kernel.
//
// Operand roles: A (32 rows) = weights of 32 filters, B (32 columns) =
// activations of 32 output pixels; lane l supplies row / column l % 32 and
// the (l / 32)-th half of the 64 k values.  Register e of the result holds,
// in lane l, the sum for filter 8*(e/4) + 4*(l/32) + e%4 and pixel l % 32.  A
// wave computes 64 (or 32) filters x 64 pixels; with pooling, the 32 pixels
// of a tile are eight 2x2 windows so that a window sits in 4 adjacent lanes.
//
// Requirements (bconv_mfma_supported): stride 1, C >= 32 (a C that is not a
// multiple of 64 is padded to whole 64-bit chunks), at most 32 taps.
#include <type_traits>

#include "fp4_expand.hpp"
#include "kernels.hpp"
#include "lane_ops.hpp"

namespace bnn {
namespace {

// Raw buffer loads: an offset at or beyond the buffer's size returns zeros,
// which is how taps outside the image read the pad word 0 without a branch
// (every load is unconditional, so the loop can keep loads in flight).
constexpr uint32_t kOutOfRange = 0x80000000u;
constexpr int kRsrcWord3 = 0x00020000;

// SPLIT: VW separate 4-byte loads, for rows whose word count leaves the
// chunks without 8- or 16-byte alignment.
template <int VW, bool SPLIT = false>
__device__ __forceinline__ void buf_load(uint32_t (&v)[VW], __amdgpu_buffer_rsrc_t r, uint32_t voff,
                                         uint32_t soff) {
  if constexpr (SPLIT) {
#pragma unroll
    for (int i = 0; i < VW; ++i) v[i] = __builtin_amdgcn_raw_buffer_load_b32(r, voff + 4 * i, soff, 0);
  } else if constexpr (VW == 4) {
    typedef unsigned int u4 __attribute__((ext_vector_type(4)));
    const u4 t = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
    v[0] = t[0];
    v[1] = t[1];
    v[2] = t[2];
    v[3] = t[3];
  } else if constexpr (VW == 2) {
    typedef unsigned int u2 __attribute__((ext_vector_type(2)));
    const u2 t = __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0);
    v[0] = t[0];
    v[1] = t[1];
  } else {
    v[0] = __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0);
  }
}

// Unsigned division by a run-time invariant divisor d >= 1 with a multiply
// and shifts (Granlund and Montgomery, "Division by invariant integers using
// multiplication", 1994): exact for every 32-bit n.
struct FastDiv {
  uint32_t d, m;
  int s1, s2;
};

inline FastDiv make_fastdiv(uint32_t d) {
  int l = 0;
  while ((uint64_t{1} << l) < d) ++l;  // l = ceil(log2 d)
  FastDiv f;
  f.d = d;
  f.m = static_cast<uint32_t>(((uint64_t{1} << 32) * ((uint64_t{1} << l) - d)) / d + 1);
  f.s1 = l < 1 ? l : 1;
  f.s2 = l > 1 ? l - 1 : 0;
  return f;
}

__device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv& f) {
  const uint32_t t = __umulhi(f.m, n);
  return (t + ((n - t) >> f.s1)) >> f.s2;
}

struct Mfma32Args {
  const uint32_t* in;
  const uint32_t* w;
  const int32_t* thr;
  const uint32_t* flip;
  int32_t* sums;
  uint32_t* bits;
  int32_t H, W, Cw, F, Fw, KH, KW, pad, Ho, Wo, Hp, Wp;
  int32_t fstride;   // words per filter, KH*KW*Cw
  int32_t items;     // output pixels covered (N*Ho*Wo, or 4*N*Hp*Wp when pooling)
  int32_t K;         // valid bits per window, KH*KW*C
  int32_t in_bytes;  // raw-buffer ranges
  int32_t w_bytes;
  FastDiv div_w, div_h;  // Wo, Ho (or Wp, Hp when pooling)
  int32_t xcd_map;   // 1: one-dimensional grid in the XCD order of block_tile;
                     // 2: the same with the filter tiles split over XCD groups
  FastDiv div_f;     // filter tiles per XCD group (all of them with xcd_fs = 0)
  int32_t xcd_fs;    // log2 of the XCD groups the filter tiles are split over
  FastDiv div_c;     // word chunks per tap (Cc / (2 VW))
  int32_t Cc;        // words per tap the loop walks: Cw rounded up to whole chunks
  uint32_t tmask_c;  // valid bits of a pixel's last word (tail_mask(C))
  int32_t pad_bits;  // bit positions per window past C (KH KW (32 Cc - C))
  // Prepared weights (operand form, see prepare_weights_kernel): w holds
  // 16-byte entries [F / 32][KH][KW][Cp][32] and corr the per-filter offsets
  // B_f the sums come out too high by; null for packed weights.
  const int32_t* corr;
  int32_t Cp;        // entries per tap and filter of the prepared weights
};

// The workgroup's pixel block and filter tile.  The workgroups of a launch
// are handed to the 8 XCDs in turn (workgroup b to XCD b mod 8), and each
// XCD has its own L2.  In the XCD order the XCDs form p = 8 / g pixel groups
// times g filter groups (g = 2^xcd_fs): XCD x takes the filter tiles
// t = x mod g (mod g) and the pixel blocks x div g (mod p), and its k-th
// workgroup takes its filter tile k mod (fy / g) of its pixel block
// k div (fy / g).  The filter tiles of a pixel block run one after another
// on one XCD, so its activations are fetched into one L2, and with g = 1
// each output row (one piece per filter tile) is complete in that L2 before
// it is written back.  With g > 1 each L2 fetches only 1/g of the weights
// (tile_grid picks g from the layer's activation and weight bytes).
// Otherwise (a 2-D grid, pixel blocks varying fastest) a row's pieces come
// from workgroups far apart in time on all 8 XCDs and are written back piece
// by piece.  The padding workgroups past the last pixel block run through
// with every pixel invalid (their loads read the pad word, their stores are
// skipped): an early return would be a branch on a kernel argument that
// makes the kernel wait for that argument before it even loads the others.
__device__ __forceinline__ void block_tile(const Mfma32Args& a, int& pb, int& ft) {
  const uint32_t b = blockIdx.x;
  const uint32_t k = b >> 3, x = b & 7;
  const uint32_t q = fdiv(k, a.div_f);
  const uint32_t g1 = (1u << a.xcd_fs) - 1u;
  const int ftx = static_cast<int>(((k - q * a.div_f.d) << a.xcd_fs) + (x & g1));
  const int pbx = static_cast<int>((q << (3 - a.xcd_fs)) + (x >> a.xcd_fs));
  pb = a.xcd_map ? pbx : static_cast<int>(blockIdx.x);
  ft = a.xcd_map ? ftx : static_cast<int>(blockIdx.y);
}

// This lane's pixel in each of the TP 32-pixel tiles of a wave: byte offset
// of its first activation load, which taps fall inside the image, and the
// output coordinates for the epilogue.
template <int TP, bool POOL, int VW>
struct PixTiles {
  int pbase[TP], pn[TP], pi[TP], pj[TP];
  uint32_t tapmask[TP];
  bool pv[TP];

  __device__ __forceinline__ void init(const Mfma32Args& a, int p0, int h, int c) {
#pragma unroll
    for (int tp = 0; tp < TP; ++tp) {
      const int item = p0 + tp * 32 + c;
      pv[tp] = item < a.items;
      const uint32_t m = pv[tp] ? static_cast<uint32_t>(item) : 0u;
      uint32_t pix = POOL ? (m >> 2) : m;
      const uint32_t t = fdiv(pix, a.div_w);
      const uint32_t jj = pix - t * a.div_w.d;
      const uint32_t nn = fdiv(t, a.div_h);
      const uint32_t ii = t - nn * a.div_h.d;
      pn[tp] = static_cast<int>(nn);
      if constexpr (POOL) {
        pi[tp] = 2 * static_cast<int>(ii) + static_cast<int>((m >> 1) & 1);
        pj[tp] = 2 * static_cast<int>(jj) + static_cast<int>(m & 1);
      } else {
        pi[tp] = static_cast<int>(ii);
        pj[tp] = static_cast<int>(jj);
      }
      pbase[tp] = (((pn[tp] * a.H + pi[tp]) * a.W + pj[tp]) * a.Cw + h * VW) * 4;
      // rows kh with 0 <= i + kh - pad < H, columns likewise
      const int rlo = max(0, a.pad - pi[tp]), rhi = min(a.KH, a.H + a.pad - pi[tp]);
      const int clo = max(0, a.pad - pj[tp]), chi = min(a.KW, a.W + a.pad - pj[tp]);
      const uint32_t cm = chi > clo ? ((1u << chi) - 1u) & ~((1u << clo) - 1u) : 0u;
      uint32_t mk = 0;
      for (int kh = rlo; kh < rhi; ++kh) mk |= cm << (kh * a.KW);
      tapmask[tp] = pv[tp] ? mk : 0u;
    }
  }
};

// Loop position of the next load (wave-uniform): iteration l_it is tap
// (l_kh, l_kw), word chunk l_cc.  Advanced incrementally (no divisions in the
// loop); it stops at the last iteration it1 - 1, so extra loads past the end
// repeat it.
struct Cursor {
  int l_it, l_cc, l_kh, l_kw, it1;

  __device__ __forceinline__ void init(const Mfma32Args& a, int it0, int it1_, int nchunk,
                                       int vw) {
    it1 = it1_;
    l_it = it0;
    const int tap = it0 / nchunk;
    l_cc = (it0 - tap * nchunk) * 2 * vw;
    l_kh = tap / a.KW;
    l_kw = tap - l_kh * a.KW;
  }
  __device__ __forceinline__ int tap(const Mfma32Args& a) const { return l_kh * a.KW + l_kw; }
  __device__ __forceinline__ void advance(const Mfma32Args& a, int vw) {
    if (l_it + 1 < it1) {
      ++l_it;
      l_cc += 2 * vw;
      if (l_cc == a.Cc) {
        l_cc = 0;
        if (++l_kw == a.KW) {
          l_kw = 0;
          ++l_kh;
        }
      }
    }
  }
};

// Activation words of the cursor's iteration for the TP pixel tiles; taps
// outside the image read the out-of-range offset, i.e. the pad word 0.
template <int TP, bool POOL, int VW, bool SPLIT = false>
__device__ __forceinline__ void load_act(uint32_t (&aw)[TP][VW], const Mfma32Args& a,
                                         const Cursor& cur, const PixTiles<TP, POOL, VW>& px,
                                         __amdgpu_buffer_rsrc_t rin) {
  const int tap = cur.tap(a);
  const int dshift = (((cur.l_kh - a.pad) * a.W + (cur.l_kw - a.pad)) * a.Cw + cur.l_cc) * 4;
  const uint32_t bit = 1u << tap;
#pragma unroll
  for (int tp = 0; tp < TP; ++tp) {
    const uint32_t off = (px.tapmask[tp] & bit) ? static_cast<uint32_t>(px.pbase[tp] + dshift)
                                                : kOutOfRange;
    buf_load<VW, SPLIT>(aw[tp], rin, off, 0u);
  }
}

// Sums, threshold / flip, OR-pool and stores of a wave's TF x TP tiles.
// The thresholds and flip words are fetched at kernel start (EpiParams::
// fetch), so their global loads overlap the main loop instead of delaying its
// first loads or the epilogue; the block's thresholds then meet in LDS right
// before the epilogue.  Each is kept as thr - 0.5 in fp32 after clamping to
// [-K-1, K+1] (|S| <= K, so the clamp keeps every comparison, and the values
// stay exact in fp32 for any int32 threshold): S >= thr  <=>  (thr - 0.5) - S
// < 0 for integer S.
template <int TF>
struct EpiParams {
  int32_t thr;       // this thread's filter's threshold (threads < 32 TF)
  int32_t corr;      // how much too high this thread's filter's sums come out
  uint32_t fl[TF];   // flip words of the TF filter tiles (wave-uniform)

  __device__ __forceinline__ void fetch(const Mfma32Args& a, int f0) {
    thr = 0;
    const int f = min(f0 + static_cast<int>(threadIdx.x), a.F - 1);
    if (a.bits && threadIdx.x < 32 * TF) thr = a.thr[f];
    // packed weights: the zeroed padding positions (pad_bits, the same for
    // every filter); prepared weights: the filter's B_f
    corr = a.pad_bits;
    if (a.corr && threadIdx.x < 32 * TF) corr = a.corr[f];
#pragma unroll
    for (int tf = 0; tf < TF; ++tf) {
      const int wi = f0 / 32 + tf;
      fl[tf] = a.flip ? a.flip[wi < a.Fw ? wi : a.Fw - 1] : 0u;
    }
  }
  // Writes the block's thresholds to LDS, as thr + corr - 0.5 (or, with
  // `neg`, as 0.5 - thr - corr, the accumulators' start value), and with
  // prepared weights and sums wanted the offsets corr to cl; a barrier must
  // follow.
  __device__ __forceinline__ void stage(const Mfma32Args& a, float* thl, int32_t* cl,
                                        bool neg) const {
    if (a.bits && threadIdx.x < 32 * TF) {
      const float t = static_cast<float>(min(max(thr, -a.K - 1), a.K + 1) + corr) - 0.5f;
      thl[threadIdx.x] = neg ? -t : t;
    }
    if (a.corr && a.sums && threadIdx.x < 32 * TF) cl[threadIdx.x] = corr;
  }
};

// Accumulator start values.  With `pre` (bits wanted, no sums, thresholds
// already in LDS as 0.5 - thr) every accumulator of filter f starts at
// 0.5 - thr_f, so it ends at S - thr_f + 0.5, which is negative exactly when
// S < thr_f: its sign bit is the complement of the output bit, and the
// epilogue needs no subtraction.  The sums stay exact: |S - thr + 0.5| <=
// 2K + 1.5 < 2^23, half-integers exact in fp32 (K < 2^22,
// bconv_mfma_supported).
// Otherwise they start at 0.
template <int TF, int TP>
__device__ __forceinline__ void init_acc(v16f (&acc)[TF][TP], bool pre, const float* thl, int h) {
#pragma unroll
  for (int tf = 0; tf < TF; ++tf) {
    v16f t;
    if (pre) {
#pragma unroll
      for (int e = 0; e < 16; ++e) t[e] = thl[tf * 32 + 8 * (e >> 2) + 4 * h + (e & 3)];
    } else {
#pragma unroll
      for (int e = 0; e < 16; ++e) t[e] = 0.0f;
    }
#pragma unroll
    for (int tp = 0; tp < TP; ++tp) acc[tf][tp] = t;
  }
}

// Output bits of a wave's TF x TP tiles: threshold, flip, OR-pool, stores.
// PRE: the accumulators hold S - thr + 0.5 (init_acc), whose sign bit is the
// complement of the output bit; otherwise they hold S and the sign bit of
// (thr - 0.5) - S is the output bit.
// Both lane halves hold bits of every tile's word.  One v_permlane32_swap of
// two tiles' words leaves lane half h with the whole h-th word of the pair:
// with TF = 2 the pair is the two filter tiles of a pixel tile, with TF = 1
// the two pixel tiles, and every lane stores its own word.
template <bool PRE, int TF, int TP, bool POOL, int VW>
__device__ __forceinline__ void epi_bits(const Mfma32Args& a, v16f (&acc)[TF][TP],
                                         const PixTiles<TP, POOL, VW>& px, int p0, int f0,
                                         int h, int c, const float* thl,
                                         const EpiParams<TF>& ep) {
  static_assert(TP == 2 && (TF == 1 || TF == 2), "tile pairs");
  float th[TF][16];
  if constexpr (!PRE) {
#pragma unroll
    for (int tf = 0; tf < TF; ++tf)
#pragma unroll
      for (int e = 0; e < 16; ++e) th[tf][e] = thl[tf * 32 + 8 * (e >> 2) + 4 * h + (e & 3)];
  }
  // Filters 8 g + 4 h + r (r = 0..3) of register group g go to bits
  // 31 - 8 g - 4 h - r: shift the four signs into a nibble (v_alignbit takes
  // the sign bit of each value), then place the nibble.
  auto signs = [&](int tf, int tp) {
    uint32_t wd = 0u;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      uint32_t nib = 0u;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float d = PRE ? acc[tf][tp][4 * g + r] : th[tf][4 * g + r] - acc[tf][tp][4 * g + r];
        nib = __builtin_amdgcn_alignbit(nib, __float_as_uint(d), 31);
      }
      wd |= nib << (28 - 8 * g - 4 * h);  // nib < 16: four bits shifted into 0
    }
    return wd;
  };
  auto pair = [](uint32_t w0, uint32_t w1) {
    const auto sw = __builtin_amdgcn_permlane32_swap(w0, w1, false, false);
    return sw[0] | sw[1];
  };
  if constexpr (TF == 2) {
    const int wi = f0 / 32 + h;  // this lane half's filter word
    const uint32_t fl = h ? ep.fl[1] : ep.fl[0];
    const uint32_t fx = PRE ? ~fl : fl;
    const uint32_t fm = wi == a.Fw - 1 ? tail_mask(a.F) : ~0u;
#pragma unroll
    for (int tp = 0; tp < TP; ++tp) {
      uint32_t wd = (pair(signs(0, tp), signs(1, tp)) ^ fx) & fm;
      if constexpr (POOL) wd = or_quad(wd);
      const int item = p0 + tp * 32 + c;
      if ((!POOL || (c & 3) == 0) && px.pv[tp] && wi < a.Fw)
        a.bits[static_cast<size_t>(POOL ? (item >> 2) : item) * a.Fw + wi] = wd;
    }
  } else {
    const int wi = f0 / 32;
    const uint32_t fx = PRE ? ~ep.fl[0] : ep.fl[0];
    const uint32_t fm = wi == a.Fw - 1 ? tail_mask(a.F) : ~0u;
    uint32_t wd = (pair(signs(0, 0), signs(0, 1)) ^ fx) & fm;
    if constexpr (POOL) wd = or_quad(wd);
    const int item = p0 + h * 32 + c;  // lane half h: pixel tile h
    const bool pv = h ? px.pv[1] : px.pv[0];
    if ((!POOL || (c & 3) == 0) && pv)
      a.bits[static_cast<size_t>(POOL ? (item >> 2) : item) * a.Fw + wi] = wd;
  }
}

template <int TF, int TP, bool POOL, int VW>
__device__ __forceinline__ void epilogue(const Mfma32Args& a, v16f (&acc)[TF][TP],
                                         const PixTiles<TP, POOL, VW>& px, int p0, int f0,
                                         int h, int c, const float* thl, const int32_t* cl,
                                         const EpiParams<TF>& ep, bool pre) {
  // Filters past F (a partial last tile) read zero weights through the
  // buffer range and are masked out of every output.
  const bool ftail = f0 + 32 * TF > a.F;
  if (a.sums) {
#pragma unroll
    for (int tp = 0; tp < TP; ++tp) {
      if (!px.pv[tp]) continue;
      int32_t* sp = a.sums +
                    (static_cast<size_t>(px.pn[tp] * a.Ho + px.pi[tp]) * a.Wo + px.pj[tp]) * a.F +
                    f0 + 4 * h;
#pragma unroll
      for (int tf = 0; tf < TF; ++tf)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int fb = f0 + tf * 32 + 8 * g + 4 * h;  // first of 4 filters
          int cb[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) cb[e] = a.corr ? cl[tf * 32 + 8 * g + 4 * h + e] : a.pad_bits;
          if (!ftail && (a.F & 3) == 0) {
            int4 t;
            t.x = static_cast<int>(acc[tf][tp][4 * g + 0]) - cb[0];
            t.y = static_cast<int>(acc[tf][tp][4 * g + 1]) - cb[1];
            t.z = static_cast<int>(acc[tf][tp][4 * g + 2]) - cb[2];
            t.w = static_cast<int>(acc[tf][tp][4 * g + 3]) - cb[3];
            *reinterpret_cast<int4*>(sp + tf * 32 + 8 * g) = t;
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (fb + e < a.F)
                sp[tf * 32 + 8 * g + e] = static_cast<int>(acc[tf][tp][4 * g + e]) - cb[e];
          }
        }
    }
  }
  if (a.bits) {
    if (pre)
      epi_bits<true, TF, TP, POOL, VW>(a, acc, px, p0, f0, h, c, thl, ep);
    else
      epi_bits<false, TF, TP, POOL, VW>(a, acc, px, p0, f0, h, c, thl, ep);
  }
}

// Template parameters:
//   VW   words each lane loads per operand row and iteration (1, 2 or 4).
//        One MFMA k-step covers 2 words (one per lane half), so an
//        iteration (a chunk of 2*VW words of one tap) feeds VW k-steps.
//   POOL pixels of a 32-tile ordered as eight 2x2 windows (4 adjacent lanes).
//   TF   32-filter tiles per wave (1 or 2); a wave always covers 64 pixels.
//   KS   1: the 4 waves of a block take 4 consecutive 64-pixel groups;
//        >1: the KS (2..8; 2 or 4 with TF = 2) waves of a block split the
//        iterations of one tile and add their partial sums in LDS (grids too
//        small to fill the chip).
//   PD   register sets of loads in flight (prefetch depth).
//   LATE (KS = 1) the block's thresholds meet in LDS after the main loop, so
//        their load latency overlaps it; this costs a block barrier between
//        the loop and the epilogue, which pays on grids of at most about two
//        waves per SIMD but not on larger ones, where a wave's epilogue
//        otherwise overlaps the other waves' loops (then they are staged at
//        kernel start).  With KS > 1 they always meet after the loop, at the
//        barrier the partial sums need anyway.
//   TAIL C not a multiple of 64: activation words loaded one by one (rows of
//        an odd word count leave wider loads unaligned).
//   PREP weights in the prepared operand form (prepare_weights_kernel): each
//        weight word is one 16-byte load of its four registers, and the
//        activations take the cheaper encoding of act_operand; otherwise
//        each wave loads packed weight words and expands both operands with
//        expand_fp4 / expand_pair.
template <int VW, bool POOL, int TF, int KS, int PD, bool LATE, bool TAIL = false,
          bool PREP = false>
__global__ __launch_bounds__(KS == 1 ? 256 : 64 * KS) void bconv_mfma32_kernel(Mfma32Args a) {
  constexpr int TP = 2;
  using WReg = typename std::conditional<PREP, v4i, uint32_t>::type;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int h = lane >> 5;   // k half (operands) / row quad (result)
  const int c = lane & 31;   // operand row / column within a 32-tile
  int pb, ft;
  block_tile(a, pb, ft);
  const int p0 = (KS == 1 ? pb * 4 + wave : pb) * 64;
  const int f0 = ft * (32 * TF);
  const int nchunk = a.Cc / (2 * VW);
  const int iters = a.KH * a.KW * nchunk;
  int it0 = 0, it1 = iters;
  if constexpr (KS > 1) {
    const int per = (iters + KS - 1) / KS;
    it0 = min(iters, wave * per);
    it1 = min(iters, it0 + per);
  }

  __shared__ float thl[32 * TF];
  __shared__ int32_t cl[PREP ? 32 * TF : 1];
  EpiParams<TF> ep;
  ep.fetch(a, f0);
  // Thresholds staged at kernel start: the accumulators start from them.
  const bool pre = KS == 1 && !LATE && a.bits && !a.sums;
  if constexpr (KS == 1 && !LATE) {
    ep.stage(a, thl, cl, pre);
    __syncthreads();
  }

  PixTiles<TP, POOL, VW> px;
  px.init(a, p0, h, c);

  v16f acc[TF][TP];
  init_acc<TF, TP>(acc, pre, thl, h);

  const __amdgpu_buffer_rsrc_t rin = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint32_t*>(a.in), 0, a.in_bytes, kRsrcWord3);
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint32_t*>(a.w), 0, a.w_bytes, kRsrcWord3);
  // Byte offset of this lane's first weight word.  Prepared weights: the
  // 16-byte entries of word j of one tap for 32 consecutive filters are
  // adjacent, so each load instruction reads two runs of 512 bytes.
  uint32_t woff[TF];
#pragma unroll
  for (int tf = 0; tf < TF; ++tf)
    woff[tf] = PREP ? static_cast<uint32_t>((((f0 / 32 + tf) * a.fstride + h * VW) * 32 + c) * 16)
                    : static_cast<uint32_t>(((f0 + tf * 32 + c) * a.fstride + h * VW) * 4);
  const uint32_t smask = __builtin_amdgcn_readfirstlane(0x88888888u);
  uint32_t vfill;
  asm("v_mov_b32 %0, 0x22222222" : "=v"(vfill));

  Cursor cur;
  cur.init(a, it0, it1, nchunk, VW);
  auto load_next = [&](WReg (&ww)[TF][VW], uint32_t (&aw)[TP][VW]) {
    if constexpr (PREP) {
      const uint32_t wsoff = static_cast<uint32_t>((cur.tap(a) * a.Cp + cur.l_cc) * 512);
#pragma unroll
      for (int tf = 0; tf < TF; ++tf)
#pragma unroll
        for (int v = 0; v < VW; ++v)
          ww[tf][v] = __builtin_bit_cast(
              v4i, __builtin_amdgcn_raw_buffer_load_b128(rw, woff[tf] + 512 * v, wsoff, 0));
    } else {
      const uint32_t wsoff = static_cast<uint32_t>((cur.tap(a) * a.Cw + cur.l_cc) * 4);
#pragma unroll
      for (int tf = 0; tf < TF; ++tf) buf_load<VW, TAIL>(ww[tf], rw, woff[tf], wsoff);
    }
    load_act<TP, POOL, VW, TAIL>(aw, a, cur, px, rin);
    if constexpr (TAIL && !PREP) {
      // C not a multiple of 64: words past a pixel's Cw (read from the next
      // tap or pixel) and the tail bits of its last word are zeroed in both
      // operands.  Each such position then adds (+1)(+1) = 1 to the sum,
      // pad_bits per window in all, which the epilogue takes off.  (Prepared
      // weights hold 0.0 at those positions, so their products vanish.)
#pragma unroll
      for (int v = 0; v < VW; ++v) {
        const int wi = cur.l_cc + h * VW + v;
        const uint32_t m = wi < a.Cw - 1 ? ~0u : (wi == a.Cw - 1 ? a.tmask_c : 0u);
#pragma unroll
        for (int tf = 0; tf < TF; ++tf) ww[tf][v] &= m;
#pragma unroll
        for (int tp = 0; tp < TP; ++tp) aw[tp][v] &= m;
      }
    }
    cur.advance(a, VW);
  };
  auto compute = [&](const WReg (&ww)[TF][VW], const uint32_t (&aw)[TP][VW]) {
    constexpr int VP = (VW == 1 || PREP) ? 1 : 2;  // k-steps expanded together
#pragma unroll
    for (int v0 = 0; v0 < VW; v0 += VP) {
      v8i A[TF][VP], B[TP][VP];
      if constexpr (PREP) {
#pragma unroll
        for (int tf = 0; tf < TF; ++tf)
          A[tf][0] = v8i{ww[tf][v0][0], ww[tf][v0][1], ww[tf][v0][2], ww[tf][v0][3], 0, 0, 0, 0};
#pragma unroll
        for (int tp = 0; tp < TP; ++tp) B[tp][0] = act_operand(aw[tp][v0], smask, vfill);
      } else {
#pragma unroll
        for (int tf = 0; tf < TF; ++tf) {
          if constexpr (VP == 1) A[tf][0] = expand_fp4(ww[tf][v0], smask, vfill);
          else expand_pair(ww[tf][v0], ww[tf][v0 + 1], smask, vfill, A[tf][0], A[tf][1]);
        }
#pragma unroll
        for (int tp = 0; tp < TP; ++tp) {
          if constexpr (VP == 1) B[tp][0] = expand_fp4(aw[tp][v0], smask, vfill);
          else expand_pair(aw[tp][v0], aw[tp][v0 + 1], smask, vfill, B[tp][0], B[tp][1]);
        }
      }
#pragma unroll
      for (int v = 0; v < VP; ++v)
#pragma unroll
        for (int tf = 0; tf < TF; ++tf)
#pragma unroll
          for (int tp = 0; tp < TP; ++tp)
            acc[tf][tp] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                A[tf][v], B[tp][v], acc[tf][tp], 4, 4, 0, 127, 0, 127);
    }
  };

  if (it0 < it1) {
    // PD register sets in a ring: the loads of iteration it + PD are issued
    // right after iteration it's MFMAs, so PD - 1 iterations of loads are
    // always in flight.  The scheduling barriers keep each load in place
    // (the scheduler would otherwise sink it below the next MFMAs).
    WReg wr[PD][TF][VW];
    uint32_t xr[PD][TP][VW];
#pragma unroll
    for (int d = 0; d < PD; ++d) load_next(wr[d], xr[d]);
    for (int it = it0; it < it1; it += PD) {
#pragma unroll
      for (int d = 0; d < PD; ++d) {
        __builtin_amdgcn_sched_barrier(0);
        if (it + d < it1) compute(wr[d], xr[d]);
        __builtin_amdgcn_sched_barrier(0);
        load_next(wr[d], xr[d]);
      }
    }
  }

  if constexpr (KS == 1) {
    if constexpr (LATE) {
      ep.stage(a, thl, cl, false);
      __syncthreads();
    }
  } else {
    // Partial sums of the KS waves meet in LDS.  KS = 2: wave 1 stores its
    // tile and, after one barrier, wave 0 adds it to its own.  KS >= 4: every
    // wave stores its tile, all threads add the slots slice by slice into
    // slot 0 and wave 0 takes the totals (one barrier more, but wave 0 then
    // reads one tile instead of KS - 1).  Exact either way: integer sums
    // below 2^24.  (256 x 4096 -> 4096 GEMM, KS = 2: 8.36 -> 7.51 us with
    // the one-barrier form; the conv layers at batch 1, KS = 4: 0.04-0.12 us
    // slower with it.)
    constexpr int NV = TF * TP * 16 * 64;  // values per wave
    constexpr int SLOTS = KS == 2 ? 1 : KS;
    __shared__ float part[SLOTS][NV];
    ep.stage(a, thl, cl, false);
    if (KS > 2 || wave > 0) {
      const int slot = KS == 2 ? 0 : wave;
#pragma unroll
      for (int tf = 0; tf < TF; ++tf)
#pragma unroll
        for (int tp = 0; tp < TP; ++tp)
#pragma unroll
          for (int e = 0; e < 16; ++e)
            part[slot][((tf * TP + tp) * 16 + e) * 64 + lane] = acc[tf][tp][e];
    }
    __syncthreads();
    if constexpr (KS > 2) {
      for (int v = threadIdx.x; v < NV; v += 64 * KS) {
        float t = part[0][v];
#pragma unroll
        for (int w = 1; w < KS; ++w) t += part[w][v];
        part[0][v] = t;
      }
      __syncthreads();
    }
    if (wave > 0) return;
#pragma unroll
    for (int tf = 0; tf < TF; ++tf)
#pragma unroll
      for (int tp = 0; tp < TP; ++tp)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float t = part[0][((tf * TP + tp) * 16 + e) * 64 + lane];
          acc[tf][tp][e] = KS == 2 ? acc[tf][tp][e] + t : t;
        }
  }
  epilogue<TF, TP, POOL, VW>(a, acc, px, p0, f0, h, c, thl, cl, ep, pre);
}

// The same conv with the weights shared through LDS.  The 4 waves of a block
// take 4 pixel groups of 64 and the same TF filter tiles (TF = 1 or 2).
// The weight words of QS iterations at a time (a stage) are loaded once per
// block, expanded to fp4 once per block (instead of once per wave), and
// stored in LDS in the exact layout of the MFMA's A operand, so each k-step
// reads its TF operands with one conflict-free ds_read_b128 each.  Stages are
// double-buffered: the next stage's words are loaded during the current
// stage's MFMAs and expanded after them, and one barrier per stage separates
// the buffers.  Activations are loaded and expanded per wave as above.
constexpr int kQS = 4;  // iterations per stage

template <int VW, int TF>
struct LdsStage {
  // [buffer][iteration q][k-step v][filter tile][lane] x 16 bytes
  static constexpr int kOps = kQS * VW * TF;            // operand slots per buffer
  static constexpr int kChunks = kQS * TF * 32;         // (iteration, filter) pairs
  static constexpr int kPerThread = (kChunks + 255) / 256;
};

template <int VW, bool POOL, int TF, int PD, bool PRE>
__global__ __launch_bounds__(256) void bconv_mfma_lds_kernel(Mfma32Args a) {
  constexpr int TP = 2;
  using St = LdsStage<VW, TF>;
  __shared__ v4i wlds[2][St::kOps * 64];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int h = lane >> 5;
  const int c = lane & 31;
  int pb, ft;
  block_tile(a, pb, ft);
  const int p0 = (pb * 4 + wave) * 64;
  const int f0 = ft * (32 * TF);
  const int nchunk = a.Cc / (2 * VW);
  const int iters = a.KH * a.KW * nchunk;
  const int stages = (iters + kQS - 1) / kQS;

  PixTiles<TP, POOL, VW> px;
  px.init(a, p0, h, c);

  const __amdgpu_buffer_rsrc_t rin = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint32_t*>(a.in), 0, a.in_bytes, kRsrcWord3);
  const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint32_t*>(a.w), 0, a.w_bytes, kRsrcWord3);
  const uint32_t smask = __builtin_amdgcn_readfirstlane(0x88888888u);
  uint32_t vfill;
  asm("v_mov_b32 %0, 0x22222222" : "=v"(vfill));

  // Staging: thread t handles (iteration q, filter fi) pairs k = t + 256 j,
  // fi = k % (32 TF), q = k / (32 TF); it loads that filter's 2 VW words of
  // the stage's q-th iteration and writes their 2 VW expanded operands.
  uint32_t sw[St::kPerThread][2 * VW];
  auto stage_load = [&](int s) {
#pragma unroll
    for (int j = 0; j < St::kPerThread; ++j) {
      const int k = threadIdx.x + 256 * j;
      const int fi = k % (32 * TF), q = k / (32 * TF);
      const int it = s * kQS + q;
      uint32_t off = kOutOfRange;
      if (k < St::kChunks && it < iters) {
        const int tap = static_cast<int>(fdiv(static_cast<uint32_t>(it), a.div_c));
        const int cc = (it - tap * nchunk) * 2 * VW;
        off = static_cast<uint32_t>(((f0 + fi) * a.fstride + tap * a.Cw + cc) * 4);
      }
      if constexpr (VW == 2) {
        typedef unsigned int u4 __attribute__((ext_vector_type(4)));
        const u4 t = __builtin_amdgcn_raw_buffer_load_b128(rw, off, 0, 0);
        sw[j][0] = t[0];
        sw[j][1] = t[1];
        sw[j][2] = t[2];
        sw[j][3] = t[3];
      } else {
        typedef unsigned int u2 __attribute__((ext_vector_type(2)));
        const u2 t = __builtin_amdgcn_raw_buffer_load_b64(rw, off, 0, 0);
        sw[j][0] = t[0];
        sw[j][1] = t[1];
      }
    }
  };
  auto stage_store = [&](int buf) {
#pragma unroll
    for (int j = 0; j < St::kPerThread; ++j) {
      const int k = threadIdx.x + 256 * j;
      if (k >= St::kChunks) continue;
      const int fi = k % (32 * TF), q = k / (32 * TF);
      const int tf = fi >> 5, cr = fi & 31;
      // word wj of the chunk: lane half hh = wj / VW, k-step v = wj % VW
      v8i e[2 * VW];
      if constexpr (VW == 1) {
        e[0] = expand_fp4(sw[j][0], smask, vfill);
        e[1] = expand_fp4(sw[j][1], smask, vfill);
      } else {
#pragma unroll
        for (int wj = 0; wj < 2 * VW; wj += 2)
          expand_pair(sw[j][wj], sw[j][wj + 1], smask, vfill, e[wj], e[wj + 1]);
      }
#pragma unroll
      for (int wj = 0; wj < 2 * VW; ++wj) {
        const int hh = wj / VW, v = wj % VW;
        wlds[buf][((q * VW + v) * TF + tf) * 64 + hh * 32 + cr] =
            v4i{e[wj][0], e[wj][1], e[wj][2], e[wj][3]};
      }
    }
  };

  Cursor cur;
  cur.init(a, 0, iters, nchunk, VW);
  uint32_t xr[2][TP][VW];

  // Thresholds staged at kernel start (the barrier after the first weight
  // stage covers them), so no threshold register stays live in the loop;
  // the accumulators start from them.
  EpiParams<TF> ep;
  ep.fetch(a, f0);
  __shared__ float thl[32 * TF];
  // PRE (a template choice: a run-time one costs registers) = bits wanted
  // and no sums.
  constexpr bool pre = PRE;
  __shared__ int32_t cl_unused[1];  // (packed weights: no per-filter offsets)
  ep.stage(a, thl, cl_unused, pre);
  stage_load(0);
  stage_store(0);
#pragma unroll
  for (int d = 0; d < 2; ++d) {
    load_act<TP, POOL, VW>(xr[d], a, cur, px, rin);
    cur.advance(a, VW);
  }
  __syncthreads();
  v16f acc[TF][TP];
  init_acc<TF, TP>(acc, pre, thl, h);

  for (int s = 0; s < stages; ++s) {
    const int buf = s & 1;
    const bool more = s + 1 < stages;
    if (more) stage_load(s + 1);
#pragma unroll
    for (int q = 0; q < kQS; ++q) {
      const int it = s * kQS + q;
      __builtin_amdgcn_sched_barrier(0);
      if (it < iters) {
        v8i B[TP][VW];
#pragma unroll
        for (int tp = 0; tp < TP; ++tp) expand_words<VW>(xr[q & 1][tp], smask, vfill, B[tp]);
#pragma unroll
        for (int v = 0; v < VW; ++v) {
          v8i A[TF];
#pragma unroll
          for (int tf = 0; tf < TF; ++tf) {
            const v4i t = wlds[buf][((q * VW + v) * TF + tf) * 64 + lane];
            A[tf] = v8i{t[0], t[1], t[2], t[3], 0, 0, 0, 0};
          }
#pragma unroll
          for (int tf = 0; tf < TF; ++tf)
#pragma unroll
            for (int tp = 0; tp < TP; ++tp)
              acc[tf][tp] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                  A[tf], B[tp][v], acc[tf][tp], 4, 4, 0, 127, 0, 127);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      load_act<TP, POOL, VW>(xr[q & 1], a, cur, px, rin);
      cur.advance(a, VW);
    }
    if (more) stage_store(buf ^ 1);
    __syncthreads();
  }
  epilogue<TF, TP, POOL, VW>(a, acc, px, p0, f0, h, c, thl, cl_unused, ep, pre);
}

// Grid of `pblocks` pixel blocks x `fy` filter tiles: one-dimensional in the
// XCD order of block_tile, or 2-D.  The XCD order needs at least 8 pixel
// blocks: with fewer it would leave XCDs idle (all filter tiles of pixel
// block 0 on XCD 0), while the 2-D grid spreads the filter tiles over the
// XCDs.  With xcd_map = 2 the filter tiles are split over g = 1, 2, 4 or 8
// XCD groups (g dividing fy), g chosen to minimise the bytes the 8 L2s move
// in all, g * (activation bytes) + (8 / g) * (weight bytes) + g * (output
// bytes): each L2 then fetches 1/g of the weights, but every output row is
// written back in g pieces from g L2s.  (8x8x512 -> 512 pool at batch 64
// with prepared weights: 3.3 instead of 9.6 MB fetched, 0.5 instead of
// 0.06 MB written, 2 % slower; 8x8x256 -> 512: 6 % slower.  So xcd_map = 1,
// g = 1, is the default.)
dim3 tile_grid(Mfma32Args& a, unsigned pblocks, unsigned fy) {
  a.xcd_fs = 0;
  if (pblocks < 8) a.xcd_map = 0;
  if (!a.xcd_map) {
    a.div_f = make_fastdiv(fy);
    return dim3(pblocks, fy);
  }
  if (a.xcd_map == 2) {
    const int64_t out = a.sums ? int64_t{a.items} * a.F * 4 : int64_t{a.items} * a.Fw * 4;
    int64_t best = int64_t{a.in_bytes} + 8 * int64_t{a.w_bytes} + out;
    for (int fs = 1; fs <= 3; ++fs) {
      const int64_t g = int64_t{1} << fs;
      const int64_t t = g * a.in_bytes + (8 / g) * int64_t{a.w_bytes} + g * out;
      if (fy % g == 0 && t < best) {
        best = t;
        a.xcd_fs = fs;
      }
    }
  }
  const unsigned fyx = fy >> a.xcd_fs, p = 8u >> a.xcd_fs;
  a.div_f = make_fastdiv(fyx);
  return dim3((pblocks + p - 1) / p * 8 * fyx);
}

template <int VW, bool POOL, bool PREP>
hipError_t launch32(Mfma32Args a, int tf, int ks, bool lds, bool late, bool tail,
                    hipStream_t s) {
  const unsigned fy = static_cast<unsigned>((a.F + 32 * tf - 1) / (32 * tf));
  const unsigned groups = static_cast<unsigned>((a.items + 63) / 64);
  if (tail) {
    // C not a multiple of 64 (run_mfma: 32-filter tiles, thresholds after
    // the loop, no LDS staging).
    if (ks == 1) {
      const dim3 grid = tile_grid(a, (groups + 3) / 4, fy), block(256);
      bconv_mfma32_kernel<VW, POOL, 1, 1, 2, true, true, PREP><<<grid, block, 0, s>>>(a);
    } else {
      const dim3 grid = tile_grid(a, groups, fy), block(64 * ks);
      if (ks == 2)
        bconv_mfma32_kernel<VW, POOL, 1, 2, 2, true, true, PREP><<<grid, block, 0, s>>>(a);
      else
        bconv_mfma32_kernel<VW, POOL, 1, 4, 2, true, true, PREP><<<grid, block, 0, s>>>(a);
    }
    return hipGetLastError();
  }
  if constexpr (VW <= 2 && !PREP) {
    if (lds) {
      const dim3 grid = tile_grid(a, (groups + 3) / 4, fy), block(256);
      const bool pre = a.bits && !a.sums;
      if (tf == 2 && pre)
        bconv_mfma_lds_kernel<VW, POOL, 2, 2, true><<<grid, block, 0, s>>>(a);
      else if (tf == 2)
        bconv_mfma_lds_kernel<VW, POOL, 2, 2, false><<<grid, block, 0, s>>>(a);
      else if (pre)
        bconv_mfma_lds_kernel<VW, POOL, 1, 2, true><<<grid, block, 0, s>>>(a);
      else
        bconv_mfma_lds_kernel<VW, POOL, 1, 2, false><<<grid, block, 0, s>>>(a);
      return hipGetLastError();
    }
  }
  if (ks == 1) {
    const dim3 grid = tile_grid(a, (groups + 3) / 4, fy), block(256);
    if (tf == 2 && late)
      bconv_mfma32_kernel<VW, POOL, 2, 1, 2, true, false, PREP><<<grid, block, 0, s>>>(a);
    else if (tf == 2)
      bconv_mfma32_kernel<VW, POOL, 2, 1, 2, false, false, PREP><<<grid, block, 0, s>>>(a);
    else if (late)
      bconv_mfma32_kernel<VW, POOL, 1, 1, 2, true, false, PREP><<<grid, block, 0, s>>>(a);
    else
      bconv_mfma32_kernel<VW, POOL, 1, 1, 2, false, false, PREP><<<grid, block, 0, s>>>(a);
  } else {
    const dim3 grid = tile_grid(a, groups, fy), block(64 * ks);
    if (tf == 2) {
      if (ks == 2)
        bconv_mfma32_kernel<VW, POOL, 2, 2, 2, true, false, PREP><<<grid, block, 0, s>>>(a);
      else
        bconv_mfma32_kernel<VW, POOL, 2, 4, 2, true, false, PREP><<<grid, block, 0, s>>>(a);
    } else if (ks == 2) {
      bconv_mfma32_kernel<VW, POOL, 1, 2, 2, true, false, PREP><<<grid, block, 0, s>>>(a);
    } else if (ks == 4) {
      bconv_mfma32_kernel<VW, POOL, 1, 4, 2, true, false, PREP><<<grid, block, 0, s>>>(a);
    } else {
      bconv_mfma32_kernel<VW, POOL, 1, 8, 2, true, false, PREP><<<grid, block, 0, s>>>(a);
    }
  }
  return hipGetLastError();
}

template <int VW, bool POOL>
hipError_t launch_vw(Mfma32Args a, int tf, int ks, bool lds, bool late, bool tail,
                     hipStream_t s) {
  if (a.corr) return launch32<VW, POOL, true>(a, tf, ks, false, late, tail, s);
  return launch32<VW, POOL, false>(a, tf, ks, lds, late, tail, s);
}

// Launch plan of the matrix-core conv for a geometry: words per lane and
// iteration (vw), filter tiles per wave (tf), K split (ks), weights through
// LDS (lds), late threshold staging (late), C not a multiple of 64 (tail),
// and whether prepared weights pay (prep).
struct Plan {
  int vw, tf, ks;
  bool lds, late, tail, short8, prep;
};

Plan plan_mfma(const ConvGeom& g, bool pool) {
  const bnn_options& opt = options();
  Plan p;
  const int64_t items = pool ? 4 * int64_t{g.N} * g.Hp * g.Wp : int64_t{g.N} * g.Ho * g.Wo;
  const int64_t groups = (items + 63) / 64;
  const int64_t ftiles = (g.F + 31) / 32;
  // Words per lane, row and iteration: 8-word chunks (128-bit loads) where
  // the channels allow, which halves the vector-memory instructions per MFMA
  // (the texture-address unit is the busiest unit of the small grids), but
  // not when that leaves fewer than 8 iterations to split.
  // C not a multiple of 64: the loop walks Cc >= Cw words per tap, whole
  // chunks of 2 VW words, with the words past Cw zeroed and every word
  // loaded on its own (bconv_mfma32_kernel, TAIL).  VW is the largest of 4,
  // 2, 1 whose padding stays within 1/8 of the row.
  p.tail = g.C % 64 != 0;
  int vw = g.Cw % 8 == 0 ? 4 : g.Cw % 4 == 0 ? 2 : 1;
  // Windows of at most 4 eight-word chunks (K <= 1024 bits, e.g. FC layers
  // of 1024 inputs) on grids too small to fill the chip keep 8-word chunks
  // and no K split: there the split's LDS reduction costs more than it
  // hides (1024 -> 1024 and 1024 -> 10 at 64 rows: 4.15 and 4.30 us against
  // 4.42 and 4.57 us with 2-word chunks split 4 ways).
  const int chunks8 = g.KH * g.KW * (g.Cw / 8);
  p.short8 = !p.tail && vw == 4 && chunks8 <= 4 && groups * ftiles < 1024;
  if (vw == 4 && chunks8 < 8 && !p.short8) vw = 2;
  // Option lds_weights = 1 asks for the LDS-weights kernel wherever no K
  // split is used; it takes chunks of at most 2 words.
  if (opt.lds_weights == 1 && vw == 4) vw = 2;
  if (p.tail) {
    vw = 1;
    for (int t = 4; t >= 2 && vw == 1; t /= 2)
      if (((g.Cw + 2 * t - 1) / (2 * t) * (2 * t) - g.Cw) * 8 <= g.Cw) vw = t;
  }
  p.vw = vw;
  const int Cc = (g.Cw + 2 * vw - 1) / (2 * vw) * (2 * vw);
  const int iters = g.KH * g.KW * (Cc / (2 * vw));

  // Tile shape and K split: 64-filter wave tiles down to ~1 wave per SIMD
  // (1024 waves), then 32-filter tiles with a K split over up to 4 waves
  // until there are ~1 (8-word chunks) or ~2 (smaller chunks) waves per
  // SIMD, keeping at least 2 iterations per wave.  Splitting 8 ways never
  // beat 4 (the LDS reduction then costs more than it hides).  With 2-word
  // chunks, grids of >= 4096 64-filter tiles stage the weights through LDS
  // (5-20 % faster there, slower on smaller grids); 8-word chunks without
  // staging were as fast or faster wherever the channels allow them.  All
  // measured on every layer shape of the networks here.
  int tf = 2, ks = 1;
  if (g.F % 64 != 0 || groups * (g.F / 64) < 1024) {
    tf = 1;
    const int64_t target = vw == 4 ? 1024 : 2048;
    while (!p.short8 && ks < 4 && groups * ftiles * ks < target && iters >= 4 * ks) ks *= 2;
  }
  bool lds = opt.lds_weights == -1 ? vw <= 2 && tf == 2 && groups * (g.F / 64) >= 4096
                                    : opt.lds_weights == 1;
  if (ks > 1 || vw == 4) lds = false;
  if (p.tail) {
    tf = 1;
    lds = false;
    if (ks > 4) ks = 4;
  }
  p.tf = tf;
  p.ks = ks;
  p.lds = lds;
  // Thresholds staged after the main loop on grids of at most 2 waves per
  // SIMD (2048 waves) with 32-filter tiles, at kernel start otherwise, where
  // the accumulators can then start from them (16x16x128 -> 256 and
  // 16x16x256 -> 256 pool at batch 64: 5.98 / 7.50 us early against
  // 6.25 / 7.94 us late; 8x8x256 -> 512 with 32-filter tiles: 6.11 us late,
  // 6.22 us early).  Option late_thresholds overrides.
  const int64_t waves = (groups + 3) / 4 * 4 * ((g.F + 32 * tf - 1) / (32 * tf));
  p.late = p.tail || (opt.late_thresholds == -1 ? waves <= 2048 && tf == 1
                                                 : opt.late_thresholds == 1);
  // Prepared weights where they pay (graph-timed on every conv shape of the
  // networks here): 32-filter tiles, where a wave's vector-ALU work per MFMA
  // then drops from 12 to 8 instructions (8x8x512 -> 512 pool at batch 64:
  // 9.7 -> 8.2 us; 8x8x256 -> 512: 6.6 -> 6.0 us), and rows of at most 2
  // words.  With 64-filter tiles over 256 or more channels the prepared
  // operands' registers cost a wave per SIMD (180 against 154 VGPRs) and
  // 4x the weight bytes through L1: 56x56x256 -> 256 took 54 us packed and
  // 60-65 us prepared.  Rows of 4 words without LDS staging also pay
  // (16x16x128 -> 256 at batch 64: 6.3 -> 5.9 us); with LDS staging the
  // packed words are expanded once per block, which prepared operands
  // cannot match (48x48x128 -> 128 pool at batch 256: 48 against 54 us).
  p.prep = tf == 1 || g.Cw <= 2 || (g.Cw <= 4 && !lds);
  return p;
}

// wprep: prepared weights (prepare_weights_kernel), used instead of the
// packed w where plan_mfma says they pay, or null.
hipError_t run_mfma(const ConvGeom& g, bool pool, const uint32_t* in, const uint32_t* w,
                    const void* wprep, const int32_t* thr, const uint32_t* flip, int32_t* sums,
                    uint32_t* bits, hipStream_t s) {
  const Plan p = plan_mfma(g, pool);
  if (!p.prep) wprep = nullptr;
  Mfma32Args a;
  a.in = in;
  a.w = wprep ? static_cast<const uint32_t*>(wprep) : w;
  a.thr = thr;
  a.flip = flip;
  a.sums = sums;
  a.bits = bits;
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
  a.corr = nullptr;
  a.Cp = 0;
  if (wprep) {
    a.Cp = prepared_words_per_tap(g.C);
    a.fstride = g.KH * g.KW * a.Cp;  // entries per filter
    a.w_bytes = static_cast<int32_t>(static_cast<int64_t>(g.F + 31) / 32 * 32 * a.fstride * 16);
    a.corr = reinterpret_cast<const int32_t*>(static_cast<const char*>(wprep) + a.w_bytes);
  }
  a.div_w = make_fastdiv(static_cast<uint32_t>(pool ? g.Wp : g.Wo));
  a.div_h = make_fastdiv(static_cast<uint32_t>(pool ? g.Hp : g.Ho));
  a.xcd_map = options().xcd_order;
  const int vw = p.vw;
  a.Cc = (g.Cw + 2 * vw - 1) / (2 * vw) * (2 * vw);
  a.tmask_c = tail_mask(g.C);
  // (prepared weights hold 0.0 at the padding positions: no correction)
  a.pad_bits = wprep ? 0 : g.KH * g.KW * (32 * a.Cc - g.C);
  a.div_c = make_fastdiv(static_cast<uint32_t>(a.Cc / (2 * vw)));
  if (vw == 4)
    return pool ? launch_vw<4, true>(a, p.tf, p.ks, false, p.late, p.tail, s)
                : launch_vw<4, false>(a, p.tf, p.ks, false, p.late, p.tail, s);
  if (vw == 2)
    return pool ? launch_vw<2, true>(a, p.tf, p.ks, p.lds, p.late, p.tail, s)
                : launch_vw<2, false>(a, p.tf, p.ks, p.lds, p.late, p.tail, s);
  return pool ? launch_vw<1, true>(a, p.tf, p.ks, p.lds, p.late, p.tail, s)
              : launch_vw<1, false>(a, p.tf, p.ks, p.lds, p.late, p.tail, s);
}

// Prepared weights: entry (f, tap, j), j < Cp, holds the four fp4 registers
// of weight word j of filter f at that tap in the encoding act_operand pairs
// with.  Register r, nibble n carries bit 4n + r of the word: for r = 3 it is
// -1.0 (bit 1) or +1.0 (bit 0), for r = 0, 1, 2 it is +m or -m (bit 1 / bit
// 0) with m = 4, 2, 1; positions past C (tail bits, words past Cw) and
// filters past F hold 0.0.  The entries are stored [F / 32][tap][j][f % 32],
// the order in which a wave's 32-filter tile reads them.  corr[f] = B_f, the
// sum of s(w) over the valid positions of registers 0-2, is how much too high
// the matrix cores' window sums come out.  One block per filter (F rounded up
// to 32); done once per network, so written for clarity.
__global__ __launch_bounds__(256) void prepare_weights_kernel(const uint32_t* w, int32_t F,
                                                              int32_t taps, int32_t Cw,
                                                              int32_t Cp, int32_t C, v4i* out,
                                                              int32_t* corr) {
  const int f = blockIdx.x;
  __shared__ int32_t total;
  if (threadIdx.x == 0) total = 0;
  __syncthreads();
  int32_t cnt = 0;
  for (int e = threadIdx.x; e < taps * Cp; e += blockDim.x) {
    const int t = e / Cp, j = e - t * Cp;
    const bool fv = f < F;
    const uint32_t word = fv && j < Cw ? w[(static_cast<size_t>(f) * taps + t) * Cw + j] : 0u;
    const uint32_t valid =
        !fv ? 0u : j < Cw - 1 ? ~0u : (j == Cw - 1 ? tail_mask(C) : 0u);
    uint32_t reg[4] = {0u, 0u, 0u, 0u};
    for (int b = 0; b < 32; ++b) {
      if (!((valid >> b) & 1u)) continue;
      const int r = b & 3, n = b >> 2;
      const bool one = (word >> b) & 1u;
      uint32_t nib;
      if (r == 3) {
        nib = one ? 0xAu : 0x2u;
      } else {
        nib = (r == 0 ? 0x6u : r == 1 ? 0x4u : 0x2u) | (one ? 0u : 0x8u);
        cnt += one ? 1 : -1;
      }
      reg[r] |= nib << (4 * n);
    }
    out[((static_cast<size_t>(f / 32) * taps + t) * Cp + j) * 32 + f % 32] =
        v4i{static_cast<int>(reg[0]), static_cast<int>(reg[1]), static_cast<int>(reg[2]),
            static_cast<int>(reg[3])};
  }
  atomicAdd(&total, cnt);
  __syncthreads();
  if (threadIdx.x == 0 && f < F) corr[f] = total;
}

}  // namespace

bool bconv_mfma_supported(const ConvGeom& g) {
  // At least 32 channels (a C that is not a multiple of 64 is padded to
  // whole chunks, at most half of them padding), at most 32 taps (per-lane
  // tap masks), fewer than 2^22 bit positions per window, padding included
  // (the fp32 accumulators, which may start at 0.5 - thr, stay exact), and
  // inputs and weights under 2 GiB (32-bit byte offsets of the raw buffer
  // loads).
  return g.C >= 32 && g.KH * g.KW <= 32 &&
         static_cast<int64_t>(g.KH) * g.KW * 32 * (g.Cw + 7) < (int64_t{1} << 22) &&
         static_cast<int64_t>(g.N) * g.H * g.W * g.Cw < (int64_t{1} << 29) &&
         static_cast<int64_t>(g.F) * g.KH * g.KW * g.Cw < (int64_t{1} << 29);
}

hipError_t launch_bconv_mfma(const ConvGeom& g, const uint32_t* in, const uint32_t* w,
                             const void* wprep, const int32_t* thr, const uint32_t* flip,
                             int32_t* sums, uint32_t* bits, hipStream_t s) {
  if (g.pool == 2 && sums && ((g.Ho & 1) || (g.Wo & 1))) {
    hipError_t e = run_mfma(g, false, in, w, wprep, thr, flip, sums, nullptr, s);
    if (e != hipSuccess || !bits) return e;
    return run_mfma(g, true, in, w, wprep, thr, flip, nullptr, bits, s);
  }
  return run_mfma(g, g.pool == 2, in, w, wprep, thr, flip, sums, bits, s);
}

// Entries per tap and filter: Cw where C % 64 == 0 (every chunk width the
// launcher picks then divides Cw), else Cw rounded up to 8 (the loop walks
// whole chunks of up to 8 words past Cw, whose entries must read 0.0).
int32_t prepared_words_per_tap(int32_t C) {
  const int32_t Cw = static_cast<int32_t>(words_of(C));
  return C % 64 == 0 ? Cw : (Cw + 7) / 8 * 8;
}

int64_t prepared_weights_bytes(int32_t F, int32_t KH, int32_t KW, int32_t C) {
  return (int64_t{F} + 31) / 32 * 32 * KH * KW * prepared_words_per_tap(C) * 16 +
         (int64_t{F} * 4 + 15) / 16 * 16;
}

bool bconv_mfma_prep_supported(const ConvGeom& g) {
  return bconv_mfma_supported(g) &&
         prepared_weights_bytes(g.F, g.KH, g.KW, g.C) < (int64_t{1} << 31);
}

hipError_t launch_prepare_weights(int32_t F, int32_t KH, int32_t KW, int32_t C,
                                  const uint32_t* w, void* out, hipStream_t s) {
  const int32_t Cp = prepared_words_per_tap(C);
  const int32_t Fp = (F + 31) / 32 * 32;
  const int64_t entries = int64_t{Fp} * KH * KW * Cp;
  prepare_weights_kernel<<<dim3(static_cast<unsigned>(Fp)), dim3(256), 0, s>>>(
      w, F, KH * KW, static_cast<int32_t>(words_of(C)), Cp, C, static_cast<v4i*>(out),
      reinterpret_cast<int32_t*>(static_cast<char*>(out) + entries * 16));
  return hipGetLastError();
}

}  // namespace bnn
