// Binary convolution and binary GEMM on the vector ALUs of gfx950:
// XOR + popcount dot products (Eq. 4 of the paper) over packed +-1 words, with
// the threshold / flip / 2x2 OR-pool epilogue fused in.
//
// Conv (Eq. 3, implicit im2col): lane = one output pixel, wave = 64 pixels x
// one group of 32 filters, so each lane ends with exactly one output word
// (32 filters' bits).  Per window word the lane does, for each of the 32
// filters, v_xor_b32 (activation in a VGPR, weight in an SGPR) and
// v_bcnt_u32_b32 (popcount plus accumulate): 2 VALU instructions per 32
// bit-MACs.  Weight words are wave-uniform, so they arrive through scalar
// loads and never occupy VGPRs or LDS.  Activation words come straight from
// global memory with 128-bit loads; each one feeds 64 VALU operations.
// Taps outside the image use the word 0 (all -1), the paper's pad value, so
// padding costs no extra arithmetic.  A FC layer / GEMM is the same kernel on
// a 1 x M "image" with a 1x1 kernel.
//
// Pooling: with pool == 2 the four lanes 4q..4q+3 of a wave hold the four
// pixels of one 2x2 window, so the OR-pool is two cross-lane shuffles.
//
// Small grids (FC layers at batch 64, late conv layers at batch 1) split the
// window words over up to 8 waves of a block and add the partial counts in
// LDS before the epilogue.
#include "kernels.hpp"

namespace bnn {
namespace {

// Weight words are read through the constant address space so that the
// compiler may use scalar loads for them (their addresses are wave-uniform).
typedef __attribute__((address_space(4))) const uint32_t cu32;

struct ConvArgs {
  const uint32_t* in;
  const uint32_t* w;
  const int32_t* thr;
  const uint32_t* flip;
  int32_t* sums;
  uint32_t* bits;
  int32_t N, H, W, Cw, F, Fw, KH, KW, pad, Ho, Wo, Hp, Wp;
  int32_t K;         // valid bits per window, KH*KW*C
  uint32_t tmask;    // valid bits of each pixel's last word
  int32_t fstride;   // words per filter, KH*KW*Cw
  int32_t items;     // N*Ho*Wo (no pool) or N*Hp*Wp (pool: one per window)
  int32_t nchunk;    // Cw / CH
  int32_t iters;     // KH*KW*nchunk
  int32_t per_wave;  // window iterations per wave when split over waves
};

template <int CH>
__device__ __forceinline__ void load_words(uint32_t (&v)[CH],
                                           const uint32_t* p, bool inside) {
  if constexpr (CH >= 4) {
#pragma unroll
    for (int q = 0; q < CH / 4; ++q) {
      uint4 t = inside ? reinterpret_cast<const uint4*>(p)[q] : make_uint4(0, 0, 0, 0);
      v[4 * q + 0] = t.x;
      v[4 * q + 1] = t.y;
      v[4 * q + 2] = t.z;
      v[4 * q + 3] = t.w;
    }
  } else if constexpr (CH == 2) {
    uint2 t = inside ? *reinterpret_cast<const uint2*>(p) : make_uint2(0, 0);
    v[0] = t.x;
    v[1] = t.y;
  } else {
    v[0] = inside ? *p : 0u;
  }
}

// KS == 1: the waves of a block take different filter groups.
// KS  > 1: the KS waves of a block share one filter group and split the
//          window iterations; partial counts are added in LDS.
template <int CH, bool POOL, bool FULL, bool TAIL, int KS>
__global__ __launch_bounds__(512) void bconv_valu_kernel(ConvArgs a) {
  const int lane = threadIdx.x & 63;
  // The wave index is uniform across the wave; readfirstlane tells the
  // compiler so, which keeps the weight addresses (and loads) scalar.
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  int fg, it0, it1;
  if constexpr (KS == 1) {
    fg = blockIdx.y * (blockDim.x >> 6) + wave;
    if (fg >= a.Fw) return;  // wave-uniform; this variant has no barrier
    it0 = 0;
    it1 = a.iters;
  } else {
    fg = blockIdx.y;
    it0 = wave * a.per_wave;
    it1 = min(a.iters, it0 + a.per_wave);
  }
  const int nf = FULL ? 32 : min(32, a.F - fg * 32);

  // Output pixel of this lane.
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

  uint32_t acc[32];
#pragma unroll
  for (int f = 0; f < 32; ++f) acc[f] = 0;

  cu32* wg = (cu32*)(a.w) + static_cast<size_t>(fg) * 32 * a.fstride;
#pragma unroll 1
  for (int it = it0; it < it1; ++it) {
    const int cc = it % a.nchunk;
    const int tap = it / a.nchunk;
    const int kh = tap / a.KW;
    const int kw = tap - kh * a.KW;
    const int hi = i + kh - a.pad;
    const int wi = j + kw - a.pad;
    const bool inside = valid && static_cast<unsigned>(hi) < static_cast<unsigned>(a.H) &&
                        static_cast<unsigned>(wi) < static_cast<unsigned>(a.W);
    const int c0 = cc * CH;
    const uint32_t* ap =
        a.in + (static_cast<size_t>(n * a.H + hi) * a.W + wi) * a.Cw + c0;
    uint32_t av[CH];
    load_words<CH>(av, ap, inside);
    const bool last = TAIL && (cc == a.nchunk - 1);
    if (last) av[CH - 1] &= a.tmask;
    cu32* wt = wg + tap * a.Cw + c0;
#pragma unroll
    for (int f = 0; f < 32; ++f) {
      if (FULL || f < nf) {
        cu32* wf = wt + f * a.fstride;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
          uint32_t wv = wf[c];
          if (c == CH - 1 && last) wv &= a.tmask;
          acc[f] += __builtin_popcount(av[c] ^ wv);
        }
      }
    }
  }

  if constexpr (KS > 1) {
    __shared__ uint32_t part[KS - 1][32][64];
    if (wave > 0) {
#pragma unroll
      for (int f = 0; f < 32; ++f) part[wave - 1][f][lane] = acc[f];
    }
    __syncthreads();
    if (wave > 0) return;
#pragma unroll
    for (int w = 0; w < KS - 1; ++w) {
#pragma unroll
      for (int f = 0; f < 32; ++f) acc[f] += part[w][f][lane];
    }
  }

  // Epilogue: S = K - 2 * popcount total; sums before pooling.
  if (a.sums && valid) {
    int32_t* sp = a.sums + (static_cast<size_t>(n * a.Ho + i) * a.Wo + j) * a.F + fg * 32;
    if (FULL && (a.F & 3) == 0) {
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        int4 t;
        t.x = a.K - 2 * static_cast<int>(acc[4 * q + 0]);
        t.y = a.K - 2 * static_cast<int>(acc[4 * q + 1]);
        t.z = a.K - 2 * static_cast<int>(acc[4 * q + 2]);
        t.w = a.K - 2 * static_cast<int>(acc[4 * q + 3]);
        reinterpret_cast<int4*>(sp)[q] = t;
      }
    } else {
#pragma unroll
      for (int f = 0; f < 32; ++f)
        if (f < nf) sp[f] = a.K - 2 * static_cast<int>(acc[f]);
    }
  }
  if (a.bits) {
    const int32_t* th = a.thr + fg * 32;
    uint32_t word = 0;
#pragma unroll
    for (int f = 0; f < 32; ++f) {
      if (FULL || f < nf) {
        const int s = a.K - 2 * static_cast<int>(acc[f]);
        word |= static_cast<uint32_t>(s >= th[f]) << (31 - f);
      }
    }
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

template <int CH, bool POOL, bool FULL, bool TAIL>
hipError_t dispatch_ks(const ConvArgs& a, int ks, hipStream_t s) {
  const int per_block = POOL ? 16 : 64;
  const unsigned gx = static_cast<unsigned>((a.items + per_block - 1) / per_block);
  if (ks == 1) {
    const int wpb = a.Fw < 4 ? a.Fw : 4;
    dim3 grid(gx, static_cast<unsigned>((a.Fw + wpb - 1) / wpb));
    bconv_valu_kernel<CH, POOL, FULL, TAIL, 1><<<grid, dim3(64 * wpb), 0, s>>>(a);
  } else {
    dim3 grid(gx, static_cast<unsigned>(a.Fw));
    if (ks == 2)
      bconv_valu_kernel<CH, POOL, FULL, TAIL, 2><<<grid, dim3(128), 0, s>>>(a);
    else if (ks == 4)
      bconv_valu_kernel<CH, POOL, FULL, TAIL, 4><<<grid, dim3(256), 0, s>>>(a);
    else
      bconv_valu_kernel<CH, POOL, FULL, TAIL, 8><<<grid, dim3(512), 0, s>>>(a);
  }
  return hipGetLastError();
}

template <int CH>
hipError_t dispatch_flags(const ConvArgs& a, bool pool, int ks, hipStream_t s) {
  const bool full = (a.F & 31) == 0;
  const bool tail = a.tmask != ~0u;
#define BNN_CASE(P, FU, T)                                                 \
  if (pool == P && full == FU && tail == T) return dispatch_ks<CH, P, FU, T>(a, ks, s);
  BNN_CASE(false, true, false)
  BNN_CASE(false, true, true)
  BNN_CASE(false, false, false)
  BNN_CASE(false, false, true)
  BNN_CASE(true, true, false)
  BNN_CASE(true, true, true)
  BNN_CASE(true, false, false)
  BNN_CASE(true, false, true)
#undef BNN_CASE
  return hipErrorInvalidValue;
}

hipError_t run_conv(const ConvGeom& g, bool pool, const uint32_t* in,
                    const uint32_t* w, const int32_t* thr, const uint32_t* flip,
                    int32_t* sums, uint32_t* bits, hipStream_t s) {
  const int CH = (g.Cw % 8 == 0) ? 8 : (g.Cw % 4 == 0) ? 4 : (g.Cw % 2 == 0) ? 2 : 1;
  ConvArgs a;
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
  a.K = g.KH * g.KW * g.C;
  a.tmask = tail_mask(g.C);
  a.fstride = g.KH * g.KW * g.Cw;
  a.items = pool ? g.N * g.Hp * g.Wp : g.N * g.Ho * g.Wo;
  a.nchunk = g.Cw / CH;
  a.iters = g.KH * g.KW * a.nchunk;

  // Split the window over waves when the grid alone cannot fill the chip
  // (about 2 waves per SIMD of the 1024 SIMDs).
  const int per_block = pool ? 16 : 64;
  const int64_t waves = static_cast<int64_t>((a.items + per_block - 1) / per_block) * a.Fw;
  int ks = 1;
  while (ks < 8 && waves * ks < 2048 && a.iters >= 2 * ks * 2) ks *= 2;
  a.per_wave = (a.iters + ks - 1) / ks;

  switch (CH) {
    case 8: return dispatch_flags<8>(a, pool, ks, s);
    case 4: return dispatch_flags<4>(a, pool, ks, s);
    case 2: return dispatch_flags<2>(a, pool, ks, s);
    default: return dispatch_flags<1>(a, pool, ks, s);
  }
}

// ---------------------------------------------------------------- GEMV ----
struct GemvArgs {
  const uint32_t* A;
  const uint32_t* B;
  const int32_t* thr;
  const uint32_t* flip;
  int32_t* sums;
  uint32_t* bits;
  int32_t M, N, Kw, K, Nw;
  uint32_t tmask;
};

// Binary GEMV / small GEMM for M <= 16 rows: a block of 16 waves computes 32
// output columns, wave w columns 2w and 2w+1.  Its 64 lanes stride along the
// K words of those two weight rows (coalesced 256-byte reads) and of the M
// activation rows, XOR + popcount into per-lane counts, and a wave
// reduction (cross-lane shuffles) gives each column's counts.  They meet in
// LDS, where the first 32 M threads turn them into sums and threshold bits,
// packed 32 columns to a word by ballot.
constexpr int kGemvWaves = 16;

template <int MT>
__global__ __launch_bounds__(1024) void bgemv_valu_kernel(GemvArgs a) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int n0 = blockIdx.x * 32;
  const int na = n0 + 2 * wave, nb = na + 1;
  const bool va = na < a.N, vb = nb < a.N;
  const uint32_t* ra = a.B + static_cast<size_t>(va ? na : 0) * a.Kw;
  const uint32_t* rb = a.B + static_cast<size_t>(vb ? nb : 0) * a.Kw;
  uint32_t ca[MT], cb[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) ca[m] = cb[m] = 0;
  // U strides of 64 words per trip, all loads issued before the popcounts:
  // one memory round trip per 64 U words rather than per 64 (18432 -> 100
  // at one row: 576 words, 3 trips instead of 9).
  constexpr int U = MT <= 2 ? 4 : (MT <= 4 ? 2 : 1);
  for (int j0 = lane; j0 < a.Kw; j0 += 64 * U) {
    uint32_t ba[U], bb[U], mk[U], av[U][MT];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + 64 * u;
      const bool in = j < a.Kw;
      mk[u] = !in ? 0u : (j == a.Kw - 1 ? a.tmask : ~0u);
      ba[u] = va && in ? ra[j] : 0u;
      bb[u] = vb && in ? rb[j] : 0u;
#pragma unroll
      for (int m = 0; m < MT; ++m)
        av[u][m] = m < a.M && in ? a.A[static_cast<size_t>(m) * a.Kw + j] : 0u;
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        ca[m] += __builtin_popcount((av[u][m] ^ ba[u]) & mk[u]);
        cb[m] += __builtin_popcount((av[u][m] ^ bb[u]) & mk[u]);
      }
  }
#pragma unroll
  for (int m = 0; m < MT; ++m) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      ca[m] += __shfl_xor(ca[m], off);
      cb[m] += __shfl_xor(cb[m], off);
    }
  }
  __shared__ uint32_t cnt[MT][32];
  if (lane == 0) {
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      cnt[m][2 * wave] = ca[m];
      cnt[m][2 * wave + 1] = cb[m];
    }
  }
  __syncthreads();
  const int t = threadIdx.x;
  if (t >= 32 * MT || t >= 32 * a.M) return;
  const int m = t >> 5, k = t & 31, n = n0 + k;
  const bool nvalid = n < a.N;
  const int S = a.K - 2 * static_cast<int>(cnt[m][k]);
  if (a.sums && nvalid) a.sums[static_cast<size_t>(m) * a.N + n] = S;
  if (a.bits) {
    // lanes 0..31 of a wave hold row m's 32 columns, lanes 32..63 row m + 1
    const bool bit = nvalid && S >= a.thr[n];
    const uint64_t mask = __ballot(bit);
    if (k == 0) {
      const int wi = n0 / 32;
      uint32_t word = __brev(static_cast<uint32_t>((lane & 32) ? (mask >> 32) : mask));
      if (a.flip) word ^= a.flip[wi];
      if (wi == a.Nw - 1) word &= tail_mask(a.N);
      a.bits[static_cast<size_t>(m) * a.Nw + wi] = word;
    }
  }
}

}  // namespace

hipError_t launch_bconv_valu(const ConvGeom& g, const uint32_t* in,
                             const uint32_t* w, const int32_t* thr,
                             const uint32_t* flip, int32_t* sums,
                             uint32_t* bits, hipStream_t s) {
  if (g.pool == 2 && sums && ((g.Ho & 1) || (g.Wo & 1))) {
    // Odd pre-pool sizes: the windows do not cover the last row / column, so
    // produce the sums with the unpooled mapping and the bits separately.
    hipError_t e = run_conv(g, false, in, w, thr, flip, sums, nullptr, s);
    if (e != hipSuccess || !bits) return e;
    return run_conv(g, true, in, w, thr, flip, nullptr, bits, s);
  }
  return run_conv(g, g.pool == 2, in, w, thr, flip, sums, bits, s);
}

hipError_t launch_bgemv_valu(int64_t M, int64_t N, int64_t K,
                             const uint32_t* A, const uint32_t* B,
                             const int32_t* thr, const uint32_t* flip,
                             int32_t* sums, uint32_t* bits, hipStream_t s) {
  GemvArgs a;
  a.A = A;
  a.B = B;
  a.thr = thr;
  a.flip = flip;
  a.sums = sums;
  a.bits = bits;
  a.M = static_cast<int32_t>(M);
  a.N = static_cast<int32_t>(N);
  a.Kw = static_cast<int32_t>(words_of(K));
  a.K = static_cast<int32_t>(K);
  a.Nw = static_cast<int32_t>(words_of(N));
  a.tmask = tail_mask(K);
  dim3 grid(static_cast<unsigned>((N + 31) / 32));
  dim3 block(64 * kGemvWaves);
  if (M <= 1)
    bgemv_valu_kernel<1><<<grid, block, 0, s>>>(a);
  else if (M <= 2)
    bgemv_valu_kernel<2><<<grid, block, 0, s>>>(a);
  else if (M <= 4)
    bgemv_valu_kernel<4><<<grid, block, 0, s>>>(a);
  else if (M <= 8)
    bgemv_valu_kernel<8><<<grid, block, 0, s>>>(a);
  else
    bgemv_valu_kernel<16><<<grid, block, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace bnn
