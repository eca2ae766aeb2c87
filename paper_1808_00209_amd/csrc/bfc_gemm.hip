// Binary FC layer / GEMM (Sec. III-B, Eq. 4) for long rows at modest row
// counts: S[m][n] = sum_k a[m][k] b[n][k] over +-1 values, with the
// threshold / flip epilogue of bnn_bgemm.  K is at least 1024 bits; an N that
// is not a multiple of 32 leaves the last output tile partial (its weight rows
// past N read as 0 through the buffer range, and its outputs past N are
// neither stored nor set in the bits).  The FC tail needs whole tiles.
//
// A workgroup computes one 32 x 32 output tile (32 rows x 32 outputs) with 8
// waves, each taking one eighth of the K bits.  A wave loads its slice of
// both operands -- 32 weight rows and 32 data rows -- in chunks of up to 32
// words per row with 16-byte loads that cover whole cache lines, stages them
// in its own LDS region (only that wave touches it, and LDS operations of a
// wave complete in order, so no barrier), and runs the chunk's k-steps from
// there on the fp4 matrix cores.  The 8 partial tiles are summed in LDS
// (exact: integer sums below 2^24) and wave 0 writes the sums and/or bits.
// Grids of more than 512 tiles (N a multiple of 64) take 2 x 2 tiles per
// workgroup instead, two waves per tile with half of K each: a workgroup
// holds about 100 KB of LDS, so one runs per CU, and 1024 one-tile
// workgroups took four rounds.  Rows whose length is not whole k-steps per
// wave are padded with cleared words (the KT form of the kernel).
// The general matrix-core kernel loads each operand row straight from memory,
// 32 rows per load instruction, and runs the K split inside a workgroup of
// one output tile column: the 8192 -> 1024 layer at 64 rows ran on 32
// workgroups there, bound by those CUs' fetch path.

#include "fp4_expand.hpp"
#include "kernels.hpp"
#include "lane_ops.hpp"

namespace bnn {
namespace {

constexpr int kNW = 8;
constexpr int kNT = 64 * kNW;
constexpr int kCH = 32;        // words per row and chunk
constexpr int kRS = kCH + 2;   // LDS words per staged row (8-byte aligned rows)

struct GmArgs {
  const uint32_t* A;      // [M][Kw]
  const uint32_t* B;      // [N][Kw]
  const int32_t* thr;     // [N] (bits) or null
  const uint32_t* flip;   // [ceil(N / 32)] or null
  int32_t* sums;          // [M][N] or null
  uint32_t* bits;         // [M][ceil(N / 32)] or null
  int32_t M, N, Kw;       // Kw = ceil(K / 32), the row length in words
  int32_t Kwp;            // Kw rounded up to 4 KS words (whole k-steps per wave)
  int32_t K;              // bits
  int32_t a_bytes, b_bytes;
};

// The second layer of an FC tail (bnn_forward's FC pairs whose second layer
// has at most 32 outputs): w1 [N1][N / 32], thr1 / flip1 for bits out (else
// int32 sums out), and the accumulators: acc [kTailMaxRows][32] and wacc
// [kTailMaxRows], zero on entry and left zero.
struct TailArgs {
  const uint32_t* w1;
  const int32_t* thr1;
  const uint32_t* flip1;
  int32_t* sums;   // [M][N1] or null
  uint32_t* bits;  // [M][1] or null
  uint32_t* acc;
  unsigned long long* wacc;
  int32_t N1;
};

constexpr uint32_t kRsrcWord3 = 0x00020000;

// Sign bits of a 32 x 32 tile's accumulators: register e of lane (h, c)
// holds output 8 (e / 4) + 4 h + e % 4 of row c, which goes to bit 31 - that
// output; each lane half holds half of every row's word.
__device__ __forceinline__ uint32_t sign_word(const v16f& acc, int h) {
  uint32_t wd = 0u;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    uint32_t nib = 0u;
#pragma unroll
    for (int r = 0; r < 4; ++r)
      nib = __builtin_amdgcn_alignbit(nib, __float_as_uint(acc[4 * g + r]), 31);
    wd |= nib << (28 - 8 * g - 4 * h);
  }
  return wd;
}

// The tail of an FC pair, run by every thread of the workgroup that holds
// the first layer's 32 x 32 sums of rows m0 .. m0 + 31 and outputs
// 32 ft .. 32 ft + 31 in `tile` (MFMA layout).  Wave 0 thresholds them into
// one word per row; then each (row, tail output j) adds its partial sum over
// these 32 inputs, p = 32 - 2 popcount(word xor w1[j][ft]) (Eq. 4 on one
// word), to its accumulator with one atomic add of 2^17 + (p + 32): the high
// bits count the slices added, the low 17 bits their biased sum (at most
// 64 G < 2^17 for G = N / 32 <= 1024 slices).  The add that brings the count
// to G returns every other slice's contribution, so that thread alone writes
// the sum S = low bits + p + 32 - 32 G (or its bit) and zeroes the
// accumulator.  Bits out: the thread that finishes output j of a row adds
// 2^32 + its bit to the row's 64-bit word accumulator, and the add that
// brings that count to N1 writes the flipped word.  Read-modify-writes on
// one location are totally ordered, so no fence and no waiting between
// workgroups is needed, whichever XCD each runs on.
__device__ __forceinline__ void fc_tail(const GmArgs& a, const TailArgs& t, const float* tile,
                                        const float* th, const uint32_t* w1c,
                                        const int32_t* thr1s, int tid, int lane, int h, int c,
                                        int ft, int m0) {
  __shared__ uint32_t wrow[32];
  const int G = a.N / 32;
  if (tid < 64) {
    v16f d;
#pragma unroll
    for (int e = 0; e < 16; ++e) d[e] = tile[e * 64 + lane] + th[8 * (e >> 2) + 4 * h + (e & 3)];
    // output bit = (S >= thr) xor flip = sign xor ~flip
    const uint32_t word = or_xor32(sign_word(d, h)) ^ ~(a.flip ? a.flip[ft] : 0u);
    if (h == 0) wrow[c] = word;
  }
  __syncthreads();
  const int rows = min(32, a.M - m0);
  for (int e = tid; e < rows * t.N1; e += kNT) {
    const int cc = e / t.N1, j = e - cc * t.N1;
    const int m = m0 + cc;
    const int p = 32 - 2 * __builtin_popcount(wrow[cc] ^ w1c[j]);
    uint32_t* acc = &t.acc[m * 32 + j];
    const uint32_t add = (1u << 17) + static_cast<uint32_t>(p + 32);
    const uint32_t old =
        __hip_atomic_fetch_add(acc, add, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (static_cast<int>(old >> 17) != G - 1) continue;
    __hip_atomic_store(acc, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int32_t S = static_cast<int32_t>(old & 0x1FFFFu) + p + 32 - 32 * G;
    if (t.sums) {
      t.sums[static_cast<size_t>(m) * t.N1 + j] = S;
      continue;
    }
    const unsigned long long wadd =
        (1ull << 32) | (S >= thr1s[j] ? (0x80000000ull >> j) : 0ull);
    unsigned long long* wa = &t.wacc[m];
    const unsigned long long wold =
        __hip_atomic_fetch_add(wa, wadd, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (static_cast<int>(wold >> 32) != t.N1 - 1) continue;
    __hip_atomic_store(wa, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint32_t word = static_cast<uint32_t>(wold + wadd);
    t.bits[m] = (word ^ (t.flip1 ? t.flip1[0] : 0u)) & tail_mask(t.N1);
  }
}

// TPB x TFB output tiles of 32 x 32 per workgroup (rows x outputs) and KS
// waves per tile, each taking 1 / KS of K (TPB TFB KS = 8 waves): wave w
// computes tile (w % TPB, (w / TPB) % TFB) over slice w / (TPB TFB) of K.
// With TAIL (one tile per workgroup only) the tile's thresholded bits feed the
// tail layer instead of memory (fc_tail above).  With KT, K is not 32 Kwp:
// words at or past Kw read as 0 and the bits of the last word past K are
// cleared, in both operands.  Each such bit is +1.0 in both fp4 operands, so
// every sum comes out P = 32 Kwp - K too high, an exact integer that the
// epilogue takes off (thresholds included).
template <int TPB, int TFB, int KS, bool TAIL = false, bool KT = false>
__global__ __launch_bounds__(kNT) void bfc_gemm_kernel(GmArgs a, TailArgs t) {
  static_assert(TPB * TFB * KS == kNW, "8 waves");
  static_assert(!TAIL || (TPB * TFB == 1 && KS > 1), "the tail takes one tile per workgroup");
  constexpr int NTL = TPB * TFB;  // tiles per workgroup
  __shared__ __attribute__((aligned(16))) uint32_t stg[kNW][2][32 * kRS];
  __shared__ float part[kNW][16 * 64];
  __shared__ float th[32 * TFB];
  __shared__ uint32_t w1c[TAIL ? 32 : 1];
  __shared__ int32_t thr1s[TAIL ? 32 : 1];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = lane >> 5, c = lane & 31;
  const int ftb = (a.N + 32 * TFB - 1) / (32 * TFB);  // filter-tile groups
  const int ft0 = TFB * (blockIdx.x % ftb);         // first filter tile
  const int m00 = 32 * TPB * (blockIdx.x / ftb);    // first row
  const int tp = wave % TPB, tf = (wave / TPB) % TFB, ks = wave / NTL;
  const int ft = ft0 + tf;
  const int m0 = m00 + 32 * tp, n0 = 32 * ft;
  const bool want_bits = TAIL || a.bits != nullptr;
  // Thresholds (and the tail's weight words and thresholds) are loaded here
  // but stored to LDS only after the main loop, so that the wait for them
  // does not hold back the first operand loads.
  int32_t thv = 0, t1v = 0;
  uint32_t w1v = 0;
  const bool th_lane = want_bits && tid < 32 * TFB;
  if (th_lane && 32 * ft0 + tid < a.N) thv = a.thr[32 * ft0 + tid];
  const bool tail_lane = TAIL && tid >= 64 && tid < 64 + t.N1;
  if (tail_lane) {
    w1v = t.w1[static_cast<size_t>(tid - 64) * (a.N / 32) + ft0];
    if (t.thr1) t1v = t.thr1[tid - 64];
  }

  const __amdgpu_buffer_rsrc_t ra =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint32_t*>(a.A), 0, a.a_bytes, kRsrcWord3);
  const __amdgpu_buffer_rsrc_t rb =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint32_t*>(a.B), 0, a.b_bytes, kRsrcWord3);
  const uint32_t smask = __builtin_amdgcn_readfirstlane(0x88888888u);
  uint32_t vfill;
  asm("v_mov_b32 %0, 0x22222222" : "=v"(vfill));

  // This wave's K slice: words k0 .. k0 + sw - 1 of every row.
  const int sw = a.Kwp / KS;
  const uint32_t lastmask = tail_mask(a.K);  // valid bits of word Kw - 1
  // Clears the words of a loaded piece (words g .. g + 3) at or past Kw and
  // the bits past K of word Kw - 1.
  auto clip = [&](v4i& v, int g) {
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const uint32_t x = static_cast<uint32_t>(v[w]);
      v[w] = static_cast<int>(g + w < a.Kw - 1 ? x : g + w == a.Kw - 1 ? x & lastmask : 0u);
    }
  };
  const int k0 = ks * sw;
  v16f acc = {};
  // A chunk of ch words (a multiple of 4, at most 32) of 32 rows is 8 ch
  // 16-byte pieces; piece p = row (p / (ch / 4)), words 4 (p % (ch / 4)) ..
  // +3.  Load i of lane l takes piece 64 i + l.  Rows past M read row M - 1.
  for (int kc = 0; kc < sw; kc += kCH) {
    const int ch = min(kCH, sw - kc);
    const int ppr = ch / 4;  // pieces per row
    // p / ppr as (p rmag) >> 16: exact for p < 4096 and ppr <= 8, and two
    // vector instructions where an integer division takes dozens.
    const int rmag = (65536 + ppr - 1) / ppr;
    v4i pa[4], pb[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int p = min(64 * i + lane, 8 * ch - 1);
      const int row = (p * rmag) >> 16, col = 4 * (p - row * ppr);
      const int m = min(m0 + row, a.M - 1);
      const uint32_t wo = static_cast<uint32_t>(k0 + kc + col) * 4;
      pa[i] = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(
                                          ra, static_cast<uint32_t>(m) * a.Kw * 4 + wo, 0, 0));
      pb[i] = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(
                                          rb, static_cast<uint32_t>(n0 + row) * a.Kw * 4 + wo, 0, 0));
      if (KT && k0 + kc + ch >= a.Kw) {  // (wave-uniform: chunks that reach word Kw - 1)
        clip(pa[i], k0 + kc + col);
        clip(pb[i], k0 + kc + col);
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int p = 64 * i + lane;
      if (p < 8 * ch) {
        const int row = (p * rmag) >> 16, col = 4 * (p - row * ppr);
        uint32_t* da = &stg[wave][0][row * kRS + col];  // 8-byte aligned
        uint32_t* db = &stg[wave][1][row * kRS + col];
        *reinterpret_cast<uint2*>(da) = uint2{static_cast<uint32_t>(pa[i][0]),
                                              static_cast<uint32_t>(pa[i][1])};
        *reinterpret_cast<uint2*>(da + 2) = uint2{static_cast<uint32_t>(pa[i][2]),
                                                  static_cast<uint32_t>(pa[i][3])};
        *reinterpret_cast<uint2*>(db) = uint2{static_cast<uint32_t>(pb[i][0]),
                                              static_cast<uint32_t>(pb[i][1])};
        *reinterpret_cast<uint2*>(db + 2) = uint2{static_cast<uint32_t>(pb[i][2]),
                                                  static_cast<uint32_t>(pb[i][3])};
      }
    }
    // k-steps: lane (h, c) takes words 4 it + 2 h and 4 it + 2 h + 1 of
    // weight row c (operand A) and of data row c (operand B).
    for (int it = 0; it < ch / 4; ++it) {
      const uint2 wv = *reinterpret_cast<const uint2*>(&stg[wave][1][c * kRS + 4 * it + 2 * h]);
      const uint2 xv = *reinterpret_cast<const uint2*>(&stg[wave][0][c * kRS + 4 * it + 2 * h]);
      v8i A0, A1, B0, B1;
      expand_pair(wv.x, wv.y, smask, vfill, A0, A1);
      expand_pair(xv.x, xv.y, smask, vfill, B0, B1);
      acc = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(A0, B0, acc, 4, 4, 0, 127, 0, 127);
      acc = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(A1, B1, acc, 4, 4, 0, 127, 0, 127);
    }
  }
  const int32_t P = 32 * a.Kwp - a.K;  // sums come out P too high (KT)
  if (th_lane) {
    const int32_t K = a.K;
    th[tid] = 0.5f - static_cast<float>(min(max(thv, -K - 1), K + 1)) - static_cast<float>(P);
  }
  if (tail_lane) {
    w1c[tid - 64] = w1v;
    thr1s[tid - 64] = t1v;
  }
  // The KS partial tiles of each output tile meet in LDS (exact: integer
  // sums below 2^24): with one tile all threads add the slots slice by
  // slice; with several, the slice-0 wave of each tile adds the others'.
  if constexpr (KS > 1) {
    if (NTL == 1 || ks > 0) {
#pragma unroll
      for (int e = 0; e < 16; ++e) part[wave][e * 64 + lane] = acc[e];
    }
    __syncthreads();
    if constexpr (NTL == 1) {
#pragma unroll
      for (int i = 0; i < 16 * 64 / kNT; ++i) {
        const int v = tid + i * kNT;
        float t = part[0][v];
#pragma unroll
        for (int w = 1; w < kNW; ++w) t += part[w][v];
        part[0][v] = t;
      }
      __syncthreads();
      if constexpr (TAIL) {
        fc_tail(a, t, part[0], th, w1c, thr1s, tid, lane, h, c, ft, m0);
        return;
      }
      if (wave > 0) return;
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[e] = part[0][e * 64 + lane];
    } else {
      if (ks > 0) return;
#pragma unroll
      for (int q = 1; q < KS; ++q)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[e] += part[wave + q * NTL][e * 64 + lane];
    }
  }
  const int m = m0 + c;
  if (a.sums) {
    // The tile goes through this wave's staging region as [row][output], so
    // that each lane stores 16 consecutive bytes of a row.
    int32_t* ts = reinterpret_cast<int32_t*>(&stg[wave][0][0]);  // 32 x 33 words
#pragma unroll
    for (int e = 0; e < 16; ++e)
      ts[c * 33 + 8 * (e >> 2) + 4 * h + (e & 3)] = static_cast<int32_t>(acc[e]) - P;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = 8 * i + (lane >> 3), col = 4 * (lane & 7);
      const int* src = &ts[row * 33 + col];
      int32_t* dst = &a.sums[static_cast<size_t>(m0 + row) * a.N + n0 + col];
      if (m0 + row < a.M && n0 + col + 4 <= a.N && (a.N & 3) == 0) {
        *reinterpret_cast<int4*>(dst) = int4{src[0], src[1], src[2], src[3]};
      } else if (m0 + row < a.M) {
        // N not a multiple of 4: rows are not 16-byte aligned; past N: nothing
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (n0 + col + e < a.N) dst[e] = src[e];
      }
    }
  }
  if (want_bits) {
    v16f d;
#pragma unroll
    for (int e = 0; e < 16; ++e)
      d[e] = acc[e] + th[32 * tf + 8 * (e >> 2) + 4 * h + (e & 3)];
    // output bit = (S >= thr) xor flip = sign xor ~flip
    const int nw = (a.N + 31) / 32;
    const uint32_t word = (or_xor32(sign_word(d, h)) ^ ~(a.flip ? a.flip[ft] : 0u)) &
                          (ft == nw - 1 ? tail_mask(a.N) : ~0u);
    if (h == 0 && m < a.M) a.bits[static_cast<size_t>(m) * nw + ft] = word;
  }
}

// Kernel arguments for M x K rows against N x K weight rows, the row length
// padded to a multiple of `split` words (4 words per wave of the K split).
GmArgs gm_args(int64_t M, int64_t N, int64_t K, const uint32_t* A, const uint32_t* B,
               const int32_t* thr, const uint32_t* flip, int32_t* sums, uint32_t* bits,
               int split) {
  GmArgs a;
  a.A = A;
  a.B = B;
  a.thr = thr;
  a.flip = flip;
  a.sums = sums;
  a.bits = bits;
  a.M = static_cast<int32_t>(M);
  a.N = static_cast<int32_t>(N);
  a.Kw = static_cast<int32_t>((K + 31) / 32);
  a.Kwp = (a.Kw + split - 1) / split * split;
  a.K = static_cast<int32_t>(K);
  a.a_bytes = static_cast<int32_t>(M * a.Kw * 4);
  a.b_bytes = static_cast<int32_t>(N * a.Kw * 4);
  return a;
}

template <int TPB, int TFB, int KS>
void launch_tiles(const GmArgs& a, hipStream_t s) {
  const unsigned blocks =
      static_cast<unsigned>(((a.M + 32 * TPB - 1) / (32 * TPB)) *
                            ((a.N + 32 * TFB - 1) / (32 * TFB)));
  if (a.K == 32 * a.Kwp)
    bfc_gemm_kernel<TPB, TFB, KS><<<blocks, kNT, 0, s>>>(a, TailArgs{});
  else
    bfc_gemm_kernel<TPB, TFB, KS, false, true><<<blocks, kNT, 0, s>>>(a, TailArgs{});
}

}  // namespace

bool bfc_gemm_supported(int64_t M, int64_t N, int64_t K) {
  const int64_t kw = (K + 31) / 32 + 32;  // row words with the padding
  return M >= 1 && N >= 1 && K >= 1024 && K < (int64_t{1} << 28) &&
         M * kw * 4 < (int64_t{1} << 31) && N * kw * 4 < (int64_t{1} << 31) &&
         ((M + 31) / 32) * ((N + 31) / 32) < (int64_t{1} << 31);
}

hipError_t launch_bfc_gemm(int64_t M, int64_t N, int64_t K, const uint32_t* A,
                           const uint32_t* B, const int32_t* thr, const uint32_t* flip,
                           int32_t* sums, uint32_t* bits, hipStream_t s) {
  // One output tile per workgroup (K split 8 ways) up to 512 tiles; larger
  // grids take 2 x 2 tiles per workgroup with K split 2 ways (rows and
  // outputs in whole pairs of tiles).
  const int64_t tiles = ((M + 31) / 32) * ((N + 31) / 32);
  if (tiles <= 512 || N % 64 != 0)
    launch_tiles<1, 1, 8>(gm_args(M, N, K, A, B, thr, flip, sums, bits, 32), s);
  else
    launch_tiles<2, 2, 2>(gm_args(M, N, K, A, B, thr, flip, sums, bits, 8), s);
  return hipGetLastError();
}

bool bfc_tail_supported(int64_t M, int64_t K0, int64_t N0, int64_t N1) {
  return bfc_gemm_supported(M, N0, K0) && N0 % 32 == 0 && M <= kTailMaxRows &&
         N0 <= 32 * 1024 && N1 >= 1 &&
         N1 <= 32 && ((M + 31) / 32) * (N0 / 32) <= 512;
}

hipError_t launch_bfc_tail(int64_t M, int64_t K0, int64_t N0, int64_t N1, const uint32_t* A,
                           const uint32_t* w0, const int32_t* thr0, const uint32_t* flip0,
                           const uint32_t* w1, const int32_t* thr1, const uint32_t* flip1,
                           int32_t* sums, uint32_t* bits, void* accum, hipStream_t s) {
  const GmArgs a = gm_args(M, N0, K0, A, w0, thr0, flip0, nullptr, nullptr, 32);
  TailArgs t;
  t.w1 = w1;
  t.thr1 = thr1;
  t.flip1 = flip1;
  t.sums = sums;
  t.bits = bits;
  t.acc = static_cast<uint32_t*>(accum);
  t.wacc = reinterpret_cast<unsigned long long*>(static_cast<uint32_t*>(accum) +
                                                  kTailMaxRows * 32);
  t.N1 = static_cast<int32_t>(N1);
  const unsigned blocks = static_cast<unsigned>(((M + 31) / 32) * (N0 / 32));
  if (a.K == 32 * a.Kwp)
    bfc_gemm_kernel<1, 1, 8, true><<<blocks, kNT, 0, s>>>(a, t);
  else
    bfc_gemm_kernel<1, 1, 8, true, true><<<blocks, kNT, 0, s>>>(a, t);
  return hipGetLastError();
}

}  // namespace bnn
