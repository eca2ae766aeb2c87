// Two consecutive binary FC layers in one launch (Sec. III-B, Eq. 4 twice):
// the first with its threshold and flip, the second to int32 sums (the
// logits layer) or to thresholded bits, the first layer's output bits kept in
// LDS.  For the last FC layers of a net, whose per-layer launches are bound
// by latency rather than work: 1024 -> 1024 -> 10 at 64 rows took two
// launches of 3.9 and 4.4 us.
//
// A workgroup takes 32 rows (one MFMA pixel tile) and 8 waves:
//   1. It stages its rows' K0 input bits in LDS as fp4 operands (rows past M
//      read as row M - 1 and are never stored), and both layers' thresholds.
//   2. First layer: wave w computes filter tiles FTW w .. FTW w + FTW - 1
//      (N0 = 256 FTW outputs) over all K0 bits.  Its filters' rows are one
//      contiguous block of the packed weights: it loads them (two filter
//      tiles at a time) with 16-byte loads that cover whole cache lines and
//      writes them to its own LDS region, from which each k-step reads the
//      32 rows of an operand.  (Operands loaded straight from the rows touched
//      32 cache lines per load and took 10.4 us for 1024 -> 1024 -> 10, the
//      two separate launches 8.6 us.)  The accumulators start at 0.5 - thr,
//      and each output word is flipped, expanded and stored in LDS.
//   3. Second layer (N1 <= 32 outputs, one filter tile): the N0 / 64 k-steps
//      are dealt out to the 8 waves, their partial tiles summed in LDS (exact:
//      integer sums below 2^24), then int32 sums or thresholded bits go out.
// The ±1 dot products run on v_mfma_scale_f32_32x32x64_f8f6f4 with fp4
// operands, exact for these integer sums.

#include "fp4_expand.hpp"
#include "kernels.hpp"
#include "lane_ops.hpp"

namespace bnn {
namespace {

constexpr int kNW = 8;
constexpr int kNT = 64 * kNW;
constexpr int kMaxN0W = 32;  // first-layer output words (N0 <= 1024)
constexpr uint32_t kRsrcWord3 = 0x00020000;

struct FpArgs {
  const uint32_t* A;      // [M][K0W]
  const uint32_t* w0;     // [N0][K0W]
  const int32_t* thr0;    // [N0]
  const uint32_t* flip0;  // [N0 / 32] or null
  const uint32_t* w1;     // [N1][N0 / 32]
  const int32_t* thr1;    // [N1] (bits output) or null (sums output)
  const uint32_t* flip1;  // [1] or null
  int32_t* sums;          // [M][N1] or null
  uint32_t* bits;         // [M][1] or null
  int32_t M, N1;
  int32_t w0_bytes, w1_bytes;
};

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

// K0W: words per input row (K0 = 32 K0W); FTW: 32-output tiles of the first
// layer per wave (N0 = 256 FTW).
template <int K0W, int FTW>
__global__ __launch_bounds__(kNT) void bfc_pair_kernel(FpArgs a) {
  constexpr int N0 = 256 * FTW;
  constexpr int N0W = N0 / 32;
  constexpr int PSA = K0W + 1;         // entries per staged input row (one spare)
  constexpr int PSB = N0W + 1;         // entries per first-layer output row
  constexpr int NXA = 32 * K0W;        // staged input words
  constexpr int XIT = (NXA + kNT - 1) / kNT;
  constexpr int ITERS = K0W / 4;       // 4 words (2 k-steps) per iteration
  constexpr int HF = FTW < 2 ? FTW : 2;  // filter tiles staged at a time
  constexpr int NH = FTW / HF;         // stages
  constexpr int RSW = K0W + 2;         // LDS words per staged filter row
  constexpr int NLD = HF * K0W / 8;    // 16-byte loads per lane per stage
  __shared__ v4i xa[32 * PSA];
  __shared__ v4i xb[32 * PSB];
  __shared__ float th0[N0];
  __shared__ float part[kNW][16 * 64];
  __shared__ __attribute__((aligned(16))) uint32_t wsm[kNW][HF * 32 * RSW];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = lane >> 5, c = lane & 31;
  const int m0 = blockIdx.x * 32;

  // 1. Staging (clamped row addresses: rows past M repeat row M - 1).
  uint32_t xw[XIT];
#pragma unroll
  for (int i = 0; i < XIT; ++i) {
    const int e = min(tid + i * kNT, NXA - 1);
    const int row = min(m0 + e / K0W, a.M - 1);
    xw[i] = a.A[static_cast<size_t>(row) * K0W + e % K0W];
  }
  const int32_t t0 = a.thr0[min(tid, N0 - 1)];
  const int32_t t0b = N0 > kNT ? a.thr0[min(tid + kNT, N0 - 1)] : 0;
  const __amdgpu_buffer_rsrc_t r0 =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint32_t*>(a.w0), 0, a.w0_bytes, kRsrcWord3);
  // Stage st of this wave's weights: filters 32 (FTW wave + HF st) onward,
  // HF 32 rows of K0W words, contiguous; load i of lane l reads bytes
  // 1024 i + 16 l of that block: row (1024 i + 16 l) / (4 K0W), words
  // from ((1024 i + 16 l) / 4) mod K0W.
  v4i wl[NLD];
  auto load_stage = [&](int st) {
    const uint32_t base = static_cast<uint32_t>(32 * (FTW * wave + HF * st) * K0W * 4);
#pragma unroll
    for (int i = 0; i < NLD; ++i)
      wl[i] = __builtin_bit_cast(
          v4i, __builtin_amdgcn_raw_buffer_load_b128(r0, base + 1024 * i + 16 * lane, 0, 0));
  };
  auto store_stage = [&]() {
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      const int byte = 1024 * i + 16 * lane;
      const int row = byte / (4 * K0W), wd = (byte / 4) % K0W;
      uint32_t* d = &wsm[wave][row * RSW + wd];  // 8-byte aligned: RSW, wd even
      *reinterpret_cast<uint2*>(d) = uint2{static_cast<uint32_t>(wl[i][0]),
                                           static_cast<uint32_t>(wl[i][1])};
      *reinterpret_cast<uint2*>(d + 2) = uint2{static_cast<uint32_t>(wl[i][2]),
                                               static_cast<uint32_t>(wl[i][3])};
    }
  };
  // (All stages' loads issued here instead: 7.7 against 7.45 us.)
  load_stage(0);

  const uint32_t smask = __builtin_amdgcn_readfirstlane(0x88888888u);
  uint32_t vfill;
  asm("v_mov_b32 %0, 0x22222222" : "=v"(vfill));
#pragma unroll
  for (int i = 0; i < XIT; ++i) {
    const int e = tid + i * kNT;
    if (e < NXA) {
      const v8i x = expand_fp4(xw[i], smask, vfill);
      xa[(e / K0W) * PSA + e % K0W] = v4i{x[0], x[1], x[2], x[3]};
    }
  }
  // Start values 0.5 - thr, thr clamped to [-K0-1, K0+1] (|S| <= K0 keeps
  // every comparison): the sign bit of S - thr + 0.5 is set exactly when
  // S < thr, the complement of the output bit.
  constexpr int K0 = 32 * K0W;
  if (tid < N0) th0[tid] = 0.5f - static_cast<float>(min(max(t0, -K0 - 1), K0 + 1));
  if (N0 > kNT && tid + kNT < N0)
    th0[tid + kNT] = 0.5f - static_cast<float>(min(max(t0b, -K0 - 1), K0 + 1));
  __syncthreads();

  // 2. First layer.
  v16f acc[FTW];
#pragma unroll
  for (int t = 0; t < FTW; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e)
      acc[t][e] = th0[32 * (FTW * wave + t) + 8 * (e >> 2) + 4 * h + (e & 3)];
  // Each stage: the wave's weight block goes to its own LDS region (written
  // and read by this wave only, so no barrier; LDS operations of a wave
  // complete in order), the next stage's loads go out, and the k-steps read
  // lane (h, c)'s words 4 it + 2 h, 4 it + 2 h + 1 of filter 32 t + c.
#pragma unroll
  for (int st = 0; st < NH; ++st) {
    store_stage();
    if (st + 1 < NH) load_stage(st + 1);
#pragma unroll
    for (int it = 0; it < ITERS; ++it) {
      v8i B[2];
#pragma unroll
      for (int v = 0; v < 2; ++v) {
        const v4i x = xa[c * PSA + 4 * it + 2 * h + v];
        B[v] = v8i{x[0], x[1], x[2], x[3], 0, 0, 0, 0};
      }
#pragma unroll
      for (int t = 0; t < HF; ++t) {
        const uint2 ww = *reinterpret_cast<const uint2*>(
            &wsm[wave][(32 * t + c) * RSW + 4 * it + 2 * h]);
        v8i A0, A1;
        expand_pair(ww.x, ww.y, smask, vfill, A0, A1);
        v16f& ac = acc[HF * st + t];
        ac = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(A0, B[0], ac, 4, 4, 0, 127, 0, 127);
        ac = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(A1, B[1], ac, 4, 4, 0, 127, 0, 127);
      }
    }
  }
  // Output words: lane half h assembles the word of tile t0 + h of each
  // tile pair with one v_permlane32_swap (a lone tile: both halves hold it).
  auto put = [&](int f, uint32_t word) {
    const uint32_t nf = ~(a.flip0 ? a.flip0[f] : 0u);  // out = sign xor ~flip
    const v8i x = expand_fp4(word ^ nf, smask, vfill);
    xb[c * PSB + f] = v4i{x[0], x[1], x[2], x[3]};
  };
#pragma unroll
  for (int t = 0; t + 1 < FTW; t += 2) {
    const auto s = __builtin_amdgcn_permlane32_swap(sign_word(acc[t], h), sign_word(acc[t + 1], h),
                                                    false, false);
    put(FTW * wave + t + h, s[0] | s[1]);
  }
  if constexpr (FTW % 2 == 1) {
    const uint32_t w = or_xor32(sign_word(acc[FTW - 1], h));
    if (h == 0) put(FTW * wave + FTW - 1, w);
  }
  __syncthreads();

  // 3. Second layer: k-step j (words 2 j, 2 j + 1 of a row) goes to wave
  // j mod 8; lane (h, c) holds word 2 j + h of row c and of output c.
  {
    const __amdgpu_buffer_rsrc_t r1 =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint32_t*>(a.w1), 0, a.w1_bytes, kRsrcWord3);
    constexpr int KS1 = N0W / 2;        // k-steps
    constexpr int JW = (KS1 + kNW - 1) / kNW;
    uint32_t w1v[JW];
#pragma unroll
    for (int q = 0; q < JW; ++q) {
      const int j = wave + kNW * q;
      // outputs past N1 read past the buffer: 0 (their sums are not stored)
      w1v[q] = j < KS1 ? __builtin_amdgcn_raw_buffer_load_b32(
                             r1, static_cast<uint32_t>((c * N0W + 2 * j + h) * 4), 0, 0)
                       : 0u;
    }
    v16f s1 = {};
#pragma unroll
    for (int q = 0; q < JW; ++q) {
      const int j = wave + kNW * q;
      if (j < KS1) {
        const v4i x = xb[c * PSB + 2 * j + h];
        s1 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
            expand_fp4(w1v[q], smask, vfill), v8i{x[0], x[1], x[2], x[3], 0, 0, 0, 0}, s1, 4, 4,
            0, 127, 0, 127);
      }
    }
#pragma unroll
    for (int e = 0; e < 16; ++e) part[wave][e * 64 + lane] = s1[e];
  }
  __syncthreads();
  // The 8 partial tiles summed slice by slice into slot 0.
#pragma unroll
  for (int i = 0; i < 16 * 64 / kNT; ++i) {
    const int v = tid + i * kNT;
    float t = part[0][v];
#pragma unroll
    for (int w = 1; w < kNW; ++w) t += part[w][v];
    part[0][v] = t;
  }
  __syncthreads();
  if (wave > 0) return;
  const int m = m0 + c;
  if (a.sums) {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int n = 8 * (e >> 2) + 4 * h + (e & 3);
      if (m < a.M && n < a.N1)
        a.sums[static_cast<size_t>(m) * a.N1 + n] = static_cast<int32_t>(part[0][e * 64 + lane]);
    }
    return;
  }
  // Bits: S - thr + 0.5 per output (thr clamped to [-N0-1, N0+1]), sign
  // word, lane halves joined, flipped, tail bits cleared.
  v16f d;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int n = 8 * (e >> 2) + 4 * h + (e & 3);
    const int32_t tn = a.thr1[min(n, a.N1 - 1)];
    d[e] = part[0][e * 64 + lane] + (0.5f - static_cast<float>(min(max(tn, -N0 - 1), N0 + 1)));
  }
  const uint32_t word = or_xor32(sign_word(d, h)) ^ ~(a.flip1 ? a.flip1[0] : 0u);
  if (h == 0 && m < a.M) a.bits[m] = word & tail_mask(a.N1);
}

template <int K0W>
hipError_t launch_k0(const FpArgs& a, int ftw, unsigned blocks, hipStream_t s) {
  switch (ftw) {
    case 1: bfc_pair_kernel<K0W, 1><<<blocks, kNT, 0, s>>>(a); break;
    case 2: bfc_pair_kernel<K0W, 2><<<blocks, kNT, 0, s>>>(a); break;
    default: bfc_pair_kernel<K0W, 4><<<blocks, kNT, 0, s>>>(a); break;
  }
  return hipGetLastError();
}

}  // namespace

bool bfc_pair_supported(int64_t M, int64_t K0, int64_t N0, int64_t N1) {
  return M >= 1 && M <= (int64_t{1} << 26) && (K0 == 512 || K0 == 1024) &&
         (N0 == 256 || N0 == 512 || N0 == 1024) && N1 >= 1 && N1 <= 32;
}

hipError_t launch_bfc_pair(int64_t M, int64_t K0, int64_t N0, int64_t N1, const uint32_t* A,
                           const uint32_t* w0, const int32_t* thr0, const uint32_t* flip0,
                           const uint32_t* w1, const int32_t* thr1, const uint32_t* flip1,
                           int32_t* sums, uint32_t* bits, hipStream_t s) {
  FpArgs a;
  a.A = A;
  a.w0 = w0;
  a.thr0 = thr0;
  a.flip0 = flip0;
  a.w1 = w1;
  a.thr1 = thr1;
  a.flip1 = flip1;
  a.sums = sums;
  a.bits = sums ? nullptr : bits;
  a.M = static_cast<int32_t>(M);
  a.N1 = static_cast<int32_t>(N1);
  a.w0_bytes = static_cast<int32_t>(N0 * K0 / 8);
  a.w1_bytes = static_cast<int32_t>(N1 * N0 / 8);
  const unsigned blocks = static_cast<unsigned>((M + 31) / 32);
  const int ftw = static_cast<int>(N0 / 256);
  return K0 == 512 ? launch_k0<16>(a, ftw, blocks, s) : launch_k0<32>(a, ftw, blocks, s);
}

}  // namespace bnn
