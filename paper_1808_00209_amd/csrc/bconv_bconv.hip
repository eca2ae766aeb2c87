// Two consecutive binary 3x3 convs in one launch (Eq. 3 and Eq. 4 twice,
// each with its threshold and flip, the second with an optional 2x2 OR-pool;
// the conv -> conv steps of Table II's layer order): the first conv's output
// bits stay in LDS and never go to global memory.  Shapes: 16-pixel-wide
// images, pad 1 in both convs, 64, 128 or 256 input channels and 256 filters
// in each conv (the CIFAR-shaped net's 16 x 16 stage).
//
// A block owns 4 rows of one image (its second conv's output rows i0 .. i0 + 3,
// all 16 columns, all 256 filters), with 8 waves, one per 32-filter tile:
//   1. It stages the 8 input rows the first conv's windows need (i0 - 2 ..
//      i0 + 5) with one pad column on each side, every word already expanded
//      to its fp4 operand (pad and rows outside the image: the word 0, i.e.
//      -1), the thresholds of both convs, and the pad columns of the first
//      conv's output.  All global loads issue before the first LDS store.
//   2. First conv on the 6 rows i0 - 1 .. i0 + 4 (96 pixels, 3 tiles of 32):
//      wave w computes filter tile w on all three pixel tiles (one weight
//      operand per k-step serves three MFMAs), accumulators started at
//      0.5 - thr, and stores each output word, flipped and expanded, in LDS.
//      Rows outside the image get the pad word 0.
//   3. Second conv on the 4 output rows (64 pixels, 2 tiles): wave w computes
//      filter tile w with operands straight from LDS, then the threshold /
//      flip / OR-pool epilogue and the packed store.
// The ±1 dot products run on v_mfma_scale_f32_32x32x64_f8f6f4 with both
// operands in fp4 (E2M1 holds ±1 exactly; integer sums below 2^24 are exact
// in the fp32 accumulators).

#include "fp4_expand.hpp"
#include "kernels.hpp"
#include "lane_ops.hpp"

namespace bnn {
namespace {

constexpr int kW = 16;              // image width (both convs, pad 1)
constexpr int kF = 256;             // filters of each conv
constexpr int kNW = kF / 32;        // waves: one per 32-filter tile
constexpr int kNT = 64 * kNW;       // threads
constexpr int kCols = kW + 2;       // staged columns (one pad column each side)
constexpr int kCW1 = kF / 32;       // words per first-conv output pixel (8)
constexpr uint32_t kRsrcWord3 = 0x00020000;

struct BbArgs {
  const uint32_t* in;     // [N][H][16][CW0] packed input bits
  const uint32_t* w0;     // [256][9][CW0]
  const int32_t* thr0;    // [256]
  const uint32_t* flip0;  // [8] or null
  const uint32_t* w1;     // [256][9][8]
  const int32_t* thr1;    // [256]
  const uint32_t* flip1;  // [8] or null
  uint32_t* bits;         // [N][Hp][Wp][8]
  int32_t N, H;
  int32_t K0, K1;         // window bits of each conv (9 C)
  int32_t w0_bytes, w1_bytes;
  int32_t Hp, Wp;         // stored output (pooled dims when pooling)
};

constexpr int64_t kCUs = 256;       // compute units of the chip

// LDS row stride (in 16-byte entries) of a staged row of kCols pixels with
// ps entries each: a multiple of 8 plus 4, so that the 16-byte reads of
// lanes two rows apart fall on different banks.
constexpr int row_stride(int ps) { return kCols * ps + ((4 - (kCols * ps) % 8) + 8) % 8; }

// Iterations of a 3x3 window over CW words per pixel: one tap and a chunk
// of 2 VW words each.
template <int CW>
constexpr int window_iters() { return 9 * (CW / (2 * (CW % 4 == 0 ? 2 : 1))); }

// One 32-filter tile (filter tile `ft`) over TP pixel tiles of a conv whose
// activation operands sit in LDS: act[abase[tp] + tap offset + word] holds
// pixel tp's word as its fp4 operand.  Weights: packed words [F][9][CW],
// read through a buffer resource, expanded per k-step.  Iterations IT0 ..
// IT1 - 1 of the window (all of it by default).  Accumulators start from
// acc.
// Weight words of iteration `it` for lane (h, c) of 32-filter tile ft: VW
// words of filter 32 ft + c at tap it / NCH, words 2 VW (it % NCH) + h VW ..
template <int CW>
__device__ __forceinline__ void tile_w_load(const uint32_t* w, int w_bytes, int ft, int lane,
                                            int it, uint32_t (&ww)[CW % 4 == 0 ? 2 : 1]) {
  constexpr int VW = CW % 4 == 0 ? 2 : 1;
  constexpr int NCH = CW / (2 * VW);
  const int h = lane >> 5, c = lane & 31;
  const __amdgpu_buffer_rsrc_t rw =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint32_t*>(w), 0, w_bytes, kRsrcWord3);
  const uint32_t woff = static_cast<uint32_t>(((32 * ft + c) * 9 * CW + h * VW) * 4);
  const int tap = it / NCH, cc = (it - tap * NCH) * 2 * VW;
  const uint32_t so = static_cast<uint32_t>((tap * CW + cc) * 4);
  if constexpr (VW == 2) {
    typedef unsigned int u2 __attribute__((ext_vector_type(2)));
    const u2 t = __builtin_amdgcn_raw_buffer_load_b64(rw, woff, so, 0);
    ww[0] = t[0];
    ww[1] = t[1];
  } else {
    ww[0] = __builtin_amdgcn_raw_buffer_load_b32(rw, woff, so, 0);
  }
}

// With `first` non-null it holds iteration IT0's weight words, loaded by the
// caller (tile_w_load) ahead of its staging.
template <int CW, int TP, int RS, int PS, int IT0 = 0, int IT1 = window_iters<CW>()>
__device__ __forceinline__ void conv_tile(const v4i* act, const int (&abase)[TP],
                                          const uint32_t* w, int w_bytes, int ft, int lane,
                                          uint32_t smask, uint32_t vfill, v16f (&acc)[TP],
                                          const uint32_t* first = nullptr) {
  constexpr int VW = CW % 4 == 0 ? 2 : 1;  // words per lane per iteration
  constexpr int NCH = CW / (2 * VW);       // iterations per tap
  auto load_w = [&](int it, uint32_t (&ww)[VW]) { tile_w_load<CW>(w, w_bytes, ft, lane, it, ww); };
  uint32_t wr[2][VW];
  if (first) {
#pragma unroll
    for (int v = 0; v < VW; ++v) wr[0][v] = first[v];
  } else {
    load_w(IT0, wr[0]);
  }
#pragma unroll
  for (int it = IT0; it < IT1; ++it) {
    const int cur = (it - IT0) & 1;
    if (it + 1 < IT1) load_w(it + 1, wr[cur ^ 1]);
    const int tap = it / NCH, cc = (it - tap * NCH) * 2 * VW;
    const int kh = tap / 3, kw = tap - kh * 3;
    const int ao = kh * RS + kw * PS + cc;
    v8i B[TP][VW], A[VW];
#pragma unroll
    for (int tp = 0; tp < TP; ++tp)
#pragma unroll
      for (int v = 0; v < VW; ++v) {
        const v4i t = act[abase[tp] + ao + v];
        B[tp][v] = v8i{t[0], t[1], t[2], t[3], 0, 0, 0, 0};
      }
    expand_words<VW>(wr[cur], smask, vfill, A);
#pragma unroll
    for (int v = 0; v < VW; ++v)
#pragma unroll
      for (int tp = 0; tp < TP; ++tp)
        acc[tp] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(A[v], B[tp][v], acc[tp], 4, 4, 0,
                                                                  127, 0, 127);
  }
}

// Sign bits of a 32 x 32 tile's accumulators (S - thr + 0.5): register e of
// lane (h, c) holds filter 8 (e / 4) + 4 h + e % 4 at pixel c, which goes to
// bit 31 - that filter.  Each lane half holds half of every pixel's word.
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

// TH: second-conv output rows per block, 4, or 2 on grids smaller than the
// chip (twice the blocks, each with 4 first-conv rows for 2 output rows
// instead of 6 for 4).
template <int TH, int CW0, bool POOL>
__global__ __launch_bounds__(kNT) void bconv_bconv_kernel(BbArgs a) {
  constexpr int kTH = TH;
  constexpr int kRA = kTH + 2;         // first-conv rows a block computes
  constexpr int kRI = kTH + 4;         // input rows it stages
  constexpr int kPTA = kRA * kW / 32;  // first-conv pixel tiles (3 or 2)
  constexpr int kPTB = kTH * kW / 32;  // second-conv pixel tiles (2 or 1)
  constexpr int PSA = CW0 + 1;  // entries per staged input pixel (one spare)
  constexpr int RSA = row_stride(PSA);
  constexpr int PSB = kCW1 + 1;
  constexpr int RSB = row_stride(PSB);
  constexpr int NXA = kRI * kCols * CW0;        // staged input words
  constexpr int XIT = (NXA + kNT - 1) / kNT;
  constexpr int NPB = kRA * 2 * kCW1;           // pad-column entries of xb
  __shared__ v4i xa[kRI * RSA];
  __shared__ v4i xb[kRA * RSB];
  __shared__ float th0[kF];
  __shared__ float th1[kF];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int tiles_h = (a.H + kTH - 1) / kTH;  // (kTH rows per block)
  const int n = blockIdx.x / tiles_h;
  const int i0 = (blockIdx.x - n * tiles_h) * kTH;

  // 1. Staging: input words (clamped addresses, so the loads need no branch;
  // words outside the image are replaced by 0 afterwards), thresholds.
  uint32_t xw[XIT];
  bool xin[XIT];
#pragma unroll
  for (int i = 0; i < XIT; ++i) {
    const int e = tid + i * kNT;
    const int wd = e % CW0, t = e / CW0;
    const int col = t % kCols, row = t / kCols;
    const int y = i0 - 2 + row, x = col - 1;
    xin[i] = e < NXA && y >= 0 && y < a.H && x >= 0 && x < kW;
    const int yc = min(max(y, 0), a.H - 1), xc = min(max(x, 0), kW - 1);
    xw[i] = a.in[((static_cast<size_t>(n) * a.H + yc) * kW + xc) * CW0 + wd];
  }
  // thread t < 256: thr0[t]; t >= 256: thr1[t - 256]
  const int32_t thv = tid < kF ? a.thr0[tid] : a.thr1[tid - kF];
  const uint32_t nf0 = ~(a.flip0 ? a.flip0[wave] : 0u);
  const uint32_t nf1 = ~(a.flip1 ? a.flip1[wave] : 0u);

  const uint32_t smask = __builtin_amdgcn_readfirstlane(0x88888888u);
  uint32_t vfill;
  asm("v_mov_b32 %0, 0x22222222" : "=v"(vfill));

#pragma unroll
  for (int i = 0; i < XIT; ++i) {
    const int e = tid + i * kNT;
    if (e < NXA) {
      const int wd = e % CW0, t = e / CW0;
      const int col = t % kCols, row = t / kCols;
      const v8i x = expand_fp4(xin[i] ? xw[i] : 0u, smask, vfill);
      xa[row * RSA + col * PSA + wd] = v4i{x[0], x[1], x[2], x[3]};
    }
  }
  // The first conv's output columns -1 and 16 are the second conv's pad.
  {
    const v8i z = expand_fp4(0u, smask, vfill);
    for (int e = tid; e < NPB; e += kNT) {
      const int wd = e % kCW1, t = e / kCW1;
      const int side = t & 1, row = t >> 1;
      xb[row * RSB + (side ? kCols - 1 : 0) * PSB + wd] = v4i{z[0], z[1], z[2], z[3]};
    }
  }
  // Start values 0.5 - thr (thr clamped to [-K-1, K+1], which keeps every
  // comparison since |S| <= K): the sign bit of S - thr + 0.5 is set exactly
  // when S < thr, the complement of the output bit.
  if (tid < kF)
    th0[tid] = 0.5f - static_cast<float>(min(max(thv, -a.K0 - 1), a.K0 + 1));
  else
    th1[tid - kF] = 0.5f - static_cast<float>(min(max(thv, -a.K1 - 1), a.K1 + 1));
  __syncthreads();

  const int h = lane >> 5, c = lane & 31;
  // 2. First conv, filter tile `wave`, pixel tiles 0..kPTA-1 of the region
  // (pixel q = 32 tp + c at region row q / 16 = image row i0 - 1 + q / 16,
  // column q % 16).  Its window starts at staged row q / 16, column q % 16.
  {
    int abase[kPTA];
#pragma unroll
    for (int tp = 0; tp < kPTA; ++tp)
      abase[tp] = (2 * tp + (c >> 4)) * RSA + (c & 15) * PSA + h * (CW0 % 4 == 0 ? 2 : 1);
    v16f acc[kPTA];
    {
      v16f t;
#pragma unroll
      for (int e = 0; e < 16; ++e) t[e] = th0[32 * wave + 8 * (e >> 2) + 4 * h + (e & 3)];
#pragma unroll
      for (int tp = 0; tp < kPTA; ++tp) acc[tp] = t;
    }
    conv_tile<CW0, kPTA, RSA, PSA>(xa, abase, a.w0, a.w0_bytes, wave, lane, smask, vfill, acc);
    // Lane half h assembles the word of pixel tile h (tiles 0, 1) with one
    // v_permlane32_swap, and every lane the word of tile 2 (when there is one).
    const auto s01 = __builtin_amdgcn_permlane32_swap(sign_word(acc[0], h), sign_word(acc[1], h),
                                                      false, false);
    const uint32_t w01 = s01[0] | s01[1];
    auto put = [&](int tp, uint32_t word) {
      const int rq = 2 * tp + (c >> 4), cq = c & 15;
      const int y = i0 - 1 + rq;
      // output bit = (S >= thr) xor flip = sign xor ~flip; rows outside the
      // image are the second conv's pad (word 0)
      const v8i x = expand_fp4(y >= 0 && y < a.H ? word ^ nf0 : 0u, smask, vfill);
      xb[rq * RSB + (cq + 1) * PSB + wave] = v4i{x[0], x[1], x[2], x[3]};
    };
    put(h, w01);
    if constexpr (kPTA == 3) {
      const uint32_t w2 = or_xor32(sign_word(acc[2], h));
      if (h == 0) put(2, w2);
    }
  }
  __syncthreads();

  // 3. Second conv, filter tile `wave`, pixel tiles 0..kPTB-1 of the output
  // rows: tile tp, lane c is output pixel (2 tp + (c / 2) % 2,
  // 2 (c / 4) + c % 2), so each 2x2 pooling window sits in 4 adjacent lanes.
  // Its window starts at first-conv region row 2 tp + (c / 2) % 2, column
  // 2 (c / 4) + c % 2 (the region and its pad columns are offset by one).
  int bbase[kPTB];
#pragma unroll
  for (int tp = 0; tp < kPTB; ++tp)
    bbase[tp] = (2 * tp + ((c >> 1) & 1)) * RSB + (2 * (c >> 2) + (c & 1)) * PSB + h * 2;
  v16f acc[kPTB];
  {
    v16f t;
#pragma unroll
    for (int e = 0; e < 16; ++e) t[e] = th1[32 * wave + 8 * (e >> 2) + 4 * h + (e & 3)];
#pragma unroll
    for (int tp = 0; tp < kPTB; ++tp) acc[tp] = t;
  }
  conv_tile<kCW1, kPTB, RSB, PSB>(xb, bbase, a.w1, a.w1_bytes, wave, lane, smask, vfill, acc);
  // Lane half h gets the word of pixel tile h (with one tile, both halves
  // hold tile 0's word and half 0 stores it).
  uint32_t word;
  if constexpr (kPTB == 2) {
    const auto sw = __builtin_amdgcn_permlane32_swap(sign_word(acc[0], h), sign_word(acc[1], h),
                                                     false, false);
    word = (sw[0] | sw[1]) ^ nf1;
  } else {
    word = or_xor32(sign_word(acc[0], h)) ^ nf1;
  }
  const bool owner = kPTB == 2 || h == 0;
  const int pr = 2 * h + ((c >> 1) & 1), pc = 2 * (c >> 2) + (c & 1);
  if constexpr (POOL) {
    word = or_quad(word);
    const int ip = (i0 >> 1) + h, jp = c >> 2;
    if (owner && (c & 3) == 0 && ip < a.Hp)
      a.bits[(static_cast<size_t>(n * a.Hp + ip) * a.Wp + jp) * kCW1 + wave] = word;
  } else {
    const int i = i0 + pr;
    if (owner && i < a.H) a.bits[(static_cast<size_t>(n * a.H + i) * kW + pc) * kCW1 + wave] = word;
  }
}

template <int TH, int CW0>
hipError_t launch_cw(const BbArgs& a, bool pool, unsigned blocks, hipStream_t s) {
  if (pool)
    bconv_bconv_kernel<TH, CW0, true><<<blocks, kNT, 0, s>>>(a);
  else
    bconv_bconv_kernel<TH, CW0, false><<<blocks, kNT, 0, s>>>(a);
  return hipGetLastError();
}

template <int TH>
hipError_t launch_th(const BbArgs& a, int cw0, bool pool, hipStream_t s) {
  const unsigned blocks = static_cast<unsigned>(a.N) * ((a.H + TH - 1) / TH);
  switch (cw0) {
    case 2: return launch_cw<TH, 2>(a, pool, blocks, s);
    case 4: return launch_cw<TH, 4>(a, pool, blocks, s);
    default: return launch_cw<TH, 8>(a, pool, blocks, s);
  }
}

// One binary 3x3 conv with pad 1 on 8 x 8 maps (Eq. 3 and Eq. 4 with the
// threshold / flip / OR-pool epilogue), bits only.  An 8 x 8 image is
// exactly two 32-pixel tiles, so a block takes one image and 128 filters (64
// on small grids), with 2 waves per 32-filter tile: filter tile w / 2, half
// w % 2 of the window's iterations (the halves' partial tiles meet in LDS).  The image and its pad ring
// (10 x 10 pixels) are staged once per block, each word already expanded to
// its fp4 operand, so the k-steps read activations straight from LDS: no
// activation loads or expansion in the loop, where the general kernel loads
// every pixel's words once per tap and expands them per use.
struct ImArgs {
  const uint32_t* in;     // [N][8][8][CW]
  const uint32_t* w;      // [F][9][CW]
  const int32_t* thr;     // [F]
  const uint32_t* flip;   // [F / 32] or null
  uint32_t* bits;         // [N][Hp][Wp][F / 32]
  int32_t N, F, K;        // K = 9 C
  int32_t w_bytes;
};

constexpr int row_stride10(int ps) { return 10 * ps + ((4 - (10 * ps) % 8) + 8) % 8; }

// FPB: filters per block (128 or 64); 2 FPB / 32 waves.
template <int CW, bool POOL, int FPB>
__global__ __launch_bounds__(2 * FPB * 2) void bconv_img8_kernel(ImArgs a) {
  constexpr int NT = 2 * FPB * 2;  // threads: 2 waves per 32-filter tile
  constexpr int PS = CW + 1;  // entries per staged pixel (one spare)
  constexpr int RS = row_stride10(PS);
  constexpr int NX = 100 * CW;  // staged words
  constexpr int XIT = (NX + NT - 1) / NT;
  constexpr int ITERS = window_iters<CW>();
  constexpr int HALF = ITERS / 2;
  __shared__ v4i xa[10 * RS];
  __shared__ float th[FPB];
  __shared__ float part[FPB / 32][2 * 16 * 64];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int fgroups = a.F / FPB;
  const int n = blockIdx.x / fgroups;
  const int fg = blockIdx.x - n * fgroups;
  const int ft = (FPB / 32) * fg + (wave >> 1);  // filter tile
  const int kh = wave & 1;              // half of the window

  // Staging (clamped addresses; the pad ring gets the word 0, i.e. -1).
  uint32_t xw[XIT];
  bool xin[XIT];
#pragma unroll
  for (int i = 0; i < XIT; ++i) {
    const int e = tid + i * NT;
    const int wd = e % CW, t = e / CW;
    const int col = t % 10, row = t / 10;
    const int y = row - 1, x = col - 1;
    xin[i] = e < NX && y >= 0 && y < 8 && x >= 0 && x < 8;
    const int yc = min(max(y, 0), 7), xc = min(max(x, 0), 7);
    xw[i] = a.in[((static_cast<size_t>(n) * 8 + yc) * 8 + xc) * CW + wd];
  }
  const int32_t thv = a.thr[min(FPB * fg + tid, a.F - 1)];
  const uint32_t nfl = ~(a.flip ? a.flip[ft] : 0u);
  // This wave's first weight words, in flight during the staging.
  uint32_t wfirst[CW % 4 == 0 ? 2 : 1];
  tile_w_load<CW>(a.w, a.w_bytes, ft, lane, kh ? HALF : 0, wfirst);
  const uint32_t smask = __builtin_amdgcn_readfirstlane(0x88888888u);
  uint32_t vfill;
  asm("v_mov_b32 %0, 0x22222222" : "=v"(vfill));
#pragma unroll
  for (int i = 0; i < XIT; ++i) {
    const int e = tid + i * NT;
    if (e < NX) {
      const int wd = e % CW, t = e / CW;
      const v8i x = expand_fp4(xin[i] ? xw[i] : 0u, smask, vfill);
      xa[(t / 10) * RS + (t % 10) * PS + wd] = v4i{x[0], x[1], x[2], x[3]};
    }
  }
  // Start values 0.5 - thr (clamped to [-K-1, K+1]) for the first half;
  // the sign bit of the total is then the complement of the output bit.
  if (tid < FPB) th[tid] = 0.5f - static_cast<float>(min(max(thv, -a.K - 1), a.K + 1));
  __syncthreads();

  // Pixel tile tp = image rows 4 tp .. 4 tp + 3; lane c holds pixel
  // (4 tp + 2 (c / 16) + (c / 2) % 2, 2 ((c / 4) % 4) + c % 2), so each 2x2
  // pooling window sits in 4 adjacent lanes.  Its window starts at staged
  // row = that row, column = that column (the pad ring offsets by one).
  const int h = lane >> 5, c = lane & 31;
  const int qr = 2 * (c >> 4) + ((c >> 1) & 1), qc = 2 * ((c >> 2) & 3) + (c & 1);
  int bbase[2];
#pragma unroll
  for (int tp = 0; tp < 2; ++tp)
    bbase[tp] = (4 * tp + qr) * RS + qc * PS + h * (CW % 4 == 0 ? 2 : 1);
  v16f acc[2];
  {
    v16f t;
#pragma unroll
    for (int e = 0; e < 16; ++e)
      t[e] = kh ? 0.0f : th[32 * (wave >> 1) + 8 * (e >> 2) + 4 * h + (e & 3)];
    acc[0] = t;
    acc[1] = t;
  }
  if (kh)
    conv_tile<CW, 2, RS, PS, HALF, ITERS>(xa, bbase, a.w, a.w_bytes, ft, lane, smask, vfill, acc,
                                          wfirst);
  else
    conv_tile<CW, 2, RS, PS, 0, HALF>(xa, bbase, a.w, a.w_bytes, ft, lane, smask, vfill, acc,
                                      wfirst);
  // The second half's partial tiles to LDS, one barrier, the first half adds
  // them (exact: integer sums below 2^24).
  float* pp = part[wave >> 1];
  if (kh) {
#pragma unroll
    for (int tp = 0; tp < 2; ++tp)
#pragma unroll
      for (int e = 0; e < 16; ++e) pp[(tp * 16 + e) * 64 + lane] = acc[tp][e];
  }
  __syncthreads();
  if (kh) return;
#pragma unroll
  for (int tp = 0; tp < 2; ++tp)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[tp][e] += pp[(tp * 16 + e) * 64 + lane];
  // Lane half h gets the word of pixel tile h; output bit = sign xor ~flip.
  const auto sw = __builtin_amdgcn_permlane32_swap(sign_word(acc[0], h), sign_word(acc[1], h),
                                                   false, false);
  uint32_t word = (sw[0] | sw[1]) ^ nfl;
  const int fw = a.F / 32;
  if constexpr (POOL) {
    word = or_quad(word);
    const int ip = 2 * h + (c >> 4), jp = (c >> 2) & 3;
    if ((c & 3) == 0) a.bits[((static_cast<size_t>(n) * 4 + ip) * 4 + jp) * fw + ft] = word;
  } else {
    const int i = 4 * h + qr;
    a.bits[((static_cast<size_t>(n) * 8 + i) * 8 + qc) * fw + ft] = word;
  }
}

template <int CW, int FPB>
hipError_t launch_img8_cw(const ImArgs& a, bool pool, unsigned blocks, hipStream_t s) {
  if (pool)
    bconv_img8_kernel<CW, true, FPB><<<blocks, 4 * FPB, 0, s>>>(a);
  else
    bconv_img8_kernel<CW, false, FPB><<<blocks, 4 * FPB, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace

bool bconv_img8_supported(const ConvGeom& g) {
  return g.KH == 3 && g.KW == 3 && g.pad == 1 && g.H == 8 && g.W == 8 &&
         (g.C == 64 || g.C == 128 || g.C == 256 || g.C == 512) && g.F % 128 == 0 &&
         (g.pool == 0 || g.pool == 2) && int64_t{g.N} * (g.F / 128) < (int64_t{1} << 31);
}

hipError_t launch_bconv_img8(const ConvGeom& g, const uint32_t* in, const uint32_t* w,
                             const int32_t* thr, const uint32_t* flip, uint32_t* bits,
                             hipStream_t s) {
  ImArgs a;
  a.in = in;
  a.w = w;
  a.thr = thr;
  a.flip = flip;
  a.bits = bits;
  a.N = g.N;
  a.F = g.F;
  a.K = 9 * g.C;
  a.w_bytes = g.F * 9 * g.Cw * 4;
  // 128 filters per block where that gives a block per compute unit, 64 on
  // smaller grids (CIFAR L4 / L5 at batch 64: 5.1 / 6.7 us with 128, 5.3 /
  // 6.9 us with 64; the batch-1 forward 30.4 us with 64, 31.1 us with 128).
  const bool pool = g.pool == 2;
  if (int64_t{g.N} * (g.F / 128) >= kCUs) {
    const unsigned blocks = static_cast<unsigned>(g.N) * (g.F / 128);
    switch (g.Cw) {
      case 2: return launch_img8_cw<2, 128>(a, pool, blocks, s);
      case 4: return launch_img8_cw<4, 128>(a, pool, blocks, s);
      case 8: return launch_img8_cw<8, 128>(a, pool, blocks, s);
      default: return launch_img8_cw<16, 128>(a, pool, blocks, s);
    }
  }
  const unsigned blocks = static_cast<unsigned>(g.N) * (g.F / 64);
  switch (g.Cw) {
    case 2: return launch_img8_cw<2, 64>(a, pool, blocks, s);
    case 4: return launch_img8_cw<4, 64>(a, pool, blocks, s);
    case 8: return launch_img8_cw<8, 64>(a, pool, blocks, s);
    default: return launch_img8_cw<16, 64>(a, pool, blocks, s);
  }
}

bool bconv_bconv_supported(const ConvGeom& g0, const ConvGeom& g1) {
  return g0.KH == 3 && g0.KW == 3 && g0.pad == 1 && g0.pool == 0 && g0.W == kW &&
         (g0.C == 64 || g0.C == 128 || g0.C == 256) && g0.F == kF &&
         g1.KH == 3 && g1.KW == 3 && g1.pad == 1 && (g1.pool == 0 || g1.pool == 2) &&
         g1.C == kF && g1.F == kF && g1.N == g0.N && g1.H == g0.Ho && g1.W == g0.Wo &&
         static_cast<int64_t>(g0.N) * ((g0.H + 1) / 2) < (int64_t{1} << 31);
}

hipError_t launch_bconv_bconv(const ConvGeom& g0, const ConvGeom& g1, const uint32_t* in,
                              const uint32_t* w0, const int32_t* thr0, const uint32_t* flip0,
                              const uint32_t* w1, const int32_t* thr1, const uint32_t* flip1,
                              uint32_t* bits, hipStream_t s) {
  BbArgs a;
  a.in = in;
  a.w0 = w0;
  a.thr0 = thr0;
  a.flip0 = flip0;
  a.w1 = w1;
  a.thr1 = thr1;
  a.flip1 = flip1;
  a.bits = bits;
  a.N = g0.N;
  a.H = g0.H;
  a.K0 = 9 * g0.C;
  a.K1 = 9 * g1.C;
  a.w0_bytes = g0.F * 9 * g0.Cw * 4;
  a.w1_bytes = g1.F * 9 * g1.Cw * 4;
  a.Hp = g1.Hp;
  a.Wp = g1.Wp;
  // 4-row tiles while they give at least one block per compute unit, 2-row
  // tiles on smaller grids.
  const bool pool = g1.pool == 2;
  return int64_t{g0.N} * ((g0.H + 3) / 4) >= kCUs ? launch_th<4>(a, g0.Cw, pool, s)
                                                  : launch_th<2>(a, g0.Cw, pool, s);
}

}  // namespace bnn
