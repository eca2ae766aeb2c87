// Launchers of the gfx950 kernels behind the C ABI (include/bnn.h).  The
// C-ABI layer in api.cpp validates every argument before calling these; the
// launchers assume valid shapes, 16-byte aligned buffers and non-empty work.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bnn.h"

namespace bnn {

// The calling thread's kernel-selection options (bnn_set_options).
const bnn_options& options();

// Mask of the valid (high) bits of the last word of a packed vector of
// `bits` values: value i of a word sits in bit 31 - i.
inline __host__ __device__ uint32_t tail_mask(int64_t bits) {
  const int r = static_cast<int>(bits & 31);
  return r ? (~0u << (32 - r)) : ~0u;
}

inline int64_t words_of(int64_t bits) { return (bits + 31) >> 5; }

// Geometry of one binary conv launch (stride 1).
struct ConvGeom {
  int32_t N, H, W, C, F, KH, KW, pad, pool;
  int32_t Cw, Fw, Ho, Wo, Hp, Wp;
};

hipError_t launch_pack_bits(const float* x, const float* offset, int64_t rows,
                            int64_t D, uint32_t* out, hipStream_t s);

// Binary conv via XOR + popcount on the vector ALUs.  sums / bits may be
// null; thr must be non-null when bits is.  flip may be null.
hipError_t launch_bconv_valu(const ConvGeom& g, const uint32_t* in,
                             const uint32_t* w, const int32_t* thr,
                             const uint32_t* flip, int32_t* sums,
                             uint32_t* bits, hipStream_t s);

// Binary 1x1 conv with C = 64, 128 or 256, F a multiple of 64 (at
// most 1024), no padding or pooling, over at least 65536 pixels, bits only:
// a wave keeps its pixels' fp4 operands and walks all filters.
bool bconv1x1_supported(const ConvGeom& g, bool sums);
hipError_t launch_bconv1x1(const ConvGeom& g, const uint32_t* in, const uint32_t* w,
                           const int32_t* thr, const uint32_t* flip, uint32_t* bits,
                           hipStream_t s);

// Binary conv on the matrix cores (fp4 MFMA).  Supported when
// bconv_mfma_supported(g): C >= 32 (padded to whole 64-bit chunks), at most
// 32 taps.
// wprep: the weights prepared by launch_prepare_weights (used instead of w),
// or null.
bool bconv_mfma_supported(const ConvGeom& g);
hipError_t launch_bconv_mfma(const ConvGeom& g, const uint32_t* in,
                             const uint32_t* w, const void* wprep,
                             const int32_t* thr, const uint32_t* flip,
                             int32_t* sums, uint32_t* bits, hipStream_t s);

// Prepared ("operand form") conv weights for the matrix-core kernel: 16-byte
// entries [ceil(F / 32)][KH][KW][Cp][32] (Cp = Cw when C % 64 == 0, else
// Cw rounded up to 8) holding each
// weight word's four fp4 registers, then F int32 per-filter offsets.  Supported where
// bconv_mfma_supported holds and the buffer stays under 2 GiB.
int32_t prepared_words_per_tap(int32_t C);
int64_t prepared_weights_bytes(int32_t F, int32_t KH, int32_t KW, int32_t C);
bool bconv_mfma_prep_supported(const ConvGeom& g);
hipError_t launch_prepare_weights(int32_t F, int32_t KH, int32_t KW, int32_t C,
                                  const uint32_t* w, void* out, hipStream_t s);

// Input binarization (bnn_input_mode of bnn.h) of an fp32 image into one
// code word per pixel, and the binary conv over an image binarized on the
// fly with one window packed into ceil(KH*KW*C / 32) words.  Supported when
// bconv_patch_supported(g): C, KH, KW <= 32 and KH*KW*C <= 128.  g.C is the
// binarized channel count, input_channels_of(mode, Cin).
int input_channels_of(int mode, int cin);
hipError_t launch_binarize(int mode, const float* x, const float* offset,
                           int32_t N, int32_t H, int32_t W, int32_t Cin,
                           uint32_t* out, hipStream_t s);
bool bconv_patch_supported(const ConvGeom& g);
hipError_t launch_bconv_patch(const ConvGeom& g, int mode, const float* x,
                              const float* offset, const uint32_t* w,
                              const int32_t* thr, const uint32_t* flip,
                              int32_t* sums, uint32_t* bits, hipStream_t s);

// Binary GEMM for a handful of rows (M <= 16; bnn_bgemm uses it for M <= 2):
// a wave per two output columns, its lanes along K, a block per 32 columns.
hipError_t launch_bgemv_valu(int64_t M, int64_t N, int64_t K,
                             const uint32_t* A, const uint32_t* B,
                             const int32_t* thr, const uint32_t* flip,
                             int32_t* sums, uint32_t* bits, hipStream_t s);

// Real-valued input conv with packed +-1 weights (fp32 sums).
hipError_t launch_fconv_binw(const ConvGeom& g, const float* in,
                             const uint32_t* w, const int32_t* thr,
                             const uint32_t* flip, float* sums,
                             uint32_t* bits, hipStream_t s);

// The real-valued first layer and the binary 3x3 conv after it in one launch
// (fconv_bconv.hip), the first layer's output bits kept in LDS.  g0: the
// first layer (3x3, C <= 4, 64 or 128 filters, no pooling); g1: the second
// (3x3 over g0's output, 64 or 128 filters, optional 2x2 pooling).  Writes
// the second layer's packed bits; both thr must be non-null.
bool fconv_bconv_supported(const ConvGeom& g0, const ConvGeom& g1);
// w1prep: the second layer's weights prepared by launch_prepare_weights, or
// null (packed w1).
hipError_t launch_fconv_bconv(const ConvGeom& g0, const ConvGeom& g1, const float* in,
                              const uint32_t* w0, const int32_t* thr0,
                              const uint32_t* flip0, const uint32_t* w1,
                              const void* w1prep, const int32_t* thr1,
                              const uint32_t* flip1, uint32_t* bits, hipStream_t s);
// The same kernel with the first layer a binary conv over the input
// thresholded per channel (bnn_bconv2d_input, mode THRESHOLD, 3 channels):
// input thresholding, the first binary conv and the second in one launch.
// g0 is the first binary conv (C = 3).
bool input_bconv_bconv_supported(int mode, const ConvGeom& g0, const ConvGeom& g1);
hipError_t launch_input_bconv_bconv(const ConvGeom& g0, const ConvGeom& g1, const float* in,
                                    const float* offset, const uint32_t* w0,
                                    const int32_t* thr0, const uint32_t* flip0,
                                    const uint32_t* w1, const void* w1prep,
                                    const int32_t* thr1, const uint32_t* flip1,
                                    uint32_t* bits, hipStream_t s);

// Two consecutive binary 3x3 convs in one launch (bconv_bconv.hip), the first
// conv's output bits kept in LDS: 16-pixel-wide images, pad 1 in both, the
// first with 64, 128 or 256 input channels, 256 filters and no pooling, the
// second with 256 filters and optional 2x2 pooling.  Packed weights; writes
// the second conv's packed bits; both thr must be non-null.
bool bconv_bconv_supported(const ConvGeom& g0, const ConvGeom& g1);
hipError_t launch_bconv_bconv(const ConvGeom& g0, const ConvGeom& g1, const uint32_t* in,
                              const uint32_t* w0, const int32_t* thr0, const uint32_t* flip0,
                              const uint32_t* w1, const int32_t* thr1, const uint32_t* flip1,
                              uint32_t* bits, hipStream_t s);

// One binary 3x3 conv with pad 1 on 8 x 8 maps, C = 64..512 (a power of
// two), F a multiple of 128, bits only (bconv_bconv.hip): a block per image
// and 128 filters, the image staged once in LDS as fp4 operands.
bool bconv_img8_supported(const ConvGeom& g);
hipError_t launch_bconv_img8(const ConvGeom& g, const uint32_t* in, const uint32_t* w,
                             const int32_t* thr, const uint32_t* flip, uint32_t* bits,
                             hipStream_t s);

// Binary FC layer / GEMM with K >= 1024 bits (bfc_gemm.hip): a workgroup per
// 32 x 32 output tile (the last one partial when N is not a multiple of 32),
// K split over its 8 waves, both operands staged per wave through LDS with
// whole-line loads.  sums [M][N] and/or bits [M][ceil(N / 32)]; thr non-null
// when bits is.
bool bfc_gemm_supported(int64_t M, int64_t N, int64_t K);
hipError_t launch_bfc_gemm(int64_t M, int64_t N, int64_t K, const uint32_t* A,
                           const uint32_t* B, const int32_t* thr, const uint32_t* flip,
                           int32_t* sums, uint32_t* bits, hipStream_t s);

// Two consecutive binary FC layers, the second with N1 <= 32 outputs, in one
// launch of the FC kernel (bfc_gemm.hip): a workgroup per 32 x 32 tile of the
// first layer (K0 >= 1024, N0 a multiple of 32, at most 512 tiles, at most
// kTailMaxRows rows), each adding the second layer's partial sums over its
// 32 inputs to accumulators in `accum` (kTailAccumBytes, zero on entry and
// left zero) with atomic adds; the add that completes an output writes it:
// int32 sums [M][N1] (sums non-null) or bits [M][1] (thr1 non-null).
// Packed weights; w1 [N1][N0 / 32].
constexpr int kTailMaxRows = 512;
constexpr size_t kTailAccumBytes = size_t{kTailMaxRows} * 32 * 4 + size_t{kTailMaxRows} * 8;
bool bfc_tail_supported(int64_t M, int64_t K0, int64_t N0, int64_t N1);
hipError_t launch_bfc_tail(int64_t M, int64_t K0, int64_t N0, int64_t N1, const uint32_t* A,
                           const uint32_t* w0, const int32_t* thr0, const uint32_t* flip0,
                           const uint32_t* w1, const int32_t* thr1, const uint32_t* flip1,
                           int32_t* sums, uint32_t* bits, void* accum, hipStream_t s);

// Two consecutive binary FC layers in one launch (bfc_pair.hip), the first
// layer's output bits kept in LDS: K0 = 512 or 1024 input bits,
// N0 = 256, 512 or 1024 first-layer outputs (thresholded, with flips), N1 <= 32
// second-layer outputs as int32 sums [M][N1] (sums non-null) or bits [M][1]
// (thr1 non-null).  Packed weights.
bool bfc_pair_supported(int64_t M, int64_t K0, int64_t N0, int64_t N1);
hipError_t launch_bfc_pair(int64_t M, int64_t K0, int64_t N0, int64_t N1, const uint32_t* A,
                           const uint32_t* w0, const int32_t* thr0, const uint32_t* flip0,
                           const uint32_t* w1, const int32_t* thr1, const uint32_t* flip1,
                           int32_t* sums, uint32_t* bits, hipStream_t s);

// A run of consecutive binary FC layers in one launch (bfc_chain.hip): every
// block takes R rows through all of them with the intermediate bits in LDS.
// Layer i has K_i input bits and N_i outputs; K_{i+1} = N_i; every layer but
// the last needs thr (its bits feed the next one); the last writes either
// packed bits [M][ceil(N/32)] (out_bits, with thr) or int32 sums [M][N]
// (out_sums).  Supported while every layer input is at most 1024 words.
// Weights must be 16-byte aligned.
constexpr int kFcChainMax = 4;
struct FcChainLayer {
  const uint32_t* w;     // [N][ceil(K/32)]
  const int32_t* thr;    // [N] or null
  const uint32_t* flip;  // [ceil(N/32)] or null
  int32_t K, N;
};
bool bfc_chain_supported(const FcChainLayer* layers, int n);
hipError_t launch_bfc_chain(const FcChainLayer* layers, int n, int64_t M,
                            const uint32_t* in, uint32_t* out_bits,
                            int32_t* out_sums, hipStream_t s);

}  // namespace bnn
