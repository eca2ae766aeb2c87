/*
 * bnn.h -- C ABI of libbnn.so: binarized convolutional / fully-connected
 * inference on AMD Instinct MI355X (gfx950).
 *
 * Method: Khan, Huttunen, Boutellier, "Binarized Convolutional Neural
 * Networks for Efficient Inference on GPUs", EUSIPCO 2018.  Weights and
 * activations are +-1 values packed 32 to a 32-bit word (Sec. II-D, Eq. 2);
 * a dot product of two packed vectors of W valid bits is
 * W - 2 * popcount(a XOR b) (Sec. III-A, Eq. 4).
 *
 * ---------------------------------------------------------------- layout --
 * Packed word (Eq. 2 with B = 32): value i (0-based) of a group of 32 goes to
 * bit (31 - i); bit 1 means +1, bit 0 means -1.  A vector of D values takes
 * ceil(D / 32) words; the unused low bits of a short last word are "tail"
 * bits.  Outputs of this library always hold 0 in tail bits; inputs may hold
 * anything there (every kernel masks them).
 *
 * Activations are NHWC with channels packed: u32 [N][H][W][Cw], Cw =
 * ceil(C / 32).  Conv weights are u32 [F][KH][KW][Cw] (filter f's KHxKWxC
 * window in the same packing).  FC operands are u32 [rows][ceil(K / 32)].
 * Output bits use the same packing over filters / output columns, and the
 * flip vector uses it too: flip bit for channel f is bit (31 - f % 32) of
 * word f / 32.
 *
 * ------------------------------------------------------------- semantics --
 * Binary conv (Eq. 3, a cross-correlation): for output pixel (n, i, j) and
 * filter f,
 *     S = sum_{kh, kw, c} w[f,kh,kw,c] * x[n, i*s + kh - p, j*s + kw - p, c]
 * over +-1 values, where a tap outside the image reads -1 (bit 0).  Padded
 * taps count: S has the parity of K = KH * KW * C and |S| <= K.
 * Threshold (folded BatchNorm + sign; not in the paper): output bit =
 * (S >= thr[f]) XOR flip[f].  Pooling: 2x2, stride 2, applied to the bits
 * after the threshold as a bitwise OR (= max over +-1), floor on odd sizes.
 *
 * ------------------------------------------------------ memory and errors --
 * Every pointer argument is a DEVICE pointer owned by the caller, except the
 * bnn_conv_desc / bnn_layer structs and the size outputs, which are host
 * memory read or written before the call returns.  The library allocates
 * nothing.  Its only state is per thread: the last error string and the
 * kernel-selection options of bnn_set_options (which never change a result).
 * It reads no environment variables.  Calls only
 * enqueue kernels on `stream` and return without synchronising; results are
 * ready when the stream reaches that point.  Device buffers passed to one
 * call must not overlap unless stated.
 *
 * Every call validates its arguments on the host first and returns a status
 * other than BNN_OK without launching anything when they are invalid;
 * bnn_last_error() then describes the problem.  A failed kernel launch
 * returns BNN_ERR_HIP.  No C++ exception crosses this interface.
 */
#ifndef BNN_H
#define BNN_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define BNN_ABI_VERSION 8

typedef enum bnn_status {
  BNN_OK = 0,
  BNN_ERR_NULL = 1,        /* a required pointer is NULL                    */
  BNN_ERR_SHAPE = 2,       /* a size is out of range or sizes disagree      */
  BNN_ERR_ALIGN = 3,       /* a pointer is not 16-byte aligned              */
  BNN_ERR_UNSUPPORTED = 4, /* valid in principle, not implemented (stride)  */
  BNN_ERR_HIP = 5,         /* the HIP runtime reported an error             */
  BNN_ERR_WORKSPACE = 6    /* workspace smaller than required               */
} bnn_status;

/* Text describing the last non-OK status returned on this thread ("" if
 * none).  The pointer stays valid until the next call on the same thread. */
const char* bnn_last_error(void);

/* BNN_ABI_VERSION of the loaded library. */
int32_t bnn_abi_version(void);

/*
 * Kernel selection.  Not part of the paper's method: every setting computes
 * the same bits and sums; they choose among kernels that do so, for
 * ablations (the vector-ALU XOR-popcount kernels of Eq. 4 against the
 * matrix-core ones) and for tests that must reach each kernel variant.
 * Options are per thread: bnn_set_options affects later calls made on the
 * calling thread only, and a thread that never calls it uses the defaults.
 */
typedef enum bnn_algo {
  BNN_ALGO_AUTO = 0, /* matrix cores wherever the shape allows (default)    */
  BNN_ALGO_VALU = 1  /* XOR + popcount on the vector ALU for every layer    */
} bnn_algo;

typedef struct bnn_options {
  int32_t algo;            /* bnn_algo                                       */
  int32_t fuse_input;      /* bnn_forward: an input layer and the conv(s)    */
                           /* after it as one kernel (1, default) or apart  */
  int32_t fuse_first;      /* bnn_forward: FCONV_BINW and the 3x3 conv after */
                           /* it as one kernel (1, default) or two (0)       */
  int32_t fc_chain;        /* bnn_forward: runs of small FC layers as one    */
                           /* kernel (1, default) or one launch each (0)     */
  int32_t conv1x1;         /* the short-window 1x1 kernel where it applies   */
                           /* (1, default) or the general one (0)            */
  int32_t xcd_order;       /* matrix-core conv workgroups in the XCD order   */
                           /* (1, default), on a 2-D grid (0), or in the XCD */
                           /* order with the filter tiles split over XCD     */
                           /* groups when that cuts the bytes the L2s move   */
                           /* (2)                                            */
  int32_t gemv_max_rows;   /* FC layers of at most this many rows use the    */
                           /* vector-ALU GEMV; 0..16, default 1              */
  int32_t lds_weights;     /* matrix-core conv weights staged through LDS:   */
                           /* -1 where the heuristic picks it (default), 0   */
                           /* never, 1 wherever no K split is used (with     */
                           /* 2-word chunks)                                 */
  int32_t late_thresholds; /* thresholds staged after the main loop: -1      */
                           /* heuristic (default), 0 at kernel start where   */
                           /* the variant allows, 1 after the loop           */
  int32_t fuse_pair;       /* bnn_forward: two 3x3 BCONVs that fit           */
                           /* bnn_bconv_bconv2d, or two FC layers that fit   */
                           /* bnn_bfc_pair, as one kernel (1, default) or    */
                           /* two (0)                                        */
} bnn_options;

/* The default options. */
void bnn_default_options(bnn_options* opt);

/* Set (bnn_set_options) or read (bnn_get_options) the calling thread's
 * options.  Values outside the ranges above give BNN_ERR_SHAPE and leave the
 * options unchanged; a NULL pointer gives BNN_ERR_NULL. */
bnn_status bnn_set_options(const bnn_options* opt);
bnn_status bnn_get_options(bnn_options* opt);

/*
 * Sign to bits (Eq. 1 and Eq. 2; input thresholding of Sec. II-C).
 *   out[r][j] bit (31 - i) = ((x[r][32 j + i] + offset[32 j + i]) > 0)
 * for 32 j + i < D, computed in fp32; tail bits are written 0.  x == 0 (after
 * the offset) gives bit 0 (-1), as does NaN.
 *   x      [rows][D] fp32, device.
 *   offset [D] fp32 or NULL (NULL: no offset).  Thresholding an RGB image by
 *          T in R^{1x1xC} passes rows = N*H*W, D = C, offset = T.
 *   out    [rows][ceil(D / 32)] u32, device.
 * rows >= 0 and D >= 1 (rows == 0 launches nothing).  Errors: BNN_ERR_NULL,
 * BNN_ERR_SHAPE.
 */
bnn_status bnn_pack_bits(const float* x, const float* offset, int64_t rows,
                         int64_t D, uint32_t* out, hipStream_t stream);

/* Shape of one convolution layer (Eq. 3).  stride must be 1 (other strides
 * return BNN_ERR_UNSUPPORTED); 0 <= pad, KH, KW >= 1 and the output
 * Ho = H + 2 pad - KH + 1, Wo = W + 2 pad - KW + 1 must be >= 1.  pool is 0
 * (none) or 2 (2x2 / stride 2; needs Ho, Wo >= 2). */
typedef struct bnn_conv_desc {
  int32_t N, H, W, C; /* input batch, height, width, channels (bits)       */
  int32_t F;          /* filters = output channels                          */
  int32_t KH, KW;     /* kernel height, width                               */
  int32_t stride;     /* must be 1                                          */
  int32_t pad;        /* symmetric padding (pad value -1 / 0.0)            */
  int32_t pool;       /* 0 or 2                                             */
} bnn_conv_desc;

/* Output sizes of a conv: Ho x Wo before pooling, Hp x Wp after (Hp = Ho/2,
 * Wp = Wo/2 when pool == 2, else Ho, Wo).  Validates like bnn_bconv2d. */
bnn_status bnn_conv_output_dims(const bnn_conv_desc* d, int32_t* Ho,
                                int32_t* Wo, int32_t* Hp, int32_t* Wp);

/*
 * Binary convolution with the fused threshold / flip / OR-pool epilogue
 * (Eq. 3 with Eq. 4 for the window dot products; Sec. III-A).
 *   in        [N][H][W][Cw] u32 packed activations.
 *   w         [F][KH][KW][Cw] u32 packed weights.
 *   thr       [F] int32 thresholds, or NULL when out_bits is NULL.
 *   flip      [ceil(F / 32)] u32 flip bits, or NULL for all-zero.
 *   out_sums  [N][Ho][Wo][F] int32 window sums S before the threshold and
 *             before pooling, or NULL.
 *   out_bits  [N][Hp][Wp][ceil(F / 32)] u32 thresholded (and pooled) bits,
 *             or NULL.  Needs thr.
 * At least one of out_sums / out_bits must be non-NULL.  in, w, out_sums and
 * out_bits must be 16-byte aligned.  Errors: BNN_ERR_NULL, BNN_ERR_SHAPE,
 * BNN_ERR_ALIGN, BNN_ERR_UNSUPPORTED (stride != 1), BNN_ERR_HIP.
 */
bnn_status bnn_bconv2d(const bnn_conv_desc* d, const uint32_t* in,
                       const uint32_t* w, const int32_t* thr,
                       const uint32_t* flip, int32_t* out_sums,
                       uint32_t* out_bits, hipStream_t stream);

/*
 * Prepared conv weights: the packed weights of a conv layer in the operand
 * form of the matrix-core kernel, made once per network (like a filter
 * transform) so that no kernel spends vector-ALU time expanding weight words
 * while it runs.  The form is private to this library (16-byte entries of
 * four fp4 registers per weight word, zero past C, then per-filter int32
 * offsets); only its size is part of the interface.  Results with prepared
 * weights are those of bnn_bconv2d, bit for bit (Eq. 3 and Eq. 4 with the
 * same epilogue).
 *   bnn_prepared_weights_size: bytes of the prepared form of F filters of
 *     KH x KW x C bits; BNN_ERR_SHAPE when beyond 2 GiB.
 *   bnn_prepare_weights: w [F][KH][KW][ceil(C/32)] u32 -> out (device,
 *     16-byte aligned, that many bytes).  Enqueued on `stream`.
 *   bnn_bconv2d_prepared: bnn_bconv2d with wprep = the prepared form of w.
 *     The packed w is still required: the vector-ALU ablation and the
 *     short-window 1x1 kernel read it.  wprep 16-byte aligned.
 * Errors: BNN_ERR_NULL, BNN_ERR_SHAPE, BNN_ERR_ALIGN, and as for bnn_bconv2d.
 */
bnn_status bnn_prepared_weights_size(int32_t F, int32_t KH, int32_t KW, int32_t C,
                                     size_t* bytes);
bnn_status bnn_prepare_weights(int32_t F, int32_t KH, int32_t KW, int32_t C,
                               const uint32_t* w, void* out, hipStream_t stream);
bnn_status bnn_bconv2d_prepared(const bnn_conv_desc* d, const uint32_t* in,
                                const uint32_t* w, const void* wprep,
                                const int32_t* thr, const uint32_t* flip,
                                int32_t* out_sums, uint32_t* out_bits,
                                hipStream_t stream);

/*
 * Real-valued first layer with binary weights ("no input binarization",
 * Table III; the BCNN row of Table I): Eq. 3 with an fp32 image and +-1
 * weights, pad value 0.0, then the same threshold / flip / OR-pool epilogue
 * as bnn_bconv2d.
 *   in        [N][H][W][C] fp32.
 *   w         [F][KH][KW][Cw] u32 packed weights.
 *   out_sums  [N][Ho][Wo][F] fp32 or NULL; out_bits as for bnn_bconv2d.
 * Precision.  Every product x * (+-1) is exact: the matrix-core kernels
 * split each x exactly into three bf16 parts (exact for finite |x| >= 2^-103
 * and x = 0; a smaller part may be flushed, losing less than 2^-126), the
 * vector kernels add +-x directly.  The products are summed in fp32 in an
 * unspecified order, so for finite sums the result S' satisfies
 *     |S' - S| <= n * (2^-23 * sum |x| + 2^-126),  n = 3 * KH * KW * C,
 * the sum of |x| taken over the window.  The output bit is S' >= thr,
 * compared exactly (no rounding of thr), so it equals the exact bit wherever
 * |S - thr| exceeds that bound.  When every input is a multiple of 2^-16 and
 * each window's sum of |x| is below 2^8 (e.g. |x| < 8 with at most 32 values
 * per window), every partial sum is exact in fp32, S' = S in any order and
 * the bits are unique.  Non-finite inputs give unspecified sums and bits in
 * the windows that hold them.
 * Errors as for bnn_bconv2d.
 */
bnn_status bnn_fconv2d_binw(const bnn_conv_desc* d, const float* in,
                            const uint32_t* w, const int32_t* thr,
                            const uint32_t* flip, float* out_sums,
                            uint32_t* out_bits, hipStream_t stream);

/*
 * Input binarizations of an fp32 NHWC image (Sec. II-C; Table III), each
 * giving C <= 32 bits per pixel:
 *   BNN_INPUT_THRESHOLD  C = Cin channels, bit = (x[c] + offset[c]) > 0
 *                        (RGB thresholding; offset NULL means 0).
 *   BNN_INPUT_GRAY       C = 1, bit = (gray + offset[0]) > 0 (grayscale
 *                        thresholding; offset NULL means 0).  Cin = 3.
 *   BNN_INPUT_LBP        C = 3 local-binary-pattern channels: on the gray
 *                        image, the 8 neighbours at radius 1 are numbered
 *                        clockwise from the top-left and channels 0, 1, 2
 *                        take neighbours 0, 3, 6, i.e. offsets (-1,-1),
 *                        (0,+1), (+1,-1); a bit is 1 when that neighbour's
 *                        gray value exceeds the centre's, and 0 for a
 *                        neighbour outside the image.  Cin = 3.
 * gray = (0.299 R + 0.587 G) + 0.114 B in fp32, each product rounded on its
 * own (the BT.601 luma; the paper names no conversion).  All comparisons
 * are in fp32.
 */
typedef enum bnn_input_mode {
  BNN_INPUT_THRESHOLD = 0,
  BNN_INPUT_GRAY = 1,
  BNN_INPUT_LBP = 2
} bnn_input_mode;

/*
 * Binarize an image: out[n][i][j] is the pixel's C-bit code, channel 0 at
 * bit 31 (Eq. 2 packing of the C channels, tail bits 0).
 *   x    [N][H][W][Cin] fp32.  offset as above.
 *   out  [N][H][W] u32 (one word per pixel).
 * mode THRESHOLD needs Cin <= 32 (bnn_pack_bits covers any Cin); GRAY and
 * LBP need Cin == 3.  x and out 16-byte aligned.  Errors: BNN_ERR_NULL,
 * BNN_ERR_SHAPE, BNN_ERR_ALIGN, BNN_ERR_HIP.
 */
bnn_status bnn_binarize_input(int32_t mode, const float* x, const float* offset,
                              int32_t N, int32_t H, int32_t W, int32_t Cin,
                              uint32_t* out, hipStream_t stream);

/*
 * Binary convolution over an image binarized on the fly by `mode`, with pad
 * value -1 and the bnn_bconv2d epilogue.  The result equals
 * bnn_binarize_input (or bnn_pack_bits) followed by bnn_bconv2d, bit for bit.
 * Each output pixel's whole binarized window is packed into
 * P = KH*KW*C bits (the patch packing of Algorithm 1 with B = P), in
 * ceil(P / 32) words, so every dot product takes ceil(P / 32) XOR + popcounts
 * (one for a 3x3 conv over 3 channels, P = 27).
 *   d         the conv; d->C is the binarized channel count (Cin for
 *             THRESHOLD, 1 for GRAY, 3 for LBP).
 *   x         [N][H][W][Cin] fp32 image (Cin = 3 for GRAY and LBP).
 *   offset    as for bnn_binarize_input.
 *   w         [F][KH][KW][1] u32 packed weights.
 *   thr, flip, out_sums, out_bits: as for bnn_bconv2d.
 * Needs C <= 32, KH <= 32, KW <= 32 and P <= 128 (else
 * BNN_ERR_UNSUPPORTED).  Alignment and other errors as for bnn_bconv2d.
 */
bnn_status bnn_bconv2d_input(const bnn_conv_desc* d, int32_t mode,
                             const float* x, const float* offset,
                             const uint32_t* w, const int32_t* thr,
                             const uint32_t* flip, int32_t* out_sums,
                             uint32_t* out_bits, hipStream_t stream);

/*
 * The real-valued first layer (bnn_fconv2d_binw) and a binary 3x3 conv over
 * its output bits (bnn_bconv2d) in one launch, the first layer's bits never
 * leaving the chip (the BCNN of Table I, first two layers).  The result
 * equals bnn_fconv2d_binw followed by bnn_bconv2d, bit for bit, whenever the
 * first layer's sums are exact, and under the same precision contract
 * otherwise (see bnn_fconv2d_binw).
 *   d0        the first layer: 3x3, C <= 4, F = 64 or 128, no pooling,
 *             pad 0 or 1.
 *   d1        the second: N, H, W equal to d0's N and output Ho, Wo; 3x3,
 *             C = d0's F, F = 64 or 128, pad 0 or 1, pool 0 or 2.
 *   x         [N][H][W][C] fp32 image.
 *   w0, thr0, flip0   the first layer's packed weights [F0][3][3][1], int32
 *             thresholds [F0] and flip words [F0 / 32] (flip0 may be NULL).
 *   w1, thr1, flip1   the second layer's [F1][3][3][F0 / 32], [F1],
 *             [F1 / 32] (flip1 may be NULL).
 *   w1prep    bnn_prepare_weights of w1 (then the second layer reads its
 *             weights in operand form), or NULL.
 *   out_bits  [N][Hp][Wp][F1 / 32] u32, the second layer's bits.
 * Shapes outside the above give BNN_ERR_UNSUPPORTED.  x, w0, w1, w1prep and
 * out_bits 16-byte aligned.  Errors: BNN_ERR_NULL, BNN_ERR_SHAPE, BNN_ERR_ALIGN,
 * BNN_ERR_UNSUPPORTED, BNN_ERR_HIP.
 */
bnn_status bnn_fconv_bconv2d(const bnn_conv_desc* d0, const bnn_conv_desc* d1,
                             const float* x, const uint32_t* w0,
                             const int32_t* thr0, const uint32_t* flip0,
                             const uint32_t* w1, const void* w1prep,
                             const int32_t* thr1, const uint32_t* flip1,
                             uint32_t* out_bits, hipStream_t stream);

/*
 * Input thresholding (Sec. II-C), a binary 3x3 conv over the thresholded
 * image and a binary 3x3 conv over its output bits in one launch, the first
 * conv's bits never leaving the chip (the vehicle classifier's first layers,
 * Table III thresholded RGB input).  The result equals bnn_bconv2d_input
 * followed by bnn_bconv2d, bit for bit.
 *   d0        the first conv: C = 3 (the image's channels), 3x3, F = 64 or
 *             128, no pooling, pad 0 or 1 (pad value -1).
 *   d1        the second: N, H, W equal to d0's N and output Ho, Wo; 3x3,
 *             C = d0's F, F = 64 or 128, pad 0 or 1, pool 0 or 2.
 *   mode      BNN_INPUT_THRESHOLD (other modes: BNN_ERR_UNSUPPORTED).
 *   x, offset as for bnn_bconv2d_input ([N][H][W][3] fp32, offsets [3] or
 *             NULL).
 *   w0, thr0, flip0, w1, w1prep, thr1, flip1, out_bits: as for
 *             bnn_fconv_bconv2d.
 * Alignment and errors as for bnn_fconv_bconv2d.
 */
bnn_status bnn_input_bconv_bconv2d(const bnn_conv_desc* d0, const bnn_conv_desc* d1,
                                  int32_t mode, const float* x, const float* offset,
                                  const uint32_t* w0, const int32_t* thr0,
                                  const uint32_t* flip0, const uint32_t* w1,
                                  const void* w1prep, const int32_t* thr1,
                                  const uint32_t* flip1, uint32_t* out_bits,
                                  hipStream_t stream);

/*
 * Two binary 3x3 convs in one launch (Eq. 3 and Eq. 4 with the threshold,
 * flip and pool epilogue of bnn_bconv2d, twice; a conv -> conv step of
 * Table II's layer order), the first conv's output bits never leaving the
 * chip.  The result equals bnn_bconv2d(d0) followed by bnn_bconv2d(d1), bit
 * for bit.
 *   d0        the first conv: W = 16, pad 1, 3x3, C = 64, 128 or 256,
 *             F = 256, no pooling.
 *   d1        the second: N, H, W equal to d0's N and output Ho, Wo; 3x3,
 *             pad 1, C = F = 256, pool 0 or 2.
 *   x         [N][H][16][C / 32] u32, the first conv's packed input bits.
 *   w0, thr0, flip0   the first conv's packed weights [256][3][3][C / 32],
 *             int32 thresholds [256] and flip words [8] (flip0 may be NULL).
 *   w1, thr1, flip1   the second conv's [256][3][3][8], [256], [8] (flip1
 *             may be NULL).
 *   out_bits  [N][Hp][Wp][8] u32, the second conv's bits.
 * Shapes outside the above give BNN_ERR_UNSUPPORTED.  x, w0, w1 and
 * out_bits 16-byte aligned.  Errors: BNN_ERR_NULL, BNN_ERR_SHAPE,
 * BNN_ERR_ALIGN, BNN_ERR_UNSUPPORTED, BNN_ERR_HIP.
 */
bnn_status bnn_bconv_bconv2d(const bnn_conv_desc* d0, const bnn_conv_desc* d1,
                             const uint32_t* x, const uint32_t* w0,
                             const int32_t* thr0, const uint32_t* flip0,
                             const uint32_t* w1, const int32_t* thr1,
                             const uint32_t* flip1, uint32_t* out_bits,
                             hipStream_t stream);

/*
 * Two binary FC layers in one launch (Sec. III-B, Eq. 4 twice), the first
 * layer's output bits never leaving the chip: out = layer 1 (layer 0 (A)),
 * layer 0 with its threshold and flip as in bnn_bgemm, layer 1 to int32 sums
 * (out_sums, e.g. the logits) or to bits (out_bits, with thr1).  The result
 * equals two bnn_bgemm calls, bit for bit.
 *   M         rows (>= 1, at most 2^26).
 *   K0        layer 0's input bits: 512 or 1024.
 *   N0        layer 0's outputs = layer 1's input bits: 256, 512 or 1024.
 *   N1        layer 1's outputs: 1..32.
 *   A         [M][K0 / 32] u32 packed rows.
 *   w0, thr0, flip0   layer 0's packed weights [N0][K0 / 32], int32
 *             thresholds [N0], flip words [N0 / 32] (flip0 may be NULL).
 *   w1, thr1, flip1   layer 1's [N1][N0 / 32], [N1], [1]; thr1 and flip1
 *             are read only for out_bits (flip1 may be NULL).
 *   out_sums  [M][N1] int32, or NULL;  out_bits  [M][1] u32 (tail bits 0),
 *             or NULL: exactly one of the two.
 * Shapes outside the above give BNN_ERR_UNSUPPORTED.  A, w0, w1 and the
 * output 16-byte aligned.  Errors: BNN_ERR_NULL, BNN_ERR_SHAPE (also both
 * outputs given), BNN_ERR_ALIGN, BNN_ERR_UNSUPPORTED, BNN_ERR_HIP.
 */
bnn_status bnn_bfc_pair(int64_t M, int64_t K0, int64_t N0, int64_t N1,
                        const uint32_t* A, const uint32_t* w0,
                        const int32_t* thr0, const uint32_t* flip0,
                        const uint32_t* w1, const int32_t* thr1,
                        const uint32_t* flip1, int32_t* out_sums,
                        uint32_t* out_bits, hipStream_t stream);

/*
 * Accumulators of the FC tail kernel (bnn_bfc_tail, and bnn_forward's FC
 * tails at the head of its workspace): 512 rows x 32 outputs x 4 bytes plus
 * 512 x 8 bytes, 68 KiB.  They must be zero before the first call that uses
 * them; every call that completes leaves them zero.
 */
#define BNN_FORWARD_SYNC_BYTES ((size_t)69632)

/*
 * Two binary FC layers in one launch (Sec. III-B, Eq. 4 twice), the second
 * with at most 32 outputs (the classifier tail), spread over the first
 * layer's output tiles: a workgroup per 32 rows x 32 outputs of layer 0
 * thresholds them (threshold and flip as in bnn_bgemm) and adds layer 1's
 * partial sums over those 32 inputs into atomic accumulators in `accum`;
 * the add that completes an output writes it as an int32 sum (out_sums,
 * e.g. the logits) or, with thr1, as a bit (out_bits), and zeroes its
 * accumulator.  The result equals two bnn_bgemm calls, bit for bit.
 *   M         rows, 1..512.
 *   K0        layer 0's input bits: at least 1024.
 *   N0        layer 0's outputs = layer 1's input bits: a multiple of 32,
 *             with ceil(M / 32) * N0 / 32 <= 512.
 *   N1        layer 1's outputs: 1..32.
 *   A, w0, thr0, flip0, w1, thr1, flip1, out_sums, out_bits   as for
 *             bnn_bfc_pair.
 *   accum     device, BNN_FORWARD_SYNC_BYTES, 16-byte aligned, zero on
 *             entry and left zero.  Calls that share it must not overlap in
 *             time (calls on one stream are ordered).
 * Shapes outside the above give BNN_ERR_UNSUPPORTED.  A, w0, w1, the output
 * and accum 16-byte aligned.  Errors: BNN_ERR_NULL, BNN_ERR_SHAPE (also both
 * outputs given), BNN_ERR_ALIGN, BNN_ERR_UNSUPPORTED, BNN_ERR_HIP.
 */
bnn_status bnn_bfc_tail(int64_t M, int64_t K0, int64_t N0, int64_t N1,
                        const uint32_t* A, const uint32_t* w0,
                        const int32_t* thr0, const uint32_t* flip0,
                        const uint32_t* w1, const int32_t* thr1,
                        const uint32_t* flip1, int32_t* out_sums,
                        uint32_t* out_bits, void* accum, hipStream_t stream);

/*
 * Binary fully-connected layer / GEMM (Sec. III-B, Eq. 4):
 *   S[m][n] = K - 2 * sum_j popcount(A[m][j] XOR B[n][j])   (valid bits only)
 *   A         [M][Kw] u32, Kw = ceil(K / 32): M packed input vectors.
 *   B         [N][Kw] u32: one packed weight row per output.
 *   thr, flip [N] int32 / [ceil(N / 32)] u32 as for bnn_bconv2d.
 *   out_sums  [M][N] int32 or NULL.
 *   out_bits  [M][ceil(N / 32)] u32 or NULL (needs thr).
 * M, N, K >= 1.  Alignment and errors as for bnn_bconv2d.
 */
bnn_status bnn_bgemm(int64_t M, int64_t N, int64_t K, const uint32_t* A,
                     const uint32_t* B, const int32_t* thr,
                     const uint32_t* flip, int32_t* out_sums,
                     uint32_t* out_bits, hipStream_t stream);

/* ------------------------------------------------------------ layer chain */
typedef enum bnn_layer_kind {
  BNN_LAYER_INPUT_THRESHOLD = 1, /* bnn_pack_bits with per-channel offset  */
  BNN_LAYER_FCONV_BINW = 2,      /* bnn_fconv2d_binw (fp32 input)           */
  BNN_LAYER_BCONV = 3,           /* bnn_bconv2d, bits out                   */
  BNN_LAYER_BFC = 4,             /* bnn_bgemm, bits out                     */
  BNN_LAYER_BFC_LOGITS = 5,      /* bnn_bgemm, int32 sums out (last layer)  */
  BNN_LAYER_INPUT_GRAY = 6,      /* bnn_binarize_input, BNN_INPUT_GRAY      */
  BNN_LAYER_INPUT_LBP = 7        /* bnn_binarize_input, BNN_INPUT_LBP       */
} bnn_layer_kind;

/* One layer of a chain.  Fields a kind does not use are ignored.  Device
 * pointers: w, thr, flip, offset. */
typedef struct bnn_layer {
  int32_t kind;              /* bnn_layer_kind                               */
  int32_t C;                 /* conv / input layers: input channels          */
  int32_t F, KH, KW;         /* conv: filters, kernel size                   */
  int32_t stride, pad, pool; /* conv: as in bnn_conv_desc                    */
  int32_t K, N;              /* FC: input bits, outputs                      */
  const uint32_t* w;         /* conv [F][KH][KW][Cw], 16-byte aligned;       */
                             /* FC [N][ceil(K/32)]                           */
  const int32_t* thr;        /* [F] or [N]                                   */
  const uint32_t* flip;      /* packed flip bits or NULL                     */
  const float* offset;       /* INPUT_THRESHOLD: [C] offsets T; INPUT_GRAY:  */
                             /* [1] offset T; or NULL                        */
  const void* wprep;         /* BCONV: bnn_prepare_weights of w, or NULL     */
                             /* (16-byte aligned); other kinds ignore it     */
} bnn_layer;

/*
 * Workspace bytes bnn_forward needs for `batch` images of H x W x C fp32:
 * BNN_FORWARD_SYNC_BYTES of accumulators and two ping-pong buffers of
 * packed activations (256-byte aligned).  Also
 * validates the chain: the first layer is an input layer (INPUT_THRESHOLD,
 * INPUT_GRAY, INPUT_LBP) or FCONV_BINW, the last is BFC_LOGITS, shapes agree
 * from layer to layer, and an FC layer that
 * follows a conv reads its NHWC bits flattened in (h, w, c) order, which needs
 * the channel count to be a multiple of 32 (or a 1x1 map).
 */
bnn_status bnn_forward_workspace_size(const bnn_layer* layers,
                                      int32_t n_layers, int32_t batch,
                                      int32_t H, int32_t W, int32_t C,
                                      size_t* bytes);

/*
 * Run the chain on input [batch][H][W][C] fp32 and write int32 logits
 * [batch][N_last] (Table I/II: conv, pool, ..., FC layers).  One kernel per
 * layer on `stream`, with four exceptions:
 *  - an INPUT_THRESHOLD layer of 3 channels followed by two 3x3 BCONVs of
 *    64 or 128 filters (the first without pooling) runs as one kernel
 *    (bnn_input_bconv_bconv2d); otherwise an input layer followed by a BCONV
 *    whose window fits bnn_bconv2d_input runs as that one kernel (option
 *    fuse_input = 0 keeps them all apart);
 *  - an FCONV_BINW layer (3x3, at most 4 channels, 64 or 128 filters, no
 *    pooling) followed by a 3x3 BCONV of 64 or 128 filters runs as one
 *    kernel that keeps the first layer's bits in LDS (bnn_fconv_bconv2d;
 *    option fuse_first = 0 keeps them apart);
 *  - two consecutive BCONVs that fit bnn_bconv_bconv2d (3x3, pad 1, 256
 *    filters each, on a 16-pixel-wide map) run as that one kernel (option
 *    fuse_pair = 0 keeps them apart);
 *  - two consecutive FC layers not part of a chained run, the second with
 *    at most 32 outputs (Sec. III-B, Eq. 4: the classifier tail), run as
 *    one kernel: when the batch is at most 512 and the first has K of at
 *    least 1024, N a multiple of 32 and at most 512 output tiles of 32 rows
 *    x 32 outputs, a workgroup per tile adds the second layer's partial
 *    sums over its 32 outputs into atomic accumulators (the workspace's
 *    first BNN_FORWARD_SYNC_BYTES: bnn_bfc_tail), and the add that
 *    completes an output writes it; otherwise, when they fit bnn_bfc_pair
 *    and have more rows than option gemv_max_rows, that kernel (option
 *    fuse_pair = 0 keeps them apart);
 *  - a run of 2-4 consecutive FC layers of at most 8192 weight words each,
 *    at batch <= 128, runs as one kernel that keeps the intermediate bits of
 *    each row in LDS (option fc_chain = 0 launches them one by one).
 * The results are the same either way.  workspace (device, >= the size
 * above, 256-byte aligned) holds the intermediate bits, and in its first
 * BNN_FORWARD_SYNC_BYTES the FC tail's accumulators: those bytes must be zero
 * before the first call that uses the workspace (one hipMemset after
 * allocating it), and every call that completes leaves them zero; the rest
 * needs no initialization.  Calls that use one workspace must not overlap
 * in time.  Errors: as the per-layer calls (conv weights not 16-byte
 * aligned: BNN_ERR_ALIGN, also from bnn_forward_workspace_size), plus
 * BNN_ERR_WORKSPACE.
 */
bnn_status bnn_forward(const bnn_layer* layers, int32_t n_layers,
                       int32_t batch, int32_t H, int32_t W, int32_t C,
                       const float* input, void* workspace, size_t ws_bytes,
                       int32_t* logits, hipStream_t stream);

/*
 * bnn_forward without a workspace argument, for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc.  The intermediate bits go to a device array owned by
 * the library, BNN_FORWARD_SCRATCH_BYTES (64 MiB) on each GPU the library
 * runs on, held from the first use on that GPU until the process ends.  The
 * call allocates nothing.  Results are those of bnn_forward, bit for bit.
 *   layers ... logits, stream: as for bnn_forward.  The stream must belong to
 *   the current device (else BNN_ERR_UNSUPPORTED).
 * Every call on one GPU shares that GPU's array: calls that overlap in time
 * on one GPU (other streams, or other threads without ordering between them)
 * race and give undefined results; calls on one stream are ordered.  The
 * array is laid out as bnn_forward's workspace: its first
 * BNN_FORWARD_SYNC_BYTES (the FC tail's accumulators) are zero when the library
 * is loaded and every completed call leaves them zero; nothing else in it
 * needs to start at zero (each layer writes every word of its output before
 * the next reads it), and a call leaves the last chain's bits there.  A
 * chain whose bnn_forward_workspace_size exceeds the array gives
 * BNN_ERR_WORKSPACE before anything is launched.  Other errors as for
 * bnn_forward.
 */
#define BNN_FORWARD_SCRATCH_BYTES ((size_t)64 << 20)

bnn_status bnn_forward_noalloc(const bnn_layer* layers, int32_t n_layers,
                               int32_t batch, int32_t H, int32_t W, int32_t C,
                               const float* input, int32_t* logits,
                               hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* BNN_H */
