// C ABI of libbnn.so (include/bnn.h): host-side validation, kernel dispatch
// and the layer chain.  Every entry point checks its arguments before it
// launches anything, reports problems through a status code plus a
// thread-local message, and never lets a C++ exception escape.
#include "bnn.h"

#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <atomic>
#include <mutex>
#include <new>

#include "kernels.hpp"

namespace {

thread_local char g_err[512] = "";

bnn_options default_options() {
  bnn_options o;
  o.algo = BNN_ALGO_AUTO;
  o.fuse_input = 1;
  o.fuse_first = 1;
  o.fc_chain = 1;
  o.conv1x1 = 1;
  o.xcd_order = 1;
  o.gemv_max_rows = 1;
  o.lds_weights = -1;
  o.late_thresholds = -1;
  o.fuse_pair = 1;
  return o;
}

thread_local bnn_options g_opt = default_options();

bnn_status fail(bnn_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

bnn_status ok() {
  g_err[0] = '\0';
  return BNN_OK;
}

bnn_status hip_status(hipError_t e, const char* where) {
  if (e == hipSuccess) return ok();
  return fail(BNN_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

// Kernel family for binary convs / GEMMs: the fp4 matrix-core kernel where
// the shape allows it, unless the options ask for the XOR-popcount vector
// kernels (the ablation).
bool use_mfma(const bnn::ConvGeom& g) {
  return g_opt.algo != BNN_ALGO_VALU && bnn::bconv_mfma_supported(g);
}

// 1x1 convs with K <= 256 over >= 65536 pixels, bits only: the kernel that
// keeps a wave's pixel operands and walks all filters (option conv1x1 = 0
// sends them to the general matrix-core kernel).
bool use_1x1(const bnn::ConvGeom& g, bool sums) {
  return g_opt.conv1x1 != 0 && bnn::bconv1x1_supported(g, sums);
}

// wprep: prepared weights (bnn_prepare_weights) for the general matrix-core
// kernel, or null; the other kernels take the packed w.
hipError_t launch_conv(const bnn::ConvGeom& g, const uint32_t* in, const uint32_t* w,
                       const void* wprep, const int32_t* thr, const uint32_t* flip,
                       int32_t* sums, uint32_t* bits, hipStream_t s) {
  if (use_mfma(g) && bits && use_1x1(g, sums != nullptr))
    return bnn::launch_bconv1x1(g, in, w, thr, flip, bits, s);
  if (use_mfma(g) && bits && !sums && bnn::bconv_img8_supported(g))
    return bnn::launch_bconv_img8(g, in, w, thr, flip, bits, s);
  if (use_mfma(g))
    return bnn::launch_bconv_mfma(g, in, w, wprep && bnn::bconv_mfma_prep_supported(g) ? wprep
                                                                                         : nullptr,
                                  thr, flip, sums, bits, s);
  return bnn::launch_bconv_valu(g, in, w, thr, flip, sums, bits, s);
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

constexpr int64_t kMaxItems = (int64_t{1} << 31) - 1;

// Validates a conv descriptor and fills the geometry.
bnn_status conv_geom(const bnn_conv_desc* d, bnn::ConvGeom* g) {
  if (!d) return fail(BNN_ERR_NULL, "conv descriptor is NULL");
  if (d->N < 1 || d->H < 1 || d->W < 1 || d->C < 1 || d->F < 1 || d->KH < 1 ||
      d->KW < 1)
    return fail(BNN_ERR_SHAPE,
                "conv sizes must be >= 1 (N=%d H=%d W=%d C=%d F=%d KH=%d KW=%d)",
                d->N, d->H, d->W, d->C, d->F, d->KH, d->KW);
  if (d->stride != 1)
    return fail(BNN_ERR_UNSUPPORTED, "conv stride %d: only stride 1 is implemented",
                d->stride);
  if (d->pad < 0) return fail(BNN_ERR_SHAPE, "conv pad %d < 0", d->pad);
  if (d->pool != 0 && d->pool != 2)
    return fail(BNN_ERR_SHAPE, "pool must be 0 or 2, got %d", d->pool);
  const int64_t Ho = int64_t{d->H} + 2 * int64_t{d->pad} - d->KH + 1;
  const int64_t Wo = int64_t{d->W} + 2 * int64_t{d->pad} - d->KW + 1;
  if (Ho < 1 || Wo < 1)
    return fail(BNN_ERR_SHAPE, "conv output %lldx%lld is empty", (long long)Ho,
                (long long)Wo);
  if (d->pool == 2 && (Ho < 2 || Wo < 2))
    return fail(BNN_ERR_SHAPE, "2x2 pooling needs a conv output of at least 2x2");
  const int64_t Cw = bnn::words_of(d->C);
  const int64_t in_words = int64_t{d->N} * d->H * d->W * Cw;
  const int64_t items = int64_t{d->N} * Ho * Wo;
  const int64_t wwords = int64_t{d->F} * d->KH * d->KW * Cw;
  // Launch limits: at most 8 work-items per output pixel (32-bit grid size)
  // and a filter-group count that fits the grid's y dimension.
  if (in_words > kMaxItems * 4 || items > (int64_t{1} << 28) || d->F > (1 << 20) ||
      int64_t{d->KH} * d->KW * d->C > kMaxItems / 2 || wwords > kMaxItems)
    return fail(BNN_ERR_SHAPE, "conv is too large for 32-bit indexing");
  g->N = d->N;
  g->H = d->H;
  g->W = d->W;
  g->C = d->C;
  g->F = d->F;
  g->KH = d->KH;
  g->KW = d->KW;
  g->pad = d->pad;
  g->pool = d->pool;
  g->Cw = static_cast<int32_t>(Cw);
  g->Fw = static_cast<int32_t>(bnn::words_of(d->F));
  g->Ho = static_cast<int32_t>(Ho);
  g->Wo = static_cast<int32_t>(Wo);
  g->Hp = d->pool == 2 ? g->Ho / 2 : g->Ho;
  g->Wp = d->pool == 2 ? g->Wo / 2 : g->Wo;
  return BNN_OK;
}

bnn_status check_outputs(const void* in, const uint32_t* w, const int32_t* thr,
                         const void* sums, const uint32_t* bits) {
  if (!in) return fail(BNN_ERR_NULL, "input pointer is NULL");
  if (!w) return fail(BNN_ERR_NULL, "weight pointer is NULL");
  if (!sums && !bits)
    return fail(BNN_ERR_NULL, "out_sums and out_bits are both NULL: nothing to compute");
  if (bits && !thr) return fail(BNN_ERR_NULL, "out_bits requested but thr is NULL");
  if (!aligned16(in) || !aligned16(w) || (sums && !aligned16(sums)) ||
      (bits && !aligned16(bits)))
    return fail(BNN_ERR_ALIGN, "input, weight and output pointers must be 16-byte aligned");
  return BNN_OK;
}

bnn_status gemm_check(int64_t M, int64_t N, int64_t K, const uint32_t* A,
                      const uint32_t* B, const int32_t* thr, const int32_t* sums,
                      const uint32_t* bits) {
  if (M < 1 || N < 1 || K < 1)
    return fail(BNN_ERR_SHAPE, "bgemm sizes must be >= 1 (M=%lld N=%lld K=%lld)",
                (long long)M, (long long)N, (long long)K);
  const int64_t Kw = bnn::words_of(K);
  if (M > (int64_t{1} << 28) || N > (1 << 20) || K > kMaxItems / 2 ||
      M * Kw > kMaxItems * 4 || N * Kw > kMaxItems)
    return fail(BNN_ERR_SHAPE, "bgemm is too large for 32-bit indexing");
  bnn_status st = check_outputs(A, B, thr, sums, bits);
  if (st != BNN_OK) return st;
  return BNN_OK;
}

bnn_status gemm_launch(int64_t M, int64_t N, int64_t K, const uint32_t* A,
                       const uint32_t* B, const int32_t* thr,
                       const uint32_t* flip, int32_t* sums, uint32_t* bits,
                       hipStream_t s) {
  // One row goes to the vector-ALU GEMV, whose time grows with every row;
  // from 2 rows on the matrix-core kernels are as fast or faster (the CIFAR
  // forward at 2 rows 30.7-31.0 against 29.7-29.9 us with its 8192 -> 1024
  // layer in the FC kernel; at one row the GEMV is 0.5-0.8 us faster), and
  // 3x faster at 16 rows.  Option gemv_max_rows (0..16) moves the limit.
  if (M <= g_opt.gemv_max_rows)
    return hip_status(bnn::launch_bgemv_valu(M, N, K, A, B, thr, flip, sums, bits, s),
                      "bgemm (gemv) launch");
  // K >= 1024 and N a multiple of 32: the FC kernel (bfc_gemm.hip), a
  // workgroup per 32 x 32 output tile up to 512 tiles, per 2 x 2 tiles above
  // that when N is a multiple of 64 (K not a multiple of the K split:
  // padded, see the kernel).  Graph-timed, bits only: 64 x 8192 -> 1024 4.7 us
  // against 6.65 us in the conv kernel, 256 x 18432 -> 1024 8.2 against
  // 10.4 us, 64 x 1024 -> 1024 3.7 against 4.2 us; 256 x 4096 -> 4096 with
  // int32 sums (1024 tiles) 7.55 against 9.2 us.  Larger grids with N not a
  // multiple of 64 stay with the conv kernel (one tile per workgroup took
  // 13.1 us on that shape).
  if (g_opt.algo != BNN_ALGO_VALU && bnn::bfc_gemm_supported(M, N, K) &&
      (((M + 31) / 32) * ((N + 31) / 32) <= 512 || N % 64 == 0))
    return hip_status(bnn::launch_bfc_gemm(M, N, K, A, B, thr, flip, sums, bits, s),
                      "bgemm launch");
  // M rows of A are a 1 x M image with K channels; B holds N 1x1 filters.
  bnn::ConvGeom g;
  g.N = 1;
  g.H = 1;
  g.W = static_cast<int32_t>(M);
  g.C = static_cast<int32_t>(K);
  g.F = static_cast<int32_t>(N);
  g.KH = g.KW = 1;
  g.pad = 0;
  g.pool = 0;
  g.Cw = static_cast<int32_t>(bnn::words_of(K));
  g.Fw = static_cast<int32_t>(bnn::words_of(N));
  g.Ho = 1;
  g.Wo = g.W;
  g.Hp = 1;
  g.Wp = g.W;
  return hip_status(launch_conv(g, A, B, nullptr, thr, flip, sums, bits, s), "bgemm launch");
}

}  // namespace

namespace bnn {
const bnn_options& options() { return g_opt; }
}  // namespace bnn

extern "C" {

const char* bnn_last_error(void) { return g_err; }

int32_t bnn_abi_version(void) { return BNN_ABI_VERSION; }

void bnn_default_options(bnn_options* opt) {
  if (opt) *opt = default_options();
}

bnn_status bnn_set_options(const bnn_options* o) {
  if (!o) return fail(BNN_ERR_NULL, "set_options: options pointer is NULL");
  auto flag = [](int32_t v) { return v == 0 || v == 1; };
  auto tri = [](int32_t v) { return v == -1 || v == 0 || v == 1; };
  if ((o->algo != BNN_ALGO_AUTO && o->algo != BNN_ALGO_VALU) || !flag(o->fuse_input) ||
      !flag(o->fuse_first) || !flag(o->fc_chain) || !flag(o->conv1x1) ||
      o->xcd_order < 0 || o->xcd_order > 2 ||
      o->gemv_max_rows < 0 || o->gemv_max_rows > 16 || !tri(o->lds_weights) ||
      !tri(o->late_thresholds) || !flag(o->fuse_pair))
    return fail(BNN_ERR_SHAPE,
                "set_options: out of range (algo %d, fuse_input %d, fuse_first %d, fc_chain %d, "
                "conv1x1 %d, xcd_order %d, gemv_max_rows %d, lds_weights %d, "
                "late_thresholds %d, fuse_pair %d)",
                o->algo, o->fuse_input, o->fuse_first, o->fc_chain, o->conv1x1, o->xcd_order,
                o->gemv_max_rows, o->lds_weights, o->late_thresholds, o->fuse_pair);
  g_opt = *o;
  return ok();
}

bnn_status bnn_get_options(bnn_options* o) {
  if (!o) return fail(BNN_ERR_NULL, "get_options: options pointer is NULL");
  *o = g_opt;
  return ok();
}

bnn_status bnn_pack_bits(const float* x, const float* offset, int64_t rows,
                         int64_t D, uint32_t* out, hipStream_t stream) {
  try {
    if (rows < 0 || D < 1)
      return fail(BNN_ERR_SHAPE, "pack: rows must be >= 0 and D >= 1 (rows=%lld D=%lld)",
                  (long long)rows, (long long)D);
    if (rows * bnn::words_of(D) > kMaxItems || D > kMaxItems)
      return fail(BNN_ERR_SHAPE, "pack: too large for 32-bit indexing");
    if (rows == 0) return ok();
    if (!x || !out) return fail(BNN_ERR_NULL, "pack: x and out must be non-NULL");
    return hip_status(bnn::launch_pack_bits(x, offset, rows, D, out, stream), "pack launch");
  } catch (...) {
    return fail(BNN_ERR_HIP, "pack: unexpected C++ exception");
  }
}

bnn_status bnn_conv_output_dims(const bnn_conv_desc* d, int32_t* Ho, int32_t* Wo,
                                int32_t* Hp, int32_t* Wp) {
  bnn::ConvGeom g;
  bnn_status st = conv_geom(d, &g);
  if (st != BNN_OK) return st;
  if (Ho) *Ho = g.Ho;
  if (Wo) *Wo = g.Wo;
  if (Hp) *Hp = g.Hp;
  if (Wp) *Wp = g.Wp;
  return ok();
}

bnn_status bnn_bconv2d(const bnn_conv_desc* d, const uint32_t* in, const uint32_t* w,
                       const int32_t* thr, const uint32_t* flip, int32_t* out_sums,
                       uint32_t* out_bits, hipStream_t stream) {
  try {
    bnn::ConvGeom g;
    bnn_status st = conv_geom(d, &g);
    if (st != BNN_OK) return st;
    st = check_outputs(in, w, thr, out_sums, out_bits);
    if (st != BNN_OK) return st;
    return hip_status(launch_conv(g, in, w, nullptr, thr, flip, out_sums, out_bits, stream),
                      "bconv2d launch");
  } catch (...) {
    return fail(BNN_ERR_HIP, "bconv2d: unexpected C++ exception");
  }
}

bnn_status bnn_prepared_weights_size(int32_t F, int32_t KH, int32_t KW, int32_t C,
                                     size_t* bytes) {
  if (!bytes) return fail(BNN_ERR_NULL, "prepared_weights_size: bytes is NULL");
  if (F < 1 || KH < 1 || KW < 1 || C < 1)
    return fail(BNN_ERR_SHAPE, "prepared_weights_size: F, KH, KW, C must be >= 1");
  if (int64_t{KH} * KW * C > kMaxItems / 2 || F > (1 << 20))
    return fail(BNN_ERR_SHAPE, "prepared_weights_size: too large for 32-bit indexing");
  const int64_t b = bnn::prepared_weights_bytes(F, KH, KW, C);
  if (b >= (int64_t{1} << 31))
    return fail(BNN_ERR_SHAPE, "prepared_weights_size: %lld bytes, beyond the 2 GiB supported",
                (long long)b);
  *bytes = static_cast<size_t>(b);
  return ok();
}

bnn_status bnn_prepare_weights(int32_t F, int32_t KH, int32_t KW, int32_t C,
                               const uint32_t* w, void* out, hipStream_t stream) {
  try {
    size_t bytes = 0;
    bnn_status st = bnn_prepared_weights_size(F, KH, KW, C, &bytes);
    if (st != BNN_OK) return st;
    if (!w || !out) return fail(BNN_ERR_NULL, "prepare_weights: w and out must be non-NULL");
    if (!aligned16(w) || !aligned16(out))
      return fail(BNN_ERR_ALIGN, "prepare_weights: w and out must be 16-byte aligned");
    return hip_status(bnn::launch_prepare_weights(F, KH, KW, C, w, out, stream),
                      "prepare_weights launch");
  } catch (...) {
    return fail(BNN_ERR_HIP, "prepare_weights: unexpected C++ exception");
  }
}

bnn_status bnn_bconv2d_prepared(const bnn_conv_desc* d, const uint32_t* in, const uint32_t* w,
                                const void* wprep, const int32_t* thr, const uint32_t* flip,
                                int32_t* out_sums, uint32_t* out_bits, hipStream_t stream) {
  try {
    bnn::ConvGeom g;
    bnn_status st = conv_geom(d, &g);
    if (st != BNN_OK) return st;
    st = check_outputs(in, w, thr, out_sums, out_bits);
    if (st != BNN_OK) return st;
    if (!wprep) return fail(BNN_ERR_NULL, "bconv2d_prepared: wprep is NULL");
    if (!aligned16(wprep))
      return fail(BNN_ERR_ALIGN, "bconv2d_prepared: wprep must be 16-byte aligned");
    return hip_status(launch_conv(g, in, w, wprep, thr, flip, out_sums, out_bits, stream),
                      "bconv2d_prepared launch");
  } catch (...) {
    return fail(BNN_ERR_HIP, "bconv2d_prepared: unexpected C++ exception");
  }
}

bnn_status bnn_fconv2d_binw(const bnn_conv_desc* d, const float* in, const uint32_t* w,
                            const int32_t* thr, const uint32_t* flip, float* out_sums,
                            uint32_t* out_bits, hipStream_t stream) {
  try {
    bnn::ConvGeom g;
    bnn_status st = conv_geom(d, &g);
    if (st != BNN_OK) return st;
    st = check_outputs(in, w, thr, out_sums, out_bits);
    if (st != BNN_OK) return st;
    return hip_status(
        bnn::launch_fconv_binw(g, in, w, thr, flip, out_sums, out_bits, stream),
        "fconv2d_binw launch");
  } catch (...) {
    return fail(BNN_ERR_HIP, "fconv2d_binw: unexpected C++ exception");
  }
}

bnn_status bnn_binarize_input(int32_t mode, const float* x, const float* offset, int32_t N,
                              int32_t H, int32_t W, int32_t Cin, uint32_t* out,
                              hipStream_t stream) {
  try {
    if (mode != BNN_INPUT_THRESHOLD && mode != BNN_INPUT_GRAY && mode != BNN_INPUT_LBP)
      return fail(BNN_ERR_SHAPE, "binarize_input: unknown mode %d", mode);
    if (N < 1 || H < 1 || W < 1 || Cin < 1)
      return fail(BNN_ERR_SHAPE, "binarize_input: N, H, W, Cin must be >= 1");
    if (mode == BNN_INPUT_THRESHOLD && Cin > 32)
      return fail(BNN_ERR_SHAPE, "binarize_input: thresholding takes Cin <= 32 (got %d); "
                  "bnn_pack_bits packs any channel count", Cin);
    if (mode != BNN_INPUT_THRESHOLD && Cin != 3)
      return fail(BNN_ERR_SHAPE, "binarize_input: gray and LBP need Cin == 3 (got %d)", Cin);
    if (int64_t{N} * H * W * Cin > kMaxItems)
      return fail(BNN_ERR_SHAPE, "binarize_input: image too large for 32-bit indexing");
    if (!x || !out) return fail(BNN_ERR_NULL, "binarize_input: x and out must be non-NULL");
    if (!aligned16(x) || !aligned16(out))
      return fail(BNN_ERR_ALIGN, "binarize_input: x and out must be 16-byte aligned");
    return hip_status(bnn::launch_binarize(mode, x, offset, N, H, W, Cin, out, stream),
                      "binarize_input launch");
  } catch (...) {
    return fail(BNN_ERR_HIP, "binarize_input: unexpected C++ exception");
  }
}

bnn_status bnn_bconv2d_input(const bnn_conv_desc* d, int32_t mode, const float* x,
                             const float* offset, const uint32_t* w, const int32_t* thr,
                             const uint32_t* flip, int32_t* out_sums, uint32_t* out_bits,
                             hipStream_t stream) {
  try {
    bnn::ConvGeom g;
    bnn_status st = conv_geom(d, &g);
    if (st != BNN_OK) return st;
    if (mode != BNN_INPUT_THRESHOLD && mode != BNN_INPUT_GRAY && mode != BNN_INPUT_LBP)
      return fail(BNN_ERR_SHAPE, "bconv2d_input: unknown mode %d", mode);
    if (mode != BNN_INPUT_THRESHOLD && g.C != bnn::input_channels_of(mode, 3))
      return fail(BNN_ERR_SHAPE, "bconv2d_input: mode %d gives %d channels, desc has C=%d",
                  mode, bnn::input_channels_of(mode, 3), g.C);
    if (!bnn::bconv_patch_supported(g))
      return fail(BNN_ERR_UNSUPPORTED,
                  "bconv2d_input: a %dx%d window of %d channels (%lld bits) is beyond the "
                  "supported C, KH, KW <= 32 and 128 bits",
                  g.KH, g.KW, g.C, (long long)(int64_t{g.KH} * g.KW * g.C));
    const int64_t cin = mode == BNN_INPUT_THRESHOLD ? g.C : 3;
    if (int64_t{g.N} * g.H * g.W * cin > kMaxItems)
      return fail(BNN_ERR_SHAPE, "bconv2d_input: image too large for 32-bit indexing");
    st = check_outputs(x, w, thr, out_sums, out_bits);
    if (st != BNN_OK) return st;
    return hip_status(bnn::launch_bconv_patch(g, mode, x, offset, w, thr, flip, out_sums,
                                              out_bits, stream),
                      "bconv2d_input launch");
  } catch (...) {
    return fail(BNN_ERR_HIP, "bconv2d_input: unexpected C++ exception");
  }
}

bnn_status bnn_fconv_bconv2d(const bnn_conv_desc* d0, const bnn_conv_desc* d1, const float* x,
                             const uint32_t* w0, const int32_t* thr0, const uint32_t* flip0,
                             const uint32_t* w1, const void* w1prep, const int32_t* thr1,
                             const uint32_t* flip1, uint32_t* out_bits, hipStream_t stream) {
  try {
    bnn::ConvGeom g0, g1;
    bnn_status st = conv_geom(d0, &g0);
    if (st != BNN_OK) return st;
    st = conv_geom(d1, &g1);
    if (st != BNN_OK) return st;
    if (g1.N != g0.N || g1.H != g0.Hp || g1.W != g0.Wp || g1.C != g0.F)
      return fail(BNN_ERR_SHAPE,
                  "fconv_bconv2d: second layer input %dx%dx%dx%d does not match the first "
                  "layer's output %dx%dx%dx%d",
                  g1.N, g1.H, g1.W, g1.C, g0.N, g0.Hp, g0.Wp, g0.F);
    if (!bnn::fconv_bconv_supported(g0, g1))
      return fail(BNN_ERR_UNSUPPORTED,
                  "fconv_bconv2d: needs 3x3 convs, first layer C <= 4, 64 or 128 filters and "
                  "no pooling, second layer 64 or 128 filters, pads 0 or 1");
    if (!w1) return fail(BNN_ERR_NULL, "fconv_bconv2d: w1 is NULL");
    if (!thr0) return fail(BNN_ERR_NULL, "fconv_bconv2d: thr0 is NULL");
    if (!out_bits) return fail(BNN_ERR_NULL, "fconv_bconv2d: out_bits is NULL");
    if (!aligned16(w1) || !aligned16(w1prep))
      return fail(BNN_ERR_ALIGN, "fconv_bconv2d: w1 and w1prep must be 16-byte aligned");
    st = check_outputs(x, w0, thr1, nullptr, out_bits);
    if (st != BNN_OK) return st;
    return hip_status(bnn::launch_fconv_bconv(g0, g1, x, w0, thr0, flip0, w1, w1prep, thr1, flip1,
                                              out_bits, stream),
                      "fconv_bconv2d launch");
  } catch (...) {
    return fail(BNN_ERR_HIP, "fconv_bconv2d: unexpected C++ exception");
  }
}

bnn_status bnn_input_bconv_bconv2d(const bnn_conv_desc* d0, const bnn_conv_desc* d1,
                                  int32_t mode, const float* x, const float* offset,
                                  const uint32_t* w0, const int32_t* thr0,
                                  const uint32_t* flip0, const uint32_t* w1,
                                  const void* w1prep, const int32_t* thr1,
                                  const uint32_t* flip1, uint32_t* out_bits,
                                  hipStream_t stream) {
  try {
    bnn::ConvGeom g0, g1;
    bnn_status st = conv_geom(d0, &g0);
    if (st != BNN_OK) return st;
    st = conv_geom(d1, &g1);
    if (st != BNN_OK) return st;
    if (mode != BNN_INPUT_THRESHOLD && mode != BNN_INPUT_GRAY && mode != BNN_INPUT_LBP)
      return fail(BNN_ERR_SHAPE, "input_bconv_bconv2d: unknown mode %d", mode);
    if (g1.N != g0.N || g1.H != g0.Hp || g1.W != g0.Wp || g1.C != g0.F)
      return fail(BNN_ERR_SHAPE,
                  "input_bconv_bconv2d: second layer input %dx%dx%dx%d does not match the "
                  "first layer's output %dx%dx%dx%d",
                  g1.N, g1.H, g1.W, g1.C, g0.N, g0.Hp, g0.Wp, g0.F);
    if (!bnn::input_bconv_bconv_supported(mode, g0, g1))
      return fail(BNN_ERR_UNSUPPORTED,
                  "input_bconv_bconv2d: needs mode THRESHOLD, 3 input channels, 3x3 convs, "
                  "64 or 128 filters, no pooling in the first, pads 0 or 1");
    if (!w1) return fail(BNN_ERR_NULL, "input_bconv_bconv2d: w1 is NULL");
    if (!thr0) return fail(BNN_ERR_NULL, "input_bconv_bconv2d: thr0 is NULL");
    if (!out_bits) return fail(BNN_ERR_NULL, "input_bconv_bconv2d: out_bits is NULL");
    if (!aligned16(w1) || !aligned16(w1prep))
      return fail(BNN_ERR_ALIGN, "input_bconv_bconv2d: w1 and w1prep must be 16-byte aligned");
    st = check_outputs(x, w0, thr1, nullptr, out_bits);
    if (st != BNN_OK) return st;
    return hip_status(bnn::launch_input_bconv_bconv(g0, g1, x, offset, w0, thr0, flip0, w1,
                                                    w1prep, thr1, flip1, out_bits, stream),
                      "input_bconv_bconv2d launch");
  } catch (...) {
    return fail(BNN_ERR_HIP, "input_bconv_bconv2d: unexpected C++ exception");
  }
}

bnn_status bnn_bconv_bconv2d(const bnn_conv_desc* d0, const bnn_conv_desc* d1, const uint32_t* x,
                             const uint32_t* w0, const int32_t* thr0, const uint32_t* flip0,
                             const uint32_t* w1, const int32_t* thr1, const uint32_t* flip1,
                             uint32_t* out_bits, hipStream_t stream) {
  try {
    bnn::ConvGeom g0, g1;
    bnn_status st = conv_geom(d0, &g0);
    if (st != BNN_OK) return st;
    st = conv_geom(d1, &g1);
    if (st != BNN_OK) return st;
    if (g1.N != g0.N || g1.H != g0.Hp || g1.W != g0.Wp || g1.C != g0.F)
      return fail(BNN_ERR_SHAPE,
                  "bconv_bconv2d: second conv input %dx%dx%dx%d does not match the first "
                  "conv's output %dx%dx%dx%d",
                  g1.N, g1.H, g1.W, g1.C, g0.N, g0.Hp, g0.Wp, g0.F);
    if (!bnn::bconv_bconv_supported(g0, g1))
      return fail(BNN_ERR_UNSUPPORTED,
                  "bconv_bconv2d: needs 3x3 convs with pad 1 on 16-pixel-wide images, the "
                  "first with 64, 128 or 256 channels, 256 filters and no pooling, the second "
                  "with 256 filters");
    if (!w1) return fail(BNN_ERR_NULL, "bconv_bconv2d: w1 is NULL");
    if (!thr0) return fail(BNN_ERR_NULL, "bconv_bconv2d: thr0 is NULL");
    if (!out_bits) return fail(BNN_ERR_NULL, "bconv_bconv2d: out_bits is NULL");
    if (!aligned16(w1)) return fail(BNN_ERR_ALIGN, "bconv_bconv2d: w1 must be 16-byte aligned");
    st = check_outputs(x, w0, thr1, nullptr, out_bits);
    if (st != BNN_OK) return st;
    return hip_status(bnn::launch_bconv_bconv(g0, g1, x, w0, thr0, flip0, w1, thr1, flip1,
                                              out_bits, stream),
                      "bconv_bconv2d launch");
  } catch (...) {
    return fail(BNN_ERR_HIP, "bconv_bconv2d: unexpected C++ exception");
  }
}

bnn_status bnn_bfc_pair(int64_t M, int64_t K0, int64_t N0, int64_t N1, const uint32_t* A,
                        const uint32_t* w0, const int32_t* thr0, const uint32_t* flip0,
                        const uint32_t* w1, const int32_t* thr1, const uint32_t* flip1,
                        int32_t* out_sums, uint32_t* out_bits, hipStream_t stream) {
  try {
    if (M < 1 || K0 < 1 || N0 < 1 || N1 < 1)
      return fail(BNN_ERR_SHAPE, "bfc_pair: sizes must be >= 1 (M=%lld K0=%lld N0=%lld N1=%lld)",
                  (long long)M, (long long)K0, (long long)N0, (long long)N1);
    if (!bnn::bfc_pair_supported(M, K0, N0, N1))
      return fail(BNN_ERR_UNSUPPORTED,
                  "bfc_pair: needs K0 = 512 or 1024, N0 = 256, 512 or 1024, N1 <= 32 "
                  "and at most 2^26 rows");
    if (!A || !w0 || !w1) return fail(BNN_ERR_NULL, "bfc_pair: A, w0 or w1 is NULL");
    if (!thr0) return fail(BNN_ERR_NULL, "bfc_pair: thr0 is NULL");
    if (!out_sums && !out_bits)
      return fail(BNN_ERR_NULL, "bfc_pair: out_sums and out_bits are both NULL");
    if (out_sums && out_bits)
      return fail(BNN_ERR_SHAPE, "bfc_pair: give out_sums or out_bits, not both");
    if (out_bits && !thr1) return fail(BNN_ERR_NULL, "bfc_pair: out_bits requested but thr1 is NULL");
    if (!aligned16(A) || !aligned16(w0) || !aligned16(w1) || !aligned16(out_sums) ||
        !aligned16(out_bits))
      return fail(BNN_ERR_ALIGN, "bfc_pair: A, weights and outputs must be 16-byte aligned");
    return hip_status(bnn::launch_bfc_pair(M, K0, N0, N1, A, w0, thr0, flip0, w1, thr1, flip1,
                                           out_sums, out_bits, stream),
                      "bfc_pair launch");
  } catch (...) {
    return fail(BNN_ERR_HIP, "bfc_pair: unexpected C++ exception");
  }
}

bnn_status bnn_bfc_tail(int64_t M, int64_t K0, int64_t N0, int64_t N1, const uint32_t* A,
                        const uint32_t* w0, const int32_t* thr0, const uint32_t* flip0,
                        const uint32_t* w1, const int32_t* thr1, const uint32_t* flip1,
                        int32_t* out_sums, uint32_t* out_bits, void* accum,
                        hipStream_t stream) {
  try {
    if (M < 1 || K0 < 1 || N0 < 1 || N1 < 1)
      return fail(BNN_ERR_SHAPE, "bfc_tail: sizes must be >= 1 (M=%lld K0=%lld N0=%lld N1=%lld)",
                  (long long)M, (long long)K0, (long long)N0, (long long)N1);
    if (!bnn::bfc_tail_supported(M, K0, N0, N1))
      return fail(BNN_ERR_UNSUPPORTED,
                  "bfc_tail: needs M <= 512, K0 >= 1024, N0 a multiple of 32 with "
                  "ceil(M / 32) * N0 / 32 <= 512, and N1 <= 32");
    if (!A || !w0 || !w1) return fail(BNN_ERR_NULL, "bfc_tail: A, w0 or w1 is NULL");
    if (!thr0) return fail(BNN_ERR_NULL, "bfc_tail: thr0 is NULL");
    if (!accum) return fail(BNN_ERR_NULL, "bfc_tail: accum is NULL");
    if (!out_sums && !out_bits)
      return fail(BNN_ERR_NULL, "bfc_tail: out_sums and out_bits are both NULL");
    if (out_sums && out_bits)
      return fail(BNN_ERR_SHAPE, "bfc_tail: give out_sums or out_bits, not both");
    if (out_bits && !thr1) return fail(BNN_ERR_NULL, "bfc_tail: out_bits requested but thr1 is NULL");
    if (!aligned16(A) || !aligned16(w0) || !aligned16(w1) || !aligned16(out_sums) ||
        !aligned16(out_bits) || !aligned16(accum))
      return fail(BNN_ERR_ALIGN,
                  "bfc_tail: A, weights, outputs and accum must be 16-byte aligned");
    return hip_status(bnn::launch_bfc_tail(M, K0, N0, N1, A, w0, thr0, flip0, w1, thr1, flip1,
                                           out_sums, out_bits, accum, stream),
                      "bfc_tail launch");
  } catch (...) {
    return fail(BNN_ERR_HIP, "bfc_tail: unexpected C++ exception");
  }
}

bnn_status bnn_bgemm(int64_t M, int64_t N, int64_t K, const uint32_t* A,
                     const uint32_t* B, const int32_t* thr, const uint32_t* flip,
                     int32_t* out_sums, uint32_t* out_bits, hipStream_t stream) {
  try {
    bnn_status st = gemm_check(M, N, K, A, B, thr, out_sums, out_bits);
    if (st != BNN_OK) return st;
    return gemm_launch(M, N, K, A, B, thr, flip, out_sums, out_bits, stream);
  } catch (...) {
    return fail(BNN_ERR_HIP, "bgemm: unexpected C++ exception");
  }
}

// ------------------------------------------------------------ layer chain --
namespace {

constexpr size_t kAlign = 256;

// Size of bnn_forward_noalloc's scratch array (BNN_FORWARD_SCRATCH_BYTES).
constexpr size_t kScratchBytes = BNN_FORWARD_SCRATCH_BYTES;

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// bnn_forward's workspace: BNN_FORWARD_SYNC_BYTES of the FC tail kernel's
// accumulators (zero between calls), then two buffers of `half` bytes for
// the packed activations.
static_assert(bnn::kTailAccumBytes <= BNN_FORWARD_SYNC_BYTES, "tail accumulators fit");
struct WsPlan {
  size_t half = 0;
  size_t total() const { return BNN_FORWARD_SYNC_BYTES + 2 * half; }
};

// Activation state between layers: an NHWC map of packed bits (or, before
// the first layer, the fp32 input).
struct Act {
  int64_t H, W, C;  // C in channels (bits); FC outputs are 1 x 1 x N
};

bool is_input_kind(int32_t k) {
  return k == BNN_LAYER_INPUT_THRESHOLD || k == BNN_LAYER_INPUT_GRAY || k == BNN_LAYER_INPUT_LBP;
}

int input_mode(int32_t kind) {
  return kind == BNN_LAYER_INPUT_GRAY ? BNN_INPUT_GRAY
         : kind == BNN_LAYER_INPUT_LBP ? BNN_INPUT_LBP : BNN_INPUT_THRESHOLD;
}

// Walks the chain, validating shapes; returns the workspace layout (from the
// largest activation size in bytes, packed words).
bnn_status plan_chain(const bnn_layer* L, int32_t n, int32_t batch, int32_t H,
                      int32_t W, int32_t C, WsPlan* plan) {
  if (!L) return fail(BNN_ERR_NULL, "forward: layers is NULL");
  if (n < 1) return fail(BNN_ERR_SHAPE, "forward: need at least one layer");
  if (batch < 1 || H < 1 || W < 1 || C < 1)
    return fail(BNN_ERR_SHAPE, "forward: batch, H, W, C must be >= 1");
  if (!is_input_kind(L[0].kind) && L[0].kind != BNN_LAYER_FCONV_BINW)
    return fail(BNN_ERR_SHAPE,
                "forward: layer 0 must be an input layer (INPUT_THRESHOLD, INPUT_GRAY, "
                "INPUT_LBP) or FCONV_BINW");
  if (L[n - 1].kind != BNN_LAYER_BFC_LOGITS)
    return fail(BNN_ERR_SHAPE, "forward: the last layer must be BFC_LOGITS");
  Act a{H, W, C};
  size_t mx = 0;
  for (int32_t li = 0; li < n; ++li) {
    const bnn_layer& l = L[li];
    switch (l.kind) {
      case BNN_LAYER_INPUT_THRESHOLD:
      case BNN_LAYER_INPUT_GRAY:
      case BNN_LAYER_INPUT_LBP: {
        if (li != 0) return fail(BNN_ERR_SHAPE, "forward: layer %d: an input layer must be first", li);
        if (l.C != C) return fail(BNN_ERR_SHAPE, "forward: layer 0 C=%d but input has C=%d", l.C, C);
        if (l.kind != BNN_LAYER_INPUT_THRESHOLD && C != 3)
          return fail(BNN_ERR_SHAPE, "forward: gray and LBP inputs need C == 3 (got %d)", C);
        a = Act{H, W, bnn::input_channels_of(input_mode(l.kind), C)};
        break;
      }
      case BNN_LAYER_FCONV_BINW:
      case BNN_LAYER_BCONV: {
        if (l.kind == BNN_LAYER_FCONV_BINW && li != 0)
          return fail(BNN_ERR_SHAPE, "forward: layer %d: FCONV_BINW must be first", li);
        if (l.C != a.C)
          return fail(BNN_ERR_SHAPE, "forward: layer %d expects C=%d, previous layer gives %lld",
                      li, l.C, (long long)a.C);
        if (!l.w || !l.thr) return fail(BNN_ERR_NULL, "forward: layer %d: w and thr are required", li);
        if (!aligned16(l.w) || !aligned16(l.wprep))
          return fail(BNN_ERR_ALIGN, "forward: layer %d: w and wprep must be 16-byte aligned", li);
        bnn_conv_desc d{batch, static_cast<int32_t>(a.H), static_cast<int32_t>(a.W), l.C, l.F,
                        l.KH, l.KW, l.stride, l.pad, l.pool};
        bnn::ConvGeom g;
        bnn_status st = conv_geom(&d, &g);
        if (st != BNN_OK) return fail(st, "forward: layer %d: %s", li, g_err);
        a = Act{g.Hp, g.Wp, l.F};
        break;
      }
      case BNN_LAYER_BFC:
      case BNN_LAYER_BFC_LOGITS: {
        if (li == 0) return fail(BNN_ERR_SHAPE, "forward: an FC layer cannot be first");
        if ((a.H * a.W) != 1 && (a.C % 32) != 0)
          return fail(BNN_ERR_SHAPE,
                      "forward: layer %d: flattening a %lldx%lld map needs C %% 32 == 0 (C=%lld)",
                      li, (long long)a.H, (long long)a.W, (long long)a.C);
        const int64_t K = a.H * a.W * a.C;
        if (l.K != K)
          return fail(BNN_ERR_SHAPE, "forward: layer %d expects K=%d, previous layer gives %lld",
                      li, l.K, (long long)K);
        if (l.N < 1) return fail(BNN_ERR_SHAPE, "forward: layer %d: N must be >= 1", li);
        if (!l.w) return fail(BNN_ERR_NULL, "forward: layer %d: w is required", li);
        if (l.kind == BNN_LAYER_BFC && !l.thr)
          return fail(BNN_ERR_NULL, "forward: layer %d: thr is required", li);
        if (l.kind == BNN_LAYER_BFC_LOGITS && li != n - 1)
          return fail(BNN_ERR_SHAPE, "forward: BFC_LOGITS must be the last layer");
        bnn_status st = gemm_check(batch, l.N, l.K, reinterpret_cast<const uint32_t*>(kAlign),
                                   l.w, l.thr, reinterpret_cast<const int32_t*>(kAlign), nullptr);
        if (st != BNN_OK) return fail(st, "forward: layer %d: %s", li, g_err);
        a = Act{1, 1, l.N};
        break;
      }
      default:
        return fail(BNN_ERR_SHAPE, "forward: layer %d has unknown kind %d", li, l.kind);
    }
    if (l.kind != BNN_LAYER_BFC_LOGITS) {
      const size_t bytes = static_cast<size_t>(batch) * a.H * a.W * bnn::words_of(a.C) * 4;
      if (bytes > mx) mx = bytes;
    }
  }
  plan->half = align_up(mx);
  return BNN_OK;
}

// Length of the run of FC layers starting at layer li that bnn_forward sends
// to the chained FC kernel (1: none).  Every layer in the run has at most
// kChainWords weight words (each block of the chained kernel reads all of
// them), the batch is at most 128 rows (beyond that the per-layer kernels
// have parallelism enough to hide their launches), and option fc_chain = 0
// keeps one launch per layer.
int fc_chain_run(const bnn_layer* L, int32_t li, int32_t n, int32_t batch) {
  constexpr int64_t kChainWords = 8192;
  if (g_opt.fc_chain == 0 || batch > 128) return 1;
  int run = 0;
  bnn::FcChainLayer fl[bnn::kFcChainMax];
  while (li + run < n && run < bnn::kFcChainMax) {
    const bnn_layer& q = L[li + run];
    if (q.kind != BNN_LAYER_BFC && q.kind != BNN_LAYER_BFC_LOGITS) break;
    if (int64_t{q.N} * bnn::words_of(q.K) > kChainWords || !aligned16(q.w)) break;
    const bool lg = q.kind == BNN_LAYER_BFC_LOGITS;
    fl[run] = bnn::FcChainLayer{q.w, lg ? nullptr : q.thr, lg ? nullptr : q.flip, q.K, q.N};
    ++run;
    if (lg) break;
  }
  while (run > 1 && !bnn::bfc_chain_supported(fl, run)) --run;
  return run > 1 ? run : 1;
}

}  // namespace

bnn_status bnn_forward_workspace_size(const bnn_layer* layers, int32_t n_layers,
                                      int32_t batch, int32_t H, int32_t W, int32_t C,
                                      size_t* bytes) {
  try {
    if (!bytes) return fail(BNN_ERR_NULL, "forward_workspace_size: bytes is NULL");
    WsPlan plan;
    bnn_status st = plan_chain(layers, n_layers, batch, H, W, C, &plan);
    if (st != BNN_OK) return st;
    *bytes = plan.total();
    return ok();
  } catch (...) {
    return fail(BNN_ERR_HIP, "forward_workspace_size: unexpected C++ exception");
  }
}

}  // extern "C"

// Scratch memory of bnn_forward_noalloc: a file-scope device array, one copy
// per GPU, held from the module's load on that GPU until the process ends.
// Host code never passes the array's name to a kernel (on the host it is a
// stand-in, not a device address): each GPU's copy is looked up once with
// hipGetSymbolAddress, with that GPU current, and that address is used.
static __device__ __align__(256) unsigned char scratch[BNN_FORWARD_SCRATCH_BYTES];

namespace {

// The layer chain of bnn_forward on a validated plan, with the workspace
// laid out as WsPlan says (256-byte aligned).
bnn_status run_chain(const bnn_layer* layers, int32_t n_layers, int32_t batch, int32_t H,
                     int32_t W, int32_t C, const float* input, void* workspace,
                     const WsPlan& plan, int32_t* logits, hipStream_t stream) {
  bnn_status st = BNN_OK;
  char* const ws = static_cast<char*>(workspace);
  void* const tail_accum = ws;
  uint32_t* buf[2] = {reinterpret_cast<uint32_t*>(ws + BNN_FORWARD_SYNC_BYTES),
                      reinterpret_cast<uint32_t*>(ws + BNN_FORWARD_SYNC_BYTES + plan.half)};
  // An input threshold followed by a conv whose window fits one word runs
  // as one patch-packing kernel on the fp32 image (option fuse_input = 0
  // keeps the two separate steps).
  bool fuse_input = false;
  const int mode = input_mode(layers[0].kind);
  if (n_layers > 1 && is_input_kind(layers[0].kind) && layers[1].kind == BNN_LAYER_BCONV) {
    bnn::ConvGeom g1;
    g1.KH = layers[1].KH;
    g1.KW = layers[1].KW;
    g1.C = layers[1].C;
    fuse_input = g_opt.fuse_input != 0 && bnn::bconv_patch_supported(g1);
  }
  // Input thresholding, a 3x3 binary conv of 64 or 128 filters over 3
  // channels and a second 3x3 binary conv run as one kernel that keeps the
  // first conv's bits in LDS (fconv_bconv.hip; a matrix-core kernel, so not
  // under the vector-ALU ablation; option fuse_input = 0 keeps all three
  // apart).
  bool fuse_input3 = false;
  bnn::ConvGeom g_in1;
  if (fuse_input && n_layers > 2 && layers[2].kind == BNN_LAYER_BCONV) {
    const bnn_layer& l1 = layers[1];
    const bnn_layer& l2 = layers[2];
    bnn_conv_desc d1{batch, H, W, l1.C, l1.F, l1.KH, l1.KW, l1.stride, l1.pad, l1.pool};
    bnn::ConvGeom g2;
    if (conv_geom(&d1, &g_in1) == BNN_OK) {  // (the chain is validated above)
      bnn_conv_desc d2{batch, g_in1.Hp, g_in1.Wp, l2.C, l2.F,
                       l2.KH, l2.KW, l2.stride, l2.pad, l2.pool};
      fuse_input3 = conv_geom(&d2, &g2) == BNN_OK && use_mfma(g2) &&
                    bnn::input_bconv_bconv_supported(mode, g_in1, g2);
    }
  }
  // A real-valued first layer followed by a 3x3 binary conv that fits runs
  // as one kernel with the first layer's bits in LDS (a matrix-core kernel,
  // so not under the vector-ALU ablation; option fuse_first = 0 keeps the
  // two launches).
  bool fuse_first = false;
  bnn::ConvGeom g_first;
  if (n_layers > 1 && layers[0].kind == BNN_LAYER_FCONV_BINW &&
      layers[1].kind == BNN_LAYER_BCONV) {
    const bnn_layer& l0 = layers[0];
    const bnn_layer& l1 = layers[1];
    bnn_conv_desc d0{batch, H, W, l0.C, l0.F, l0.KH, l0.KW, l0.stride, l0.pad, l0.pool};
    bnn::ConvGeom g1;
    if (conv_geom(&d0, &g_first) == BNN_OK) {  // (the chain is validated above)
      bnn_conv_desc d1{batch, g_first.Hp, g_first.Wp, l1.C, l1.F,
                       l1.KH, l1.KW, l1.stride, l1.pad, l1.pool};
      // Fused at every batch size (one image of 32 x 32: 38.6 us per
      // forward fused, 41.0 us as two launches).
      fuse_first = g_opt.fuse_first != 0 && conv_geom(&d1, &g1) == BNN_OK &&
                   use_mfma(g1) && bnn::fconv_bconv_supported(g_first, g1);
    }
  }
  int cur = 0;  // buffer holding the current packed activations
  int64_t h = H, w = W, c = C;
  for (int32_t li = 0; li < n_layers; ++li) {
    const bnn_layer& l = layers[li];
    uint32_t* dst = buf[li == 0 ? 0 : cur ^ 1];
    const uint32_t* src = buf[cur];
    hipError_t e = hipSuccess;
    switch (l.kind) {
      case BNN_LAYER_INPUT_THRESHOLD:
      case BNN_LAYER_INPUT_GRAY:
      case BNN_LAYER_INPUT_LBP:
        if (!fuse_input) {
          if (l.kind == BNN_LAYER_INPUT_THRESHOLD)
            e = bnn::launch_pack_bits(input, l.offset, int64_t{batch} * h * w, c, dst, stream);
          else
            e = bnn::launch_binarize(mode, input, l.offset, batch, static_cast<int32_t>(h),
                                     static_cast<int32_t>(w), static_cast<int32_t>(c), dst,
                                     stream);
        }
        c = bnn::input_channels_of(mode, static_cast<int>(c));
        break;
      case BNN_LAYER_FCONV_BINW:
      case BNN_LAYER_BCONV: {
        bnn_conv_desc d{batch, static_cast<int32_t>(h), static_cast<int32_t>(w), l.C, l.F,
                        l.KH, l.KW, l.stride, l.pad, l.pool};
        bnn::ConvGeom g;
        conv_geom(&d, &g);
        // Two 3x3 binary convs on a 16-pixel-wide map that fit one kernel
        // run as one, the first conv's bits kept in LDS (a matrix-core
        // kernel, so not under the vector-ALU ablation; option fuse_pair = 0
        // launches them apart).
        const bool handled = (li == 1 && (fuse_first || fuse_input || fuse_input3)) ||
                             (li == 2 && fuse_input3);
        bnn::ConvGeom g2;
        bool pair = false;
        if (!handled && l.kind == BNN_LAYER_BCONV && g_opt.fuse_pair != 0 &&
            li + 1 < n_layers && layers[li + 1].kind == BNN_LAYER_BCONV && use_mfma(g)) {
          const bnn_layer& l2 = layers[li + 1];
          bnn_conv_desc d2{batch, g.Hp, g.Wp, l2.C, l2.F, l2.KH, l2.KW, l2.stride, l2.pad, l2.pool};
          pair = conv_geom(&d2, &g2) == BNN_OK && use_mfma(g2) &&
                 bnn::bconv_bconv_supported(g, g2);
        }
        if (pair) {
          const bnn_layer& l2 = layers[li + 1];
          e = bnn::launch_bconv_bconv(g, g2, src, l.w, l.thr, l.flip, l2.w, l2.thr, l2.flip, dst,
                                      stream);
          if (e != hipSuccess) return fail(BNN_ERR_HIP, "forward: layers %d-%d launch: %s", li,
                                           li + 1, hipGetErrorString(e));
          h = g2.Hp;
          w = g2.Wp;
          c = l2.F;
          ++li;  // the pair's second conv; its output is in dst
          break;
        }
        if (l.kind == BNN_LAYER_FCONV_BINW) {
          if (!fuse_first)
            e = bnn::launch_fconv_binw(g, input, l.w, l.thr, l.flip, nullptr, dst, stream);
        } else if (li == 1 && fuse_first) {
          e = bnn::launch_fconv_bconv(g_first, g, input, layers[0].w, layers[0].thr,
                                      layers[0].flip, l.w, l.wprep, l.thr, l.flip, dst, stream);
        } else if (li == 1 && fuse_input3) {
          // (computed with layer 2)
        } else if (li == 2 && fuse_input3) {
          e = bnn::launch_input_bconv_bconv(g_in1, g, input, layers[0].offset, layers[1].w,
                                            layers[1].thr, layers[1].flip, l.w, l.wprep, l.thr,
                                            l.flip, dst, stream);
        } else if (li == 1 && fuse_input)
          e = bnn::launch_bconv_patch(g, mode, input, layers[0].offset, l.w, l.thr, l.flip,
                                      nullptr, dst, stream);
        else
          e = launch_conv(g, src, l.w, l.wprep, l.thr, l.flip, nullptr, dst, stream);
        h = g.Hp;
        w = g.Wp;
        c = l.F;
        break;
      }
      case BNN_LAYER_BFC: {
        // A run of small FC layers from here on goes to one chained kernel.
        const int run = fc_chain_run(layers, li, n_layers, batch);
        if (run > 1) {
          bnn::FcChainLayer fl[bnn::kFcChainMax];
          for (int i = 0; i < run; ++i) {
            const bnn_layer& q = layers[li + i];
            const bool lg = q.kind == BNN_LAYER_BFC_LOGITS;
            fl[i] = bnn::FcChainLayer{q.w, lg ? nullptr : q.thr, lg ? nullptr : q.flip, q.K, q.N};
          }
          const bool to_logits = layers[li + run - 1].kind == BNN_LAYER_BFC_LOGITS;
          e = bnn::launch_bfc_chain(fl, run, batch, src, to_logits ? nullptr : dst,
                                    to_logits ? logits : nullptr, stream);
          if (e != hipSuccess) return fail(BNN_ERR_HIP, "forward: layers %d-%d launch: %s", li,
                                           li + run - 1, hipGetErrorString(e));
          h = w = 1;
          c = layers[li + run - 1].N;
          li += run - 1;  // the run's last layer; its output is in dst
          break;
        }
        // Two FC layers, the second with at most 32 outputs (often the
        // logits), as one launch of the FC kernel over the first layer's
        // output tiles, which add the second layer's partial sums into
        // atomic accumulators in the workspace (bfc_gemm.hip).  A
        // matrix-core kernel, so not under the vector-ALU ablation; option
        // fuse_pair = 0 launches them apart.
        if (g_opt.fuse_pair != 0 && g_opt.algo != BNN_ALGO_VALU && li + 1 < n_layers &&
            (layers[li + 1].kind == BNN_LAYER_BFC || layers[li + 1].kind == BNN_LAYER_BFC_LOGITS) &&
            layers[li + 1].K == l.N && bnn::bfc_tail_supported(batch, l.K, l.N, layers[li + 1].N)) {
          const bnn_layer& l2 = layers[li + 1];
          const bool lg = l2.kind == BNN_LAYER_BFC_LOGITS;
          e = bnn::launch_bfc_tail(batch, l.K, l.N, l2.N, src, l.w, l.thr, l.flip, l2.w,
                                   lg ? nullptr : l2.thr, lg ? nullptr : l2.flip,
                                   lg ? logits : nullptr, lg ? nullptr : dst, tail_accum, stream);
          if (e != hipSuccess) return fail(BNN_ERR_HIP, "forward: layers %d-%d launch: %s", li,
                                           li + 1, hipGetErrorString(e));
          h = w = 1;
          c = l2.N;
          ++li;  // the pair's second layer; its output is in dst (or the logits)
          break;
        }
        // Two FC layers that fit one kernel (the second with at most 32
        // outputs, often the logits) run as one, the first layer's bits kept
        // in LDS, where the GEMM path would take them (rows above
        // gemv_max_rows; the GEMVs are faster below: 1024 -> 1024 -> 10 at one
        // row 5.2 us as two GEMVs, 7.4 us fused; at 64 rows 8.6 us as two
        // GEMMs, 7.45 us fused).  A matrix-core kernel, so not under the
        // vector-ALU ablation; option fuse_pair = 0 launches them apart.
        if (g_opt.fuse_pair != 0 && g_opt.algo != BNN_ALGO_VALU && batch > g_opt.gemv_max_rows &&
            li + 1 < n_layers &&
            (layers[li + 1].kind == BNN_LAYER_BFC || layers[li + 1].kind == BNN_LAYER_BFC_LOGITS) &&
            layers[li + 1].K == l.N && bnn::bfc_pair_supported(batch, l.K, l.N, layers[li + 1].N)) {
          const bnn_layer& l2 = layers[li + 1];
          const bool lg = l2.kind == BNN_LAYER_BFC_LOGITS;
          e = bnn::launch_bfc_pair(batch, l.K, l.N, l2.N, src, l.w, l.thr, l.flip, l2.w,
                                   lg ? nullptr : l2.thr, lg ? nullptr : l2.flip,
                                   lg ? logits : nullptr, lg ? nullptr : dst, stream);
          if (e != hipSuccess) return fail(BNN_ERR_HIP, "forward: layers %d-%d launch: %s", li,
                                           li + 1, hipGetErrorString(e));
          h = w = 1;
          c = l2.N;
          ++li;  // the pair's second layer; its output is in dst (or the logits)
          break;
        }
        st = gemm_launch(batch, l.N, l.K, src, l.w, l.thr, l.flip, nullptr, dst, stream);
        if (st != BNN_OK) return fail(st, "forward: layer %d: %s", li, g_err);
        h = w = 1;
        c = l.N;
        break;
      }
      case BNN_LAYER_BFC_LOGITS: {
        st = gemm_launch(batch, l.N, l.K, src, l.w, nullptr, nullptr, logits, nullptr, stream);
        if (st != BNN_OK) return fail(st, "forward: layer %d: %s", li, g_err);
        break;
      }
    }
    if (e != hipSuccess) return fail(BNN_ERR_HIP, "forward: layer %d launch: %s", li,
                                     hipGetErrorString(e));
    cur = (li == 0) ? 0 : cur ^ 1;
  }
  return ok();
}

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mu;

// The current device's copy of `scratch`; the stream must belong to it.
bnn_status scratch_of_device(hipStream_t stream, void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e, "forward_noalloc: hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(BNN_ERR_UNSUPPORTED, "forward_noalloc: device %d beyond the %d supported", dev,
                kMaxDevices);
  if (stream) {
    hipDevice_t sdev = -1;
    e = hipStreamGetDevice(stream, &sdev);
    if (e != hipSuccess) return hip_status(e, "forward_noalloc: hipStreamGetDevice");
    if (sdev != dev)
      return fail(BNN_ERR_UNSUPPORTED,
                  "forward_noalloc: the stream belongs to device %d but device %d is current",
                  static_cast<int>(sdev), dev);
  }
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (!p) {
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess) return hip_status(e, "forward_noalloc: hipGetSymbolAddress");
      if (!p || (reinterpret_cast<uintptr_t>(p) % kAlign) != 0)
        return fail(BNN_ERR_HIP, "forward_noalloc: bad scratch address %p", p);
      g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return BNN_OK;
}

}  // namespace

extern "C" {

bnn_status bnn_forward(const bnn_layer* layers, int32_t n_layers, int32_t batch,
                       int32_t H, int32_t W, int32_t C, const float* input,
                       void* workspace, size_t ws_bytes, int32_t* logits,
                       hipStream_t stream) {
  try {
    WsPlan plan;
    bnn_status st = plan_chain(layers, n_layers, batch, H, W, C, &plan);
    if (st != BNN_OK) return st;
    if (!input || !logits || !workspace)
      return fail(BNN_ERR_NULL, "forward: input, logits and workspace must be non-NULL");
    if (!aligned16(input) || !aligned16(logits) ||
        (reinterpret_cast<uintptr_t>(workspace) % kAlign) != 0)
      return fail(BNN_ERR_ALIGN,
                  "forward: input/logits must be 16-byte aligned, workspace 256-byte aligned");
    if (ws_bytes < plan.total())
      return fail(BNN_ERR_WORKSPACE, "forward: workspace of %zu bytes, need %zu", ws_bytes,
                  plan.total());
    return run_chain(layers, n_layers, batch, H, W, C, input, workspace, plan, logits, stream);
  } catch (...) {
    return fail(BNN_ERR_HIP, "forward: unexpected C++ exception");
  }
}

bnn_status bnn_forward_noalloc(const bnn_layer* layers, int32_t n_layers, int32_t batch,
                               int32_t H, int32_t W, int32_t C, const float* input,
                               int32_t* logits, hipStream_t stream) {
  try {
    WsPlan plan;
    bnn_status st = plan_chain(layers, n_layers, batch, H, W, C, &plan);
    if (st != BNN_OK) return st;
    if (!input || !logits)
      return fail(BNN_ERR_NULL, "forward_noalloc: input and logits must be non-NULL");
    if (!aligned16(input) || !aligned16(logits))
      return fail(BNN_ERR_ALIGN, "forward_noalloc: input/logits must be 16-byte aligned");
    if (plan.total() > kScratchBytes)
      return fail(BNN_ERR_WORKSPACE,
                  "forward_noalloc: the chain needs %zu bytes of workspace, more than the %zu "
                  "of the library's scratch array (use bnn_forward with a workspace)",
                  plan.total(), kScratchBytes);
    void* ws = nullptr;
    st = scratch_of_device(stream, &ws);
    if (st != BNN_OK) return st;
    return run_chain(layers, n_layers, batch, H, W, C, input, ws, plan, logits, stream);
  } catch (...) {
    return fail(BNN_ERR_HIP, "forward_noalloc: unexpected C++ exception");
  }
}

}  // extern "C"
