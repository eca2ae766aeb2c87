/*
 * CPU oracle for binarized convolutional / fully-connected inference
 * (Khan, Huttunen, Boutellier, "Binarized Convolutional Neural Networks for
 * Efficient Inference on GPUs", EUSIPCO 2018).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or
 * call this file: only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg use it.  It shares no source with the HIP library.
 *
 * Representation: every binary value is an int8_t holding -1 or +1 and every
 * dot product is a plain multiply-accumulate in int32.  There are no bits, no
 * XOR and no popcount here: the oracle is the definition the packed method
 * must reproduce exactly.  The one exception is orc_pack_eq2, which writes
 * out the paper's packing formula (Eq. 2) so that the packing kernel can be
 * checked against it.
 *
 * Readings of the paper taken here (each also listed in the design notes):
 *  - sign(0) = -1 (Eq. 1: -1 for x <= 0).
 *  - Binary layers pad with -1: the paper's shared-memory tile is zero
 *    initialised and then compared with "> 0" (Sec. III-A, Algorithm 1), so a
 *    pad tap reads as -1.  Padded taps count in the dot product.
 *  - The real-valued first layer pads with 0.0.
 *  - Convolution is cross-correlation (the remark after Eq. 3), with the
 *    kernel row index paired with the image row offset.
 *  - The per-channel threshold with flip bit (BatchNorm folded into sign) is
 *    not in the paper: bit = (S >= thr) XOR flip, so S == thr gives 1^flip.
 *  - 2x2 max-pooling over +-1 values, applied after the threshold, floor on
 *    odd sizes (Table II lists pooling; the paper gives no algorithm).
 */
#include <stdint.h>
#include <stddef.h>

/* Eq. (1): deterministic sign, ties (x == 0) go to -1. */
static int8_t sign_pm1(float v) { return v > 0.0f ? (int8_t)1 : (int8_t)-1; }

/*
 * Input binarization by thresholding (Sec. II-C): out = sign(x + T[d]) with
 * the addition done in fp32, the precision of the input.  offset may be NULL
 * (then T = 0, i.e. plain Eq. 1).  x, out: [rows, D] row-major.
 */
void orc_sign(const float* x, const float* offset, int64_t rows, int64_t D,
              int8_t* out) {
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r) {
    for (int64_t d = 0; d < D; ++d) {
      float v = x[r * D + d];
      if (offset) v = v + offset[d];
      out[r * D + d] = sign_pm1(v);
    }
  }
}

/*
 * Eq. (2), packing: the g-th packed value of a row is
 *     sum over i in group g of (1 + x_i) * 2^(B - 2 - ((i - 1) mod B))
 * with i 1-based.  (1 + x_i) is 0 or 2, so the term for m = (i-1) mod B is
 * 2^(B-1-m) for +1 and 0 for -1; it is evaluated here as
 * ((1 + x_i) << (B - 1 - m)) >> 1, which equals the formula exactly also for
 * m = B - 1 where the printed exponent is -1.  The paper assumes D divisible
 * by B; a shorter last group simply has fewer terms, which leaves its missing
 * low positions at 0.  x: [rows, D] of +-1; out: [rows, ceil(D / B)].
 */
void orc_pack_eq2(const int8_t* x, int64_t rows, int64_t D, int32_t B,
                  uint32_t* out) {
  const int64_t groups = (D + B - 1) / B;
  for (int64_t r = 0; r < rows; ++r) {
    for (int64_t g = 0; g < groups; ++g) {
      uint64_t acc = 0;
      for (int64_t i = g * B + 1; i <= (g + 1) * B && i <= D; ++i) {
        const int64_t m = (i - 1) % B;
        const uint64_t one_plus_x = (uint64_t)(1 + x[r * D + (i - 1)]);
        acc += (one_plus_x << (B - 1 - m)) >> 1;
      }
      out[r * groups + g] = (uint32_t)acc;
    }
  }
}

/*
 * Eq. (3) as cross-correlation over +-1 values, generalised to F filters,
 * N images, stride and symmetric padding with pad value -1:
 *   S[n,i,j,f] = sum_{kh,kw,c} w[f,kh,kw,c] * x[n, i*s + kh - p, j*s + kw - p, c]
 * x: [N,H,W,C], w: [F,KH,KW,C] (+-1 int8), out: [N,Ho,Wo,F] int32 with
 * Ho = (H + 2p - KH) / s + 1.
 */
static int32_t conv_at(const int8_t* x, const int8_t* w, int32_t H, int32_t W,
                       int32_t C, int32_t KH, int32_t KW, int32_t stride,
                       int32_t pad, int64_t n, int64_t i, int64_t j, int64_t f) {
  int32_t s = 0;
  for (int32_t kh = 0; kh < KH; ++kh) {
    for (int32_t kw = 0; kw < KW; ++kw) {
      const int64_t hi = i * stride + kh - pad;
      const int64_t wi = j * stride + kw - pad;
      const int inside = hi >= 0 && hi < H && wi >= 0 && wi < W;
      for (int32_t c = 0; c < C; ++c) {
        const int32_t xv =
            inside ? x[((n * H + hi) * W + wi) * C + c] : -1; /* pad = -1 */
        const int32_t wv = w[(((int64_t)f * KH + kh) * KW + kw) * C + c];
        s += wv * xv;
      }
    }
  }
  return s;
}

void orc_conv2d(const int8_t* x, const int8_t* w, int32_t N, int32_t H,
                int32_t W, int32_t C, int32_t F, int32_t KH, int32_t KW,
                int32_t stride, int32_t pad, int32_t* out) {
  const int32_t Ho = (H + 2 * pad - KH) / stride + 1;
  const int32_t Wo = (W + 2 * pad - KW) / stride + 1;
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int64_t n = 0; n < N; ++n) {
    for (int64_t i = 0; i < Ho; ++i) {
      for (int64_t j = 0; j < Wo; ++j) {
        for (int64_t f = 0; f < F; ++f) {
          out[((n * Ho + i) * Wo + j) * F + f] =
              conv_at(x, w, H, W, C, KH, KW, stride, pad, n, i, j, f);
        }
      }
    }
  }
}

/* The same sum at a list of output coordinates idx[k] = (n, i, j, f). */
void orc_conv2d_at(const int8_t* x, const int8_t* w, int32_t H, int32_t W,
                   int32_t C, int32_t KH, int32_t KW, int32_t stride,
                   int32_t pad, const int64_t* idx, int64_t count,
                   int32_t* out) {
#pragma omp parallel for schedule(static)
  for (int64_t k = 0; k < count; ++k) {
    out[k] = conv_at(x, w, H, W, C, KH, KW, stride, pad, idx[4 * k],
                     idx[4 * k + 1], idx[4 * k + 2], idx[4 * k + 3]);
  }
}

/*
 * Real-valued first layer with +-1 weights: cross-correlation (Eq. 3) of an
 * fp32 image with +-1 weights, pad value 0.0, accumulated in fp64.
 * x: [N,H,W,C] fp32, w: [F,KH,KW,C] +-1, out: [N,Ho,Wo,F] fp64.
 */
void orc_fconv2d(const float* x, const int8_t* w, int32_t N, int32_t H,
                 int32_t W, int32_t C, int32_t F, int32_t KH, int32_t KW,
                 int32_t stride, int32_t pad, double* out) {
  const int32_t Ho = (H + 2 * pad - KH) / stride + 1;
  const int32_t Wo = (W + 2 * pad - KW) / stride + 1;
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int64_t n = 0; n < N; ++n) {
    for (int64_t i = 0; i < Ho; ++i) {
      for (int64_t j = 0; j < Wo; ++j) {
        for (int64_t f = 0; f < F; ++f) {
          double s = 0.0;
          for (int32_t kh = 0; kh < KH; ++kh) {
            for (int32_t kw = 0; kw < KW; ++kw) {
              const int64_t hi = i * stride + kh - pad;
              const int64_t wi = j * stride + kw - pad;
              if (hi < 0 || hi >= H || wi < 0 || wi >= W) continue; /* 0.0 */
              for (int32_t c = 0; c < C; ++c) {
                const double xv = (double)x[((n * H + hi) * W + wi) * C + c];
                const double wv =
                    (double)w[((f * KH + kh) * (int64_t)KW + kw) * C + c];
                s += wv * xv;
              }
            }
          }
          out[((n * Ho + i) * Wo + j) * F + f] = s;
        }
      }
    }
  }
}

/*
 * Fully-connected layer (Sec. III-B): S[m,n] = sum_k A[m,k] * B[n,k] over +-1
 * values.  A: [M,K] (activations), B: [N,K] (one weight row per output).
 */
void orc_fc(const int8_t* A, const int8_t* B, int64_t M, int64_t N, int64_t K,
            int32_t* out) {
#pragma omp parallel for collapse(2) schedule(static)
  for (int64_t m = 0; m < M; ++m) {
    for (int64_t n = 0; n < N; ++n) {
      int32_t s = 0;
      for (int64_t k = 0; k < K; ++k) s += (int32_t)A[m * K + k] * B[n * K + k];
      out[m * N + n] = s;
    }
  }
}

/*
 * Folded BatchNorm + sign: bit = (S >= thr[f]) XOR flip[f]; the result is
 * returned as a +-1 value (bit 1 -> +1).  S: [P, F]; flip: 0/1 per channel.
 */
void orc_threshold(const int32_t* S, const int32_t* thr, const uint8_t* flip,
                   int64_t P, int64_t F, int8_t* out) {
#pragma omp parallel for schedule(static)
  for (int64_t p = 0; p < P; ++p) {
    for (int64_t f = 0; f < F; ++f) {
      const int ge = S[p * F + f] >= thr[f];
      const int bit = ge ^ (flip ? (flip[f] & 1) : 0);
      out[p * F + f] = bit ? (int8_t)1 : (int8_t)-1;
    }
  }
}

/* The same threshold for real-valued sums, compared in fp64. */
void orc_threshold_f64(const double* S, const int32_t* thr,
                       const uint8_t* flip, int64_t P, int64_t F,
                       int8_t* out) {
#pragma omp parallel for schedule(static)
  for (int64_t p = 0; p < P; ++p) {
    for (int64_t f = 0; f < F; ++f) {
      const int ge = S[p * F + f] >= (double)thr[f];
      const int bit = ge ^ (flip ? (flip[f] & 1) : 0);
      out[p * F + f] = bit ? (int8_t)1 : (int8_t)-1;
    }
  }
}

/*
 * 2x2 max-pooling with stride 2 over +-1 values (Table II), floor on odd
 * sizes.  x: [N,H,W,C] -> out: [N,H/2,W/2,C].
 */
void orc_maxpool2(const int8_t* x, int32_t N, int32_t H, int32_t W, int32_t C,
                  int8_t* out) {
  const int32_t Hp = H / 2, Wp = W / 2;
#pragma omp parallel for collapse(2) schedule(static)
  for (int64_t n = 0; n < N; ++n) {
    for (int64_t i = 0; i < Hp; ++i) {
      for (int64_t j = 0; j < Wp; ++j) {
        for (int64_t c = 0; c < C; ++c) {
          int8_t m = -1;
          for (int di = 0; di < 2; ++di) {
            for (int dj = 0; dj < 2; ++dj) {
              const int8_t v = x[((n * H + 2 * i + di) * W + 2 * j + dj) * C + c];
              if (v > m) m = v;
            }
          }
          out[((n * Hp + i) * Wp + j) * C + c] = m;
        }
      }
    }
  }
}

/*
 * Grayscale value of an RGB pixel, the input of the grayscale thresholding
 * and of the LBP binarization (Sec. II-C; Table III).  The paper does not give
 * the conversion.  The reading taken is the ITU-R BT.601 luma
 * 0.299 R + 0.587 G + 0.114 B, evaluated in fp32 as (0.299 R + 0.587 G) +
 * 0.114 B with every product rounded to fp32 on its own.  Both the oracle and
 * the kernels use exactly these operations, since the binarization decision
 * depends on their rounding.
 */
static float gray_of(const float* px) {
  const float r = 0.299f * px[0];
  const float g = 0.587f * px[1];
  const float b = 0.114f * px[2];
  const float rg = r + g;
  return rg + b;
}

/*
 * Grayscale thresholding (Table III "Thresholding Grayscale"): one channel,
 * out = sign(gray(x) + T) with the addition in fp32.  x: [rows, 3] RGB;
 * out: [rows] +-1.
 */
void orc_gray_threshold(const float* x, float T, int64_t rows, int8_t* out) {
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r) {
    const float v = gray_of(x + 3 * r) + T;
    out[r] = sign_pm1(v);
  }
}

/*
 * LBP input binarization (Sec. II-C, local binary patterns).  On the
 * grayscale image, the 8 neighbours at radius 1 of a pixel are numbered
 * clockwise from the top-left one:
 *   0: (-1,-1)  1: (-1,0)  2: (-1,+1)  3: (0,+1)
 *   4: (+1,+1)  5: (+1,0)  6: (+1,-1)  7: (0,-1)      (row, column offsets)
 * The three artificial channels take neighbours 0, 3 and 6, a clockwise
 * stride of 3 (the start point is not stated; top-left is the reading taken).
 * A channel is +1 when its neighbour's gray value exceeds the centre's
 * (strictly) and -1 otherwise; a neighbour outside the image never exceeds.
 * x: [N, H, W, 3] RGB; out: [N, H, W, 3] +-1.
 */
void orc_lbp(const float* x, int32_t N, int32_t H, int32_t W, int8_t* out) {
  static const int dr[3] = {-1, 0, 1};
  static const int dc[3] = {-1, 1, -1};
#pragma omp parallel for collapse(2) schedule(static)
  for (int64_t n = 0; n < N; ++n) {
    for (int64_t i = 0; i < H; ++i) {
      for (int64_t j = 0; j < W; ++j) {
        const float centre = gray_of(x + ((n * H + i) * W + j) * 3);
        for (int ch = 0; ch < 3; ++ch) {
          const int64_t ni = i + dr[ch], nj = j + dc[ch];
          int8_t v = -1;
          if (ni >= 0 && ni < H && nj >= 0 && nj < W) {
            const float g = gray_of(x + ((n * H + ni) * W + nj) * 3);
            if (g > centre) v = 1;
          }
          out[((n * H + i) * W + j) * 3 + ch] = v;
        }
      }
    }
  }
}

/* Number of OpenMP threads a parallel region of this library would use. */
int orc_num_threads(void) {
  int n = 1;
#pragma omp parallel
  {
#pragma omp single
    {
#ifdef _OPENMP
      extern int omp_get_num_threads(void);
      n = omp_get_num_threads();
#endif
    }
  }
  return n;
}
