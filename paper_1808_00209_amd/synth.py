"""Seeded synthetic inputs and the workload shapes they are drawn for.

This module generates data only: +-1 tensors, thresholds, flip bits and
real-valued images, from ``numpy.random.default_rng`` with fixed seeds.  It
holds none of the binarized arithmetic (no packing, no dot products), so the
oracle and the HIP path can both consume its arrays without sharing method
code.  Everything is plain numpy on the host.

Seeds: ``1808000 + 1000*cfg + 10*layer + t`` with t = 0 input, 1 weights,
2 thresholds, 3 flips.

Workloads (shapes follow the five benchmark configurations; the paper's own
network is the 5x5 vehicle classifier of Table II, whose dataset and trained
weights are not available, so every tensor here is synthetic):
  1 single 3x3 conv, 64->64 channels at 32x32, batch 1
  2 FC GEMM 256 x 4096 bits x 4096 outputs (and a 4100-bit variant)
  3 CIFAR-shaped net, fp32 first layer, batch 1 and 64
  4 vehicle-shaped net, 96x96 RGB thresholded input, batch 256
  5 large 3x3 convs at batch 64 and a 1x1 256->1024 conv
"""
from __future__ import annotations

import math

import numpy as np

SEED_BASE = 1808000
T_X, T_W, T_THR, T_FLIP = 0, 1, 2, 3


def seed(cfg: int, layer: int, t: int) -> int:
    return SEED_BASE + 1000 * cfg + 10 * layer + t


def rng(cfg: int, layer: int, t: int) -> np.random.Generator:
    return np.random.default_rng(seed(cfg, layer, t))


def pm1(g: np.random.Generator, shape) -> np.ndarray:
    """i.i.d. Bernoulli(0.5) values in {-1, +1} as int8."""
    bits = g.integers(0, 2, size=shape, dtype=np.int8)
    return (bits * 2 - 1).astype(np.int8)


def flips(g: np.random.Generator, n: int) -> np.ndarray:
    """Bernoulli(0.5) flip bits, one uint8 0/1 per channel."""
    return g.integers(0, 2, size=n, dtype=np.uint8)


def thresholds(g: np.random.Generator, n: int, lo: int, hi: int) -> np.ndarray:
    """Integer thresholds uniform on [lo, hi] (both ends included)."""
    return g.integers(lo, hi + 1, size=n, dtype=np.int64).astype(np.int32)


def balanced_range(k: int):
    """[-2 ceil(sqrt K), 2 ceil(sqrt K)]: keeps output bits near balanced."""
    r = 2 * int(math.ceil(math.sqrt(k)))
    return -r, r


def dyadic_normal(g: np.random.Generator, shape, frac_bits: int = 16,
                  limit: float = 8.0) -> np.ndarray:
    """N(0,1) fp32 values rounded to a 2^-frac_bits grid, |x| < limit.

    Sums of up to a few dozen such values are exact in fp32 in any order,
    which makes the real-valued first layer order-independent.
    """
    step = 2.0 ** -frac_bits
    v = g.standard_normal(size=shape)
    v = np.clip(np.round(v / step) * step, -limit + step, limit - step)
    return v.astype(np.float32)


def pixels(g: np.random.Generator, shape) -> np.ndarray:
    """Integer-valued pixels uniform on [0, 255], stored as fp32."""
    return g.integers(0, 256, size=shape, dtype=np.int64).astype(np.float32)


def rgb_offsets(g: np.random.Generator, c: int) -> np.ndarray:
    """Per-channel offsets T_c = -t_c with t_c integer on [64, 191]."""
    return (-g.integers(64, 192, size=c, dtype=np.int64)).astype(np.float32)


# --------------------------------------------------------------------------
# Layer descriptions.  A layer is a dict; binary tensors are +-1 int8.
#   input_threshold: C, offset[C]
#   input_gray:      C (= 3), offset[1]
#   input_lbp:       C (= 3)
#   fconv / bconv:   C, F, KH, KW, pad, pool, w[F,KH,KW,C], thr[F], flip[F]
#   bfc:             K, N, w[N,K], thr[N], flip[N]
#   bfc_logits:      K, N, w[N,K]
# --------------------------------------------------------------------------

def conv_layer(cfg, li, kind, C, F, k=3, pad=1, pool=0, thr_range=None):
    K = k * k * C
    lo, hi = thr_range if thr_range is not None else balanced_range(K)
    return dict(kind=kind, C=C, F=F, KH=k, KW=k, pad=pad, pool=pool, stride=1,
                w=pm1(rng(cfg, li, T_W), (F, k, k, C)),
                thr=thresholds(rng(cfg, li, T_THR), F, lo, hi),
                flip=flips(rng(cfg, li, T_FLIP), F))


def fc_layer(cfg, li, K, N, logits=False, thr_range=None):
    d = dict(kind="bfc_logits" if logits else "bfc", K=K, N=N,
             w=pm1(rng(cfg, li, T_W), (N, K)))
    if not logits:
        lo, hi = thr_range if thr_range is not None else balanced_range(K)
        d["thr"] = thresholds(rng(cfg, li, T_THR), N, lo, hi)
        d["flip"] = flips(rng(cfg, li, T_FLIP), N)
    return d


# Config 1: one binary 3x3 conv, batch 1, 64 ch at 32x32, 64 filters,
# thresholds uniform in [-K/4, K/4] with K = 576.
CFG1 = dict(N=1, H=32, W=32, C=64, F=64, k=3, pad=1)


def cfg1_layer():
    K = 9 * 64
    return conv_layer(1, 0, "bconv", 64, 64, thr_range=(-K // 4, K // 4))


def cfg1_input():
    return pm1(rng(1, 0, T_X), (1, 32, 32, 64))


# Config 2: FC GEMM, M = 256 rows, N = 4096 outputs, K = 4096 or 4100 bits.
def cfg2(K=4096, M=256, N=4096):
    li = 0 if K == 4096 else 1
    a = pm1(rng(2, li, T_X), (M, K))
    layer = fc_layer(2, li, K, N)
    return a, layer


# Config 3: CIFAR-shaped net (fp32 first conv, then binary convs
# 128-128(pool)-256-256(pool)-512-512(pool), FC 8192-1024-1024-10).
def cfg3_net():
    L = [conv_layer(3, 0, "fconv", 3, 128),
         conv_layer(3, 1, "bconv", 128, 128, pool=2),
         conv_layer(3, 2, "bconv", 128, 256),
         conv_layer(3, 3, "bconv", 256, 256, pool=2),
         conv_layer(3, 4, "bconv", 256, 512),
         conv_layer(3, 5, "bconv", 512, 512, pool=2),
         fc_layer(3, 6, 4 * 4 * 512, 1024),
         fc_layer(3, 7, 1024, 1024),
         fc_layer(3, 8, 1024, 10, logits=True)]
    return L


def cfg3_input(batch):
    """fp32 images [batch, 32, 32, 3] on the 2^-16 grid."""
    return dyadic_normal(rng(3, 90, T_X), (batch, 32, 32, 3))


# Config 4: vehicle-shaped net (96x96x3 RGB thresholded per channel, binary
# convs 64-64(pool)-128-128(pool)-256-256(pool)-512(pool), FC 18432-1024-4).
def cfg4_net():
    return [dict(kind="input_threshold", C=3, offset=rgb_offsets(rng(4, 0, T_W), 3)),
            conv_layer(4, 1, "bconv", 3, 64),
            conv_layer(4, 2, "bconv", 64, 64, pool=2),
            conv_layer(4, 3, "bconv", 64, 128),
            conv_layer(4, 4, "bconv", 128, 128, pool=2),
            conv_layer(4, 5, "bconv", 128, 256),
            conv_layer(4, 6, "bconv", 256, 256, pool=2),
            conv_layer(4, 7, "bconv", 256, 512, pool=2),
            fc_layer(4, 8, 6 * 6 * 512, 1024),
            fc_layer(4, 9, 1024, 4, logits=True)]


def cfg4_input(batch):
    return pixels(rng(4, 90, T_X), (batch, 96, 96, 3))


# Config 5: large binary convs at batch 64.
CFG5 = {
    "A": dict(N=64, H=56, W=56, C=256, F=256, k=3, pad=1),
    "B": dict(N=64, H=28, W=28, C=512, F=512, k=3, pad=1),
    "C": dict(N=64, H=56, W=56, C=256, F=1024, k=1, pad=0),
}


def cfg5_case(name, N=None):
    s = dict(CFG5[name])
    if N is not None:
        s["N"] = N
    li = "ABC".index(name)
    layer = conv_layer(5, li, "bconv", s["C"], s["F"], k=s["k"], pad=s["pad"])
    x = pm1(rng(5, li, T_X), (s["N"], s["H"], s["W"], s["C"]))
    return x, layer


# Paper-shaped vehicle classifier (Table II): an input binarization, binary
# convs 32@5x5 + 2x2 pool and 32@5x5 + 2x2 pool, FC 18432 -> 100, then the two
# small FC layers the paper leaves out of Table II (100 -> 100 -> 4; their
# sizes are not given, 100 is the reading).  Input binarizations of Table III:
# "rgb" (per-channel thresholds), "gray" (grayscale threshold) and "lbp".
PAPER_MODES = ("rgb", "gray", "lbp")


def paper_net(mode="rgb"):
    if mode == "rgb":
        first, c = dict(kind="input_threshold", C=3, offset=rgb_offsets(rng(6, 0, T_W), 3)), 3
    elif mode == "gray":
        first, c = dict(kind="input_gray", C=3, offset=rgb_offsets(rng(6, 0, T_W), 1)), 1
    elif mode == "lbp":
        first, c = dict(kind="input_lbp", C=3), 3
    else:
        raise ValueError(mode)
    return [first,
            conv_layer(6, 1, "bconv", c, 32, k=5, pad=2, pool=2),
            conv_layer(6, 2, "bconv", 32, 32, k=5, pad=2, pool=2),
            fc_layer(6, 3, 24 * 24 * 32, 100),
            fc_layer(6, 4, 100, 100),
            fc_layer(6, 5, 100, 4, logits=True)]


def paper_input(batch):
    return pixels(rng(6, 90, T_X), (batch, 96, 96, 3))


def bit_macs_conv(N, Ho, Wo, F, KH, KW, C):
    """Bit multiply-accumulates of one conv layer (padded taps included)."""
    return N * Ho * Wo * F * KH * KW * C
