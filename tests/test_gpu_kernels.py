"""GPU parity of the HIP kernels against the CPU oracle (bit-exact).

Inputs are seeded +-1 tensors; the GPU gets them packed by bnn_pack_bits, the
oracle gets the +-1 int8 arrays.  Expected output bits are the oracle's +-1
outputs packed with the oracle's Eq. (2) routine.  Sizes span several tiles
and ragged tails; full-size configurations are checked on sampled outputs.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_1808_00209_amd import bnn, synth
from paper_1808_00209_amd.device import pack_flips, pack_pm1, to_device, words_u32

pytestmark = pytest.mark.gpu

# Kernel families: "auto" takes the fp4 matrix-core kernel wherever the shape
# allows it (C a multiple of 64, at most 32 taps), "valu" forces the
# XOR-popcount vector kernels everywhere, "lds" is "auto" with 2-word chunks
# and the weights staged through LDS wherever no K split is used (by default
# only large grids do that; small grids with C % 256 == 0 take 8-word chunks),
# "early" is "auto" with the thresholds staged at kernel start (by default
# only grids of more than 2 waves per SIMD do that), "grid2d" is "auto" with
# the matrix-core workgroups on a 2-D grid (pixel blocks x filter tiles)
# instead of the one-dimensional XCD order; "prep" is "auto" with the conv
# weights in the prepared operand form (bnn_bconv2d_prepared), and
# "prep_early2d" that with early thresholds on the 2-D grid; "prep_xcdsplit"
# is "prep" with the filter tiles split over XCD groups where that cuts the
# bytes the L2s move (option xcd_order = 2).
ALGOS = ["auto", "valu", "lds", "early", "grid2d", "prep", "prep_early2d", "prep_xcdsplit"]
_PREP = False  # whether _run_conv passes prepared weights


@pytest.fixture(params=ALGOS)
def algo(request):
    global _PREP
    bnn.bnn_set_options(**{"auto": {}, "valu": dict(algo=bnn.ALGO_VALU),
                           "lds": dict(lds_weights=1), "early": dict(late_thresholds=0),
                           "grid2d": dict(xcd_order=0), "prep": {},
                           "prep_early2d": dict(late_thresholds=0, xcd_order=0),
                           "prep_xcdsplit": dict(xcd_order=2)}[request.param])
    _PREP = request.param.startswith("prep")
    yield request.param
    _PREP = False


def _pm1(rng, shape):
    return (rng.integers(0, 2, size=shape) * 2 - 1).astype(np.int8)


def _garble_tails(words_t, bits_valid):
    """OR random garbage into the tail bits of every last word (in place)."""
    r = bits_valid % 32
    if r == 0:
        return words_t
    g = torch.Generator(device="cpu").manual_seed(99)
    junk = torch.randint(0, 2 ** 31 - 1, words_t[..., -1].shape, generator=g, dtype=torch.int64)
    tail = (1 << (32 - r)) - 1
    words_t[..., -1] |= (junk & tail).to(torch.int32).to(words_t.device)
    return words_t


# ------------------------------------------------------------------ pack ---
@pytest.mark.parametrize("D", [1, 3, 31, 32, 33, 63, 64, 65, 100, 4100])
@pytest.mark.parametrize("with_offset", [False, True])
def test_pack_bits_matches_oracle(D, with_offset):
    rng = np.random.default_rng(1000 + D)
    rows = 37
    x = rng.standard_normal((rows, D)).astype(np.float32)
    x[0, : min(D, 4)] = [0.0, -0.0, 1e-45, -1e-45][: min(D, 4)]  # ties and denormals
    x[1] = np.round(x[1] * 4) / 4
    off = None
    if with_offset:
        off = np.round(rng.standard_normal(D) * 4).astype(np.float32) / 4
        x[2] = -off  # x + T == 0 exactly -> bit 0
    got = words_u32(bnn.bnn_pack_bits(to_device(x), None if off is None else to_device(off)))
    ref = oracle.pack_eq2(oracle.sign(x, off))
    assert np.array_equal(got, ref)


def test_pack_bits_rgb_thresholding_ties():
    # Sec. II-C on integer pixels with integer offsets: exact ties occur.
    g = synth.rng(4, 90, 0)
    x = synth.pixels(g, (3, 96, 96, 3))
    T = synth.rgb_offsets(synth.rng(4, 0, 1), 3)
    got = words_u32(bnn.bnn_pack_bits(to_device(x), to_device(T)))
    ref = oracle.pack_eq2(oracle.sign(x, T))
    assert got.shape == (3, 96, 96, 1)
    assert np.array_equal(got, ref)


def test_pack_bits_zero_rows():
    x = torch.empty((0, 64), dtype=torch.float32, device="cuda")
    out = bnn.bnn_pack_bits(x)
    assert out.shape == (0, 2)


# ------------------------------------------------------------------ conv ---
def _run_conv(x, L, pool, want_sums=True, want_bits=True, garble=False):
    N, H, W, C = x.shape
    F, KH, KW, _ = L["w"].shape
    desc = bnn.conv_desc(N, H, W, C, F, KH, KW, 1, L["pad"], pool)
    xd, wd = pack_pm1(x), pack_pm1(L["w"])
    if garble:
        _garble_tails(xd, C)
        _garble_tails(wd, C)
    thr = to_device(L["thr"], torch.int32)
    flip = pack_flips(L["flip"])
    if _PREP:
        wp = bnn.bnn_prepare_weights(wd, F, KH, KW, C)
        sums, bits = bnn.bnn_bconv2d_prepared(desc, xd, wd, wp, thr, flip, want_sums=want_sums,
                                              want_bits=want_bits)
    else:
        sums, bits = bnn.bnn_bconv2d(desc, xd, wd, thr, flip, want_sums=want_sums,
                                     want_bits=want_bits)
    torch.cuda.synchronize()
    return sums, bits


def _oracle_conv(x, L, pool):
    S = oracle.conv2d(x, L["w"], 1, L["pad"])
    b = oracle.threshold(S, L["thr"], L["flip"])
    if pool:
        b = oracle.maxpool2(b)
    return S, oracle.pack_eq2(b)


def test_cfg1_single_conv_bit_exact(algo):
    x, L = synth.cfg1_input(), synth.cfg1_layer()
    sums, bits = _run_conv(x, L, 0)
    S, B = _oracle_conv(x, L, 0)
    assert np.array_equal(sums.cpu().numpy(), S)
    assert np.array_equal(words_u32(bits), B)


CONV_CASES = [
    # N, H, W, C, F, k, pad, pool
    (2, 7, 7, 3, 64, 3, 1, 0),
    (1, 32, 32, 33, 32, 3, 1, 2),
    (3, 2, 2, 64, 40, 3, 1, 0),
    (1, 1, 1, 96, 32, 3, 1, 0),
    (2, 7, 9, 128, 96, 3, 1, 2),
    (1, 32, 7, 32, 64, 1, 0, 0),
    (2, 7, 7, 96, 33, 1, 0, 2),
    (1, 9, 11, 256, 64, 3, 1, 2),
    (1, 5, 6, 512, 32, 3, 0, 0),
    (4, 6, 6, 3, 10, 3, 1, 2),
    (1, 8, 8, 320, 64, 3, 1, 0),
    # shapes the matrix-core kernel takes (C % 128 == 0, F % 64 == 0)
    (2, 9, 7, 128, 64, 3, 1, 0),
    (1, 16, 16, 128, 128, 3, 1, 2),
    (3, 5, 7, 256, 64, 3, 1, 2),
    (1, 6, 6, 256, 192, 3, 0, 0),
    (2, 4, 4, 512, 128, 3, 1, 0),
    (1, 7, 9, 512, 64, 3, 1, 2),
    (1, 3, 3, 1024, 64, 3, 1, 0),
    (2, 11, 5, 384, 64, 1, 0, 0),
    (1, 1, 1, 128, 64, 3, 1, 0),
    (2, 5, 5, 128, 96, 3, 1, 2),
    (1, 12, 12, 256, 32, 3, 1, 0),
    (64, 8, 8, 512, 512, 3, 1, 2),
    # filter counts that are not a multiple of 32 on the matrix-core path
    (2, 6, 6, 64, 10, 3, 1, 2),
    (1, 5, 5, 128, 40, 3, 1, 0),
    (3, 4, 7, 192, 70, 1, 0, 0),
    # C >= 64 but not a multiple of 64 on the matrix-core path: words past a
    # pixel's last one and the last word's tail bits are zeroed (even and odd
    # word counts, 3x3 and 1x1, pooled)
    (2, 9, 9, 100, 64, 3, 1, 2),
    (1, 7, 5, 65, 96, 3, 1, 0),
    (1, 6, 6, 130, 32, 3, 0, 0),
    (3, 5, 5, 200, 128, 1, 0, 2),
    # 32 <= C < 64 on the matrix-core path: one word per tap padded to a
    # 2-word chunk (C = 32), or a masked second word (C = 48, 63); 5x5
    # windows as in Table II's second conv, a 1x1 and a single pixel
    (1, 48, 48, 32, 32, 5, 2, 2),
    (2, 13, 11, 32, 40, 5, 2, 0),
    (3, 9, 9, 48, 64, 3, 1, 2),
    (1, 7, 6, 63, 96, 5, 2, 0),
    (2, 10, 10, 32, 128, 1, 0, 2),
    (1, 1, 1, 32, 32, 5, 2, 0),
    # grids in the XCD order whose pixel blocks are not a multiple of 8, so
    # padding workgroups run with no valid pixel: a K split over 36 blocks,
    # 36 blocks of 4 waves, and 23 pooled blocks with a ragged last one
    (1, 48, 48, 128, 128, 3, 1, 0),
    (1, 96, 96, 64, 1024, 1, 0, 0),
    (2, 40, 72, 64, 1024, 1, 0, 2),
]


@pytest.mark.parametrize("case", CONV_CASES, ids=[str(c) for c in CONV_CASES])
@pytest.mark.parametrize("garble", [False, True])
def test_bconv_shapes_bit_exact(case, garble, algo):
    N, H, W, C, F, k, pad, pool = case
    rng = np.random.default_rng(hash(case) % 2 ** 32)
    x = _pm1(rng, (N, H, W, C))
    K = k * k * C
    L = dict(w=_pm1(rng, (F, k, k, C)), pad=pad,
             thr=rng.integers(-2 * int(np.sqrt(K)), 2 * int(np.sqrt(K)) + 1, F).astype(np.int32),
             flip=rng.integers(0, 2, F).astype(np.uint8))
    sums, bits = _run_conv(x, L, pool, garble=garble)
    S, B = _oracle_conv(x, L, pool)
    assert np.array_equal(sums.cpu().numpy(), S)
    assert np.array_equal(words_u32(bits), B)


@pytest.mark.parametrize("C", [64, 128])
def test_bconv_bits_only_and_sums_only_agree(C, algo):
    rng = np.random.default_rng(5)
    x = _pm1(rng, (2, 12, 10, C))
    L = dict(w=_pm1(rng, (64, 3, 3, C)), pad=1, thr=rng.integers(-20, 21, 64).astype(np.int32),
             flip=rng.integers(0, 2, 64).astype(np.uint8))
    s1, b1 = _run_conv(x, L, 2)
    _, b2 = _run_conv(x, L, 2, want_sums=False)
    s3, _ = _run_conv(x, L, 2, want_bits=False)
    assert torch.equal(b1, b2) and torch.equal(s1, s3)


@pytest.mark.parametrize("C,F", [(32, 32), (128, 64)])
def test_bconv_threshold_ties_exact(C, F, algo):
    # thr equal to the actual sums: every output is a tie -> bit = 1 ^ flip.
    rng = np.random.default_rng(6)
    x = _pm1(rng, (1, 4, 4, C))
    w = _pm1(rng, (F, 3, 3, C))
    S = oracle.conv2d(x, w, 1, 1)
    thr = S[0, 1, 1, :].astype(np.int32)
    flip = rng.integers(0, 2, F).astype(np.uint8)
    L = dict(w=w, pad=1, thr=thr, flip=flip)
    _, bits = _run_conv(x, L, 0)
    _, B = _oracle_conv(x, L, 0)
    assert np.array_equal(words_u32(bits), B)
    expect = oracle.pack_eq2(np.where(flip == 0, 1, -1).astype(np.int8)[None])[0]
    assert np.array_equal(words_u32(bits)[0, 1, 1], expect)


@pytest.mark.parametrize("C,F", [(64, 32), (128, 64)])
def test_bconv_extreme_thresholds(C, F, algo):
    rng = np.random.default_rng(8)
    x = _pm1(rng, (1, 5, 5, C))
    thr = np.array(([-2 ** 31, 2 ** 31 - 1, 0, 1, -1, 9 * C, -9 * C, 9 * C + 1] * F)[:F], np.int32)
    L = dict(w=_pm1(rng, (F, 3, 3, C)), pad=1, thr=thr, flip=rng.integers(0, 2, F).astype(np.uint8))
    _, bits = _run_conv(x, L, 0)
    _, B = _oracle_conv(x, L, 0)
    assert np.array_equal(words_u32(bits), B)


@pytest.mark.parametrize("C", [64, 256])
def test_bconv_odd_pool_sizes_keep_all_sums(C, algo):
    rng = np.random.default_rng(7)
    x = _pm1(rng, (2, 7, 9, C))
    L = dict(w=_pm1(rng, (64, 3, 3, C)), pad=1, thr=rng.integers(-9, 10, 64).astype(np.int32),
             flip=rng.integers(0, 2, 64).astype(np.uint8))
    sums, bits = _run_conv(x, L, 2)
    S, B = _oracle_conv(x, L, 2)
    assert sums.shape == (2, 7, 9, 64) and bits.shape == (2, 3, 4, 2)
    assert np.array_equal(sums.cpu().numpy(), S)
    assert np.array_equal(words_u32(bits), B)


def test_bconv_deterministic_repeat(algo):
    x, L = synth.cfg5_case("A", N=2)
    s1, b1 = _run_conv(x, L, 0)
    s2, b2 = _run_conv(x, L, 0)
    assert torch.equal(s1, s2) and torch.equal(b1, b2)


# ------------------------------------------------------------------ GEMM ---
def _run_gemm(a, L, garble=False):
    M, K = a.shape
    A, B = pack_pm1(a), pack_pm1(L["w"])
    if garble:
        _garble_tails(A, K)
        _garble_tails(B, K)
    thr = to_device(L["thr"], torch.int32)
    flip = pack_flips(L["flip"])
    sums, bits = bnn.bnn_bgemm(A, B, K, thr, flip)
    torch.cuda.synchronize()
    return sums.cpu().numpy(), words_u32(bits)


def _oracle_gemm(a, L):
    S = oracle.fc(a, L["w"])
    return S, oracle.pack_eq2(oracle.threshold(S, L["thr"], L["flip"]))


@pytest.mark.parametrize("K", [4096, 4100])
def test_cfg2_fc_gemm_full_size_bit_exact(K, algo):
    a, L = synth.cfg2(K)
    S, B = _run_gemm(a, L, garble=(K == 4100))
    Sr, Br = _oracle_gemm(a, L)
    assert np.array_equal(S, Sr)
    assert np.array_equal(B, Br)


GEMM_CASES = [(1, 1, 1), (1, 10, 1024), (2, 33, 31), (5, 100, 33), (16, 1024, 8192),
              (3, 40, 100), (64, 96, 4100), (7, 33, 65),
              (16, 64, 4100), (17, 40, 96), (64, 1024, 8192), (100, 70, 1000), (3, 4, 18432),
              (65, 128, 1024), (300, 64, 18432), (64, 192, 128), (64, 10, 1024),
              (40, 50, 128), (64, 33, 8192), (64, 4, 18432), (256, 1024, 8192),
              # K a multiple of 1024, N of 32, at most 512 output tiles: the
              # FC kernel with a workgroup per tile (ragged row tiles, K slices
              # of one chunk, of several chunks and of a short last chunk)
              (3, 32, 1024), (33, 64, 2048), (97, 96, 8192), (40, 32, 18432), (512, 1024, 1024),
              # more than 512 tiles and N a multiple of 64: workgroups of 2 x 2
              # tiles, two waves per tile with half of K each (a ragged second
              # row tile, one with no row in range, K slices of 16, 48, 64 and
              # 80 words); N not a multiple of 64 there stays with the conv
              # kernel
              (100, 6144, 1024), (33, 16384, 1024), (130, 4096, 3072), (256, 4096, 4096),
              (40, 16384, 5120), (600, 1056, 1024),
              # K >= 1024 not a multiple of the K split: rows padded with
              # cleared words and the last word's bits past K cleared (one
              # valid bit, 4, 12, 31), in both forms
              (5, 64, 1025), (70, 96, 4100), (100, 2048, 1100), (64, 4096, 2047),
              (300, 4096, 4100), (600, 1088, 1056),
              # two rows: the FC kernel by default (one row: the GEMV)
              (2, 1024, 8192), (2, 64, 1025), (1, 1024, 8192),
              # N not a multiple of 32 in the FC kernel: a partial last tile
              # (Table II's 18432 -> 100 at 256 rows, N % 4 != 0 with
              # element stores, a K tail, fewer than 32 outputs)
              (256, 100, 18432), (64, 50, 4096), (70, 100, 2047), (40, 1000, 5120),
              (33, 10, 1024), (5, 33, 1025)]


@pytest.mark.parametrize("case", GEMM_CASES, ids=[str(c) for c in GEMM_CASES])
def test_bgemm_shapes_bit_exact(case, algo):
    M, N, K = case
    rng = np.random.default_rng(M * 7919 + N * 31 + K)
    a = _pm1(rng, (M, K))
    L = dict(w=_pm1(rng, (N, K)), thr=rng.integers(-8, 9, N).astype(np.int32),
             flip=rng.integers(0, 2, N).astype(np.uint8))
    S, B = _run_gemm(a, L, garble=True)
    Sr, Br = _oracle_gemm(a, L)
    assert np.array_equal(S, Sr)
    assert np.array_equal(B, Br)


GEMV_CASES = [(1, 1, 1), (2, 33, 31), (3, 100, 33), (5, 1024, 8192), (8, 64, 4100),
              (12, 10, 1024), (16, 1024, 8192), (16, 4, 18432)]


@pytest.mark.parametrize("case", GEMV_CASES, ids=[str(c) for c in GEMV_CASES])
def test_bgemv_all_row_counts_bit_exact(case):
    """The vector-ALU GEMV kernel at every row count it supports (1..16);
    bnn_bgemm sends it only M = 1 by default, option gemv_max_rows = 16 forces it."""
    bnn.bnn_set_options(gemv_max_rows=16)
    M, N, K = case
    rng = np.random.default_rng(M * 7907 + N * 29 + K)
    a = _pm1(rng, (M, K))
    L = dict(w=_pm1(rng, (N, K)), thr=rng.integers(-8, 9, N).astype(np.int32),
             flip=rng.integers(0, 2, N).astype(np.uint8))
    S, B = _run_gemm(a, L, garble=True)
    Sr, Br = _oracle_gemm(a, L)
    assert np.array_equal(S, Sr)
    assert np.array_equal(B, Br)


# ---------------------------------------------------------- fp32 1st layer -
@pytest.mark.parametrize("pool", [0, 2])
@pytest.mark.parametrize("N,H,W,C,F", [(2, 32, 32, 3, 128), (1, 7, 5, 3, 128), (1, 9, 33, 3, 40),
                                       (3, 12, 10, 1, 64), (1, 10, 9, 4, 96), (1, 6, 6, 2, 32)])
def test_fconv_first_layer_exact(pool, N, H, W, C, F, algo):
    rng = np.random.default_rng(N * H + W + 7 * C + F)
    x = synth.dyadic_normal(rng, (N, H, W, C))
    w = _pm1(rng, (F, 3, 3, C))
    thr = rng.integers(-9, 10, F).astype(np.int32)
    flip = rng.integers(0, 2, F).astype(np.uint8)
    desc = bnn.conv_desc(N, H, W, C, F, 3, 3, 1, 1, pool)
    sums, bits = bnn.bnn_fconv2d_binw(desc, to_device(x), pack_pm1(w),
                                      to_device(thr, torch.int32), pack_flips(flip))
    torch.cuda.synchronize()
    S = oracle.fconv2d(x, w, 1, 1)
    b = oracle.threshold(S, thr, flip)
    if pool:
        b = oracle.maxpool2(b)
    assert np.array_equal(sums.cpu().numpy().astype(np.float64), S)
    assert np.array_equal(words_u32(bits), oracle.pack_eq2(b))


def test_fconv_cifar_first_layer_batch64(algo):
    L = synth.cfg3_net()[0]
    x = synth.cfg3_input(64)
    desc = bnn.conv_desc(64, 32, 32, 3, L["F"], 3, 3, 1, 1, 0)
    sums, bits = bnn.bnn_fconv2d_binw(desc, to_device(x), pack_pm1(L["w"]),
                                      to_device(L["thr"], torch.int32), pack_flips(L["flip"]))
    torch.cuda.synchronize()
    S = oracle.fconv2d(x, L["w"], 1, 1)
    assert np.array_equal(sums.cpu().numpy().astype(np.float64), S)
    assert np.array_equal(words_u32(bits), oracle.pack_eq2(oracle.threshold(S, L["thr"], L["flip"])))


# ------------------------------- input binarization and patch-packed conv --
# Sec. II-C / Table III input binarizations and the first conv over them with
# each window packed into ceil(KH*KW*C / 32) words (Algorithm 1's patch
# packing).  Cases: N, H, W, C, F, KH, KW, pad, pool, mode.  Several 8x32
# tiles with ragged edges, odd sizes under pooling (floor), F tails, windows
# of 18 to 121 bits (1 to 4 words, words straddled by a tap's channels), pad
# 0, a one-pixel window of 32 channels, a 32-tap column with F > 256 (two
# rounds of staged filters), and the grayscale and LBP inputs.
T, G, L = 0, 1, 2  # bnn_input_mode
PATCH_CASES = [
    (2, 12, 40, 3, 64, 3, 3, 1, 0, T),
    (1, 17, 35, 3, 64, 3, 3, 1, 2, T),
    (1, 9, 9, 3, 40, 3, 3, 1, 2, T),
    (2, 10, 11, 1, 32, 5, 5, 2, 0, T),
    (1, 8, 70, 2, 96, 3, 3, 0, 0, T),
    (1, 6, 6, 32, 33, 1, 1, 0, 2, T),
    (1, 40, 3, 1, 300, 32, 1, 3, 0, T),
    (2, 20, 37, 3, 32, 5, 5, 2, 2, T),      # 75 bits, 3 words (the paper's first layer)
    (1, 13, 19, 8, 48, 3, 3, 1, 0, T),      # 72 bits
    (1, 15, 15, 2, 40, 7, 7, 3, 0, T),      # 98 bits, 4 words
    (1, 14, 33, 1, 64, 11, 11, 5, 2, T),    # 121 bits
    (2, 12, 40, 1, 64, 3, 3, 1, 0, G),
    (1, 24, 24, 1, 32, 5, 5, 2, 2, G),
    (2, 12, 40, 3, 64, 3, 3, 1, 2, L),
    (1, 24, 35, 3, 32, 5, 5, 2, 2, L),
]


def _binarized(x, off, mode):
    """The oracle's +-1 input for a binarization mode."""
    if mode == T:
        C = x.shape[-1]
        return oracle.sign(x.reshape(-1, C), off).reshape(x.shape)
    if mode == G:
        return oracle.gray_threshold(x, float(off[0]))
    return oracle.lbp(x)


def _patch_case(seed, N, H, W, C, F, KH, KW, mode):
    rng = np.random.default_rng(seed)
    cin = C if mode == T else 3
    x = synth.pixels(rng, (N, H, W, cin))
    off = synth.rgb_offsets(rng, cin if mode == T else 1)
    w = _pm1(rng, (F, KH, KW, C))
    K = KH * KW * C
    thr = rng.integers(-K // 2, K // 2 + 1, size=F).astype(np.int32)
    flip = rng.integers(0, 2, size=F).astype(np.uint8)
    return x, off, w, thr, flip


@pytest.mark.parametrize("case", PATCH_CASES)
def test_bconv_input_patch_bit_exact(case):
    N, H, W, C, F, KH, KW, pad, pool, mode = case
    x, off, w, thr, flip = _patch_case(7 + sum(case), N, H, W, C, F, KH, KW, mode)
    desc = bnn.conv_desc(N, H, W, C, F, KH, KW, 1, pad, pool)
    offd = to_device(off) if mode != L else None
    sums, bits = bnn.bnn_bconv2d_input(desc, mode, to_device(x), offd, pack_pm1(w),
                                       to_device(thr, torch.int32), pack_flips(flip))
    torch.cuda.synchronize()
    S = oracle.conv2d(_binarized(x, off, mode), w, 1, pad)
    b = oracle.threshold(S, thr, flip)
    if pool:
        b = oracle.maxpool2(b)
    assert np.array_equal(sums.cpu().numpy(), S)
    assert np.array_equal(words_u32(bits), oracle.pack_eq2(b))


# Bits-only calls of 3x3 and 5x5 windows over 1 or 3 channels take the
# row-stream kernel (each tile row's codes as one bit stream, window rows cut
# out by funnel shifts); the extra cases add more than 64 filters (all four
# waves binarize), more than 256 (a second round of staged filters), pad 0,
# and the paper's first layer on whole 96 x 96 images.
ROWS_CASES = PATCH_CASES + [
    (1, 19, 45, 3, 100, 5, 5, 2, 2, T),
    (1, 9, 40, 3, 300, 5, 5, 2, 0, T),
    (1, 14, 40, 3, 33, 5, 5, 0, 2, T),
    (1, 30, 33, 1, 70, 5, 5, 2, 0, G),
    (1, 17, 29, 3, 96, 5, 5, 2, 2, L),
    (1, 11, 70, 3, 290, 3, 3, 1, 2, T),
    (2, 96, 96, 3, 32, 5, 5, 2, 2, T),
    (1, 96, 96, 1, 32, 5, 5, 2, 2, G),
]


@pytest.mark.parametrize("case", ROWS_CASES)
def test_bconv_input_bits_only_bit_exact(case):
    N, H, W, C, F, KH, KW, pad, pool, mode = case
    x, off, w, thr, flip = _patch_case(7 + sum(case), N, H, W, C, F, KH, KW, mode)
    desc = bnn.conv_desc(N, H, W, C, F, KH, KW, 1, pad, pool)
    offd = to_device(off) if mode != L else None
    _, bits = bnn.bnn_bconv2d_input(desc, mode, to_device(x), offd, pack_pm1(w),
                                    to_device(thr, torch.int32), pack_flips(flip),
                                    want_sums=False)
    torch.cuda.synchronize()
    b = oracle.threshold(oracle.conv2d(_binarized(x, off, mode), w, 1, pad), thr, flip)
    if pool:
        b = oracle.maxpool2(b)
    assert np.array_equal(words_u32(bits), oracle.pack_eq2(b))


@pytest.mark.parametrize("mode,cin", [(T, 3), (T, 1), (T, 32), (T, 17), (G, 3), (L, 3)])
def test_binarize_input_bit_exact(mode, cin):
    rng = np.random.default_rng(40 + 3 * mode + cin)
    x = synth.pixels(rng, (2, 13, 37, cin))
    off = synth.rgb_offsets(rng, cin if mode == T else 1)
    out = bnn.bnn_binarize_input(mode, to_device(x), to_device(off) if mode != L else None)
    torch.cuda.synchronize()
    assert np.array_equal(words_u32(out), oracle.pack_eq2(_binarized(x, off, mode)))


def test_bconv_input_matches_pack_then_bconv():
    """The fused call equals bnn_pack_bits followed by bnn_bconv2d (bits only,
    no offset), on the vehicle-shaped first layer at batch 8."""
    N, H, W, C, F = 8, 96, 96, 3, 64
    x, _, w, thr, flip = _patch_case(11, N, H, W, C, F, 3, 3, T)
    x = x - 127.0  # thresholds at 0 without an offset
    desc = bnn.conv_desc(N, H, W, C, F, 3, 3, 1, 1, 0)
    xd, wd = to_device(x), pack_pm1(w)
    td, fd = to_device(thr, torch.int32), pack_flips(flip)
    _, fused = bnn.bnn_bconv2d_input(desc, T, xd, None, wd, td, fd, want_sums=False)
    packed = bnn.bnn_pack_bits(xd)
    _, twostep = bnn.bnn_bconv2d(desc, packed, wd, td, fd, want_sums=False)
    torch.cuda.synchronize()
    assert torch.equal(fused, twostep)
    xb = oracle.sign(x[[0, 7]].reshape(-1, C)).reshape((2, H, W, C))
    ref = oracle.pack_eq2(oracle.threshold(oracle.conv2d(xb, w, 1, 1), thr, flip))
    assert np.array_equal(words_u32(fused)[[0, 7]], ref)


# ------------------------------------------------ XCD groups of filters ---
# Grids of >= 8 pixel blocks run in the XCD order; with option xcd_order = 2
# the filter tiles are split over g = 1, 2, 4 or 8 XCD groups chosen from
# the layer's activation, weight and output bytes (tile_grid): these shapes
# span the choices (family "prep_xcdsplit"; the others run them unsplit).
XCD_CASES = [  # N, H, W, C, F, pool
    (8, 16, 16, 512, 512, 2),
    (4, 16, 32, 256, 256, 0),
    (8, 16, 16, 128, 128, 2),
    (16, 16, 16, 64, 64, 0),
    (32, 32, 32, 64, 64, 2),
]


@pytest.mark.parametrize("case", XCD_CASES, ids=[str(c) for c in XCD_CASES])
def test_bconv_xcd_filter_groups_bit_exact(case, algo):
    N, H, W, C, F, pool = case
    rng = np.random.default_rng(N * 100 + C)
    x = _pm1(rng, (N, H, W, C))
    L = dict(w=_pm1(rng, (F, 3, 3, C)), pad=1,
             thr=rng.integers(-3 * int(np.sqrt(9 * C)), 3 * int(np.sqrt(9 * C)) + 1,
                              size=F).astype(np.int32),
             flip=rng.integers(0, 2, size=F).astype(np.uint8))
    sums, bits = _run_conv(x, L, pool)
    S, B = _oracle_conv(x, L, pool)
    assert np.array_equal(sums.cpu().numpy(), S)
    assert np.array_equal(words_u32(bits), B)
    _, bits_only = _run_conv(x, L, pool, want_sums=False)
    assert np.array_equal(words_u32(bits_only), B)


# ---------------------------------------------------- prepared weights ---
@pytest.mark.parametrize("F,KH,KW,C", [(40, 3, 3, 96), (33, 1, 1, 4100), (64, 3, 3, 64),
                                       (32, 5, 5, 32)])
def test_prepared_weights_decode_to_the_packed_weights(F, KH, KW, C):
    """bnn_prepare_weights decoded on the host, independently of the
    kernels: register r, nibble n of word j's entry is the fp4 value of
    channel 32 j + 31 - (4 n + r) (the Eq. 2 bit of that channel), -w for
    r = 3 and +4 w, +2 w, +1 w for r = 0, 1, 2 (w = +-1), 0 past C (garbled
    tail bits ignored) and past F; the trailing offsets are the sums of w
    over the r < 3 positions."""
    rng = np.random.default_rng(F * 1000 + C)
    w = _pm1(rng, (F, KH, KW, C))
    wd = _garble_tails(pack_pm1(w), C)
    prep = bnn.bnn_prepare_weights(wd, F, KH, KW, C)
    torch.cuda.synchronize()
    raw = prep.cpu().numpy()
    Cw = (C + 31) // 32
    Cp = Cw if C % 64 == 0 else (Cw + 7) // 8 * 8
    Fp = (F + 31) // 32 * 32
    n_ent = Fp * KH * KW * Cp
    assert raw.size == bnn.bnn_prepared_weights_size(F, KH, KW, C) >= n_ent * 16 + 4 * F
    # entries [F / 32][tap][word][f % 32][4 registers]
    ent = raw[:n_ent * 16].view(np.uint32).reshape(Fp // 32, KH * KW, Cp, 32, 4)
    ent = ent.transpose(0, 3, 1, 2, 4).reshape(Fp, KH * KW, Cp, 4)
    assert not ent[F:].any()  # filters past F: zero
    ent = ent[:F]
    corr = raw[n_ent * 16:n_ent * 16 + 4 * F].view(np.int32)
    e2m1 = {0x0: 0.0, 0x2: 1.0, 0x4: 2.0, 0x6: 4.0, 0xA: -1.0, 0xC: -2.0, 0xE: -4.0}
    lut = np.full(16, np.nan)
    for k, v in e2m1.items():
        lut[k] = v
    r = np.arange(4)[:, None]
    n = np.arange(8)[None, :]
    nib = (ent[..., :, None] >> (4 * n)) & 0xF               # [F, T, Cp, 4 r, 8 n]
    val = lut[nib]
    assert not np.isnan(val).any()
    ch = 32 * np.arange(Cp)[:, None, None] + 31 - (4 * n + r)  # [Cp, 4, 8]
    wt = np.zeros((F, KH * KW, Cp, 4, 8))
    ok = ch < C
    wf = w.reshape(F, KH * KW, C).astype(np.float64)
    wt[:, :, ok] = wf[:, :, ch[ok]]
    mag = np.array([4.0, 2.0, 1.0, -1.0])[:, None]
    assert np.array_equal(val, wt * mag)
    assert np.array_equal(corr, wt[:, :, :, :3, :].sum(axis=(1, 2, 3, 4)).astype(np.int32))
