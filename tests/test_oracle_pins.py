"""Pins of the CPU oracle to things other than itself (CPU only).

Each test ties one oracle function to what the paper or the mathematics fixes:
hand-worked values of Eq. (2), the Eq. (4) XOR-popcount identity, library
routines that compute the same definition (torch conv2d / numpy matmul in
float64, exact for these integers), closed forms at image borders, invariants
and brute force on tiny shapes.
"""
import itertools
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as tF

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _pm1(rng, shape):
    return (rng.integers(0, 2, size=shape) * 2 - 1).astype(np.int8)


def _popcount(v):
    return bin(int(v)).count("1")


# --------------------------------------------------------------- Eq. (1) ----
def test_sign_ties_and_specials():
    x = np.array([[0.0, -0.0, 1e-45, -1e-45, 3.5, -2.0, np.inf, -np.inf, np.nan]],
                 np.float32)
    got = oracle.sign(x)
    assert got.tolist() == [[-1, -1, 1, -1, 1, -1, 1, -1, -1]]


def test_sign_with_offset_thresholding():
    # Sec. II-C: sign(X + T), T per channel; ties at X == -T go to -1.
    x = np.array([[100, 101, 99], [0, 255, 128]], np.float32)
    T = np.array([-100, -100, -128], np.float32)
    got = oracle.sign(x, T)
    assert got.tolist() == [[-1, 1, -1], [-1, 1, -1]]


# --------------------------------------------------------------- Eq. (2) ----
def _golden_x(case):
    if "x" in case:
        return np.array(case["x"], np.int8)
    D = case["D"]
    x = -np.ones(D, np.int8)
    if case["x_plus_at"] == "all":
        x[:] = 1
    else:
        for i in case["x_plus_at"]:
            x[i - 1] = 1
    return x


def test_pack_eq2_hand_worked_golden():
    cases = json.load(open(os.path.join(GOLDEN, "eq2_pack_examples.json")))["cases"]
    for case in cases:
        x = _golden_x(case)[None, :]
        got = oracle.pack_eq2(x, case["B"])[0].tolist()
        assert got == case["words"], case


@pytest.mark.parametrize("D", [1, 3, 31, 32, 33, 63, 64, 65, 100, 4100])
def test_pack_eq2_b32_matches_numpy_packbits(D):
    # B = 32: first element -> most significant bit, a left-aligned short last
    # word.  numpy.packbits(bitorder="big") over the bits padded with zeros to
    # a multiple of 32, read as big-endian uint32, is the same layout.
    rng = np.random.default_rng(D)
    x = _pm1(rng, (7, D))
    bits = (x > 0).astype(np.uint8)
    Dw = (D + 31) // 32
    padded = np.zeros((7, Dw * 32), np.uint8)
    padded[:, :D] = bits
    ref = np.packbits(padded, axis=1, bitorder="big").view(">u4").astype(np.uint32)
    assert np.array_equal(oracle.pack_eq2(x, 32), ref)


@pytest.mark.parametrize("B", [25, 9, 32, 1])
def test_pack_eq2_matches_algorithm1_shift_or(B):
    # Algorithm 1 forms the same word by OR-ing (value > 0) << (B - 1 - i) for
    # the i-th (0-based) element of a group: a second formulation in the paper.
    rng = np.random.default_rng(B)
    D = 3 * B
    x = _pm1(rng, (5, D))
    ref = np.zeros((5, 3), np.uint64)
    for r in range(5):
        for g in range(3):
            v = 0
            for i in range(B):
                s = 1 if x[r, g * B + i] > 0 else 0
                v |= s << (B - 1 - i)
            ref[r, g] = v
    assert np.array_equal(oracle.pack_eq2(x, B).astype(np.uint64), ref)


def test_pack_eq2_popcount_counts_plus_ones():
    rng = np.random.default_rng(7)
    x = _pm1(rng, (50, 97))
    words = oracle.pack_eq2(x, 32)
    pc = np.array([[sum(_popcount(w) for w in row)] for row in words])
    assert np.array_equal(pc[:, 0], (x > 0).sum(1))


# --------------------------------------------------------------- Eq. (4) ----
def _unpack_msb_first(words, nbits):
    """+-1 vector from words, bit (nbits-1-i) -> element i (test helper)."""
    out = np.empty((len(words), nbits), np.int8)
    for r, w in enumerate(words):
        for i in range(nbits):
            out[r, i] = 1 if (int(w) >> (nbits - 1 - i)) & 1 else -1
    return out


def test_eq4_identity_exhaustive_8bit():
    # a . b = W - 2 popcount(a xor b) for every pair of 8-bit words.
    words = np.arange(256)
    V = _unpack_msb_first(words, 8)
    S = oracle.fc(V, V)
    ref = np.array([[8 - 2 * _popcount(a ^ b) for b in words] for a in words])
    assert np.array_equal(S, ref)


def test_eq4_identity_random_32bit_words():
    rng = np.random.default_rng(11)
    wa = rng.integers(0, 2 ** 32, size=300, dtype=np.uint64)
    wb = rng.integers(0, 2 ** 32, size=200, dtype=np.uint64)
    S = oracle.fc(_unpack_msb_first(wa, 32), _unpack_msb_first(wb, 32))
    ref = np.array([[32 - 2 * _popcount(int(a) ^ int(b)) for b in wb] for a in wa])
    assert np.array_equal(S, ref)


def test_eq4_multiword_with_zero_tail():
    # Several words per vector and a short last word whose pad bits are 0 in
    # both operands: the identity holds with W = number of valid bits.
    rng = np.random.default_rng(12)
    for D in (33, 70, 100):
        a = _pm1(rng, (9, D))
        b = _pm1(rng, (6, D))
        pa, pb = oracle.pack_eq2(a, 32), oracle.pack_eq2(b, 32)
        ref = np.array([[D - 2 * sum(_popcount(int(x) ^ int(y))
                                     for x, y in zip(ra, rb)) for rb in pb]
                        for ra in pa])
        assert np.array_equal(oracle.fc(a, b), ref)


# --------------------------------------------------------------- FC ---------
def test_fc_matches_numpy_matmul_f64():
    rng = np.random.default_rng(3)
    for M, N, K in [(1, 1, 1), (3, 5, 7), (17, 33, 100), (64, 40, 4100)]:
        a, b = _pm1(rng, (M, K)), _pm1(rng, (N, K))
        ref = a.astype(np.float64) @ b.astype(np.float64).T
        assert np.array_equal(oracle.fc(a, b), ref.astype(np.int32))


# --------------------------------------------------------------- Eq. (3) ----
def _torch_conv_pm1(x, w, stride, pad):
    """float64 torch conv2d of NHWC +-1 data after padding with -1."""
    xt = torch.from_numpy(x.astype(np.float64)).permute(0, 3, 1, 2)
    wt = torch.from_numpy(w.astype(np.float64)).permute(0, 3, 1, 2)
    xt = tF.pad(xt, (pad, pad, pad, pad), value=-1.0)
    out = tF.conv2d(xt, wt, stride=stride)
    return out.permute(0, 2, 3, 1).numpy()


CONV_SHAPES = [
    # N, H, W, C, F, KH, KW, stride, pad
    (1, 1, 1, 1, 1, 1, 1, 1, 0),
    (2, 5, 7, 3, 4, 3, 3, 1, 1),
    (1, 6, 6, 33, 5, 3, 3, 1, 1),
    (2, 4, 9, 5, 3, 1, 3, 1, 0),
    (1, 7, 5, 2, 3, 5, 3, 1, 2),
    (1, 8, 8, 4, 2, 3, 3, 2, 1),
    (1, 2, 2, 64, 7, 3, 3, 1, 1),
    (3, 3, 3, 1, 2, 3, 3, 1, 0),
    (1, 5, 6, 7, 3, 2, 4, 1, 1),
]


@pytest.mark.parametrize("shape", CONV_SHAPES)
def test_conv_matches_torch_conv2d_f64(shape):
    N, H, W, C, F, KH, KW, stride, pad = shape
    rng = np.random.default_rng(sum(shape))
    x, w = _pm1(rng, (N, H, W, C)), _pm1(rng, (F, KH, KW, C))
    ref = _torch_conv_pm1(x, w, stride, pad)
    got = oracle.conv2d(x, w, stride, pad)
    assert got.shape == ref.shape
    assert np.array_equal(got, ref.astype(np.int32))


def test_conv_bruteforce_python_loops_asymmetric_kernel():
    # Pure-Python loops on a tiny case with a non-symmetric kernel, so a
    # transposed kernel index (kh <-> kw) or a mirrored one (a true
    # convolution instead of cross-correlation) would show.
    rng = np.random.default_rng(5)
    N, H, W, C, F, KH, KW, pad = 1, 4, 5, 2, 2, 3, 2, 1
    x, w = _pm1(rng, (N, H, W, C)), _pm1(rng, (F, KH, KW, C))
    Ho, Wo = H + 2 * pad - KH + 1, W + 2 * pad - KW + 1
    ref = np.zeros((N, Ho, Wo, F), np.int64)
    for n, i, j, f in itertools.product(range(N), range(Ho), range(Wo), range(F)):
        s = 0
        for kh, kw, c in itertools.product(range(KH), range(KW), range(C)):
            r, q = i + kh - pad, j + kw - pad
            v = x[n, r, q, c] if 0 <= r < H and 0 <= q < W else -1
            s += int(w[f, kh, kw, c]) * int(v)
        ref[n, i, j, f] = s
    assert np.array_equal(oracle.conv2d(x, w, 1, pad), ref)


def test_conv_border_closed_form_golden():
    d = json.load(open(os.path.join(GOLDEN, "conv_border_closed_form.json")))
    for case in d["cases"]:
        H, W, C, F, k, pad = (case[n] for n in ("H", "W", "C", "F", "k", "pad"))
        x = np.ones((1, H, W, C), np.int8)
        w = np.ones((F, k, k, C), np.int8)
        S = oracle.conv2d(x, w, 1, pad)
        assert k * k * C == case["K"]
        for i, j, val, _ in case["points"]:
            assert (S[0, i, j, :] == val).all(), (case, i, j)


def test_conv_invariants_parity_bound_negation():
    rng = np.random.default_rng(21)
    x, w = _pm1(rng, (2, 9, 7, 37)), _pm1(rng, (5, 3, 3, 37))
    K = 3 * 3 * 37
    S = oracle.conv2d(x, w, 1, 1)
    assert ((S - K) % 2 == 0).all()                 # S = K mod 2
    assert (np.abs(S) <= K).all()                   # |S| <= K
    assert np.array_equal(oracle.conv2d(x, -w, 1, 0), -oracle.conv2d(x, w, 1, 0))
    # With padding, negating both operands leaves interior outputs unchanged
    # but not border ones (the pad stays -1).
    S2 = oracle.conv2d(-x, -w, 1, 1)
    assert np.array_equal(S2[:, 1:-1, 1:-1], S[:, 1:-1, 1:-1])


def test_conv_1x1_equals_fc():
    rng = np.random.default_rng(4)
    x, w = _pm1(rng, (2, 5, 6, 70)), _pm1(rng, (9, 1, 1, 70))
    S = oracle.conv2d(x, w, 1, 0)
    ref = oracle.fc(x.reshape(-1, 70), w.reshape(9, 70))
    assert np.array_equal(S.reshape(-1, 9), ref)


def test_fc_equals_full_kernel_conv():
    # An FC layer over an NHWC-flattened map is a conv whose kernel covers
    # the whole map with no padding.
    rng = np.random.default_rng(6)
    x, w = _pm1(rng, (3, 4, 5, 6)), _pm1(rng, (7, 4, 5, 6))
    S = oracle.conv2d(x, w, 1, 0)
    assert S.shape == (3, 1, 1, 7)
    ref = oracle.fc(x.reshape(3, -1), w.reshape(7, -1))
    assert np.array_equal(S[:, 0, 0, :], ref)


def test_conv_at_matches_full_conv():
    rng = np.random.default_rng(8)
    x, w = _pm1(rng, (2, 6, 5, 40)), _pm1(rng, (6, 3, 3, 40))
    S = oracle.conv2d(x, w, 1, 1)
    idx = np.stack([rng.integers(0, s, 200) for s in S.shape], 1)
    got = oracle.conv2d_at(x, w, idx, 1, 1)
    assert np.array_equal(got, S[tuple(idx.T)])


# --------------------------------------------------------------- fp32 layer -
def test_fconv_matches_torch_f64_zero_pad():
    rng = np.random.default_rng(9)
    x = rng.standard_normal((2, 6, 5, 3)).astype(np.float32)
    w = _pm1(rng, (4, 3, 3, 3))
    xt = torch.from_numpy(x.astype(np.float64)).permute(0, 3, 1, 2)
    wt = torch.from_numpy(w.astype(np.float64)).permute(0, 3, 1, 2)
    ref = tF.conv2d(xt, wt, padding=1).permute(0, 2, 3, 1).numpy()
    got = oracle.fconv2d(x, w, 1, 1)
    assert np.allclose(got, ref, rtol=0, atol=1e-12)


def test_fconv_exact_on_dyadic_grid_in_fp32_any_order():
    # Inputs on a 2^-16 grid with |x| < 8: every partial sum of 27 terms is a
    # multiple of 2^-16 below 2^8, exact in fp32, so fp32 in reverse order
    # equals the fp64 oracle bit for bit.
    rng = np.random.default_rng(10)
    x = np.clip(np.round(rng.standard_normal((1, 5, 5, 3)) * 65536) / 65536,
                -8 + 2 ** -16, 8 - 2 ** -16).astype(np.float32)
    w = _pm1(rng, (3, 3, 3, 3))
    got = oracle.fconv2d(x, w, 1, 1)
    xp = np.pad(x, ((0, 0), (1, 1), (1, 1), (0, 0)))
    for i, j, f in itertools.product(range(5), range(5), range(3)):
        terms = (xp[0, i:i + 3, j:j + 3, :] * w[f]).astype(np.float32).ravel()
        s = np.float32(0)
        for t in terms[::-1]:
            s = np.float32(s + t)
        assert float(s) == got[0, i, j, f]


# --------------------------------------------------------------- threshold --
def test_threshold_ties_and_flip():
    S = np.array([[5, 5, 4, 6, -3, -3]], np.int32)
    thr = np.array([5, 5, 5, 5, -3, -2], np.int32)
    flip = np.array([0, 1, 0, 1, 0, 0], np.uint8)
    got = oracle.threshold(S, thr, flip)
    # (S >= thr) XOR flip: tie gives 1 (or 0 when flipped).
    assert got.tolist() == [[1, -1, -1, -1, 1, -1]]
    assert oracle.threshold(S, thr).tolist() == [[1, 1, -1, 1, 1, -1]]
    Sf = S.astype(np.float64) + np.array([[0, 0, 0.5, -0.75, 0, 0.999]])
    assert oracle.threshold(Sf, thr, flip).tolist() == [[1, -1, -1, -1, 1, -1]]


def test_threshold_extreme_thresholds():
    S = np.array([[-2 ** 31, 2 ** 31 - 1, 0]], np.int32)
    thr = np.array([-2 ** 31, -2 ** 31, 2 ** 31 - 1], np.int32)
    assert oracle.threshold(S, thr).tolist() == [[1, 1, -1]]


# --------------------------------------------------------------- pooling ----
def test_maxpool_matches_numpy_reshape_max():
    rng = np.random.default_rng(13)
    for (N, H, W, C) in [(2, 4, 6, 3), (1, 5, 7, 33), (1, 1, 3, 2)]:
        x = _pm1(rng, (N, H, W, C))
        Hp, Wp = H // 2, W // 2
        ref = x[:, :2 * Hp, :2 * Wp].reshape(N, Hp, 2, Wp, 2, C).max(axis=(2, 4))
        assert np.array_equal(oracle.maxpool2(x), ref)


# --------------------------------------------------------------- chain ------
def test_forward_chain_matches_torch_composition():
    """A small net through the oracle vs the same chain built from torch ops
    (float64 conv2d with -1 padding, torch.where threshold, max_pool2d,
    NHWC flatten, matmul)."""
    rng = np.random.default_rng(14)
    N = 2
    x = rng.integers(0, 256, size=(N, 8, 8, 3)).astype(np.float32)
    T = -rng.integers(64, 192, size=3).astype(np.float32)

    def conv(C, F, pool):
        return dict(kind="bconv", C=C, F=F, KH=3, KW=3, pad=1, pool=pool,
                    w=_pm1(rng, (F, 3, 3, C)),
                    thr=rng.integers(-6, 7, size=F).astype(np.int32),
                    flip=rng.integers(0, 2, size=F).astype(np.uint8))

    layers = [dict(kind="input_threshold", C=3, offset=T),
              conv(3, 8, 2), conv(8, 16, 2),
              dict(kind="bfc", K=2 * 2 * 16, N=12, w=_pm1(rng, (12, 64)),
                   thr=rng.integers(-4, 5, size=12).astype(np.int32),
                   flip=rng.integers(0, 2, size=12).astype(np.uint8)),
              dict(kind="bfc_logits", K=12, N=5, w=_pm1(rng, (5, 12)))]
    got = oracle.forward(layers, x)

    a = torch.from_numpy(x.astype(np.float64))
    one = torch.ones((), dtype=torch.float64)
    a = torch.where(a + torch.from_numpy(T.astype(np.float64)) > 0, one, -one)
    a = a.permute(0, 3, 1, 2)
    for L in layers[1:3]:
        wt = torch.from_numpy(L["w"].astype(np.float64)).permute(0, 3, 1, 2)
        s = tF.conv2d(tF.pad(a, (1, 1, 1, 1), value=-1.0), wt)
        thr = torch.from_numpy(L["thr"].astype(np.float64)).view(1, -1, 1, 1)
        fl = torch.from_numpy(L["flip"].astype(bool)).view(1, -1, 1, 1)
        bit = (s >= thr) ^ fl
        a = tF.max_pool2d(torch.where(bit, one, -one), 2)
    a = a.permute(0, 2, 3, 1).reshape(N, -1)
    L = layers[3]
    s = a @ torch.from_numpy(L["w"].astype(np.float64)).T
    bit = (s >= torch.from_numpy(L["thr"].astype(np.float64))) ^ \
        torch.from_numpy(L["flip"].astype(bool))
    a = torch.where(bit, one, -one)
    ref = a @ torch.from_numpy(layers[4]["w"].astype(np.float64)).T
    assert np.array_equal(got, ref.numpy().astype(np.int32))


# ------------------------------------------- grayscale and LBP binarization --
# Sec. II-C / Table III: the grayscale-thresholded input (one channel) and the
# LBP input (three channels from the grayscale image).  The grayscale weights
# are the BT.601 luma (a reading; the paper gives none).

def test_gray_threshold_each_weight_on_its_channel_and_sum_one():
    """Pure red / green / blue pixels of value v against thresholds just off
    0.299 v, 0.587 v, 0.114 v, and a gray pixel against v: every weight sits on
    its own channel and the three add up to one."""
    v = 200.0
    for ch, wt in ((0, 0.299), (1, 0.587), (2, 0.114)):
        px = np.zeros((1, 3), np.float32)
        px[0, ch] = v
        assert oracle.gray_threshold(px, -(wt * v) + 0.01)[0, 0] == 1
        assert oracle.gray_threshold(px, -(wt * v) - 0.01)[0, 0] == -1
    g = np.full((2, 3), v, np.float32)
    assert (oracle.gray_threshold(g, -v + 0.01) == 1).all()
    assert (oracle.gray_threshold(g, -v - 0.01) == -1).all()


def test_gray_threshold_tie_is_minus_one_and_shape():
    x = np.zeros((2, 4, 5, 3), np.float32)
    out = oracle.gray_threshold(x, 0.0)
    assert out.shape == (2, 4, 5, 1) and (out == -1).all()


def test_lbp_constant_image_is_all_minus_one():
    x = np.full((2, 5, 7, 3), 77.0, np.float32)
    assert (oracle.lbp(x) == -1).all()


@pytest.mark.parametrize("i,j", [(2, 3), (0, 0), (4, 6), (0, 6), (4, 0), (1, 5)])
def test_lbp_single_bright_pixel_closed_form(i, j):
    """One bright pixel at (i, j) of a dark 5x7 image: exactly the pixels that
    see it as their selected neighbour become +1.  Neighbours are numbered
    clockwise from the top-left; channels take numbers 0, 3, 6, i.e. offsets
    (-1,-1), (0,+1), (+1,-1).  So channel 0 fires at (i+1, j+1), channel 1 at
    (i, j-1) and channel 2 at (i-1, j+1), when inside the image."""
    x = np.zeros((1, 5, 7, 3), np.float32)
    x[0, i, j] = (10.0, 20.0, 30.0)
    out = oracle.lbp(x)
    expect = -np.ones_like(out)
    for ch, (pi, pj) in enumerate([(i + 1, j + 1), (i, j - 1), (i - 1, j + 1)]):
        if 0 <= pi < 5 and 0 <= pj < 7:
            expect[0, pi, pj, ch] = 1
    assert np.array_equal(out, expect)


def test_lbp_single_dark_pixel_sees_every_neighbour_exceed():
    """A dark pixel in a bright image: its own three channels are +1 wherever
    the selected neighbour exists; no other pixel has a brighter neighbour."""
    for (i, j) in [(2, 3), (0, 0), (4, 6)]:
        x = np.full((1, 5, 7, 3), 50.0, np.float32)
        x[0, i, j] = 0.0
        out = oracle.lbp(x)
        expect = -np.ones_like(out)
        for ch, (di, dj) in enumerate([(-1, -1), (0, 1), (1, -1)]):
            if 0 <= i + di < 5 and 0 <= j + dj < 7:
                expect[0, i, j, ch] = 1
        assert np.array_equal(out, expect)


def test_lbp_invariant_to_gain_and_brightness():
    """Comparisons of gray values survive x -> 4x (exact in fp32) and
    x -> x + 16 (integer pixels: distinct gray values differ by >= 0.001)."""
    rng = np.random.default_rng(5)
    x = rng.integers(0, 240, size=(2, 9, 11, 3)).astype(np.float32)
    ref = oracle.lbp(x)
    assert np.array_equal(oracle.lbp(4.0 * x), ref)
    assert np.array_equal(oracle.lbp(x + 16.0), ref)
    assert (ref == 1).any() and (ref == -1).any()


def test_lbp_matches_a_direct_loop_on_a_tiny_image():
    """Brute force over a 3x4 image with float32 gray values computed by numpy
    in the same order: every (pixel, channel) by explicit comparison."""
    rng = np.random.default_rng(6)
    x = rng.integers(0, 256, size=(1, 3, 4, 3)).astype(np.float32)
    f = np.float32
    g = (f(0.299) * x[..., 0] + f(0.587) * x[..., 1]) + f(0.114) * x[..., 2]
    out = oracle.lbp(x)
    for i in range(3):
        for j in range(4):
            for ch, (di, dj) in enumerate([(-1, -1), (0, 1), (1, -1)]):
                ni, nj = i + di, j + dj
                exceed = 0 <= ni < 3 and 0 <= nj < 4 and g[0, ni, nj] > g[0, i, j]
                assert out[0, i, j, ch] == (1 if exceed else -1)


def _torch_gray(x):
    """BT.601 luma in float32, products rounded one by one, then summed as
    (R + G) + B: written here with torch ops, independently of the oracle."""
    f = torch.float32
    r, g, b = x[..., 0], x[..., 1], x[..., 2]
    return (torch.tensor(0.299, dtype=f) * r + torch.tensor(0.587, dtype=f) * g) + \
        torch.tensor(0.114, dtype=f) * b


def _torch_lbp(gray):
    """LBP channels of Sec. II-C from a gray image [N, H, W]: neighbours at
    offsets (-1,-1), (0,+1), (+1,-1) (numbers 0, 3, 6 clockwise from the
    top-left); +1 where the neighbour is strictly brighter, -1 otherwise and
    outside the image.  Built from padded shifted copies."""
    N, H, W = gray.shape
    pad = torch.full((N, H + 2, W + 2), -float("inf"), dtype=gray.dtype)
    pad[:, 1:H + 1, 1:W + 1] = gray
    chans = []
    for di, dj in ((-1, -1), (0, 1), (1, -1)):
        nb = pad[:, 1 + di:1 + di + H, 1 + dj:1 + dj + W]
        chans.append(torch.where(nb > gray, 1.0, -1.0))
    return torch.stack(chans, dim=-1).to(torch.float64)


@pytest.mark.parametrize("mode", ["input_gray", "input_lbp"])
def test_forward_gray_and_lbp_chains_match_torch_composition(mode):
    """Table II's layer order behind the grayscale and LBP binarizations of
    Table III (Sec. II-C): oracle.forward against the same chain composed
    from torch ops with its own grayscale and LBP, so that the chain's input
    dispatch (which binarization, which offset, how many channels) is pinned
    by something other than the HIP path."""
    rng = np.random.default_rng(15 if mode == "input_gray" else 16)
    N, H, W = 2, 10, 12
    x = rng.integers(0, 256, size=(N, H, W, 3)).astype(np.float32)
    T = np.array([-float(rng.integers(64, 192))], np.float32)
    C1 = 1 if mode == "input_gray" else 3
    F1, F2 = 6, 8
    layers = [dict(kind=mode, C=3, offset=T if mode == "input_gray" else None),
              dict(kind="bconv", C=C1, F=F1, KH=5, KW=5, pad=2, pool=2,
                   w=_pm1(rng, (F1, 5, 5, C1)),
                   thr=rng.integers(-5, 6, size=F1).astype(np.int32),
                   flip=rng.integers(0, 2, size=F1).astype(np.uint8)),
              dict(kind="bconv", C=F1, F=F2, KH=3, KW=3, pad=1, pool=0,
                   w=_pm1(rng, (F2, 3, 3, F1)),
                   thr=rng.integers(-6, 7, size=F2).astype(np.int32),
                   flip=rng.integers(0, 2, size=F2).astype(np.uint8)),
              dict(kind="bfc", K=5 * 6 * F2, N=10, w=_pm1(rng, (10, 5 * 6 * F2)),
                   thr=rng.integers(-8, 9, size=10).astype(np.int32),
                   flip=rng.integers(0, 2, size=10).astype(np.uint8)),
              dict(kind="bfc_logits", K=10, N=4, w=_pm1(rng, (4, 10)))]
    got, trace = oracle.forward(layers, x, return_all=True)

    xt = torch.from_numpy(x)
    one = torch.ones((), dtype=torch.float64)
    gray = _torch_gray(xt)
    if mode == "input_gray":
        a = torch.where(gray + torch.tensor(float(T[0]), dtype=torch.float32) > 0, one, -one)
        a = a.unsqueeze(-1)
    else:
        a = _torch_lbp(gray)
    assert np.array_equal(trace[0], a.numpy().astype(np.int8))  # the binarized input
    a = a.permute(0, 3, 1, 2)
    for L in layers[1:3]:
        p = L["pad"]
        wt = torch.from_numpy(L["w"].astype(np.float64)).permute(0, 3, 1, 2)
        s = tF.conv2d(tF.pad(a, (p, p, p, p), value=-1.0), wt)
        thr = torch.from_numpy(L["thr"].astype(np.float64)).view(1, -1, 1, 1)
        fl = torch.from_numpy(L["flip"].astype(bool)).view(1, -1, 1, 1)
        a = torch.where((s >= thr) ^ fl, one, -one)
        if L["pool"]:
            a = tF.max_pool2d(a, 2)
    a = a.permute(0, 2, 3, 1).reshape(N, -1)
    L = layers[3]
    s = a @ torch.from_numpy(L["w"].astype(np.float64)).T
    bit = (s >= torch.from_numpy(L["thr"].astype(np.float64))) ^ \
        torch.from_numpy(L["flip"].astype(bool))
    a = torch.where(bit, one, -one)
    ref = a @ torch.from_numpy(layers[4]["w"].astype(np.float64)).T
    assert np.array_equal(got, ref.numpy().astype(np.int32))
    assert len(np.unique(got)) > 2  # the chain is not degenerate
