"""GPU parity of the 1x1 short-window conv kernel (K = C <= 256 bits, at
least 65536 pixels, bits only), which keeps a wave's pixel operands in
registers and walks all filters in chunks of 64.

Every case runs twice through bnn_bconv2d, once on this kernel and once on
the general matrix-core kernel (option conv1x1 = 0), and the two outputs must agree
on every word; sampled pixels are also checked against the oracle's sums
(Eq. 3 with one tap), thresholded, flipped and packed (Eq. 2).  Shapes cover
C = 64 / 128 / 256 (1, 2 and 4 k-steps), an odd number of filter chunks, a
last block of 256 pixels that is only partly filled, ties with the
thresholds and thresholds outside [-K, K]."""
import numpy as np
import pytest
import torch

import oracle
from paper_1808_00209_amd import bnn, synth
from paper_1808_00209_amd.device import pack_flips, pack_pm1, to_device, words_u32

pytestmark = pytest.mark.gpu

#         N,   H,   W,   C,    F
CASES = [(1, 256, 256, 256, 128),
         (3, 150, 150, 64, 192),
         (1, 300, 221, 128, 64),
         (2, 181, 183, 256, 320)]


def _layer(C, F, seed, lo=None, hi=None):
    g = synth.rng(8, seed, synth.T_W)
    lo, hi = (lo, hi) if lo is not None else synth.balanced_range(C)
    return dict(w=synth.pm1(g, (F, 1, 1, C)),
                thr=synth.thresholds(synth.rng(8, seed, synth.T_THR), F, lo, hi),
                flip=synth.flips(synth.rng(8, seed, synth.T_FLIP), F), pad=0)


def _bits(x, L, use_1x1):
    bnn.bnn_set_options(conv1x1=int(use_1x1))
    N, H, W, C = x.shape
    F = L["w"].shape[0]
    desc = bnn.conv_desc(N, H, W, C, F, 1, 1, 1, 0, 0)
    _, bits = bnn.bnn_bconv2d(desc, pack_pm1(x), pack_pm1(L["w"]), to_device(L["thr"], torch.int32),
                              pack_flips(L["flip"]), want_sums=False, want_bits=True)
    torch.cuda.synchronize()
    return words_u32(bits)


def _oracle_bits_at(x, L, pix):
    """Packed output words of the pixels pix [count, 3] = (n, i, j)."""
    F = L["w"].shape[0]
    idx = np.concatenate([np.repeat(pix, F, axis=0),
                          np.tile(np.arange(F), len(pix))[:, None]], 1)
    S = oracle.conv2d_at(x, L["w"], idx, 1, 0).reshape(len(pix), F)
    return oracle.pack_eq2(oracle.threshold(S, L["thr"], L["flip"]))


def _sample_pixels(shape, count, seed):
    N, H, W = shape
    rng = np.random.default_rng(seed)
    pix = np.stack([rng.integers(0, s, count) for s in (N, H, W)], 1)
    last = np.array([[N - 1, H - 1, W - 1], [N - 1, H - 1, W - 2], [0, 0, 0]])
    return np.concatenate([pix, last])


@pytest.mark.parametrize("case", CASES, ids=[str(c) for c in CASES])
def test_conv1x1_matches_general_kernel_and_oracle(case):
    N, H, W, C, F = case
    x = synth.pm1(synth.rng(8, 50 + C, synth.T_X), (N, H, W, C))
    L = _layer(C, F, 60 + F)
    got = _bits(x, L, True)
    ref = _bits(x, L, False)
    assert np.array_equal(got, ref)
    pix = _sample_pixels((N, H, W), 150, C + F)
    assert np.array_equal(got[pix[:, 0], pix[:, 1], pix[:, 2]], _oracle_bits_at(x, L, pix))


def test_conv1x1_ties_and_extreme_thresholds():
    """Thresholds on the sums' parity grid (ties S == thr give bit 1), at
    +-K and beyond it, INT32_MIN / MAX."""
    N, H, W, C, F = 1, 260, 256, 128, 192
    x = synth.pm1(synth.rng(8, 70, synth.T_X), (N, H, W, C))
    L = _layer(C, F, 71, -8, 8)
    thr = L["thr"].copy()
    thr[thr % 2 == 1] += 1  # even, like every sum with K = 128: ties occur
    thr[:6] = [np.iinfo(np.int32).min, np.iinfo(np.int32).max, -C, C, -C - 1, C + 1]
    L["thr"] = thr.astype(np.int32)
    got = _bits(x, L, True)
    assert np.array_equal(got, _bits(x, L, False))
    pix = _sample_pixels((N, H, W), 200, 72)
    assert np.array_equal(got[pix[:, 0], pix[:, 1], pix[:, 2]], _oracle_bits_at(x, L, pix))


def test_conv1x1_cfg5_full_size_bits():
    """The 1x1 256 -> 1024 layer at 56 x 56, batch 64, bits only (the
    configuration the bench times): every word against the general kernel,
    sampled pixels against the oracle."""
    x, L = synth.cfg5_case("C")
    got = _bits(x, L, True)
    assert np.array_equal(got, _bits(x, L, False))
    pix = _sample_pixels(x.shape[:3], 60, 73)
    assert np.array_equal(got[pix[:, 0], pix[:, 1], pix[:, 2]], _oracle_bits_at(x, L, pix))


@pytest.mark.parametrize("K", [256, 192])
def test_bgemm_bits_only_through_the_1x1_kernel(K):
    """An FC layer of 70000 rows and 128 outputs runs as a 1 x M image with
    1x1 filters, bits only: with K = 256 it takes the 1x1 kernel (K = 192,
    6 words per row, is not one of its variants and goes to the general
    kernel either way), and every word must match the general kernel;
    sampled rows match the oracle's FC sums (Sec. III-B), thresholded and
    packed."""
    M, N = 70000, 128
    a = synth.pm1(synth.rng(8, 80, synth.T_X), (M, K))
    L = _layer(K, N, 81)
    w = L["w"].reshape(N, K)
    outs = []
    for use in (True, False):
        bnn.bnn_set_options(conv1x1=int(use))
        _, bits = bnn.bnn_bgemm(pack_pm1(a), pack_pm1(w), K, to_device(L["thr"], torch.int32),
                                pack_flips(L["flip"]), want_sums=False)
        torch.cuda.synchronize()
        outs.append(words_u32(bits))
    assert np.array_equal(outs[0], outs[1])
    rows = np.concatenate([np.random.default_rng(82).integers(0, M, 300), [0, M - 1]])
    S = oracle.fc(a[rows], w)
    assert np.array_equal(outs[0][rows], oracle.pack_eq2(oracle.threshold(S, L["thr"], L["flip"])))
