"""The real-valued first layer (Eq. 3 with an fp32 image and +-1 weights;
the BCNN of Table I) on general fp32 input: N(0,1) values as they come,
not rounded to any grid, at several scales, including magnitudes beyond the
fp16 range.

The library's contract (bnn_fconv2d_binw in bnn.h): every product with a
+-1 weight is exact and the sums are accumulated in fp32 in an unspecified
order, so |S_gpu - S| <= n (2^-23 sum|x| + 2^-126) over the window, with
n = 3 KH KW C (the second term covers subnormal parts and sums); the
output bit is S_gpu >= thr, compared exactly.  So the GPU sums must lie
within that bound of the oracle's fp64 sums, and the output bits must equal
the oracle's wherever |S - thr| exceeds the bound (elsewhere either bit is
correct).  The fused first-layer kernel is checked the same way through its
second layer's bits, on the outputs whose receptive field holds no
undecided first-layer value."""
import numpy as np
import pytest
import torch

import oracle
from paper_1808_00209_amd import bnn, synth
from paper_1808_00209_amd.device import pack_flips, pack_pm1, to_device, upload_layer, words_u32

pytestmark = pytest.mark.gpu


@pytest.fixture(params=["auto", "valu"])
def algo(request):
    bnn.bnn_set_options(**({"algo": bnn.ALGO_VALU} if request.param == "valu" else {}))
    return request.param


def _pm1(rng, shape):
    return (rng.integers(0, 2, size=shape) * 2 - 1).astype(np.int8)


def _inputs(seed, shape, scale):
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal(shape) * scale).astype(np.float32)
    return rng, x


def _bound(x, KH, KW, pad):
    """n (2^-23 sum|x| + 2^-126) per output pixel (fp64), n = 3 KH KW C."""
    C = x.shape[-1]
    ones = np.ones((1, KH, KW, C), np.int8)
    absum = oracle.fconv2d(np.abs(x), ones, 1, pad)[..., 0]
    return 3 * KH * KW * C * (2.0 ** -23 * absum + 2.0 ** -126)


def _thresholds(rng, F, scale, K):
    """Integers spread over the sums' range (std of S is scale sqrt(K)),
    clipped to int32."""
    t = np.round(rng.uniform(-2, 2, F) * scale * np.sqrt(K))
    return np.clip(t, -2 ** 31, 2 ** 31 - 1).astype(np.int32)


CASES = [  # N, H, W, C, F, pad, scale
    (4, 32, 32, 3, 128, 1, 1.0),
    (2, 17, 23, 3, 64, 1, 1.0),
    (2, 16, 16, 1, 64, 0, 3.0e-4),
    (2, 16, 40, 4, 128, 1, 1.0e5),   # beyond the fp16 range (65504)
    (1, 9, 9, 3, 64, 1, 3.0e8),      # sums and thresholds beyond 2^24
    (1, 8, 8, 2, 32, 1, 1.0e-30),
]


@pytest.mark.parametrize("case", CASES, ids=[str(c) for c in CASES])
@pytest.mark.parametrize("pool", [0, 2])
def test_fconv_offgrid_sums_within_bound_bits_exact_where_decided(case, pool, algo):
    N, H, W, C, F, pad, scale = case
    rng, x = _inputs(1000 + C * 7 + F, (N, H, W, C), scale)
    w = _pm1(rng, (F, 3, 3, C))
    K = 9 * C
    thr = _thresholds(rng, F, scale, K)
    flip = rng.integers(0, 2, size=F).astype(np.uint8)
    desc = bnn.conv_desc(N, H, W, C, F, 3, 3, 1, pad, pool)
    sums, bits = bnn.bnn_fconv2d_binw(desc, to_device(x), pack_pm1(w), to_device(thr, torch.int32),
                                      pack_flips(flip))
    torch.cuda.synchronize()
    S = oracle.fconv2d(x, w, 1, pad)
    bound = _bound(x, 3, 3, pad)[..., None]
    got_s = sums.cpu().numpy().astype(np.float64)
    err = np.abs(got_s - S)
    assert (err <= bound).all(), "max error / bound %.3g" % float((err / np.maximum(bound, 1e-300)).max())
    decided = np.abs(S - thr.astype(np.float64)) > bound
    b = oracle.threshold(S, thr, flip)  # +-1, pre-pool
    got_b = words_u32(bits)
    if pool:
        Hp, Wp = (H + 2 * pad - 2) // 2, (W + 2 * pad - 2) // 2
        b = oracle.maxpool2(b)
        d = decided[:, :2 * Hp, :2 * Wp].reshape(N, Hp, 2, Wp, 2, F).all(axis=(2, 4))
    else:
        d = decided
    want = oracle.pack_eq2(b)
    # compare bit by bit where decided
    unpack = lambda wds: ((wds[..., :, None] >> (31 - np.arange(32))) & 1).reshape(
        wds.shape[:-1] + (-1,))[..., :F]
    gb, wb = unpack(got_b), unpack(want)
    assert d.mean() > 0.95  # the comparison covers nearly every output
    assert np.array_equal(gb[d], wb[d])


@pytest.mark.parametrize("N", [3, 34])  # 4-row tiles with packed, 8-row with prepared w1
def test_fused_first_offgrid_second_layer_exact_where_decided(N):
    """bnn_fconv_bconv2d on N(0,1) input: the second layer's pooled bits
    against the oracle chain on every output whose 4 x 4 x F0 receptive
    field in the first layer's output holds only decided values."""
    H, W, C0, F0, F1 = 32, 32, 3, 128, 128
    rng, x = _inputs(2024, (N, H, W, C0), 1.0)
    L0 = synth.conv_layer(9, 0, "fconv", C0, F0, pad=1)
    L0["thr"] = _thresholds(rng, F0, 1.0, 9 * C0)
    L1 = synth.conv_layer(9, 1, "bconv", F0, F1, pad=1, pool=2)
    S0 = oracle.fconv2d(x, L0["w"], 1, 1)
    a0 = oracle.threshold(S0, L0["thr"], L0["flip"])
    S1 = oracle.conv2d(a0, L1["w"], 1, 1)
    want = oracle.pack_eq2(oracle.maxpool2(oracle.threshold(S1, L1["thr"], L1["flip"])))
    undecided = (np.abs(S0 - L0["thr"].astype(np.float64)) <= _bound(x, 3, 3, 1)[..., None]).any(-1)
    # a pre-pool second-layer pixel (i, j) reads first-layer pixels i-1..i+1,
    # j-1..j+1; a pooled output reads pre-pool 2ip..2ip+1, 2jp..2jp+1
    u = np.pad(undecided, ((0, 0), (1, 1), (1, 1)))
    near = np.zeros((N, H, W), bool)
    for di in range(3):
        for dj in range(3):
            near |= u[:, di:di + H, dj:dj + W]
    skip = near.reshape(N, H // 2, 2, W // 2, 2).any(axis=(2, 4))
    d0, d1 = upload_layer(L0), upload_layer(L1)
    desc0 = bnn.conv_desc(N, H, W, C0, F0, 3, 3, 1, 1, 0)
    desc1 = bnn.conv_desc(N, H, W, F0, F1, 3, 3, 1, 1, 2)
    assert (~skip).mean() > 0.8
    for w1prep in (None, d1["wprep"]):  # packed / prepared second-layer weights
        got = words_u32(bnn.bnn_fconv_bconv2d(desc0, desc1, to_device(x), d0["w"], d0["thr"],
                                              d0.get("flip"), d1["w"], d1["thr"], d1.get("flip"),
                                              w1prep=w1prep))
        torch.cuda.synchronize()
        assert np.array_equal(got[~skip], want[~skip])
