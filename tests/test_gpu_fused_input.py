"""Input thresholding (Sec. II-C), a binary 3x3 conv over the thresholded
image and a second binary 3x3 conv in one launch (bnn_input_bconv_bconv2d,
the first layers of the vehicle-shaped net): bit-exact against the oracle
chain (sign with per-channel offsets, Eq. 3 / Eq. 4 sums, threshold and
flip, 2x2 OR-pool, Eq. 2 packing) and against the two separate launches
bnn_bconv2d_input + bnn_bconv2d, with packed and with prepared second-layer
weights, on 4-row (small grids) and 8-row tiles."""
import numpy as np
import pytest
import torch

import oracle
from paper_1808_00209_amd import bnn, synth
from paper_1808_00209_amd.device import pack_flips, pack_pm1, to_device, upload_layer, words_u32

pytestmark = pytest.mark.gpu
T = bnn.INPUT_THRESHOLD

#        N,  H,  W, F0, pad0, F1, pad1, pool
CASES = [
    (2, 96, 96, 64, 1, 64, 1, 2),       # the vehicle-shaped net's first layers
    (40, 24, 40, 64, 1, 64, 1, 2),      # 8-row tiles
    (3, 13, 20, 128, 0, 64, 1, 2),      # odd sizes, first pad 0
    (1, 9, 37, 64, 1, 128, 0, 0),       # no pooling, second pad 0
    (34, 17, 33, 128, 1, 128, 1, 0),    # 8-row tiles, ragged tile edges
    (1, 3, 3, 64, 1, 64, 1, 2),         # a single 2x2 window
]


def _case(case, seed):
    N, H, W, F0, pad0, F1, pad1, pool = case
    rng = np.random.default_rng(seed)
    x = synth.pixels(rng, (N, H, W, 3))
    off = synth.rgb_offsets(rng, 3)
    L0 = synth.conv_layer(11, 0, "bconv", 3, F0, pad=pad0)
    L1 = synth.conv_layer(11, 1, "bconv", F0, F1, pad=pad1, pool=pool)
    return x, off, L0, L1


def _oracle_bits(x, off, L0, L1, use_off=True):
    C = x.shape[-1]
    xb = oracle.sign(x.reshape(-1, C), off if use_off else None).reshape(x.shape)
    a0 = oracle.threshold(oracle.conv2d(xb, L0["w"], 1, L0["pad"]), L0["thr"], L0["flip"])
    b1 = oracle.threshold(oracle.conv2d(a0, L1["w"], 1, L1["pad"]), L1["thr"], L1["flip"])
    if L1["pool"]:
        b1 = oracle.maxpool2(b1)
    return oracle.pack_eq2(b1)


@pytest.mark.parametrize("case", CASES, ids=[str(c) for c in CASES])
def test_input_bconv_bconv_matches_oracle_and_two_launches(case):
    N, H, W, F0, pad0, F1, pad1, pool = case
    print("fused input case", case, flush=True)
    x, off, L0, L1 = _case(case, 500 + sum(case))
    d0, d1 = upload_layer(L0), upload_layer(L1)
    xd, offd = to_device(x), to_device(off)
    desc0 = bnn.conv_desc(N, H, W, 3, F0, 3, 3, 1, pad0, 0)
    Ho0, Wo0 = H + 2 * pad0 - 2, W + 2 * pad0 - 2
    desc1 = bnn.conv_desc(N, Ho0, Wo0, F0, F1, 3, 3, 1, pad1, pool)
    want = _oracle_bits(x, off, L0, L1)
    _, b0 = bnn.bnn_bconv2d_input(desc0, T, xd, offd, d0["w"], d0["thr"], d0["flip"],
                                  want_sums=False)
    _, two = bnn.bnn_bconv2d(desc1, b0, d1["w"], d1["thr"], d1["flip"], want_sums=False)
    torch.cuda.synchronize()
    assert np.array_equal(words_u32(two), want)
    for w1prep in (None, d1["wprep"]):
        got = bnn.bnn_input_bconv_bconv2d(desc0, desc1, T, xd, offd, d0["w"], d0["thr"],
                                          d0["flip"], d1["w"], d1["thr"], d1["flip"],
                                          w1prep=w1prep)
        torch.cuda.synchronize()
        assert np.array_equal(words_u32(got), want), "w1prep %s" % (w1prep is not None)


def test_input_bconv_bconv_no_offset_no_flips_and_ties():
    """Offsets NULL (threshold at 0 on signed inputs with exact zeros: 0 maps
    to -1), flip words NULL, and first-layer thresholds at the extremes
    (every output 1 / every output -1) and at 0 (ties of the integer sums)."""
    N, H, W = 3, 20, 36
    rng = np.random.default_rng(77)
    x = (rng.integers(-2, 3, size=(N, H, W, 3))).astype(np.float32)
    L0 = synth.conv_layer(12, 0, "bconv", 3, 64, pad=1)
    L1 = synth.conv_layer(12, 1, "bconv", 64, 64, pad=1, pool=2)
    L0["thr"][:8] = -28        # below every sum: bit 1
    L0["thr"][8:16] = 28       # above every sum: bit 0
    L0["thr"][16:24] = 1       # sums are odd (K = 27): S >= 1 exactly when S > 0
    L0["flip"] = np.zeros_like(L0["flip"])
    L1["flip"] = np.zeros_like(L1["flip"])
    d0, d1 = upload_layer(L0), upload_layer(L1)
    desc0 = bnn.conv_desc(N, H, W, 3, 64, 3, 3, 1, 1, 0)
    desc1 = bnn.conv_desc(N, H, W, 64, 64, 3, 3, 1, 1, 2)
    got = bnn.bnn_input_bconv_bconv2d(desc0, desc1, T, to_device(x), None, d0["w"], d0["thr"],
                                      None, d1["w"], d1["thr"], None)
    torch.cuda.synchronize()
    assert np.array_equal(words_u32(got), _oracle_bits(x, None, L0, L1, use_off=False))


def test_vehicle_forward_fused_input_equals_separate_launches():
    """bnn_forward on the vehicle-shaped net: the three-layer fusion (default)
    against option fuse_input = 0 (input packing and two conv launches), at
    batch 3 (4-row tiles) and 40 (8-row tiles), and against the oracle."""
    layers = synth.cfg4_net()
    from paper_1808_00209_amd.device import upload_network
    net = upload_network(layers, 96, 96, 3)
    for batch in (3, 40):
        x = synth.cfg4_input(batch)
        xd = to_device(x)
        bnn.bnn_set_options(fuse_input=1)
        fused = bnn.bnn_forward(net, xd)
        bnn.bnn_set_options(fuse_input=0)
        apart = bnn.bnn_forward(net, xd)
        bnn.bnn_set_options()
        torch.cuda.synchronize()
        assert torch.equal(fused, apart)
        pick = [0, batch - 1]
        assert np.array_equal(fused.cpu().numpy()[pick], oracle.forward(layers, x[pick]))
