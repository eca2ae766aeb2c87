"""GPU parity of the fused first-layer kernel (the real-valued first conv and
the binary 3x3 conv after it in one launch, the first layer's bits kept in
LDS), through its own entry point bnn_fconv_bconv2d and inside bnn_forward,
against the two separate launches and the oracle.

Each net is the pair of convs followed by a logits layer over the flattened
output; every logit is a sum of +-1 products, so any differing bit of the
pair's output changes some logit by 2.  The shapes cover 1 to 4 input
channels, 64 and 128 filters in both layers, pads 0 and 1, pooling on and
off, images smaller than one 8 x 32 tile, several tiles in both directions
and odd sizes whose last pooling row and column are dropped."""
import numpy as np
import pytest
import torch

import oracle
from paper_1808_00209_amd import bnn, synth
from paper_1808_00209_amd.device import to_device, upload_layer, upload_network, words_u32

pytestmark = pytest.mark.gpu

#        H,  W, C0,  F0, pad0, F1, pad1, pool
CASES = {
    "cifar": (32, 32, 3, 128, 1, 128, 1, 2),
    "gray_64": (32, 32, 1, 64, 1, 64, 1, 0),
    "pad0_odd": (13, 20, 2, 128, 0, 64, 1, 2),
    "c4_tall": (37, 9, 4, 64, 1, 128, 0, 0),
    "tiny": (3, 3, 3, 128, 1, 128, 1, 2),
    "wide": (8, 70, 3, 128, 1, 64, 0, 2),
    "rows": (27, 33, 3, 64, 1, 128, 1, 2),
}


def _net(name):
    H, W, C0, F0, pad0, F1, pad1, pool = CASES[name]
    Ho0, Wo0 = H + 2 * pad0 - 2, W + 2 * pad0 - 2
    Ho1, Wo1 = Ho0 + 2 * pad1 - 2, Wo0 + 2 * pad1 - 2
    Hp, Wp = (Ho1 // 2, Wo1 // 2) if pool == 2 else (Ho1, Wo1)
    return [synth.conv_layer(9, 0, "fconv", C0, F0, pad=pad0),
            synth.conv_layer(9, 1, "bconv", F0, F1, pad=pad1, pool=pool),
            synth.fc_layer(9, 2, Hp * Wp * F1, 10, logits=True)]


def _run(net, xd, fuse):
    bnn.bnn_set_options(fuse_first=int(fuse))
    out = bnn.bnn_forward(net, xd)
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("name", sorted(CASES))
@pytest.mark.parametrize("batch", [1, 5, 40])  # 4-row tiles at 1 and 5, mostly 8-row at 40
def test_fused_first_matches_two_launches_and_oracle(name, batch):
    H, W, C0 = CASES[name][:3]
    layers = _net(name)
    x = synth.dyadic_normal(synth.rng(9, 90, synth.T_X), (batch, H, W, C0))
    net = upload_network(layers, H, W, C0)
    xd = to_device(x)
    got = _run(net, xd, True)
    ref = _run(net, xd, False)
    assert np.array_equal(got, ref)
    pick = sorted({0, batch - 1})
    assert np.array_equal(got[pick], oracle.forward(layers, x[pick]))


def test_fused_first_cifar_batch64_sampled():
    """The CIFAR-shaped net's first two layers at the benchmark's batch."""
    layers, x = synth.cfg3_net(), synth.cfg3_input(64)
    net = upload_network(layers, 32, 32, 3)
    xd = to_device(x)
    got = _run(net, xd, True)
    ref = _run(net, xd, False)
    assert np.array_equal(got, ref)
    pick = [0, 37, 63]
    assert np.array_equal(got[pick], oracle.forward(layers, x[pick]))


@pytest.mark.parametrize("name", sorted(CASES))
def test_fconv_bconv2d_entry_point(name):
    """bnn_fconv_bconv2d against bnn_fconv2d_binw + bnn_bconv2d and against
    the oracle's bits of the second layer (Eq. 2 packing)."""
    H, W, C0, F0, pad0, F1, pad1, pool = CASES[name]
    N = 3
    layers = _net(name)[:2]
    x = synth.dyadic_normal(synth.rng(9, 91, synth.T_X), (N, H, W, C0))
    xd = to_device(x)
    l0, l1 = (upload_layer(L) for L in layers)
    Ho0, Wo0 = H + 2 * pad0 - 2, W + 2 * pad0 - 2
    d0 = bnn.conv_desc(N, H, W, C0, F0, 3, 3, 1, pad0, 0)
    d1 = bnn.conv_desc(N, Ho0, Wo0, F0, F1, 3, 3, 1, pad1, pool)
    got = bnn.bnn_fconv_bconv2d(d0, d1, xd, l0["w"], l0["thr"], l0["flip"], l1["w"], l1["thr"],
                                l1["flip"])
    got_p = bnn.bnn_fconv_bconv2d(d0, d1, xd, l0["w"], l0["thr"], l0["flip"], l1["w"],
                                  l1["thr"], l1["flip"], w1prep=l1["wprep"])
    _, b0 = bnn.bnn_fconv2d_binw(d0, xd, l0["w"], l0["thr"], l0["flip"], want_sums=False)
    _, b1 = bnn.bnn_bconv2d(d1, b0, l1["w"], l1["thr"], l1["flip"], want_sums=False)
    torch.cuda.synchronize()
    ref = oracle.pack_eq2(oracle.forward(layers, x))
    assert np.array_equal(words_u32(got), words_u32(b1))
    assert np.array_equal(words_u32(got), ref)
    assert np.array_equal(words_u32(got_p), ref)  # prepared second-layer weights


def test_fused_first_ties_zero_windows_and_extreme_thresholds():
    """Inputs on a 0.5 grid, so first-layer sums often equal their integer
    threshold (S >= thr gives bit 1); a block of exact zeros, whose windows
    sum to 0 against thresholds of 0; and thresholds far outside any sum
    (INT32_MIN / MAX, +-10^6), which the kernel clamps without changing a
    comparison.  Fused against the two launches and the oracle."""
    H, W, C0 = 20, 36, 3
    l0 = synth.conv_layer(9, 5, "fconv", C0, 128, pad=1)
    l1 = synth.conv_layer(9, 6, "bconv", 128, 128, pad=1, pool=2)
    thr0 = l0["thr"].copy()
    thr0[:24] = 0
    thr0[24:32] = [np.iinfo(np.int32).min, np.iinfo(np.int32).max, -10**6, 10**6, 1, -1, 2, -2]
    thr0[32:40] = [0, 1, -1, 0, 3, -3, 0, 0]
    l0["thr"] = thr0.astype(np.int32)
    l1["thr"] = l1["thr"].copy()
    l1["thr"][:4] = [np.iinfo(np.int32).min, np.iinfo(np.int32).max, 0, 9 * 128]
    layers = [l0, l1, synth.fc_layer(9, 7, (H // 2) * (W // 2) * 128, 10, logits=True)]
    g = synth.rng(9, 92, synth.T_X)
    x = (g.integers(-4, 5, size=(4, H, W, C0)) * 0.5).astype(np.float32)
    x[:, 4:12, 6:20, :] = 0.0
    x[2] = 0.0
    net = upload_network(layers, H, W, C0)
    xd = to_device(x)
    got = _run(net, xd, True)
    ref = _run(net, xd, False)
    assert np.array_equal(got, ref)
    assert np.array_equal(got, oracle.forward(layers, x))
