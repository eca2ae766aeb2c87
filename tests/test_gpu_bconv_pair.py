"""Two binary 3x3 convs in one launch (bnn_bconv_bconv2d: the CIFAR-shaped
net's 16 x 16 stage, a conv -> conv step of Table II's layer order): bit-exact
against the oracle chain (Eq. 3 / Eq. 4 sums with the -1 pad, threshold and
flip, 2x2 OR-pool, Eq. 2 packing) and against two bnn_bconv2d launches, on
whole and ragged 4-row and 2-row tiles, every input width the kernel takes, with and
without pooling, NULL flips, extreme and tied thresholds, and inside
bnn_forward with option fuse_pair on and off."""
import numpy as np
import pytest
import torch

import oracle
from paper_1808_00209_amd import bnn, synth
from paper_1808_00209_amd.device import pack_pm1, to_device, upload_layer, upload_network, words_u32

pytestmark = pytest.mark.gpu

# Grids of at least 256 blocks of 4 rows take 4-row tiles, smaller ones 2-row
# tiles.
#        N,  H,  C0, pool
CASES = [
    (2, 16, 128, 2),    # the CIFAR-shaped stage, 2-row tiles
    (3, 16, 64, 0),
    (1, 16, 256, 2),
    (2, 6, 128, 2),
    (1, 5, 256, 0),     # odd height, no pooling: a last tile with one row
    (1, 3, 64, 2),      # odd height with pooling (one pooled row)
    (1, 1, 128, 0),     # a single row
    (5, 12, 128, 2),
    (86, 12, 128, 2),   # 4-row tiles
    (43, 22, 256, 0),   # 4-row tiles, a last tile with two rows
    (128, 8, 64, 2),
    (52, 19, 128, 2),   # 4-row tiles, a last tile with three rows
]


def _layers(seed, C0, pool):
    L0 = synth.conv_layer(seed, 0, "bconv", C0, 256, pad=1)
    L1 = synth.conv_layer(seed, 1, "bconv", 256, 256, pad=1, pool=pool)
    return L0, L1


def _oracle_bits(x, L0, L1, flips=True):
    a0 = oracle.threshold(oracle.conv2d(x, L0["w"], 1, 1), L0["thr"],
                          L0["flip"] if flips else np.zeros_like(L0["flip"]))
    b1 = oracle.threshold(oracle.conv2d(a0, L1["w"], 1, 1), L1["thr"],
                          L1["flip"] if flips else np.zeros_like(L1["flip"]))
    if L1["pool"]:
        b1 = oracle.maxpool2(b1)
    return oracle.pack_eq2(b1)


def _descs(N, H, C0, pool):
    return (bnn.conv_desc(N, H, 16, C0, 256, 3, 3, 1, 1, 0),
            bnn.conv_desc(N, H, 16, 256, 256, 3, 3, 1, 1, pool))


def _two_launches(d0, d1, xd, l0, l1, flips=True):
    _, b0 = bnn.bnn_bconv2d(d0, xd, l0["w"], l0["thr"], l0["flip"] if flips else None,
                            want_sums=False)
    _, b1 = bnn.bnn_bconv2d(d1, b0, l1["w"], l1["thr"], l1["flip"] if flips else None,
                            want_sums=False)
    return b1


@pytest.mark.parametrize("case", CASES, ids=[str(c) for c in CASES])
def test_bconv_pair_matches_oracle_and_two_launches(case):
    N, H, C0, pool = case
    print("conv pair case", case, flush=True)
    rng = np.random.default_rng(900 + sum(case))
    x = synth.pm1(rng, (N, H, 16, C0))
    L0, L1 = _layers(13, C0, pool)
    l0, l1 = upload_layer(L0), upload_layer(L1)
    d0, d1 = _descs(N, H, C0, pool)
    xd = pack_pm1(x)
    got = bnn.bnn_bconv_bconv2d(d0, d1, xd, l0["w"], l0["thr"], l0["flip"], l1["w"], l1["thr"],
                                l1["flip"])
    two = _two_launches(d0, d1, xd, l0, l1)
    torch.cuda.synchronize()
    assert np.array_equal(words_u32(got), _oracle_bits(x, L0, L1))
    assert torch.equal(got, two)


def test_bconv_pair_no_flips_extreme_and_tied_thresholds():
    """flip0 / flip1 NULL; thresholds at 0 (ties: K is even, so S = 0 occurs
    and gives bit 1), beyond every sum both ways, and at the int32 limits
    (clamped on the device without changing a comparison)."""
    N, H, C0, pool = 2, 10, 128, 2
    rng = np.random.default_rng(31)
    x = synth.pm1(rng, (N, H, 16, C0))
    L0, L1 = _layers(14, C0, pool)
    for L, K in ((L0, 9 * C0), (L1, 9 * 256)):
        L["thr"][:64] = 0
        L["thr"][64:80] = -K - 3
        L["thr"][80:96] = K + 3
        L["thr"][96] = np.iinfo(np.int32).max
        L["thr"][97] = np.iinfo(np.int32).min
        L["thr"][98] = K
        L["thr"][99] = -K
    l0, l1 = upload_layer(L0), upload_layer(L1)
    d0, d1 = _descs(N, H, C0, pool)
    xd = pack_pm1(x)
    got = bnn.bnn_bconv_bconv2d(d0, d1, xd, l0["w"], l0["thr"], None, l1["w"], l1["thr"], None)
    two = _two_launches(d0, d1, xd, l0, l1, flips=False)
    torch.cuda.synchronize()
    assert np.array_equal(words_u32(got), _oracle_bits(x, L0, L1, flips=False))
    assert torch.equal(got, two)


def test_bconv_pair_cifar_stage_full_batch():
    """The CIFAR-shaped net's L2 + L3 at batch 64 with the net's own weights,
    in the launch bnn_forward makes: every output word against the two
    separate launches, two images against the oracle."""
    layers = synth.cfg3_net()
    L0, L1 = layers[2], layers[3]
    N = 64
    rng = np.random.default_rng(64)
    x = synth.pm1(rng, (N, 16, 16, 128))
    l0, l1 = upload_layer(L0), upload_layer(L1)
    d0, d1 = _descs(N, 16, 128, 2)
    xd = pack_pm1(x)
    got = bnn.bnn_bconv_bconv2d(d0, d1, xd, l0["w"], l0["thr"], l0["flip"], l1["w"], l1["thr"],
                                l1["flip"])
    two = _two_launches(d0, d1, xd, l0, l1)
    torch.cuda.synchronize()
    assert torch.equal(got, two)
    pick = [0, N - 1]
    assert np.array_equal(words_u32(got)[pick], _oracle_bits(x[pick], L0, L1))


@pytest.mark.parametrize("batch", [1, 3, 64])
def test_cifar_forward_fused_pair_equals_separate_launches(batch):
    """bnn_forward on the CIFAR-shaped net with the L2 + L3 pair fused
    (default) and with option fuse_pair = 0, and against the oracle."""
    layers = synth.cfg3_net()
    net = upload_network(layers, 32, 32, 3)
    x = synth.cfg3_input(batch)
    xd = to_device(x)
    fused = bnn.bnn_forward(net, xd)
    with bnn.options(fuse_pair=0):
        apart = bnn.bnn_forward(net, xd)
    torch.cuda.synchronize()
    assert torch.equal(fused, apart)
    pick = [0, batch - 1]
    assert np.array_equal(fused.cpu().numpy()[pick], oracle.forward(layers, x[pick]))
