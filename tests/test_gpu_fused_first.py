"""GPU parity of the fused first-layer kernel (the real-valued first conv and
the binary 3x3 conv after it in one launch, the first layer's bits kept in
LDS) inside bnn_forward, against the two separate launches and the oracle.

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
from paper_1808_00209_amd.device import to_device, upload_network

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


def _run(net, xd, monkeypatch, fuse):
    monkeypatch.setenv("BNN_FUSE_FIRST", "1" if fuse else "0")
    out = bnn.bnn_forward(net, xd)
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("name", sorted(CASES))
@pytest.mark.parametrize("batch", [1, 5])
def test_fused_first_matches_two_launches_and_oracle(name, batch, monkeypatch):
    H, W, C0 = CASES[name][:3]
    layers = _net(name)
    x = synth.dyadic_normal(synth.rng(9, 90, synth.T_X), (batch, H, W, C0))
    net = upload_network(layers, H, W, C0)
    xd = to_device(x)
    got = _run(net, xd, monkeypatch, True)
    ref = _run(net, xd, monkeypatch, False)
    assert np.array_equal(got, ref)
    pick = sorted({0, batch - 1})
    assert np.array_equal(got[pick], oracle.forward(layers, x[pick]))


def test_fused_first_cifar_batch64_sampled(monkeypatch):
    """The CIFAR-shaped net's first two layers at the benchmark's batch."""
    layers, x = synth.cfg3_net(), synth.cfg3_input(64)
    net = upload_network(layers, 32, 32, 3)
    xd = to_device(x)
    got = _run(net, xd, monkeypatch, True)
    ref = _run(net, xd, monkeypatch, False)
    assert np.array_equal(got, ref)
    pick = [0, 37, 63]
    assert np.array_equal(got[pick], oracle.forward(layers, x[pick]))
