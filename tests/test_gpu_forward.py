"""GPU parity of the whole layer chain (bnn_forward) against the oracle: the
logits of every image, at small batches and at the full-size batches (64
images of the CIFAR-shaped net, 256 of the vehicle-shaped net), under every
kernel family and fusion setting."""
import functools

import numpy as np
import pytest
import torch

import oracle
from paper_1808_00209_amd import bnn, synth
from paper_1808_00209_amd.device import to_device, upload_network

pytestmark = pytest.mark.gpu


# "auto": default kernels; "valu": vector-ALU kernels only; "lds": the
# matrix-core kernel with weights staged through LDS; "nopatch": the thresholded
# input packed by bnn_pack_bits and convolved by the generic kernel instead
# of the fused patch-packing kernel; "nochain": every FC layer as its own
# launch instead of runs of small FC layers in the chained kernel; "nofuse":
# the real-valued first layer and the binary conv after it as two launches
# instead of the fused first-layer kernel.
# "packed": "auto" with packed conv weights only (no prepared operand form,
# which every other family passes in each binary conv layer).
_PREPARE = True


@pytest.fixture(params=["auto", "valu", "lds", "nopatch", "nochain", "nofuse", "packed"])
def algo(request):
    global _PREPARE
    bnn.bnn_set_options(**{"auto": {}, "valu": dict(algo=bnn.ALGO_VALU),
                           "lds": dict(lds_weights=1), "nopatch": dict(fuse_input=0),
                           "nochain": dict(fc_chain=0), "nofuse": dict(fuse_first=0),
                           "packed": {}}[request.param])
    _PREPARE = request.param != "packed"
    yield request.param
    _PREPARE = True


def _gpu_logits(layers, x):
    N, H, W, C = x.shape
    net = upload_network(layers, H, W, C, prepare=_PREPARE)
    out = bnn.bnn_forward(net, to_device(x))
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("batch", [1, 3])
def test_cifar_net_small_batch(batch, algo):
    layers, x = synth.cfg3_net(), synth.cfg3_input(batch)
    got = _gpu_logits(layers, x)
    ref = oracle.forward(layers, x)
    assert got.shape == (batch, 10)
    assert np.array_equal(got, ref)


def test_vehicle_net_small_batch(algo):
    layers, x = synth.cfg4_net(), synth.cfg4_input(2)
    got = _gpu_logits(layers, x)
    ref = oracle.forward(layers, x)
    assert got.shape == (2, 4)
    assert np.array_equal(got, ref)


@functools.lru_cache(maxsize=2)
def _oracle_logits(cfg, batch):
    """The oracle's logits for every image of a full-size batch (computed once
    per module run: about 1 s for 64 CIFAR-shaped images and 11 s for 256
    vehicle-shaped ones on 16 host threads)."""
    if cfg == 3:
        return oracle.forward(synth.cfg3_net(), synth.cfg3_input(batch))
    return oracle.forward(synth.cfg4_net(), synth.cfg4_input(batch))


def test_cifar_net_batch64_every_image(algo):
    layers, x = synth.cfg3_net(), synth.cfg3_input(64)
    got = _gpu_logits(layers, x)
    assert np.array_equal(got, _oracle_logits(3, 64))


def test_vehicle_net_batch256_every_image(algo):
    layers, x = synth.cfg4_net(), synth.cfg4_input(256)
    got = _gpu_logits(layers, x)
    assert np.array_equal(got, _oracle_logits(4, 256))


def test_forward_is_deterministic_and_batch_independent():
    layers, x = synth.cfg3_net(), synth.cfg3_input(8)
    a = _gpu_logits(layers, x)
    b = _gpu_logits(layers, x)
    c = _gpu_logits(layers, x[5:6])
    assert np.array_equal(a, b)
    assert np.array_equal(a[5:6], c)


@pytest.mark.parametrize("mode", synth.PAPER_MODES)
def test_paper_net_small_batch(mode, algo):
    """Table II's 5x5 vehicle classifier behind each input binarization of
    Table III (RGB / grayscale thresholding, LBP)."""
    layers, x = synth.paper_net(mode), synth.paper_input(2)
    got = _gpu_logits(layers, x)
    ref = oracle.forward(layers, x)
    assert got.shape == (2, 4)
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("mode", synth.PAPER_MODES)
def test_paper_net_batch64_every_image(mode):
    layers, x = synth.paper_net(mode), synth.paper_input(64)
    got = _gpu_logits(layers, x)
    assert np.array_equal(got, oracle.forward(layers, x))
