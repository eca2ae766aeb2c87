"""bnn_forward_noalloc (the chain with the intermediate bits in the library's
per-GPU scratch array, for callers that cannot allocate) against bnn_forward
with a caller workspace: bit-exact logits on consecutive calls, the later
ones on smaller inputs, so that each reuses the array the call before left
its bits in."""
import numpy as np
import pytest
import torch

import oracle
from paper_1808_00209_amd import bnn, synth
from paper_1808_00209_amd.device import to_device, upload_network

pytestmark = pytest.mark.gpu


def _both(layers, x, H, W, C):
    net = upload_network(layers, H, W, C)
    xd = to_device(x)
    ref = bnn.bnn_forward(net, xd)
    got = bnn.bnn_forward_noalloc(net, xd)
    torch.cuda.synchronize()
    return got.cpu().numpy(), ref.cpu().numpy()


def test_noalloc_matches_forward_on_calls_of_decreasing_size():
    cases = [("vehicle b256", synth.cfg4_net(), synth.cfg4_input(256), 96, 96),
             ("cifar b64", synth.cfg3_net(), synth.cfg3_input(64), 32, 32),
             ("cifar b3", synth.cfg3_net(), synth.cfg3_input(3), 32, 32)]
    for name, layers, x, H, W in cases:
        print("forward_noalloc:", name, flush=True)
        got, ref = _both(layers, x, H, W, 3)
        assert np.array_equal(got, ref), name
        if x.shape[0] <= 3:
            assert np.array_equal(got, oracle.forward(layers, x)), name


def test_noalloc_rejects_a_chain_beyond_the_scratch_array():
    layers = synth.cfg4_net()
    net = upload_network(layers, 96, 96, 3)
    assert net.workspace_size(512) > bnn.FORWARD_SCRATCH_BYTES
    x = torch.zeros((512, 96, 96, 3), dtype=torch.float32, device="cuda")
    with pytest.raises(bnn.BnnError, match="BNN_ERR_WORKSPACE"):
        bnn.bnn_forward_noalloc(net, x)
