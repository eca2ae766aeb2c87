"""bnn_forward captured into a HIP graph: every replay must equal the eager
result, with other eager work and synchronisations between replays (the
library records no memset or allocation, so the calls are capture-safe)."""
import numpy as np
import pytest
import torch

import oracle
from paper_1808_00209_amd import bnn, synth
from paper_1808_00209_amd.device import to_device, upload_network

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("batch", [1, 4])
def test_forward_graph_replays_match_eager(batch):
    layers = synth.cfg3_net()
    net = upload_network(layers, 32, 32, 3)
    x_host = synth.cfg3_input(batch + 3)
    x = to_device(x_host[:batch]).contiguous()
    ws = net.alloc_workspace(batch)
    out = torch.empty((batch, 10), dtype=torch.int32, device="cuda")
    eager = bnn.bnn_forward(net, x, ws, torch.empty_like(out))
    torch.cuda.synchronize()
    ref = oracle.forward(layers, x_host[:batch])
    assert np.array_equal(eager.cpu().numpy(), ref)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        bnn.bnn_forward(net, x, ws, out)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        bnn.bnn_forward(net, x, ws, out)
    other = to_device(x_host[batch:batch + 1]).contiguous()
    for rep in range(4):
        out.fill_(-7)
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(out.cpu().numpy(), ref), "replay %d" % rep
        # unrelated eager work through the same workspace between replays
        bnn.bnn_forward(net, other, net.alloc_workspace(1))
        torch.cuda.synchronize()
    # new input copied into the captured buffer
    x.copy_(to_device(x_host[3:3 + batch]))
    g.replay()
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy(), oracle.forward(layers, x_host[3:3 + batch]))
