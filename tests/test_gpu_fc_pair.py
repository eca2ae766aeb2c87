"""Two binary FC layers in one launch (the CIFAR-shaped net's 1024 -> 1024 ->
10 tail, Sec. III-B): bnn_bfc_pair, and the FC tail kernel inside
bnn_forward.  Bit-exact against the oracle (Eq. 4 sums, threshold and flip,
Eq. 2 packing) and against the layers launched apart, for every K0 / N0 the
kernels take, int32 sums and bits, ragged row counts, NULL flips, tied and
extreme thresholds, and one workspace through calls of several batch
sizes."""
import numpy as np
import pytest
import torch

import oracle
from paper_1808_00209_amd import bnn, synth
from paper_1808_00209_amd.device import pack_flips, pack_pm1, to_device, upload_network, words_u32

pytestmark = pytest.mark.gpu

#        M,    K0,   N0, N1, logits
CASES = [
    (64, 1024, 1024, 10, True),    # the CIFAR-shaped net's tail at batch 64
    (1, 1024, 1024, 10, True),
    (3, 512, 256, 32, False),
    (33, 1024, 512, 1, True),      # a ragged second row block
    (100, 512, 1024, 17, False),
    (2, 512, 256, 4, True),
]


def _case(case, seed):
    M, K0, N0, N1, logits = case
    rng = np.random.default_rng(seed)
    a = synth.pm1(rng, (M, K0))
    L0 = synth.fc_layer(20 + seed % 7, 0, K0, N0)
    L1 = synth.fc_layer(20 + seed % 7, 1, N0, N1, logits=logits)
    return a, L0, L1


def _oracle(a, L0, L1, flips=True):
    f0 = L0["flip"] if flips else np.zeros_like(L0["flip"])
    h = oracle.threshold(oracle.fc(a, L0["w"]), L0["thr"], f0)
    S = oracle.fc(h, L1["w"])
    if "thr" not in L1:
        return S
    f1 = L1["flip"] if flips else np.zeros_like(L1["flip"])
    return oracle.pack_eq2(oracle.threshold(S, L1["thr"], f1))


def _dev(L, flips=True):
    d = dict(w=pack_pm1(L["w"]))
    if "thr" in L:
        d["thr"] = to_device(L["thr"], torch.int32)
        d["flip"] = pack_flips(L["flip"]) if flips else None
    return d


@pytest.mark.parametrize("case", CASES, ids=[str(c) for c in CASES])
def test_fc_pair_matches_oracle_and_two_gemms(case):
    M, K0, N0, N1, logits = case
    print("fc pair case", case, flush=True)
    a, L0, L1 = _case(case, 40 + M + N1)
    d0, d1 = _dev(L0), _dev(L1)
    A = pack_pm1(a)
    got = bnn.bnn_bfc_pair(A, K0, d0["w"], d0["thr"], d0["flip"], d1["w"], N1,
                           d1.get("thr"), d1.get("flip"))
    _, hb = bnn.bnn_bgemm(A, d0["w"], K0, d0["thr"], d0["flip"], want_sums=False)
    if logits:
        two, _ = bnn.bnn_bgemm(hb, d1["w"], N0, want_bits=False)
    else:
        _, two = bnn.bnn_bgemm(hb, d1["w"], N0, d1["thr"], d1["flip"], want_sums=False)
    torch.cuda.synchronize()
    want = _oracle(a, L0, L1)
    if logits:
        assert np.array_equal(got.cpu().numpy(), want)
    else:
        assert np.array_equal(words_u32(got), want)
    assert torch.equal(got, two)


def test_fc_pair_no_flips_extreme_and_tied_thresholds():
    """flip0 / flip1 NULL; thresholds at 0 (K even: S = 0 occurs, bit 1),
    beyond every sum both ways and at the int32 limits."""
    M, K0, N0, N1 = 40, 1024, 512, 32
    a, L0, L1 = _case((M, K0, N0, N1, False), 5)
    for L, K in ((L0, K0), (L1, N0)):
        L["thr"][:8] = 0
        L["thr"][8:12] = -K - 3
        L["thr"][12:16] = K + 3
        L["thr"][16] = np.iinfo(np.int32).max
        L["thr"][17] = np.iinfo(np.int32).min
        L["thr"][18] = K
        L["thr"][19] = -K
    d0, d1 = _dev(L0, flips=False), _dev(L1, flips=False)
    got = bnn.bnn_bfc_pair(pack_pm1(a), K0, d0["w"], d0["thr"], None, d1["w"], N1, d1["thr"],
                           None)
    torch.cuda.synchronize()
    assert np.array_equal(words_u32(got), _oracle(a, L0, L1, flips=False))


# FC tails inside bnn_forward: two FC layers whose second has at most 32
# outputs, the first with K >= 1024 and N a multiple of 32, run as one launch
# of the FC kernel (a workgroup per 32 x 32 tile of the first layer, the last
# workgroup of each 32-row block adding the second layer's partial sums).
# The stacks sit behind a real-valued first layer on a 1 x 1 image (3x3,
# pad 1) whose outputs are the first FC layer's input bits; option
# fc_chain = 0 keeps small stacks off the chained kernel.
TAILS = {
    "cifar": (1024, [1024, 10]),        # the CIFAR-shaped net's tail
    "bits_tail": (2048, [512, 32, 10]),  # the pair's second layer writes bits
    "one_output": (1024, [64, 1]),
    "three_slices": (3072, [96, 17]),
    "padded_k": (1100, [256, 12]),      # K not a multiple of 32: padded rows
}


def _tail_net(name):
    K0, sizes = TAILS[name]
    layers = [synth.conv_layer(9, 0, "fconv", 3, K0)]
    k = K0
    for i, n in enumerate(sizes):
        layers.append(synth.fc_layer(9, i + 1, k, n, logits=(i == len(sizes) - 1)))
        k = n
    return layers


def _tail_run(net, xd, fused, ws=None):
    with bnn.options(fc_chain=0, fuse_pair=int(fused)):
        out = bnn.bnn_forward(net, xd, ws)
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("name", sorted(TAILS))
@pytest.mark.parametrize("batch", [1, 2, 3, 31, 32, 33, 64, 100, 200, 512, 513])
def test_fc_tail_in_forward_matches_apart_and_oracle(name, batch):
    print("fc tail", name, batch, flush=True)
    layers = _tail_net(name)
    x = synth.dyadic_normal(synth.rng(9, 90 + batch, synth.T_X), (batch, 1, 1, 3))
    net = upload_network(layers, 1, 1, 3)
    xd = to_device(x)
    got = _tail_run(net, xd, True)
    assert np.array_equal(got, _tail_run(net, xd, False))
    assert np.array_equal(got, oracle.forward(layers, x))


def test_fc_tail_bits_ties_extremes_and_no_flips():
    """The tail's second layer writing bits: thresholds at 0 (N0 even: S = 0
    occurs, bit 1), beyond every sum both ways, at +-N0 and at the int32
    limits, with flips and without."""
    layers = _tail_net("bits_tail")
    L = layers[2]
    N0 = L["K"]
    L["thr"][:8] = 0
    L["thr"][8:12] = -N0 - 3
    L["thr"][12:16] = N0 + 3
    L["thr"][16] = np.iinfo(np.int32).max
    L["thr"][17] = np.iinfo(np.int32).min
    L["thr"][18] = N0
    L["thr"][19] = -N0
    x = synth.dyadic_normal(synth.rng(9, 7, synth.T_X), (70, 1, 1, 3))
    xd = to_device(x)
    for flips in (True, False):
        if not flips:
            L["flip"][:] = 0
        net = upload_network(layers, 1, 1, 3)
        got = _tail_run(net, xd, True)
        assert np.array_equal(got, _tail_run(net, xd, False))
        assert np.array_equal(got, oracle.forward(layers, x))


def test_fc_tail_counters_left_zero_across_calls_and_batches():
    """One workspace through calls of different batch sizes (different row
    block counts): every call must find the counters zero, so every result
    is exact, and the counter bytes are zero after each call."""
    layers = _tail_net("cifar")
    net = upload_network(layers, 1, 1, 3)
    ws = net.alloc_workspace(200)
    for batch in (200, 33, 1, 200, 64):
        x = synth.dyadic_normal(synth.rng(9, 300 + batch, synth.T_X), (batch, 1, 1, 3))
        got = _tail_run(net, to_device(x), True, ws)
        assert np.array_equal(got, oracle.forward(layers, x)), batch
        assert not ws[:bnn.FORWARD_SYNC_BYTES].any().item()


#             M,   K0,   N0, N1, logits
TAIL_CASES = [(64, 1024, 1024, 10, True),   # the CIFAR-shaped net's tail at batch 64
              (1, 1024, 1024, 10, True),
              (3, 2048, 512, 32, False),
              (33, 1024, 64, 1, True),       # a ragged second row block
              (100, 3072, 96, 17, False),    # three first-layer slices
              (512, 1024, 1024, 10, True),   # 512 rows and 512 tiles, the limits
              (200, 1024, 2048, 5, False),
              (50, 1500, 64, 7, True),       # K0 not a multiple of 32: padded rows
              (20, 2047, 128, 32, False)]


@pytest.mark.parametrize("case", TAIL_CASES, ids=[str(c) for c in TAIL_CASES])
def test_fc_tail_kernel_matches_oracle_and_two_gemms(case):
    """bnn_bfc_tail through the C ABI, twice on one accumulator buffer: the
    oracle, two bnn_bgemm calls, and the buffer zero after each call."""
    M, K0, N0, N1, logits = case
    print("fc tail kernel case", case, flush=True)
    a, L0, L1 = _case(case, 60 + M + N1)
    d0, d1 = _dev(L0), _dev(L1)
    A = pack_pm1(a)
    accum = bnn.accum_buffer()
    _, hb = bnn.bnn_bgemm(A, d0["w"], K0, d0["thr"], d0["flip"], want_sums=False)
    if logits:
        two, _ = bnn.bnn_bgemm(hb, d1["w"], N0, want_bits=False)
    else:
        _, two = bnn.bnn_bgemm(hb, d1["w"], N0, d1["thr"], d1["flip"], want_sums=False)
    want = _oracle(a, L0, L1)
    for rep in range(2):
        got = bnn.bnn_bfc_tail(A, K0, d0["w"], d0["thr"], d0["flip"], d1["w"], N1, accum,
                               d1.get("thr"), d1.get("flip"))
        torch.cuda.synchronize()
        if logits:
            assert np.array_equal(got.cpu().numpy(), want), rep
        else:
            assert np.array_equal(words_u32(got), want), rep
        assert torch.equal(got, two)
        assert not accum.any().item()
