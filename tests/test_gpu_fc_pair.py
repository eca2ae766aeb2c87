"""Two binary FC layers in one launch (bnn_bfc_pair: the CIFAR-shaped net's
1024 -> 1024 -> 10 tail, Sec. III-B): bit-exact against the oracle (Eq. 4
sums, threshold and flip, Eq. 2 packing) and against two bnn_bgemm calls, for
every K0 / N0 the kernel takes, int32 sums and bits, ragged row counts,
NULL flips and tied / extreme thresholds."""
import numpy as np
import pytest
import torch

import oracle
from paper_1808_00209_amd import bnn, synth
from paper_1808_00209_amd.device import pack_flips, pack_pm1, to_device, words_u32

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
