"""Binary 3x3 convs on 8 x 8 maps, bits only (bnn_bconv2d without sums takes
the whole-image kernel there; the CIFAR-shaped net's L4 and L5): bit-exact
against the oracle (Eq. 3 / Eq. 4 sums with the -1 pad, threshold and flip,
2x2 OR-pool, Eq. 2 packing) and against the same call with int32 sums, which
runs the general matrix-core kernel; every channel count the kernel takes,
128 to 512 filters, with and without pooling, NULL flips, tied and extreme
thresholds."""
import numpy as np
import pytest
import torch

import oracle
from paper_1808_00209_amd import bnn, synth
from paper_1808_00209_amd.device import pack_flips, pack_pm1, to_device, words_u32

pytestmark = pytest.mark.gpu

# Grids of at least 256 blocks of 128 filters take those, smaller ones blocks
# of 64 filters.
#        N,   C,   F, pool
CASES = [
    (64, 256, 512, 0),   # the CIFAR-shaped net's L4 at batch 64
    (64, 512, 512, 2),   # and L5
    (1, 64, 128, 0),
    (3, 128, 256, 2),
    (5, 512, 128, 0),
    (2, 256, 384, 2),
    (200, 128, 256, 2),  # blocks of 128 filters with a filter group count of 2
]


def _oracle_bits(x, w, thr, flip, pool):
    b = oracle.threshold(oracle.conv2d(x, w, 1, 1), thr, flip)
    if pool:
        b = oracle.maxpool2(b)
    return oracle.pack_eq2(b)


def _run(case, x, w, thr, flip, use_flip=True):
    N, C, F, pool = case
    desc = bnn.conv_desc(N, 8, 8, C, F, 3, 3, 1, 1, pool)
    xd, wd = pack_pm1(x), pack_pm1(w)
    td = to_device(thr, torch.int32)
    fd = pack_flips(flip) if use_flip else None
    _, bits = bnn.bnn_bconv2d(desc, xd, wd, td, fd, want_sums=False)
    _, bits2 = bnn.bnn_bconv2d(desc, xd, wd, td, fd, want_sums=True)
    torch.cuda.synchronize()
    return bits, bits2


@pytest.mark.parametrize("case", CASES, ids=[str(c) for c in CASES])
def test_img8_conv_matches_oracle_and_general_kernel(case):
    N, C, F, pool = case
    print("img8 case", case, flush=True)
    rng = np.random.default_rng(7000 + N + C + F + pool)
    x = synth.pm1(rng, (N, 8, 8, C))
    L = synth.conv_layer(15, C // 64, "bconv", C, F, pad=1, pool=pool)
    bits, bits2 = _run(case, x, L["w"], L["thr"], L["flip"])
    assert np.array_equal(words_u32(bits), _oracle_bits(x, L["w"], L["thr"], L["flip"], pool))
    assert torch.equal(bits, bits2)


def test_img8_no_flips_extreme_and_tied_thresholds():
    """NULL flips; thresholds at 0 (K even: ties), beyond every sum both ways
    and at the int32 limits."""
    case = (4, 256, 128, 2)
    N, C, F, pool = case
    rng = np.random.default_rng(81)
    x = synth.pm1(rng, (N, 8, 8, C))
    L = synth.conv_layer(16, 0, "bconv", C, F, pad=1, pool=pool)
    K = 9 * C
    L["thr"][:32] = 0
    L["thr"][32:40] = -K - 3
    L["thr"][40:48] = K + 3
    L["thr"][48] = np.iinfo(np.int32).max
    L["thr"][49] = np.iinfo(np.int32).min
    L["thr"][50] = K
    L["thr"][51] = -K
    bits, bits2 = _run(case, x, L["w"], L["thr"], L["flip"], use_flip=False)
    assert np.array_equal(words_u32(bits),
                          _oracle_bits(x, L["w"], L["thr"], np.zeros_like(L["flip"]), pool))
    assert torch.equal(bits, bits2)
