"""Bit-exactness at the benchmark sizes, in the modes the benchmark times.

Every output word, and every int32 sum where a call returns sums, of the
full-size workloads is compared with the CPU oracle:
* the large layers (56x56x256 -> 256 and 28x28x512 -> 512 3x3, 56x56x256 ->
  1024 1x1, batch 64) bits-only, exactly as bench.py times them, and with
  int32 sums (Eq. 3 and Eq. 4 with the threshold / flip epilogue);
* each layer of the CIFAR-shaped net at batch 64 and of the vehicle-shaped
  net at batch 256 through its own entry point, bits only as bnn_forward
  calls it, fed with the oracle's activations of the layer before, and the
  fused kernels bnn_forward runs (first layers, conv pairs, the FC tail)
  the same way (the logits of every image through bnn_forward are in
  test_gpu_forward.py).
The oracle's results are computed once per module run.
"""
import functools

import numpy as np
import pytest
import torch

import oracle
from paper_1808_00209_amd import bnn, synth
from paper_1808_00209_amd.device import pack_pm1, to_device, upload_layer, words_u32

pytestmark = pytest.mark.gpu


@pytest.fixture(params=["auto", "prep", "valu"])
def algo(request):
    """"auto": the default kernels (the matrix cores) with packed weights;
    "prep": the same with the conv weights in the prepared operand form
    (bnn_bconv2d_prepared, as bnn_forward runs the networks and bench.py
    times the layers); "valu": the vector-ALU XOR-popcount kernels (the
    ablation the benchmark also times)."""
    bnn.bnn_set_options(**({"algo": bnn.ALGO_VALU} if request.param == "valu" else {}))
    return request.param


# ------------------------------------------------ large layers, batch 64 ---
@functools.lru_cache(maxsize=3)
def _cfg5_oracle(name):
    x, L = synth.cfg5_case(name)
    S = oracle.conv2d(x, L["w"], 1, L["pad"])
    return S, oracle.pack_eq2(oracle.threshold(S, L["thr"], L["flip"]))


def _conv(desc, src, d, algo, want_sums):
    """One conv layer through bnn_bconv2d_prepared (family "prep") or
    bnn_bconv2d."""
    if algo == "prep":
        return bnn.bnn_bconv2d_prepared(desc, src, d["w"], d["wprep"], d["thr"], d.get("flip"),
                                        want_sums=want_sums)
    return bnn.bnn_bconv2d(desc, src, d["w"], d["thr"], d.get("flip"), want_sums=want_sums)


def _cfg5_gpu(name, want_sums, algo):
    """The call bench.py times: packed input and layer on the device, one
    conv call, bits only unless sums are asked for."""
    x, L = synth.cfg5_case(name)
    N, H, W, C = x.shape
    desc = bnn.conv_desc(N, H, W, C, L["F"], L["KH"], L["KW"], 1, L["pad"], L.get("pool", 0))
    dl = upload_layer(L)
    sums, bits = _conv(desc, pack_pm1(x), dl, algo, want_sums)
    torch.cuda.synchronize()
    return (sums.cpu().numpy() if want_sums else None), words_u32(bits)


@pytest.mark.parametrize("name", ["A", "B", "C"])
def test_cfg5_bits_only_every_word(name, algo):
    print("cfg5 %s bits only, %s" % (name, algo), flush=True)
    _, bits = _cfg5_gpu(name, False, algo)
    _, B = _cfg5_oracle(name)
    assert bits.shape == B.shape
    assert np.array_equal(bits, B)


@pytest.mark.parametrize("name", ["A", "B", "C"])
def test_cfg5_sums_and_bits_every_value(name, algo):
    print("cfg5 %s sums + bits, %s" % (name, algo), flush=True)
    sums, bits = _cfg5_gpu(name, True, algo)
    S, B = _cfg5_oracle(name)
    assert np.array_equal(sums, S)
    assert np.array_equal(bits, B)


# ------------------------------------- every layer of the full-size nets ---
@functools.lru_cache(maxsize=2)
def _chain_oracle(cfg, batch):
    """Input, layers and the oracle's output of every layer (+-1 activations;
    int32 logits for the last)."""
    layers = synth.cfg3_net() if cfg == 3 else synth.cfg4_net()
    x = synth.cfg3_input(batch) if cfg == 3 else synth.cfg4_input(batch)
    logits, trace = oracle.forward(layers, x, return_all=True)
    outs, k = [], 0
    for L in layers:  # input layers leave one trace entry, the others two (S, output)
        if L["kind"].startswith("input"):
            outs.append(trace[k])
            k += 1
        else:
            outs.append(trace[k + 1])
            k += 2
    assert k == len(trace) and np.array_equal(outs[-1], logits)
    return layers, x, outs


def _packed(a):
    return oracle.pack_eq2(a)


def _pair_fusable(L0, L1, w, c):
    """The conv pairs bnn_bconv_bconv2d takes (and bnn_forward fuses): 3x3,
    pad 1, 256 filters each, a 16-wide map, 64 / 128 / 256 input channels,
    no pooling in the first."""
    return (L0["KH"] == L0["KW"] == 3 and L0["pad"] == 1 and not L0.get("pool", 0)
            and w == 16 and c in (64, 128, 256) and L0["F"] == 256
            and L1["KH"] == L1["KW"] == 3 and L1["pad"] == 1 and L1["F"] == 256)


@pytest.mark.parametrize("cfg,batch", [(3, 64), (4, 256)], ids=["cifar_b64", "vehicle_b256"])
def test_every_layer_bits_at_full_batch(cfg, batch, algo):
    layers, x, outs = _chain_oracle(cfg, batch)
    N, H, W, C = x.shape
    dev = [upload_layer(L) for L in layers]
    xd = to_device(x)
    h, w = H, W
    descs = {}
    for li, L in enumerate(layers):
        k = L["kind"]
        print("cfg%d batch %d layer %d (%s), %s" % (cfg, batch, li, k, algo), flush=True)
        d = dev[li]
        if k == "input_threshold":
            got = words_u32(bnn.bnn_pack_bits(xd, d["offset"]))
            assert np.array_equal(got, _packed(outs[li]))
            continue
        if k in ("fconv", "bconv"):
            desc = bnn.conv_desc(N, h, w, L["C"], L["F"], L["KH"], L["KW"], 1, L["pad"],
                                 L.get("pool", 0))
            if k == "fconv":
                _, bits = bnn.bnn_fconv2d_binw(desc, xd, d["w"], d["thr"], d.get("flip"),
                                               want_sums=False)
            else:
                _, bits = _conv(desc, pack_pm1(outs[li - 1]), d, algo, False)
            torch.cuda.synchronize()
            assert np.array_equal(words_u32(bits), _packed(outs[li])), "layer %d" % li
            # the fused kernels bnn_forward runs for the first two layers
            if li == 1 and layers[0]["kind"] == "fconv" and algo != "valu":
                d0 = bnn.conv_desc(N, H, W, C, layers[0]["F"], 3, 3, 1, layers[0]["pad"], 0)
                fb = bnn.bnn_fconv_bconv2d(d0, desc, xd, dev[0]["w"], dev[0]["thr"],
                                           dev[0].get("flip"), d["w"], d["thr"], d.get("flip"),
                                           w1prep=d["wprep"] if algo == "prep" else None)
                torch.cuda.synchronize()
                assert np.array_equal(words_u32(fb), _packed(outs[li])), "fused L0+L1"
            if li == 1 and layers[0]["kind"] == "input_threshold":
                _, pb = bnn.bnn_bconv2d_input(desc, bnn.INPUT_THRESHOLD, xd, dev[0]["offset"],
                                              d["w"], d["thr"], d.get("flip"), want_sums=False)
                torch.cuda.synchronize()
                assert np.array_equal(words_u32(pb), _packed(outs[li])), "patch L0+L1"
            # the conv pair bnn_forward runs as one kernel (bnn_bconv_bconv2d)
            p = descs.get(li - 1)
            if (k == "bconv" and p is not None and layers[li - 1]["kind"] == "bconv"
                    and algo != "valu" and _pair_fusable(layers[li - 1], L, p.W, p.C)):
                dp = dev[li - 1]
                pb = bnn.bnn_bconv_bconv2d(p, desc, pack_pm1(outs[li - 2]), dp["w"], dp["thr"],
                                           dp.get("flip"), d["w"], d["thr"], d.get("flip"))
                torch.cuda.synchronize()
                assert np.array_equal(words_u32(pb), _packed(outs[li])), "fused pair %d" % li
            descs[li] = desc
            Ho, Wo, Hp, Wp = bnn.bnn_conv_output_dims(desc)
            h, w = Hp, Wp
            continue
        src = pack_pm1(outs[li - 1].reshape(N, -1))
        if k == "bfc":
            _, bits = bnn.bnn_bgemm(src, d["w"], L["K"], d["thr"], d.get("flip"),
                                    want_sums=False)
            torch.cuda.synchronize()
            assert np.array_equal(words_u32(bits), _packed(outs[li])), "layer %d" % li
        else:
            sums, _ = bnn.bnn_bgemm(src, d["w"], L["K"], want_bits=False)
            torch.cuda.synchronize()
            assert np.array_equal(sums.cpu().numpy(), outs[li]), "logits"
        # the FC tail bnn_forward runs as one kernel (bnn_bfc_tail)
        P = layers[li - 1]
        if (P["kind"] == "bfc" and L["N"] <= 32 and algo != "valu" and N <= 512
                and P["K"] % 1024 == 0 and P["N"] % 32 == 0
                and ((N + 31) // 32) * (P["N"] // 32) <= 512):
            dp = dev[li - 1]
            lg = k == "bfc_logits"
            tb = bnn.bnn_bfc_tail(pack_pm1(outs[li - 2].reshape(N, -1)), P["K"], dp["w"],
                                  dp["thr"], dp.get("flip"), d["w"], L["N"], bnn.accum_buffer(),
                                  None if lg else d["thr"], None if lg else d.get("flip"))
            torch.cuda.synchronize()
            if lg:
                assert np.array_equal(tb.cpu().numpy(), outs[li]), "FC tail"
            else:
                assert np.array_equal(words_u32(tb), _packed(outs[li])), "FC tail"
