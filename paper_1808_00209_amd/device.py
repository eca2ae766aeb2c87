"""Moving seeded host data onto the GPU in the library's packed layout.

+-1 int8 host arrays are copied to the device as fp32 and packed there by
``bnn_pack_bits`` (the library's own packing kernel); 0/1 flip bits are
packed the same way.  Used by the tests, the benchmark and the smoke check.
"""
from __future__ import annotations

import numpy as np
import torch

from . import bnn


def to_device(a, dtype=None, device="cuda"):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.to(device)


def pack_pm1(a, device="cuda"):
    """+-1 int8 array [..., D] -> packed words on the device (int32 storage)."""
    x = to_device(a, torch.float32, device)
    return bnn.bnn_pack_bits(x)


def pack_flips(flip, device="cuda"):
    """0/1 per channel -> packed flip words [ceil(F/32)]."""
    pm = np.where(np.asarray(flip) != 0, 1, -1).astype(np.int8)
    return pack_pm1(pm, device)


def upload_layer(L, device="cuda", prepare=True):
    """A host layer dict (see synth) -> device tensors + C-struct fields.
    Binary conv layers also get their weights in the prepared operand form
    (bnn_prepare_weights) unless ``prepare`` is False."""
    kind = L["kind"]
    d = {}
    if kind in ("input_threshold", "input_gray", "input_lbp"):
        d.update(kind={"input_threshold": bnn.LAYER_INPUT_THRESHOLD,
                       "input_gray": bnn.LAYER_INPUT_GRAY,
                       "input_lbp": bnn.LAYER_INPUT_LBP}[kind], C=L["C"])
        if L.get("offset") is not None:
            d["offset"] = to_device(L["offset"], torch.float32, device)
        return d
    if kind in ("fconv", "bconv"):
        d.update(kind=bnn.LAYER_FCONV_BINW if kind == "fconv" else bnn.LAYER_BCONV,
                 C=L["C"], F=L["F"], KH=L["KH"], KW=L["KW"], stride=L.get("stride", 1),
                 pad=L["pad"], pool=L.get("pool", 0))
    else:
        d.update(kind=bnn.LAYER_BFC if kind == "bfc" else bnn.LAYER_BFC_LOGITS,
                 K=L["K"], N=L["N"])
    d["w"] = pack_pm1(L["w"], device)
    if prepare and kind == "bconv":
        d["wprep"] = bnn.bnn_prepare_weights(d["w"], L["F"], L["KH"], L["KW"], L["C"])
    if L.get("thr") is not None:
        d["thr"] = to_device(L["thr"], torch.int32, device)
    if L.get("flip") is not None:
        d["flip"] = pack_flips(L["flip"], device)
    return d


def upload_network(layers, H, W, C, device="cuda", prepare=True):
    return bnn.Network([upload_layer(L, device, prepare) for L in layers], H, W, C)


def words_u32(t) -> np.ndarray:
    """Device packed words (int32 storage) -> host uint32 array."""
    return t.cpu().numpy().view(np.uint32)
