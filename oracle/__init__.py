"""CPU oracle for binarized conv / FC inference -- TEST INFRASTRUCTURE ONLY.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The product library never links or calls it, and it
imports nothing from the product package.

Binary values are int8 arrays holding -1/+1; sums are int32 (binary layers) or
fp64 (the real-valued first layer).  The arithmetic lives in ``bnn_oracle.c``
(plain direct loops, OpenMP over independent outputs); this module marshals
numpy arrays and composes a layer chain.  Each function names the passage of
the paper (Khan et al., EUSIPCO 2018) it follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "bnn_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile ``bnn_oracle.c`` with gcc (-O2, OpenMP) into ``liboracle.so``."""
    if force or not os.path.exists(_LIB_PATH) or (
            os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC)):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared",
                               "-std=c11", "-Wall", "-ffp-contract=off", "-o", tmp, _SRC])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _bind(path: str):
    """Load an oracle shared library at ``path`` and declare its signatures."""
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    i32, i64 = ctypes.c_int32, ctypes.c_int64
    lib.orc_sign.argtypes = [P, P, i64, i64, P]
    lib.orc_pack_eq2.argtypes = [P, i64, i64, i32, P]
    lib.orc_conv2d.argtypes = [P, P] + [i32] * 9 + [P]
    lib.orc_conv2d_at.argtypes = [P, P] + [i32] * 7 + [P, i64, P]
    lib.orc_fconv2d.argtypes = [P, P] + [i32] * 9 + [P]
    lib.orc_fc.argtypes = [P, P, i64, i64, i64, P]
    lib.orc_threshold.argtypes = [P, P, P, i64, i64, P]
    lib.orc_threshold_f64.argtypes = [P, P, P, i64, i64, P]
    lib.orc_maxpool2.argtypes = [P, i32, i32, i32, i32, P]
    lib.orc_gray_threshold.argtypes = [P, ctypes.c_float, i64, P]
    lib.orc_lbp.argtypes = [P, i32, i32, i32, P]
    lib.orc_num_threads.restype = ctypes.c_int
    return lib


def _load():
    """Load liboracle.so (building it if needed).  ``BNN_ORACLE_LIB`` names
    another build instead: the mutation tests plant a mistake in a copy of the
    C source and check that the pins catch it."""
    global _lib
    if _lib is None:
        alt = os.environ.get("BNN_ORACLE_LIB")
        if alt:
            _lib = _bind(alt)
        else:
            build()
            _lib = _bind(_LIB_PATH)
    return _lib


def _c(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data


def _pm1(a):
    a = np.ascontiguousarray(a, dtype=np.int8)
    if a.size and not np.all((a == 1) | (a == -1)):
        raise ValueError("oracle binary inputs must hold only -1/+1")
    return a, a.ctypes.data


def num_threads() -> int:
    return int(_load().orc_num_threads())


def sign(x, offset=None):
    """Eq. (1) on ``x + offset`` (Sec. II-C thresholding), fp32 add. [rows, D]"""
    lib = _load()
    x, xp = _c(x, np.float32)
    D = x.shape[-1] if x.ndim else 1
    rows = x.size // D if D else 0
    op = None
    if offset is not None:
        offset, op = _c(offset, np.float32)
        assert offset.shape == (D,)
    out = np.empty(x.shape, np.int8)
    lib.orc_sign(xp, op, rows, D, out.ctypes.data)
    return out


def pack_eq2(x, B: int = 32):
    """Eq. (2): pack each row of +-1 values into ceil(D/B) words."""
    lib = _load()
    x, xp = _pm1(x)
    D = x.shape[-1]
    rows = x.size // D if D else 0
    out = np.zeros(x.shape[:-1] + ((D + B - 1) // B,), np.uint32)
    lib.orc_pack_eq2(xp, rows, D, B, out.ctypes.data)
    return out


def conv_out_size(H, K, stride, pad):
    return (H + 2 * pad - K) // stride + 1


def conv2d(x, w, stride: int = 1, pad: int = 0):
    """Eq. (3) over +-1 values, pad value -1.  x [N,H,W,C], w [F,KH,KW,C]."""
    lib = _load()
    x, xp = _pm1(x)
    w, wp = _pm1(w)
    N, H, W, C = x.shape
    F, KH, KW, C2 = w.shape
    assert C == C2
    Ho, Wo = conv_out_size(H, KH, stride, pad), conv_out_size(W, KW, stride, pad)
    out = np.empty((N, Ho, Wo, F), np.int32)
    lib.orc_conv2d(xp, wp, N, H, W, C, F, KH, KW, stride, pad, out.ctypes.data)
    return out


def conv2d_at(x, w, idx, stride: int = 1, pad: int = 0):
    """Eq. (3) at output coordinates idx [count, 4] = (n, i, j, f)."""
    lib = _load()
    x, xp = _pm1(x)
    w, wp = _pm1(w)
    N, H, W, C = x.shape
    F, KH, KW, _ = w.shape
    idx, ip = _c(idx, np.int64)
    assert idx.ndim == 2 and idx.shape[1] == 4
    out = np.empty(idx.shape[0], np.int32)
    lib.orc_conv2d_at(xp, wp, H, W, C, KH, KW, stride, pad, ip, idx.shape[0],
                      out.ctypes.data)
    return out


def fconv2d(x, w, stride: int = 1, pad: int = 0):
    """Eq. (3) for an fp32 image and +-1 weights, pad 0.0, fp64 sums."""
    lib = _load()
    x, xp = _c(x, np.float32)
    w, wp = _pm1(w)
    N, H, W, C = x.shape
    F, KH, KW, _ = w.shape
    Ho, Wo = conv_out_size(H, KH, stride, pad), conv_out_size(W, KW, stride, pad)
    out = np.empty((N, Ho, Wo, F), np.float64)
    lib.orc_fconv2d(xp, wp, N, H, W, C, F, KH, KW, stride, pad, out.ctypes.data)
    return out


def fc(a, b):
    """Sec. III-B: S[m,n] = sum_k a[m,k] b[n,k] over +-1 values."""
    lib = _load()
    a, ap = _pm1(a)
    b, bp = _pm1(b)
    M, K = a.shape
    N, K2 = b.shape
    assert K == K2
    out = np.empty((M, N), np.int32)
    lib.orc_fc(ap, bp, M, N, K, out.ctypes.data)
    return out


def threshold(S, thr, flip=None):
    """bit = (S >= thr) XOR flip, returned as +-1; S [..., F] int32 or fp64."""
    lib = _load()
    F = S.shape[-1]
    thr, tp = _c(thr, np.int32)
    fp = None
    if flip is not None:
        flip, fp = _c(flip, np.uint8)
    out = np.empty(S.shape, np.int8)
    P = S.size // F if F else 0
    if np.issubdtype(S.dtype, np.floating):
        S, sp = _c(S, np.float64)
        lib.orc_threshold_f64(sp, tp, fp, P, F, out.ctypes.data)
    else:
        S, sp = _c(S, np.int32)
        lib.orc_threshold(sp, tp, fp, P, F, out.ctypes.data)
    return out


def maxpool2(x):
    """2x2 / stride 2 max over +-1 values (Table II pooling rows)."""
    lib = _load()
    x, xp = _pm1(x)
    N, H, W, C = x.shape
    out = np.empty((N, H // 2, W // 2, C), np.int8)
    lib.orc_maxpool2(xp, N, H, W, C, out.ctypes.data)
    return out


def gray_threshold(x, T):
    """Grayscale thresholding (Table III): sign(gray(x) + T), fp32.
    x [..., 3] RGB -> [..., 1] +-1."""
    lib = _load()
    x, xp = _c(x, np.float32)
    assert x.shape[-1] == 3
    rows = x.size // 3
    out = np.empty(x.shape[:-1] + (1,), np.int8)
    lib.orc_gray_threshold(xp, float(T), rows, out.ctypes.data)
    return out


def lbp(x):
    """LBP input binarization (Sec. II-C): x [N,H,W,3] RGB -> [N,H,W,3] +-1."""
    lib = _load()
    x, xp = _c(x, np.float32)
    N, H, W, C = x.shape
    assert C == 3
    out = np.empty((N, H, W, 3), np.int8)
    lib.orc_lbp(xp, N, H, W, out.ctypes.data)
    return out


def forward(layers, x, return_all: bool = False):
    """Run a layer chain (Table II order: conv, pool, ..., FC) on ``x``.

    ``layers`` is a list of dicts (kinds: input_threshold, input_gray,
    input_lbp, fconv, bconv, bfc, bfc_logits) holding +-1 int8 weights, int32 thresholds and 0/1 flips.
    Conv activations are NHWC; FC layers flatten them in (h, w, c) order.
    Returns the int32 logits of the last layer (and every intermediate, on
    request, as +-1 arrays or sums).
    """
    a = np.ascontiguousarray(x, np.float32)
    trace = []
    for L in layers:
        k = L["kind"]
        if k == "input_threshold":
            a = sign(a, L.get("offset"))
        elif k == "input_gray":
            a = gray_threshold(a, float(L["offset"][0]))
        elif k == "input_lbp":
            a = lbp(a)
        elif k in ("fconv", "bconv"):
            conv = fconv2d if k == "fconv" else conv2d
            S = conv(a, L["w"], L.get("stride", 1), L["pad"])
            a = threshold(S, L["thr"], L.get("flip"))
            if L.get("pool", 0):
                a = maxpool2(a)
            trace.append(S)
        elif k in ("bfc", "bfc_logits"):
            a2 = a.reshape(a.shape[0], -1)
            S = fc(a2, L["w"])
            trace.append(S)
            if k == "bfc_logits":
                a = S
            else:
                a = threshold(S, L["thr"], L.get("flip"))
        else:
            raise ValueError("unknown layer kind %r" % k)
        trace.append(a)
    return (a, trace) if return_all else a
