"""ctypes binding of libbnn.so (C ABI in include/bnn.h).

Argument marshalling only: every function checks tensor dtypes, devices and
contiguity, allocates outputs with torch when the caller does not pass them,
and calls the C entry point of the same name on the current HIP stream.  All
computation happens in the library's HIP kernels.  Loading fails loudly when
libbnn.so has not been built (``python -m paper_1808_00209_amd.build``).
"""
from __future__ import annotations

import contextlib
import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libbnn.so")

BNN_OK = 0
STATUS_NAMES = {0: "BNN_OK", 1: "BNN_ERR_NULL", 2: "BNN_ERR_SHAPE", 3: "BNN_ERR_ALIGN",
                4: "BNN_ERR_UNSUPPORTED", 5: "BNN_ERR_HIP", 6: "BNN_ERR_WORKSPACE"}

LAYER_INPUT_THRESHOLD = 1
LAYER_FCONV_BINW = 2
LAYER_BCONV = 3
LAYER_BFC = 4
LAYER_BFC_LOGITS = 5
LAYER_INPUT_GRAY = 6
LAYER_INPUT_LBP = 7
INPUT_THRESHOLD = 0
INPUT_GRAY = 1
INPUT_LBP = 2

# Every symbol include/bnn.h declares.
EXPORTED = ["bnn_last_error", "bnn_abi_version", "bnn_default_options", "bnn_set_options",
            "bnn_get_options", "bnn_pack_bits", "bnn_conv_output_dims",
            "bnn_bconv2d", "bnn_prepared_weights_size", "bnn_prepare_weights",
            "bnn_bconv2d_prepared", "bnn_fconv2d_binw", "bnn_binarize_input", "bnn_bconv2d_input",
            "bnn_fconv_bconv2d", "bnn_input_bconv_bconv2d", "bnn_bconv_bconv2d", "bnn_bfc_pair", "bnn_bfc_tail",
            "bnn_bgemm",
            "bnn_forward_workspace_size", "bnn_forward", "bnn_forward_noalloc"]

# Bytes of bnn_forward_noalloc's per-GPU scratch array (BNN_FORWARD_SCRATCH_BYTES).
FORWARD_SCRATCH_BYTES = 64 << 20
# Leading workspace bytes that must be zero before a workspace's first use
# (BNN_FORWARD_SYNC_BYTES: the FC tail kernel's accumulators, left zero by every call).
FORWARD_SYNC_BYTES = 69632


class BnnError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__("%s: %s" % (STATUS_NAMES.get(status, status), message))
        self.status = status


ALGO_AUTO = 0
ALGO_VALU = 1


class Options(ctypes.Structure):
    """bnn_options: the calling thread's kernel selection (never changes a result)."""
    _fields_ = [(n, ctypes.c_int32) for n in
                ("algo", "fuse_input", "fuse_first", "fc_chain", "conv1x1", "xcd_order",
                 "gemv_max_rows", "lds_weights", "late_thresholds", "fuse_pair")]


class ConvDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("N", "H", "W", "C", "F", "KH", "KW", "stride", "pad", "pool")]


class Layer(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("C", ctypes.c_int32), ("F", ctypes.c_int32),
                ("KH", ctypes.c_int32), ("KW", ctypes.c_int32), ("stride", ctypes.c_int32),
                ("pad", ctypes.c_int32), ("pool", ctypes.c_int32), ("K", ctypes.c_int32),
                ("N", ctypes.c_int32), ("w", ctypes.c_void_p), ("thr", ctypes.c_void_p),
                ("flip", ctypes.c_void_p), ("offset", ctypes.c_void_p), ("wprep", ctypes.c_void_p)]


_lib = None


def load(path: str = LIB_PATH):
    """Load libbnn.so and declare the C signatures (raises if it is missing)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError("libbnn.so not found at %s: build it with "
                           "`python -m paper_1808_00209_amd.build` (no fallback exists)" % path)
    lib = ctypes.CDLL(path)
    P, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.bnn_last_error.restype = ctypes.c_char_p
    lib.bnn_last_error.argtypes = []
    lib.bnn_abi_version.restype = i32
    lib.bnn_abi_version.argtypes = []
    lib.bnn_default_options.restype = None
    lib.bnn_default_options.argtypes = [ctypes.POINTER(Options)]
    lib.bnn_set_options.argtypes = [ctypes.POINTER(Options)]
    lib.bnn_get_options.argtypes = [ctypes.POINTER(Options)]
    lib.bnn_pack_bits.argtypes = [P, P, i64, i64, P, P]
    lib.bnn_conv_output_dims.argtypes = [ctypes.POINTER(ConvDesc)] + [ctypes.POINTER(i32)] * 4
    lib.bnn_bconv2d.argtypes = [ctypes.POINTER(ConvDesc), P, P, P, P, P, P, P]
    lib.bnn_prepared_weights_size.argtypes = [i32, i32, i32, i32, ctypes.POINTER(ctypes.c_size_t)]
    lib.bnn_prepare_weights.argtypes = [i32, i32, i32, i32, P, P, P]
    lib.bnn_bconv2d_prepared.argtypes = [ctypes.POINTER(ConvDesc), P, P, P, P, P, P, P, P]
    lib.bnn_fconv2d_binw.argtypes = [ctypes.POINTER(ConvDesc), P, P, P, P, P, P, P]
    lib.bnn_bgemm.argtypes = [i64, i64, i64, P, P, P, P, P, P, P]
    lib.bnn_binarize_input.argtypes = [i32, P, P, i32, i32, i32, i32, P, P]
    lib.bnn_bconv2d_input.argtypes = [ctypes.POINTER(ConvDesc), i32, P, P, P, P, P, P, P, P]
    lib.bnn_fconv_bconv2d.argtypes = [ctypes.POINTER(ConvDesc), ctypes.POINTER(ConvDesc),
                                      P, P, P, P, P, P, P, P, P, P]
    lib.bnn_input_bconv_bconv2d.argtypes = [ctypes.POINTER(ConvDesc), ctypes.POINTER(ConvDesc),
                                            i32, P, P, P, P, P, P, P, P, P, P, P]
    lib.bnn_bconv_bconv2d.argtypes = [ctypes.POINTER(ConvDesc), ctypes.POINTER(ConvDesc),
                                      P, P, P, P, P, P, P, P, P]
    lib.bnn_bfc_pair.argtypes = [i64, i64, i64, i64, P, P, P, P, P, P, P, P, P, P]
    lib.bnn_bfc_tail.argtypes = [i64, i64, i64, i64, P, P, P, P, P, P, P, P, P, P, P]
    lib.bnn_forward_workspace_size.argtypes = [ctypes.POINTER(Layer), i32, i32, i32, i32, i32,
                                               ctypes.POINTER(ctypes.c_size_t)]
    lib.bnn_forward.argtypes = [ctypes.POINTER(Layer), i32, i32, i32, i32, i32, P, P,
                                ctypes.c_size_t, P, P]
    lib.bnn_forward_noalloc.argtypes = [ctypes.POINTER(Layer), i32, i32, i32, i32, i32, P, P, P]
    for name in EXPORTED:
        if name not in ("bnn_last_error", "bnn_abi_version", "bnn_default_options"):
            getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def last_error() -> str:
    return load().bnn_last_error().decode()


def _check(status: int):
    if status != BNN_OK:
        raise BnnError(status, last_error())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dev(t, dtype, name):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or t.dtype != dtype or not t.is_cuda:
        raise TypeError("%s must be a CUDA(HIP) tensor of %s" % (name, dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    return t


def words(bits: int) -> int:
    return (bits + 31) // 32


def _u32(t):
    """torch has no uint32 arithmetic; packed words travel as int32 storage."""
    return _dev(t, torch.int32, "packed words")


# ---------------------------------------------------------------- options ---
def bnn_default_options() -> Options:
    o = Options()
    load().bnn_default_options(ctypes.byref(o))
    return o


def bnn_get_options() -> Options:
    o = Options()
    _check(load().bnn_get_options(ctypes.byref(o)))
    return o


def bnn_set_options(opt: Options = None, **fields) -> Options:
    """Set the calling thread's options: ``opt`` (default: the library
    defaults) with ``fields`` replaced.  Returns the options in force before."""
    prev = bnn_get_options()
    o = Options.from_buffer_copy(opt) if opt is not None else bnn_default_options()
    for k, v in fields.items():
        if k not in dict(Options._fields_):
            raise KeyError("unknown option %r" % k)
        setattr(o, k, int(v))
    _check(load().bnn_set_options(ctypes.byref(o)))
    return prev


@contextlib.contextmanager
def options(**fields):
    """``with bnn.options(algo=bnn.ALGO_VALU): ...`` -- the defaults with
    ``fields`` replaced, restored to what was in force on exit."""
    prev = bnn_set_options(None, **fields)
    try:
        yield
    finally:
        _check(load().bnn_set_options(ctypes.byref(prev)))


# ------------------------------------------------------------------ calls ---
def bnn_pack_bits(x, offset=None, out=None, stream=None):
    """Eq. (1)+(2): x [..., D] fp32 -> packed words [..., ceil(D/32)] (int32 storage)."""
    lib = load()
    x = _dev(x, torch.float32, "x")
    D = x.shape[-1]
    rows = x.numel() // D if D else 0
    if offset is not None:
        offset = _dev(offset, torch.float32, "offset")
    if out is None:
        out = torch.empty(tuple(x.shape[:-1]) + (words(D),), dtype=torch.int32, device=x.device)
    _u32(out)
    _check(lib.bnn_pack_bits(_ptr(x), _ptr(offset), rows, D, _ptr(out), _stream(stream)))
    return out


def conv_desc(N, H, W, C, F, KH=3, KW=3, stride=1, pad=1, pool=0) -> ConvDesc:
    return ConvDesc(N, H, W, C, F, KH, KW, stride, pad, pool)


def bnn_conv_output_dims(desc: ConvDesc):
    lib = load()
    o = [ctypes.c_int32() for _ in range(4)]
    _check(lib.bnn_conv_output_dims(ctypes.byref(desc), *[ctypes.byref(v) for v in o]))
    return tuple(v.value for v in o)


def bnn_bconv2d(desc: ConvDesc, x, w, thr=None, flip=None, want_sums=True, want_bits=True,
                out_sums=None, out_bits=None, stream=None):
    """Binary conv (Eq. 3/4) with fused threshold/flip/OR-pool.  Returns
    (sums [N,Ho,Wo,F] int32 or None, bits [N,Hp,Wp,Fw] int32-storage or None)."""
    lib = load()
    Ho, Wo, Hp, Wp = bnn_conv_output_dims(desc)
    _u32(x)
    _u32(w)
    thr = _dev(thr, torch.int32, "thr")
    flip = _dev(flip, torch.int32, "flip")
    if want_sums and out_sums is None:
        out_sums = torch.empty((desc.N, Ho, Wo, desc.F), dtype=torch.int32, device=x.device)
    if want_bits and out_bits is None:
        out_bits = torch.empty((desc.N, Hp, Wp, words(desc.F)), dtype=torch.int32,
                               device=x.device)
    _check(lib.bnn_bconv2d(ctypes.byref(desc), _ptr(x), _ptr(w), _ptr(thr), _ptr(flip),
                           _ptr(out_sums), _ptr(out_bits), _stream(stream)))
    return out_sums, out_bits


def bnn_prepared_weights_size(F, KH, KW, C) -> int:
    out = ctypes.c_size_t()
    _check(load().bnn_prepared_weights_size(F, KH, KW, C, ctypes.byref(out)))
    return out.value


def bnn_prepare_weights(w, F, KH, KW, C, out=None, stream=None):
    """Packed conv weights [F, KH, KW, ceil(C/32)] -> the matrix-core operand
    form (a uint8 device buffer of bnn_prepared_weights_size bytes)."""
    lib = load()
    _u32(w)
    if out is None:
        out = torch.empty(bnn_prepared_weights_size(F, KH, KW, C), dtype=torch.uint8,
                          device=w.device)
    _check(lib.bnn_prepare_weights(F, KH, KW, C, _ptr(w), _ptr(out), _stream(stream)))
    return out


def bnn_bconv2d_prepared(desc: ConvDesc, x, w, wprep, thr=None, flip=None, want_sums=True,
                         want_bits=True, out_sums=None, out_bits=None, stream=None):
    """bnn_bconv2d with prepared weights (wprep = bnn_prepare_weights of w)."""
    lib = load()
    Ho, Wo, Hp, Wp = bnn_conv_output_dims(desc)
    _u32(x)
    _u32(w)
    _dev(wprep, torch.uint8, "wprep")
    thr = _dev(thr, torch.int32, "thr")
    flip = _dev(flip, torch.int32, "flip")
    if want_sums and out_sums is None:
        out_sums = torch.empty((desc.N, Ho, Wo, desc.F), dtype=torch.int32, device=x.device)
    if want_bits and out_bits is None:
        out_bits = torch.empty((desc.N, Hp, Wp, words(desc.F)), dtype=torch.int32,
                               device=x.device)
    _check(lib.bnn_bconv2d_prepared(ctypes.byref(desc), _ptr(x), _ptr(w), _ptr(wprep), _ptr(thr),
                                    _ptr(flip), _ptr(out_sums), _ptr(out_bits),
                                    _stream(stream)))
    return out_sums, out_bits


def bnn_fconv2d_binw(desc: ConvDesc, x, w, thr=None, flip=None, want_sums=True,
                     want_bits=True, out_sums=None, out_bits=None, stream=None):
    """fp32-input conv with packed +-1 weights; sums fp32 [N,Ho,Wo,F]."""
    lib = load()
    Ho, Wo, Hp, Wp = bnn_conv_output_dims(desc)
    _dev(x, torch.float32, "x")
    _u32(w)
    thr = _dev(thr, torch.int32, "thr")
    flip = _dev(flip, torch.int32, "flip")
    if want_sums and out_sums is None:
        out_sums = torch.empty((desc.N, Ho, Wo, desc.F), dtype=torch.float32, device=x.device)
    if want_bits and out_bits is None:
        out_bits = torch.empty((desc.N, Hp, Wp, words(desc.F)), dtype=torch.int32,
                               device=x.device)
    _check(lib.bnn_fconv2d_binw(ctypes.byref(desc), _ptr(x), _ptr(w), _ptr(thr), _ptr(flip),
                                _ptr(out_sums), _ptr(out_bits), _stream(stream)))
    return out_sums, out_bits


def bnn_binarize_input(mode, x, offset=None, out=None, stream=None):
    """Input binarization (Sec. II-C): mode INPUT_THRESHOLD / INPUT_GRAY /
    INPUT_LBP on x [N,H,W,Cin] fp32 -> one code word per pixel [N,H,W,1]."""
    lib = load()
    _dev(x, torch.float32, "x")
    offset = _dev(offset, torch.float32, "offset")
    N, H, W, Cin = x.shape
    if out is None:
        out = torch.empty((N, H, W, 1), dtype=torch.int32, device=x.device)
    _check(lib.bnn_binarize_input(int(mode), _ptr(x), _ptr(offset), N, H, W, Cin, _ptr(out),
                                  _stream(stream)))
    return out


def bnn_bconv2d_input(desc: ConvDesc, mode, x, offset, w, thr=None, flip=None, want_sums=True,
                      want_bits=True, out_sums=None, out_bits=None, stream=None):
    """Binary conv over an fp32 image binarized on the fly by ``mode`` (Sec. II-C),
    each window packed into ceil(KH*KW*C / 32) words (Algorithm 1's patch
    packing).  desc.C is the binarized channel count.  Same outputs as
    bnn_binarize_input / bnn_pack_bits followed by bnn_bconv2d."""
    lib = load()
    Ho, Wo, Hp, Wp = bnn_conv_output_dims(desc)
    _dev(x, torch.float32, "x")
    offset = _dev(offset, torch.float32, "offset")
    _u32(w)
    thr = _dev(thr, torch.int32, "thr")
    flip = _dev(flip, torch.int32, "flip")
    if want_sums and out_sums is None:
        out_sums = torch.empty((desc.N, Ho, Wo, desc.F), dtype=torch.int32, device=x.device)
    if want_bits and out_bits is None:
        out_bits = torch.empty((desc.N, Hp, Wp, words(desc.F)), dtype=torch.int32,
                               device=x.device)
    _check(lib.bnn_bconv2d_input(ctypes.byref(desc), int(mode), _ptr(x), _ptr(offset), _ptr(w),
                                 _ptr(thr), _ptr(flip), _ptr(out_sums), _ptr(out_bits),
                                 _stream(stream)))
    return out_sums, out_bits


def bnn_fconv_bconv2d(desc0: ConvDesc, desc1: ConvDesc, x, w0, thr0, flip0, w1, thr1,
                      flip1=None, out_bits=None, stream=None, w1prep=None):
    """The real-valued first layer and a binary 3x3 conv over its bits in one
    launch (the first two layers of Table I's BCNN): returns the second
    layer's packed bits [N, Hp, Wp, F1/32], the same as bnn_fconv2d_binw
    followed by bnn_bconv2d.  w1prep: bnn_prepare_weights of w1, or None."""
    lib = load()
    _, _, Hp, Wp = bnn_conv_output_dims(desc1)
    _dev(x, torch.float32, "x")
    _u32(w0)
    _u32(w1)
    thr0 = _dev(thr0, torch.int32, "thr0")
    thr1 = _dev(thr1, torch.int32, "thr1")
    flip0 = _dev(flip0, torch.int32, "flip0")
    flip1 = _dev(flip1, torch.int32, "flip1")
    if out_bits is None:
        out_bits = torch.empty((desc1.N, Hp, Wp, words(desc1.F)), dtype=torch.int32,
                               device=x.device)
    _dev(w1prep, torch.uint8, "w1prep")
    _check(lib.bnn_fconv_bconv2d(ctypes.byref(desc0), ctypes.byref(desc1), _ptr(x), _ptr(w0),
                                 _ptr(thr0), _ptr(flip0), _ptr(w1), _ptr(w1prep), _ptr(thr1),
                                 _ptr(flip1), _ptr(out_bits), _stream(stream)))
    return out_bits


def bnn_input_bconv_bconv2d(desc0: ConvDesc, desc1: ConvDesc, mode, x, offset, w0, thr0, flip0,
                            w1, thr1, flip1=None, out_bits=None, stream=None, w1prep=None):
    """Input thresholding, a binary 3x3 conv and a binary 3x3 conv over its
    bits in one launch: returns the second conv's packed bits
    [N, Hp, Wp, F1/32], the same as bnn_bconv2d_input followed by
    bnn_bconv2d.  w1prep: bnn_prepare_weights of w1, or None."""
    lib = load()
    _, _, Hp, Wp = bnn_conv_output_dims(desc1)
    _dev(x, torch.float32, "x")
    offset = _dev(offset, torch.float32, "offset")
    _u32(w0)
    _u32(w1)
    thr0 = _dev(thr0, torch.int32, "thr0")
    thr1 = _dev(thr1, torch.int32, "thr1")
    flip0 = _dev(flip0, torch.int32, "flip0")
    flip1 = _dev(flip1, torch.int32, "flip1")
    if out_bits is None:
        out_bits = torch.empty((desc1.N, Hp, Wp, words(desc1.F)), dtype=torch.int32,
                               device=x.device)
    _dev(w1prep, torch.uint8, "w1prep")
    _check(lib.bnn_input_bconv_bconv2d(ctypes.byref(desc0), ctypes.byref(desc1), int(mode),
                                       _ptr(x), _ptr(offset), _ptr(w0), _ptr(thr0), _ptr(flip0),
                                       _ptr(w1), _ptr(w1prep), _ptr(thr1), _ptr(flip1),
                                       _ptr(out_bits), _stream(stream)))
    return out_bits


def bnn_bconv_bconv2d(desc0: ConvDesc, desc1: ConvDesc, x, w0, thr0, flip0, w1, thr1,
                      flip1=None, out_bits=None, stream=None):
    """Two binary 3x3 convs in one launch, the first conv's bits kept on
    chip: returns the second conv's packed bits [N, Hp, Wp, F1/32], the same
    as bnn_bconv2d(desc0) followed by bnn_bconv2d(desc1)."""
    lib = load()
    _, _, Hp, Wp = bnn_conv_output_dims(desc1)
    _u32(x)
    _u32(w0)
    _u32(w1)
    thr0 = _dev(thr0, torch.int32, "thr0")
    thr1 = _dev(thr1, torch.int32, "thr1")
    flip0 = _dev(flip0, torch.int32, "flip0")
    flip1 = _dev(flip1, torch.int32, "flip1")
    if out_bits is None:
        out_bits = torch.empty((desc1.N, Hp, Wp, words(desc1.F)), dtype=torch.int32,
                               device=x.device)
    _check(lib.bnn_bconv_bconv2d(ctypes.byref(desc0), ctypes.byref(desc1), _ptr(x), _ptr(w0),
                                 _ptr(thr0), _ptr(flip0), _ptr(w1), _ptr(thr1), _ptr(flip1),
                                 _ptr(out_bits), _stream(stream)))
    return out_bits


def bnn_bfc_pair(A, K0, w0, thr0, flip0, w1, N1, thr1=None, flip1=None, out=None,
                 stream=None):
    """Two binary FC layers in one launch: layer 0 (K0 -> N0 outputs, its
    threshold and flip) then layer 1 (N0 -> N1 <= 32).  With thr1 None the
    result is layer 1's int32 sums [M, N1]; otherwise its bits [M, 1].  The
    same as two bnn_bgemm calls."""
    lib = load()
    _u32(A)
    _u32(w0)
    _u32(w1)
    M, N0 = A.shape[0], w0.shape[0]
    thr0 = _dev(thr0, torch.int32, "thr0")
    flip0 = _dev(flip0, torch.int32, "flip0")
    thr1 = _dev(thr1, torch.int32, "thr1")
    flip1 = _dev(flip1, torch.int32, "flip1")
    if out is None:
        out = torch.empty((M, N1) if thr1 is None else (M, 1), dtype=torch.int32, device=A.device)
    _check(lib.bnn_bfc_pair(M, K0, N0, N1, _ptr(A), _ptr(w0), _ptr(thr0), _ptr(flip0), _ptr(w1),
                            _ptr(thr1), _ptr(flip1), _ptr(out) if thr1 is None else None,
                            None if thr1 is None else _ptr(out), _stream(stream)))
    return out


def bnn_bfc_tail(A, K0, w0, thr0, flip0, w1, N1, accum, thr1=None, flip1=None, out=None,
                 stream=None):
    """The FC tail kernel: the same two layers as bnn_bfc_pair, spread over
    layer 0's 32 x 32 output tiles, layer 1's partial sums added in `accum`
    (FORWARD_SYNC_BYTES, zero on entry and left zero: see accum_buffer)."""
    lib = load()
    _u32(A)
    _u32(w0)
    _u32(w1)
    M, N0 = A.shape[0], w0.shape[0]
    thr0 = _dev(thr0, torch.int32, "thr0")
    flip0 = _dev(flip0, torch.int32, "flip0")
    thr1 = _dev(thr1, torch.int32, "thr1")
    flip1 = _dev(flip1, torch.int32, "flip1")
    if out is None:
        out = torch.empty((M, N1) if thr1 is None else (M, 1), dtype=torch.int32, device=A.device)
    _check(lib.bnn_bfc_tail(M, K0, N0, N1, _ptr(A), _ptr(w0), _ptr(thr0), _ptr(flip0), _ptr(w1),
                            _ptr(thr1), _ptr(flip1), _ptr(out) if thr1 is None else None,
                            None if thr1 is None else _ptr(out), _ptr(accum), _stream(stream)))
    return out


def accum_buffer(device="cuda"):
    """A zeroed accumulator buffer for bnn_bfc_tail (FORWARD_SYNC_BYTES)."""
    return torch.zeros(FORWARD_SYNC_BYTES, dtype=torch.uint8, device=device)


def bnn_bgemm(A, B, K, thr=None, flip=None, want_sums=True, want_bits=True, out_sums=None,
              out_bits=None, stream=None):
    """Binary GEMM / FC (Sec. III-B): A [M,Kw], B [N,Kw] packed -> sums [M,N],
    bits [M,ceil(N/32)]."""
    lib = load()
    _u32(A)
    _u32(B)
    M, N = A.shape[0], B.shape[0]
    thr = _dev(thr, torch.int32, "thr")
    flip = _dev(flip, torch.int32, "flip")
    if want_sums and out_sums is None:
        out_sums = torch.empty((M, N), dtype=torch.int32, device=A.device)
    if want_bits and out_bits is None:
        out_bits = torch.empty((M, words(N)), dtype=torch.int32, device=A.device)
    _check(lib.bnn_bgemm(M, N, K, _ptr(A), _ptr(B), _ptr(thr), _ptr(flip), _ptr(out_sums),
                         _ptr(out_bits), _stream(stream)))
    return out_sums, out_bits


class Network:
    """A layer chain for bnn_forward.  ``layers`` holds dicts with the C
    struct's fields and device tensors (w, thr, flip, offset); the tensors are
    kept alive by this object."""

    def __init__(self, layers, H, W, C):
        self.H, self.W, self.C = H, W, C
        self._tensors = layers
        arr = (Layer * len(layers))()
        for i, d in enumerate(layers):
            L = arr[i]
            L.kind = d["kind"]
            for f in ("C", "F", "KH", "KW", "stride", "pad", "pool", "K", "N"):
                setattr(L, f, int(d.get(f, 0)))
            for f in ("w", "thr", "flip", "offset", "wprep"):
                t = d.get(f)
                setattr(L, f, None if t is None else t.data_ptr())
        self.layers = arr
        self.n = len(layers)

    def workspace_size(self, batch: int) -> int:
        lib = load()
        out = ctypes.c_size_t()
        _check(lib.bnn_forward_workspace_size(self.layers, self.n, batch, self.H, self.W,
                                              self.C, ctypes.byref(out)))
        return out.value

    def alloc_workspace(self, batch: int, device="cuda"):
        """A bnn_forward workspace for `batch` images, its accumulator bytes zeroed."""
        ws = torch.empty(self.workspace_size(batch), dtype=torch.uint8, device=device)
        ws[:FORWARD_SYNC_BYTES].zero_()
        return ws


def bnn_forward(net: Network, x, workspace=None, logits=None, stream=None):
    """Run the chain on x [batch, H, W, C] fp32; returns int32 logits."""
    lib = load()
    _dev(x, torch.float32, "x")
    batch = x.shape[0]
    if workspace is None:
        workspace = net.alloc_workspace(batch, x.device)
    n_out = net.layers[net.n - 1].N
    if logits is None:
        logits = torch.empty((batch, n_out), dtype=torch.int32, device=x.device)
    _check(lib.bnn_forward(net.layers, net.n, batch, net.H, net.W, net.C, _ptr(x),
                           _ptr(workspace), workspace.numel(), _ptr(logits),
                           _stream(stream)))
    return logits


def bnn_forward_noalloc(net: Network, x, logits=None, stream=None):
    """bnn_forward with the intermediate bits in the library's per-GPU scratch
    array instead of a workspace (for callers that cannot allocate); returns
    int32 logits."""
    lib = load()
    _dev(x, torch.float32, "x")
    batch = x.shape[0]
    n_out = net.layers[net.n - 1].N
    if logits is None:
        logits = torch.empty((batch, n_out), dtype=torch.int32, device=x.device)
    _dev(logits, torch.int32, "logits")
    _check(lib.bnn_forward_noalloc(net.layers, net.n, batch, net.H, net.W, net.C, _ptr(x),
                                   _ptr(logits), _stream(stream)))
    return logits


# Short aliases.
pack_bits = bnn_pack_bits
bconv2d = bnn_bconv2d
fconv2d_binw = bnn_fconv2d_binw
bconv2d_input = bnn_bconv2d_input
fconv_bconv2d = bnn_fconv_bconv2d
binarize_input = bnn_binarize_input
bgemm = bnn_bgemm
forward = bnn_forward
