"""The C-ABI library on the CPU: it loads, exports every symbol bnn.h declares,
and rejects invalid arguments before launching anything (no GPU needed: each
call here fails validation on the host)."""
import ctypes
import os
import re

import pytest

from paper_1808_00209_amd import bnn

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bnn.h")

needs_lib = pytest.mark.skipif(not os.path.exists(bnn.LIB_PATH),
                               reason="libbnn.so not built (run __graft_entry__.build())")

A = 4096  # a 16-byte-aligned stand-in address; never dereferenced here


def declared_functions():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"^\S[^\n(]*?\b(bnn_[a-z0-9_]+)\(", src, re.M)))


def test_header_lists_the_binding_symbols():
    assert declared_functions() == sorted(bnn.EXPORTED)


@needs_lib
def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(bnn.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name


@needs_lib
def test_abi_version_and_empty_error():
    lib = bnn.load()
    header = open(HEADER).read()
    assert "#define BNN_ABI_VERSION %d" % lib.bnn_abi_version() in header
    assert isinstance(bnn.last_error(), str)


def test_missing_library_fails_loudly(tmp_path):
    saved = bnn._lib
    bnn._lib = None
    try:
        with pytest.raises(RuntimeError, match="not found"):
            bnn.load(str(tmp_path / "nope.so"))
    finally:
        bnn._lib = saved


def _conv(**kw):
    d = dict(N=1, H=8, W=8, C=64, F=64, KH=3, KW=3, stride=1, pad=1, pool=0)
    d.update(kw)
    return bnn.ConvDesc(*[d[k] for k in ("N", "H", "W", "C", "F", "KH", "KW", "stride",
                                         "pad", "pool")])


def _bconv(desc, inp=A, w=A, thr=A, flip=None, sums=A, bits=A):
    lib = bnn.load()
    return lib.bnn_bconv2d(ctypes.byref(desc), inp, w, thr, flip, sums, bits, None)


@needs_lib
@pytest.mark.parametrize("kw,status,text", [
    (dict(stride=2), 4, "stride"),
    (dict(pool=3), 2, "pool"),
    (dict(N=0), 2, ">= 1"),
    (dict(C=-1), 2, ">= 1"),
    (dict(KH=0), 2, ">= 1"),
    (dict(pad=-1), 2, "pad"),
    (dict(H=1, W=1, pad=0), 2, "empty"),
    (dict(H=2, W=2, pad=0, KH=2, KW=2, pool=2), 2, "pooling"),
])
def test_bconv_shape_errors(kw, status, text):
    assert _bconv(_conv(**kw)) == status
    assert text in bnn.last_error()


@needs_lib
def test_bconv_null_and_alignment_errors():
    d = _conv()
    assert _bconv(d, inp=None) == 1 and "input" in bnn.last_error()
    assert _bconv(d, w=None) == 1 and "weight" in bnn.last_error()
    assert _bconv(d, sums=None, bits=None) == 1 and "nothing" in bnn.last_error()
    assert _bconv(d, thr=None) == 1 and "thr" in bnn.last_error()
    assert _bconv(d, inp=A + 4) == 3 and "aligned" in bnn.last_error()
    assert _bconv(d, bits=A + 8) == 3
    lib = bnn.load()
    assert lib.bnn_bconv2d(None, A, A, A, None, A, A, None) == 1


@needs_lib
def test_bconv_input_errors():
    lib = bnn.load()

    def call(desc, mode=0, x=A, off=None, w=A, thr=A, sums=A, bits=A):
        return lib.bnn_bconv2d_input(ctypes.byref(desc), mode, x, off, w, thr, None, sums, bits,
                                     None)

    # the window must fit 128 bits with C, KH, KW <= 32: 5x5x6 = 150 does not
    assert call(_conv(C=6, KH=5, KW=5)) == 4 and "150 bits" in bnn.last_error()
    assert call(_conv(C=33, KH=1, KW=1)) == 4
    assert call(_conv(C=1, KH=33, KW=1, H=40)) == 4
    assert call(_conv(C=3, stride=2)) == 4 and "stride" in bnn.last_error()
    assert call(_conv(C=3, pool=3)) == 2
    assert call(_conv(C=3), mode=3) == 2 and "mode" in bnn.last_error()
    assert call(_conv(C=3), mode=1) == 2 and "channels" in bnn.last_error()  # gray is 1 channel
    assert call(_conv(C=1), mode=2) == 2                                     # LBP is 3
    assert call(_conv(C=3), x=None) == 1 and "input" in bnn.last_error()
    assert call(_conv(C=3), thr=None) == 1 and "thr" in bnn.last_error()
    assert call(_conv(C=3), sums=None, bits=None) == 1
    assert call(_conv(C=3), x=A + 4) == 3
    assert lib.bnn_bconv2d_input(None, 0, A, None, A, A, None, A, A, None) == 1


@needs_lib
def test_fconv_bconv_errors():
    lib = bnn.load()
    d0 = _conv(N=2, H=32, W=32, C=3, F=128)
    d1 = _conv(N=2, H=32, W=32, C=128, F=128, pool=2)

    def call(a=d0, b=d1, x=A, w0=A, thr0=A, w1=A, thr1=A, bits=A):
        return lib.bnn_fconv_bconv2d(ctypes.byref(a), ctypes.byref(b), x, w0, thr0, None, w1,
                                     None, thr1, None, bits, None)

    # the second layer must read the first one's output
    assert call(b=_conv(N=2, H=30, W=32, C=128, F=128)) == 2 and "match" in bnn.last_error()
    assert call(b=_conv(N=2, H=32, W=32, C=64, F=128)) == 2
    assert call(b=_conv(N=1, H=32, W=32, C=128, F=128)) == 2
    # shapes the fused kernel does not cover
    assert call(a=_conv(N=2, H=32, W=32, C=5, F=128)) == 4 and "C <= 4" in bnn.last_error()
    assert call(a=_conv(N=2, H=32, W=32, C=3, F=96),
                b=_conv(N=2, H=32, W=32, C=96, F=128)) == 4
    assert call(b=_conv(N=2, H=32, W=32, C=128, F=256)) == 4
    assert call(a=_conv(N=2, H=32, W=32, C=3, F=128, pool=2),
                b=_conv(N=2, H=16, W=16, C=128, F=128)) == 4
    assert call(a=_conv(N=2, H=32, W=32, C=3, F=128, KH=5, KW=5, pad=2)) == 4
    assert call(b=_conv(N=2, H=32, W=32, C=128, F=128, pad=2)) == 4
    # pointers
    assert call(x=None) == 1
    assert call(w1=None) == 1 and "w1" in bnn.last_error()
    assert call(thr0=None) == 1 and "thr0" in bnn.last_error()
    assert call(thr1=None) == 1
    assert call(bits=None) == 1
    assert call(w1=A + 4) == 3
    assert call(x=A + 4) == 3


@needs_lib
def test_input_bconv_bconv_errors():
    lib = bnn.load()
    d0 = _conv(N=2, H=32, W=32, C=3, F=64)
    d1 = _conv(N=2, H=32, W=32, C=64, F=64, pool=2)

    def call(a=d0, b=d1, mode=0, x=A, w0=A, thr0=A, w1=A, thr1=A, bits=A):
        return lib.bnn_input_bconv_bconv2d(ctypes.byref(a), ctypes.byref(b), mode, x, None, w0,
                                           thr0, None, w1, None, thr1, None, bits, None)

    # modes: unknown, or not thresholding
    assert call(mode=3) == 2 and "mode" in bnn.last_error()
    assert call(mode=1) == 4 and "THRESHOLD" in bnn.last_error()
    assert call(mode=2) == 4
    # the second layer must read the first one's output
    assert call(b=_conv(N=2, H=30, W=32, C=64, F=64)) == 2 and "match" in bnn.last_error()
    assert call(b=_conv(N=2, H=32, W=32, C=128, F=64)) == 2
    # shapes the fused kernel does not cover: 3 input channels only
    assert call(a=_conv(N=2, H=32, W=32, C=4, F=64), b=d1) == 4
    assert call(a=_conv(N=2, H=32, W=32, C=1, F=64), b=d1) == 4
    assert call(a=_conv(N=2, H=32, W=32, C=3, F=96),
                b=_conv(N=2, H=32, W=32, C=96, F=64)) == 4
    assert call(b=_conv(N=2, H=32, W=32, C=64, F=256)) == 4
    assert call(a=_conv(N=2, H=32, W=32, C=3, F=64, pool=2),
                b=_conv(N=2, H=16, W=16, C=64, F=64)) == 4
    # pointers and alignment
    assert call(x=None) == 1
    assert call(w1=None) == 1 and "w1" in bnn.last_error()
    assert call(thr0=None) == 1 and "thr0" in bnn.last_error()
    assert call(thr1=None) == 1
    assert call(bits=None) == 1
    assert call(w1=A + 4) == 3
    assert call(x=A + 4) == 3


@needs_lib
def test_bconv_bconv_errors():
    """bnn_bconv_bconv2d: shape chaining, the shapes its kernel covers, NULL
    pointers and alignment, all refused on the host before any launch."""
    lib = bnn.load()
    d0 = _conv(N=2, H=16, W=16, C=128, F=256, pad=1)
    d1 = _conv(N=2, H=16, W=16, C=256, F=256, pad=1, pool=2)

    def call(a=d0, b=d1, x=A, w0=A, thr0=A, w1=A, thr1=A, bits=A):
        return lib.bnn_bconv_bconv2d(ctypes.byref(a), ctypes.byref(b), x, w0, thr0, None, w1,
                                     thr1, None, bits, None)

    assert lib.bnn_bconv_bconv2d(None, ctypes.byref(d1), A, A, A, None, A, A, None, A,
                                 None) == 1
    # the second conv must read the first one's output
    assert call(b=_conv(N=2, H=14, W=16, C=256, F=256, pad=1)) == 2 and "match" in bnn.last_error()
    assert call(b=_conv(N=1, H=16, W=16, C=256, F=256, pad=1)) == 2
    assert call(b=_conv(N=2, H=16, W=16, C=128, F=256, pad=1)) == 2
    # shapes the kernel does not cover
    assert call(a=_conv(N=2, H=8, W=8, C=256, F=256, pad=1),
                b=_conv(N=2, H=8, W=8, C=256, F=256, pad=1)) == 4
    assert call(a=_conv(N=2, H=16, W=16, C=96, F=256, pad=1)) == 4
    assert call(a=_conv(N=2, H=16, W=16, C=128, F=128, pad=1),
                b=_conv(N=2, H=16, W=16, C=128, F=256, pad=1)) == 4
    assert call(b=_conv(N=2, H=16, W=16, C=256, F=512, pad=1)) == 4
    assert call(a=_conv(N=2, H=16, W=16, C=128, F=256, pad=0),
                b=_conv(N=2, H=14, W=14, C=256, F=256, pad=1)) == 4
    assert call(b=_conv(N=2, H=16, W=16, C=256, F=256, pad=0)) == 4
    assert call(a=_conv(N=2, H=16, W=16, C=128, F=256, pad=1, pool=2),
                b=_conv(N=2, H=8, W=8, C=256, F=256, pad=1)) == 4
    # pointers and alignment
    assert call(x=None) == 1
    assert call(w0=None) == 1
    assert call(w1=None) == 1 and "w1" in bnn.last_error()
    assert call(thr0=None) == 1 and "thr0" in bnn.last_error()
    assert call(thr1=None) == 1
    assert call(bits=None) == 1
    assert call(w1=A + 4) == 3
    assert call(w0=A + 4) == 3
    assert call(x=A + 4) == 3
    assert call(bits=A + 4) == 3


@needs_lib
def test_bfc_pair_errors():
    """bnn_bfc_pair: sizes, the shapes its kernel covers, one output of the
    two, NULL pointers and alignment, all refused on the host."""
    lib = bnn.load()

    def call(M=64, K0=1024, N0=1024, N1=10, a=A, w0=A, thr0=A, w1=A, thr1=None, sums=A,
             bits=None):
        return lib.bnn_bfc_pair(M, K0, N0, N1, a, w0, thr0, None, w1, thr1, None, sums, bits,
                                None)

    for bad in (dict(M=0), dict(K0=0), dict(N0=0), dict(N1=0), dict(N1=-3)):
        assert call(**bad) == 2, bad
    for uns in (dict(K0=1000), dict(K0=2048), dict(K0=4096), dict(N0=128), dict(N0=2048), dict(N1=33),
                dict(M=(1 << 26) + 1)):
        assert call(**uns) == 4, uns
    assert call(a=None) == 1
    assert call(w0=None) == 1
    assert call(w1=None) == 1
    assert call(thr0=None) == 1 and "thr0" in bnn.last_error()
    assert call(sums=None, bits=None) == 1
    assert call(sums=A, bits=A, thr1=A) == 2 and "not both" in bnn.last_error()
    assert call(sums=None, bits=A, thr1=None) == 1 and "thr1" in bnn.last_error()
    assert call(a=A + 4) == 3
    assert call(w1=A + 4) == 3
    assert call(sums=A + 4) == 3
    assert call(sums=None, bits=A + 4, thr1=A) == 3


@needs_lib
def test_bfc_tail_errors():
    """bnn_bfc_tail: sizes, the shapes its kernel covers (rows, K0, N0, tile
    count, N1), one output of the two, NULL pointers (accum included) and
    alignment, all refused on the host."""
    lib = bnn.load()

    def call(M=64, K0=1024, N0=1024, N1=10, a=A, w0=A, thr0=A, w1=A, thr1=None, sums=A,
             bits=None, accum=A):
        return lib.bnn_bfc_tail(M, K0, N0, N1, a, w0, thr0, None, w1, thr1, None, sums, bits,
                                accum, None)

    for bad in (dict(M=0), dict(K0=0), dict(N0=0), dict(N1=0), dict(N1=-3)):
        assert call(**bad) == 2, bad
    # K0 below 1024, N0 not a multiple of 32, more than 512 rows or 512
    # tiles (64 rows x 9216 outputs: 2 x 288), N1 > 32
    for uns in (dict(K0=1000), dict(K0=1023), dict(N0=1000), dict(M=513), dict(N0=9216),
                dict(M=40, N0=9216), dict(N1=33)):
        assert call(**uns) == 4, uns
    assert call(a=None) == 1
    assert call(w0=None) == 1
    assert call(w1=None) == 1
    assert call(thr0=None) == 1 and "thr0" in bnn.last_error()
    assert call(accum=None) == 1 and "accum" in bnn.last_error()
    assert call(sums=None, bits=None) == 1
    assert call(sums=A, bits=A, thr1=A) == 2 and "not both" in bnn.last_error()
    assert call(sums=None, bits=A, thr1=None) == 1 and "thr1" in bnn.last_error()
    assert call(a=A + 4) == 3
    assert call(w1=A + 4) == 3
    assert call(sums=A + 4) == 3
    assert call(accum=A + 4) == 3
    assert call(sums=None, bits=A + 4, thr1=A) == 3


@needs_lib
def test_binarize_input_errors():
    lib = bnn.load()
    assert lib.bnn_binarize_input(5, A, None, 1, 4, 4, 3, A, None) == 2
    assert lib.bnn_binarize_input(0, A, None, 0, 4, 4, 3, A, None) == 2
    assert lib.bnn_binarize_input(0, A, None, 1, 4, 4, 33, A, None) == 2
    assert lib.bnn_binarize_input(1, A, None, 1, 4, 4, 4, A, None) == 2
    assert lib.bnn_binarize_input(2, A, None, 1, 4, 4, 1, A, None) == 2
    assert lib.bnn_binarize_input(2, None, None, 1, 4, 4, 3, A, None) == 1
    assert lib.bnn_binarize_input(2, A, None, 1, 4, 4, 3, A + 4, None) == 3


@needs_lib
def test_conv_output_dims():
    assert bnn.bnn_conv_output_dims(_conv(H=32, W=30, pool=2)) == (32, 30, 16, 15)
    assert bnn.bnn_conv_output_dims(_conv(H=7, W=5, pool=2, KH=1, KW=1, pad=0)) == (7, 5, 3, 2)
    assert bnn.bnn_conv_output_dims(_conv(H=5, W=5, KH=5, KW=3, pad=0)) == (1, 3, 1, 3)
    with pytest.raises(bnn.BnnError) as e:
        bnn.bnn_conv_output_dims(_conv(stride=3))
    assert e.value.status == 4


@needs_lib
def test_bgemm_errors():
    lib = bnn.load()
    assert lib.bnn_bgemm(0, 4, 4, A, A, A, None, A, A, None) == 2
    assert lib.bnn_bgemm(4, 4, 0, A, A, A, None, A, A, None) == 2
    assert lib.bnn_bgemm(4, 4, 4, None, A, A, None, A, A, None) == 1
    assert lib.bnn_bgemm(4, 4, 4, A, A, None, None, A, A, None) == 1
    assert lib.bnn_bgemm(4, 4, 4, A, A + 4, A, None, A, None, None) == 3
    assert lib.bnn_bgemm(1 << 40, 4, 4, A, A, A, None, A, A, None) == 2


@needs_lib
def test_pack_errors_and_empty():
    lib = bnn.load()
    assert lib.bnn_pack_bits(A, None, -1, 4, A, None) == 2
    assert lib.bnn_pack_bits(A, None, 4, 0, A, None) == 2
    assert lib.bnn_pack_bits(None, None, 4, 4, A, None) == 1
    assert lib.bnn_pack_bits(None, None, 0, 4, None, None) == 0  # nothing to do


def _layers(specs):
    arr = (bnn.Layer * len(specs))()
    for i, d in enumerate(specs):
        for k, v in d.items():
            setattr(arr[i], k, v)
    return arr


@needs_lib
def test_forward_chain_validation():
    lib = bnn.load()
    size = ctypes.c_size_t()
    good = [dict(kind=1, C=3),
            dict(kind=3, C=3, F=64, KH=3, KW=3, stride=1, pad=1, pool=2, w=A, thr=A),
            dict(kind=3, C=64, F=64, KH=3, KW=3, stride=1, pad=1, pool=2, w=A, thr=A),
            dict(kind=5, K=2 * 2 * 64, N=4, w=A)]
    L = _layers(good)
    assert lib.bnn_forward_workspace_size(L, 4, 8, 8, 8, 3, ctypes.byref(size)) == 0
    # the FC tail's 69632 accumulator bytes and two buffers of the largest
    # packed map, the thresholded input: 8 images x 8x8 pixels x 1 word x 4
    # bytes, 256-byte aligned
    assert size.value == 69632 + 2 * 256 * ((8 * 8 * 8 * 1 * 4 + 255) // 256)
    bad_k = [dict(good[0]), dict(good[1]), dict(good[2]), dict(good[3], K=100)]
    assert lib.bnn_forward_workspace_size(_layers(bad_k), 4, 8, 8, 8, 3, ctypes.byref(size)) == 2
    assert "expects K" in bnn.last_error()
    no_logits = good[:3]
    assert lib.bnn_forward_workspace_size(_layers(no_logits), 3, 8, 8, 8, 3,
                                          ctypes.byref(size)) == 2
    # flattening a map whose channel count is not a multiple of 32
    odd = [dict(kind=1, C=3), dict(kind=3, C=3, F=40, KH=3, KW=3, stride=1, pad=1, w=A, thr=A),
           dict(kind=5, K=8 * 8 * 40, N=4, w=A)]
    assert lib.bnn_forward_workspace_size(_layers(odd), 3, 1, 8, 8, 3, ctypes.byref(size)) == 2
    assert "flattening" in bnn.last_error()
    # conv weights must be 16-byte aligned, as for bnn_bconv2d
    skew = [dict(good[0]), dict(good[1], w=A + 4), dict(good[2]), dict(good[3])]
    assert lib.bnn_forward_workspace_size(_layers(skew), 4, 8, 8, 8, 3, ctypes.byref(size)) == 3
    assert "16-byte aligned" in bnn.last_error()
    # a too-small workspace is refused before any launch
    assert lib.bnn_forward(L, 4, 8, 8, 8, 3, A, A, 256, A, None) == 6
    assert lib.bnn_forward(L, 4, 8, 8, 8, 3, A, A + 16, 1 << 20, A, None) == 3


@needs_lib
def test_forward_noalloc_validation_before_any_device_call():
    """bnn_forward_noalloc checks the chain, its pointers and the size of
    its intermediate bits against the scratch array before it touches the
    device: a chain that needs more than BNN_FORWARD_SCRATCH_BYTES gives
    BNN_ERR_WORKSPACE, NULL / misaligned pointers their errors."""
    lib = bnn.load()
    header = open(HEADER).read()
    assert "#define BNN_FORWARD_SCRATCH_BYTES ((size_t)64 << 20)" in header
    assert bnn.FORWARD_SCRATCH_BYTES == 64 << 20
    good = [dict(kind=1, C=3),
            dict(kind=3, C=3, F=64, KH=3, KW=3, stride=1, pad=1, pool=2, w=A, thr=A),
            dict(kind=3, C=64, F=64, KH=3, KW=3, stride=1, pad=1, pool=2, w=A, thr=A),
            dict(kind=5, K=2 * 2 * 64, N=4, w=A)]
    L = _layers(good)
    size = ctypes.c_size_t()
    # 8 x 8 images: BNN_FORWARD_SYNC_BYTES of accumulators and two buffers of
    # the thresholded input, batch * 64 pixels * 1 word * 4 bytes; the
    # largest batch that fits the 64 MiB array is (64 MiB - 69632) / 512 = 130936
    assert "#define BNN_FORWARD_SYNC_BYTES ((size_t)69632)" in header
    assert bnn.FORWARD_SYNC_BYTES == 69632
    for batch, fits in ((130936, True), (130937, False)):
        assert lib.bnn_forward_workspace_size(L, 4, batch, 8, 8, 3, ctypes.byref(size)) == 0
        assert size.value == 69632 + 2 * batch * 256
        assert (size.value <= bnn.FORWARD_SCRATCH_BYTES) == fits
    assert lib.bnn_forward_noalloc(L, 4, 130937, 8, 8, 3, A, A, None) == 6
    assert "scratch" in bnn.last_error()
    assert lib.bnn_forward_noalloc(L, 4, 8, 8, 8, 3, None, A, None) == 1
    assert lib.bnn_forward_noalloc(L, 4, 8, 8, 8, 3, A, A + 4, None) == 3
    assert lib.bnn_forward_noalloc(L, 3, 8, 8, 8, 3, A, A, None) == 2  # no logits layer


@needs_lib
def test_options_defaults_set_get_and_range_checks():
    """Kernel-selection options: defaults, a round trip, per-field range
    checks (an invalid set leaves the options unchanged), NULL pointers."""
    lib = bnn.load()
    d = bnn.bnn_default_options()
    assert (d.algo, d.fuse_input, d.fuse_first, d.fc_chain, d.conv1x1, d.xcd_order,
            d.gemv_max_rows, d.lds_weights, d.late_thresholds,
            d.fuse_pair) == (0, 1, 1, 1, 1, 1, 1, -1, -1, 1)
    try:
        bnn.bnn_set_options(algo=bnn.ALGO_VALU, gemv_max_rows=16, lds_weights=1)
        got = bnn.bnn_get_options()
        assert (got.algo, got.gemv_max_rows, got.lds_weights) == (1, 16, 1)
        for field, bad in [("algo", 2), ("fuse_input", 2), ("fuse_first", -1), ("fc_chain", 3),
                           ("conv1x1", 2), ("xcd_order", -1), ("xcd_order", 3),
                           ("gemv_max_rows", 17),
                           ("gemv_max_rows", -1), ("lds_weights", 2), ("late_thresholds", -2),
                           ("fuse_pair", 2), ("fuse_pair", -1)]:
            with pytest.raises(bnn.BnnError, match="out of range"):
                bnn.bnn_set_options(**{field: bad})
            got = bnn.bnn_get_options()
            assert (got.algo, got.gemv_max_rows, got.lds_weights) == (1, 16, 1)
        assert lib.bnn_set_options(None) == 1 and "NULL" in bnn.last_error()
        assert lib.bnn_get_options(None) == 1
        with bnn.options(fc_chain=0):
            assert bnn.bnn_get_options().fc_chain == 0
            assert bnn.bnn_get_options().algo == 0  # the block starts from the defaults
        assert bnn.bnn_get_options().algo == 1  # restored on exit
    finally:
        bnn.bnn_set_options()


@needs_lib
def test_options_are_per_thread():
    import threading
    seen = {}
    try:
        bnn.bnn_set_options(algo=bnn.ALGO_VALU)

        def other():
            seen["algo"] = bnn.bnn_get_options().algo

        t = threading.Thread(target=other)
        t.start()
        t.join()
        assert seen["algo"] == bnn.ALGO_AUTO
        assert bnn.bnn_get_options().algo == bnn.ALGO_VALU
    finally:
        bnn.bnn_set_options()


def test_library_sources_read_no_environment():
    """The launch path reads no environment variables: every kernel choice
    comes from the arguments and the per-thread options."""
    csrc = os.path.join(ROOT, "paper_1808_00209_amd", "csrc")
    for f in os.listdir(csrc):
        src = open(os.path.join(csrc, f)).read()
        assert "getenv" not in src and "environ" not in src, f


@needs_lib
def test_prepared_weights_size_and_argument_errors():
    """bnn_prepared_weights_size: 16-byte entries [ceil(F/32)*32][KH][KW][Cp]
    with Cp = Cw = ceil(C/32) when C % 64 == 0, else Cw rounded up to 8, then
    F int32 offsets rounded up to 16
    bytes; shape, NULL and alignment errors of the three calls come before
    any launch."""
    lib = bnn.load()
    size = ctypes.c_size_t()
    for F, KH, KW, C in [(64, 3, 3, 64), (40, 3, 3, 96), (1024, 1, 1, 4100), (1, 1, 1, 1)]:
        assert lib.bnn_prepared_weights_size(F, KH, KW, C, ctypes.byref(size)) == 0
        Cw = (C + 31) // 32
        Cp = Cw if C % 64 == 0 else (Cw + 7) // 8 * 8
        assert size.value == (F + 31) // 32 * 32 * KH * KW * Cp * 16 + (4 * F + 15) // 16 * 16
    assert lib.bnn_prepared_weights_size(0, 3, 3, 64, ctypes.byref(size)) == 2
    assert lib.bnn_prepared_weights_size(64, 3, 3, 64, None) == 1
    # beyond 2 GiB
    assert lib.bnn_prepared_weights_size(1 << 20, 3, 3, 4096, ctypes.byref(size)) == 2
    assert "2 GiB" in bnn.last_error()
    assert lib.bnn_prepare_weights(64, 3, 3, 64, None, A, None) == 1
    assert lib.bnn_prepare_weights(64, 3, 3, 64, A, A + 4, None) == 3
    assert lib.bnn_prepare_weights(64, 3, 0, 64, A, A, None) == 2
    d = _conv()
    assert lib.bnn_bconv2d_prepared(ctypes.byref(d), A, A, None, A, None, A, A, None) == 1
    assert "wprep" in bnn.last_error()
    assert lib.bnn_bconv2d_prepared(ctypes.byref(d), A, A, A + 8, A, None, A, A, None) == 3
    assert lib.bnn_bconv2d_prepared(ctypes.byref(_conv(stride=2)), A, A, A, A, None, A, A,
                                    None) == 4
    # bnn_forward checks a conv layer's wprep alignment like its w
    good = [dict(kind=1, C=3),
            dict(kind=3, C=3, F=64, KH=3, KW=3, stride=1, pad=1, pool=2, w=A, thr=A, wprep=A + 4),
            dict(kind=5, K=4 * 4 * 64, N=4, w=A)]
    assert lib.bnn_forward_workspace_size(_layers(good), 3, 8, 8, 8, 3, ctypes.byref(size)) == 3
    assert "wprep" in bnn.last_error()
