"""The C-ABI library loads and validates arguments on the host (no GPU).

Every call below is built to fail validation, which happens before anything
is enqueued, so none of them reaches the HIP runtime; the fake pointers are
never dereferenced.
"""
import ctypes
import os
import re

import pytest

from paper_1810_11066_amd import bitserial as bs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bitserial.h")

FAKE = ctypes.c_void_p(0x10000)        # aligned, never dereferenced
MISALIGNED = ctypes.c_void_p(0x10004)
NULL = ctypes.c_void_p(0)
STREAM = ctypes.c_void_p(0)


@pytest.fixture(scope="module")
def lib():
    return bs.load_library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(bs_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert "bs_conv2d" in names and "bs_pack" in names
    for name in names:
        assert hasattr(lib, name), name
    assert set(names) == set(bs.EXPORTED)


def test_abi_version_and_words(lib):
    assert lib.bs_abi_version() == 109
    for k, w in [(0, 0), (1, 1), (31, 1), (32, 1), (33, 2), (4096, 128)]:
        assert lib.bs_packed_words(k) == w


def test_timing_events_set_and_clear(lib):
    # host-side state only: nothing is launched, the handles are not touched
    assert lib.bs_set_timing_events(FAKE, FAKE) == bs.BS_OK
    assert lib.bs_set_timing_events(NULL, NULL) == bs.BS_OK


def test_status_strings(lib):
    for s in range(5):
        assert lib.bs_status_string(s)
    assert lib.bs_status_string(99) == b"unknown status"


def test_quantize_validation(lib):
    q = lib.bs_quantize
    assert q(NULL, FAKE, 8, 1.0, 2, 0, STREAM) == bs.BS_ERR_INVALID_ARG
    assert b"x is NULL" in lib.bs_last_error()
    assert q(FAKE, MISALIGNED, 8, 1.0, 2, 0, STREAM) == bs.BS_ERR_INVALID_ARG
    assert b"aligned" in lib.bs_last_error()
    assert q(FAKE, FAKE, -1, 1.0, 2, 0, STREAM) == bs.BS_ERR_INVALID_ARG
    for bits in (0, 9):
        assert q(FAKE, FAKE, 8, 1.0, bits, 0, STREAM) == bs.BS_ERR_INVALID_ARG
    for scale in (0.0, -1.0, float("inf"), float("nan")):
        assert q(FAKE, FAKE, 8, scale, 2, 0, STREAM) == bs.BS_ERR_INVALID_ARG
    assert q(FAKE, FAKE, 8, 1.0, 2, 1, STREAM) == bs.BS_ERR_INVALID_ARG
    assert q(FAKE, FAKE, 8, 1.0, 1, 7, STREAM) == bs.BS_ERR_INVALID_ARG
    # signed codes need a sign plane and a magnitude plane
    assert q(FAKE, FAKE, 8, 1.0, 1, 2, STREAM) == bs.BS_ERR_INVALID_ARG
    assert b"signed" in lib.bs_last_error()
    assert q(FAKE, FAKE, 0, 1.0, 2, 2, STREAM) == bs.BS_OK


def test_empty_is_ok_without_launch(lib):
    # n == 0 / rows == 0 enqueue nothing
    assert lib.bs_quantize(FAKE, FAKE, 0, 1.0, 2, 0, STREAM) == bs.BS_OK
    assert lib.bs_pack(FAKE, FAKE, 0, 64, 2, STREAM) == bs.BS_OK
    assert lib.bs_quantize_pack(FAKE, FAKE, 0, 64, 1.0, 2, 0, STREAM) == bs.BS_OK
    assert lib.bs_last_error() == b""


def test_pack_validation(lib):
    p = lib.bs_pack
    assert p(NULL, FAKE, 4, 64, 2, STREAM) == bs.BS_ERR_INVALID_ARG
    assert p(FAKE, NULL, 4, 64, 2, STREAM) == bs.BS_ERR_INVALID_ARG
    assert p(FAKE, FAKE, -1, 64, 2, STREAM) == bs.BS_ERR_INVALID_ARG
    assert p(FAKE, FAKE, 4, 0, 2, STREAM) == bs.BS_ERR_INVALID_ARG
    assert p(FAKE, FAKE, 4, 64, 9, STREAM) == bs.BS_ERR_INVALID_ARG
    qp = lib.bs_quantize_pack
    assert qp(FAKE, FAKE, 4, 64, 1.0, 2, 1, STREAM) == bs.BS_ERR_INVALID_ARG
    assert qp(FAKE, FAKE, 4, 64, 0.0, 2, 0, STREAM) == bs.BS_ERR_INVALID_ARG
    assert qp(FAKE, FAKE, 4, 64, 1.0, 1, 2, STREAM) == bs.BS_ERR_INVALID_ARG


def test_pack_ex_validation(lib):
    p = lib.bs_pack_ex
    assert p(NULL, FAKE, 2, 64, 9, 2, 0, STREAM) == bs.BS_ERR_INVALID_ARG
    assert p(FAKE, MISALIGNED, 2, 64, 9, 2, 0, STREAM) == bs.BS_ERR_INVALID_ARG
    assert p(FAKE, FAKE, -1, 64, 9, 2, 0, STREAM) == bs.BS_ERR_INVALID_ARG
    assert p(FAKE, FAKE, 2, 0, 9, 2, 0, STREAM) == bs.BS_ERR_INVALID_ARG
    assert p(FAKE, FAKE, 2, 64, 0, 2, 0, STREAM) == bs.BS_ERR_INVALID_ARG
    assert p(FAKE, FAKE, 2, 64, 9, 9, 0, STREAM) == bs.BS_ERR_INVALID_ARG
    for layout in (-1, 3):
        assert p(FAKE, FAKE, 2, 64, 9, 2, layout,
                 STREAM) == bs.BS_ERR_INVALID_ARG
    assert b"layout" in lib.bs_last_error()
    assert p(FAKE, FAKE, 1 << 30, 1 << 20, 1 << 10, 2, 0,
             STREAM) == bs.BS_ERR_UNSUPPORTED
    assert p(FAKE, FAKE, 0, 64, 9, 2, 1, STREAM) == bs.BS_OK   # nothing to do


def params(**kw):
    base = dict(n=1, h=8, w=8, c=64, oc=64, kh=3, kw=3, stride_h=1,
                stride_w=1, pad_h=1, pad_w=1, abits=2, wbits=1, aenc=0,
                wenc=0)
    base.update(kw)
    return bs.ConvParams(**base)


@pytest.mark.parametrize("bad,status", [
    (dict(n=0), bs.BS_ERR_INVALID_ARG),
    (dict(c=0), bs.BS_ERR_INVALID_ARG),
    (dict(oc=-3), bs.BS_ERR_INVALID_ARG),
    (dict(kh=0), bs.BS_ERR_INVALID_ARG),
    (dict(stride_w=0), bs.BS_ERR_INVALID_ARG),
    (dict(pad_h=-1), bs.BS_ERR_INVALID_ARG),
    (dict(abits=0), bs.BS_ERR_INVALID_ARG),
    (dict(wbits=9), bs.BS_ERR_INVALID_ARG),
    (dict(wenc=2), bs.BS_ERR_INVALID_ARG),
    (dict(kh=11, pad_h=1), bs.BS_ERR_INVALID_ARG),     # oh < 1
    (dict(aenc=3), bs.BS_ERR_INVALID_ARG),             # unknown encoding
    (dict(aenc=2, abits=1), bs.BS_ERR_INVALID_ARG),    # signed needs 2 bits
    (dict(wenc=-1), bs.BS_ERR_INVALID_ARG),
    (dict(abits=8, wbits=8, c=(1 << 31) // (255 * 255 * 9) + 1),
     bs.BS_ERR_OVERFLOW),
])
def test_conv_validation(lib, bad, status):
    p = params(**bad)
    assert lib.bs_conv2d(ctypes.byref(p), FAKE, FAKE, FAKE, STREAM) == status
    assert lib.bs_last_error() != b""


def test_conv_pointer_validation(lib):
    p = params()
    assert lib.bs_conv2d(ctypes.byref(p), NULL, FAKE, FAKE,
                         STREAM) == bs.BS_ERR_INVALID_ARG
    assert lib.bs_conv2d(ctypes.byref(p), FAKE, MISALIGNED, FAKE,
                         STREAM) == bs.BS_ERR_INVALID_ARG
    assert lib.bs_conv2d(None, FAKE, FAKE, FAKE,
                         STREAM) == bs.BS_ERR_INVALID_ARG


@pytest.mark.parametrize("bad,status", [
    (dict(n=0), bs.BS_ERR_INVALID_ARG),
    (dict(kh=11, pad_h=1), bs.BS_ERR_INVALID_ARG),
    (dict(wenc=-1), bs.BS_ERR_INVALID_ARG),
    (dict(abits=8, wbits=8, c=(1 << 31) // (255 * 255 * 9) + 1),
     bs.BS_ERR_OVERFLOW),
    # shapes no fused kernel covers: refused before any launch
    (dict(c=48), bs.BS_ERR_UNSUPPORTED),            # c not a multiple of 32
    (dict(oc=6), bs.BS_ERR_UNSUPPORTED),            # oc not a multiple of 4
    (dict(kh=5, kw=5, pad_h=2, pad_w=2), bs.BS_ERR_UNSUPPORTED),
    (dict(wbits=5), bs.BS_ERR_UNSUPPORTED),         # filters above 4 bits
    (dict(abits=5), bs.BS_ERR_UNSUPPORTED),         # codes above 4 bits
    (dict(aenc=2, wenc=2, wbits=2), bs.BS_ERR_UNSUPPORTED),  # signed
    (dict(aenc=1, abits=1), bs.BS_ERR_UNSUPPORTED),  # +-1 activations
    (dict(c=96), bs.BS_ERR_UNSUPPORTED),            # 3 words per plane
    (dict(c=1024), bs.BS_ERR_UNSUPPORTED),          # 32 words, 3x3 window
])
def test_fused_conv_validation(lib, bad, status):
    # disjoint fake buffers, so that the overlap check passes
    p = params(**bad)
    act, wts, out = at(0), at(1 << 26), at(1 << 28)
    assert lib.bs_conv2d_codes(ctypes.byref(p), act, wts, out,
                               STREAM) == status
    assert lib.bs_last_error() != b""


def test_fused_conv_pointer_validation(lib):
    p = params()
    assert lib.bs_conv2d_codes(ctypes.byref(p), NULL, FAKE, FAKE,
                               STREAM) == bs.BS_ERR_INVALID_ARG
    assert lib.bs_conv2d_codes(ctypes.byref(p), MISALIGNED, FAKE, FAKE,
                               STREAM) == bs.BS_ERR_INVALID_ARG
    # the output may not overlap the codes (n*h*w*c = 4096 bytes) ...
    assert lib.bs_conv2d_codes(ctypes.byref(p), at(0), at(1 << 20),
                               at(4096 - 16), STREAM) == bs.BS_ERR_INVALID_ARG
    assert b"overlaps act_codes" in lib.bs_last_error()
    # ... nor the packed filters (64 x 9 x 1 plane x 2 words x 4 B)
    assert lib.bs_conv2d_codes(ctypes.byref(p), at(0), at(1 << 20),
                               at((1 << 20) + 4608 - 16),
                               STREAM) == bs.BS_ERR_INVALID_ARG
    assert b"overlaps w_packed" in lib.bs_last_error()


def at(offset):
    """A fake device address `offset` bytes past FAKE (never dereferenced)."""
    return ctypes.c_void_p(0x10000 + offset)


FAR = ctypes.c_void_p(0x40000000)


def test_output_overlapping_an_input_is_rejected(lib):
    """An output sharing a byte with an input is an invalid argument, found
    before anything is enqueued (fake pointers, nothing is launched)."""
    E = bs.BS_ERR_INVALID_ARG
    # 8 floats span 32 bytes; codes at byte 16 overlap them
    assert lib.bs_quantize(FAKE, at(16), 8, 1.0, 2, 0, STREAM) == E
    assert b"overlaps" in lib.bs_last_error()
    assert lib.bs_pack(FAKE, at(16), 4, 64, 2, STREAM) == E
    assert lib.bs_pack_ex(FAKE, at(16), 2, 64, 9, 2, 0, STREAM) == E
    assert lib.bs_quantize_pack(FAKE, at(16), 4, 64, 1.0, 2, 0, STREAM) == E
    # the output placed first, the input starting inside it
    assert lib.bs_pack(at(16), FAKE, 4, 64, 2, STREAM) == E
    p = params()                       # 1x8x8x64 A2 -> 8x8x64 int32
    assert lib.bs_conv2d(ctypes.byref(p), FAKE, FAR, at(1008),
                         STREAM) == E    # out from the last 16 of act's 1 KB
    assert b"act_packed" in lib.bs_last_error()
    assert lib.bs_conv2d(ctypes.byref(p), FAR, FAKE, at(4592),
                         STREAM) == E    # ... of the filters' 4608 B
    assert b"w_packed" in lib.bs_last_error()
    assert lib.bs_conv2d_requant(ctypes.byref(p), FAKE, FAR, 0.5, 2, at(16),
                                 STREAM) == E
    assert lib.bs_dense(4, 4, 64, 2, 2, 0, FAKE, FAKE, at(16),
                        STREAM) == E
    assert lib.bs_dense_ex(4, 4, 64, 2, 0, 2, 0, FAR, FAKE, at(16),
                           STREAM) == E


def test_overflow_guard_boundary(lib):
    # (2^8-1)^2 * 9 * c <= 2^31-1  <=>  c <= 3669
    limit = (2 ** 31 - 1) // (255 * 255 * 9)
    p = params(abits=8, wbits=8, c=limit + 1)
    assert lib.bs_conv2d(ctypes.byref(p), FAKE, FAKE, FAKE,
                         STREAM) == bs.BS_ERR_OVERFLOW
    # dense bound (2^a-1)(2^w-1) k
    k = (2 ** 31 - 1) // (255 * 255) + 1
    assert lib.bs_dense(4, 4, k, 8, 8, 0, FAKE, FAKE, FAKE,
                        STREAM) == bs.BS_ERR_OVERFLOW


def test_overflow_guard_encodings(lib):
    """The bound uses the largest magnitude of each encoding: 2^(B-1) for
    signed codes, 2^B - 1 for unipolar and bipolar ones (checked on the host
    through bs_conv2d_describe, which launches nothing)."""
    buf = ctypes.create_string_buffer(256)
    d = lib.bs_conv2d_describe
    uni = (2 ** 31 - 1) // (255 * 255 * 9)
    sgn = (2 ** 31 - 1) // (128 * 128 * 9)
    ok = params(abits=8, wbits=8, aenc=2, wenc=2, c=uni + 1)
    assert d(ctypes.byref(ok), buf, 256) == bs.BS_OK
    bad = params(abits=8, wbits=8, aenc=2, wenc=2, c=sgn + 1)
    assert d(ctypes.byref(bad), buf, 256) == bs.BS_ERR_OVERFLOW
    bip = params(abits=8, wbits=8, aenc=1, wenc=1, c=uni + 1)
    assert d(ctypes.byref(bip), buf, 256) == bs.BS_ERR_OVERFLOW
    assert lib.bs_dense_ex(4, 4, (2 ** 31 - 1) // (128 * 255) + 1, 8, 2, 8, 0,
                           FAKE, FAKE, FAKE, STREAM) == bs.BS_ERR_OVERFLOW


def test_dense_ex_validation(lib):
    d = lib.bs_dense_ex
    assert d(4, 4, 64, 1, 2, 2, 0, FAKE, FAKE, FAKE,
             STREAM) == bs.BS_ERR_INVALID_ARG        # 1-bit signed
    assert d(4, 4, 64, 2, 5, 2, 0, FAKE, FAKE, FAKE,
             STREAM) == bs.BS_ERR_INVALID_ARG        # unknown encoding
    assert d(4, 4, 64, 2, 0, 2, 0, NULL, FAKE, FAKE,
             STREAM) == bs.BS_ERR_INVALID_ARG
    assert d(0, 4, 64, 1, 1, 1, 1, FAKE, FAKE, FAKE,
             STREAM) == bs.BS_ERR_INVALID_ARG


def test_dense_validation(lib):
    d = lib.bs_dense
    assert d(0, 4, 64, 2, 2, 0, FAKE, FAKE, FAKE, STREAM) == bs.BS_ERR_INVALID_ARG
    assert d(4, 4, 64, 2, 2, 3, FAKE, FAKE, FAKE, STREAM) == bs.BS_ERR_INVALID_ARG
    assert d(4, 4, 64, 0, 2, 0, FAKE, FAKE, FAKE, STREAM) == bs.BS_ERR_INVALID_ARG
    assert d(4, 4, 64, 2, 2, 0, FAKE, NULL, FAKE, STREAM) == bs.BS_ERR_INVALID_ARG


def test_out_shape(lib):
    oh, ow = ctypes.c_int32(), ctypes.c_int32()
    for (h, k, s, pd) in [(56, 3, 1, 1), (56, 3, 2, 1), (56, 1, 2, 0),
                          (7, 3, 1, 1), (9, 5, 3, 2)]:
        p = params(h=h, w=h + 1, kh=k, kw=k, stride_h=s, stride_w=s, pad_h=pd,
                   pad_w=pd)
        assert lib.bs_conv2d_out_shape(ctypes.byref(p), ctypes.byref(oh),
                                       ctypes.byref(ow)) == bs.BS_OK
        assert oh.value == (h + 2 * pd - k) // s + 1
        assert ow.value == (h + 1 + 2 * pd - k) // s + 1


def test_binding_out_shape_matches_the_library(lib):
    # the binding computes (oh, ow) itself to size its tensor checks; it must
    # agree with bs_conv2d_out_shape wherever that accepts the parameters,
    # and report the library's error wherever it does not
    import itertools
    oh, ow = ctypes.c_int32(), ctypes.c_int32()
    for h, w, k, s, pd in itertools.product((1, 2, 7, 14, 57), (1, 3, 56),
                                            (1, 2, 3, 5), (0, 1, 2, 3),
                                            (0, 1, 2)):
        p = params(h=h, w=w, kh=k, kw=k, stride_h=s, stride_w=s, pad_h=pd,
                   pad_w=pd)
        st = lib.bs_conv2d_out_shape(ctypes.byref(p), ctypes.byref(oh),
                                     ctypes.byref(ow))
        if st == bs.BS_OK:
            assert bs._out_hw(p) == (oh.value, ow.value)
        else:
            with pytest.raises(bs.BitserialError) as e:
                bs._out_hw(p)
            assert e.value.status == st


def test_kernel_mode(lib):
    assert lib.bs_set_kernel_mode(4) == bs.BS_ERR_INVALID_ARG
    assert lib.bs_set_kernel_mode(-1) == bs.BS_ERR_INVALID_ARG
    for m in (1, 2, 3):
        assert lib.bs_set_kernel_mode(m) == bs.BS_OK
    assert lib.bs_set_kernel_mode(0) == bs.BS_OK


def test_units_per_wave(lib):
    assert lib.bs_set_units_per_wave(-1) == bs.BS_ERR_INVALID_ARG
    p = params(n=64, h=56, w=56, c=64, oc=64)
    try:
        assert lib.bs_set_units_per_wave(5) == bs.BS_OK
        d = bs.bs_conv2d_describe(p)
        # 64*56*56 / 64 groups x 16 quads = 50176 units, 5 per wave
        assert "units=50176 units_per_wave=5" in d
        waves = -(-50176 // 5)
        assert "grid=%d " % -(-waves // 4) in d
    finally:
        assert lib.bs_set_units_per_wave(0) == bs.BS_OK


def test_describe_store_bound_1x1_runs(lib):
    # 1x1 layers with A*W*words <= 16 run one tile chunk (4 quads) per wave;
    # others keep the balanced plan (not 4 here: 50176 units on the CPU's
    # stand-in of one block per CU)
    import re

    def run_of(p):
        return int(re.search(r"units_per_wave=(\d+)",
                             bs.bs_conv2d_describe(p)).group(1))

    l3 = params(n=128, h=56, w=56, c=64, oc=64, kh=1, kw=1, pad_h=0, pad_w=0)
    assert run_of(l3) == 4
    a3w3 = params(n=128, h=14, w=14, c=256, oc=512, kh=1, kw=1, pad_h=0,
                  pad_w=0, abits=3, wbits=3)
    assert run_of(a3w3) != 4
    assert run_of(params(n=64, h=56, w=56, c=64, oc=64)) != 4


def test_describe_batch_split(lib):
    # the pixel kernel addresses its tensors with 32-bit offsets: an int32
    # output past 2 GB (128 x 56 x 56 x 1344) is split into image chunks of
    # 127 and 1 (2^31 - 64 KiB / 16.9 MB per image), one below stays whole
    big = params(n=128, h=56, w=56, c=32, oc=1344, kh=1, kw=1, pad_h=0,
                 pad_w=0, abits=1, wbits=1)
    d = bs.bs_conv2d_describe(big)
    assert d.startswith("conv_pix_kernel") and "batch split" in d
    assert "units=%d " % (127 * 56 * 56 // 64 * 1344 // 4) in d
    small = params(n=126, h=56, w=56, c=32, oc=1344, kh=1, kw=1, pad_h=0,
                   pad_w=0, abits=1, wbits=1)
    assert "batch split" not in bs.bs_conv2d_describe(small)


def test_binding_refuses_cpu_tensors():
    import torch
    x = torch.zeros(16, dtype=torch.float32)
    q = torch.zeros(16, dtype=torch.uint8)
    with pytest.raises(ValueError, match="GPU tensor"):
        bs.bs_quantize(x, q, 1.0, 2)


def test_describe_names_the_kernel_each_mode_picks(lib):
    # host-only planning: no device memory is touched
    p = params(n=64, h=56, w=56, c=64, oc=64)
    try:
        assert bs.bs_conv2d_describe(p).startswith(
            "conv_pix_kernel<A=2,W=1,unipolar,K=3,S=1,CW=2> patch=9taps x 2words "
            "slice=1ch x 9taps")
        bs.bs_set_kernel_mode(2)
        assert bs.bs_conv2d_describe(p).startswith(
            "conv_ocl_kernel<A=2,W=1,unipolar,K=3,S=1,P=7,CW=2>")
        bs.bs_set_kernel_mode(1)
        assert bs.bs_conv2d_describe(p).startswith("conv_generic_kernel")
        bs.bs_set_kernel_mode(3)
        # oc not a multiple of 4: the pixel kernel does not apply
        assert bs.bs_conv2d_describe(params(oc=70)).startswith(
            "conv_generic_kernel")
    finally:
        bs.bs_set_kernel_mode(0)
    # 5-bit activations: no specialised kernel
    assert bs.bs_conv2d_describe(params(abits=5)).startswith(
        "conv_generic_kernel")


def test_error_string_and_kernel_mode_are_per_thread(lib):
    """The library's only state (last error, kernel mode) is per host
    thread: another thread's error and mode do not leak into this one."""
    import threading
    p = params(n=64, h=56, w=56, c=64, oc=64)
    seen = {}
    ready, resume = threading.Event(), threading.Event()

    def worker():
        bs.bs_set_kernel_mode(1)
        seen["status"] = lib.bs_quantize(NULL, FAKE, 8, 1.0, 2, 0, STREAM)
        seen["err"] = lib.bs_last_error()
        ready.set()
        resume.wait(30)
        seen["err_after"] = lib.bs_last_error()
        seen["desc"] = bs.bs_conv2d_describe(p)
        bs.bs_set_kernel_mode(0)

    t = threading.Thread(target=worker)
    t.start()
    try:
        assert ready.wait(30)
        assert lib.bs_set_units_per_wave(0) == bs.BS_OK   # clears this one
        assert lib.bs_last_error() == b""
        assert bs.bs_conv2d_describe(p).startswith("conv_pix_kernel")
    finally:
        resume.set()
        t.join(30)
    assert seen["status"] == bs.BS_ERR_INVALID_ARG
    assert b"NULL" in seen["err"] and seen["err_after"] == seen["err"]
    assert seen["desc"].startswith("conv_generic_kernel")


ENC = ("unipolar", "bipolar", "signed")


@pytest.mark.parametrize("aenc", [0, 1, 2])
@pytest.mark.parametrize("wenc", [0, 1, 2])
@pytest.mark.parametrize("bits", [1, 2, 3])
def test_describe_kernel_encodings_match_the_call(lib, aenc, wenc, bits):
    """Whatever kernel serves a call was compiled for the call's encodings:
    a pixels-on-lanes specialisation names its own (activation x weight)
    encodings, which must be the requested ones (host-only planning)."""
    abits = 1 if aenc == 1 else max(bits, 2 if aenc == 2 else 1)
    wbits = 1 if wenc == 1 else max(bits, 2 if wenc == 2 else 1)
    for a_, w_ in ((abits, wbits), (abits, abits)):
        if (aenc == 1 and a_ != 1) or (wenc == 1 and w_ != 1) or \
                (wenc == 2 and w_ < 2):
            continue
        d = bs.bs_conv2d_describe(params(abits=a_, wbits=w_, aenc=aenc,
                                         wenc=wenc))
        if not d.startswith("conv_pix_kernel"):
            continue
        kenc = d.split(",")[2]
        want = ENC[wenc] if aenc == 0 else "%s x %s" % (ENC[aenc], ENC[wenc])
        assert kenc == want, d


def test_describe_pixel_kernel_serves_new_encodings(lib):
    for kw in (dict(abits=1, wbits=1, aenc=1, wenc=1),     # XNOR
               dict(abits=1, wbits=1, aenc=1, wenc=0),
               dict(abits=2, wbits=2, aenc=0, wenc=2),
               dict(abits=3, wbits=3, aenc=2, wenc=2)):
        d = bs.bs_conv2d_describe(params(**kw))
        assert d.startswith("conv_pix_kernel"), (kw, d)
    # signed activations with unipolar weights: no specialisation, plain loops
    d = bs.bs_conv2d_describe(params(abits=2, wbits=2, aenc=2, wenc=0))
    assert d.startswith("conv_generic_kernel"), d


def test_describe_validation_and_truncation(lib):
    buf = ctypes.create_string_buffer(8)
    assert lib.bs_conv2d_describe(ctypes.byref(params()), buf, 8) == bs.BS_OK
    assert len(buf.value) == 7
    assert lib.bs_conv2d_describe(ctypes.byref(params()), None,
                                  8) == bs.BS_ERR_INVALID_ARG
    assert lib.bs_conv2d_describe(ctypes.byref(params()), buf,
                                  0) == bs.BS_ERR_INVALID_ARG
    assert lib.bs_conv2d_describe(ctypes.byref(params(kh=0)), buf,
                                  8) == bs.BS_ERR_INVALID_ARG


def test_requant_validation(lib):
    r = lib.bs_conv2d_requant
    p = params()
    assert r(ctypes.byref(p), FAKE, FAKE, 0.5, 0, FAKE,
             STREAM) == bs.BS_ERR_INVALID_ARG
    assert r(ctypes.byref(p), FAKE, FAKE, 0.5, 9, FAKE,
             STREAM) == bs.BS_ERR_INVALID_ARG
    for scale in (0.0, -2.0, float("inf"), float("nan")):
        assert r(ctypes.byref(p), FAKE, FAKE, scale, 2, FAKE,
                 STREAM) == bs.BS_ERR_INVALID_ARG
    assert r(ctypes.byref(p), FAKE, FAKE, 0.5, 2, NULL,
             STREAM) == bs.BS_ERR_INVALID_ARG
    assert r(ctypes.byref(p), FAKE, MISALIGNED, 0.5, 2, FAKE,
             STREAM) == bs.BS_ERR_INVALID_ARG
    assert r(ctypes.byref(params(aenc=3)), FAKE, FAKE, 0.5, 2, FAKE,
             STREAM) == bs.BS_ERR_INVALID_ARG
    assert r(ctypes.byref(params(abits=8, wbits=8, c=4000)), FAKE, FAKE, 0.5,
             2, FAKE, STREAM) == bs.BS_ERR_OVERFLOW


def _staged_region(n, h, w, k, s, pad, oc, run):
    """Largest input region (pixels) a 4-wave block of `run` units per wave
    packs for a fused conv: the flat NHWC input rows from the first tap row
    of the block's first output pixel to the last tap row of its last one,
    without the columns of those two rows (when they are inside the image)
    that only pixels outside the block read, checked here to hold every
    in-range tap of every output pixel of the block; for strided 1x1
    windows, one gathered input pixel per output pixel of the block."""
    oh = (h + 2 * pad - k) // s + 1
    ow = (w + 2 * pad - k) // s + 1
    npix = n * oh * ow
    gu = oc // 4
    units = -(-npix // 64) * gu
    best = 0
    for ub0 in range(0, units, 4 * run):
        ub1 = min(ub0 + 4 * run, units)
        p0, p1 = ub0 // gu * 64, min((ub1 - 1) // gu * 64 + 63, npix - 1)
        if k == 1 and s > 1:
            # strided 1x1 windows: one gathered input pixel per output pixel
            best = max(best, p1 + 1 - p0)
            continue
        (n0, y0, x0), (n1, y1, x1) = [
            ((p // ow) // oh, (p // ow) % oh, p % ow) for p in (p0, p1)]
        a, b = y0 * s - pad, y1 * s - pad + k - 1
        lo = (n0 * h + min(max(a, 0), h)) * w
        hi = (n1 * h + max(min(b, h - 1), -1)) * w + w
        if 0 <= a < h:
            lo += min(max(x0 * s - pad, 0), w - 1)
        if 0 <= b < h:
            hi -= w - 1 - max(min(x1 * s - pad + k - 1, w - 1), 0)
        hi = max(hi, lo)
        for p in range(p0, p1 + 1):
            img, y, x = (p // ow) // oh, (p // ow) % oh, p % ow
            for dy in range(k):
                for dx in range(k):
                    iy, ix = y * s - pad + dy, x * s - pad + dx
                    if 0 <= iy < h and 0 <= ix < w:
                        assert lo <= (img * h + iy) * w + ix < hi
        best = max(best, hi - lo)
    return best


@pytest.mark.parametrize("shape", [
    dict(n=2, h=9, w=10, k=3, s=1, pad=1, oc=16, run=3),
    dict(n=3, h=7, w=13, k=3, s=2, pad=1, oc=64, run=5),
    dict(n=2, h=12, w=12, k=1, s=2, pad=0, oc=128, run=2)])
def test_codes_describe_reports_the_staged_plan(lib, shape):
    # the fused call's plan: its own kernel (staged codes), run length and
    # the input region of its largest block
    sh = dict(shape)
    run = sh.pop("run")
    p = params(n=sh["n"], h=sh["h"], w=sh["w"], c=64, oc=sh["oc"],
               kh=sh["k"], kw=sh["k"], stride_h=sh["s"], stride_w=sh["s"],
               pad_h=sh["pad"], pad_w=sh["pad"], abits=2, wbits=1)
    try:
        assert lib.bs_set_units_per_wave(run) == bs.BS_OK
        d = bs.bs_conv2d_codes_describe(p)
    finally:
        assert lib.bs_set_units_per_wave(0) == bs.BS_OK
    assert d.startswith("conv_pix_kernel<A=2,W=1,unipolar,K=%d,S=%d,CW=2> "
                        "staged codes:" % (sh["k"], sh["s"]))
    assert "units_per_wave=%d" % run in d
    assert " region=%dpx " % _staged_region(run=run, **sh) in d


def test_codes_describe_refusals(lib):
    buf = ctypes.create_string_buffer(64)
    d = lib.bs_conv2d_codes_describe
    assert d(ctypes.byref(params()), None, 64) == bs.BS_ERR_INVALID_ARG
    assert d(ctypes.byref(params()), buf, 0) == bs.BS_ERR_INVALID_ARG
    # c = 96 has no fused kernel: refused as bs_conv2d_codes refuses it
    assert d(ctypes.byref(params(c=96)), buf, 64) == bs.BS_ERR_UNSUPPORTED
    assert buf.value == b""
    assert b"no fused kernel" in lib.bs_last_error()


def test_quantized_refusals(lib):
    buf = ctypes.create_string_buffer(64)
    q = lib.bs_conv2d_quantized
    one = params(kh=1, kw=1, pad_h=0, pad_w=0)
    assert q(ctypes.byref(one), None, ctypes.c_float(1.0), FAKE, FAKE,
             STREAM) == bs.BS_ERR_INVALID_ARG
    for bad_scale in (0.0, -1.0, float("inf"), float("nan")):
        assert q(ctypes.byref(one), FAKE, ctypes.c_float(bad_scale), FAKE,
                 FAKE, STREAM) == bs.BS_ERR_INVALID_ARG
    # the quantizer is unipolar; signed or +-1 activations are refused
    for aenc in (1, 2):
        assert q(ctypes.byref(params(kh=1, kw=1, pad_h=0, pad_w=0,
                                     abits=2 if aenc == 2 else 1,
                                     aenc=aenc)),
                 FAKE, ctypes.c_float(1.0), FAKE, FAKE,
                 STREAM) == bs.BS_ERR_UNSUPPORTED
    # 3x3 windows have no fused float32 kernel (refused before any launch,
    # as the describe call shows without a GPU)
    d = lib.bs_conv2d_quantized_describe
    assert d(ctypes.byref(params()), buf, 64) == bs.BS_ERR_UNSUPPORTED
    assert buf.value == b""
    assert b"no fused kernel" in lib.bs_last_error()
    assert d(ctypes.byref(one), None, 64) == bs.BS_ERR_INVALID_ARG


@pytest.mark.parametrize("s,run", [(1, 4), (2, 3)])
def test_quantized_describe_reports_the_staged_plan(lib, s, run):
    sh = dict(n=2, h=13, w=11, k=1, s=s, pad=0, oc=64)
    p = params(n=2, h=13, w=11, c=128, oc=64, kh=1, kw=1, stride_h=s,
               stride_w=s, pad_h=0, pad_w=0, abits=3, wbits=2)
    try:
        assert lib.bs_set_units_per_wave(run) == bs.BS_OK
        d = bs.bs_conv2d_quantized_describe(p)
        codes = bs.bs_conv2d_codes_describe(p)
    finally:
        assert lib.bs_set_units_per_wave(0) == bs.BS_OK
    assert d.startswith("conv_pix_kernel<A=3,W=2,unipolar,K=1,S=%d,CW=4> "
                        "staged float32:" % s)
    assert " region=%dpx " % _staged_region(run=run, **sh) in d
    # the same plan as the fused call on codes
    assert d.split(": ", 1)[1] == codes.split(": ", 1)[1]
