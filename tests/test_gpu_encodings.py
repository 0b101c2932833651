"""GPU parity for the encodings and packed layouts beyond unipolar data:
+-1 (bipolar) activations, signed (two's complement) activations and
weights, and bs_pack_ex's strided reduction axis and bit-axis positions.

Every call goes through the C ABI; every result is compared bit for bit with
the CPU oracle, into sentinel-filled buffers with guard bands (so unwritten
elements and stray writes fail too).
"""
import numpy as np
import pytest
import torch

from paper_1810_11066_amd import bitserial as bs
from tests.test_gpu_parity import (SENT32, Guarded, as_words, dev, say,
                                   special_floats)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU parity tests need the MI355X"
    bs.load_library()
    bs.bs_set_kernel_mode(0)
    yield
    bs.bs_set_kernel_mode(0)


# ------------------------------------------------------- signed quantize --

@pytest.mark.parametrize("n", [1, 17, 1000, 100003])
@pytest.mark.parametrize("bits,scale", [(2, 1.0), (3, 0.7), (4, 1.5),
                                        (8, 1.3), (2, 3e38)])
def test_quantize_signed(oracle, n, bits, scale):
    say("quantize signed n=%d bits=%d scale=%g" % (n, bits, scale))
    rng = np.random.default_rng(7 * n + bits)
    x = rng.permutation(special_floats(rng, n))[:n]
    want = oracle.quantize(x, scale, bits, oracle.SIGNED)
    g = Guarded(n, torch.uint8, 0xAB)
    bs.bs_quantize(dev(x), g.t, scale, bits, bs.SIGNED)
    torch.cuda.synchronize()
    assert np.array_equal(g.t.cpu().numpy(), want)
    g.check_guards()


@pytest.mark.parametrize("k", [32, 96, 256, 33, 100])
@pytest.mark.parametrize("rows", [1, 130])
@pytest.mark.parametrize("bits", [2, 4, 8])
def test_quantize_pack_signed(oracle, k, rows, bits):
    say("quantize_pack signed rows=%d k=%d bits=%d" % (rows, k, bits))
    rng = np.random.default_rng(k + 5 * rows + bits)
    x = rng.permutation(special_floats(rng, rows * k))[:rows * k]
    x = x.reshape(rows, k)
    want = oracle.pack(oracle.quantize(x, 1.7, bits, oracle.SIGNED), bits)
    g = Guarded(want.size, torch.int32, SENT32)
    bs.bs_quantize_pack(dev(x), g.t, rows, k, 1.7, bits, bs.SIGNED)
    torch.cuda.synchronize()
    assert np.array_equal(as_words(g.t).reshape(want.shape), want)
    g.check_guards()


# ---------------------------------------------------------------- pack_ex --

PACK_EX_CASES = [
    # shape, axis
    ((2, 64, 5, 8), 1),       # NCHW, inner = 40 (4 rows per thread)
    ((3, 45, 7, 3), 1),       # NCHW, inner = 21 (one row per thread), tail
    ((1, 300, 16), 1),        # many words, inner = 16
    ((17, 100), 1),           # inner = 1: contiguous reduction axis
    ((64, 3, 3, 64), 3),      # OHWI filters, inner = 1
    ((8, 64, 3, 3), 1),       # OIHW filters, inner = 9
    ((5, 1), 1),              # k = 1
]


@pytest.mark.parametrize("layout", [bs.LAYOUT_MBK, bs.LAYOUT_MKB,
                                    bs.LAYOUT_BMK])
@pytest.mark.parametrize("case", PACK_EX_CASES, ids=lambda c: str(c[0]))
@pytest.mark.parametrize("bits", [1, 2, 5])
def test_pack_ex(oracle, case, layout, bits):
    shape, axis = case
    say("pack_ex", shape, "axis", axis, "layout", layout, "bits", bits)
    rng = np.random.default_rng(sum(shape) + 3 * layout + bits)
    q = rng.integers(0, 256, size=shape, dtype=np.uint8)    # high bits too
    want = oracle.pack_ex(q, bits, axis=axis, layout=layout)
    k = shape[axis]
    outer = int(np.prod(shape[:axis], dtype=np.int64))
    inner = int(np.prod(shape[axis + 1:], dtype=np.int64))
    g = Guarded(want.size, torch.int32, SENT32)
    bs.bs_pack_ex(dev(q), g.t, outer, k, inner, bits, layout)
    torch.cuda.synchronize()
    assert np.array_equal(as_words(g.t).reshape(want.shape), want)
    g.check_guards()


def test_pack_ex_grid_stride(oracle):
    # more work items than one pass of the largest grid
    shape = (4, 96, 120, 96)        # NCHW, inner % 4 == 0
    say("pack_ex grid stride", shape)
    rng = np.random.default_rng(3)
    q = rng.integers(0, 4, size=shape, dtype=np.uint8)
    want = oracle.pack_ex(q, 2, axis=1)
    got = bs.pack_ex(dev(q), 2, axis=1)
    torch.cuda.synchronize()
    assert np.array_equal(as_words(got).reshape(want.shape), want)


def test_nchw_pack_feeds_conv(oracle):
    """NCHW codes packed along C with bs_pack_ex are the packed NHWC tensor
    the conv reads: the conv of them equals the oracle's NHWC conv."""
    n, c, h, w, oc = 2, 70, 9, 8, 12
    rng = np.random.default_rng(21)
    x = rng.integers(0, 4, size=(n, c, h, w), dtype=np.uint8)
    wq = rng.integers(0, 2, size=(oc, 3, 3, c), dtype=np.uint8)
    nhwc = np.ascontiguousarray(x.transpose(0, 2, 3, 1))
    op = oracle.conv_params(n, h, w, c, oc, 3, 3, 1, 1, 2, 1)
    want = oracle.conv2d(op, oracle.pack(nhwc, 2), oracle.pack(wq, 1))
    spec = bs.Conv2dSpec(n, h, w, c, oc, 3, 3, 1, 1, 2, 1)
    got = bs.conv2d(spec, bs.pack_ex(dev(x), 2, axis=1), bs.pack(dev(wq), 1))
    torch.cuda.synchronize()
    assert np.array_equal(got.cpu().numpy(), want)


# ------------------------------------------------ conv with any encodings --

def codes(rng, shape, bits):
    return rng.integers(0, 1 << bits, size=shape, dtype=np.uint8)


def run_conv_enc(oracle, shape, abits, aenc, wbits, wenc, seed, mode=0,
                 expect_pix=None):
    n, h, w, c, oc, k, s, pad = shape
    rng = np.random.default_rng(seed)
    a, wq = codes(rng, (n, h, w, c), abits), codes(rng, (oc, k, k, c), wbits)
    ap, wp = oracle.pack(a, abits), oracle.pack(wq, wbits)
    op = oracle.conv_params(n, h, w, c, oc, k, k, s, pad, abits, wbits,
                            aenc, wenc)
    want = oracle.conv2d(op, ap, wp)
    p = bs.ConvParams(n, h, w, c, oc, k, k, s, s, pad, pad, abits, wbits,
                      aenc, wenc)
    oh, ow = bs.bs_conv2d_out_shape(p)
    g = Guarded(n * oh * ow * oc, torch.int32, SENT32)
    bs.bs_set_kernel_mode(mode)
    try:
        desc = bs.bs_conv2d_describe(p)
        bs.bs_conv2d(p, dev(ap.view(np.int32)), dev(wp.view(np.int32)), g.t)
    finally:
        bs.bs_set_kernel_mode(0)
    torch.cuda.synchronize()
    if expect_pix is not None:
        assert desc.startswith("conv_pix_kernel") == expect_pix, desc
    got = g.t.cpu().numpy().reshape(want.shape)
    g.check_guards()
    assert np.array_equal(got, want)


ENC_SHAPES = [
    # n, h, w, c, oc, k, s, pad
    (2, 9, 10, 64, 12, 3, 1, 1),     # whole window in registers
    (1, 13, 11, 128, 8, 3, 2, 1),    # 3-tap filter slices, stride 2
    (1, 7, 9, 256, 8, 3, 1, 1),      # row blocks, partial sums in the tile
    (1, 6, 5, 512, 4, 3, 1, 1),      # tap blocks
    (2, 8, 9, 45, 12, 3, 1, 1),      # ragged channels (tail bits)
    (1, 10, 10, 100, 8, 3, 2, 0),    # no padding, ragged channels
    (1, 5, 67, 33, 4, 3, 1, 2),      # pad 2: taps out of range on 2 sides
    (3, 7, 7, 64, 16, 1, 1, 0),      # 1x1
    (1, 12, 9, 1024, 8, 1, 2, 0),    # 1x1, word chunks
]

# (abits, aenc, wbits, wenc) served by the pixels-on-lanes kernel
PIX_ENCODINGS = ([(1, 1, 1, 1), (1, 1, 1, 0)] +
                 [(a, 0, w, 2) for a in (1, 2, 3, 4) for w in (2, 3, 4)] +
                 [(b, 2, b, 2) for b in (2, 3, 4)])


@pytest.mark.parametrize("enc", PIX_ENCODINGS,
                         ids=lambda e: "A%d%sW%d%s" % (e[0], "ubs"[e[1]],
                                                       e[2], "ubs"[e[3]]))
@pytest.mark.parametrize("shape", ENC_SHAPES,
                         ids=lambda s: "x".join(map(str, s)))
def test_conv_encodings_pixel(oracle, shape, enc):
    abits, aenc, wbits, wenc = enc
    say("conv enc", shape, enc)
    run_conv_enc(oracle, shape, abits, aenc, wbits, wenc,
                 seed=sum(shape) * 31 + abits * 7 + wbits + 3 * aenc + wenc,
                 expect_pix=True)


@pytest.mark.parametrize("seed", range(40))
def test_conv_encodings_pixel_random(oracle, seed):
    """Random shapes inside the pixel kernel's domain with a random encoding
    it serves (signed data, the XNOR case, +-1 activations with unipolar
    filters) at a random run length; the plan must be the pixel kernel."""
    rng = np.random.default_rng(7000 + seed)
    abits, aenc, wbits, wenc = PIX_ENCODINGS[
        int(rng.integers(0, len(PIX_ENCODINGS)))]
    k, s, pad = int(rng.choice([1, 3])), int(rng.choice([1, 2])), \
        int(rng.integers(0, 3))
    cw = int(rng.choice([1, 2, 4, 8, 16] + ([32] if k == 1 else [])))
    c = int(rng.integers(32 * (cw - 1) + 1, 32 * cw + 1))
    oc = 4 * int(rng.integers(1, 25))
    n = int(rng.integers(1, 3))
    h = max(int(rng.integers(1, 25)), k - 2 * pad)
    w = max(int(rng.integers(1, 25)), k - 2 * pad)
    run = int(rng.choice([0, 1, 2, 3, 5, 7, 13]))
    shape = (n, h, w, c, oc, k, s, pad)
    say("conv enc pixel random", shape, (abits, aenc, wbits, wenc), "run", run)
    bs.bs_set_units_per_wave(run)
    try:
        run_conv_enc(oracle, shape, abits, aenc, wbits, wenc, seed=seed,
                     mode=3, expect_pix=True)
    finally:
        bs.bs_set_units_per_wave(0)


@pytest.mark.parametrize("aenc", [0, 1, 2])
@pytest.mark.parametrize("wenc", [0, 1, 2])
@pytest.mark.parametrize("seed", range(4))
def test_conv_encodings_random(oracle, aenc, wenc, seed):
    rng = np.random.default_rng(4000 + 9 * seed + 3 * aenc + wenc)
    n, h, w = int(rng.integers(1, 3)), int(rng.integers(1, 12)), \
        int(rng.integers(1, 12))
    c, oc = int(rng.integers(1, 140)), int(rng.integers(1, 40))
    k = int(rng.choice([1, 2, 3, 5]))
    s, pad = int(rng.integers(1, 3)), int(rng.integers(0, 3))
    while h + 2 * pad < k or w + 2 * pad < k:
        pad += 1
    lo_a = 2 if aenc == 2 else 1
    lo_w = 2 if wenc == 2 else 1
    abits = int(rng.integers(lo_a, 6))
    wbits = int(rng.integers(lo_w, 6))
    shape = (n, h, w, c, oc, k, s, pad)
    for mode in (0, 1):
        say("conv enc random", shape, abits, aenc, wbits, wenc, "mode", mode)
        run_conv_enc(oracle, shape, abits, aenc, wbits, wenc, seed=seed,
                     mode=mode)


@pytest.mark.parametrize("aenc,wenc", [(1, 1), (1, 0), (0, 2), (2, 2), (2, 0),
                                       (1, 2), (2, 1)])
@pytest.mark.parametrize("mkn", [(64, 40, 4096), (130, 8, 100), (1, 4, 32)])
def test_dense_encodings(oracle, aenc, wenc, mkn):
    m, n, k = mkn
    abits = 1 if aenc == 1 else 2
    wbits = 1 if wenc == 1 else (3 if wenc == 2 else 2)
    say("dense enc", mkn, aenc, wenc)
    rng = np.random.default_rng(m + n + k + aenc + 3 * wenc)
    a, w = codes(rng, (m, k), abits), codes(rng, (n, k), wbits)
    ap, wp = oracle.pack(a, abits), oracle.pack(w, wbits)
    want = oracle.dense(ap, wp, m, n, k, abits, wbits, wenc, aenc)
    g = Guarded(m * n, torch.int32, SENT32)
    bs.bs_dense_ex(m, n, k, abits, aenc, wbits, wenc, dev(ap.view(np.int32)),
                   dev(wp.view(np.int32)), g.t)
    torch.cuda.synchronize()
    assert np.array_equal(g.t.cpu().numpy().reshape(m, n), want)
    g.check_guards()


def test_xnor_conv_worked_padding(oracle):
    """All +1 activations against +1 filters at 3x3 pad 1: every output is
    c times its number of in-range taps (zero padding of +-1 data)."""
    n, h, w, c, oc = 1, 7, 9, 100, 8
    a = np.ones((n, h, w, c), np.uint8)
    wq = np.ones((oc, 3, 3, c), np.uint8)
    p = bs.ConvParams(n, h, w, c, oc, 3, 3, 1, 1, 1, 1, 1, 1, 1, 1)
    got = bs.conv2d(bs.Conv2dSpec(n, h, w, c, oc, 3, 3, 1, 1, 1, 1,
                                  wenc=1, aenc=1),
                    bs.pack(dev(a), 1), bs.pack(dev(wq), 1)).cpu().numpy()
    assert bs.bs_conv2d_describe(p).startswith("conv_pix_kernel")
    taps = np.full((h, w), 9)
    taps[0, :] = taps[-1, :] = 6
    taps[:, 0] = taps[:, -1] = 6
    taps[0, 0] = taps[0, -1] = taps[-1, 0] = taps[-1, -1] = 4
    for o in range(oc):
        assert np.array_equal(got[0, :, :, o], c * taps)


def test_requant_other_encodings(oracle):
    """Requantized output of +-1 and signed convs (plain-loop requantizing
    kernel) equals the oracle's conv -> quantize -> pack."""
    for (abits, aenc, wbits, wenc) in [(1, 1, 1, 1), (2, 0, 3, 2),
                                       (3, 2, 3, 2)]:
        n, h, w, c, oc, k, s, pad = 2, 7, 8, 64, 40, 3, 1, 1
        say("requant enc", abits, aenc, wbits, wenc)
        rng = np.random.default_rng(abits + wenc)
        a = codes(rng, (n, h, w, c), abits)
        wq = codes(rng, (oc, k, k, c), wbits)
        ap, wp = oracle.pack(a, abits), oracle.pack(wq, wbits)
        conv = oracle.conv2d(oracle.conv_params(n, h, w, c, oc, k, k, s, pad,
                                                abits, wbits, aenc, wenc),
                             ap, wp)
        scale, obits = 0.05, 2
        want = oracle.pack(oracle.quantize(conv.astype(np.float32), scale,
                                           obits), obits)
        p = bs.ConvParams(n, h, w, c, oc, k, k, s, s, pad, pad, abits, wbits,
                          aenc, wenc)
        g = Guarded(want.size, torch.int32, SENT32)
        bs.bs_conv2d_requant(p, dev(ap.view(np.int32)),
                             dev(wp.view(np.int32)), scale, obits, g.t)
        torch.cuda.synchronize()
        assert np.array_equal(as_words(g.t).reshape(want.shape), want)
        g.check_guards()
