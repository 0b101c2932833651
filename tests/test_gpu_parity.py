"""GPU parity: the HIP library against the CPU oracle, bit for bit.

All calls go through the C ABI (the ctypes binding).  Outputs are written into
buffers pre-filled with a sentinel and flanked by guard bands, so a test also
fails if a kernel leaves an element unwritten or writes past its output.
Results are exact integers; the bar is equality.
"""
import ctypes

import numpy as np
import pytest
import torch

from paper_1810_11066_amd import bitserial as bs
from paper_1810_11066_amd import workloads as wl

pytestmark = pytest.mark.gpu

SENT32 = 0x7FFFFFFF
GUARD = 1024       # elements on each side (4 KiB for int32)


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU parity tests need the MI355X"
    bs.load_library()
    bs.bs_set_kernel_mode(0)
    yield
    bs.bs_set_kernel_mode(0)


def say(*a):
    print(*a, flush=True)


class Guarded:
    """A device buffer of `numel` elements with sentinel-filled guard bands."""

    def __init__(self, numel, dtype, sentinel):
        self.numel, self.sent = numel, sentinel
        self.buf = torch.full((numel + 2 * GUARD,), sentinel, dtype=dtype,
                              device="cuda")
        self.t = self.buf[GUARD:GUARD + numel]

    def view(self, *shape):
        return self.t.view(*shape)

    def check_guards(self):
        b = self.buf.cpu()
        assert bool((b[:GUARD] == self.sent).all()), "write before output"
        assert bool((b[GUARD + self.numel:] == self.sent).all()), \
            "write past output"


def dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def as_words(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().view(np.uint32)


# ---------------------------------------------------------------- quantize --

def special_floats(rng, n):
    parts = [rng.standard_normal(n).astype(np.float32) * 3,
             (rng.integers(-20, 600, n) / 2).astype(np.float32),
             rng.uniform(-1e-38, 1e-38, n).astype(np.float32),
             np.array([np.nan, np.inf, -np.inf, -0.0, 0.0, 1e30, -1e30,
                       0.5, 1.5, 2.5, 3.5], np.float32)]
    return np.concatenate(parts)


@pytest.mark.parametrize("n", [1, 15, 16, 17, 1000, 100003])
@pytest.mark.parametrize("bits,scale,enc", [
    (1, 1.0, 0), (2, 1.0, 0), (2, 1.5, 0), (3, 0.7, 0), (4, 3.0, 0),
    (8, 1.3, 0), (2, 3e38, 0), (1, 1.0, 1)])
def test_quantize(oracle, n, bits, scale, enc):
    say("quantize n=%d bits=%d scale=%g enc=%d" % (n, bits, scale, enc))
    rng = np.random.default_rng(n + bits)
    x = rng.permutation(special_floats(rng, n))[:n]
    want = oracle.quantize(x, scale, bits, enc)
    g = Guarded(n, torch.uint8, 0xAB)
    bs.bs_quantize(dev(x), g.t, scale, bits, enc)
    torch.cuda.synchronize()
    assert np.array_equal(g.t.cpu().numpy(), want)
    g.check_guards()


def test_quantize_golden(oracle):
    import json
    import os
    path = os.path.join(os.path.dirname(__file__), "golden",
                        "quantize_cases.json")
    for c in json.load(open(path))["cases"]:
        x = np.array([int(c["x"], 16)], np.uint32).view(np.float32)
        s = np.array([int(c["scale"], 16)], np.uint32).view(np.float32)[0]
        enc = 1 if c["enc"] == "bipolar" else 0
        q = torch.empty(1, dtype=torch.uint8, device="cuda")
        bs.bs_quantize(dev(x), q, float(s), c["bits"], enc)
        assert int(q.item()) == c["q"], c


# -------------------------------------------------------------------- pack --

@pytest.mark.parametrize("k", [1, 5, 31, 32, 33, 64, 70, 96, 128, 257, 512,
                               4096])
@pytest.mark.parametrize("bits", [1, 2, 3, 8])
@pytest.mark.parametrize("rows", [1, 3, 257])
def test_pack(oracle, k, bits, rows):
    say("pack rows=%d k=%d bits=%d" % (rows, k, bits))
    rng = np.random.default_rng(k * 7 + bits + rows)
    q = rng.integers(0, 256, size=(rows, k), dtype=np.uint8)  # high bits too
    want = oracle.pack(q, bits)
    g = Guarded(want.size, torch.int32, SENT32)
    bs.bs_pack(dev(q), g.t, rows, k, bits)
    torch.cuda.synchronize()
    assert np.array_equal(as_words(g.t).reshape(want.shape), want)
    g.check_guards()


def test_pack_grid_stride(oracle):
    # more words than one pass of the largest grid covers (8192 blocks x 512
    # words), so waves take several chunks, and a ragged last chunk
    rows, k, bits = 70001, 2048, 2
    say("pack grid stride rows=%d k=%d" % (rows, k))
    rng = np.random.default_rng(11)
    q = rng.integers(0, 256, size=(rows, k), dtype=np.uint8)
    want = oracle.pack(q, bits)
    g = Guarded(want.size, torch.int32, SENT32)
    bs.bs_pack(dev(q), g.t, rows, k, bits)
    torch.cuda.synchronize()
    assert np.array_equal(as_words(g.t).reshape(want.shape), want)
    g.check_guards()


def test_quantize_pack_grid_stride(oracle):
    # more words than one pass of the largest grid (8192 blocks x 256 words)
    rows, k, bits = 70001, 1024, 2
    say("quantize_pack grid stride rows=%d k=%d" % (rows, k))
    rng = np.random.default_rng(12)
    x = rng.standard_normal((rows, k), dtype=np.float32)
    want = oracle.pack(oracle.quantize(x, 1.3, bits), bits)
    g = Guarded(want.size, torch.int32, SENT32)
    bs.bs_quantize_pack(dev(x), g.t, rows, k, 1.3, bits)
    torch.cuda.synchronize()
    assert np.array_equal(as_words(g.t).reshape(want.shape), want)
    g.check_guards()


@pytest.mark.parametrize("k", [32, 64, 96, 100, 128, 256, 33, 4096])
@pytest.mark.parametrize("rows", [1, 5, 130])
@pytest.mark.parametrize("bits,enc", [(1, 0), (2, 0), (3, 0), (8, 0), (1, 1)])
def test_quantize_pack(oracle, k, rows, bits, enc):
    say("quantize_pack rows=%d k=%d bits=%d enc=%d" % (rows, k, bits, enc))
    rng = np.random.default_rng(k + rows * 3 + bits)
    x = rng.permutation(special_floats(rng, rows * k))[:rows * k]
    x = x.reshape(rows, k)
    want = oracle.pack(oracle.quantize(x, 1.7, bits, enc), bits)
    g = Guarded(want.size, torch.int32, SENT32)
    bs.bs_quantize_pack(dev(x), g.t, rows, k, 1.7, bits, enc)
    torch.cuda.synchronize()
    assert np.array_equal(as_words(g.t).reshape(want.shape), want)
    g.check_guards()


# -------------------------------------------------------------------- conv --

def run_conv(oracle, n, h, w, c, oc, kh, kw, sh, sw, ph, pw, abits, wbits,
             bipolar, seed, mode=0, check="full"):
    rng = np.random.default_rng(seed)
    a = rng.integers(0, 1 << abits, size=(n, h, w, c), dtype=np.uint8)
    wq = rng.integers(0, 1 << wbits, size=(oc, kh, kw, c), dtype=np.uint8)
    op = oracle.ConvParams(n, h, w, c, oc, kh, kw, sh, sw, ph, pw, abits,
                           wbits, 0, int(bipolar))
    ap, wp = oracle.pack(a, abits), oracle.pack(wq, wbits)
    p = bs.ConvParams(n, h, w, c, oc, kh, kw, sh, sw, ph, pw, abits, wbits,
                      0, int(bipolar))
    oh, ow = bs.bs_conv2d_out_shape(p)
    g = Guarded(n * oh * ow * oc, torch.int32, SENT32)
    # the library's own pack feeds the conv, as on the benchmark path
    a_dev = bs.pack(dev(a), abits)
    w_dev = bs.pack(dev(wq), wbits)
    bs.bs_set_kernel_mode(mode)
    try:
        bs.bs_conv2d(p, a_dev, w_dev, g.t)
    finally:
        bs.bs_set_kernel_mode(0)
    torch.cuda.synchronize()
    assert np.array_equal(as_words(a_dev).reshape(ap.shape), ap)
    assert np.array_equal(as_words(w_dev).reshape(wp.shape), wp)
    got = g.t.cpu().numpy().reshape(n, oh, ow, oc)
    g.check_guards()
    want = oracle.conv2d(op, ap, wp)
    assert np.array_equal(got, want)
    return got


def random_conv(rng):
    n = int(rng.integers(1, 3))
    h, w = int(rng.integers(1, 12)), int(rng.integers(1, 12))
    c = int(rng.integers(1, 140))
    oc = int(rng.integers(1, 80))
    kh, kw = int(rng.choice([1, 2, 3, 5])), int(rng.choice([1, 2, 3, 5]))
    sh, sw = int(rng.integers(1, 4)), int(rng.integers(1, 4))
    ph, pw = int(rng.integers(0, 3)), int(rng.integers(0, 3))
    if h + 2 * ph < kh:
        ph = (kh - h + 1) // 2
    if w + 2 * pw < kw:
        pw = (kw - w + 1) // 2
    abits, wbits = int(rng.integers(1, 9)), int(rng.integers(1, 9))
    return (n, h, w, c, oc, kh, kw, sh, sw, ph, pw, abits, wbits,
            bool(rng.integers(0, 2)))


@pytest.mark.parametrize("seed", range(40))
def test_conv_random_generic(oracle, seed):
    args = random_conv(np.random.default_rng(900 + seed))
    say("conv generic", args)
    run_conv(oracle, *args, seed=seed, mode=1)


def random_pixel_conv(rng):
    """A random shape inside the pixels-on-lanes kernel's domain: A, W <= 4
    (bipolar filters at W = 1), 1x1 or 3x3 windows, stride 1 or 2, padding
    0-2, a word count per plane the kernel is specialised for with a random
    tail, output channels a multiple of 4."""
    k = int(rng.choice([1, 3]))
    s = int(rng.choice([1, 2]))
    pad = int(rng.integers(0, 3))
    cw = int(rng.choice([1, 2, 4, 8, 16] + ([32] if k == 1 else [])))
    c = int(rng.integers(32 * (cw - 1) + 1, 32 * cw + 1))
    oc = 4 * int(rng.integers(1, 25))
    n = int(rng.integers(1, 3))
    h, w = int(rng.integers(1, 25)), int(rng.integers(1, 25))
    h, w = max(h, k - 2 * pad), max(w, k - 2 * pad)
    bipolar = bool(rng.integers(0, 2))
    abits = int(rng.integers(1, 5))
    wbits = 1 if bipolar else int(rng.integers(1, 5))
    return (n, h, w, c, oc, k, k, s, s, pad, pad, abits, wbits, bipolar)


@pytest.mark.parametrize("seed", range(60))
def test_conv_random_pixel_domain(oracle, seed):
    """Random shapes the pixel kernel takes (checked through the plan it
    reports), each at a random run length so that group visits and tile
    chunks break at varied places."""
    rng = np.random.default_rng(5000 + seed)
    args = random_pixel_conv(rng)
    run = int(rng.choice([0, 1, 2, 3, 5, 7, 13]))
    say("conv pixel domain", args, "run", run)
    p = bs.ConvParams(*args[:13], 0, int(args[13]))
    bs.bs_set_kernel_mode(3)
    try:
        assert bs.bs_conv2d_describe(p).startswith("conv_pix_kernel")
    finally:
        bs.bs_set_kernel_mode(0)
    bs.bs_set_units_per_wave(run)
    try:
        run_conv(oracle, *args, seed=seed, mode=3)
    finally:
        bs.bs_set_units_per_wave(0)


@pytest.mark.parametrize("mode", [0, 2, 3])
@pytest.mark.parametrize("seed", range(40))
def test_conv_random_fast(oracle, seed, mode):
    args = random_conv(np.random.default_rng(900 + seed))
    say("conv mode", mode, args)
    run_conv(oracle, *args, seed=seed, mode=mode)


# shapes that take the specialised kernel: K in {1,3}, S in {1,2}, even word
# count, A, W <= 4; ragged oc, widths that are not multiples of the group
# size, borders on every side, several images
FAST_SHAPES = [
    # n, h, w, c, oc, k, s, pad
    (2, 9, 11, 64, 64, 3, 1, 1),
    (1, 10, 9, 32, 68, 3, 1, 1),
    (2, 8, 7, 20, 36, 3, 2, 1),
    (1, 12, 12, 128, 40, 1, 1, 0),
    (1, 14, 14, 64, 100, 3, 1, 1),
    (3, 7, 7, 128, 64, 3, 1, 1),
    (2, 10, 13, 64, 70, 3, 2, 1),
    (1, 8, 8, 192, 64, 1, 1, 0),
    (2, 9, 9, 64, 65, 1, 2, 0),
    (1, 5, 17, 256, 33, 3, 1, 0),
    (1, 6, 6, 64, 128, 3, 2, 0),
    (2, 16, 9, 64, 64, 3, 1, 2),
]


# mode 2: output-channels-on-lanes kernel, mode 3: pixels-on-lanes kernel
# (each falls back to the generic kernel where it does not apply)
@pytest.mark.parametrize("mode", [2, 3])
@pytest.mark.parametrize("shape", FAST_SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("abits,wbits,bip", [
    (1, 1, False), (1, 1, True), (2, 1, False), (2, 1, True), (2, 2, False),
    (3, 3, False), (3, 3, True), (4, 4, False), (1, 4, False), (4, 1, True)])
def test_conv_fast_shapes(oracle, shape, abits, wbits, bip, mode):
    n, h, w, c, oc, k, s, pad = shape
    say("conv fast", shape, abits, wbits, bip, "mode", mode)
    run_conv(oracle, n, h, w, c, oc, k, k, s, s, pad, pad, abits, wbits, bip,
             seed=hash((shape, abits, wbits, bip)) % 10000, mode=mode)


# Runs of units (64 pixels x 4 channels) that start and end inside groups,
# cross group boundaries, and flush 4, 8, 12 and 16 channel tiles.
RUN_SHAPES = [
    # n, h, w, c, oc, k, s, pad
    (2, 9, 11, 64, 64, 3, 1, 1),      # 4 groups (last one partial) x 16 quads
    (1, 10, 9, 32, 12, 3, 1, 1),      # 3 quads per group
    (2, 8, 7, 64, 36, 3, 2, 1),       # 9 quads, stride 2
    (1, 12, 12, 128, 40, 1, 1, 0),    # 1x1, 10 quads, 3 groups
    (3, 7, 7, 128, 20, 3, 1, 1),      # 4 words per plane
]


@pytest.mark.parametrize("run", [1, 2, 3, 5, 7, 16, 37, 100000])
@pytest.mark.parametrize("shape", RUN_SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("abits,wbits,bip", [(2, 1, False), (1, 1, True),
                                             (2, 2, False)])
def test_conv_pixel_runs(oracle, shape, run, abits, wbits, bip):
    n, h, w, c, oc, k, s, pad = shape
    say("conv pixel runs", shape, run, abits, wbits, bip)
    bs.bs_set_units_per_wave(run)
    try:
        run_conv(oracle, n, h, w, c, oc, k, k, s, s, pad, pad, abits, wbits,
                 bip, seed=run * 7 + oc, mode=3)
    finally:
        bs.bs_set_units_per_wave(0)


# Wide layers: the pixel kernel holds one filter row or one tap of the patch
# at a time and adds tap-block partial sums in its LDS tile.
WIDE_SHAPES = [
    # n, h, w, c, oc, k, s, pad
    (2, 6, 7, 256, 24, 3, 1, 1),
    (1, 5, 5, 512, 20, 3, 2, 1),
    (2, 7, 6, 256, 36, 3, 2, 0),
    (1, 4, 9, 512, 8, 3, 1, 1),
    (1, 9, 4, 224, 28, 3, 1, 1),     # 7 words per plane: generic fallback
]


@pytest.mark.parametrize("shape", WIDE_SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("abits,wbits,bip", [
    (1, 1, False), (1, 1, True), (2, 1, False), (2, 1, True), (2, 2, False),
    (3, 3, False)])
def test_conv_wide_shapes(oracle, shape, abits, wbits, bip):
    n, h, w, c, oc, k, s, pad = shape
    say("conv wide", shape, abits, wbits, bip)
    run_conv(oracle, n, h, w, c, oc, k, k, s, s, pad, pad, abits, wbits, bip,
             seed=hash((shape, abits, wbits, bip, 1)) % 10000, mode=3)


@pytest.mark.parametrize("run", [1, 3, 5, 9, 100000])
@pytest.mark.parametrize("shape", WIDE_SHAPES[:3], ids=lambda s: "x".join(map(str, s)))
def test_conv_wide_runs(oracle, shape, run):
    n, h, w, c, oc, k, s, pad = shape
    say("conv wide runs", shape, run)
    bs.bs_set_units_per_wave(run)
    try:
        run_conv(oracle, n, h, w, c, oc, k, k, s, s, pad, pad, 2, 1, True,
                 seed=run + oc, mode=3)
    finally:
        bs.bs_set_units_per_wave(0)


# 1x1 layers and dense rows too wide for one patch: the reduction is split
# into blocks of 8 or 16 words per plane (double-buffered patch blocks).
@pytest.mark.parametrize("m,n,k", [(64, 8, 4096), (100, 20, 2048),
                                   (130, 12, 1024), (70, 36, 4096)])
@pytest.mark.parametrize("abits,wbits,bip", [(2, 2, False), (1, 1, True),
                                             (2, 1, False), (3, 3, False)])
def test_dense_word_blocks(oracle, m, n, k, abits, wbits, bip):
    say("dense word blocks", m, n, k, abits, wbits, bip)
    rng = np.random.default_rng(m * 31 + n + k + abits)
    a = rng.integers(0, 1 << abits, size=(m, k), dtype=np.uint8)
    w = rng.integers(0, 1 << wbits, size=(n, k), dtype=np.uint8)
    ap, wp = oracle.pack(a, abits), oracle.pack(w, wbits)
    want = oracle.dense(ap, wp, m, n, k, abits, wbits, int(bip))
    g = Guarded(m * n, torch.int32, SENT32)
    bs.bs_set_kernel_mode(3)
    try:
        bs.bs_dense(m, n, k, abits, wbits, int(bip), dev(ap.view(np.int32)),
                    dev(wp.view(np.int32)), g.t)
    finally:
        bs.bs_set_kernel_mode(0)
    torch.cuda.synchronize()
    assert np.array_equal(g.t.cpu().numpy().reshape(m, n), want)
    g.check_guards()


def test_conv_deterministic(oracle):
    args = (2, 14, 14, 64, 64, 3, 3, 1, 1, 1, 1, 2, 1, False)
    a = run_conv(oracle, *args, seed=5)
    b = run_conv(oracle, *args, seed=5)
    assert np.array_equal(a, b)


# ------------------------------------------------------------------- dense --

@pytest.mark.parametrize("seed", range(16))
def test_dense_random(oracle, seed):
    rng = np.random.default_rng(300 + seed)
    m, n = int(rng.integers(1, 300)), int(rng.integers(1, 200))
    k = int(rng.choice([1, 31, 64, 100, 256, 1000, 2048]))
    abits, wbits = int(rng.integers(1, 5)), int(rng.integers(1, 5))
    bip = bool(rng.integers(0, 2))
    say("dense", m, n, k, abits, wbits, bip)
    a = rng.integers(0, 1 << abits, size=(m, k), dtype=np.uint8)
    w = rng.integers(0, 1 << wbits, size=(n, k), dtype=np.uint8)
    ap, wp = oracle.pack(a, abits), oracle.pack(w, wbits)
    want = oracle.dense(ap, wp, m, n, k, abits, wbits, int(bip))
    g = Guarded(m * n, torch.int32, SENT32)
    bs.bs_dense(m, n, k, abits, wbits, int(bip), dev(ap.view(np.int32)),
                dev(wp.view(np.int32)), g.t)
    torch.cuda.synchronize()
    assert np.array_equal(g.t.cpu().numpy().reshape(m, n), want)
    g.check_guards()


def test_dense_operands_may_alias(oracle):
    """A . A^T from one packed matrix passed as both operands: inputs may
    alias each other (only an output overlapping an input is refused)."""
    rng = np.random.default_rng(77)
    m, k, bits = 96, 320, 2
    say("dense alias", m, k, bits)
    a = rng.integers(0, 1 << bits, size=(m, k), dtype=np.uint8)
    ap = oracle.pack(a, bits)
    want = oracle.dense(ap, ap, m, m, k, bits, bits, 0)
    a_dev = dev(ap.view(np.int32))
    out = torch.empty((m, m), dtype=torch.int32, device="cuda")
    bs.bs_dense(m, m, k, bits, bits, 0, a_dev, a_dev, out)
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy(), want)


def test_conv_output_adjacent_and_overlapping(oracle):
    """One allocation holding the packed input and, right after its last
    byte, the output: a valid call.  With the output moved 16 bytes back
    onto the input, the call is refused and writes nothing."""
    rng = np.random.default_rng(78)
    n, h, w, c, oc = 2, 9, 11, 64, 24
    codes = rng.integers(0, 4, size=(n * h * w, c), dtype=np.uint8)
    filt = rng.integers(0, 2, size=(oc * 9, c), dtype=np.uint8)
    ap, wp = oracle.pack(codes, 2), oracle.pack(filt, 1)
    spec = bs.Conv2dSpec(n, h, w, c, oc, 3, 3, 1, 1, 2, 1)
    want = oracle.conv2d(oracle.conv_params(n, h, w, c, oc, 3, 3, 1, 1, 2, 1),
                         ap, wp)
    act_words = ap.size
    out_elems = n * h * w * oc
    say("conv adjacent", act_words, out_elems)
    buf = torch.full((act_words + out_elems,), SENT32, dtype=torch.int32,
                     device="cuda")
    buf[:act_words] = dev(ap.view(np.int32).ravel())
    w_dev = dev(wp.view(np.int32))
    act = buf[:act_words]
    out = buf[act_words:]
    bs.bs_conv2d(spec.params(), act, w_dev, out)
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy().reshape(want.shape), want)
    assert np.array_equal(as_words(act).reshape(ap.shape), ap)
    before = buf.clone()
    lib = bs.load_library()
    st = lib.bs_conv2d(ctypes.byref(spec.params()), act.data_ptr(),
                       w_dev.data_ptr(), buf[act_words - 4:].data_ptr(),
                       ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == bs.BS_ERR_INVALID_ARG
    assert b"overlaps" in lib.bs_last_error()
    torch.cuda.synchronize()
    assert torch.equal(buf, before)


def test_concurrent_threads_and_streams(oracle):
    """Four host threads, each on its own stream (default priority) and in
    its own kernel mode, pack and convolve different shapes at the same
    time; every result equals the oracle's."""
    import threading
    # (n, h, w, c, oc, k, stride, pad, abits, wbits, bipolar w, kernel mode)
    jobs = [(2, 14, 14, 64, 64, 3, 1, 1, 2, 1, False, 0),
            (1, 9, 13, 96, 40, 3, 2, 1, 1, 1, True, 2),
            (3, 7, 7, 128, 36, 1, 1, 0, 3, 2, False, 3),
            (1, 6, 6, 32, 12, 3, 1, 1, 2, 2, False, 1)]
    prepared = []
    for i, (n, h, w, c, oc, k, st, pd, ab, wb, bip, mode) in enumerate(jobs):
        rng = np.random.default_rng(900 + i)
        codes = rng.integers(0, 1 << ab, size=(n, h, w, c), dtype=np.uint8)
        filt = rng.integers(0, 1 << wb, size=(oc, k, k, c), dtype=np.uint8)
        wenc = 1 if bip else 0
        want = oracle.conv2d(
            oracle.conv_params(n, h, w, c, oc, k, k, st, pd, ab, wb,
                               wenc=wenc),
            oracle.pack(codes.reshape(-1, c), ab),
            oracle.pack(filt.reshape(-1, c), wb))
        spec = bs.Conv2dSpec(n, h, w, c, oc, k, k, st, pd, ab, wb, wenc)
        prepared.append((dev(codes), bs.pack(dev(filt.reshape(-1, c)), wb),
                         spec, ab, mode, want))
    torch.cuda.synchronize()
    errors = []

    def run(x, w_dev, spec, ab, mode, want):
        try:
            bs.bs_set_kernel_mode(mode)
            stream = torch.cuda.Stream()
            outs = []
            with torch.cuda.stream(stream):
                for _ in range(25):
                    a_dev = bs.pack(x.view(-1, x.shape[-1]), ab)
                    outs.append(bs.conv2d(spec, a_dev, w_dev))
            stream.synchronize()
            for o in outs:
                if not np.array_equal(o.cpu().numpy(), want):
                    errors.append("mode %d: result differs" % mode)
                    break
        except Exception as e:        # reported in the main thread
            errors.append("mode %d: %r" % (mode, e))
        finally:
            bs.bs_set_kernel_mode(0)

    say("concurrent", len(prepared), "threads")
    threads = [threading.Thread(target=run, args=job) for job in prepared]
    for t in threads:
        t.start()
    for t in threads:
        t.join(120)
    assert not any(t.is_alive() for t in threads)
    assert errors == []


# ------------------------------------------- requantized (chained) output --

def run_requant(oracle, n, h, w, c, oc, k, s, pad, abits, wbits, bip, scale,
                obits, seed, mode=0, run=0):
    rng = np.random.default_rng(seed)
    a = rng.integers(0, 1 << abits, size=(n, h, w, c), dtype=np.uint8)
    wq = rng.integers(0, 1 << wbits, size=(oc, k, k, c), dtype=np.uint8)
    ap, wp = oracle.pack(a, abits), oracle.pack(wq, wbits)
    conv = oracle.conv2d(oracle.conv_params(n, h, w, c, oc, k, k, s, pad,
                                            abits, wbits, wenc=int(bip)),
                         ap, wp)
    # the next layer's input: quantize the float32 values, pack over channels
    want = oracle.pack(oracle.quantize(conv.astype(np.float32), scale, obits),
                       obits)
    p = bs.ConvParams(n, h, w, c, oc, k, k, s, s, pad, pad, abits, wbits, 0,
                      int(bip))
    g = Guarded(want.size, torch.int32, SENT32)
    bs.bs_set_kernel_mode(mode)
    bs.bs_set_units_per_wave(run)
    try:
        bs.bs_conv2d_requant(p, dev(ap.view(np.int32)), dev(wp.view(np.int32)),
                             scale, obits, g.t)
    finally:
        bs.bs_set_kernel_mode(0)
        bs.bs_set_units_per_wave(0)
    torch.cuda.synchronize()
    assert np.array_equal(as_words(g.t).reshape(want.shape), want)
    g.check_guards()


REQUANT_SHAPES = [
    # n, h, w, c, oc, k, s, pad
    (2, 9, 11, 64, 64, 3, 1, 1),
    (1, 10, 9, 32, 36, 3, 1, 1),      # a partial last word (4 channels)
    (2, 8, 7, 64, 96, 3, 2, 1),
    (1, 12, 12, 128, 40, 1, 1, 0),
    (2, 6, 7, 256, 64, 3, 1, 1),      # row blocks: partial sums in the tile
    (1, 5, 5, 512, 32, 3, 2, 1),      # tap blocks
    (1, 7, 6, 64, 70, 3, 1, 1),       # oc % 4 != 0: plain-loop kernel
]


@pytest.mark.parametrize("seed", range(30))
def test_conv_requant_random(oracle, seed):
    """Random pixel-domain shapes (output channels often not a multiple of
    8, so the last packed byte is partial) with 1- to 8-bit requantized
    output at a random run length; shapes are drawn where the plain conv's
    plan is the pixel kernel, whose requantizing variant then runs."""
    rng = np.random.default_rng(8000 + seed)
    k, s, pad = int(rng.choice([1, 3])), int(rng.choice([1, 2])), \
        int(rng.integers(0, 3))
    cw = int(rng.choice([1, 2, 4, 8] + ([16] if k == 1 else [])))
    c = int(rng.integers(32 * (cw - 1) + 1, 32 * cw + 1))
    oc = 4 * int(rng.integers(1, 25))
    n = int(rng.integers(1, 3))
    h = max(int(rng.integers(1, 20)), k - 2 * pad)
    w = max(int(rng.integers(1, 20)), k - 2 * pad)
    bip = bool(rng.integers(0, 2))
    abits = int(rng.integers(1, 5))
    wbits = 1 if bip else int(rng.integers(1, 5))
    obits = int(rng.integers(1, 9))
    run = int(rng.choice([0, 1, 2, 3, 5, 7, 13]))
    # a scale that spreads the results over the output codes
    scale = ((1 << obits) - 1) / (0.5 * k * k * c * ((1 << abits) - 1) + 1)
    p = bs.ConvParams(n, h, w, c, oc, k, k, s, s, pad, pad, abits, wbits, 0,
                      int(bip))
    bs.bs_set_kernel_mode(3)
    try:
        assert bs.bs_conv2d_describe(p).startswith("conv_pix_kernel")
    finally:
        bs.bs_set_kernel_mode(0)
    say("conv requant random", (n, h, w, c, oc, k, s, pad), abits, wbits,
        bip, obits, "run", run)
    run_requant(oracle, n, h, w, c, oc, k, s, pad, abits, wbits, bip, scale,
                obits, seed=seed, mode=0, run=run)


@pytest.mark.parametrize("seed", range(30))
def test_conv_channels_on_lanes_random(oracle, seed):
    """Random shapes inside the channels-on-lanes kernel's domain (even word
    counts per plane, any number of output channels); the plan must be
    that kernel."""
    rng = np.random.default_rng(9000 + seed)
    k, s, pad = int(rng.choice([1, 3])), int(rng.choice([1, 2])), \
        int(rng.integers(0, 3))
    cw = int(rng.choice([2, 4, 8]))
    c = int(rng.integers(32 * (cw - 1) + 1, 32 * cw + 1))
    oc = int(rng.integers(1, 150))
    n = int(rng.integers(1, 3))
    h = max(int(rng.integers(1, 20)), k - 2 * pad)
    w = max(int(rng.integers(1, 30)), k - 2 * pad)
    bip = bool(rng.integers(0, 2))
    abits = int(rng.integers(1, 5))
    wbits = 1 if bip else int(rng.integers(1, 5))
    p = bs.ConvParams(n, h, w, c, oc, k, k, s, s, pad, pad, abits, wbits, 0,
                      int(bip))
    bs.bs_set_kernel_mode(2)
    try:
        assert bs.bs_conv2d_describe(p).startswith("conv_ocl_kernel")
    finally:
        bs.bs_set_kernel_mode(0)
    args = (n, h, w, c, oc, k, k, s, s, pad, pad, abits, wbits, bip)
    say("conv channels-on-lanes random", args)
    run_conv(oracle, *args, seed=seed, mode=2)


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("shape", REQUANT_SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("abits,wbits,bip,obits", [
    (2, 1, False, 2), (1, 1, True, 1), (2, 2, False, 3), (3, 3, False, 8)])
def test_conv_requant(oracle, shape, abits, wbits, bip, obits, mode):
    n, h, w, c, oc, k, s, pad = shape
    say("conv requant", shape, abits, wbits, bip, obits, "mode", mode)
    # a scale that spreads the results over the output codes
    scale = ((1 << obits) - 1) / (0.5 * k * k * c * ((1 << abits) - 1) + 1)
    run_requant(oracle, n, h, w, c, oc, k, s, pad, abits, wbits, bip, scale,
                obits, seed=hash((shape, abits, obits)) % 10000, mode=mode)


@pytest.mark.parametrize("run", [1, 2, 3, 100000])
@pytest.mark.parametrize("shape", REQUANT_SHAPES[:3] + REQUANT_SHAPES[4:5],
                         ids=lambda s: "x".join(map(str, s)))
def test_conv_requant_runs(oracle, shape, run):
    n, h, w, c, oc, k, s, pad = shape
    say("conv requant runs", shape, run)
    run_requant(oracle, n, h, w, c, oc, k, s, pad, 2, 1, False, 0.01, 2,
                seed=run + 3 * oc, mode=3, run=run)


def test_conv_requant_special_scales(oracle):
    # saturation (every result at the top code), everything rounding to 0,
    # and ties: a scale of 0.5 puts odd results exactly halfway
    for scale in (1e6, 1e-9, 0.5):
        run_requant(oracle, 2, 9, 11, 64, 64, 3, 1, 1, 2, 1, False, scale, 2,
                    seed=17)


# ------------------------------------------------- int8 comparison baseline --

# ------------------------------------------------ batch split past 2 GB --

def test_conv_batch_split_over_2gb(oracle):
    # an int32 output of 2.16 GB is more than one launch of the pixel kernel
    # addresses (32-bit offsets): the batch is split into image chunks.  The
    # chunk boundary (127 images, then 1) is checked against the oracle on
    # whole images and against the generic kernel everywhere.
    n, h, w, c, oc = 128, 56, 56, 32, 1344
    say("conv batch split", n, h, w, c, oc)
    rng = np.random.default_rng(2048)
    a = rng.integers(0, 2, size=(n, h, w, c), dtype=np.uint8)
    wq = rng.integers(0, 2, size=(oc, 1, 1, c), dtype=np.uint8)
    ap, wp = oracle.pack(a, 1), oracle.pack(wq, 1)
    spec = bs.Conv2dSpec(n, h, w, c, oc, 1, 1, 1, 0, 1, 1)
    assert "batch split" in bs.bs_conv2d_describe(spec.params())
    a_dev, w_dev = dev(ap.view(np.int32)), dev(wp.view(np.int32))
    out = bs.conv2d(spec, a_dev, w_dev)
    bs.bs_set_kernel_mode(1)
    try:
        ref = bs.conv2d(spec, a_dev, w_dev)
    finally:
        bs.bs_set_kernel_mode(0)
    torch.cuda.synchronize()
    assert torch.equal(out, ref)
    del ref
    per_image = h * w * oc
    idx = np.concatenate([np.arange(125 * per_image, n * per_image),
                          rng.integers(0, n * per_image, 65536)])
    got = out.view(-1)[torch.from_numpy(idx).cuda()].cpu().numpy()
    want = oracle.conv2d_at(oracle.conv_params(n, h, w, c, oc, 1, 1, 1, 0, 1,
                                               1), ap, wp, idx)
    assert np.array_equal(got, want)
