"""GPU parity of the fused call bs_conv2d_codes (bit-pack of uint8 codes
inside the conv kernel) against the oracle's pack -> conv2d on the same
seeded inputs, for whole-window kernels and for kernels that split the
reduction into blocks read from the staged region.

Each workgroup of these kernels packs the input rows its outputs read into
LDS, so the tests vary what decides those regions: image sizes, strides,
padding, and the run of units each wave takes (blocks that start and end
inside images and span image boundaries)."""
import numpy as np
import pytest
import torch

from paper_1810_11066_amd import bitserial as bs
from paper_1810_11066_amd import workloads as wl

pytestmark = pytest.mark.gpu

SENT32 = 0x7FFFFFFF
GUARD = 1024


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU parity tests need the MI355X"
    bs.load_library()
    bs.bs_set_kernel_mode(0)
    yield
    bs.bs_set_units_per_wave(0)


def say(*a):
    print(*a, flush=True)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


class Guarded:
    """int32 device buffer with sentinel guard bands on both sides."""

    def __init__(self, numel):
        self.numel = numel
        self.buf = torch.full((numel + 2 * GUARD,), SENT32, dtype=torch.int32,
                              device="cuda")
        self.t = self.buf[GUARD:GUARD + numel]

    def check_guards(self):
        b = self.buf.cpu()
        assert bool((b[:GUARD] == SENT32).all()), "write before output"
        assert bool((b[GUARD + self.numel:] == SENT32).all()), \
            "write past output"


def window_words(k, abits, cw):
    return k * k * abits * cw


def random_staged(rng):
    """A shape the fused kernels cover: c a multiple of 32, oc of 4, 1x1 or
    3x3 windows, stride 1 or 2, unipolar activations of 1-4 bits with
    unipolar filters of 1-2 bits or bipolar 1-bit filters, and the whole
    window within 72 words."""
    while True:
        k = int(rng.choice([1, 3]))
        s = int(rng.choice([1, 2]))
        pad = int(rng.integers(0, 3))
        abits = int(rng.integers(1, 5))
        bipolar = bool(rng.integers(0, 2))
        wbits = 1 if bipolar else int(rng.integers(1, 3))
        cw = int(rng.choice([1, 2, 4, 8, 16]))
        if window_words(k, abits, cw) <= 72 and wbits * cw <= 24:
            break
    n = int(rng.integers(1, 4))
    h, w = int(rng.integers(1, 25)), int(rng.integers(1, 25))
    h, w = max(h, k - 2 * pad), max(w, k - 2 * pad)
    oc = 4 * int(rng.integers(1, 25))
    return n, h, w, 32 * cw, oc, k, s, pad, abits, wbits, bipolar


LDS_BYTES = 64 * 1024          # per workgroup
TILE_BYTES = 4 * 64 * 17 * 4   # the four waves' output tiles


def smallest_plan_fits(n, h, w, c, oc, k, s, pad, abits):
    """Whether the packed input rows of the smallest share a workgroup can
    take (4 units of 64 output pixels x 4 channels) fit its LDS: the fused
    call may refuse a shape only when they do not."""
    oh, ow = (h + 2 * pad - k) // s + 1, (w + 2 * pad - k) // s + 1
    npix, gu = n * oh * ow, oc // 4
    units = (npix + 63) // 64 * gu
    pwb = abits * (c // 32) * 4
    worst = 0
    for ub0 in range(0, units, 4):
        ub1 = min(ub0 + 4, units)
        p0, p1 = ub0 // gu * 64, min((ub1 - 1) // gu * 64 + 63, npix - 1)
        n0, y0 = divmod(p0 // ow, oh)
        n1, y1 = divmod(p1 // ow, oh)
        lo_row = min(max(y0 * s - pad, 0), h)
        hi_row = max(min(y1 * s - pad + k - 1, h - 1), -1)
        lo = (n0 * h + lo_row) * w
        hi = max((n1 * h + hi_row) * w + w, lo)
        worst = max(worst, hi - lo)
    return TILE_BYTES + (worst + 1) * pwb <= LDS_BYTES


def call_fused(fn, p, run, shape):
    """fn() under the run-length override; a run that makes a workgroup's
    rows too large for LDS is retried with the library's own plan, and a
    refusal of that is accepted only when even the smallest plan cannot
    fit.  Returns False when the shape was (rightly) refused."""
    bs.bs_set_units_per_wave(run)
    try:
        fn()
        return True
    except bs.BitserialError as e:
        if e.status != bs.BS_ERR_UNSUPPORTED:
            raise
    finally:
        bs.bs_set_units_per_wave(0)
    if run != 0:
        try:
            fn()
            return True
        except bs.BitserialError as e:
            if e.status != bs.BS_ERR_UNSUPPORTED:
                raise
    assert not smallest_plan_fits(*shape), "refused a shape that fits"
    say("refused: the smallest plan's input rows exceed the LDS")
    return False


def expect(oracle, codes, wq, n, h, w, c, oc, k, s, pad, abits, wbits, bip):
    ap = oracle.pack(codes, abits)
    wp = oracle.pack(wq, wbits)
    p = oracle.conv_params(n, h, w, c, oc, k, k, s, pad, abits, wbits,
                           wenc=int(bip))
    return oracle.conv2d(p, ap, wp)


def run_codes(oracle, args, seed, run=0):
    n, h, w, c, oc, k, s, pad, abits, wbits, bip = args
    rng = np.random.default_rng(seed)
    # every byte value: bits at or above abits must be ignored
    codes = rng.integers(0, 256, size=(n, h, w, c), dtype=np.uint8)
    wq = rng.integers(0, 1 << wbits, size=(oc, k, k, c), dtype=np.uint8)
    want = expect(oracle, codes, wq, *args)
    spec = bs.Conv2dSpec(n, h, w, c, oc, k, k, s, pad, abits, wbits,
                         int(bip))
    p = spec.params()
    oh, ow = bs.bs_conv2d_out_shape(p)
    g = Guarded(n * oh * ow * oc)
    w_dev = bs.pack(dev(wq), wbits)
    c_dev = dev(codes)
    if not call_fused(lambda: bs.bs_conv2d_codes(p, c_dev, w_dev, g.t), p,
                      run, (n, h, w, c, oc, k, s, pad, abits)):
        return
    torch.cuda.synchronize()
    got = g.t.cpu().numpy().reshape(n, oh, ow, oc)
    g.check_guards()
    assert np.array_equal(got, want)


@pytest.mark.parametrize("seed", range(60))
def test_conv2d_codes_random(oracle, seed):
    rng = np.random.default_rng(7100 + seed)
    args = random_staged(rng)
    run = int(rng.choice([0, 0, 1, 2, 3, 5, 7, 13]))
    say("conv2d_codes", args, "run", run)
    run_codes(oracle, args, seed=seed, run=run)


def random_staged_blocks(rng):
    """A shape whose fused kernel splits the reduction into blocks (the
    kh x kw x abits x c/32-word window above 72 words: one filter row, one
    tap, or one tap and part of each plane per block), or whose filters
    have 3 or 4 bits."""
    while True:
        k = int(rng.choice([1, 3]))
        s = int(rng.choice([1, 2]))
        pad = int(rng.integers(0, 2)) if k == 3 else 0
        abits = int(rng.integers(1, 5))
        bipolar = bool(rng.integers(0, 3) == 0)
        wbits = 1 if bipolar else int(rng.integers(1, 5))
        cw = int(rng.choice([4, 8, 16] if k == 3 else [16, 32, 64, 128]))
        if window_words(k, abits, cw) > 72 or wbits >= 3:
            break
    n = int(rng.integers(1, 3))
    h, w = int(rng.integers(1, 13)), int(rng.integers(1, 13))
    h, w = max(h, k - 2 * pad), max(w, k - 2 * pad)
    oc = 4 * int(rng.integers(1, 13))
    return n, h, w, 32 * cw, oc, k, s, pad, abits, wbits, bipolar


@pytest.mark.parametrize("seed", range(40))
def test_conv2d_codes_blocks_random(oracle, seed):
    rng = np.random.default_rng(7300 + seed)
    args = random_staged_blocks(rng)
    run = int(rng.choice([0, 0, 1, 2, 3, 5, 7, 13]))
    say("conv2d_codes blocks", args, "run", run)
    run_codes(oracle, args, seed=seed, run=run)


# fixed shapes: ResNet-style layers at small batch, blocks spanning images
CODES_SHAPES = [
    # n, h, w, c, oc, k, s, pad, abits, wbits, bipolar
    (3, 14, 14, 64, 64, 3, 1, 1, 2, 1, False),
    (2, 9, 11, 64, 64, 3, 1, 1, 2, 1, True),
    (3, 8, 8, 128, 128, 3, 2, 1, 2, 1, False),
    (4, 7, 7, 128, 36, 3, 1, 1, 2, 1, False),
    (2, 12, 12, 64, 128, 1, 2, 0, 2, 1, False),
    (2, 6, 6, 256, 64, 1, 1, 0, 2, 1, False),
    (2, 5, 5, 32, 8, 3, 1, 2, 4, 2, False),
    (5, 3, 3, 64, 4, 3, 2, 1, 1, 1, True),
    # padding above K - 1: whole output rows and blocks in the padding
    (2, 24, 22, 64, 68, 1, 1, 2, 4, 1, False),
    (3, 5, 6, 64, 8, 1, 2, 2, 2, 1, False),
    (2, 4, 4, 32, 8, 3, 1, 3, 2, 1, False),
    # reduction blocks: filter rows, taps, taps x part of each plane
    (2, 14, 14, 256, 64, 3, 1, 1, 2, 1, False),
    (2, 14, 14, 256, 32, 3, 1, 1, 4, 4, False),
    (2, 14, 14, 256, 64, 3, 2, 1, 3, 3, False),
    (3, 7, 7, 512, 16, 3, 1, 1, 2, 1, False),
    (2, 9, 9, 512, 8, 3, 1, 1, 1, 1, True),
    (2, 10, 9, 128, 36, 3, 2, 1, 3, 3, False),
    (1, 5, 7, 4096, 16, 1, 1, 0, 2, 2, False),
    (2, 6, 6, 1024, 8, 1, 2, 0, 4, 3, False),
]


@pytest.mark.parametrize("run", [0, 1, 3, 16, 100000])
@pytest.mark.parametrize("shape", CODES_SHAPES,
                         ids=lambda s: "x".join(map(str, s)))
def test_conv2d_codes_shapes(oracle, shape, run):
    say("conv2d_codes shape", shape, "run", run)
    run_codes(oracle, shape, seed=run + 17 * shape[4], run=run)


def test_conv2d_codes_unsupported_writes_nothing(oracle):
    # c not a multiple of 32: the fused kernels do not cover it
    n, h, w, c, oc = 1, 6, 6, 48, 8
    spec = bs.Conv2dSpec(n, h, w, c, oc, 3, 3, 1, 1, 2, 1)
    g = Guarded(n * h * w * oc)
    codes = torch.zeros((n, h, w, c), dtype=torch.uint8, device="cuda")
    w_dev = torch.zeros((oc * 9 * 1 * 2,), dtype=torch.int32, device="cuda")
    with pytest.raises(bs.BitserialError) as e:
        bs.bs_conv2d_codes(spec.params(), codes, w_dev, g.t)
    assert e.value.status == bs.BS_ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert bool((g.t == SENT32).all().item())
    g.check_guards()


def test_config2_conv2d_codes_full(oracle):
    """Config 2 (the benchmark's workload) through the fused call, every
    output element against the oracle."""
    case = wl.config2()
    say(case.name)
    codes = case.activations()
    wq = case.weights()
    want = expect(oracle, codes, wq, case.n, case.h, case.w, case.c, case.oc,
                  case.k, case.stride, case.pad, case.abits, case.wbits,
                  False)
    spec = bs.Conv2dSpec(case.n, case.h, case.w, case.c, case.oc, case.k,
                         case.k, case.stride, case.pad, case.abits,
                         case.wbits)
    got = bs.conv2d_codes(spec, dev(codes), bs.pack(dev(wq), case.wbits))
    assert np.array_equal(got.cpu().numpy(), want)


def test_conv2d_codes_split_by_codes_size(oracle):
    """Codes of more than 2 GiB: the call splits the batch into launches
    whose uint8 codes stay within one buffer (the packed words, a quarter
    of the size, would fit one launch).  Every output against the oracle."""
    n, h, w, c, oc = 1025, 64, 64, 512, 4
    args = (n, h, w, c, oc, 1, 1, 0, 2, 1, False)
    say("conv2d_codes split", args)
    assert n * h * w * c > 2 ** 31
    rng = np.random.default_rng(424242)
    codes = rng.integers(0, 256, size=(n, h, w, c), dtype=np.uint8)
    wq = rng.integers(0, 2, size=(oc, 1, 1, c), dtype=np.uint8)
    want = expect(oracle, codes, wq, *args)
    spec = bs.Conv2dSpec(n, h, w, c, oc, 1, 1, 1, 0, 2, 1)
    g = Guarded(n * h * w * oc)
    c_dev = dev(codes)
    del codes
    bs.bs_conv2d_codes(spec.params(), c_dev, bs.pack(dev(wq), 1), g.t)
    torch.cuda.synchronize()
    got = g.t.cpu().numpy().reshape(n, h, w, oc)
    g.check_guards()
    assert np.array_equal(got, want)
