"""GPU parity of the paired call bs_conv2d_pair (a KxK conv and the 1x1 conv
of the same stride whose input pixel is the window's centre tap, one pass)
and of bs_conv2d_pair_requant, against the oracle's two convolutions (and
its quantize -> pack of each result for the requantized form).

Shapes cover the paired kernels' domain (3x3 windows, whole patches, up to
16 filter words per quad of the 1x1 conv), shapes outside it (run as two
convolutions), several run lengths per wave, and the three downsampling
pairs of ResNet-18 (Table 1 layers 4/5, 7/8, 10/11) at batch 128."""
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


def oracle_pair(oracle, codes, w3, w1, n, h, w, c, oc, k, s, abits, wbits,
                bip):
    """The oracle's KxK conv (pad (k-1)/2) and 1x1 conv (pad 0), each the
    plain definition on the packed operands."""
    ap = oracle.pack(codes, abits)
    p3 = oracle.conv_params(n, h, w, c, oc, k, k, s, (k - 1) // 2, abits,
                            wbits, wenc=int(bip))
    p1 = oracle.conv_params(n, h, w, c, oc, 1, 1, s, 0, abits, wbits,
                            wenc=int(bip))
    return (oracle.conv2d(p3, ap, oracle.pack(w3, wbits)),
            oracle.conv2d(p1, ap, oracle.pack(w1, wbits)))


def draw(rng, n, h, w, c, oc, k, abits, wbits):
    codes = rng.integers(0, 1 << abits, size=(n, h, w, c), dtype=np.uint8)
    w3 = rng.integers(0, 1 << wbits, size=(oc, k, k, c), dtype=np.uint8)
    w1 = rng.integers(0, 1 << wbits, size=(oc, 1, 1, c), dtype=np.uint8)
    return codes, w3, w1


def run_pair(oracle, shape, seed, run=0, requant_bits=0):
    n, h, w, c, oc, k, s, abits, wbits, bip = shape
    rng = np.random.default_rng(seed)
    codes, w3, w1 = draw(rng, n, h, w, c, oc, k, abits, wbits)
    want3, want1 = oracle_pair(oracle, codes, w3, w1, *shape)
    spec = bs.Conv2dSpec(n, h, w, c, oc, k, k, s, (k - 1) // 2, abits, wbits,
                         int(bip))
    p = spec.params()
    oh, ow = bs.bs_conv2d_out_shape(p)
    assert want3.shape == want1.shape == (n, oh, ow, oc)
    a_dev = bs.pack(dev(codes), abits)
    w3_dev = bs.pack(dev(w3), wbits)
    w1_dev = bs.pack(dev(w1), wbits)
    if requant_bits:
        ob = requant_bits
        # scales that map about twice the mean result to the top code
        mean3 = max(float(np.abs(want3).mean()), 1.0)
        mean1 = max(float(np.abs(want1).mean()), 1.0)
        sc3, sc1 = ((1 << ob) - 1) / (2 * mean3), ((1 << ob) - 1) / (2 * mean1)
        numel = n * oh * ow * ob * bs.words(oc)
        g3, g1 = Guarded(numel), Guarded(numel)
        bs.bs_set_units_per_wave(run)
        try:
            bs.bs_conv2d_pair_requant(p, a_dev, w3_dev, w1_dev, sc3, sc1, ob,
                                      g3.t, g1.t)
        finally:
            bs.bs_set_units_per_wave(0)
        torch.cuda.synchronize()
        for g, want, sc in ((g3, want3, sc3), (g1, want1, sc1)):
            q = oracle.pack(oracle.quantize(want.astype(np.float32), sc, ob),
                            ob)
            got = g.t.cpu().numpy().view(np.uint32).reshape(q.shape)
            g.check_guards()
            assert np.array_equal(got, q)
        return
    g3, g1 = Guarded(n * oh * ow * oc), Guarded(n * oh * ow * oc)
    bs.bs_set_units_per_wave(run)
    try:
        bs.bs_conv2d_pair(p, a_dev, w3_dev, w1_dev, g3.t, g1.t)
    finally:
        bs.bs_set_units_per_wave(0)
    torch.cuda.synchronize()
    for g, want in ((g3, want3), (g1, want1)):
        got = g.t.cpu().numpy().reshape(want.shape)
        g.check_guards()
        assert np.array_equal(got, want)


def random_pair(rng):
    """3x3 stride 1 or 2 (sometimes 1x1 or 5x5 windows, which the plain
    kernels take), activations 1-4 bits, unipolar filters of 1-2 bits or
    bipolar 1-bit ones, 1-8 words per plane (8: outside the paired kernels),
    output channels mostly a multiple of 4."""
    k = int(rng.choice([3, 3, 3, 1, 5]))
    s = int(rng.choice([1, 2]))
    abits = int(rng.integers(1, 5))
    bip = bool(rng.integers(0, 2))
    wbits = 1 if bip else int(rng.integers(1, 3))
    cw = int(rng.choice([1, 2, 4, 8]))
    c = int(rng.integers(32 * (cw - 1) + 1, 32 * cw + 1))
    oc = 4 * int(rng.integers(1, 20)) + (int(rng.integers(0, 4))
                                         if rng.integers(0, 5) == 0 else 0)
    n = int(rng.integers(1, 4))
    h, w = int(rng.integers(1, 20)), int(rng.integers(1, 20))
    return n, h, w, c, oc, k, s, abits, wbits, bip


@pytest.mark.parametrize("seed", range(50))
def test_pair_random(oracle, seed):
    rng = np.random.default_rng(8100 + seed)
    shape = random_pair(rng)
    run = int(rng.choice([0, 0, 1, 2, 3, 7, 13]))
    say("pair", shape, "run", run)
    run_pair(oracle, shape, seed, run)


@pytest.mark.parametrize("seed", range(30))
def test_pair_requant_random(oracle, seed):
    rng = np.random.default_rng(8300 + seed)
    shape = random_pair(rng)
    run = int(rng.choice([0, 0, 1, 3, 5]))
    ob = int(rng.integers(1, 5))
    say("pair requant", shape, "run", run, "bits", ob)
    run_pair(oracle, shape, seed, run, requant_bits=ob)


PAIR_SHAPES = [
    # n, h, w, c, oc, k, s, abits, wbits, bipolar
    (3, 14, 14, 64, 128, 3, 2, 2, 1, False),   # ResNet-18 layers 4/5 shape
    (2, 14, 14, 128, 256, 3, 2, 2, 1, False),  # layers 7/8
    (2, 7, 7, 256, 128, 3, 2, 2, 1, False),    # layers 10/11 (two launches)
    (2, 9, 11, 64, 64, 3, 1, 1, 1, True),
    (4, 5, 5, 32, 36, 3, 2, 4, 2, False),
]


@pytest.mark.parametrize("run", [0, 1, 3, 16, 100000])
@pytest.mark.parametrize("shape", PAIR_SHAPES,
                         ids=lambda s: "x".join(map(str, s)))
def test_pair_shapes(oracle, shape, run):
    say("pair shape", shape, "run", run)
    run_pair(oracle, shape, seed=run + shape[4], run=run)
    run_pair(oracle, shape, seed=run + shape[4], run=run, requant_bits=2)


def test_pair_rejects_other_windows(oracle):
    """Windows whose centre tap is not the 1x1 conv's input pixel (padding
    other than (k-1)/2, unequal strides, even windows) are refused and
    nothing is written."""
    codes = torch.zeros((1, 8, 8, 64), dtype=torch.uint8, device="cuda")
    a = bs.pack(codes, 2)
    w1 = torch.zeros((16 * 2,), dtype=torch.int32, device="cuda")
    for p in (bs.ConvParams(1, 8, 8, 64, 16, 3, 3, 1, 1, 0, 1, 2, 1, 0, 0),
              bs.ConvParams(1, 8, 8, 64, 16, 3, 3, 1, 2, 1, 1, 2, 1, 0, 0),
              bs.ConvParams(1, 8, 8, 64, 16, 2, 2, 1, 1, 0, 0, 2, 1, 0, 0)):
        oh, ow = bs.bs_conv2d_out_shape(p)
        w3 = torch.zeros((16 * p.kh * p.kw * 2,), dtype=torch.int32,
                         device="cuda")
        out = torch.full((oh * ow * 16,), SENT32, dtype=torch.int32,
                         device="cuda")
        out1 = torch.full_like(out, SENT32)
        with pytest.raises(bs.BitserialError) as e:
            bs.bs_conv2d_pair(p, a, w3, w1, out, out1)
        assert e.value.status == bs.BS_ERR_INVALID_ARG
        torch.cuda.synchronize()
        assert bool((out == SENT32).all().item())
        assert bool((out1 == SENT32).all().item())


RESNET_PAIRS = [(4, 5), (7, 8), (10, 11)]


@pytest.mark.parametrize("main,short", RESNET_PAIRS,
                         ids=lambda v: "L%d" % v)
def test_resnet18_downsampling_pairs_full(oracle, main, short):
    """Table 1's downsampling pairs at batch 128, A2W1, the input quantized
    from float32 N(0,1) with config 4's scale for the main layer: both
    outputs, every element, against the oracle."""
    case = {c.name: c for c in wl.config4()}["resnet18_L%d_b128" % main]
    case1 = {c.name: c for c in wl.config4()}["resnet18_L%d_b128" % short]
    assert (case.h, case.c, case.oc, case.stride) == \
        (case1.h, case1.c, case1.oc, case1.stride)
    say(case.name, "+", case1.name)
    x = case.activations()
    codes = oracle.quantize(x, case.act_scale, case.abits)
    w3 = case.weights()
    w1 = case1.weights()
    want3, want1 = oracle_pair(oracle, codes, w3, w1, case.n, case.h, case.w,
                               case.c, case.oc, 3, case.stride, case.abits,
                               case.wbits, False)
    spec = bs.Conv2dSpec(case.n, case.h, case.w, case.c, case.oc, 3, 3,
                         case.stride, 1, case.abits, case.wbits)
    a_dev = bs.quantize_pack(dev(x), case.act_scale, case.abits)
    got3, got1 = bs.conv2d_pair(spec, a_dev, bs.pack(dev(w3), case.wbits),
                                bs.pack(dev(w1), case.wbits))
    assert np.array_equal(got3.cpu().numpy(), want3)
    assert np.array_equal(got1.cpu().numpy(), want1)
