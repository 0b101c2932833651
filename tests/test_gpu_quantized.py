"""GPU parity of the fused call bs_conv2d_quantized (float32 activations
quantized and bit-packed inside a 1x1 conv kernel) against the oracle's
quantize -> pack -> conv2d on the same seeded inputs.

The quantizer is the library's reading of Sec. 3.1 (round half to even of
the binary32 product, clamped, NaN to 0), so the inputs mix N(0,1) values
with the cases that reading decides: exact halfway points, values past
the top code, negatives, -0, NaN and +-inf.  Strided windows gather one
input pixel per output pixel; padding, strides and run lengths vary which
pixels a workgroup gathers."""
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


def activations(rng, shape, scale, abits):
    """N(0,1) values, a fifth of them replaced by the quantizer's edge
    cases."""
    x = rng.standard_normal(shape, dtype=np.float32)
    qmax = (1 << abits) - 1
    edge = np.array([np.nan, np.inf, -np.inf, -0.0, 0.0, -1.0,
                     (qmax + 0.5) / scale, (qmax + 7) / scale,
                     0.5 / scale, 1.5 / scale, 2.5 / scale,
                     (qmax - 0.5) / scale], dtype=np.float32)
    pick = rng.random(shape) < 0.2
    x[pick] = rng.choice(edge, size=int(pick.sum()))
    return x


LDS_BYTES = 64 * 1024          # per workgroup
TILE_BYTES = 4 * 64 * 17 * 4   # the four waves' output tiles


def smallest_plan_fits(n, h, w, c, oc, s, ph, pw, abits):
    """Whether the packed input pixels of the smallest share a workgroup can
    take (4 units of 64 output pixels x 4 channels) fit its LDS: at stride 2
    the pixels gathered for its output pixels, at stride 1 the flat input
    range its outputs read.  The fused call may refuse a shape only when
    they do not."""
    oh, ow = (h + 2 * ph - 1) // s + 1, (w + 2 * pw - 1) // s + 1
    npix, gu = n * oh * ow, oc // 4
    units = (npix + 63) // 64 * gu
    worst = 0
    for ub0 in range(0, units, 4):
        ub1 = min(ub0 + 4, units)
        p0, p1 = ub0 // gu * 64, min((ub1 - 1) // gu * 64 + 63, npix - 1)
        if s > 1:
            worst = max(worst, p1 + 1 - p0)
            continue
        # stride 1: input pixel (y - ph, x - pw) of output pixel (y, x)
        taps = [(img * h + y - ph) * w + x - pw
                for img, y, x in (((q // ow) // oh, (q // ow) % oh, q % ow)
                                  for q in range(p0, p1 + 1))
                if 0 <= y - ph < h and 0 <= x - pw < w]
        if taps:
            worst = max(worst, max(taps) + 1 - min(taps))
    return TILE_BYTES + (worst + 1) * abits * (c // 32) * 4 <= LDS_BYTES


def run_quantized(oracle, n, h, w, c, oc, s, ph, pw, abits, wbits, bip,
                  scale, seed, run=0):
    rng = np.random.default_rng(seed)
    x = activations(rng, (n, h, w, c), scale, abits)
    wq = rng.integers(0, 1 << wbits, size=(oc, 1, 1, c), dtype=np.uint8)
    op = oracle.conv_params(n, h, w, c, oc, 1, 1, (s, s), (ph, pw), abits,
                            wbits, wenc=int(bip))
    want = oracle.conv2d(op, oracle.pack(oracle.quantize(x, scale, abits),
                                         abits), oracle.pack(wq, wbits))
    p = bs.ConvParams(n, h, w, c, oc, 1, 1, s, s, ph, pw, abits, wbits, 0,
                      int(bip))
    try:
        assert bs.bs_conv2d_quantized_describe(p).startswith(
            "conv_pix_kernel<A=%d,W=%d" % (abits, wbits))
    except bs.BitserialError as e:
        assert e.status == bs.BS_ERR_UNSUPPORTED
        assert not smallest_plan_fits(n, h, w, c, oc, s, ph, pw, abits), \
            "refused a shape that fits"
        say("refused: the smallest plan's input pixels exceed the LDS")
        return
    oh, ow = bs.bs_conv2d_out_shape(p)
    numel = n * oh * ow * oc
    buf = torch.full((numel + 2 * GUARD,), SENT32, dtype=torch.int32,
                     device="cuda")
    x_dev, w_dev = dev(x), bs.pack(dev(wq), wbits)
    out = buf[GUARD:GUARD + numel]
    bs.bs_set_units_per_wave(run)
    try:
        bs.bs_conv2d_quantized(p, x_dev, scale, w_dev, out)
    except bs.BitserialError as e:
        # a forced run whose workgroups' pixels overflow the LDS is refused;
        # the library's own plan shortens runs until they fit
        if e.status != bs.BS_ERR_UNSUPPORTED or run == 0:
            raise
        bs.bs_set_units_per_wave(0)
        bs.bs_conv2d_quantized(p, x_dev, scale, w_dev, out)
    finally:
        bs.bs_set_units_per_wave(0)
    torch.cuda.synchronize()
    b = buf.cpu()
    assert bool((b[:GUARD] == SENT32).all()), "write before output"
    assert bool((b[GUARD + numel:] == SENT32).all()), "write past output"
    assert np.array_equal(out.cpu().numpy().reshape(want.shape), want)


@pytest.mark.parametrize("seed", range(50))
def test_conv2d_quantized_random(oracle, seed):
    rng = np.random.default_rng(9300 + seed)
    s = int(rng.choice([1, 2]))
    ph, pw = int(rng.integers(0, 2)), int(rng.integers(0, 2))
    cw = int(rng.choice([1, 2, 4, 8, 16, 32]))
    abits = int(rng.integers(1, 5))
    bip = bool(rng.integers(0, 2))
    wbits = 1 if bip else int(rng.integers(1, 5))
    n = int(rng.integers(1, 4))
    h, w = int(rng.integers(1, 20)), int(rng.integers(1, 20))
    oc = 4 * int(rng.integers(1, 33))
    scale = float(rng.choice([0.7, 1.0, 1.3, 2.9]))
    run = int(rng.choice([0, 0, 1, 2, 3, 4, 5, 7, 13]))
    args = (n, h, w, 32 * cw, oc, s, ph, pw, abits, wbits, bip, scale)
    say("conv2d_quantized", args, "run", run)
    run_quantized(oracle, *args, seed=seed, run=run)


def test_conv2d_quantized_refuses_3x3(oracle):
    p = bs.ConvParams(1, 8, 8, 64, 64, 3, 3, 1, 1, 1, 1, 2, 1, 0, 0)
    x = torch.zeros((1, 8, 8, 64), dtype=torch.float32, device="cuda")
    w = torch.zeros((64, 3, 3, 1, 2), dtype=torch.int32, device="cuda")
    out = torch.full((1, 8, 8, 64), 7, dtype=torch.int32, device="cuda")
    with pytest.raises(bs.BitserialError) as e:
        bs.bs_conv2d_quantized(p, x, 1.0, w, out)
    assert e.value.status == bs.BS_ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert bool((out == 7).all()), "a refused call wrote its output"


@pytest.mark.parametrize("case", [c for c in wl.config4() if c.k == 1],
                         ids=lambda c: c.name)
def test_config4_1x1_layers_quantized(oracle, case):
    """Config 4's 1x1 layers (float32 N(0,1) activations at the layer's
    scale) through the fused call, every output element against the
    oracle."""
    say(case.name)
    x = case.activations()
    wq = case.weights()
    p = bs.ConvParams(case.n, case.h, case.w, case.c, case.oc, 1, 1,
                      case.stride, case.stride, case.pad, case.pad,
                      case.abits, case.wbits, 0, case.wenc)
    oh, ow = bs.bs_conv2d_out_shape(p)
    out = torch.empty((case.n, oh, ow, case.oc), dtype=torch.int32,
                      device="cuda")
    bs.bs_conv2d_quantized(p, dev(x), case.act_scale,
                           bs.pack(dev(wq), case.wbits), out)
    torch.cuda.synchronize()
    op = oracle.conv_params(case.n, case.h, case.w, case.c, case.oc, 1, 1,
                            case.stride, case.pad, case.abits, case.wbits,
                            wenc=case.wenc)
    want = oracle.conv2d(op, oracle.pack(oracle.quantize(x, case.act_scale,
                                                         case.abits),
                                         case.abits),
                         oracle.pack(wq, case.wbits))
    got = out.cpu().numpy()
    bad = np.flatnonzero(got.ravel() != want.ravel())
    assert bad.size == 0, "%d outputs differ from the oracle, first at %d" % (
        bad.size, bad[0])


@pytest.mark.parametrize("stride", [1, 2])
def test_conv2d_quantized_split_by_input_size(oracle, stride):
    """Float32 activations of more than 2 GiB: the call splits the batch
    into launches whose float32 input stays within one buffer (32-bit
    offsets); at stride 2 each launch gathers its pixels.  Every output
    against the oracle."""
    n, h, w, c, oc, abits, scale = 257, 64, 64, 512, 4, 2, 1.3
    say("conv2d_quantized split", (n, h, w, c, oc, stride))
    assert n * h * w * c * 4 > 2 ** 31
    rng = np.random.default_rng(515151 + stride)
    x = rng.standard_normal((n, h, w, c), dtype=np.float32)
    wq = rng.integers(0, 2, size=(oc, 1, 1, c), dtype=np.uint8)
    op = oracle.conv_params(n, h, w, c, oc, 1, 1, stride, 0, abits, 1)
    want = oracle.conv2d(op, oracle.pack(oracle.quantize(x, scale, abits),
                                         abits), oracle.pack(wq, 1))
    p = bs.ConvParams(n, h, w, c, oc, 1, 1, stride, stride, 0, 0, abits, 1,
                      0, 0)
    oh, ow = bs.bs_conv2d_out_shape(p)
    numel = n * oh * ow * oc
    buf = torch.full((numel + 2 * GUARD,), SENT32, dtype=torch.int32,
                     device="cuda")
    x_dev = dev(x)
    del x
    bs.bs_conv2d_quantized(p, x_dev, scale, bs.pack(dev(wq), 1),
                           buf[GUARD:GUARD + numel])
    torch.cuda.synchronize()
    del x_dev
    b = buf.cpu()
    assert bool((b[:GUARD] == SENT32).all()), "write before output"
    assert bool((b[GUARD + numel:] == SENT32).all()), "write past output"
    got = b[GUARD:GUARD + numel].numpy().reshape(want.shape)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("stride", [1, 2])
def test_conv2d_quantized_subnormals(oracle, stride):
    """Subnormal activations times a scale of 2e38 land on codes 0-2 (the
    quantizer keeps subnormals; flushed to zero they would all give 0)."""
    n, h, w, c, oc, abits, scale = 2, 11, 13, 128, 20, 2, 2e38
    say("conv2d_quantized subnormals", (n, h, w, c, oc, stride))
    rng = np.random.default_rng(616 + stride)
    x = rng.uniform(-1.2e-38, 1.2e-38, size=(n, h, w, c)).astype(np.float32)
    assert (np.abs(x) < np.finfo(np.float32).tiny).mean() > 0.9
    wq = rng.integers(0, 2, size=(oc, 1, 1, c), dtype=np.uint8)
    codes = oracle.quantize(x, scale, abits)
    assert codes.max() == 2 and (codes > 0).mean() > 0.3
    op = oracle.conv_params(n, h, w, c, oc, 1, 1, stride, 0, abits, 1)
    want = oracle.conv2d(op, oracle.pack(codes, abits), oracle.pack(wq, 1))
    p = bs.ConvParams(n, h, w, c, oc, 1, 1, stride, stride, 0, 0, abits, 1,
                      0, 0)
    oh, ow = bs.bs_conv2d_out_shape(p)
    out = torch.empty((n, oh, ow, oc), dtype=torch.int32, device="cuda")
    bs.bs_conv2d_quantized(p, dev(x), scale, bs.pack(dev(wq), 1), out)
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy(), want)
