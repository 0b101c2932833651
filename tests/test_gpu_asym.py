"""GPU parity with different padding above/below and left/right (pad_h !=
pad_w), through the pixels-on-lanes kernel on packed input and the fused
call on uint8 codes, against the oracle's conv2d of the same seeded inputs.

The pixel kernels take the row padding and the column padding separately:
a window's first row and column, the taps that read zeros, and the fused
kernel's staged input range (whose first and last tap rows are cut at
columns derived from the column padding) each depend on one of them, so
equal paddings would hide a swap of the two."""
import numpy as np
import pytest
import torch

from paper_1810_11066_amd import bitserial as bs

pytestmark = pytest.mark.gpu

SENT32 = 0x7FFFFFFF
GUARD = 1024


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU parity tests need the MI355X"
    bs.load_library()
    bs.bs_set_kernel_mode(0)
    yield
    bs.bs_set_kernel_mode(0)
    bs.bs_set_units_per_wave(0)


def say(*a):
    print(*a, flush=True)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def guarded(numel):
    return torch.full((numel + 2 * GUARD,), SENT32, dtype=torch.int32,
                      device="cuda")


def check_guards(buf, numel):
    b = buf.cpu()
    assert bool((b[:GUARD] == SENT32).all()), "write before output"
    assert bool((b[GUARD + numel:] == SENT32).all()), "write past output"


def random_shape(rng, staged):
    """A square 1x1 or 3x3 window, stride 1 or 2, different row and column
    padding (0-2), and widths the pixel kernels take (the fused call: c a
    multiple of 32, 1-2 bit unipolar or 1-bit bipolar filters)."""
    k = int(rng.choice([1, 3]))
    s = int(rng.choice([1, 2]))
    ph, pw = [int(x) for x in rng.choice(3, size=2, replace=False)]
    cw = int(rng.choice([1, 2, 4]))
    c = 32 * cw if staged else int(rng.integers(32 * (cw - 1) + 1,
                                                32 * cw + 1))
    oc = 4 * int(rng.integers(1, 20))
    n = int(rng.integers(1, 4))
    h = max(int(rng.integers(1, 20)), k - 2 * ph)
    w = max(int(rng.integers(1, 20)), k - 2 * pw)
    bipolar = bool(rng.integers(0, 2))
    abits = int(rng.integers(1, 5))
    wbits = 1 if bipolar else int(rng.integers(1, 3))
    return n, h, w, c, oc, k, s, ph, pw, abits, wbits, bipolar


def conv_case(oracle, shape, seed, codes_range):
    n, h, w, c, oc, k, s, ph, pw, abits, wbits, bip = shape
    rng = np.random.default_rng(seed)
    codes = rng.integers(0, codes_range, size=(n, h, w, c), dtype=np.uint8)
    wq = rng.integers(0, 1 << wbits, size=(oc, k, k, c), dtype=np.uint8)
    op = oracle.conv_params(n, h, w, c, oc, k, k, (s, s), (ph, pw), abits,
                            wbits, wenc=int(bip))
    want = oracle.conv2d(op, oracle.pack(codes, abits),
                         oracle.pack(wq, wbits))
    p = bs.ConvParams(n, h, w, c, oc, k, k, s, s, ph, pw, abits, wbits, 0,
                      int(bip))
    return codes, wq, p, want


@pytest.mark.parametrize("seed", range(30))
def test_pixel_kernel_asymmetric_padding(oracle, seed):
    rng = np.random.default_rng(8100 + seed)
    shape = random_shape(rng, staged=False)
    run = int(rng.choice([0, 1, 3, 5, 7]))
    say("pixel kernel, pad_h != pad_w", shape, "run", run)
    n, h, w, c, oc, k, s, ph, pw, abits, wbits, bip = shape
    codes, wq, p, want = conv_case(oracle, shape, seed, 1 << abits)
    bs.bs_set_kernel_mode(3)
    try:
        assert bs.bs_conv2d_describe(p).startswith("conv_pix_kernel")
        oh, ow = bs.bs_conv2d_out_shape(p)
        buf = guarded(n * oh * ow * oc)
        bs.bs_set_units_per_wave(run)
        bs.bs_conv2d(p, bs.pack(dev(codes), abits), bs.pack(dev(wq), wbits),
                     buf[GUARD:GUARD + n * oh * ow * oc])
    finally:
        bs.bs_set_units_per_wave(0)
        bs.bs_set_kernel_mode(0)
    torch.cuda.synchronize()
    got = buf[GUARD:GUARD + n * oh * ow * oc].cpu().numpy()
    check_guards(buf, n * oh * ow * oc)
    assert np.array_equal(got.reshape(want.shape), want)


@pytest.mark.parametrize("seed", range(30))
def test_fused_codes_asymmetric_padding(oracle, seed):
    rng = np.random.default_rng(8200 + seed)
    shape = random_shape(rng, staged=True)
    run = int(rng.choice([0, 1, 2, 3, 5, 7, 13]))
    say("fused codes, pad_h != pad_w", shape, "run", run)
    n, h, w, c, oc, k, s, ph, pw, abits, wbits, bip = shape
    # every byte value: code bits at or above abits must be ignored
    codes, wq, p, want = conv_case(oracle, shape, seed, 256)
    assert bs.bs_conv2d_codes_describe(p).startswith("conv_pix_kernel")
    oh, ow = bs.bs_conv2d_out_shape(p)
    buf = guarded(n * oh * ow * oc)
    c_dev, w_dev = dev(codes), bs.pack(dev(wq), wbits)
    out = buf[GUARD:GUARD + n * oh * ow * oc]
    bs.bs_set_units_per_wave(run)
    try:
        bs.bs_conv2d_codes(p, c_dev, w_dev, out)
    except bs.BitserialError as e:
        # a forced run whose workgroups' input rows overflow the LDS is
        # refused; the library's own plan shortens runs until they fit
        if e.status != bs.BS_ERR_UNSUPPORTED or run == 0:
            raise
        bs.bs_set_units_per_wave(0)
        bs.bs_conv2d_codes(p, c_dev, w_dev, out)
    finally:
        bs.bs_set_units_per_wave(0)
    torch.cuda.synchronize()
    got = buf[GUARD:GUARD + n * oh * ow * oc].cpu().numpy()
    check_guards(buf, n * oh * ow * oc)
    assert np.array_equal(got.reshape(want.shape), want)
