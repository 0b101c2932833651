"""GPU parity of the int8 matrix-core comparison baselines (hand-written
implicit-GEMM MFMA conv, and the library GEMM routes) against the oracle.

The oracle computes the same integer convolution from bit-packed codes:
activations as unipolar codes of up to 7 bits (int8 values 0..127) and
filters as signed 8-bit two's complement codes (int8 -128..127)."""
import numpy as np
import pytest
import torch

from paper_1810_11066_amd import int8_baseline as ib
from paper_1810_11066_amd import workloads as wl

pytestmark = pytest.mark.gpu

SENT32 = 0x7FFFFFFF


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU parity tests need the MI355X"
    ib.load_library()


def say(*a):
    print(*a, flush=True)


def oracle_conv(oracle, x, w, stride, pad, abits, wbits, wenc):
    """The oracle's conv of unsigned activation codes x (NHWC) and filter
    codes w (OHWI, two's complement bytes for signed filters)."""
    n, h, wd, c = x.shape
    oc, k = w.shape[0], w.shape[1]
    p = oracle.conv_params(n, h, wd, c, oc, k, k, stride, pad, abits, wbits,
                           wenc=wenc)
    return oracle.conv2d(p, oracle.pack(x.view(np.uint8), abits),
                         oracle.pack(w.view(np.uint8), wbits))


def run_mfma(x, w, stride, pad):
    n, h, wd, c = x.shape
    oc, k = w.shape[0], w.shape[1]
    oh = (h + 2 * pad - k) // stride + 1
    ow = (wd + 2 * pad - k) // stride + 1
    guard = 1024
    buf = torch.full((n * oh * ow * oc + 2 * guard,), SENT32,
                     dtype=torch.int32, device="cuda")
    out = buf[guard:guard + n * oh * ow * oc]
    ib.conv2d_mfma(torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda(),
                   stride, pad, out=out)
    torch.cuda.synchronize()
    b = buf.cpu().numpy()
    assert (b[:guard] == SENT32).all() and (b[-guard:] == SENT32).all()
    return out.cpu().numpy().reshape(n, oh, ow, oc)


@pytest.mark.parametrize("seed", range(30))
def test_mfma_conv_random(oracle, seed):
    rng = np.random.default_rng(9100 + seed)
    while True:   # filters within the kernel's 64 KiB of LDS
        k = int(rng.choice([1, 3]))
        c = 64 * int(rng.integers(1, 4))
        oc = 64 * int(rng.integers(1, 3))
        if oc * k * k * c <= 65536:
            break
    s = int(rng.choice([1, 2]))
    pad = int(rng.integers(0, 3))
    n = int(rng.integers(1, 4))
    h, w = int(rng.integers(1, 20)), int(rng.integers(1, 20))
    h, w = max(h, k - 2 * pad), max(w, k - 2 * pad)
    say("int8 mfma conv", (n, h, w, c, oc, k, s, pad))
    x = rng.integers(0, 128, size=(n, h, w, c), dtype=np.int8)
    wq = rng.integers(-128, 128, size=(oc, k, k, c), dtype=np.int8)
    got = run_mfma(x, wq, s, pad)
    assert np.array_equal(got, oracle_conv(oracle, x, wq, s, pad, 7, 8, 2))


@pytest.mark.parametrize("shape", [
    # (n, h, w, c, oc, k, stride, pad)
    (1, 6, 300, 64, 64, 3, 1, 1),    # input rows too wide for LDS: direct
    (2, 5, 260, 64, 128, 1, 2, 0),   # direct 1x1
    (3, 23, 29, 64, 64, 3, 2, 1),    # staged, tiles across images
    (2, 17, 19, 128, 128, 1, 1, 0),  # staged 1x1, two slices, two blocks
    (1, 1, 1, 64, 64, 3, 1, 1),      # one pixel, eight padded taps
    (5, 7, 9, 64, 64, 3, 1, 2),      # pad wider than the window reach
])
def test_mfma_conv_kernel_paths(oracle, shape):
    n, h, w, c, oc, k, s, pad = shape
    rng = np.random.default_rng(hash(shape) & 0xFFFF)
    say("int8 mfma conv", shape)
    x = rng.integers(0, 128, size=(n, h, w, c), dtype=np.int8)
    wq = rng.integers(-128, 128, size=(oc, k, k, c), dtype=np.int8)
    got = run_mfma(x, wq, s, pad)
    assert np.array_equal(got, oracle_conv(oracle, x, wq, s, pad, 7, 8, 2))


def test_mfma_conv_config2_full(oracle):
    """Config 2 (A2W1 ResNet-18 layer 2 at batch 64): the codes as int8
    through the matrix cores, every output against the oracle."""
    case = wl.config2()
    say(case.name)
    x = case.activations().astype(np.int8)
    wq = case.weights().astype(np.int8)
    got = run_mfma(x, wq, case.stride, case.pad)
    want = oracle_conv(oracle, x, wq, case.stride, case.pad, case.abits,
                       case.wbits, 0)
    assert np.array_equal(got, want)


def test_mfma_conv_refuses_uncovered_shapes():
    x = torch.zeros((1, 8, 8, 32), dtype=torch.int8, device="cuda")
    w = torch.zeros((64, 3, 3, 32), dtype=torch.int8, device="cuda")
    with pytest.raises(RuntimeError, match="status 2"):
        ib.conv2d_mfma(x, w, 1, 1)


def test_library_gemm_routes_against_oracle(oracle):
    """The library routes (im2col + torch._int_mm for the conv, one
    torch._int_mm for dense) on small shapes, against the oracle."""
    rng = np.random.default_rng(77)
    x = rng.integers(0, 4, size=(2, 9, 7, 64), dtype=np.uint8)
    wq = rng.integers(0, 2, size=(64, 3, 3, 64), dtype=np.uint8)
    got = ib.conv2d_int8(torch.from_numpy(x).cuda(),
                         torch.from_numpy(wq).cuda(), 1, 1).cpu().numpy()
    assert np.array_equal(got, oracle_conv(oracle, x, wq, 1, 1, 2, 1, 0))
    a = rng.integers(0, 4, size=(48, 256), dtype=np.uint8)
    wd = rng.integers(0, 4, size=(80, 256), dtype=np.uint8)
    got = ib.dense_int8(torch.from_numpy(a).cuda(),
                        torch.from_numpy(wd).cuda()).cpu().numpy()
    want = oracle.dense(oracle.pack(a, 2), oracle.pack(wd, 2), 48, 80, 256,
                        2, 2)
    assert np.array_equal(got, want)
