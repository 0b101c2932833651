"""Pin the oracle's conv2d and dense to things other than itself.

* brute force: an int64 numpy convolution / matmul on the UNPACKED codes (no
  bit-planes involved), weight value w for unipolar and 2w - (2^W - 1) for
  bipolar weights (bit 1 = +1, bit 0 = -1 per plane, Sec. 2.2);
* Eq. 2 evaluated literally with numpy popcounts over the packed words, the
  bipolar form being popcount(a AND w) - popcount(a AND NOT w);
* the bit-plane identity: an A-bit conv equals sum_i 2^i times the 1-bit
  convs of the activation planes (Eq. 2 weighting);
* closed forms: all-ones data at 3x3 pad 1 gives (2^A-1)(2^W-1) C times the
  number of in-range taps (4 corner, 6 edge, 9 interior); and
  conv_bipolar(a, w) = 2 conv_unipolar(a, w) - (2^W - 1) conv_unipolar(a, 1).
"""
import numpy as np
import pytest

from paper_1810_11066_amd import workloads as wl


def weight_values(q, wbits, bipolar):
    q = q.astype(np.int64)
    return 2 * q - ((1 << wbits) - 1) if bipolar else q


def brute_conv(a, wv, sh, sw, ph, pw):
    """a: [n][h][w][c] codes, wv: [oc][kh][kw][c] integer weight values."""
    n, h, w, c = a.shape
    oc, kh, kw, _ = wv.shape
    xp = np.zeros((n, h + 2 * ph, w + 2 * pw, c), np.int64)
    xp[:, ph:ph + h, pw:pw + w, :] = a
    oh = (h + 2 * ph - kh) // sh + 1
    ow = (w + 2 * pw - kw) // sw + 1
    out = np.zeros((n, oh, ow, oc), np.int64)
    for r in range(kh):
        for s in range(kw):
            patch = xp[:, r:r + sh * (oh - 1) + 1:sh, s:s + sw * (ow - 1) + 1:sw]
            out += np.tensordot(patch, wv[:, r, s, :], axes=([3], [1]))
    return out


def random_conv_case(rng):
    n = int(rng.integers(1, 3))
    h, w = int(rng.integers(1, 10)), int(rng.integers(1, 10))
    c = int(rng.integers(1, 71))
    oc = int(rng.integers(1, 10))
    kh, kw = int(rng.choice([1, 2, 3, 5])), int(rng.choice([1, 2, 3, 5]))
    sh, sw = int(rng.integers(1, 4)), int(rng.integers(1, 4))
    ph, pw = int(rng.integers(0, 3)), int(rng.integers(0, 3))
    if h + 2 * ph < kh:
        ph = (kh - h + 1) // 2
    if w + 2 * pw < kw:
        pw = (kw - w + 1) // 2
    abits, wbits = int(rng.integers(1, 5)), int(rng.integers(1, 5))
    bipolar = bool(rng.integers(0, 2))
    return n, h, w, c, oc, kh, kw, sh, sw, ph, pw, abits, wbits, bipolar


@pytest.mark.parametrize("seed", range(120))
def test_conv_bruteforce_random(oracle, seed):
    rng = np.random.default_rng(1000 + seed)
    (n, h, w, c, oc, kh, kw, sh, sw, ph, pw, abits, wbits,
     bipolar) = random_conv_case(rng)
    a = rng.integers(0, 1 << abits, size=(n, h, w, c), dtype=np.uint8)
    wq = rng.integers(0, 1 << wbits, size=(oc, kh, kw, c), dtype=np.uint8)
    p = oracle.ConvParams(n, h, w, c, oc, kh, kw, sh, sw, ph, pw, abits,
                          wbits, 0, int(bipolar))
    got = oracle.conv2d(p, oracle.pack(a, abits), oracle.pack(wq, wbits))
    want = brute_conv(a, weight_values(wq, wbits, bipolar), sh, sw, ph, pw)
    assert got.shape == want.shape
    assert np.array_equal(got.astype(np.int64), want)


@pytest.mark.parametrize("seed", range(40))
def test_dense_bruteforce_random(oracle, seed):
    rng = np.random.default_rng(5000 + seed)
    m, n, k = (int(rng.integers(1, 20)), int(rng.integers(1, 20)),
               int(rng.integers(1, 200)))
    abits, wbits = int(rng.integers(1, 9)), int(rng.integers(1, 9))
    bipolar = bool(rng.integers(0, 2))
    a = rng.integers(0, 1 << abits, size=(m, k), dtype=np.uint8)
    w = rng.integers(0, 1 << wbits, size=(n, k), dtype=np.uint8)
    got = oracle.dense(oracle.pack(a, abits), oracle.pack(w, wbits), m, n, k,
                       abits, wbits, int(bipolar))
    want = a.astype(np.int64) @ weight_values(w, wbits, bipolar).T
    assert np.array_equal(got.astype(np.int64), want)


def eq2_dense(ap, wp, bipolar):
    """Eq. 2 written with numpy popcounts over packed words.
    ap: [m][A][kw], wp: [n][W][kw] uint32."""
    m, A, _ = ap.shape
    n, W, _ = wp.shape
    out = np.zeros((m, n), np.int64)
    for i in range(A):
        for j in range(W):
            x = ap[:, i, None, :]
            y = wp[None, :, j, :]
            term = np.bitwise_count(x & y).sum(axis=2).astype(np.int64)
            if bipolar:
                term -= np.bitwise_count(x & ~y).sum(axis=2).astype(np.int64)
            out += term << (i + j)
    return out


@pytest.mark.parametrize("seed", range(20))
def test_dense_equals_eq2(oracle, seed):
    rng = np.random.default_rng(7000 + seed)
    m, n, k = 5, 6, int(rng.integers(1, 300))
    abits, wbits = int(rng.integers(1, 5)), int(rng.integers(1, 5))
    bipolar = bool(rng.integers(0, 2))
    a = rng.integers(0, 1 << abits, size=(m, k), dtype=np.uint8)
    w = rng.integers(0, 1 << wbits, size=(n, k), dtype=np.uint8)
    ap, wp = oracle.pack(a, abits), oracle.pack(w, wbits)
    got = oracle.dense(ap, wp, m, n, k, abits, wbits, int(bipolar))
    assert np.array_equal(got.astype(np.int64), eq2_dense(ap, wp, bipolar))


@pytest.mark.parametrize("abits", [2, 3, 4])
def test_conv_bitplane_identity(oracle, abits):
    rng = np.random.default_rng(abits)
    n, h, w, c, oc = 2, 7, 6, 45, 5
    a = rng.integers(0, 1 << abits, size=(n, h, w, c), dtype=np.uint8)
    wq = rng.integers(0, 4, size=(oc, 3, 3, c), dtype=np.uint8)
    wp = oracle.pack(wq, 2)
    p = oracle.ConvParams(n, h, w, c, oc, 3, 3, 1, 2, 1, 1, abits, 2, 0, 0)
    full = oracle.conv2d(p, oracle.pack(a, abits), wp).astype(np.int64)
    total = np.zeros_like(full)
    for i in range(abits):
        plane = ((a >> i) & 1).astype(np.uint8)
        p1 = oracle.ConvParams(n, h, w, c, oc, 3, 3, 1, 2, 1, 1, 1, 2, 0, 0)
        total += oracle.conv2d(p1, oracle.pack(plane, 1), wp).astype(
            np.int64) << i
    assert np.array_equal(full, total)


@pytest.mark.parametrize("abits,wbits", [(1, 1), (2, 1), (3, 3), (8, 8)])
def test_conv_all_ones_closed_form(oracle, abits, wbits):
    n, h, w, c, oc = 1, 5, 6, 37, 3
    a = np.full((n, h, w, c), (1 << abits) - 1, np.uint8)
    wq = np.full((oc, 3, 3, c), (1 << wbits) - 1, np.uint8)
    p = oracle.ConvParams(n, h, w, c, oc, 3, 3, 1, 1, 1, 1, abits, wbits,
                          0, 0)
    out = oracle.conv2d(p, oracle.pack(a, abits), oracle.pack(wq, wbits))
    unit = ((1 << abits) - 1) * ((1 << wbits) - 1) * c
    taps = np.full((h, w), 9)
    taps[0, :] = taps[-1, :] = 6
    taps[:, 0] = taps[:, -1] = 6
    taps[0, 0] = taps[0, -1] = taps[-1, 0] = taps[-1, -1] = 4
    for o in range(oc):
        assert np.array_equal(out[0, :, :, o], unit * taps)


@pytest.mark.parametrize("wbits", [1, 2, 3])
def test_conv_bipolar_identity(oracle, wbits):
    rng = np.random.default_rng(40 + wbits)
    n, h, w, c, oc = 2, 6, 7, 70, 4
    a = rng.integers(0, 4, size=(n, h, w, c), dtype=np.uint8)
    wq = rng.integers(0, 1 << wbits, size=(oc, 3, 3, c), dtype=np.uint8)
    ap = oracle.pack(a, 2)

    def run(wbits_, wenc, wcodes):
        p = oracle.ConvParams(n, h, w, c, oc, 3, 3, 2, 1, 1, 1, 2, wbits_, 0,
                              wenc)
        return oracle.conv2d(p, ap, oracle.pack(wcodes, wbits_)).astype(
            np.int64)

    bip = run(wbits, 1, wq)
    uni = run(wbits, 0, wq)
    ones = run(1, 0, np.ones_like(wq))
    assert np.array_equal(bip, 2 * uni - ((1 << wbits) - 1) * ones)


def test_conv_at_matches_full(oracle):
    rng = np.random.default_rng(3)
    n, h, w, c, oc = 2, 9, 8, 33, 7
    a = rng.integers(0, 8, size=(n, h, w, c), dtype=np.uint8)
    wq = rng.integers(0, 2, size=(oc, 3, 3, c), dtype=np.uint8)
    p = oracle.ConvParams(n, h, w, c, oc, 3, 3, 2, 2, 1, 1, 3, 1, 0, 1)
    ap, wp = oracle.pack(a, 3), oracle.pack(wq, 1)
    full = oracle.conv2d(p, ap, wp)
    idx = rng.integers(0, full.size, 300)
    assert np.array_equal(oracle.conv2d_at(p, ap, wp, idx), full.ravel()[idx])


def test_conv_rejects(oracle):
    ok = dict(n=1, h=4, w=4, c=8, oc=2, kh=3, kw=3, stride_h=1, stride_w=1,
              pad_h=1, pad_w=1, abits=2, wbits=1, aenc=0, wenc=0)
    a = np.zeros((1, 4, 4, 2, 1), np.uint32)
    w = np.zeros((2, 3, 3, 1, 1), np.uint32)
    for bad in (dict(abits=0), dict(wbits=9), dict(aenc=3), dict(stride_h=0),
                dict(pad_w=-1), dict(kh=7, pad_h=0), dict(wenc=2),
                dict(aenc=2, abits=1), dict(wenc=-1)):
        p = oracle.ConvParams(**{**ok, **bad})
        with pytest.raises((oracle.OracleError, ValueError)):
            oracle.conv2d(p, a, w)


# --- full-size checks against an independent library routine ---------------

def torch_conv_f64(a, wv, stride, pad):
    """torch CPU conv2d in float64 on integer values: exact, since every
    partial sum is an integer far below 2^53."""
    import torch
    x = torch.from_numpy(a.astype(np.float64)).permute(0, 3, 1, 2)
    k = torch.from_numpy(wv.astype(np.float64)).permute(0, 3, 1, 2)
    y = torch.nn.functional.conv2d(x, k, stride=stride, padding=pad)
    return y.permute(0, 2, 3, 1).numpy().astype(np.int64)


def _case_inputs(oracle, case):
    a = case.activations()
    if case.act_scale is not None:
        a = oracle.quantize(a, case.act_scale, case.abits)
    wq = case.weights()
    if case.weights_from_signs:
        wq = oracle.quantize(wq, 1.0, 1, oracle.BIPOLAR)
    return a, wq


def test_fullsize_config1(oracle):
    case = wl.config1()
    a, wq = _case_inputs(oracle, case)
    p = oracle.conv_params(case.n, case.h, case.w, case.c, case.oc, case.k,
                           case.k, case.stride, case.pad, case.abits,
                           case.wbits, wenc=case.wenc)
    got = oracle.conv2d(p, oracle.pack(a, case.abits),
                        oracle.pack(wq, case.wbits))
    want = torch_conv_f64(a, weight_values(wq, case.wbits, False), 1, 1)
    assert np.array_equal(got.astype(np.int64), want)


@pytest.mark.slow
def test_fullsize_config2_slice(oracle):
    """ResNet-18 layer-2 shape at A2W1: the first 4 images of the batch."""
    case = wl.config2()
    a, wq = _case_inputs(oracle, case)
    a = a[:4]
    p = oracle.conv_params(4, case.h, case.w, case.c, case.oc, case.k,
                           case.k, case.stride, case.pad, case.abits,
                           case.wbits)
    got = oracle.conv2d(p, oracle.pack(a, case.abits),
                        oracle.pack(wq, case.wbits))
    want = torch_conv_f64(a, weight_values(wq, case.wbits, False), 1, 1)
    assert np.array_equal(got.astype(np.int64), want)


@pytest.mark.slow
def test_fullsize_config3_rows(oracle):
    """Dense A2W2 at K = N = 4096, 32 of the 256 activation rows."""
    case = wl.config3()
    a, w = case.activations()[:32], case.weights()
    got = oracle.dense(oracle.pack(a, 2), oracle.pack(w, 2), 32, case.n,
                       case.k, 2, 2)
    want = a.astype(np.float64) @ w.astype(np.float64).T
    assert np.array_equal(got.astype(np.int64), want.astype(np.int64))


@pytest.mark.slow
@pytest.mark.parametrize("case", wl.config4(batch=2) + wl.config5(batch=2),
                         ids=lambda c: c.name)
def test_fullsize_layer_shapes(oracle, case):
    """Every Table 1 layer and the bipolar/A3W3 shapes, at batch 2."""
    a, wq = _case_inputs(oracle, case)
    p = oracle.conv_params(case.n, case.h, case.w, case.c, case.oc, case.k,
                           case.k, case.stride, case.pad, case.abits,
                           case.wbits, wenc=case.wenc)
    got = oracle.conv2d(p, oracle.pack(a, case.abits),
                        oracle.pack(wq, case.wbits))
    want = torch_conv_f64(a, weight_values(wq, case.wbits,
                                           case.wenc == wl.BIPOLAR),
                          case.stride, case.pad)
    assert np.array_equal(got.astype(np.int64), want)


def test_int8_baseline_matches_oracle(oracle):
    # the labelled int8 comparison path (im2col + integer GEMM) computes the
    # same exact integers; checked here with torch's CPU integer GEMM
    import torch
    from paper_1810_11066_amd import int8_baseline as ib
    rng = np.random.default_rng(77)
    for (n, h, w, c, oc, k, s, p, ab, wb) in [(2, 9, 7, 64, 24, 3, 2, 1, 2, 1),
                                              (1, 6, 6, 96, 16, 3, 1, 1, 3, 3),
                                              (1, 5, 8, 64, 8, 1, 1, 0, 4, 2)]:
        a = rng.integers(0, 1 << ab, size=(n, h, w, c), dtype=np.uint8)
        wq = rng.integers(0, 1 << wb, size=(oc, k, k, c), dtype=np.uint8)
        got = ib.conv2d_int8(torch.from_numpy(a), torch.from_numpy(wq), s,
                             p).numpy()
        want = oracle.conv2d(oracle.conv_params(n, h, w, c, oc, k, k, s, p,
                                                ab, wb),
                             oracle.pack(a, ab), oracle.pack(wq, wb))
        assert np.array_equal(got, want)
