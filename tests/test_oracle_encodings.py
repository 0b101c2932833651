"""Pin the oracle's bipolar-activation, signed and packed-layout paths to
things other than itself.

* quantize (signed): numpy's own binary32 multiply, np.rint and clip, then
  the two's complement code of the clamped value; plus a table of ties,
  saturation and specials worked out by hand.
* pack_ex: np.packbits(bitorder='little') after moving the reduction axis
  last, with the bit axis placed by numpy transposes (MBK', MK'B, BMK').
* conv2d / dense with every encoding pair: an int64 brute force on the
  UNPACKED codes, each decoded by a formula other than the oracle's
  (bipolar 2q - (2^B - 1); signed q - 2^B when q >= 2^(B-1)), with zero
  padding of the value tensor.
* the paper's XNOR form for +-1 data (Sec. 2.2): a . w = K - 2 popcount(a XOR w)
  over packed words, both for dense and for the in-range taps of a conv.
* signed data as Eq. 2 with every binary dot product weighted by the sign of
  its planes (Sec. 2.2), written with numpy popcounts.
* closed forms that fix the padding convention of bipolar activations: all
  +1 (or all -1) data against +1 filters gives +-C times the number of
  in-range taps (4 corner, 6 edge, 9 interior at 3x3, pad 1).
"""
import numpy as np
import pytest

from tests.test_oracle_conv_dense import brute_conv


def decode(q, bits, enc):
    q = q.astype(np.int64)
    if enc == 1:                               # bipolar, per plane +-1
        return 2 * q - ((1 << bits) - 1)
    if enc == 2:                               # two's complement
        return np.where(q >= (1 << (bits - 1)), q - (1 << bits), q)
    return q


def numpy_quantize_signed(x, scale, bits):
    lo, hi = -(1 << (bits - 1)), (1 << (bits - 1)) - 1
    with np.errstate(over="ignore", invalid="ignore"):
        r = np.rint(np.float32(x) * np.float32(scale))
        r = np.where(np.isnan(r), 0.0, r)
        v = np.clip(r, lo, hi).astype(np.int64)
    return (v & ((1 << bits) - 1)).astype(np.uint8)


@pytest.mark.parametrize("bits", [2, 3, 4, 8])
@pytest.mark.parametrize("scale", [1.0, 0.5, 1.5, 7.0, 1e38])
def test_quantize_signed_matches_numpy(oracle, bits, scale):
    rng = np.random.default_rng(300 + bits * 7 + int(scale) % 13)
    x = np.concatenate([
        rng.standard_normal(3000).astype(np.float32) * 4,
        (rng.integers(-600, 600, 2000) / 2).astype(np.float32),
        np.array([np.nan, np.inf, -np.inf, -0.0, 0.0, 1e30, -1e30],
                 np.float32)])
    got = oracle.quantize(x, scale, bits, oracle.SIGNED)
    assert np.array_equal(got, numpy_quantize_signed(x, scale, bits))


def test_quantize_signed_table(oracle):
    # 2-bit two's complement: values -2..1, codes 2, 3, 0, 1.
    x = np.array([0.5, 1.5, -0.5, -1.5, -2.5, -3.0, 7.0, np.nan, np.inf,
                  -np.inf, -0.0, -1.0], np.float32)
    want = [0,    1,   0,    2,    2,    2,    1,   0,      1,
            2,       0,    3]
    assert oracle.quantize(x, 1.0, 2, oracle.SIGNED).tolist() == want
    # 4 bits at scale 1.5: -4.5 -> -6.75 -> -7 (code 9); 5.1 -> 7.65 -> 7
    x = np.array([-4.5, 5.1, 1.0 / 3.0], np.float32)
    assert oracle.quantize(x, 1.5, 4, oracle.SIGNED).tolist() == [9, 7, 0]


@pytest.mark.parametrize("args", [dict(bits=1, enc=2), dict(bits=2, enc=3)])
def test_quantize_signed_rejects(oracle, args):
    with pytest.raises(oracle.OracleError):
        oracle.quantize(np.zeros(4, np.float32), 1.0, **args)


def numpy_pack_axis(q, bits, axis, layout):
    """Reference for pack_ex: move the reduction axis last, pack each plane
    with np.packbits, then place the bit axis."""
    q = np.moveaxis(q, axis, -1)
    k = q.shape[-1]
    q = q.reshape(-1, k)
    kw = (k + 31) // 32
    padded = np.zeros((q.shape[0], 32 * kw), np.uint8)
    padded[:, :k] = q
    planes = []
    for b in range(bits):
        by = np.packbits((padded >> b) & 1, axis=1, bitorder="little")
        planes.append(np.ascontiguousarray(by).view("<u4"))
    mbk = np.stack(planes, axis=1)                    # [rows][bits][kw]
    if layout == 0:
        return mbk
    if layout == 1:
        return np.ascontiguousarray(mbk.transpose(0, 2, 1))
    return np.ascontiguousarray(mbk.transpose(1, 0, 2))


@pytest.mark.parametrize("layout", [0, 1, 2])
@pytest.mark.parametrize("shape,axis", [((5, 70), 1), ((2, 37, 3, 4), 1),
                                        ((3, 64, 7), 1), ((33, 6), 0),
                                        ((2, 3, 100), 2)])
@pytest.mark.parametrize("bits", [1, 3])
def test_pack_ex_matches_packbits(oracle, layout, shape, axis, bits):
    rng = np.random.default_rng(len(shape) * 10 + axis + layout)
    q = rng.integers(0, 256, size=shape, dtype=np.uint8)
    got = oracle.pack_ex(q, bits, axis=axis, layout=layout)
    assert np.array_equal(got, numpy_pack_axis(q, bits, axis, layout))


def test_pack_ex_nchw_is_nhwc_pack(oracle):
    """NCHW codes packed along C give the packed NHWC tensor (Sec. 3.2
    layouts): pack_ex(x_nchw, axis=1) == pack(x_nhwc)."""
    rng = np.random.default_rng(11)
    x = rng.integers(0, 4, size=(2, 45, 5, 6), dtype=np.uint8)
    got = oracle.pack_ex(x, 2, axis=1)
    want = oracle.pack(np.ascontiguousarray(x.transpose(0, 2, 3, 1)), 2)
    assert np.array_equal(got, want.reshape(got.shape))


ENC_PAIRS = [(ae, we) for ae in (0, 1, 2) for we in (0, 1, 2)]


def _bits_for(rng, enc, hi=5):
    return int(rng.integers(2 if enc == 2 else 1, hi))


@pytest.mark.parametrize("aenc,wenc", ENC_PAIRS)
@pytest.mark.parametrize("seed", range(8))
def test_conv_encodings_bruteforce(oracle, aenc, wenc, seed):
    rng = np.random.default_rng(9000 + 31 * seed + 3 * aenc + wenc)
    n, h, w = int(rng.integers(1, 3)), int(rng.integers(1, 9)), \
        int(rng.integers(1, 9))
    c, oc = int(rng.integers(1, 71)), int(rng.integers(1, 7))
    k = int(rng.choice([1, 3, 5]))
    s, p = int(rng.integers(1, 3)), int(rng.integers(0, 3))
    while h + 2 * p < k or w + 2 * p < k:
        p += 1
    abits = 1 if aenc == 1 and seed % 2 == 0 else _bits_for(rng, aenc)
    wbits = _bits_for(rng, wenc)
    a = rng.integers(0, 1 << abits, size=(n, h, w, c), dtype=np.uint8)
    wq = rng.integers(0, 1 << wbits, size=(oc, k, k, c), dtype=np.uint8)
    prm = oracle.ConvParams(n, h, w, c, oc, k, k, s, s, p, p, abits, wbits,
                            aenc, wenc)
    got = oracle.conv2d(prm, oracle.pack(a, abits), oracle.pack(wq, wbits))
    want = brute_conv(decode(a, abits, aenc), decode(wq, wbits, wenc),
                      s, s, p, p)
    assert np.array_equal(got.astype(np.int64), want)


@pytest.mark.parametrize("aenc,wenc", ENC_PAIRS)
def test_dense_encodings_bruteforce(oracle, aenc, wenc):
    rng = np.random.default_rng(600 + 3 * aenc + wenc)
    for _ in range(4):
        m, n, k = (int(rng.integers(1, 12)), int(rng.integers(1, 12)),
                   int(rng.integers(1, 150)))
        abits, wbits = _bits_for(rng, aenc, 9), _bits_for(rng, wenc, 9)
        a = rng.integers(0, 1 << abits, size=(m, k), dtype=np.uint8)
        w = rng.integers(0, 1 << wbits, size=(n, k), dtype=np.uint8)
        got = oracle.dense(oracle.pack(a, abits), oracle.pack(w, wbits), m, n,
                           k, abits, wbits, wenc, aenc)
        want = decode(a, abits, aenc) @ decode(w, wbits, wenc).T
        assert np.array_equal(got.astype(np.int64), want)


def test_dense_xnor_closed_form(oracle):
    """+-1 vectors (Sec. 2.2): x . y = K - 2 popcount(x XOR y)."""
    rng = np.random.default_rng(17)
    for k in (1, 31, 32, 33, 100, 4096):
        a = rng.integers(0, 2, size=(6, k), dtype=np.uint8)
        w = rng.integers(0, 2, size=(5, k), dtype=np.uint8)
        ap, wp = oracle.pack(a, 1)[:, 0], oracle.pack(w, 1)[:, 0]
        ham = np.bitwise_count(ap[:, None, :] ^ wp[None, :, :]).sum(axis=2)
        got = oracle.dense(oracle.pack(a, 1), oracle.pack(w, 1), 6, 5, k, 1,
                           1, oracle.BIPOLAR, oracle.BIPOLAR)
        assert np.array_equal(got.astype(np.int64), k - 2 * ham.astype(np.int64))


def test_conv_xnor_interior(oracle):
    """At pixels whose 3x3 window is in range, a +-1 conv is
    9 C - 2 * (Hamming distance of the packed window and filter)."""
    rng = np.random.default_rng(23)
    n, h, w, c, oc = 2, 7, 8, 70, 3
    a = rng.integers(0, 2, size=(n, h, w, c), dtype=np.uint8)
    wq = rng.integers(0, 2, size=(oc, 3, 3, c), dtype=np.uint8)
    ap, wp = oracle.pack(a, 1), oracle.pack(wq, 1)
    prm = oracle.ConvParams(n, h, w, c, oc, 3, 3, 1, 1, 1, 1, 1, 1, 1, 1)
    out = oracle.conv2d(prm, ap, wp).astype(np.int64)
    for y in range(1, h - 1):
        for x in range(1, w - 1):
            win = ap[:, y - 1:y + 2, x - 1:x + 2, 0, :]       # [n][3][3][kw]
            ham = np.bitwise_count(win[:, None] ^ wp[None, :, :, :, 0, :])
            ham = ham.reshape(n, oc, -1).sum(axis=2).astype(np.int64)
            assert np.array_equal(out[:, y, x, :], 9 * c - 2 * ham)


def signed_eq2_dense(ap, wp, asigned, wsigned):
    """Eq. 2 with each plane pair weighted by the sign of its planes:
    the top plane of a two's complement operand counts -2^(B-1)."""
    m, A, _ = ap.shape
    n, W, _ = wp.shape
    out = np.zeros((m, n), np.int64)
    for i in range(A):
        for j in range(W):
            sign = (-1 if asigned and i == A - 1 else 1) * \
                   (-1 if wsigned and j == W - 1 else 1)
            pc = np.bitwise_count(ap[:, i, None, :] & wp[None, :, j, :])
            out += sign * (pc.sum(axis=2).astype(np.int64) << (i + j))
    return out


@pytest.mark.parametrize("aenc,wenc", [(2, 0), (0, 2), (2, 2)])
def test_dense_signed_eq2(oracle, aenc, wenc):
    rng = np.random.default_rng(40 + aenc + 2 * wenc)
    m, n, k, abits, wbits = 7, 9, 200, 3, 4
    a = rng.integers(0, 1 << abits, size=(m, k), dtype=np.uint8)
    w = rng.integers(0, 1 << wbits, size=(n, k), dtype=np.uint8)
    ap, wp = oracle.pack(a, abits), oracle.pack(w, wbits)
    got = oracle.dense(ap, wp, m, n, k, abits, wbits, wenc, aenc)
    want = signed_eq2_dense(ap, wp, aenc == 2, wenc == 2)
    assert np.array_equal(got.astype(np.int64), want)


@pytest.mark.parametrize("sign", [1, -1])
def test_conv_bipolar_activation_padding(oracle, sign):
    """All +1 (code 1) or all -1 (code 0) activations against +1 filters:
    padded taps contribute nothing, so out = sign * C * (in-range taps)."""
    n, h, w, c, oc = 1, 5, 6, 37, 2
    a = np.full((n, h, w, c), 1 if sign > 0 else 0, np.uint8)
    wq = np.ones((oc, 3, 3, c), np.uint8)
    prm = oracle.ConvParams(n, h, w, c, oc, 3, 3, 1, 1, 1, 1, 1, 1, 1, 1)
    out = oracle.conv2d(prm, oracle.pack(a, 1), oracle.pack(wq, 1))
    taps = np.full((h, w), 9)
    taps[0, :] = taps[-1, :] = 6
    taps[:, 0] = taps[:, -1] = 6
    taps[0, 0] = taps[0, -1] = taps[-1, 0] = taps[-1, -1] = 4
    for o in range(oc):
        assert np.array_equal(out[0, :, :, o], sign * c * taps)


def test_conv_signed_msb_identity(oracle):
    """Two's complement: a_signed = a_code - 2^A * a_top, so the signed conv
    is the unipolar conv of the codes minus 2^A times the conv of the top
    activation plane."""
    rng = np.random.default_rng(5)
    n, h, w, c, oc, A = 2, 6, 5, 50, 4, 3
    a = rng.integers(0, 1 << A, size=(n, h, w, c), dtype=np.uint8)
    wq = rng.integers(0, 4, size=(oc, 3, 3, c), dtype=np.uint8)
    wp = oracle.pack(wq, 2)

    def run(codes, bits, aenc):
        prm = oracle.ConvParams(n, h, w, c, oc, 3, 3, 2, 2, 1, 1, bits, 2,
                                aenc, 0)
        return oracle.conv2d(prm, oracle.pack(codes, bits), wp).astype(
            np.int64)

    top = ((a >> (A - 1)) & 1).astype(np.uint8)
    assert np.array_equal(run(a, A, 2), run(a, A, 0) - (1 << A) * run(top, 1, 0))
