"""Pin the oracle's quantizer and bit packer to numpy's own routines.

* quantize: numpy evaluates the reading of Sec. 3.1 with its own IEEE binary32
  multiply and round-half-even (np.rint) -- a separate implementation of the
  same IEEE operations.
* pack: np.packbits(bitorder='little') lays out bit-planes (Sec. 2.2) with
  element u at bit u; viewing its bytes as little-endian uint32 gives the MBK'
  words of Sec. 3.1.
"""
import numpy as np
import pytest


def numpy_quantize(x, scale, bits):
    with np.errstate(over="ignore", invalid="ignore"):
        p = np.float32(x) * np.float32(scale)      # binary32 product
        r = np.rint(p)                              # ties to even
        r = np.where(np.isnan(r), 0.0, r)
        return np.clip(r, 0, (1 << bits) - 1).astype(np.uint8)


def random_floats(rng, n):
    """A mix that exercises rounding ties, saturation, signs, specials."""
    parts = [
        rng.standard_normal(n).astype(np.float32) * 3,
        (rng.integers(-20, 600, n) / 2).astype(np.float32),   # exact halves
        rng.uniform(-1e-38, 1e-38, n).astype(np.float32),     # subnormals
        np.array([np.nan, np.inf, -np.inf, -0.0, 0.0, 1e30, -1e30],
                 dtype=np.float32),
    ]
    return np.concatenate(parts)


@pytest.mark.parametrize("bits", [1, 2, 3, 4, 8])
@pytest.mark.parametrize("scale", [1.0, 0.5, 1.5, 1.3, 7.0, 1e38])
def test_quantize_matches_numpy(oracle, bits, scale):
    rng = np.random.default_rng(bits * 100 + int(scale * 10) % 97)
    x = random_floats(rng, 4000)
    q = oracle.quantize(x, scale, bits)
    assert np.array_equal(q, numpy_quantize(x, scale, bits))


def test_quantize_bipolar_is_sign(oracle):
    rng = np.random.default_rng(5)
    x = random_floats(rng, 3000)
    q = oracle.quantize(x, 1.0, 1, oracle.BIPOLAR)
    with np.errstate(invalid="ignore"):
        expect = (x >= 0).astype(np.uint8)    # NaN compares false -> 0
    assert np.array_equal(q, expect)


@pytest.mark.parametrize("args", [
    dict(scale=0.0, bits=2), dict(scale=-1.0, bits=2),
    dict(scale=float("inf"), bits=2), dict(scale=float("nan"), bits=2),
    dict(scale=1.0, bits=0), dict(scale=1.0, bits=9),
    dict(scale=1.0, bits=2, enc=1)])
def test_quantize_rejects(oracle, args):
    with pytest.raises(oracle.OracleError):
        oracle.quantize(np.zeros(4, np.float32), **args)


def numpy_pack(q, bits):
    rows, k = q.shape
    kw = (k + 31) // 32
    out = np.zeros((rows, bits, kw), dtype=np.uint32)
    padded = np.zeros((rows, kw * 32), dtype=np.uint8)
    padded[:, :k] = q
    for b in range(bits):
        plane = (padded >> b) & 1
        by = np.packbits(plane, axis=1, bitorder="little")   # [rows][kw*4]
        out[:, b, :] = by.view("<u4")
    return out


@pytest.mark.parametrize("k", [1, 5, 31, 32, 33, 64, 70, 100, 128, 257])
@pytest.mark.parametrize("bits", [1, 2, 3, 8])
def test_pack_matches_packbits(oracle, k, bits):
    rng = np.random.default_rng(k * 10 + bits)
    q = rng.integers(0, 256, size=(7, k), dtype=np.uint8)   # high bits too
    assert np.array_equal(oracle.pack(q, bits), numpy_pack(q, bits))


def test_pack_known_word(oracle):
    # elements 0, 1, 4, 6 set -> bits 0, 1, 4, 6 -> 0x53
    q = np.zeros((1, 32), np.uint8)
    q[0, [0, 1, 4, 6]] = 1
    assert oracle.pack(q, 1)[0, 0, 0] == 0x53
    # element 31 is the top bit, element 32 starts the next word
    q = np.zeros((1, 33), np.uint8)
    q[0, 31] = 1
    q[0, 32] = 1
    assert list(oracle.pack(q, 1)[0, 0]) == [0x80000000, 1]


def test_pack_roundtrip_and_popcount(oracle):
    rng = np.random.default_rng(11)
    for bits in (1, 2, 3, 5):
        q = rng.integers(0, 1 << bits, size=(9, 77), dtype=np.uint8)
        pk = oracle.pack(q, bits)
        # unpack by hand: bit u of word t of plane b -> element 32t+u
        back = np.zeros_like(q, dtype=np.int64)
        for b in range(bits):
            for e in range(77):
                back[:, e] |= ((pk[:, b, e // 32] >> (e % 32)) & 1).astype(
                    np.int64) << b
        assert np.array_equal(back, q)
        # popcount of each plane = number of elements with that bit set
        for b in range(bits):
            assert np.array_equal(
                np.bitwise_count(pk[:, b, :]).sum(axis=1),
                ((q >> b) & 1).sum(axis=1))
        # tail bits (past k = 77) are zero
        assert np.all(pk[:, :, 2] >> (77 - 64) == 0)


def test_pack_masks_high_bits(oracle):
    q = np.full((2, 40), 0xFF, np.uint8)
    pk = oracle.pack(q, 2)
    assert np.all(pk[:, :, 0] == 0xFFFFFFFF)
    assert np.all(pk[:, :, 1] == 0xFF)
