"""Pin the oracle to hand-worked examples (tests/golden/*.json).

The paper's worked dot product (Fig. 1) is an image that is not available,
so the fixtures were worked out by hand from Eq. 1, Eq. 2 and the bipolar rule
of Sec. 2.2; each fixture names the passage it illustrates.
"""
import json
import os

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


DOT = _load("worked_dot_products.json")["cases"]


@pytest.mark.parametrize("case", DOT, ids=[c["cite"] + " " + str(c["dot"])
                                           for c in DOT])
def test_worked_planes_and_dot(oracle, case):
    x = np.array(case["x"], dtype=np.uint8)
    y = np.array(case["y"], dtype=np.uint8)
    xp = oracle.pack(x[None, :], case["xbits"])[0]
    yp = oracle.pack(y[None, :], case["ybits"])[0]
    # the bit-planes written by hand in the fixture
    assert list(xp[:, 0]) == case["x_planes"]
    assert list(yp[:, 0]) == case["y_planes"]
    enc = oracle.BIPOLAR if case["yenc"] == "bipolar" else oracle.UNIPOLAR
    k = len(case["x"])
    out = oracle.dense(xp, yp, 1, 1, k, case["xbits"], case["ybits"], enc)
    assert out[0, 0] == case["dot"]
    # the same dot product through the conv path: a 1x1 conv over one pixel
    p = oracle.conv_params(1, 1, 1, k, 1, 1, 1, 1, 0, case["xbits"],
                           case["ybits"], wenc=enc)
    assert oracle.conv2d(p, xp, yp)[0, 0, 0, 0] == case["dot"]


CONV = _load("worked_conv2d.json")


@pytest.mark.parametrize("case", CONV["cases"],
                         ids=["s%d_p%d" % (c["stride"], c["pad"])
                              for c in CONV["cases"]])
def test_worked_conv2d(oracle, case):
    x = np.array(CONV["input_2bit"], dtype=np.uint8).reshape(1, 3, 3, 1)
    w = np.array(CONV["weight_1bit"], dtype=np.uint8).reshape(1, 3, 3, 1)
    p = oracle.conv_params(1, 3, 3, 1, 1, 3, 3, case["stride"], case["pad"],
                           2, 1)
    out = oracle.conv2d(p, oracle.pack(x, 2), oracle.pack(w, 1))
    assert out[0, :, :, 0].tolist() == case["out"]


QUANT = _load("quantize_cases.json")["cases"]


def _f32(hexstr):
    return np.array([int(hexstr, 16)], dtype=np.uint32).view(np.float32)[0]


@pytest.mark.parametrize("case", QUANT, ids=[c["dec"] + "/" + c["enc"] +
                                             str(c["bits"]) for c in QUANT])
def test_worked_quantize(oracle, case):
    enc = oracle.BIPOLAR if case["enc"] == "bipolar" else oracle.UNIPOLAR
    q = oracle.quantize(np.array([_f32(case["x"])], dtype=np.float32),
                        _f32(case["scale"]), case["bits"], enc)
    assert int(q[0]) == case["q"]
