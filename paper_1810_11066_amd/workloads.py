"""Seeded synthetic workloads for the bitserial operators.

This module only draws inputs: shapes, value ranges and seeds.  It holds none
of the method's arithmetic (no quantization, packing or convolution), so both
the GPU path and the CPU oracle can be fed from it without sharing any of the
computation.  All arrays are host numpy arrays drawn from numpy's PCG64
generator, so the same seed gives the same bytes on every machine.

Shapes follow the paper's workloads: the ResNet-18 conv layers 2-12 of
Table 1 (the first layer is left out there because its input depth is too
small to pack), a square-ish dense layer for the matrix-multiply study
(Sec. 6.2.1) and the W/A naming of Sec. 6.1 (WxAy = x-bit weights, y-bit
activations).  No dataset or trained weights are used: values are uniform over
the code range (or N(0,1) floats where a layer quantizes its own input).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

UNIPOLAR = 0
BIPOLAR = 1
SIGNED = 2

SEED_BASE = 1810 * 100


def seed_for(config: int, sub: int = 0) -> int:
    """Base seed of case ``sub`` of workload ``config``; a case draws its
    activations from this seed and its weights from this seed + 1."""
    return SEED_BASE + 1000 * config + 10 * sub


def uniform_codes(shape, bits: int, seed: int) -> np.ndarray:
    """uint8 values uniform over {0 .. 2^bits - 1}."""
    rng = np.random.default_rng(seed)
    return rng.integers(0, 1 << bits, size=shape, dtype=np.uint8)


def normal_floats(shape, seed: int) -> np.ndarray:
    """float32 values drawn from N(0, 1)."""
    rng = np.random.default_rng(seed)
    return rng.standard_normal(size=shape, dtype=np.float32)


def sign_floats(shape, seed: int) -> np.ndarray:
    """float32 values +1.0 / -1.0 with equal probability (bipolar weights)."""
    rng = np.random.default_rng(seed)
    return np.where(rng.integers(0, 2, size=shape) == 1, 1.0,
                    -1.0).astype(np.float32)


@dataclass
class ConvCase:
    """One conv2d workload: NHWC activations, OHWI filters."""
    name: str
    n: int
    h: int
    w: int
    c: int
    oc: int
    k: int
    stride: int
    pad: int
    abits: int
    wbits: int
    wenc: int = UNIPOLAR
    seed: int = SEED_BASE
    # activations arrive as float32 N(0,1) and are quantized per call with
    # this scale (otherwise they arrive as uint8 codes)
    act_scale: Optional[float] = None
    # bipolar weights arrive as float +-1 and go through the bipolar quantizer
    weights_from_signs: bool = False
    # encoding of the activation codes (quantized with it when act_scale is
    # set); the codes are drawn uniformly over their 2^abits patterns
    aenc: int = UNIPOLAR

    @property
    def oh(self) -> int:
        return (self.h + 2 * self.pad - self.k) // self.stride + 1

    @property
    def ow(self) -> int:
        return (self.w + 2 * self.pad - self.k) // self.stride + 1

    @property
    def macs(self) -> int:
        """Low-precision multiply-accumulates, padded taps included."""
        return self.n * self.oh * self.ow * self.oc * self.k * self.k * self.c

    def activations(self) -> np.ndarray:
        shape = (self.n, self.h, self.w, self.c)
        if self.act_scale is not None:
            return normal_floats(shape, self.seed + 0)
        return uniform_codes(shape, self.abits, self.seed + 0)

    def weights(self) -> np.ndarray:
        shape = (self.oc, self.k, self.k, self.c)
        if self.weights_from_signs:
            return sign_floats(shape, self.seed + 1)
        return uniform_codes(shape, self.wbits, self.seed + 1)


@dataclass
class DenseCase:
    name: str
    m: int
    n: int
    k: int
    abits: int
    wbits: int
    wenc: int = UNIPOLAR
    seed: int = SEED_BASE

    @property
    def macs(self) -> int:
        return self.m * self.n * self.k

    def activations(self) -> np.ndarray:
        return uniform_codes((self.m, self.k), self.abits, self.seed + 0)

    def weights(self) -> np.ndarray:
        return uniform_codes((self.n, self.k), self.wbits, self.seed + 1)


# ResNet-18 conv layers 2-12 (Table 1): (layer, H=W, IC, OC, K, S)
RESNET18_TABLE1 = [
    (2, 56, 64, 64, 3, 1),
    (3, 56, 64, 64, 1, 1),
    (4, 56, 64, 128, 3, 2),
    (5, 56, 64, 128, 1, 2),
    (6, 28, 128, 128, 3, 1),
    (7, 28, 128, 256, 3, 2),
    (8, 28, 128, 256, 1, 2),
    (9, 14, 256, 256, 3, 1),
    (10, 14, 256, 512, 3, 2),
    (11, 14, 256, 512, 1, 2),
    (12, 7, 512, 512, 3, 1),
]


def config1() -> ConvCase:
    """A1W1 unipolar, 1x14x14x64 -> 64 filters 3x3, stride 1, pad 1."""
    return ConvCase("a1w1_1x14x14x64_3x3", 1, 14, 14, 64, 64, 3, 1, 1, 1, 1,
                    seed=seed_for(1))


def config2(batch: int = 64) -> ConvCase:
    """ResNet-18 layer-2 shape, A2W1 unipolar, 3x3 stride 1 pad 1."""
    return ConvCase("a2w1_%dx56x56x64_3x3" % batch, batch, 56, 56, 64, 64, 3,
                    1, 1, 2, 1, seed=seed_for(2))


def config3() -> DenseCase:
    """Dense A2W2 unipolar: 256x4096 activations, 4096x4096 weights."""
    return DenseCase("dense_a2w2_256x4096x4096", 256, 4096, 4096, 2, 2,
                     seed=seed_for(3))


def config4(batch: int = 128) -> List[ConvCase]:
    """Table 1 layers 2-12 at A2W1, float32 N(0,1) inputs quantized per layer
    with the fixed scale 1.0 + 0.1 (L - 2); pad (K - 1) / 2."""
    cases = []
    for (layer, hw, ic, oc, k, s) in RESNET18_TABLE1:
        cases.append(ConvCase(
            "resnet18_L%d_b%d" % (layer, batch), batch, hw, hw, ic, oc, k, s,
            (k - 1) // 2, 2, 1, seed=seed_for(4, layer),
            act_scale=1.0 + 0.1 * (layer - 2)))
    return cases


def config5(batch: int = 128) -> List[ConvCase]:
    """Bipolar-weight A1W1 and unipolar A3W3 on a 3x3 stride-2 conv
    (128x28x28x128 -> 256) and a 1x1 stride-2 conv (128x14x14x256 -> 512);
    the 1x1 cases are also given at stride 1."""
    out = []
    for sub, (hw, c, oc, k, s, p) in enumerate([
            (28, 128, 256, 3, 2, 1), (14, 256, 512, 1, 2, 0),
            (14, 256, 512, 1, 1, 0)]):
        tag = "%dx%dx%dx%d_%dx%d_s%d" % (batch, hw, hw, c, k, k, s)
        out.append(ConvCase("a1w1bip_" + tag, batch, hw, hw, c, oc, k, s, p,
                            1, 1, wenc=BIPOLAR, seed=seed_for(5, 2 * sub),
                            weights_from_signs=True))
        out.append(ConvCase("a3w3_" + tag, batch, hw, hw, c, oc, k, s, p,
                            3, 3, seed=seed_for(5, 2 * sub + 1)))
    return out


def encodings(batch: int = 128) -> List[ConvCase]:
    """Config 5's shapes (3x3 stride-2 conv 128x28x28x128 -> 256, 1x1 conv
    128x14x14x256 -> 512 at stride 2 and 1) with the other encodings of
    Sec. 2.2: +-1 activations and +-1 weights (the XNOR case; activations
    N(0,1) floats binarized by sign per call, weights float signs), signed
    3-bit activations and weights (N(0,1) activations quantized per call at
    scale 2, weight codes uniform over the 3-bit two's complement range), and
    unipolar 2-bit activations with signed 2-bit weights."""
    out = []
    for sub, (hw, c, oc, k, s, p) in enumerate([
            (28, 128, 256, 3, 2, 1), (14, 256, 512, 1, 2, 0),
            (14, 256, 512, 1, 1, 0)]):
        tag = "%dx%dx%dx%d_%dx%d_s%d" % (batch, hw, hw, c, k, k, s)
        out.append(ConvCase("a1w1xnor_" + tag, batch, hw, hw, c, oc, k, s, p,
                            1, 1, wenc=BIPOLAR, aenc=BIPOLAR,
                            seed=seed_for(7, 3 * sub), act_scale=1.0,
                            weights_from_signs=True))
        out.append(ConvCase("a3w3signed_" + tag, batch, hw, hw, c, oc, k, s,
                            p, 3, 3, wenc=SIGNED, aenc=SIGNED,
                            seed=seed_for(7, 3 * sub + 1), act_scale=2.0))
        out.append(ConvCase("a2uw2s_" + tag, batch, hw, hw, c, oc, k, s, p,
                            2, 2, wenc=SIGNED, aenc=UNIPOLAR,
                            seed=seed_for(7, 3 * sub + 2), act_scale=1.5))
    return out


def bitwidth_sweep(batch: int = 128) -> List[ConvCase]:
    """The limit study of Sec. 6.2.2 on ResNet-18 layer 9 (Table 1: 14x14,
    256 -> 256 channels, 3x3, stride 1, pad 1): every activation width 1..4
    with every unipolar weight width 1..4, codes uniform over their range."""
    out = []
    for abits in range(1, 5):
        for wbits in range(1, 5):
            out.append(ConvCase(
                "resnet18_L9_b%d_A%dW%d" % (batch, abits, wbits), batch, 14,
                14, 256, 256, 3, 1, 1, abits, wbits,
                seed=seed_for(6, 10 * abits + wbits)))
    return out


@dataclass
class ChainLayer:
    """One conv of a chained network: input shape, filters, next-layer
    requantization scale (None for the last layer, which keeps int32).
    A downsampling layer also has its 1x1 projection shortcut (same input,
    stride and output grid), whose requantized output the residual branch
    would take."""
    name: str
    h: int
    w: int
    c: int
    oc: int
    k: int
    stride: int
    pad: int
    seed: int
    out_scale: Optional[float] = None
    shortcut_scale: Optional[float] = None   # set: the layer has a shortcut

    def weights(self, wbits: int) -> np.ndarray:
        return uniform_codes((self.oc, self.k, self.k, self.c), wbits,
                             self.seed + 1)

    def shortcut_weights(self, wbits: int) -> np.ndarray:
        return uniform_codes((self.oc, 1, 1, self.c), wbits, self.seed + 2)


def resnet18_chain(abits: int = 2, wbits: int = 1) -> List[ChainLayer]:
    """The 19 convs of ResNet-18 after conv1: the 16 3x3 convs (Table 1
    layers 2, 4, 6, 7, 9, 10, 12 with their multiplicities 4, 1, 3, 1, 3, 1,
    3), chained, and the 1x1 stride-2 shortcuts (layers 5, 8, 11) on the
    inputs of layers 4, 7 and 10, without the residual adds.  Each output is
    requantized to abits-bit codes with a scale that maps twice the mean
    result of uniform codes, (2^A - 1)/2 * (2^W - 1)/2 * K*K*C, to the top
    code; the last layer keeps its int32 output."""
    stages = [(2, 56, 64, 64, 1, 4), (4, 56, 64, 128, 2, 1),
              (6, 28, 128, 128, 1, 3), (7, 28, 128, 256, 2, 1),
              (9, 14, 256, 256, 1, 3), (10, 14, 256, 512, 2, 1),
              (12, 7, 512, 512, 1, 3)]
    qa, qw = (1 << abits) - 1, (1 << wbits) - 1
    out = []
    for (layer, hw, c, oc, s, reps) in stages:
        for r in range(reps):
            mean = qa / 2 * qw / 2 * 9 * c
            mean1 = qa / 2 * qw / 2 * c
            out.append(ChainLayer("L%d.%d" % (layer, r), hw, hw, c, oc, 3, s,
                                  1, seed_for(7, 10 * len(out)),
                                  qa / (2 * mean),
                                  qa / (2 * mean1) if s == 2 else None))
    out[-1].out_scale = None
    return out
