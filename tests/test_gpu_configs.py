"""GPU parity at the benchmark workloads' full sizes, through the same library
calls and launch configuration the benchmark times.

Every output element of configs 1-5, the encodings workloads, the one-GPU
share of config 4 and the bit-width sweep (16 workloads of ResNet-18 layer 9
at batch 128, up to A4W4) is compared with the oracle's (the full oracle
conv2d / dense at the workload's size).  In addition, as an extra and not as
the reference, every kernel family is compared with the default kernel on
the whole output.  Packed activations and weights are compared with the
oracle's in full.
"""
import numpy as np
import pytest
import torch

from paper_1810_11066_amd import bitserial as bs
from paper_1810_11066_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU parity tests need the MI355X"
    bs.load_library()
    bs.bs_set_kernel_mode(0)


def say(*a):
    print(*a, flush=True)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def words_np(t):
    return t.cpu().numpy().view(np.uint32)


def prepare(oracle, case: wl.ConvCase):
    """Host inputs, oracle-packed operands, and the GPU-packed operands."""
    x = case.activations()
    wsrc = case.weights()
    if case.act_scale is not None:
        a_codes = oracle.quantize(x, case.act_scale, case.abits, case.aenc)
        a_dev = bs.quantize_pack(dev(x), case.act_scale, case.abits,
                                 case.aenc)
    else:
        a_codes = x
        a_dev = bs.pack(dev(x), case.abits)
    if case.weights_from_signs:
        w_codes = oracle.quantize(wsrc, 1.0, 1, oracle.BIPOLAR)
        w_dev = bs.pack(bs.quantize(dev(wsrc), 1.0, 1, bs.BIPOLAR), 1)
    else:
        w_codes = wsrc
        w_dev = bs.pack(dev(wsrc), case.wbits)
    ap = oracle.pack(a_codes, case.abits)
    wp = oracle.pack(w_codes, case.wbits)
    torch.cuda.synchronize()
    assert np.array_equal(words_np(a_dev).reshape(ap.shape), ap)
    assert np.array_equal(words_np(w_dev).reshape(wp.shape), wp)
    return ap, wp, a_dev, w_dev


def spec_of(case):
    return bs.Conv2dSpec(case.n, case.h, case.w, case.c, case.oc, case.k,
                         case.k, case.stride, case.pad, case.abits,
                         case.wbits, case.wenc, case.aenc)


def oracle_params(oracle, case):
    return oracle.conv_params(case.n, case.h, case.w, case.c, case.oc,
                              case.k, case.k, case.stride, case.pad,
                              case.abits, case.wbits, aenc=case.aenc,
                              wenc=case.wenc)


def run_modes(spec, a_dev, w_dev, modes):
    """The conv's output under each kernel mode (0 default, 1 generic,
    2 channels-on-lanes, 3 pixels-on-lanes)."""
    outs = {}
    for mode in modes:
        bs.bs_set_kernel_mode(mode)
        try:
            outs[mode] = bs.conv2d(spec, a_dev, w_dev)
        finally:
            bs.bs_set_kernel_mode(0)
    torch.cuda.synchronize()
    return outs


def check_full(oracle, case, modes=(0, 2, 3)):
    """Every output element of each kernel mode against the oracle."""
    ap, wp, a_dev, w_dev = prepare(oracle, case)
    want = oracle.conv2d(oracle_params(oracle, case), ap, wp)
    for mode, out in run_modes(spec_of(case), a_dev, w_dev, modes).items():
        assert np.array_equal(out.cpu().numpy(), want), "kernel mode %d" % mode


def check_full_default(oracle, case):
    """The default kernel's whole output against the oracle's; the other
    kernel families against the default kernel on the whole output (an extra
    check between kernels, not the reference)."""
    ap, wp, a_dev, w_dev = prepare(oracle, case)
    outs = run_modes(spec_of(case), a_dev, w_dev, (0, 1, 2, 3))
    got = outs[0].cpu().numpy()
    want = oracle.conv2d(oracle_params(oracle, case), ap, wp)
    bad = np.flatnonzero(got.ravel() != want.ravel())
    assert bad.size == 0, "%d outputs differ from the oracle, first at %d" % (
        bad.size, bad[0])
    for mode in (1, 2, 3):
        assert torch.equal(outs[mode], outs[0]), "kernel mode %d" % mode


def test_config1_a1w1(oracle):
    case = wl.config1()
    say(case.name)
    check_full(oracle, case)


def test_config2_a2w1(oracle):
    case = wl.config2()
    say(case.name)
    check_full(oracle, case)


def test_config3_dense(oracle):
    case = wl.config3()
    say(case.name)
    a, w = case.activations(), case.weights()
    a_dev = bs.pack(dev(a), case.abits)
    w_dev = bs.pack(dev(w), case.wbits)
    ap, wp = oracle.pack(a, case.abits), oracle.pack(w, case.wbits)
    got = bs.dense(a_dev, w_dev, case.m, case.n, case.k, case.abits,
                   case.wbits).cpu().numpy()
    assert np.array_equal(words_np(a_dev).reshape(ap.shape), ap)
    assert np.array_equal(words_np(w_dev).reshape(wp.shape), wp)
    want = oracle.dense(ap, wp, case.m, case.n, case.k, case.abits,
                        case.wbits)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("case", wl.config4(), ids=lambda c: c.name)
def test_config4_resnet18_layer(oracle, case):
    say(case.name)
    check_full_default(oracle, case)


@pytest.mark.parametrize("case", wl.config4(batch=16), ids=lambda c: c.name)
def test_config4_one_gpu_share(oracle, case):
    """Config 4 at batch 16, one GPU's share of the batch-128 run sharded
    over 8 GPUs by images: the planner lays out the smaller grid."""
    say(case.name)
    check_full_default(oracle, case)


@pytest.mark.parametrize("case", wl.config5(), ids=lambda c: c.name)
def test_config5_bipolar_a3w3(oracle, case):
    say(case.name)
    check_full_default(oracle, case)


@pytest.mark.parametrize("case", wl.encodings(), ids=lambda c: c.name)
def test_encodings_xnor_signed(oracle, case):
    say(case.name)
    check_full_default(oracle, case)


@pytest.mark.parametrize("case", wl.bitwidth_sweep(), ids=lambda c: c.name)
def test_bitwidth_sweep_layer9(oracle, case):
    say(case.name)
    check_full_default(oracle, case)


def test_resnet18_chain_batch2(oracle):
    # the 16 chained 3x3 convs (bs_conv2d_requant between layers, the three
    # downsampling ones paired with their 1x1 shortcuts) on two images,
    # against the oracle's conv -> quantize(float32) -> pack per layer
    batch, abits, wbits = 2, 2, 1
    layers = wl.resnet18_chain(abits, wbits)
    x = wl.normal_floats((batch, 56, 56, 64), wl.seed_for(7))
    cur_dev = bs.quantize_pack(dev(x), 1.0, abits)
    cur = oracle.pack(oracle.quantize(x, 1.0, abits), abits)
    torch.cuda.synchronize()
    assert np.array_equal(words_np(cur_dev).reshape(cur.shape), cur)
    for L in layers:
        say("chain", L.name)
        wq = L.weights(wbits)
        w_dev = bs.pack(dev(wq), wbits)
        spec = bs.Conv2dSpec(batch, L.h, L.w, L.c, L.oc, L.k, L.k, L.stride,
                             L.pad, abits, wbits)
        conv = oracle.conv2d(oracle.conv_params(batch, L.h, L.w, L.c, L.oc,
                                                L.k, L.k, L.stride, L.pad,
                                                abits, wbits),
                             cur, oracle.pack(wq, wbits))
        if L.out_scale is None:
            got = bs.conv2d(spec, cur_dev, w_dev).cpu().numpy()
            assert np.array_equal(got, conv)
        elif L.shortcut_scale is not None:
            # the downsampling layer and its 1x1 shortcut in one pass
            w1 = L.shortcut_weights(wbits)
            short = oracle.conv2d(
                oracle.conv_params(batch, L.h, L.w, L.c, L.oc, 1, 1,
                                   L.stride, 0, abits, wbits),
                cur, oracle.pack(w1, wbits))
            want1 = oracle.pack(oracle.quantize(short.astype(np.float32),
                                                L.shortcut_scale, abits),
                                abits)
            cur = oracle.pack(oracle.quantize(conv.astype(np.float32),
                                              L.out_scale, abits), abits)
            cur_dev, sc_dev = bs.conv2d_pair_requant(
                spec, cur_dev, w_dev, bs.pack(dev(w1), wbits), L.out_scale,
                L.shortcut_scale, abits)
            torch.cuda.synchronize()
            assert np.array_equal(words_np(cur_dev).reshape(cur.shape), cur)
            assert np.array_equal(words_np(sc_dev).reshape(want1.shape),
                                  want1)
        else:
            cur = oracle.pack(oracle.quantize(conv.astype(np.float32),
                                              L.out_scale, abits), abits)
            cur_dev = bs.conv2d_requant(spec, cur_dev, w_dev, L.out_scale,
                                        abits)
            torch.cuda.synchronize()
            assert np.array_equal(words_np(cur_dev).reshape(cur.shape), cur)
