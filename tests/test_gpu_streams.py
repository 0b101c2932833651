"""GPU parity of independent calls in flight on two HIP streams at once, as
the benchmark issues its steps: consecutive batches alternate between two
streams, each with its own input and output buffers, with no
synchronisation until all are enqueued.  Every batch's output is compared
with the oracle's, for the fused call (bs_conv2d_codes), for bs_pack +
bs_conv2d, and for the requantizing chain step (bs_conv2d_requant)."""
import numpy as np
import pytest
import torch

from paper_1810_11066_amd import bitserial as bs
from paper_1810_11066_amd import workloads as wl

pytestmark = pytest.mark.gpu

BATCHES = 6
N, H, W, C, OC = 4, 56, 56, 64, 64      # the ResNet-18 layer-2 shape


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU parity tests need the MI355X"
    bs.load_library()
    bs.bs_set_kernel_mode(0)


def inputs():
    acts = [wl.uniform_codes((N, H, W, C), 2, wl.seed_for(90, b))
            for b in range(BATCHES)]
    wts = wl.uniform_codes((OC, 3, 3, C), 1, wl.seed_for(90, 99))
    return acts, wts


def oracle_conv(oracle, a, wts):
    p = oracle.conv_params(N, H, W, C, OC, 3, 3, 1, 1, 2, 1)
    return oracle.conv2d(p, oracle.pack(a, 2), oracle.pack(wts, 1))


@pytest.mark.parametrize("path", ["fused", "pack_conv"])
def test_two_streams_int32(oracle, path):
    acts, wts = inputs()
    spec = bs.Conv2dSpec(N, H, W, C, OC, 3, 3, 1, 1, 2, 1)
    p = spec.params()
    w_dev = bs.pack(torch.from_numpy(wts).cuda(), 1)
    xs = [torch.from_numpy(a).cuda() for a in acts]
    packed = [torch.empty((N * H * W, 2, bs.words(C)), dtype=torch.int32,
                          device="cuda") for _ in acts]
    outs = [torch.full((N, H, W, OC), 0x7FFFFFFF, dtype=torch.int32,
                       device="cuda") for _ in acts]
    torch.cuda.synchronize()
    streams = [torch.cuda.current_stream(), torch.cuda.Stream()]
    start = torch.cuda.Event()
    start.record(streams[0])
    streams[1].wait_event(start)
    for b in range(BATCHES):
        s = streams[b % 2]
        if path == "fused":
            bs.bs_conv2d_codes(p, xs[b], w_dev, outs[b], s)
        else:
            bs.bs_pack(xs[b], packed[b], N * H * W, C, 2, s)
            bs.bs_conv2d(p, packed[b], w_dev, outs[b], s)
    torch.cuda.synchronize()
    for b in range(BATCHES):
        want = oracle_conv(oracle, acts[b], wts)
        assert np.array_equal(outs[b].cpu().numpy(), want), "batch %d" % b


def test_two_streams_requant(oracle):
    acts, wts = inputs()
    spec = bs.Conv2dSpec(N, H, W, C, OC, 3, 3, 1, 1, 2, 1)
    p = spec.params()
    w_dev = bs.pack(torch.from_numpy(wts).cuda(), 1)
    packed = [bs.pack(torch.from_numpy(a).cuda(), 2) for a in acts]
    scale = 3.0 / 864.0        # twice the mean result (432) to the top code
    outs = [torch.empty((N, H, W, 2, bs.words(OC)), dtype=torch.int32,
                        device="cuda") for _ in acts]
    torch.cuda.synchronize()
    streams = [torch.cuda.current_stream(), torch.cuda.Stream()]
    start = torch.cuda.Event()
    start.record(streams[0])
    streams[1].wait_event(start)
    for b in range(BATCHES):
        bs.bs_conv2d_requant(p, packed[b], w_dev, scale, 2, outs[b],
                             streams[b % 2])
    torch.cuda.synchronize()
    for b in range(BATCHES):
        conv = oracle_conv(oracle, acts[b], wts).astype(np.float32)
        want = oracle.pack(oracle.quantize(conv, scale, 2), 2)
        got = outs[b].cpu().numpy().view(np.uint32).reshape(want.shape)
        assert np.array_equal(got, want), "batch %d" % b
