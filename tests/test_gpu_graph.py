"""GPU: the hot path captured in a HIP graph (torch.cuda.CUDAGraph) and
replayed.

No entry point allocates device memory, copies, or synchronises: each
enqueues only its kernels on the caller's stream, so a capture holds
exactly those kernels.  The captured graph -- quantize + pack of float32
activations, the conv, the requantizing conv and the next layer's conv on
its packed output, and the fused conv of uint8 codes -- is replayed several
times with new inputs copied into the captured buffers and eager calls of
the same entry points in between (and, quantized inside the kernel, a 1x1
stride-2 conv of the float32 input), and every replay is checked against the
oracle, element by element."""
import numpy as np
import pytest
import torch

from paper_1810_11066_amd import bitserial as bs

pytestmark = pytest.mark.gpu

N, H, W, C, OC, OC2, K = 2, 9, 10, 64, 68, 32, 3
OC3 = 36   # the 1x1 stride-2 conv of the float32 input
OH3, OW3 = (H - 1) // 2 + 1, (W - 1) // 2 + 1
ABITS, WBITS, OBITS = 2, 1, 2
SCALE = 1.3
# spreads the first conv's results over the 2-bit output codes
SCALE2 = 3.0 / (0.5 * K * K * C * 3 + 1)


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU parity tests need the MI355X"
    bs.load_library()
    bs.bs_set_kernel_mode(0)
    bs.bs_set_units_per_wave(0)
    yield


def say(*a):
    print(*a, flush=True)


def inputs(replay):
    rng = np.random.default_rng(4400 + replay)
    x = rng.standard_normal((N, H, W, C), dtype=np.float32)
    codes = rng.integers(0, 256, size=(N, H, W, C), dtype=np.uint8)
    return x, codes


def expected(oracle, x, codes, w1, w2, w3):
    p1 = oracle.conv_params(N, H, W, C, OC, K, K, 1, 1, ABITS, WBITS)
    p3 = oracle.conv_params(N, H, W, C, OC3, 1, 1, 2, 0, ABITS, WBITS)
    p2 = oracle.conv_params(N, H, W, OC, OC2, K, K, 1, 1, OBITS, WBITS)
    wp1, wp2 = oracle.pack(w1, WBITS), oracle.pack(w2, WBITS)
    ap = oracle.pack(oracle.quantize(x, SCALE, ABITS), ABITS)
    conv1 = oracle.conv2d(p1, ap, wp1)
    req = oracle.pack(oracle.quantize(conv1.astype(np.float32), SCALE2,
                                      OBITS), OBITS)
    conv2 = oracle.conv2d(p2, req, wp2)
    convc = oracle.conv2d(p1, oracle.pack(codes, ABITS), wp1)
    conv3 = oracle.conv2d(p3, ap, oracle.pack(w3, WBITS))
    return ap, conv1, req, conv2, convc, conv3


def test_hot_path_in_a_graph(oracle):
    rng = np.random.default_rng(4399)
    w1 = rng.integers(0, 2, size=(OC, K, K, C), dtype=np.uint8)
    w2 = rng.integers(0, 2, size=(OC2, K, K, OC), dtype=np.uint8)
    w3 = rng.integers(0, 2, size=(OC3, 1, 1, C), dtype=np.uint8)
    dev = torch.device("cuda")
    w1_dev = bs.pack(torch.from_numpy(w1).to(dev), WBITS)
    w2_dev = bs.pack(torch.from_numpy(w2).to(dev), WBITS)
    w3_dev = bs.pack(torch.from_numpy(w3).to(dev), WBITS)
    p1 = bs.ConvParams(N, H, W, C, OC, K, K, 1, 1, 1, 1, ABITS, WBITS, 0, 0)
    p2 = bs.ConvParams(N, H, W, OC, OC2, K, K, 1, 1, 1, 1, OBITS, WBITS, 0,
                       0)
    p3 = bs.ConvParams(N, H, W, C, OC3, 1, 1, 2, 2, 0, 0, ABITS, WBITS, 0, 0)
    # every buffer the graph touches exists before the capture
    x_dev = torch.empty((N, H, W, C), dtype=torch.float32, device=dev)
    codes_dev = torch.empty((N, H, W, C), dtype=torch.uint8, device=dev)
    a_dev = torch.empty((N * H * W, ABITS, bs.words(C)), dtype=torch.int32,
                        device=dev)
    out1 = torch.empty((N, H, W, OC), dtype=torch.int32, device=dev)
    req = torch.empty((N, H, W, OBITS, bs.words(OC)), dtype=torch.int32,
                      device=dev)
    out2 = torch.empty((N, H, W, OC2), dtype=torch.int32, device=dev)
    outc = torch.empty((N, H, W, OC), dtype=torch.int32, device=dev)
    out3 = torch.empty((N, OH3, OW3, OC3), dtype=torch.int32, device=dev)

    def path():
        bs.bs_quantize_pack(x_dev, a_dev, N * H * W, C, SCALE, ABITS)
        bs.bs_conv2d(p1, a_dev, w1_dev, out1)
        bs.bs_conv2d_requant(p1, a_dev, w1_dev, SCALE2, OBITS, req)
        bs.bs_conv2d(p2, req, w2_dev, out2)
        bs.bs_conv2d_codes(p1, codes_dev, w1_dev, outc)
        bs.bs_conv2d_quantized(p3, x_dev, SCALE, w3_dev, out3)

    x, codes = inputs(0)
    x_dev.copy_(torch.from_numpy(x))
    codes_dev.copy_(torch.from_numpy(codes))
    # the calls once outside the capture, on a side stream (plans cached,
    # kernels loaded)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        path()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        path()
    torch.cuda.synchronize()

    for replay in range(4):
        x, codes = inputs(replay)
        x_dev.copy_(torch.from_numpy(x))
        codes_dev.copy_(torch.from_numpy(codes))
        # eager calls of the same entry points on other buffers in between
        other = bs.quantize_pack(torch.from_numpy(inputs(99 + replay)[0])
                                 .to(dev), SCALE, ABITS)
        bs.conv2d(bs.Conv2dSpec(N, H, W, C, OC, K, K, 1, 1, ABITS, WBITS),
                  other, w1_dev)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        ap, conv1, rq, conv2, convc, conv3 = expected(oracle, x, codes, w1,
                                                      w2, w3)
        say("replay", replay)
        assert np.array_equal(a_dev.cpu().numpy().view(np.uint32)
                              .reshape(ap.shape), ap)
        assert np.array_equal(out1.cpu().numpy(), conv1)
        assert np.array_equal(req.cpu().numpy().view(np.uint32)
                              .reshape(rq.shape), rq)
        assert np.array_equal(out2.cpu().numpy(), conv2)
        assert np.array_equal(outc.cpu().numpy(), convc)
        assert np.array_equal(out3.cpu().numpy(), conv3)
