#!/usr/bin/env python3
"""Benchmark: bitserial conv2d effective GOPS on one MI355X.

One step = the hot path over one batch: bit-pack the activations
(bs_pack, included as in the paper's timings) and run the bitserial conv2d
(bs_conv2d).  The filters are packed once beforehand (the paper excludes
weight packing from its timings).  Workload: the ResNet-18 layer-2 shape at
batch 64, NHWC 64x56x56x64 codes in {0..3} (2-bit activations), 64 filters
3x3x64 in {0,1} (1-bit weights), stride 1, pad 1, int32 output.

Effective ops = 2 * MACs, MACs = n*oh*ow*oc*kh*kw*c (padded taps counted).
Inputs are resident in HBM before timing starts; several input/output sets
are rotated so the working set exceeds the 256 MB Infinity Cache.

Steps are independent batches, each with its own buffer set.  The warmup
is --warmup steps and at least 0.2 s of them (the GPU's clocks settle only
after tens of ms of load); the timed region runs the steps alternately on
two HIP streams, so that one batch's conv
starts while the previous one drains (a serving loop with two batches in
flight), and then once more on one stream; a line reports the faster of the
two with both beside it.  Kernel durations come from separate passes on one
stream.

Prints ONE JSON line.  Roofline: the conv kernel's live average duration
(HIP events on the launch stream) against the popcount-VALU peak
256 CU x 64 lanes x 2.4 GHz / 2 instructions per 32-bit word pair
x 32 binary MACs per pair / (A*W) x 2 ops per MAC = 629.1 TOPS at A2W1.
cpu_baseline: the CPU oracle, timed on this host on a bounded slice of the
same batch, which it also uses to check the GPU output.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_LANE_OPS = 256 * 64 * 2.4e9           # 32-bit VALU lane-ops / s
HBM_PEAK_GBS = 8000.0
PROFILES = os.path.join(ROOT, "profiles")
# sources of the conv kernels: a committed traffic figure is used only while
# their hash matches the one recorded with it
CONV_SOURCES = ["paper_1810_11066_amd/csrc/" + f for f in (
    "bs_internal.h", "conv.hip", "conv_fast.h", "conv_fast_inst.hip",
    "conv_pix.h", "conv_pix.hip", "conv_pix_inst.hip")]


def popcount_roofline_tops(abits: int, wbits: int) -> float:
    """Effective (2 * A-bit x W-bit MAC) TOPS at the popcount-VALU peak."""
    binary_macs = PEAK_LANE_OPS / 2 * 32        # AND + BCNT per 32 MACs
    return 2 * binary_macs / (abits * wbits) / 1e12


def strip_comments(src: str) -> str:
    """C/C++ source without its comments, whitespace runs collapsed, so that
    the hash below follows the code and not its documentation."""
    out, i, n = [], 0, len(src)
    while i < n:
        c = src[i]
        if c in "\"'":                       # string or character literal
            j = i + 1
            while j < n and src[j] != c:
                j += 2 if src[j] == "\\" else 1
            out.append(src[i:j + 1])
            i = j + 1
        elif src.startswith("//", i):
            j = src.find("\n", i)
            i = n if j < 0 else j
        elif src.startswith("/*", i):
            j = src.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def kernel_source_hash() -> str:
    """Hash of the conv kernel sources' code (comments excluded): a recorded
    counter figure stays valid while only comments change."""
    h = hashlib.sha256()
    for rel in CONV_SOURCES:
        with open(os.path.join(ROOT, rel), encoding="utf-8") as f:
            h.update(strip_comments(f.read()).encode())
            h.update(b"\0")
    return h.hexdigest()[:16]


def committed_traffic(workload: str):
    """HBM bytes per conv launch from the committed rocprofv3 counter summary,
    or None if there is none or the kernel source changed since."""
    path = os.path.join(PROFILES, "conv2d_%s_traffic.md" % workload)
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_src = re.search(r"kernel_source_sha256:\s*([0-9a-f]+)", text)
    m_val = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not m_src or not m_val or m_src.group(1) != kernel_source_hash():
        return None
    return float(m_val.group(1))


def committed_kernel_trace(workload: str, ops: float, peak_tops: float):
    """The conv kernel's average duration in the committed rocprofv3 kernel
    trace of this workload, with the roofline fraction it gives, or None if
    there is none or the kernel source changed since."""
    path = os.path.join(PROFILES, "conv2d_%s_kernel_trace.md" % workload)
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_src = re.search(r"kernel_source_sha256:\s*([0-9a-f]+)", text)
    m_val = re.search(r"conv_kernel_avg_ns:\s*([0-9.eE+]+)", text)
    if not m_src or not m_val or m_src.group(1) != kernel_source_hash():
        return None
    ns = float(m_val.group(1))
    return {"kernel_ms": round(ns * 1e-6, 5),
            "frac": round(ops / (ns * 1e-9) / 1e12 / peak_tops, 4),
            "source": os.path.relpath(path, ROOT)}


def cpu_model() -> str:
    """The host CPU's model name (/proc/cpuinfo), or '' if unknown."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return ""


def oracle_one_thread():
    """The oracle on one host thread, on bounded samples of configs 1-3
    (pack of the activations + conv / dense; about 2 s each)."""
    from oracle import bsref
    from paper_1810_11066_amd import workloads as wl
    out = {}
    bsref.set_threads(1)
    try:
        for name, case in (("config1", wl.config1()), ("config2", wl.config2()),
                           ("config3", wl.config3())):
            if isinstance(case, wl.DenseCase):
                rows = 8
                a = case.activations()[:rows]
                wp = bsref.pack(case.weights(), case.wbits)
                macs = rows * case.n * case.k

                def run():
                    ap = bsref.pack(a, case.abits)
                    bsref.dense(ap, wp, rows, case.n, case.k, case.abits,
                                case.wbits)
                what = "%d of %d rows" % (rows, case.m)
            else:
                n_img = 1
                a = case.activations()[:n_img]
                wp = bsref.pack(case.weights(), case.wbits)
                p = bsref.conv_params(n_img, case.h, case.w, case.c, case.oc,
                                      case.k, case.k, case.stride, case.pad,
                                      case.abits, case.wbits)
                macs = n_img * case.oh * case.ow * case.oc * case.k ** 2 * \
                    case.c

                def run():
                    bsref.conv2d(p, bsref.pack(a, case.abits), wp)
                what = "%d of %d images" % (n_img, case.n)
            reps, t0 = 0, time.perf_counter()
            while True:
                run()
                reps += 1
                el = time.perf_counter() - t0
                if el >= 2.0:
                    break
            out[name] = {"value": round(2 * macs * reps / el / 1e9, 4),
                         "unit": "GOPS",
                         "sample": "%d x (pack + %s) of %s, %.1f s" % (
                             reps, "dense" if "rows" in what else "conv",
                             what, el)}
    finally:
        bsref.set_threads(os.cpu_count() or 1)
    return out


def cpu_baseline(case, a_host, w_host, gpu_out_fn, budget_s: float):
    """Time the oracle (pack + conv) on the first images of the batch until
    `budget_s` of wall time is spent; check the GPU output on that slice."""
    import numpy as np
    from oracle import bsref
    bsref.build(force=False)
    n_img = min(case.n, 8)
    a = a_host[:n_img]
    p = bsref.conv_params(n_img, case.h, case.w, case.c, case.oc, case.k,
                          case.k, case.stride, case.pad, case.abits,
                          case.wbits)
    reps, t0 = 0, time.perf_counter()
    while True:
        ap = bsref.pack(a, case.abits)
        wp = bsref.pack(w_host, case.wbits)
        ref = bsref.conv2d(p, ap, wp)
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    macs = n_img * case.oh * case.ow * case.oc * case.k * case.k * case.c
    cores = bsref.threads()
    gpu = gpu_out_fn(n_img)
    return {
        "value": round(2 * macs * reps / el / 1e9, 3),
        "unit": "GOPS",
        "cores": cores,
        "kind": "oracle",
        "sample": "%d x (pack + conv) of the first %d of %d images, %.1f s"
                  % (reps, n_img, case.n, el),
        "cpu_model": cpu_model(),
        "one_thread": oracle_one_thread(),
    }, all(bool(np.array_equal(g, ref)) for g in gpu)


class Measured:
    """Times of one workload: the clean step (steps spread over the bench's
    streams, and on one stream), and per-launch kernel times."""

    main_tput_ms = None   # main kernel alone, launches spread over streams

    def __init__(self, ms_by_streams, host_ms, pre_ms, main_ms, describe,
                 pre_b2b_ms, pre_ev_ms, main_ev_ms):
        # the step as timed with each stream count; the faster one counts
        self.ms_by_streams = ms_by_streams
        self.n_streams = min(ms_by_streams, key=ms_by_streams.get)
        self.ms_step = ms_by_streams[self.n_streams]
        self.host_ms = host_ms
        self.pre_ms = pre_ms          # activation (quantize +) pack kernel
        self.pre_b2b_ms = pre_b2b_ms  # the same, back-to-back launches
        self.main_ms = main_ms        # conv / dense kernel
        self.pre_ev_ms = pre_ev_ms    # event pairs recorded around launches
        self.main_ev_ms = main_ev_ms
        self.describe = describe


# how the description of a fused step's kernel starts
FUSED_CODES = "activation codes bit-packed into LDS: "
FUSED_FLOAT = "float32 activations quantized and bit-packed into LDS: "


def is_fused(describe: str) -> bool:
    return describe.startswith((FUSED_CODES, FUSED_FLOAT))


def prepare(case, n_sets, bs, torch, np, fused=False):
    """Device buffers for `n_sets` rotated steps of a conv or dense case, and
    the per-step launch function.  Inputs are the workload's seeded host
    arrays (rolled along the batch axis for sets beyond the first); weights
    are packed once, outside the timed steps.

    fused: the step is one call that bit-packs the activations inside the
    conv kernel -- uint8 codes (bs_conv2d_codes) instead of bs_pack followed
    by bs_conv2d, or float32 values quantized per call (bs_conv2d_quantized,
    1x1 windows) instead of bs_quantize_pack followed by bs_conv2d; None is
    returned when the fused kernels do not cover the case (dense, other
    shapes)."""
    from paper_1810_11066_amd import workloads as wl
    main_stream = torch.cuda.current_stream()
    dense = isinstance(case, wl.DenseCase)
    if fused and dense:
        return None
    if dense:
        rows, k, abits = case.m, case.k, case.abits
    else:
        rows, k, abits = case.n * case.h * case.w, case.c, case.abits
    words = bs.words(k)
    x_host = case.activations()
    wsrc = case.weights()
    if not dense and case.weights_from_signs:
        w_packed = bs.pack(bs.quantize(torch.from_numpy(wsrc).cuda(), 1.0, 1,
                                       bs.BIPOLAR), 1)
    else:
        w_packed = bs.pack(torch.from_numpy(wsrc).cuda(), case.wbits)
    if dense:
        out_shape = (case.m, case.n)
        params = None
    else:
        params = bs.Conv2dSpec(case.n, case.h, case.w, case.c, case.oc,
                               case.k, case.k, case.stride, case.pad,
                               case.abits, case.wbits, case.wenc,
                               case.aenc).params()
        oh, ow = bs.bs_conv2d_out_shape(params)
        out_shape = (case.n, oh, ow, case.oc)
    quantized = (not dense) and case.act_scale is not None
    sets = []
    for i in range(n_sets):
        xi = x_host if i == 0 else np.roll(x_host, i, axis=0)
        x = torch.from_numpy(np.ascontiguousarray(xi)).cuda()
        packed = torch.empty((rows, abits, words), dtype=torch.int32,
                             device="cuda")
        out = torch.empty(out_shape, dtype=torch.int32, device="cuda")
        sets.append((x, packed, out))
    torch.cuda.synchronize()

    def pack_launch(x, packed, stream):
        if quantized:
            bs.bs_quantize_pack(x, packed, rows, k, case.act_scale, abits,
                                case.aenc, stream)
        else:
            bs.bs_pack(x, packed, rows, k, abits, stream)

    def main_launch(x, packed, out, stream):
        if dense:
            bs.bs_dense(case.m, case.n, case.k, case.abits, case.wbits,
                        bs.UNIPOLAR, packed, w_packed, out, stream)
        elif fused and quantized:
            bs.bs_conv2d_quantized(params, x, case.act_scale, w_packed, out,
                                   stream)
        elif fused:
            bs.bs_conv2d_codes(params, x, w_packed, out, stream)
        else:
            bs.bs_conv2d(params, packed, w_packed, out, stream)

    def step(i, ev=None, pack_only=False, dispatch_ev=None, stream=None,
             main_only=False):
        """One step on set i, on `stream` (default: the current stream at
        preparation).  ev: three events recorded around the launches;
        dispatch_ev: two (start, stop) pairs the library attaches to the pack
        and the conv dispatch themselves.  pack_only: the standalone
        activation pack alone (also for a fused step, as a reference);
        main_only: the conv (or dense) launch alone, on the set's packed
        activations of an earlier step."""
        stream = main_stream if stream is None else stream
        x, packed, out = sets[i % len(sets)]
        if pack_only:
            pack_launch(x, packed, stream)
            return
        if main_only:
            main_launch(x, packed, out, stream)
            return
        if ev is not None:
            ev[0].record(stream)
        if not fused:
            if dispatch_ev is not None:
                bs.bs_set_timing_events(*dispatch_ev[0])
            pack_launch(x, packed, stream)
        if ev is not None:
            ev[1].record(stream)
        if dispatch_ev is not None:
            bs.bs_set_timing_events(*dispatch_ev[1])
        main_launch(x, packed, out, stream)
        if dispatch_ev is not None:
            bs.bs_set_timing_events(None, None)
        if ev is not None:
            ev[2].record(stream)

    step.fused = fused
    step.n_sets = n_sets
    if fused:
        try:
            step(0)
        except bs.BitserialError as e:
            if e.status == bs.BS_ERR_UNSUPPORTED:
                return None
            raise
    if dense:
        describe = bs.bs_conv2d_describe(bs.Conv2dSpec(
            1, 1, case.m, case.k, case.n, 1, 1, 1, 0, case.abits,
            case.wbits).params())
    elif fused and quantized:
        describe = FUSED_FLOAT + bs.bs_conv2d_quantized_describe(params)
    elif fused:
        describe = FUSED_CODES + bs.bs_conv2d_codes_describe(params)
    else:
        describe = bs.bs_conv2d_describe(params)
    # initialisation: one step per set writes every packed and output buffer
    # once, so that no buffer is first written inside a timed region
    for i in range(n_sets):
        step(i)
        if fused:
            step(i, pack_only=True)
    torch.cuda.synchronize()
    return sets, step, params, w_packed, describe, quantized


def stream_of(j, steps, n_streams):
    """Stream index of step j of `steps` timed steps: consecutive steps
    alternate, and the first one runs on stream 0, right behind the start
    event (a first launch on another stream sits behind a wait for that
    event and starts several us later)."""
    return j % n_streams


def check_sets_streams(n_sets, n_streams):
    """Steps i and j share a buffer set when i = j mod n_sets; with n_sets a
    multiple of n_streams they then share a stream as well, so no two steps
    that write the same buffers ever run concurrently.  n_sets = 0: the
    steps write only fresh buffers."""
    if n_streams > 1 and n_sets % n_streams:
        raise ValueError("buffer sets (%d) must be a multiple of the streams "
                         "(%d)" % (n_sets, n_streams))


def timed_steps(step, first, steps, torch, streams):
    """Wall time per step of `steps` steps from index `first`, bracketed by
    device synchronisations and one event pair on streams[0].  Step j runs
    on streams[stream_of(j, ...)], so consecutive steps (independent
    batches with buffers of their own) alternate streams and the first one
    follows the start event on streams[0]; each other stream waits for the
    start event just before its first step, and streams[0] waits for the
    other streams' last steps before the stop event.
    Returns (ms per step, host enqueue ms per step)."""
    main = streams[0]
    ns = len(streams)
    check_sets_streams(getattr(step, "n_sets", 0), ns)
    torch.cuda.synchronize()
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    h0 = time.perf_counter()
    t_start.record(main)
    for j in range(steps):
        k = stream_of(j, steps, ns)
        if j == k and k > 0:
            streams[k].wait_event(t_start)
        step(first + j, stream=streams[k])
    for s in streams[1:min(ns, steps)]:
        done = torch.cuda.Event()
        done.record(s)
        main.wait_event(done)
    t_end.record(main)
    host_ms = (time.perf_counter() - h0) * 1e3 / steps
    torch.cuda.synchronize()
    return t_start.elapsed_time(t_end) / steps, host_ms


N_STREAMS = 2
# the GPU's clocks settle only after tens of ms of sustained load: a config-2
# step timed right after an idle period runs up to 20 % slower than one timed
# after 30 ms of work, so the warmup runs at least this long
WARMUP_MIN_S = 0.2


def warm_up(step, warmup, torch, streams, chunk=32):
    """At least `warmup` steps, and more until the GPU has been busy for
    WARMUP_MIN_S of wall time, spread over the streams as timed steps are
    (step i on streams[i % len]); ends with a device synchronisation.
    Returns the number of steps issued (the next step index)."""
    ns = len(streams)
    check_sets_streams(getattr(step, "n_sets", 0), ns)
    t0 = time.perf_counter()
    i = 0
    while i < warmup or time.perf_counter() - t0 < WARMUP_MIN_S:
        for _ in range(chunk):
            step(i, stream=streams[i % ns])
            i += 1
        torch.cuda.synchronize()
    return i


_STREAMS = []


def make_streams(torch, n):
    """Streams for timed steps: the current stream when n is 1, else n
    streams of the default priority created once per process and reused.
    The runtime spreads streams over a few hardware queues (4 by default)
    as they are created, so streams made afresh for every measurement would
    sooner or later share one queue and run one after the other."""
    if n == 1:
        return [torch.cuda.current_stream()]
    while len(_STREAMS) < n:
        _STREAMS.append(torch.cuda.Stream())
    return _STREAMS[:n]


def measure(step, describe, steps, warmup, torch):
    """Clean timed regions: the steps spread over N_STREAMS streams, then
    the same steps on one stream (the step counts at the faster of the two;
    both are reported), then the main kernel alone spread over the streams.
    Then the same steps again with dispatch-stamped events on each launch
    for kernel times and once more with event pairs around each launch,
    then the activation pack launches alone, back to back under one event
    pair.  The kernel-time passes run on one stream.

    Each timed region is bracketed by device synchronisations: it starts on
    an idle GPU after the warmup steps have finished, so it includes the
    host's enqueue of its first launch."""
    streams = make_streams(torch, N_STREAMS)
    stream = torch.cuda.current_stream()     # the single-stream passes
    first = warm_up(step, warmup, torch, streams)
    by = {}
    if N_STREAMS > 1:
        by[N_STREAMS], host_ms = timed_steps(step, first, steps, torch,
                                             streams)
    by[1], host_one = timed_steps(step, first, steps, torch,
                                  make_streams(torch, 1))
    if N_STREAMS == 1:
        host_ms = host_one
    main_tput_ms = None
    if N_STREAMS > 1:
        # the main kernel alone with its launches spread over the streams:
        # its throughput once the launches' fixed costs overlap (the
        # activation pack of a fused step is inside this kernel).  Timed
        # before the passes below: the memory-bound pack launches leave
        # the GPU at clocks that slow the next compute-bound pass.
        def main_only(i, stream=None):
            step(i, stream=stream, main_only=True)
        main_only.n_sets = getattr(step, "n_sets", 0)
        main_tput_ms = timed_steps(main_only, first, steps, torch,
                                   streams)[0]
    # kernel durations: events the runtime stamps with each dispatch's own
    # start and end (the library launches through hipExtLaunchKernel while
    # they are set), the figure a kernel trace reports
    def mk():
        return torch.cuda.Event(enable_timing=True)
    dev = [((mk(), mk()), (mk(), mk())) for _ in range(steps)]
    for i in range(steps):
        step(i, dispatch_ev=dev[i])
    torch.cuda.synchronize()
    pre_ms = None if step.fused else \
        sum(d[0][0].elapsed_time(d[0][1]) for d in dev) / steps
    main_ms = sum(d[1][0].elapsed_time(d[1][1]) for d in dev) / steps
    # for comparison: event pairs recorded on the stream around each launch
    # (they also count part of each launch's overhead)
    ev = [tuple(mk() for _ in range(3)) for _ in range(steps)]
    for i in range(steps):
        step(i, ev[i])
    torch.cuda.synchronize()
    pre_ev_ms = None if step.fused else \
        sum(e[0].elapsed_time(e[1]) for e in ev) / steps
    main_ev_ms = sum(e[1].elapsed_time(e[2]) for e in ev) / steps
    p_start = torch.cuda.Event(enable_timing=True)
    p_end = torch.cuda.Event(enable_timing=True)
    p_start.record(stream)
    for i in range(steps):
        step(i, pack_only=True)
    p_end.record(stream)
    torch.cuda.synchronize()
    pre_b2b_ms = p_start.elapsed_time(p_end) / steps
    m = Measured(by, host_ms, pre_ms, main_ms, describe, pre_b2b_ms,
                 pre_ev_ms, main_ev_ms)
    m.main_tput_ms = main_tput_ms
    return m


def throughput_of(m, t_roof_s):
    """The main kernel alone, launches spread over the streams: ms per
    launch and its fraction of the roofline (None on one stream)."""
    if m.main_tput_ms is None:
        return None
    return {"streams": N_STREAMS, "ms_per_launch": round(m.main_tput_ms, 5),
            "frac": round(t_roof_s / (m.main_tput_ms * 1e-3), 4)}


def by_streams(m):
    """{streams: ms per step} of a measured workload, for the JSON line."""
    return {str(k): round(v, 5) for k, v in sorted(m.ms_by_streams.items())}


def pack_roofline(nbytes, m):
    """The standalone activation (quantize +) pack kernel against the HBM
    peak, timed by dispatch-stamped events (back-to-back launches when the
    step is fused and has no pack launch of its own); the other timings
    beside it."""
    if m.pre_ms is not None:
        ms, how = m.pre_ms, "dispatch-stamped events (hipExtLaunchKernel) " \
            "on each pack launch"
    else:
        ms, how = m.pre_b2b_ms, "back-to-back standalone pack launches " \
            "under one event pair (not part of the fused step)"
    gbs = nbytes / (ms * 1e-3) / 1e9
    out = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS,
           "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
           "bytes": nbytes, "kernel_ms": round(ms, 5), "timing": how,
           "kernel_ms_back_to_back": round(m.pre_b2b_ms, 5)}
    if m.pre_ev_ms is not None:
        out["kernel_ms_events_around_launch"] = round(m.pre_ev_ms, 5)
    return out


def case_bytes(case, fused=False):
    """Algorithmic HBM bytes of (activation pack, main kernel); fused: the
    main kernel reads the unpacked activations instead of packed ones.  The
    pack handles every input pixel; the main kernel reads the pixels its
    windows touch: all of them, except for 1x1 windows at stride 2 (one per
    output pixel)."""
    from paper_1810_11066_amd import workloads as wl
    if isinstance(case, wl.DenseCase):
        rows, k, out = case.m, case.k, case.m * case.n * 4
        read = rows
        wbytes = case.n * case.wbits * ((case.k + 31) // 32) * 4
    else:
        rows, k = case.n * case.h * case.w, case.c
        out = case.n * case.oh * case.ow * case.oc * 4
        read = case.n * case.oh * case.ow if case.k == 1 and \
            case.stride > 1 else rows
        wbytes = case.oc * case.k * case.k * case.wbits * \
            ((case.c + 31) // 32) * 4
    per_packed = case.abits * ((k + 31) // 32) * 4
    per_src = k * (4 if getattr(case, "act_scale", None) else 1)
    return (rows * (per_src + per_packed),
            read * (per_src if fused else per_packed) + wbytes + out)


def sets_for(case, minimum: int) -> int:
    """Rotated buffer sets for a case: at least `minimum`, and enough that
    the sets together pass 512 MB (twice the 256 MB Infinity Cache), so
    timed steps read their inputs from HBM; at most 256 (tiny workloads stay
    cache-resident whatever the count)."""
    from paper_1810_11066_amd import workloads as wl
    if isinstance(case, wl.DenseCase):
        out = case.m * case.n * 4
    else:
        out = case.n * case.oh * case.ow * case.oc * 4
    pre_bytes, _ = case_bytes(case)
    per_set = pre_bytes + out
    need = -(-512 * 10**6 // per_set)
    n = max(minimum, min(256, need))
    return -(-n // N_STREAMS) * N_STREAMS     # a multiple of the streams


ENC_NAMES = ("unipolar", "bipolar", "signed")


def roofline_of(case, m, ops, main_bytes):
    """Roofline object of the step's main (conv / dense) kernel."""
    peak = popcount_roofline_tops(case.abits, case.wbits)
    t_alu = ops / (peak * 1e12)
    t_hbm = main_bytes / (HBM_PEAK_GBS * 1e9)
    bound = "alu" if t_alu >= t_hbm else "hbm"
    main_s = m.main_ms * 1e-3
    roof = {"bound": bound, "kernel": m.describe,
            "kernel_ms": round(m.main_ms, 5),
            "timing": "dispatch-stamped events (hipExtLaunchKernel) on each "
                      "launch",
            "kernel_ms_events_around_launch": round(m.main_ev_ms, 5)}
    if bound == "alu":
        roof.update(achieved=round(ops / main_s / 1e12, 2),
                    peak=round(peak, 1), unit="TOPS (effective ops, "
                    "popcount VALU)", frac=round(t_alu / main_s, 4))
    else:
        roof.update(achieved=round(main_bytes / main_s / 1e9, 1),
                    peak=HBM_PEAK_GBS, unit="GB/s (algorithmic bytes)",
                    frac=round(t_hbm / main_s, 4))
    roof["throughput_streams"] = throughput_of(m, t_alu if bound == "alu"
                                               else t_hbm)
    return roof


def per_step_name(case, fused):
    from paper_1810_11066_amd import workloads as wl
    q = getattr(case, "act_scale", None) is not None
    if fused and q:
        return ("bs_conv2d_quantized (quantize and bit-pack of the float32 "
                "activations inside the conv kernel)")
    if fused:
        return ("bs_conv2d_codes (bit-pack of the uint8 activation codes "
                "inside the conv kernel)")
    return ("bs_quantize_pack" if q else "bs_pack") + "(activations) + " + \
        ("bs_dense" if isinstance(case, wl.DenseCase) else "bs_conv2d")


def case_line(case, m, args, other=None):
    """One JSON result object for a workload other than the headline one.
    m: the step reported (the faster of the fused call and pack + conv
    where both cover the case); other: the other path's step, reported
    beside it under "fused" or "unfused"."""
    ops = 2 * case.macs
    fused = is_fused(m.describe)
    pre_bytes, main_bytes = case_bytes(case, fused=fused)
    line = {
        "metric": "bitserial conv2d effective GOPS (2*MACs/s) + % of "
                  "popcount-VALU roofline",
        "value": round(ops / (m.ms_step * 1e-3) / 1e9, 1),
        "unit": "GOPS", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "warmup_min_s": WARMUP_MIN_S,
        "ms_per_step": round(m.ms_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "u32", "data": "synthetic",
        "config": {"workload": case.name,
                   "per_step": per_step_name(case, fused),
                   "streams": m.n_streams,
                   "abits": case.abits, "wbits": case.wbits,
                   "encoding": ENC_NAMES[getattr(case, "wenc", 0)],
                   "act_encoding": ENC_NAMES[getattr(case, "aenc", 0)]},
        "roofline": roofline_of(case, m, ops, main_bytes),
        "pack_roofline": pack_roofline(pre_bytes, m),
        "host_enqueue_ms_per_step": round(m.host_ms, 5),
        "ms_per_step_by_streams": by_streams(m),
    }
    if other is not None and other is not m:
        ofused = is_fused(other.describe)
        _, obytes = case_bytes(case, fused=ofused)
        line["fused" if ofused else "unfused"] = {
            "per_step": per_step_name(case, ofused),
            "ms_per_step": round(other.ms_step, 5),
            "ms_per_step_by_streams": by_streams(other),
            "value": round(ops / (other.ms_step * 1e-3) / 1e9, 1),
            "roofline": roofline_of(case, other, ops, obytes)}
    return line


def pairs_lines(args, bs, torch, np, wl) -> int:
    """ResNet-18's downsampling pairs (Table 1 layers 4/5, 7/8, 10/11) at
    batch 128, A2W1: one step quantizes and packs the float32 input, then
    runs the 3x3 stride-2 conv and its 1x1 stride-2 shortcut -- as one paired
    launch (bs_conv2d_pair) and, for comparison, as two bs_conv2d launches.
    One line per pair, with the step and kernel times of both."""
    layers = {c.name: c for c in wl.config4(batch=args.batch or 128)}
    main_stream = torch.cuda.current_stream()
    for main, short in ((4, 5), (7, 8), (10, 11)):
        c3 = layers["resnet18_L%d_b%d" % (main, args.batch or 128)]
        c1 = layers["resnet18_L%d_b%d" % (short, args.batch or 128)]
        rows = c3.n * c3.h * c3.w
        spec3 = bs.Conv2dSpec(c3.n, c3.h, c3.w, c3.c, c3.oc, 3, 3, c3.stride,
                              1, c3.abits, c3.wbits).params()
        spec1 = bs.Conv2dSpec(c1.n, c1.h, c1.w, c1.c, c1.oc, 1, 1, c1.stride,
                              0, c1.abits, c1.wbits).params()
        oh, ow = bs.bs_conv2d_out_shape(spec3)
        w3 = bs.pack(torch.from_numpy(c3.weights()).cuda(), c3.wbits)
        w1 = bs.pack(torch.from_numpy(c1.weights()).cuda(), c1.wbits)
        x_host = c3.activations()
        per_set = x_host.nbytes + 2 * c3.n * oh * ow * c3.oc * 4
        n_sets = max(args.sets, min(64, -(-512 * 10**6 // per_set)))
        n_sets = -(-n_sets // N_STREAMS) * N_STREAMS
        sets = []
        for i in range(n_sets):
            xi = x_host if i == 0 else np.roll(x_host, i, axis=0)
            sets.append((torch.from_numpy(np.ascontiguousarray(xi)).cuda(),
                         torch.empty((rows, c3.abits, bs.words(c3.c)),
                                     dtype=torch.int32, device="cuda"),
                         torch.empty((c3.n, oh, ow, c3.oc), dtype=torch.int32,
                                     device="cuda"),
                         torch.empty((c3.n, oh, ow, c3.oc), dtype=torch.int32,
                                     device="cuda")))

        def mk_step(paired):
            def step(i, ev=None, pack_only=False, dispatch_ev=None,
                     stream=None, main_only=False):
                stream = main_stream if stream is None else stream
                x, packed, o3, o1 = sets[i % n_sets]
                if not pack_only and dispatch_ev is not None:
                    bs.bs_set_timing_events(*dispatch_ev[0])
                if not main_only:
                    bs.bs_quantize_pack(x, packed, rows, c3.c, c3.act_scale,
                                        c3.abits, bs.UNIPOLAR, stream)
                if pack_only:
                    return
                if ev is not None:
                    ev[0].record(stream)
                    ev[1].record(stream)
                if dispatch_ev is not None:
                    bs.bs_set_timing_events(*dispatch_ev[1])
                if paired:
                    bs.bs_conv2d_pair(spec3, packed, w3, w1, o3, o1, stream)
                else:
                    # one pair of dispatch events over both launches: start
                    # stamped by the first, stop by the last
                    bs.bs_conv2d(spec3, packed, w3, o3, stream)
                    bs.bs_conv2d(spec1, packed, w1, o1, stream)
                if dispatch_ev is not None:
                    bs.bs_set_timing_events(None, None)
                if ev is not None:
                    ev[2].record(stream)
            step.fused = False
            step.n_sets = n_sets
            return step

        res = {}
        for paired in (True, False):
            step = mk_step(paired)
            for i in range(n_sets):
                step(i)
            torch.cuda.synchronize()
            res[paired] = measure(step, "", args.steps, args.warmup, torch)
        macs = c3.macs + c1.macs
        mp, ms = res[True], res[False]
        print(json.dumps({
            "pairs": "resnet18 L%d (3x3 s2) + L%d (1x1 s2 shortcut), batch "
                     "%d, A2W1, float32 input quantized + packed per step"
                     % (main, short, c3.n),
            "paired_kernel": bs.bs_conv2d_describe(spec3).split(" patch=")[0]
                             + " with the centre-tap 1x1 conv (bs_conv2d_pair;"
                             " runs of 4 units where oc % 16 == 0; 8 words "
                             "per plane run as two launches)",
            "paired_ms_per_step": round(mp.ms_step, 5),
            "separate_ms_per_step": round(ms.ms_step, 5),
            "paired_ms_per_step_by_streams": by_streams(mp),
            "separate_ms_per_step_by_streams": by_streams(ms),
            "paired_conv_ms": round(mp.main_ms, 5),
            "separate_convs_ms": round(ms.main_ms, 5),
            "paired_conv_ms_streams": round(mp.main_tput_ms, 5)
            if mp.main_tput_ms is not None else None,
            "separate_convs_ms_streams": round(ms.main_tput_ms, 5)
            if ms.main_tput_ms is not None else None,
            "quantize_pack_ms": round(mp.pre_ms, 5),
            "paired_step_effective_tops": round(
                2 * macs / (mp.ms_step * 1e-3) / 1e12, 1),
            "separate_step_effective_tops": round(
                2 * macs / (ms.ms_step * 1e-3) / 1e12, 1),
        }), flush=True)
        del sets
        torch.cuda.empty_cache()
    return 0


INT8_MFMA_PEAK_TOPS = 5000.0   # dense int8 MFMA, MI355X


def chain_line(args, bs, torch, np, wl, batch=128, abits=2, wbits=1) -> int:
    """ResNet-18's conv path chained on the GPU: the float32 input is
    quantized and packed once, every 3x3 conv but the last writes the next
    layer's packed codes (bs_conv2d_requant), the three downsampling layers
    with their 1x1 shortcuts in one paired launch (bs_conv2d_pair_requant,
    the shortcut's packed codes for the residual branch), the last writes
    int32.  Consecutive passes are independent batches: each stream has a
    buffer set of its own and passes alternate streams, as steps do."""
    layers = wl.resnet18_chain(abits, wbits)
    x_host = wl.normal_floats((batch, 56, 56, 64), wl.seed_for(7))
    specs, wts, wts1 = [], [], []
    for L in layers:
        spec = bs.Conv2dSpec(batch, L.h, L.w, L.c, L.oc, L.k, L.k, L.stride,
                             L.pad, abits, wbits)
        specs.append(spec.params())
        wts.append(bs.pack(torch.from_numpy(L.weights(wbits)).cuda(), wbits))
        wts1.append(bs.pack(torch.from_numpy(
            L.shortcut_weights(wbits)).cuda(), wbits)
            if L.shortcut_scale is not None else None)

    def buffers(i):
        """Input, packed input and per-layer outputs of buffer set i."""
        xi = x_host if i == 0 else np.roll(x_host, i, axis=0)
        x = torch.from_numpy(np.ascontiguousarray(xi)).cuda()
        packed_in = torch.empty((batch * 56 * 56, abits, bs.words(64)),
                                dtype=torch.int32, device="cuda")
        outs, outs1 = [], []
        for L, p in zip(layers, specs):
            oh, ow = bs.bs_conv2d_out_shape(p)
            if L.out_scale is None:
                outs.append(torch.empty((batch, oh, ow, L.oc),
                                        dtype=torch.int32, device="cuda"))
            else:
                outs.append(torch.empty((batch, oh, ow, abits,
                                         bs.words(L.oc)),
                                        dtype=torch.int32, device="cuda"))
            outs1.append(torch.empty_like(outs[-1])
                         if L.shortcut_scale is not None else None)
        return x, packed_in, outs, outs1

    sets = [buffers(i) for i in range(N_STREAMS)]
    main_stream = torch.cuda.current_stream()
    macs = sum(batch * ((L.h + 2 * L.pad - L.k) // L.stride + 1) ** 2 *
               L.oc * (L.k * L.k + (1 if L.shortcut_scale else 0)) * L.c
               for L in layers)

    def run(i, ev=None, stream=None, **_):
        stream = main_stream if stream is None else stream
        x, packed_in, outs, outs1 = sets[i % len(sets)]
        bs.bs_quantize_pack(x, packed_in, batch * 56 * 56, 64, 1.0, abits,
                            bs.UNIPOLAR, stream)
        src = packed_in
        for k, L in enumerate(layers):
            if ev is not None:
                ev[k][0].record(stream)
            if L.out_scale is None:
                bs.bs_conv2d(specs[k], src, wts[k], outs[k], stream)
            elif L.shortcut_scale is not None:
                bs.bs_conv2d_pair_requant(specs[k], src, wts[k], wts1[k],
                                          L.out_scale, L.shortcut_scale,
                                          abits, outs[k], outs1[k], stream)
            else:
                bs.bs_conv2d_requant(specs[k], src, wts[k], L.out_scale,
                                     abits, outs[k], stream)
            if ev is not None:
                ev[k][1].record(stream)
            src = outs[k]
    run.n_sets = len(sets)

    streams = make_streams(torch, N_STREAMS)
    first = warm_up(run, args.warmup, torch, streams, chunk=4)
    by = {1: timed_steps(run, first, args.steps, torch,
                         make_streams(torch, 1))[0]}
    if len(streams) > 1:
        by[len(streams)] = timed_steps(run, first, args.steps, torch,
                                       streams)[0]
    n_best = min(by, key=by.get)
    ms = by[n_best]
    ev = [[(torch.cuda.Event(enable_timing=True),
            torch.cuda.Event(enable_timing=True)) for _ in layers]
          for _ in range(args.steps)]
    for r in range(args.steps):
        run(r, ev[r])
    torch.cuda.synchronize()
    per = [sum(ev[r][k][0].elapsed_time(ev[r][k][1])
               for r in range(args.steps)) / args.steps
           for k in range(len(layers))]
    print(json.dumps({
        "chain": "resnet18 convs after conv1 (16 3x3 chained by "
                 "bs_conv2d_requant, the 3 downsampling ones paired with "
                 "their 1x1 shortcuts by bs_conv2d_pair_requant), batch %d, "
                 "A%dW%d, no residual adds" % (batch, abits, wbits),
        "layers": len(layers),
        "shortcuts": sum(1 for L in layers if L.shortcut_scale is not None),
        "streams": n_best,
        "ms_per_pass": round(ms, 4),
        "effective_tops": round(2 * macs / (ms * 1e-3) / 1e12, 1),
        "frac_of_roofline": round(2 * macs / (ms * 1e-3) / 1e12 /
                                  popcount_roofline_tops(abits, wbits), 4),
        "ms_per_pass_by_streams": {str(k): round(v, 4)
                                   for k, v in sorted(by.items())},
        "layer_ms": {L.name: round(t, 4) for L, t in zip(layers, per)},
    }))
    return 0


def int8_baseline_lines(args, bs, torch, np, wl) -> int:
    """The int8 matrix-core comparison (baselines, not the bitserial path):
    config 2 through the hand-written implicit-GEMM MFMA conv and through
    im2col + the library int8 GEMM, config 3 through one library GEMM, each
    next to the bitserial step and checked equal to the bitserial result
    (both are checked against the oracle by the GPU tests)."""
    from paper_1810_11066_amd import int8_baseline as ib

    def per_launch(fn, n_sets):
        """ms per launch: back-to-back launches over n_sets rotated buffer
        sets after warmup, spread over the streams as the bitserial steps
        are (timed_steps).  n_sets = 0: fn writes only fresh outputs."""
        streams = make_streams(torch, N_STREAMS)

        def step(i, stream=None):
            with torch.cuda.stream(stream or streams[0]):
                fn(i)
        step.n_sets = n_sets
        first = warm_up(step, max(args.warmup, n_sets), torch, streams)
        return timed_steps(step, first, args.steps, torch, streams)[0]

    ok_all = True
    for case in (wl.config2(), wl.config3()):
        dense = isinstance(case, wl.DenseCase)
        n_sets = sets_for(case, args.sets)
        fz = prepare(case, n_sets, bs, torch, np, fused=True)
        sets, step, params, w_packed, describe, _ = prepare(case, n_sets, bs,
                                                            torch, np)
        m = measure(step, describe, args.steps, args.warmup, torch)
        mf = (measure(fz[1], fz[4], args.steps, args.warmup, torch)
              if fz is not None else None)
        ops = 2 * case.macs
        line = {"baseline": ib.LABEL, "workload": case.name,
                "bitserial_kernel_ms": round(m.main_ms, 5),
                "bitserial_step_ms": round(m.ms_step, 5),
                "bitserial_fused_step_ms": round(mf.ms_step, 5)
                if mf is not None else None}
        if dense:
            a8 = torch.from_numpy(case.activations()).cuda()
            w8 = torch.from_numpy(case.weights()).cuda()
            wt = w8.to(torch.int8).t().contiguous()
            a8 = a8.to(torch.int8)
            gemm_ms = per_launch(lambda i: torch._int_mm(a8, wt), 0)
            ref = torch._int_mm(a8, wt)
            line.update(int8_gemm=ib.LABEL_GEMM,
                        int8_gemm_ms=round(gemm_ms, 5),
                        int8_gemm_tops=round(ops / (gemm_ms * 1e-3) / 1e12, 1),
                        int8_gemm_frac_of_mfma_peak=round(
                            ops / (gemm_ms * 1e-3) / 1e12 /
                            INT8_MFMA_PEAK_TOPS, 4))
        else:
            x8s = [s_[0].to(torch.int8) for s_ in sets]
            w8 = torch.from_numpy(case.weights()).cuda().to(torch.int8)
            outs = [torch.empty_like(s_[2]) for s_ in sets]
            mfma_ms = per_launch(lambda i: ib.conv2d_mfma(
                x8s[i % n_sets], w8, case.stride, case.pad,
                out=outs[i % n_sets]), n_sets)
            ref = ib.conv2d_mfma(x8s[0], w8, case.stride, case.pad)
            in_b = case.n * case.h * case.w * case.c
            out_b = case.n * case.oh * case.ow * case.oc * 4
            w_b = case.oc * case.k * case.k * case.c
            hbm = (in_b + out_b + w_b) / (mfma_ms * 1e-3) / 1e9
            cols = ib.im2col_nhwc(x8s[0], case.k, case.stride,
                                  case.pad).contiguous()
            wt = w8.reshape(case.oc, -1).t().contiguous()
            gemm_ms = per_launch(lambda i: torch._int_mm(cols, wt), 0)
            im2col_ms = per_launch(lambda i: ib.im2col_nhwc(
                x8s[i % n_sets], case.k, case.stride, case.pad).contiguous(),
                n_sets)
            line.update(
                int8_conv=ib.LABEL_CONV,
                int8_conv_ms=round(mfma_ms, 5),
                int8_conv_tops=round(ops / (mfma_ms * 1e-3) / 1e12, 1),
                int8_conv_frac_of_mfma_peak=round(
                    ops / (mfma_ms * 1e-3) / 1e12 / INT8_MFMA_PEAK_TOPS, 4),
                int8_conv_hbm_gbs=round(hbm, 1),
                int8_conv_frac_of_hbm=round(hbm / HBM_PEAK_GBS, 4),
                int8_conv_over_bitserial_step=round(
                    mfma_ms / (mf.ms_step if mf is not None else m.ms_step),
                    3),
                int8_gemm=ib.LABEL_GEMM,
                int8_gemm_ms=round(gemm_ms, 5),
                int8_im2col_ms=round(im2col_ms, 5),
                int8_gemm_tops=round(ops / (gemm_ms * 1e-3) / 1e12, 1))
        step(0)
        torch.cuda.synchronize()
        same = bool(torch.equal(ref.reshape(-1), sets[0][2].reshape(-1)))
        ok_all &= same
        line["outputs_equal_bitserial"] = same
        print(json.dumps(line), flush=True)
        del sets, fz
        torch.cuda.empty_cache()
    return 0 if ok_all else 1


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--batch", type=int, default=None,
                    help="images per call: config 2 (default 64) and "
                         "configs 4, 5 and --encodings (default 128); "
                         "config 4 at 16 is one GPU's share of a batch-128 "
                         "run sharded over 8")
    ap.add_argument("--sets", type=int, default=6,
                    help="at least this many input/output buffer sets "
                         "rotated across steps (more where needed to pass "
                         "512 MB in all)")
    ap.add_argument("--cpu-budget", type=float, default=10.0,
                    help="seconds of oracle time for cpu_baseline (0: skip)")
    ap.add_argument("--path", choices=["both", "fused", "unfused"],
                    default="both",
                    help="which steps to time: the fused call that bit-packs "
                         "the activation codes inside the conv kernel "
                         "(bs_conv2d_codes, where it covers the workload), "
                         "the two-kernel step (bs_pack or bs_quantize_pack, "
                         "then bs_conv2d), or both (default; the line's "
                         "value is the fused step where there is one)")
    ap.add_argument("--streams", type=int, default=2, choices=[1, 2, 3, 4],
                    help="HIP streams the timed steps alternate over (the "
                         "line reports the faster of this many and one); 1 "
                         "for profiling runs, whose kernel traces then give "
                         "per-launch durations of kernels that never "
                         "overlap")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="also run one device copy of this size (for HBM "
                         "counter calibration under rocprofv3 --pmc)")
    ap.add_argument("--config", type=int, default=2, choices=[1, 2, 3, 4, 5],
                    help="workload: 2 (default) is the headline ResNet-18 "
                         "layer-2 A2W1 line; 1, 3, 4, 5 print one line per "
                         "case of that workload")
    ap.add_argument("--int8-baseline", action="store_true",
                    help="time the labelled int8 matrix-core baselines "
                         "(hand-written implicit-GEMM MFMA conv; im2col + "
                         "library int8 GEMM; library GEMM for dense) on "
                         "configs 2 and 3 next to the bitserial steps, "
                         "checking equal outputs")
    ap.add_argument("--chain", action="store_true",
                    help="the 16 3x3 convs of ResNet-18 (batch 128, A2W1) "
                         "chained with bs_conv2d_requant: quantize+pack of "
                         "the float input, 15 requantizing convs, one int32 "
                         "conv; one line with the total and per-layer times")
    ap.add_argument("--pairs", action="store_true",
                    help="ResNet-18's downsampling pairs (layers 4/5, 7/8, "
                         "10/11, batch 128): the 3x3 stride-2 conv and its "
                         "1x1 shortcut as one paired launch against two "
                         "launches; one line per pair")
    ap.add_argument("--encodings", action="store_true",
                    help="config 5's shapes with +-1 activations and weights "
                         "(XNOR), signed A3W3, and unipolar A2 x signed W2: "
                         "one line per case")
    ap.add_argument("--sweep", action="store_true",
                    help="bit-width sweep A1-4 x W1-4 on ResNet-18 layer 9 "
                         "(batch 128): one line per pair, then a summary "
                         "line with the time ratios the paper reports")
    args = ap.parse_args()

    global N_STREAMS
    N_STREAMS = args.streams
    if args.gpus != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr)
        return 2

    import numpy as np
    import torch
    from paper_1810_11066_amd import bitserial as bs
    from paper_1810_11066_amd import workloads as wl

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    torch.cuda.set_device(0)
    bs.load_library()

    if args.copy_calibration_mib > 0:
        # one device copy of known size: the reference that scales the HBM
        # counters of a rocprofv3 --pmc pass over this run
        nbytes = args.copy_calibration_mib << 20
        src = torch.ones(nbytes // 4, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    if args.int8_baseline:
        return int8_baseline_lines(args, bs, torch, np, wl)
    if args.chain:
        return chain_line(args, bs, torch, np, wl)
    if args.pairs:
        return pairs_lines(args, bs, torch, np, wl)

    if args.sweep or args.encodings or args.config != 2:
        b = {} if args.batch is None else {"batch": args.batch}
        if args.sweep:
            cases = wl.bitwidth_sweep()
        elif args.encodings:
            cases = wl.encodings(**b)
        else:
            cases = {1: lambda: [wl.config1()], 3: lambda: [wl.config3()],
                     4: lambda: wl.config4(**b),
                     5: lambda: wl.config5(**b)}[args.config]()
        times = {}
        for case in cases:
            n_sets = sets_for(case, args.sets)
            mu = mf = None
            if args.path != "fused":
                sets, step, _, _, describe, _ = prepare(case, n_sets, bs,
                                                        torch, np)
                mu = measure(step, describe, args.steps, args.warmup, torch)
                times[(case.abits, case.wbits)] = mu.main_ms
                del sets, step
                torch.cuda.empty_cache()
            fz = None if args.path == "unfused" else prepare(
                case, n_sets, bs, torch, np, fused=True)
            if fz is not None:
                mf = measure(fz[1], fz[4], args.steps, args.warmup, torch)
                del fz
                torch.cuda.empty_cache()
            if mf is not None and mu is not None:
                # the faster path first, the other beside it
                first, second = (mf, mu) if mf.ms_step <= mu.ms_step \
                    else (mu, mf)
                print(json.dumps(case_line(case, first, args, second)),
                      flush=True)
            elif mf is not None or mu is not None:
                print(json.dumps(case_line(case, mf or mu, args)),
                      flush=True)
        if args.sweep and len(times) == 16:
            # the paper's limit study quotes W1A1 against W4A4 and W2A2
            # against W1A4 (activation width A, weight width W)
            print(json.dumps({
                "sweep": "resnet18_L9_b128 conv kernel time ratios",
                "A4W4_over_A1W1": round(times[(4, 4)] / times[(1, 1)], 2),
                "A4W1_over_A2W2": round(times[(4, 1)] / times[(2, 2)], 3),
                "kernel_ms": {"A%dW%d" % k: round(v, 5)
                              for k, v in sorted(times.items())}}))
        return 0

    case = wl.config2(batch=args.batch or 64)
    n_sets = sets_for(case, args.sets)
    fz = None if args.path == "unfused" else prepare(case, n_sets, bs, torch,
                                                     np, fused=True)
    mf = mu = None
    if fz is not None:
        mf = measure(fz[1], fz[4], args.steps, args.warmup, torch)
    sets = step = None
    if args.path != "fused" or fz is None:
        sets, step, params, w_packed, describe, _ = prepare(case, n_sets, bs,
                                                            torch, np)
        mu = measure(step, describe, args.steps, args.warmup, torch)
    # the faster of the fused call and pack + conv (the fused call where
    # only it ran); the other is reported beside it
    m = mf if mf is not None and (mu is None or mf.ms_step <= mu.ms_step) \
        else mu
    other = (mu if m is mf else mf) if mf is not None and mu is not None \
        else None
    m_fused = m is mf
    macs = case.macs
    value_gops = 2 * macs / (m.ms_step * 1e-3) / 1e9
    peak = popcount_roofline_tops(case.abits, case.wbits)
    pack_bytes, _ = case_bytes(case)

    def conv_roofline(mm, workload):
        achieved = 2 * macs / (mm.main_ms * 1e-3) / 1e12
        return {
            "bound": "alu",
            "achieved": round(achieved, 2),
            "peak": round(peak, 1),
            "unit": "TOPS (effective A2W1 ops, popcount VALU)",
            "frac": round(achieved / peak, 4),
            "traffic": committed_traffic(workload),
            "kernel": mm.describe,
            "kernel_ms": round(mm.main_ms, 5),
            "timing": "dispatch-stamped events (hipExtLaunchKernel) on each "
                      "conv launch, in a second pass over the same steps",
            "kernel_ms_events_around_launch": round(mm.main_ev_ms, 5),
            "kernel_trace": committed_kernel_trace(workload, 2 * macs, peak),
            "throughput_streams": throughput_of(mm, 2 * macs / (peak * 1e12)),
        }

    shape = "a2w1_b%d_56x56x64_3x3" % case.n
    result = {
        "metric": "bitserial conv2d effective GOPS (2*MACs/s) + % of "
                  "popcount-VALU roofline",
        "value": round(value_gops, 1),
        "unit": "GOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "warmup_min_s": WARMUP_MIN_S,
        "ms_per_step": round(m.ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic",
        "config": {
            "workload": "resnet18_layer2_conv3x3_A2W1_pack_plus_conv",
            "batch": case.n, "h": case.h, "w": case.w, "c": case.c,
            "oc": case.oc, "kernel": case.k, "stride": case.stride,
            "pad": case.pad, "abits": case.abits, "wbits": case.wbits,
            "encoding": "unipolar", "output": "int32 NHWC",
            "per_step": per_step_name(case, m_fused),
            "buffer_sets": n_sets,
            "streams": m.n_streams,
        },
        "roofline": conv_roofline(
            m, ("codes_" if m_fused else "") + shape),
        "host_enqueue_ms_per_step": round(m.host_ms, 5),
        "ms_per_step_by_streams": by_streams(m),
        "pack_roofline": pack_roofline(pack_bytes, mu if mu is not None
                                       else m),
    }
    if other is not None:
        result["unfused" if m_fused else "fused"] = {
            "per_step": per_step_name(case, not m_fused),
            "ms_per_step": round(other.ms_step, 5),
            "ms_per_step_by_streams": by_streams(other),
            "value": round(2 * macs / (other.ms_step * 1e-3) / 1e9, 1),
            "roofline": conv_roofline(
                other, ("" if m_fused else "codes_") + shape)}

    if args.cpu_budget > 0:
        a_host = case.activations()
        w_host = case.weights()

        def gpu_slice(n_img):
            """The first images of set 0 from the unfused and (if timed) the
            fused step, stacked; the oracle's slice must equal each."""
            outs = []
            if step is not None:
                step(0)
                outs.append(sets[0][2][:n_img].cpu().numpy())
            if fz is not None:
                fz[1](0)
                outs.append(fz[0][0][2][:n_img].cpu().numpy())
            torch.cuda.synchronize()
            return outs
        cpu, ok = cpu_baseline(case, a_host, w_host, gpu_slice,
                               args.cpu_budget)
        result["cpu_baseline"] = cpu
        result["verified_against_oracle"] = ok
        if not ok:
            print(json.dumps(result))
            print("GPU output differs from the oracle", file=sys.stderr)
            return 1
    print(json.dumps(result))
    return 0


if __name__ == "__main__":
    sys.exit(main())
