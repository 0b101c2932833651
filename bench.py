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
CONV_SOURCES = ["paper_1810_11066_amd/csrc/bs_internal.h",
                "paper_1810_11066_amd/csrc/conv.hip",
                "paper_1810_11066_amd/csrc/conv_fast.h",
                "paper_1810_11066_amd/csrc/conv_pix.h",
                "paper_1810_11066_amd/csrc/conv_pix.hip"]


def popcount_roofline_tops(abits: int, wbits: int) -> float:
    """Effective (2 * A-bit x W-bit MAC) TOPS at the popcount-VALU peak."""
    binary_macs = PEAK_LANE_OPS / 2 * 32        # AND + BCNT per 32 MACs
    return 2 * binary_macs / (abits * wbits) / 1e12


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for rel in CONV_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
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
    gpu = gpu_out_fn(n_img)
    return {
        "value": round(2 * macs * reps / el / 1e9, 3),
        "unit": "GOPS",
        "cores": bsref.threads(),
        "kind": "oracle",
        "sample": "%d x (pack + conv) of the first %d of %d images, %.1f s"
                  % (reps, n_img, case.n, el),
    }, bool(np.array_equal(gpu, ref))


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--batch", type=int, default=64)
    ap.add_argument("--sets", type=int, default=6,
                    help="input/output buffer sets rotated across steps")
    ap.add_argument("--cpu-budget", type=float, default=10.0,
                    help="seconds of oracle time for cpu_baseline (0: skip)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="also run one device copy of this size (for HBM "
                         "counter calibration under rocprofv3 --pmc)")
    args = ap.parse_args()

    if args.gpus != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
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

    case = wl.config2(batch=args.batch)
    spec = bs.Conv2dSpec(case.n, case.h, case.w, case.c, case.oc, case.k,
                         case.k, case.stride, case.pad, case.abits,
                         case.wbits)
    params = spec.params()
    oh, ow = bs.bs_conv2d_out_shape(params)
    rows, k = case.n * case.h * case.w, case.c
    words = bs.words(k)

    a_host = case.activations()
    w_host = case.weights()
    w_packed = bs.pack(torch.from_numpy(w_host).cuda(), case.wbits)
    sets = []
    for i in range(args.sets):
        q = torch.from_numpy(a_host).cuda() if i == 0 else \
            torch.from_numpy(np.roll(a_host, i, axis=0)).cuda()
        packed = torch.empty((case.n, case.h, case.w, case.abits, words),
                             dtype=torch.int32, device="cuda")
        out = torch.empty((case.n, oh, ow, case.oc), dtype=torch.int32,
                          device="cuda")
        sets.append((q, packed, out))
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()

    def step(i, ev=None):
        q, packed, out = sets[i % len(sets)]
        if ev is not None:
            ev[0].record(stream)
        bs.bs_pack(q, packed, rows, k, case.abits, stream)
        if ev is not None:
            ev[1].record(stream)
        bs.bs_conv2d(params, packed, w_packed, out, stream)
        if ev is not None:
            ev[2].record(stream)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # timed region: the steps back to back, bracketed by one pair of events
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    h0 = time.perf_counter()
    t_start.record(stream)
    for i in range(args.steps):
        step(i)
    t_end.record(stream)
    host_ms = (time.perf_counter() - h0) * 1e3 / args.steps
    torch.cuda.synchronize()
    ms_total = t_start.elapsed_time(t_end)
    ms_step = ms_total / args.steps

    # kernel durations: the same steps again with an event pair around each
    # launch (events between launches add gaps, so they stay out of the
    # timed region above)
    step_ev = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(3))
               for _ in range(args.steps)]
    for i in range(args.steps):
        step(i, step_ev[i])
    torch.cuda.synchronize()
    pack_ms = sum(e[0].elapsed_time(e[1]) for e in step_ev) / args.steps
    conv_ms = sum(e[1].elapsed_time(e[2]) for e in step_ev) / args.steps
    # packing moves its codes in (one byte each) and its bit-planes out
    pack_bytes = rows * k + rows * case.abits * words * 4
    macs = case.macs
    value_gops = 2 * macs / (ms_step * 1e-3) / 1e9
    peak = popcount_roofline_tops(case.abits, case.wbits)
    achieved = 2 * macs / (conv_ms * 1e-3) / 1e12

    if args.copy_calibration_mib > 0:
        nbytes = args.copy_calibration_mib << 20
        src = torch.ones(nbytes // 4, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()

    workload = "a2w1_b%d_56x56x64_3x3" % case.n
    result = {
        "metric": "bitserial conv2d effective GOPS (2*MACs/s) + % of "
                  "popcount-VALU roofline",
        "value": round(value_gops, 1),
        "unit": "GOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
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
            "per_step": "bs_pack(activations) + bs_conv2d",
            "buffer_sets": args.sets,
        },
        "roofline": {
            "bound": "alu",
            "achieved": round(achieved, 2),
            "peak": round(peak, 1),
            "unit": "TOPS (effective A2W1 ops, popcount VALU)",
            "frac": round(achieved / peak, 4),
            "traffic": committed_traffic(workload),
            "kernel": bs.bs_conv2d_describe(params),
            "kernel_ms": round(conv_ms, 5),
            "timing": "per-launch HIP events on the launch stream, in a "
                      "second pass over the same steps",
        },
        "host_enqueue_ms_per_step": round(host_ms, 5),
        "pack_roofline": {
            "bound": "hbm",
            "achieved": round(pack_bytes / (pack_ms * 1e-3) / 1e9, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(pack_bytes / (pack_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                          4),
            "bytes": pack_bytes,
            "kernel_ms": round(pack_ms, 5),
        },
    }

    if args.cpu_budget > 0:
        def gpu_slice(n_img):
            q, packed, out = sets[0]
            bs.bs_pack(q, packed, rows, k, case.abits, stream)
            bs.bs_conv2d(params, packed, w_packed, out, stream)
            torch.cuda.synchronize()
            return out[:n_img].cpu().numpy()
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
