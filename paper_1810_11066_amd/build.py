"""Build libbitserial.so in-tree with hipcc for gfx950.

    python -m paper_1810_11066_amd.build

Every compile unit below is compiled to an object in parallel, then linked
into paper_1810_11066_amd/libbitserial.so.  The kernel instantiation sources
(conv_fast_inst.hip, conv_pix_inst.hip) are compiled once per unit, each with
its own -D selection, so that the specialisations compile in parallel.
Flags:
  --offload-arch=gfx950          MI355X only
  -ffp-contract=off              the quantizer's product must stay a lone
                                 binary32 multiply (no FMA contraction)
  -target-feature -packed-fp32-ops
                                 keep the compiler from emitting packed FP32
                                 instructions
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libbitserial.so")
# the int8 matrix-core comparison baseline: a library of its own
INT8_LIB = os.path.join(HERE, "libint8mfma.so")
INT8_SOURCE = "int8_mfma.hip"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# (source, object name, defines)
UNITS = ([("api.hip", "api", ()), ("quant_pack.hip", "quant_pack", ()),
          ("conv.hip", "conv", ()), ("conv_pix.hip", "conv_pix", ())] +
         [("conv_fast_inst.hip", "conv_fast_a%d" % a, ("BS_A=%d" % a,))
          for a in range(1, 5)] +
         [("conv_pix_inst.hip", "conv_pix_a%d" % a,
           ("BS_PIX_FAMILY=0", "BS_A=%d" % a)) for a in range(1, 5)] +
         [("conv_pix_inst.hip", "conv_pix_s%d" % a,
           ("BS_PIX_FAMILY=1", "BS_A=%d" % a)) for a in range(1, 5)] +
         [("conv_pix_inst.hip", "conv_pix_b", ("BS_PIX_FAMILY=2",))])
# every source file the library is built from (headers included)
SOURCES = sorted({u[0] for u in UNITS} |
                 {"bs_internal.h", "conv_fast.h", "conv_pix.h"})

CFLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-ffp-contract=off", "-Wall",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", CSRC,
]


def _compile(src: str, obj: str, extra=()) -> None:
    cmd = [HIPCC] + CFLAGS + list(extra) + ["-c", os.path.join(CSRC, src),
                                            "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed on %s:\n%s%s" % (src, r.stdout,
                                                          r.stderr))


def _link(objs, out):
    out_tmp = out + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC"] + objs + \
          ["-o", out_tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s%s" % (r.stdout, r.stderr))
    os.replace(out_tmp, out)


def build_int8(verbose: bool = False, out: str = INT8_LIB) -> str:
    """Compile and link the int8 MFMA baseline library; returns its path."""
    with tempfile.TemporaryDirectory(prefix="i8_build_") as tmp:
        obj = os.path.join(tmp, "int8_mfma.o")
        _compile(INT8_SOURCE, obj)
        _link([obj], out)
    if verbose:
        print("built", out)
    return out


def build(verbose: bool = False, out: str = LIB, defines=()) -> str:
    """Compile and link the library (to `out`, with extra -D `defines`);
    returns its path."""
    extra = ["-D" + d for d in defines]
    with tempfile.TemporaryDirectory(prefix="bs_build_") as tmp:
        objs = [os.path.join(tmp, u[1] + ".o") for u in UNITS]
        with cf.ThreadPoolExecutor(max_workers=min(8, len(UNITS))) as ex:
            list(ex.map(lambda a: _compile(
                a[0][0], a[1], extra + ["-D" + d for d in a[0][2]]),
                zip(UNITS, objs)))
        _link(objs, out)
    if verbose:
        print("built", out)
    return out


if __name__ == "__main__":
    build(verbose=True)
    build_int8(verbose=True)
    sys.exit(0)
