"""int8 matrix-core comparison baselines (not part of the bitserial path).

The paper compares its bitserial operators with optimized 8-bit and 16-bit
integer implementations on the same CPU (Sec. 6.2.1, 6.2.2).  The GPU
analogue is an int8 x int8 -> int32 product on the matrix cores (MFMA):

* ``conv2d_mfma``: a hand-written implicit-GEMM conv (libint8mfma.so,
  include/int8_mfma.h): NHWC int8 activations read once per tap straight into
  v_mfma_i32_16x16x64_i8 fragments, OHWI int8 filters staged in LDS, int32
  NHWC output -- no im2col copy;
* ``dense_int8``: the vendor GEMM behind ``torch._int_mm`` (hipBLASLt);
* ``conv2d_int8``: NHWC im2col of the codes followed by that GEMM, kept as
  the library route for comparison.

Codes of up to 7 bits fit int8 unchanged, so the products are exactly the
integer results the bitserial kernels compute; the tests check them against
the oracle.  Nothing here is used by the bitserial library.
"""
from __future__ import annotations

import ctypes
import os
import threading

import torch
import torch.nn.functional as F

LABEL = "int8 MFMA baseline, not bitserial"
LABEL_GEMM = "int8 MFMA baseline (torch._int_mm -> hipBLASLt), not bitserial"
LABEL_CONV = ("int8 MFMA baseline (hand-written implicit-GEMM conv, "
              "v_mfma_i32_16x16x64_i8), not bitserial")

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libint8mfma.so")
_lock = threading.Lock()
_lib = None


class ConvParams(ctypes.Structure):
    """Mirror of ``i8mfma_conv_params``."""
    _fields_ = [(f, ctypes.c_int32) for f in (
        "n", "h", "w", "c", "oc", "kh", "kw", "stride", "pad")]


def load_library():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError("libint8mfma.so is not built (%s); run "
                                   "`python -m paper_1810_11066_amd.build`"
                                   % LIB_PATH)
            lib = ctypes.CDLL(LIB_PATH)
            P = ctypes.c_void_p
            lib.i8mfma_conv2d.argtypes = [ctypes.POINTER(ConvParams), P, P, P,
                                          P]
            lib.i8mfma_conv2d.restype = ctypes.c_int
            lib.i8mfma_last_error.restype = ctypes.c_char_p
            _lib = lib
        return _lib


def conv2d_mfma(x: torch.Tensor, w: torch.Tensor, stride: int, pad: int,
                out: torch.Tensor = None, stream=None) -> torch.Tensor:
    """NHWC int8 x [N][H][W][C], OHWI int8 w [OC][K][K][C] -> int32 NHWC on
    the matrix cores (hand-written kernel).  Raises on shapes the kernel does
    not cover (c or oc not a multiple of 64, windows other than 1x1 / 3x3,
    filters over 64 KiB)."""
    for t, name in ((x, "x"), (w, "w")):
        if t.dtype != torch.int8 or not t.is_cuda or not t.is_contiguous():
            raise TypeError("%s must be a contiguous int8 GPU tensor" % name)
    n, h, wd, c = x.shape
    oc, k = w.shape[0], w.shape[1]
    oh = (h + 2 * pad - k) // stride + 1
    ow = (wd + 2 * pad - k) // stride + 1
    if out is None:
        out = torch.empty((n, oh, ow, oc), dtype=torch.int32, device=x.device)
    elif (out.dtype != torch.int32 or not out.is_contiguous()
          or out.numel() != n * oh * ow * oc):
        raise ValueError("out must be a contiguous int32 [n][oh][ow][oc]")
    if stream is None:
        stream = torch.cuda.current_stream()
    lib = load_library()
    p = ConvParams(n, h, wd, c, oc, k, k, stride, pad)
    st = lib.i8mfma_conv2d(ctypes.byref(p), ctypes.c_void_p(x.data_ptr()),
                           ctypes.c_void_p(w.data_ptr()),
                           ctypes.c_void_p(out.data_ptr()),
                           ctypes.c_void_p(stream.cuda_stream))
    if st != 0:
        raise RuntimeError("i8mfma_conv2d status %d: %s" % (
            st, lib.i8mfma_last_error().decode()))
    return out


def dense_int8(a_codes: torch.Tensor, w_codes: torch.Tensor) -> torch.Tensor:
    """out[m][n] = sum_k a[m][k] w[n][k] in int32; a: [M][K], w: [N][K]
    uint8 codes < 128 on the GPU."""
    a = a_codes.to(torch.int8)
    wt = w_codes.to(torch.int8).t().contiguous()
    return torch._int_mm(a, wt)


def im2col_nhwc(x: torch.Tensor, k: int, stride: int, pad: int) -> torch.Tensor:
    """[N][H][W][C] int8 -> [N*OH*OW][K*K*C], columns ordered (ky, kx, c),
    zero padding."""
    n, h, w, c = x.shape
    xp = F.pad(x, (0, 0, pad, pad, pad, pad))
    win = xp.unfold(1, k, stride).unfold(2, k, stride)   # N,OH,OW,C,ky,kx
    oh, ow = win.shape[1], win.shape[2]
    return win.permute(0, 1, 2, 4, 5, 3).reshape(n * oh * ow, k * k * c)


def conv2d_int8(x_codes: torch.Tensor, w_codes: torch.Tensor, stride: int,
                pad: int) -> torch.Tensor:
    """NHWC codes [N][H][W][C] and OHWI filter codes [OC][K][K][C] (uint8,
    < 128) -> int32 NHWC output via im2col + int8 GEMM."""
    n, h, w, c = x_codes.shape
    oc, k = w_codes.shape[0], w_codes.shape[1]
    cols = im2col_nhwc(x_codes.to(torch.int8), k, stride, pad)
    wt = w_codes.to(torch.int8).reshape(oc, k * k * c).t().contiguous()
    oh = (h + 2 * pad - k) // stride + 1
    ow = (w + 2 * pad - k) // stride + 1
    return torch._int_mm(cols, wt).reshape(n, oh, ow, oc)
