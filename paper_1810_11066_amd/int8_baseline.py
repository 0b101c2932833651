"""int8 matrix-core comparison baseline (not part of the bitserial path).

The paper compares its bitserial operators with optimized 8-bit and 16-bit
integer implementations on the same CPU (Sec. 6.2).  The GPU analogue is an
int8 x int8 -> int32 product on the matrix cores (MFMA), which this module
takes from the vendor GEMM behind ``torch._int_mm`` (hipBLASLt on ROCm):

* dense: the activation codes [M][K] and weight codes [N][K] as int8, one
  GEMM;
* conv2d: NHWC im2col of the codes (the K x K window of every output pixel,
  tap-major then channel, matching OHWI filters) followed by one GEMM with
  the [OC][K*K*C] filters.

Codes of up to 7 bits fit int8 unchanged, so the products are exactly the
integer results the bitserial kernels compute; the tests use that to check
both paths against each other.  Nothing here is used by the bitserial
library.
"""
from __future__ import annotations

import torch
import torch.nn.functional as F

LABEL = "int8 MFMA baseline (torch._int_mm -> hipBLASLt), not bitserial"


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
