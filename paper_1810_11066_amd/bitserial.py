"""Python binding of libbitserial.so (include/bitserial.h).

The ``bs_*`` functions carry the C entry points' names and semantics and only
marshal arguments: torch tensors supply device pointers, shapes are checked,
and the current HIP stream is passed through.  Every operation runs in the
library's HIP kernels; there is no host fallback -- if the library is missing
or the device is not a GPU, the call raises.

Packed bit-plane tensors are torch.int32 tensors holding the uint32 words'
bit patterns, shaped [rows, bits, ceil(k/32)] (activations: [n, h, w, bits,
words]; conv filters: [oc, kh, kw, bits, words]).

Convenience wrappers (``quantize``, ``pack``, ``quantize_pack``, ``conv2d``,
``dense``) allocate the output with torch and call the entry point.
"""
from __future__ import annotations

import ctypes
import os
import threading
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# BITSERIAL_LIBRARY selects another build of the same library
LIB_PATH = os.environ.get("BITSERIAL_LIBRARY",
                          os.path.join(_HERE, "libbitserial.so"))

BS_OK = 0
BS_ERR_INVALID_ARG = 1
BS_ERR_UNSUPPORTED = 2
BS_ERR_OVERFLOW = 3
BS_ERR_HIP = 4

UNIPOLAR = 0
BIPOLAR = 1
SIGNED = 2

LAYOUT_MBK = 0
LAYOUT_MKB = 1
LAYOUT_BMK = 2

EXPORTED = ("bs_packed_words", "bs_quantize", "bs_pack", "bs_pack_ex",
            "bs_quantize_pack",
            "bs_conv2d_out_shape", "bs_conv2d", "bs_conv2d_requant",
            "bs_conv2d_codes", "bs_conv2d_pair", "bs_conv2d_pair_requant",
            "bs_conv2d_describe", "bs_conv2d_codes_describe",
            "bs_conv2d_quantized", "bs_conv2d_quantized_describe",
            "bs_dense", "bs_dense_ex", "bs_status_string",
            "bs_last_error", "bs_set_kernel_mode", "bs_set_units_per_wave",
            "bs_set_timing_events", "bs_abi_version")


class BitserialError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__("bitserial status %d: %s" % (status, msg))
        self.status = status


class ConvParams(ctypes.Structure):
    """Mirror of ``bs_conv2d_params``."""
    _fields_ = [(name, ctypes.c_int32) for name in (
        "n", "h", "w", "c", "oc", "kh", "kw", "stride_h", "stride_w",
        "pad_h", "pad_w", "abits", "wbits", "aenc", "wenc")]


_lock = threading.Lock()
_lib = None


def load_library():
    """Load libbitserial.so (built in-tree by paper_1810_11066_amd.build)."""
    global _lib
    if _lib is not None:
        return _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                "libbitserial.so is not built (%s); run "
                "`python -m paper_1810_11066_amd.build`" % LIB_PATH)
        lib = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        i64, ci, cf = ctypes.c_int64, ctypes.c_int, ctypes.c_float
        sig = {
            "bs_packed_words": (i64, [i64]),
            "bs_quantize": (ci, [P, P, i64, cf, ci, ci, P]),
            "bs_pack": (ci, [P, P, i64, i64, ci, P]),
            "bs_pack_ex": (ci, [P, P, i64, i64, i64, ci, ci, P]),
            "bs_quantize_pack": (ci, [P, P, i64, i64, cf, ci, ci, P]),
            "bs_conv2d_out_shape": (ci, [ctypes.POINTER(ConvParams),
                                         ctypes.POINTER(ctypes.c_int32),
                                         ctypes.POINTER(ctypes.c_int32)]),
            "bs_conv2d": (ci, [ctypes.POINTER(ConvParams), P, P, P, P]),
            "bs_conv2d_codes": (ci, [ctypes.POINTER(ConvParams), P, P, P,
                                     P]),
            "bs_conv2d_pair": (ci, [ctypes.POINTER(ConvParams), P, P, P, P, P,
                                    P]),
            "bs_conv2d_pair_requant": (ci, [ctypes.POINTER(ConvParams), P, P,
                                            P, cf, cf, ci, P, P, P]),
            "bs_conv2d_requant": (ci, [ctypes.POINTER(ConvParams), P, P, cf,
                                       ci, P, P]),
            "bs_conv2d_describe": (ci, [ctypes.POINTER(ConvParams),
                                        ctypes.c_char_p, ctypes.c_int32]),
            "bs_conv2d_codes_describe": (ci, [ctypes.POINTER(ConvParams),
                                              ctypes.c_char_p,
                                              ctypes.c_int32]),
            "bs_conv2d_quantized": (ci, [ctypes.POINTER(ConvParams), P, cf,
                                         P, P, P]),
            "bs_conv2d_quantized_describe": (ci, [ctypes.POINTER(ConvParams),
                                                  ctypes.c_char_p,
                                                  ctypes.c_int32]),
            "bs_dense": (ci, [i64, i64, i64, ci, ci, ci, P, P, P, P]),
            "bs_dense_ex": (ci, [i64, i64, i64, ci, ci, ci, ci, P, P, P, P]),
            "bs_status_string": (ctypes.c_char_p, [ci]),
            "bs_last_error": (ctypes.c_char_p, []),
            "bs_set_kernel_mode": (ci, [ci]),
            "bs_set_units_per_wave": (ci, [ci]),
            "bs_set_timing_events": (ci, [P, P]),
            "bs_abi_version": (ci, []),
        }
        for name, (res, args) in sig.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
        return lib


def _check(status: int):
    if status != BS_OK:
        lib = load_library()
        raise BitserialError(status, lib.bs_last_error().decode())


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dev(t: torch.Tensor, name: str, dtype: torch.dtype, numel: int):
    """Device address of a contiguous GPU tensor of the given dtype and
    element count; raises with the reason otherwise."""
    if (isinstance(t, torch.Tensor) and t.is_cuda and t.dtype == dtype
            and t.numel() == numel and t.is_contiguous()):
        return t.data_ptr()
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if t.device.type != "cuda":
        raise ValueError("%s must be a GPU tensor (got %s)" % (name, t.device))
    if t.dtype != dtype:
        raise TypeError("%s must be %s (got %s)" % (name, dtype, t.dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if t.numel() != numel:
        raise ValueError("%s has %d elements, expected %d" % (name, t.numel(),
                                                             numel))
    return ctypes.c_void_p(t.data_ptr())


def words(k: int) -> int:
    return (k + 31) // 32


# ---- entry points (same names as the C ABI) --------------------------------

def bs_quantize(x: torch.Tensor, q: torch.Tensor, scale: float, bits: int,
                enc: int = UNIPOLAR, stream=None) -> None:
    n = x.numel()
    _check(load_library().bs_quantize(
        _dev(x, "x", torch.float32, n), _dev(q, "q", torch.uint8, n), n,
        float(scale), int(bits), int(enc), _stream(stream)))


def bs_pack(q: torch.Tensor, packed: torch.Tensor, rows: int, k: int,
            bits: int, stream=None) -> None:
    _check(load_library().bs_pack(
        _dev(q, "q", torch.uint8, rows * k),
        _dev(packed, "packed", torch.int32, rows * bits * words(k)),
        rows, k, int(bits), _stream(stream)))


def bs_quantize_pack(x: torch.Tensor, packed: torch.Tensor, rows: int, k: int,
                     scale: float, bits: int, enc: int = UNIPOLAR,
                     stream=None) -> None:
    _check(load_library().bs_quantize_pack(
        _dev(x, "x", torch.float32, rows * k),
        _dev(packed, "packed", torch.int32, rows * bits * words(k)),
        rows, k, float(scale), int(bits), int(enc), _stream(stream)))


def _out_hw(p: ConvParams):
    """(oh, ow) of the conv p as bs_conv2d_out_shape computes it, without a
    library call; for parameters it would reject, the library's error."""
    if p.stride_h >= 1 and p.stride_w >= 1:
        eh = p.h + 2 * p.pad_h - p.kh
        ew = p.w + 2 * p.pad_w - p.kw
        if eh >= 0 and ew >= 0:
            return eh // p.stride_h + 1, ew // p.stride_w + 1
    return bs_conv2d_out_shape(p)


def bs_conv2d_out_shape(p: ConvParams):
    oh, ow = ctypes.c_int32(), ctypes.c_int32()
    _check(load_library().bs_conv2d_out_shape(ctypes.byref(p),
                                              ctypes.byref(oh),
                                              ctypes.byref(ow)))
    return oh.value, ow.value


def bs_conv2d_requant(p: ConvParams, act_packed: torch.Tensor,
                      w_packed: torch.Tensor, out_scale: float, out_bits: int,
                      out_packed: torch.Tensor, stream=None) -> None:
    """bs_conv2d with its result requantized to out_bits and bit-packed as
    [n][oh][ow][out_bits][ceil(oc/32)] words (the next layer's input)."""
    lib = load_library()
    oh, ow = _out_hw(p)
    cw = words(p.c)
    _check(lib.bs_conv2d_requant(
        ctypes.byref(p),
        _dev(act_packed, "act_packed", torch.int32,
             p.n * p.h * p.w * p.abits * cw),
        _dev(w_packed, "w_packed", torch.int32,
             p.oc * p.kh * p.kw * p.wbits * cw),
        float(out_scale), int(out_bits),
        _dev(out_packed, "out_packed", torch.int32,
             p.n * oh * ow * out_bits * words(p.oc)),
        _stream(stream)))


def conv2d_requant(spec: "Conv2dSpec", act_packed: torch.Tensor,
                   w_packed: torch.Tensor, out_scale: float,
                   out_bits: int) -> torch.Tensor:
    p = spec.params()
    oh, ow = _out_hw(p)
    out = torch.empty((p.n, oh, ow, out_bits, words(p.oc)), dtype=torch.int32,
                      device=act_packed.device)
    bs_conv2d_requant(p, act_packed, w_packed, out_scale, out_bits, out)
    return out


def bs_conv2d_describe(p: ConvParams) -> str:
    """Kernel and launch configuration bs_conv2d would use for ``p`` under
    this thread's kernel mode (host only)."""
    buf = ctypes.create_string_buffer(256)
    _check(load_library().bs_conv2d_describe(ctypes.byref(p), buf, 256))
    return buf.value.decode()


def bs_conv2d_codes_describe(p: ConvParams) -> str:
    """Kernel and launch plan bs_conv2d_codes would use for ``p`` (the
    staged plan, with its LDS region; host only)."""
    buf = ctypes.create_string_buffer(320)
    _check(load_library().bs_conv2d_codes_describe(ctypes.byref(p), buf, 320))
    return buf.value.decode()


def bs_conv2d_quantized_describe(p: ConvParams) -> str:
    """Kernel and launch plan bs_conv2d_quantized would use for ``p`` (host
    only)."""
    buf = ctypes.create_string_buffer(320)
    _check(load_library().bs_conv2d_quantized_describe(ctypes.byref(p), buf,
                                                        320))
    return buf.value.decode()


def bs_conv2d(p: ConvParams, act_packed: torch.Tensor, w_packed: torch.Tensor,
              out: torch.Tensor, stream=None) -> None:
    lib = load_library()
    oh, ow = _out_hw(p)
    cw = words(p.c)
    _check(lib.bs_conv2d(
        ctypes.byref(p),
        _dev(act_packed, "act_packed", torch.int32,
             p.n * p.h * p.w * p.abits * cw),
        _dev(w_packed, "w_packed", torch.int32,
             p.oc * p.kh * p.kw * p.wbits * cw),
        _dev(out, "out", torch.int32, p.n * oh * ow * p.oc),
        _stream(stream)))


def bs_conv2d_codes(p: ConvParams, act_codes: torch.Tensor,
                    w_packed: torch.Tensor, out: torch.Tensor,
                    stream=None) -> None:
    """bs_pack of the uint8 NHWC codes fused into bs_conv2d."""
    oh, ow = _out_hw(p)
    _check(load_library().bs_conv2d_codes(
        ctypes.byref(p),
        _dev(act_codes, "act_codes", torch.uint8, p.n * p.h * p.w * p.c),
        _dev(w_packed, "w_packed", torch.int32,
             p.oc * p.kh * p.kw * p.wbits * words(p.c)),
        _dev(out, "out", torch.int32, p.n * oh * ow * p.oc),
        _stream(stream)))


def bs_conv2d_quantized(p: ConvParams, act: torch.Tensor, act_scale: float,
                        w_packed: torch.Tensor, out: torch.Tensor,
                        stream=None) -> None:
    """bs_quantize_pack of the float32 NHWC activations (unipolar,
    act_scale, p.abits bits) fused into bs_conv2d (1x1 windows)."""
    oh, ow = _out_hw(p)
    _check(load_library().bs_conv2d_quantized(
        ctypes.byref(p),
        _dev(act, "act", torch.float32, p.n * p.h * p.w * p.c),
        float(act_scale),
        _dev(w_packed, "w_packed", torch.int32,
             p.oc * p.kh * p.kw * p.wbits * words(p.c)),
        _dev(out, "out", torch.int32, p.n * oh * ow * p.oc),
        _stream(stream)))


def bs_conv2d_pair(p: ConvParams, act_packed: torch.Tensor,
                   w_packed: torch.Tensor, w1_packed: torch.Tensor,
                   out: torch.Tensor, out1: torch.Tensor,
                   stream=None) -> None:
    """The KxK conv p and its centre-tap 1x1 conv in one pass."""
    oh, ow = _out_hw(p)
    cw = words(p.c)
    _check(load_library().bs_conv2d_pair(
        ctypes.byref(p),
        _dev(act_packed, "act_packed", torch.int32,
             p.n * p.h * p.w * p.abits * cw),
        _dev(w_packed, "w_packed", torch.int32,
             p.oc * p.kh * p.kw * p.wbits * cw),
        _dev(w1_packed, "w1_packed", torch.int32, p.oc * p.wbits * cw),
        _dev(out, "out", torch.int32, p.n * oh * ow * p.oc),
        _dev(out1, "out1", torch.int32, p.n * oh * ow * p.oc),
        _stream(stream)))


def bs_conv2d_pair_requant(p: ConvParams, act_packed: torch.Tensor,
                           w_packed: torch.Tensor, w1_packed: torch.Tensor,
                           out_scale: float, out1_scale: float,
                           out_bits: int, out_packed: torch.Tensor,
                           out1_packed: torch.Tensor, stream=None) -> None:
    oh, ow = _out_hw(p)
    cw = words(p.c)
    n_out = p.n * oh * ow * out_bits * words(p.oc)
    _check(load_library().bs_conv2d_pair_requant(
        ctypes.byref(p),
        _dev(act_packed, "act_packed", torch.int32,
             p.n * p.h * p.w * p.abits * cw),
        _dev(w_packed, "w_packed", torch.int32,
             p.oc * p.kh * p.kw * p.wbits * cw),
        _dev(w1_packed, "w1_packed", torch.int32, p.oc * p.wbits * cw),
        float(out_scale), float(out1_scale), int(out_bits),
        _dev(out_packed, "out_packed", torch.int32, n_out),
        _dev(out1_packed, "out1_packed", torch.int32, n_out),
        _stream(stream)))


def bs_dense(m: int, n: int, k: int, abits: int, wbits: int, wenc: int,
             a_packed: torch.Tensor, w_packed: torch.Tensor,
             out: torch.Tensor, stream=None) -> None:
    _check(load_library().bs_dense(
        m, n, k, int(abits), int(wbits), int(wenc),
        _dev(a_packed, "a_packed", torch.int32, m * abits * words(k)),
        _dev(w_packed, "w_packed", torch.int32, n * wbits * words(k)),
        _dev(out, "out", torch.int32, m * n), _stream(stream)))


def bs_dense_ex(m: int, n: int, k: int, abits: int, aenc: int, wbits: int,
                wenc: int, a_packed: torch.Tensor, w_packed: torch.Tensor,
                out: torch.Tensor, stream=None) -> None:
    _check(load_library().bs_dense_ex(
        m, n, k, int(abits), int(aenc), int(wbits), int(wenc),
        _dev(a_packed, "a_packed", torch.int32, m * abits * words(k)),
        _dev(w_packed, "w_packed", torch.int32, n * wbits * words(k)),
        _dev(out, "out", torch.int32, m * n), _stream(stream)))


def bs_pack_ex(q: torch.Tensor, packed: torch.Tensor, outer: int, k: int,
               inner: int, bits: int, layout: int = LAYOUT_MBK,
               stream=None) -> None:
    _check(load_library().bs_pack_ex(
        _dev(q, "q", torch.uint8, outer * k * inner),
        _dev(packed, "packed", torch.int32, outer * inner * bits * words(k)),
        outer, k, inner, int(bits), int(layout), _stream(stream)))


def bs_set_kernel_mode(mode: int) -> None:
    _check(load_library().bs_set_kernel_mode(int(mode)))


def bs_set_units_per_wave(units: int) -> None:
    _check(load_library().bs_set_units_per_wave(int(units)))


def bs_set_timing_events(start=None, stop=None) -> None:
    """Attach torch.cuda.Event start/stop (or None) to the library's later
    kernel dispatches from this thread (bs_set_timing_events).  The events
    are recorded once on the current stream first, so that their HIP events
    exist; after a call, start.elapsed_time(stop) is its kernel's duration."""
    handles = []
    for e in (start, stop):
        if e is None:
            handles.append(None)
            continue
        if not isinstance(e, torch.cuda.Event):
            raise TypeError("timing events must be torch.cuda.Event")
        e.record(torch.cuda.current_stream())
        handles.append(ctypes.c_void_p(e.cuda_event))
    _check(load_library().bs_set_timing_events(*handles))


def bs_packed_words(k: int) -> int:
    return load_library().bs_packed_words(k)


def bs_abi_version() -> int:
    return load_library().bs_abi_version()


# ---- allocating conveniences -----------------------------------------------

@dataclass
class Conv2dSpec:
    n: int
    h: int
    w: int
    c: int
    oc: int
    kh: int
    kw: int
    stride: int = 1
    pad: int = 0
    abits: int = 1
    wbits: int = 1
    wenc: int = UNIPOLAR
    aenc: int = UNIPOLAR

    def params(self) -> ConvParams:
        return ConvParams(self.n, self.h, self.w, self.c, self.oc, self.kh,
                          self.kw, self.stride, self.stride, self.pad,
                          self.pad, self.abits, self.wbits, self.aenc,
                          self.wenc)


def quantize(x: torch.Tensor, scale: float, bits: int, enc: int = UNIPOLAR):
    q = torch.empty(x.shape, dtype=torch.uint8, device=x.device)
    bs_quantize(x, q, scale, bits, enc)
    return q


def pack(q: torch.Tensor, bits: int) -> torch.Tensor:
    """q: [..., k] uint8 -> [..., bits, ceil(k/32)] int32 words."""
    k = q.shape[-1]
    rows = q.numel() // k
    out = torch.empty(tuple(q.shape[:-1]) + (bits, words(k)),
                      dtype=torch.int32, device=q.device)
    bs_pack(q, out, rows, k, bits)
    return out


def pack_ex(q: torch.Tensor, bits: int, axis: int = -1,
            layout: int = LAYOUT_MBK) -> torch.Tensor:
    """Pack q (any rank, uint8) along ``axis``; the packed rows are the
    other axes in order.  Returns [rows][bits][words] (MBK'),
    [rows][words][bits] (MK'B) or [bits][rows][words] (BMK') int32 words."""
    axis = axis % q.dim()
    k = q.shape[axis]
    outer = 1
    for d in q.shape[:axis]:
        outer *= d
    inner = q.numel() // (outer * k)
    rows, kw = outer * inner, words(k)
    shape = {LAYOUT_MBK: (rows, bits, kw), LAYOUT_MKB: (rows, kw, bits),
             LAYOUT_BMK: (bits, rows, kw)}[layout]
    out = torch.empty(shape, dtype=torch.int32, device=q.device)
    bs_pack_ex(q, out, outer, k, inner, bits, layout)
    return out


def quantize_pack(x: torch.Tensor, scale: float, bits: int,
                  enc: int = UNIPOLAR) -> torch.Tensor:
    k = x.shape[-1]
    rows = x.numel() // k
    out = torch.empty(tuple(x.shape[:-1]) + (bits, words(k)),
                      dtype=torch.int32, device=x.device)
    bs_quantize_pack(x, out, rows, k, scale, bits, enc)
    return out


def conv2d(spec: Conv2dSpec, act_packed: torch.Tensor,
           w_packed: torch.Tensor) -> torch.Tensor:
    p = spec.params()
    oh, ow = _out_hw(p)
    out = torch.empty((spec.n, oh, ow, spec.oc), dtype=torch.int32,
                      device=act_packed.device)
    bs_conv2d(p, act_packed, w_packed, out)
    return out


def conv2d_codes(spec: Conv2dSpec, act_codes: torch.Tensor,
                 w_packed: torch.Tensor) -> torch.Tensor:
    """Conv of uint8 NHWC codes, the activation pack fused into the conv."""
    p = spec.params()
    oh, ow = _out_hw(p)
    out = torch.empty((spec.n, oh, ow, spec.oc), dtype=torch.int32,
                      device=act_codes.device)
    bs_conv2d_codes(p, act_codes, w_packed, out)
    return out


def conv2d_pair(spec: Conv2dSpec, act_packed: torch.Tensor,
                w_packed: torch.Tensor, w1_packed: torch.Tensor):
    """(out, out1): the KxK conv and its centre-tap 1x1 conv."""
    p = spec.params()
    oh, ow = _out_hw(p)
    out = torch.empty((spec.n, oh, ow, spec.oc), dtype=torch.int32,
                      device=act_packed.device)
    out1 = torch.empty_like(out)
    bs_conv2d_pair(p, act_packed, w_packed, w1_packed, out, out1)
    return out, out1


def conv2d_pair_requant(spec: Conv2dSpec, act_packed: torch.Tensor,
                        w_packed: torch.Tensor, w1_packed: torch.Tensor,
                        out_scale: float, out1_scale: float, out_bits: int):
    p = spec.params()
    oh, ow = _out_hw(p)
    shape = (p.n, oh, ow, out_bits, words(p.oc))
    out = torch.empty(shape, dtype=torch.int32, device=act_packed.device)
    out1 = torch.empty(shape, dtype=torch.int32, device=act_packed.device)
    bs_conv2d_pair_requant(p, act_packed, w_packed, w1_packed, out_scale,
                           out1_scale, out_bits, out, out1)
    return out, out1


def dense(a_packed: torch.Tensor, w_packed: torch.Tensor, m: int, n: int,
          k: int, abits: int, wbits: int, wenc: int = UNIPOLAR,
          aenc: int = UNIPOLAR):
    out = torch.empty((m, n), dtype=torch.int32, device=a_packed.device)
    if aenc == UNIPOLAR:
        bs_dense(m, n, k, abits, wbits, wenc, a_packed, w_packed, out)
    else:
        bs_dense_ex(m, n, k, abits, aenc, wbits, wenc, a_packed, w_packed,
                    out)
    return out
