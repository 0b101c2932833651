"""CPU oracle for low-precision bitserial operators -- Python face of ``bsref.c``.

TEST INFRASTRUCTURE ONLY.  Imported by the tests, the smoke check and the
benchmark's CPU-baseline leg; the product path (the HIP library and its
binding) never imports it, and it imports nothing from the product package.

Every function takes and returns host numpy arrays and calls the plain C
oracle (``libbsref.so``, built here with gcc).  The semantics of each call are
documented in ``bsref.h``; the paper passages they follow are:

* ``quantize``  -- quantization of float data to k bits (Sec. 3.1)
* ``pack``      -- bit-plane split and packing into uint32 words (Sec. 2.2,
  Sec. 3.1, layout MBK')
* ``pack_ex``   -- the same with any reduction-axis stride and bit-axis
  position (MBK', MK'B, BMK'; Sec. 3.1)
* ``conv2d``    -- bitserial conv2d, NHWC / OHWI (Sec. 3.2; Eq. 1, Eq. 2 reach
  exactly the integer convolution, which is what the oracle evaluates)
* ``dense``     -- bitserial dense / matmul (Sec. 3.2, Sec. 6.2.1)

Encodings (Sec. 2.2): unipolar codes, bipolar (+-1) codes and signed (two's
complement) codes, for activations and weights alike.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "bsref.c")
_LIB_PATH = os.path.join(_HERE, "libbsref.so")
# BSREF_LIBRARY: load this compiled copy of bsref.c instead (the mutation
# tests point it at deliberately broken copies, to show that the pins reject
# them)
_OVERRIDE = os.environ.get("BSREF_LIBRARY")

UNIPOLAR = 0
BIPOLAR = 1
SIGNED = 2

LAYOUT_MBK = 0
LAYOUT_MKB = 1
LAYOUT_BMK = 2

_lock = threading.Lock()
_lib = None


def compile_to(src: str, out: str) -> None:
    """gcc command line of the oracle: plain C11 + OpenMP, IEEE float."""
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
           "-ffp-contract=off", "-fno-fast-math", "-Wall", "-Wextra",
           src, "-o", out, "-lm"]
    subprocess.run(cmd, check=True, cwd=os.path.dirname(src))


def build(force: bool = True) -> str:
    """Compile ``libbsref.so`` with gcc (plain C11 + OpenMP).  Returns its path."""
    if _OVERRIDE:
        return _OVERRIDE
    if not force and os.path.exists(_LIB_PATH) and \
            os.path.getmtime(_LIB_PATH) >= os.path.getmtime(_SRC):
        return _LIB_PATH
    tmp = _LIB_PATH + ".tmp%d" % os.getpid()
    compile_to(_SRC, tmp)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


class ConvParams(ctypes.Structure):
    """Mirror of ``bsref_conv2d_params`` (bsref.h)."""
    _fields_ = [(name, ctypes.c_int32) for name in (
        "n", "h", "w", "c", "oc", "kh", "kw", "stride_h", "stride_w",
        "pad_h", "pad_w", "abits", "wbits", "aenc", "wenc")]


def _load():
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        lib = ctypes.CDLL(build(force=False))
        P = ctypes.c_void_p
        i64 = ctypes.c_int64
        ci = ctypes.c_int
        lib.bsref_quantize.argtypes = [P, P, i64, ctypes.c_float, ci, ci]
        lib.bsref_pack.argtypes = [P, P, i64, i64, ci]
        lib.bsref_pack_ex.argtypes = [P, P, i64, i64, i64, ci, ci]
        lib.bsref_conv2d_out_shape.argtypes = [
            ctypes.POINTER(ConvParams), ctypes.POINTER(ctypes.c_int32),
            ctypes.POINTER(ctypes.c_int32)]
        lib.bsref_conv2d.argtypes = [ctypes.POINTER(ConvParams), P, P, P]
        lib.bsref_conv2d_at.argtypes = [ctypes.POINTER(ConvParams), P, P, P,
                                        i64, P]
        lib.bsref_dense.argtypes = [i64, i64, i64, ci, ci, ci, P, P, P]
        lib.bsref_dense_ex.argtypes = [i64, i64, i64, ci, ci, ci, ci, P, P, P]
        for fn in ("bsref_quantize", "bsref_pack", "bsref_pack_ex",
                   "bsref_conv2d_out_shape", "bsref_conv2d", "bsref_conv2d_at",
                   "bsref_dense", "bsref_dense_ex", "bsref_threads",
                   "bsref_set_threads"):
            getattr(lib, fn).restype = ci
        _lib = lib
        return lib


class OracleError(RuntimeError):
    pass


def _check(rc: int, what: str):
    if rc != 0:
        raise OracleError("%s returned %d" % (what, rc))


def _ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data)


def threads() -> int:
    return _load().bsref_threads()


def set_threads(n: int) -> None:
    """Host threads for later oracle calls from this thread (timing only;
    results do not depend on it)."""
    lib = _load()
    lib.bsref_set_threads.argtypes = [ctypes.c_int]
    _check(lib.bsref_set_threads(n), "bsref_set_threads")


def words(k: int) -> int:
    return (k + 31) // 32


def quantize(x: np.ndarray, scale: float, bits: int, enc: int = UNIPOLAR):
    x = np.ascontiguousarray(x, dtype=np.float32)
    q = np.empty(x.shape, dtype=np.uint8)
    _check(_load().bsref_quantize(_ptr(x), _ptr(q), x.size, float(scale),
                                  bits, enc), "bsref_quantize")
    return q


def pack(q: np.ndarray, bits: int):
    """q: [..., k] uint8 -> [..., bits, ceil(k/32)] uint32."""
    q = np.ascontiguousarray(q, dtype=np.uint8)
    k = q.shape[-1]
    rows = q.size // k
    out = np.empty(q.shape[:-1] + (bits, words(k)), dtype=np.uint32)
    _check(_load().bsref_pack(_ptr(q), _ptr(out), rows, k, bits),
           "bsref_pack")
    return out


def pack_ex(q: np.ndarray, bits: int, axis: int = -1,
            layout: int = LAYOUT_MBK):
    """Pack along ``axis`` of q (any rank).  The packed rows are the other
    axes in order (the leading ones, then the trailing ones); the result is
    [rows][bits][words] (MBK'), [rows][words][bits] (MK'B) or
    [bits][rows][words] (BMK'), rows flattened."""
    q = np.ascontiguousarray(q, dtype=np.uint8)
    axis = axis % q.ndim
    k = q.shape[axis]
    outer = int(np.prod(q.shape[:axis], dtype=np.int64))
    inner = int(np.prod(q.shape[axis + 1:], dtype=np.int64))
    rows, kw = outer * inner, words(k)
    shape = {LAYOUT_MBK: (rows, bits, kw), LAYOUT_MKB: (rows, kw, bits),
             LAYOUT_BMK: (bits, rows, kw)}[layout]
    out = np.empty(shape, dtype=np.uint32)
    _check(_load().bsref_pack_ex(_ptr(q), _ptr(out), outer, k, inner, bits,
                                 layout), "bsref_pack_ex")
    return out


def conv_params(n, h, w, c, oc, kh, kw, stride=(1, 1), pad=(0, 0),
                abits=1, wbits=1, aenc=UNIPOLAR, wenc=UNIPOLAR) -> ConvParams:
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    ph, pw = (pad, pad) if np.isscalar(pad) else pad
    return ConvParams(n, h, w, c, oc, kh, kw, sh, sw, ph, pw, abits, wbits,
                      aenc, wenc)


def conv2d_out_shape(p: ConvParams):
    oh, ow = ctypes.c_int32(), ctypes.c_int32()
    _check(_load().bsref_conv2d_out_shape(ctypes.byref(p), ctypes.byref(oh),
                                          ctypes.byref(ow)),
           "bsref_conv2d_out_shape")
    return oh.value, ow.value


def _conv_inputs(p: ConvParams, act: np.ndarray, wts: np.ndarray):
    act = np.ascontiguousarray(act, dtype=np.uint32)
    wts = np.ascontiguousarray(wts, dtype=np.uint32)
    cw = words(p.c)
    if act.size != p.n * p.h * p.w * p.abits * cw:
        raise ValueError("packed activation size mismatch")
    if wts.size != p.oc * p.kh * p.kw * p.wbits * cw:
        raise ValueError("packed weight size mismatch")
    return act, wts


def conv2d(p: ConvParams, act: np.ndarray, wts: np.ndarray) -> np.ndarray:
    act, wts = _conv_inputs(p, act, wts)
    oh, ow = conv2d_out_shape(p)
    out = np.empty((p.n, oh, ow, p.oc), dtype=np.int32)
    _check(_load().bsref_conv2d(ctypes.byref(p), _ptr(act), _ptr(wts),
                                _ptr(out)), "bsref_conv2d")
    return out


def conv2d_at(p: ConvParams, act: np.ndarray, wts: np.ndarray,
              idx: np.ndarray) -> np.ndarray:
    """Outputs at flat indices ``idx`` into the [n][oh][ow][oc] result."""
    act, wts = _conv_inputs(p, act, wts)
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    vals = np.empty(idx.shape, dtype=np.int32)
    _check(_load().bsref_conv2d_at(ctypes.byref(p), _ptr(act), _ptr(wts),
                                   _ptr(idx), idx.size, _ptr(vals)),
           "bsref_conv2d_at")
    return vals


def dense(a: np.ndarray, w: np.ndarray, m: int, n: int, k: int, abits: int,
          wbits: int, wenc: int = UNIPOLAR, aenc: int = UNIPOLAR) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.uint32)
    w = np.ascontiguousarray(w, dtype=np.uint32)
    if a.size != m * abits * words(k) or w.size != n * wbits * words(k):
        raise ValueError("packed operand size mismatch")
    out = np.empty((m, n), dtype=np.int32)
    _check(_load().bsref_dense_ex(m, n, k, abits, aenc, wbits, wenc, _ptr(a),
                                  _ptr(w), _ptr(out)), "bsref_dense_ex")
    return out
