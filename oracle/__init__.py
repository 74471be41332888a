"""CPU oracle for reduced-precision integer convolution -- TEST INFRASTRUCTURE.

Only the test suite, the smoke check and the CPU-baseline leg of the benchmark
may import this package.  The GPU library never imports it, and it imports
nothing from the GPU library: the two share no code.

The arithmetic lives in ``qconv_oracle.c`` (plain C loops, exact int64 sums);
this module builds it with gcc on first use, loads it with ctypes and composes
the steps of the path:

    relayout_pack   int8 NCHW / KCRS  ->  packed NHWC / KRSC   (Sec. 1, Sec. 3.3)
    unpack          packed words      ->  integer values       (Sec. 1)
    conv2d          direct convolution, exact int32 result      (Sec. 2.1, Sec. 3.2.1)
    requant         multiplier, round-half-up shift, ReLU, clamp (Sec. 3.2.2)
    pack_output     4-bit nibbles (8 per word) or int8          (Sec. 3.2.3)

Every function is exact, so there is exactly one correct output for each input.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "qconv_oracle.c")
_BUILD = os.path.join(_HERE, "_build")
_LIB = os.path.join(_BUILD, "liboracle.so")
_lock = threading.Lock()
_lib = None

OK = 0
EINVAL = -1
EOVERFLOW = -5


def build(force: bool = False) -> str:
    """Compile the C oracle into ``oracle/_build/liboracle.so`` (gcc -O2 -fopenmp)."""
    os.makedirs(_BUILD, exist_ok=True)
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-Wall", "-Wextra",
               _SRC, "-o", tmp]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        lib = ctypes.CDLL(build())
        i64, i32, vp = ctypes.c_int64, ctypes.c_int, ctypes.c_void_p
        lib.oracle_out_dim.argtypes = [i64, i64, i64, i64]
        lib.oracle_out_dim.restype = i64
        lib.oracle_saturate.argtypes = [i64, i32, i32]
        lib.oracle_saturate.restype = i64
        lib.oracle_unpack4.argtypes = [vp, i64, i32, vp]
        lib.oracle_unpack4.restype = None
        lib.oracle_pack4.argtypes = [vp, i64, i32, vp]
        lib.oracle_pack4.restype = i32
        lib.oracle_relayout_pack.argtypes = [vp, i64, i64, i64, i64, i32, i32, vp]
        lib.oracle_relayout_pack.restype = i32
        lib.oracle_conv2d.argtypes = [vp, vp] + [i64] * 11 + [vp, i64, vp, i32]
        lib.oracle_conv2d.restype = i32
        lib.oracle_requant.argtypes = [vp, i64, i64, vp, i32, i32, i64, i64, vp]
        lib.oracle_requant.restype = i32
        lib.oracle_requant_ext.argtypes = [vp, i64, i64, vp, vp, i32, vp, i32, i64, i64, vp]
        lib.oracle_requant_ext.restype = i32
        lib.oracle_max_threads.argtypes = []
        lib.oracle_max_threads.restype = i32
        _lib = lib
        return lib


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.c_void_p)


class OracleError(RuntimeError):
    pass


def max_threads() -> int:
    return int(_load().oracle_max_threads())


def out_dim(size: int, window: int, stride: int, pad: int) -> int:
    """Output extent floor((size + 2*pad - window) / stride) + 1 (Sec. 2.1 reading)."""
    v = int(_load().oracle_out_dim(size, window, stride, pad))
    if v < 1:
        raise OracleError("window does not fit the padded input")
    return v


def saturate(v: int, bits: int, is_signed: bool) -> int:
    return int(_load().oracle_saturate(int(v), bits, int(bool(is_signed))))


def unpack4(words: np.ndarray, count: int, is_signed: bool) -> np.ndarray:
    """4-bit values from uint32 words; value 8j+i is bits [4i,4i+3] of word j."""
    words = np.ascontiguousarray(words, dtype=np.uint32).reshape(-1)
    if count % 8 or count > 8 * words.size:
        raise OracleError("count must be a multiple of 8 within the words given")
    out = np.empty(count, dtype=np.int32)
    _load().oracle_unpack4(_ptr(words), count, int(bool(is_signed)), _ptr(out))
    return out


def pack4(vals: np.ndarray, is_signed: bool) -> np.ndarray:
    """Pack in-range 4-bit values (count a multiple of 8) into uint32 words."""
    vals = np.ascontiguousarray(vals, dtype=np.int32).reshape(-1)
    if vals.size % 8:
        raise OracleError("count must be a multiple of 8")
    words = np.empty(vals.size // 8, dtype=np.uint32)
    rc = _load().oracle_pack4(_ptr(vals), vals.size, int(bool(is_signed)), _ptr(words))
    if rc != OK:
        raise OracleError("value outside the 4-bit range")
    return words


def relayout_pack(src: np.ndarray, bits: int, is_signed: bool) -> np.ndarray:
    """int8 N x C x H x W -> saturated, channel-packed N x H x W x ... .

    bits=4: uint32 array of shape (N, H, W, C//8); bits=8: int8 (N, H, W, C).
    Filters use the same call with (K, C, R, S) -> (K, R, S, ...).
    """
    src = np.ascontiguousarray(src, dtype=np.int8)
    n, c, h, w = src.shape
    if bits == 4:
        if c % 8:
            raise OracleError("4-bit packing needs C % 8 == 0")
        dst = np.empty((n, h, w, c // 8), dtype=np.uint32)
    elif bits == 8:
        dst = np.empty((n, h, w, c), dtype=np.int8)
    else:
        raise OracleError("bits must be 4 or 8")
    rc = _load().oracle_relayout_pack(_ptr(src), n, c, h, w, bits, int(bool(is_signed)), _ptr(dst))
    if rc != OK:
        raise OracleError("relayout_pack failed (%d)" % rc)
    return dst


def unpack_tensor(packed: np.ndarray, channels: int, bits: int, is_signed: bool) -> np.ndarray:
    """Packed N x H x W x (...) -> int32 N x H x W x C values."""
    lead = packed.shape[:-1]
    if bits == 4:
        flat = unpack4(packed.reshape(-1), int(np.prod(lead)) * channels, is_signed)
        return flat.reshape(*lead, channels)
    if bits == 8:
        return np.asarray(packed, dtype=np.int8).astype(np.int32).reshape(*lead, channels)
    raise OracleError("bits must be 4 or 8")


def conv2d(x_nhwc: np.ndarray, w_krsc: np.ndarray, stride=(1, 1), pad=(0, 0),
           pixels: np.ndarray | None = None, threads: int = 1) -> np.ndarray:
    """Exact direct convolution (Sec. 2.1) of int values; returns int32.

    x: N x H x W x C, w: K x R x S x C.  Without ``pixels`` the result is
    N x P x Q x K; with ``pixels`` (flat output indices n*P*Q + p*Q + q) it is
    len(pixels) x K.  Raises OracleError if any |acc| >= 2^31 (Sec. 3.2.1).
    """
    x = np.ascontiguousarray(x_nhwc, dtype=np.int32)
    w = np.ascontiguousarray(w_krsc, dtype=np.int32)
    n, h, wd, c = x.shape
    k, r, s, c2 = w.shape
    if c != c2:
        raise OracleError("channel mismatch")
    sh, sw = stride
    ph, pw = pad
    p = out_dim(h, r, sh, ph)
    q = out_dim(wd, s, sw, pw)
    if pixels is None:
        acc = np.empty((n, p, q, k), dtype=np.int32)
        pix_ptr, npix = None, n * p * q
    else:
        pixels = np.ascontiguousarray(pixels, dtype=np.int64)
        acc = np.empty((pixels.size, k), dtype=np.int32)
        pix_ptr, npix = _ptr(pixels), pixels.size
    rc = _load().oracle_conv2d(_ptr(x), _ptr(w), n, h, wd, c, k, r, s, sh, sw, ph, pw,
                               pix_ptr, npix, _ptr(acc), int(threads))
    if rc == EOVERFLOW:
        raise OracleError("accumulator outside the int32 range")
    if rc != OK:
        raise OracleError("conv2d failed (%d)" % rc)
    return acc


def requant(acc: np.ndarray, mult: np.ndarray, shift: int, relu: bool, lo: int, hi: int,
            bias: np.ndarray | None = None, residual: np.ndarray | None = None) -> np.ndarray:
    """Per-channel scale, round half up, ReLU, clamp (Sec. 3.2.2 order); channels last.
    With ``bias`` (int32 per channel, accumulator units, added before scaling)
    and/or ``residual`` (int values shaped like acc, output units, added after
    rounding and before ReLU and clipping)."""
    acc = np.ascontiguousarray(acc, dtype=np.int32)
    mult = np.ascontiguousarray(mult, dtype=np.int32).reshape(-1)
    k = acc.shape[-1]
    if mult.size != k:
        raise OracleError("one multiplier per output channel")
    out = np.empty_like(acc)
    if bias is None and residual is None:
        rc = _load().oracle_requant(_ptr(acc), acc.size // k, k, _ptr(mult), int(shift), int(bool(relu)),
                                    int(lo), int(hi), _ptr(out))
    else:
        b = None if bias is None else np.ascontiguousarray(bias, dtype=np.int32).reshape(-1)
        if b is not None and b.size != k:
            raise OracleError("one bias per output channel")
        r = None if residual is None else np.ascontiguousarray(residual, dtype=np.int32)
        if r is not None and r.shape != acc.shape:
            raise OracleError("residual must be shaped like the accumulators")
        rc = _load().oracle_requant_ext(_ptr(acc), acc.size // k, k, _ptr(mult), None if b is None else _ptr(b),
                                        int(shift), None if r is None else _ptr(r), int(bool(relu)), int(lo), int(hi),
                                        _ptr(out))
    if rc != OK:
        raise OracleError("requant: shift must be in [1, 62] and lo <= hi")
    return out


def pack_output(vals: np.ndarray, bits: int, is_signed: bool) -> np.ndarray:
    """Requantised N x P x Q x K values -> the packed layout the next layer reads."""
    vals = np.ascontiguousarray(vals, dtype=np.int32)
    lead, k = vals.shape[:-1], vals.shape[-1]
    if bits == 4:
        if k % 8:
            raise OracleError("4-bit output needs K % 8 == 0")
        return pack4(vals.reshape(-1), is_signed).reshape(*lead, k // 8)
    if bits == 8:
        if vals.min(initial=0) < -128 or vals.max(initial=0) > 127:
            raise OracleError("value outside int8")
        return vals.astype(np.int8)
    raise OracleError("bits must be 4 or 8")


def qconv_layer(x_nchw: np.ndarray, w_kcrs: np.ndarray, *, bits: int, x_signed: bool, w_signed: bool,
                stride=(1, 1), pad=(0, 0), mult=None, shift=None, relu=False, lo=None, hi=None,
                threads: int = 1, packed_x: np.ndarray | None = None, bias: np.ndarray | None = None,
                residual: np.ndarray | None = None) -> dict:
    """The whole path for one layer, step by step.

    Returns a dict with ``x_packed``, ``w_packed``, ``acc`` (int32 N x P x Q x K)
    and, when ``mult`` is given, ``y`` (requantised values) and ``y_packed``.
    ``packed_x`` may be given instead of ``x_nchw`` (a chained layer's input);
    ``bias`` and ``residual`` extend the epilogue as in :func:`requant`.
    """
    if packed_x is None:
        x_packed = relayout_pack(x_nchw, bits, x_signed)
    else:
        x_packed = packed_x
    w_packed = relayout_pack(w_kcrs, bits, w_signed)
    c = w_kcrs.shape[1]
    xv = unpack_tensor(x_packed, c, bits, x_signed)
    wv = unpack_tensor(w_packed, c, bits, w_signed)
    acc = conv2d(xv, wv, stride, pad, threads=threads)
    out = {"x_packed": x_packed, "w_packed": w_packed, "acc": acc}
    if mult is not None:
        y = requant(acc, mult, shift, relu, lo, hi, bias=bias, residual=residual)
        out["y"] = y
        out["y_packed"] = pack_output(y, bits, lo < 0)
    return out
