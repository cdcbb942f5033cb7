"""CPU oracle for the bitpacked binary convolution (arXiv 2011.09398, Sec. 3.2).

TEST INFRASTRUCTURE.  Only tests/, __graft_entry__.smoke() and bench.py's
cpu_baseline leg may import this package.  The HIP path never calls it.

Thin ctypes wrapper over the plain C definitions in lce_oracle.c plus the
composition of the four steps (binarize/pack -> convolve -> clamp -> output
transform).  Shapes follow the operator's NHWC activations and OHWI filters.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import numpy as np

from . import build as _build

_lib = None

_i8p = np.ctypeslib.ndpointer(np.int8, flags="C_CONTIGUOUS")
_i32p = np.ctypeslib.ndpointer(np.int32, flags="C_CONTIGUOUS")
_u32p = np.ctypeslib.ndpointer(np.uint32, flags="C_CONTIGUOUS")
_f32p = np.ctypeslib.ndpointer(np.float32, flags="C_CONTIGUOUS")
_f64p = np.ctypeslib.ndpointer(np.float64, flags="C_CONTIGUOUS")
_i64 = ctypes.c_int64
_int = ctypes.c_int


def lib():
    global _lib
    if _lib is None:
        # LCE_ORACLE_LIB lets the mutation tests load a deliberately broken copy.
        path = os.environ.get("LCE_ORACLE_LIB") or _build.LIB
        if path == _build.LIB and not os.path.exists(path):
            _build.build()
        L = ctypes.CDLL(path)
        L.oracle_num_threads.restype = _int
        L.oracle_set_num_threads.argtypes = [_int]
        L.oracle_out_size.argtypes = [_int, _int, _int, _int,
                                      ctypes.POINTER(_int), ctypes.POINTER(_int)]
        L.oracle_out_size.restype = _int
        L.oracle_binarize.argtypes = [_f32p, _i64, _i8p]
        L.oracle_pack.argtypes = [_i8p, _i64, _int, _u32p]
        L.oracle_unpack.argtypes = [_u32p, _i64, _int, _i8p]
        L.oracle_conv_dot.argtypes = [_i8p, _int, _int, _int, _int, _i8p, _int, _int, _int,
                                      _int, _int, _int, _i32p]
        L.oracle_conv_dot.restype = _int
        L.oracle_conv_dot_padded.argtypes = [_i8p, _int, _int, _int, _int, _i8p, _int, _int,
                                             _int, _int, _int, _int, _int, _i32p]
        L.oracle_conv_dot_padded.restype = _int
        L.oracle_bmaxpool.argtypes = [_i8p, _int, _int, _int, _int, _int, _int, _int, _int,
                                      _int, _i8p]
        L.oracle_bmaxpool.restype = _int
        L.oracle_sign_of_affine.argtypes = [_i32p, _i64, ctypes.c_float, ctypes.c_float,
                                            np.ctypeslib.ndpointer(np.uint8, flags="C_CONTIGUOUS")]
        L.oracle_clamp.argtypes = [_i32p, _i64, ctypes.c_int32, ctypes.c_int32, _i32p]
        L.oracle_out_float.argtypes = [_i32p, _i64, _int, ctypes.c_void_p, ctypes.c_void_p, _f64p]
        L.oracle_out_bits.argtypes = [_i32p, _i64, _int, _f32p, _u32p]
        _lib = L
    return _lib


def num_threads() -> int:
    return lib().oracle_num_threads()


def set_num_threads(n: int) -> None:
    lib().oracle_set_num_threads(int(n))


def out_size(in_: int, k: int, s: int, padding: str) -> Tuple[int, int]:
    """(output size, leading pad) of one spatial dimension; TF SAME/VALID."""
    o, p = _int(), _int()
    if lib().oracle_out_size(in_, k, s, 1 if padding == "same" else 0,
                             ctypes.byref(o), ctypes.byref(p)) != 0:
        raise ValueError("shape has no output")
    return o.value, p.value


def binarize(x: np.ndarray) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    s = np.empty(x.shape, np.int8)
    lib().oracle_binarize(x.reshape(-1), x.size, s.reshape(-1))
    return s


def pack(s: np.ndarray) -> np.ndarray:
    """+-1 int8 [..., C] -> uint32 [..., ceil(C/32)]."""
    s = np.ascontiguousarray(s, dtype=np.int8)
    c = s.shape[-1]
    rows = s.size // c if c else 0
    out = np.empty(s.shape[:-1] + ((c + 31) // 32,), np.uint32)
    lib().oracle_pack(s.reshape(-1), rows, c, out.reshape(-1))
    return out


def unpack(words: np.ndarray, channels: int) -> np.ndarray:
    """uint32 [..., ceil(C/32)] -> +-1 int8 [..., C]."""
    words = np.ascontiguousarray(words, dtype=np.uint32)
    rows = words.size // words.shape[-1]
    s = np.empty(words.shape[:-1] + (channels,), np.int8)
    lib().oracle_unpack(words.reshape(-1), rows, channels, s.reshape(-1))
    return s


def conv_dot(a: np.ndarray, w: np.ndarray, stride=1, padding: str = "same",
             pad_value: int = 1) -> np.ndarray:
    """+-1 cross-correlation: int8 NHWC x int8 OHWI -> int32 NHWC.

    pad_value 1 = one-padding (padded bits read as +1), 0 = zero-padding."""
    a = np.ascontiguousarray(a, dtype=np.int8)
    w = np.ascontiguousarray(w, dtype=np.int8)
    n, h, wd, c = a.shape
    cout, kh, kw, c2 = w.shape
    assert c == c2
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    oh, _ = out_size(h, kh, sh, padding)
    ow, _ = out_size(wd, kw, sw, padding)
    dot = np.empty((n, oh, ow, cout), np.int32)
    rc = lib().oracle_conv_dot_padded(a.reshape(-1), n, h, wd, c, w.reshape(-1), cout, kh, kw,
                                      sh, sw, 1 if padding == "same" else 0, int(pad_value),
                                      dot.reshape(-1))
    if rc != 0:
        raise ValueError("shape has no output")
    return dot


def clamp(dot: np.ndarray, lo: int, hi: int) -> np.ndarray:
    dot = np.ascontiguousarray(dot, dtype=np.int32)
    out = np.empty_like(dot)
    lib().oracle_clamp(dot.reshape(-1), dot.size, int(lo), int(hi), out.reshape(-1))
    return out


def out_float(c: np.ndarray, mult: Optional[np.ndarray], bias: Optional[np.ndarray]) -> np.ndarray:
    c = np.ascontiguousarray(c, dtype=np.int32)
    cout = c.shape[-1]
    m = c.size // cout
    y = np.empty(c.shape, np.float64)
    mu = None if mult is None else np.ascontiguousarray(mult, dtype=np.float32)
    bi = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    lib().oracle_out_float(c.reshape(-1), m, cout,
                           None if mu is None else mu.ctypes.data,
                           None if bi is None else bi.ctypes.data, y.reshape(-1))
    return y


def out_bits(c: np.ndarray, thr: np.ndarray) -> np.ndarray:
    c = np.ascontiguousarray(c, dtype=np.int32)
    cout = c.shape[-1]
    m = c.size // cout
    thr = np.ascontiguousarray(thr, dtype=np.float32)
    words = np.empty(c.shape[:-1] + ((cout + 31) // 32,), np.uint32)
    lib().oracle_out_bits(c.reshape(-1), m, cout, thr, words.reshape(-1))
    return words


INT32_MIN = -(2 ** 31)
INT32_MAX = 2 ** 31 - 1


def bmaxpool(a: np.ndarray, kh: int, kw: int, stride=1, padding: str = "valid") -> np.ndarray:
    """Max pooling of +-1 int8 NHWC values (padded locations ignored)."""
    a = np.ascontiguousarray(a, dtype=np.int8)
    n, h, wd, c = a.shape
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    oh, _ = out_size(h, kh, sh, padding)
    ow, _ = out_size(wd, kw, sw, padding)
    out = np.empty((n, oh, ow, c), np.int8)
    if lib().oracle_bmaxpool(a.reshape(-1), n, h, wd, c, kh, kw, sh, sw,
                             1 if padding == "same" else 0, out.reshape(-1)) != 0:
        raise ValueError("shape has no output")
    return out


def sign_of_affine(c: np.ndarray, mult: float, bias: float) -> np.ndarray:
    """1 where fmaf(float(c), mult, bias) < 0, else 0 (exact sign)."""
    c = np.ascontiguousarray(c, dtype=np.int32)
    bits = np.empty(c.shape, np.uint8)
    lib().oracle_sign_of_affine(c.reshape(-1), c.size, float(np.float32(mult)),
                                float(np.float32(bias)), bits.reshape(-1))
    return bits


def bconv2d(a: np.ndarray, w: np.ndarray, *, stride=1, padding="same",
            clamp_range=(INT32_MIN, INT32_MAX), out="float",
            mult=None, bias=None, thr=None, pad_value=1, flip=None) -> np.ndarray:
    """The whole operator on +-1 activations a (int8 NHWC) and +-1 filters w.

    out="int32"     -> clamped accumulator, int32 NHWC
    out="float"     -> fp64 NHWC values of clamp(dot) * mult + bias
    out="bitpacked" -> uint32 NHWC words (bit 1 iff clamp(dot) < thr, XOR flip[co]
                       when a per-channel 0/1 `flip` is given)
    pad_value        -> 1 one-padding, 0 zero-padding
    """
    dot = conv_dot(a, w, stride, padding, pad_value)
    lo, hi = clamp_range
    c = clamp(dot, lo, hi)
    if out == "int32":
        return c
    if out == "float":
        return out_float(c, mult, bias)
    if out == "bitpacked":
        words = out_bits(c, thr)
        if flip is not None:
            flip = np.asarray(flip, dtype=np.uint8)
            cout = c.shape[-1]
            signs = unpack(words, cout)
            signs = np.where(flip.astype(bool), -signs, signs).astype(np.int8)
            words = pack(signs)
        return words
    raise ValueError(out)
