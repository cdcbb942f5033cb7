"""MI355X (gfx950) bitpacked binary convolution: Python binding of include/lce.h.

Argument marshalling only: every step of the operator runs in the HIP
kernels of liblce.so.  torch supplies device memory and the current stream.
If the library is not built this module raises; there is no CPU fallback.

    bitpack(x)                        LceQuantize: float [..., C] -> int32 [..., ceil(C/32)]
    bconv2d(x_packed, w_packed, c_in) LceBConv2d with the fused output transform
    quantize_bconv2d(x, w_packed)     LceQuantize + LceBConv2d in one launch (float input)
    pad_correction(w_packed, c_in)    zero-padding correction table of a filter tensor
    fold_thresholds(m, b, k, clamp)   float transform + binarization -> thresholds, flip
    mfma_weights(w_packed, c_in)      filters widened to 4-bit +-1.0 for the matrix-core path
    bconv2d_mfma(x_packed, w_fp4, ..) LceBConv2d on the matrix cores (same result)
    bmaxpool2d(x_packed, channels)    LceBMaxPool2d: AND over each window of packed words
    dequantize(x_packed, channels)    LceDequantize: packed bits -> +-1.0 float32
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence, Tuple, Union

from . import build as _build

LCE_OK, LCE_EINVAL, LCE_EUNSUPPORTED, LCE_EALIGN, LCE_EHIP = 0, 1, 2, 3, 4
STATUS_NAMES = {0: "LCE_OK", 1: "LCE_EINVAL", 2: "LCE_EUNSUPPORTED", 3: "LCE_EALIGN",
                4: "LCE_EHIP"}
PADDING = {"valid": 0, "same": 1}
PAD_VALUE = {"one": 0, "zero": 1}
OUT_TYPE = {"float": 0, "bitpacked": 1, "int32": 2}
INT32_MIN = -(2 ** 31)
INT32_MAX = 2 ** 31 - 1

# Every symbol include/lce.h declares.
EXPORTS = ("lce_packed_words", "lce_bconv2d_out_shape", "lce_bitpack", "lce_bconv2d",
           "lce_bconv2d_pad_correction_size", "lce_bconv2d_pad_correction",
           "lce_fold_thresholds", "lce_bmaxpool2d_out_shape", "lce_bmaxpool2d",
           "lce_dequantize", "lce_bconv2d_mfma_weights_size", "lce_bconv2d_mfma_weights",
           "lce_bconv2d_mfma", "lce_quantize_bconv2d", "lce_quantize_bconv2d_mfma",
           "lce_set_tuning", "lce_get_tuning",
           "lce_last_error")

# lce_tuning_key values, by the names tuning() takes.
TUNING_KEYS = {"xor_nb": 0, "xor_ks": 1, "mfma_schedule": 2, "mfma_fs_ks": 3, "mfma_fs_s": 4,
               "mfma_fs_wpc": 5, "mfma_fs_pad": 6, "mfma_packed": 7, "mfma_tile_m": 8,
               "mfma_tile_n": 9, "mfma_fs_window": 10}
MFMA_SCHEDULES = {"auto": 0, "fs": 1, "ksplit": 2, "pixel": 3}


class Desc(ctypes.Structure):
    """lce_bconv2d_desc: fourteen int32 fields, in header order."""
    _fields_ = [(name, ctypes.c_int32) for name in (
        "n", "h", "w", "c_in", "c_out", "kh", "kw", "stride_h", "stride_w",
        "padding", "pad_value", "clamp_min", "clamp_max", "out_type")]


class PoolDesc(ctypes.Structure):
    """lce_bmaxpool2d_desc: nine int32 fields, in header order."""
    _fields_ = [(name, ctypes.c_int32) for name in (
        "n", "h", "w", "channels", "kh", "kw", "stride_h", "stride_w", "padding")]


class LceError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded liblce.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            raise ImportError(f"{_build.LIB} is not built; run paper_2011_09398_amd.build.build()")
        L = ctypes.CDLL(_build.LIB)
        vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        L.lce_packed_words.argtypes = [i32]
        L.lce_packed_words.restype = i32
        L.lce_bconv2d_out_shape.argtypes = [ctypes.POINTER(Desc), ctypes.POINTER(i32),
                                            ctypes.POINTER(i32)]
        L.lce_bconv2d_out_shape.restype = ctypes.c_int
        L.lce_bitpack.argtypes = [vp, vp, i64, i32, vp]
        L.lce_bitpack.restype = ctypes.c_int
        L.lce_bconv2d.argtypes = [ctypes.POINTER(Desc), vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.lce_bconv2d.restype = ctypes.c_int
        L.lce_bconv2d_pad_correction_size.argtypes = [ctypes.POINTER(Desc),
                                                       ctypes.POINTER(i64)]
        L.lce_bconv2d_pad_correction_size.restype = ctypes.c_int
        L.lce_bconv2d_pad_correction.argtypes = [ctypes.POINTER(Desc), vp, vp, vp]
        L.lce_bconv2d_pad_correction.restype = ctypes.c_int
        L.lce_fold_thresholds.argtypes = [vp, vp, i32, i32, i32, i32, vp, vp]
        L.lce_fold_thresholds.restype = ctypes.c_int
        L.lce_bmaxpool2d_out_shape.argtypes = [ctypes.POINTER(PoolDesc), ctypes.POINTER(i32),
                                               ctypes.POINTER(i32)]
        L.lce_bmaxpool2d_out_shape.restype = ctypes.c_int
        L.lce_bmaxpool2d.argtypes = [ctypes.POINTER(PoolDesc), vp, vp, vp]
        L.lce_bmaxpool2d.restype = ctypes.c_int
        L.lce_dequantize.argtypes = [vp, vp, i64, i32, vp]
        L.lce_dequantize.restype = ctypes.c_int
        L.lce_bconv2d_mfma_weights_size.argtypes = [ctypes.POINTER(Desc), ctypes.POINTER(i64)]
        L.lce_bconv2d_mfma_weights_size.restype = ctypes.c_int
        L.lce_bconv2d_mfma_weights.argtypes = [ctypes.POINTER(Desc), vp, vp, vp]
        L.lce_bconv2d_mfma_weights.restype = ctypes.c_int
        L.lce_bconv2d_mfma.argtypes = [ctypes.POINTER(Desc), vp, vp, vp, vp, vp, vp, vp, vp]
        L.lce_bconv2d_mfma.restype = ctypes.c_int
        L.lce_quantize_bconv2d.argtypes = [ctypes.POINTER(Desc), vp, vp, vp, vp, vp, vp, vp, vp]
        L.lce_quantize_bconv2d.restype = ctypes.c_int
        L.lce_quantize_bconv2d_mfma.argtypes = [ctypes.POINTER(Desc), vp, vp, vp, vp, vp, vp,
                                                vp, vp]
        L.lce_quantize_bconv2d_mfma.restype = ctypes.c_int
        L.lce_set_tuning.argtypes = [i32, i32]
        L.lce_set_tuning.restype = ctypes.c_int
        L.lce_get_tuning.argtypes = [i32]
        L.lce_get_tuning.restype = i32
        L.lce_last_error.argtypes = []
        L.lce_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def last_error() -> str:
    return lib().lce_last_error().decode()


def _check(status: int) -> None:
    if status != LCE_OK:
        raise LceError(status, last_error())


def set_tuning(**overrides) -> None:
    """Schedule overrides (lce_set_tuning), e.g. set_tuning(xor_nb=2,
    mfma_schedule="fs"); 0 restores the automatic choice.  Process-wide."""
    for name, value in overrides.items():
        if name not in TUNING_KEYS:
            raise KeyError(f"unknown tuning key {name!r}")
        if name == "mfma_schedule" and isinstance(value, str):
            value = MFMA_SCHEDULES[value]
        _check(lib().lce_set_tuning(TUNING_KEYS[name], int(value)))


def get_tuning(name: str) -> int:
    return int(lib().lce_get_tuning(TUNING_KEYS[name]))


class tuning:
    """Context manager: the given overrides inside, every key back to
    automatic (0) on exit."""

    def __init__(self, **overrides):
        self.overrides = overrides

    def __enter__(self):
        set_tuning(**self.overrides)
        return self

    def __exit__(self, *exc):
        set_tuning(**{k: 0 for k in TUNING_KEYS})
        return False


def packed_words(channels: int) -> int:
    return int(lib().lce_packed_words(int(channels)))


def make_desc(n, h, w, c_in, c_out, kh, kw, stride=1, padding="same", pad_value="one",
              clamp: Optional[Tuple[int, int]] = None, out_type="float") -> Desc:
    sh, sw = (stride, stride) if isinstance(stride, int) else tuple(stride)
    lo, hi = (INT32_MIN, INT32_MAX) if clamp is None else clamp
    return Desc(n, h, w, c_in, c_out, kh, kw, sh, sw,
                PADDING[padding] if isinstance(padding, str) else padding,
                PAD_VALUE[pad_value] if isinstance(pad_value, str) else pad_value,
                lo, hi, OUT_TYPE[out_type] if isinstance(out_type, str) else out_type)


def out_shape(desc: Desc) -> Tuple[int, int]:
    oh, ow = ctypes.c_int32(), ctypes.c_int32()
    _check(lib().lce_bconv2d_out_shape(ctypes.byref(desc), ctypes.byref(oh), ctypes.byref(ow)))
    return oh.value, ow.value


def _stream_handle(t) -> int:
    import torch
    return torch.cuda.current_stream(t.device).cuda_stream


def _require(t, dtype, name):
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device tensor, got {t.device}")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def bitpack(x, out=None):
    """LceQuantize on a float32 device tensor [..., C] -> int32 [..., ceil(C/32)]."""
    import torch
    _require(x, torch.float32, "x")
    c = x.shape[-1]
    cw = packed_words(c)
    rows = x.numel() // c if c else 0
    if out is None:
        out = torch.empty(tuple(x.shape[:-1]) + (cw,), dtype=torch.int32, device=x.device)
    else:
        _require(out, torch.int32, "out")
        if out.numel() != rows * cw:
            raise ValueError("out has the wrong size")
    _check(lib().lce_bitpack(x.data_ptr(), out.data_ptr(), rows, c, _stream_handle(x)))
    return out


def _filter_desc(w_packed, c_in, padding="same", pad_value="zero", stride=1) -> Desc:
    """A descriptor for filter-only calls (the input dims do not matter)."""
    cout, kh, kw, _ = w_packed.shape
    return make_desc(1, kh, kw, c_in, cout, kh, kw, stride, padding, pad_value, None, "int32")


def pad_correction_size(desc: Desc) -> int:
    n = ctypes.c_int64()
    _check(lib().lce_bconv2d_pad_correction_size(ctypes.byref(desc), ctypes.byref(n)))
    return n.value


def pad_correction(w_packed, c_in: int, out=None):
    """Zero-padding correction table of w_packed: int32 [(KH+1)*KW*(KW+1)/2, Cout]."""
    import torch
    _require(w_packed, torch.int32, "w_packed")
    cout, kh, kw, cw = w_packed.shape
    if cw != packed_words(c_in):
        raise ValueError(f"packed channel words {cw} do not match c_in={c_in}")
    desc = _filter_desc(w_packed, c_in)
    size = pad_correction_size(desc)
    if out is None:
        out = torch.empty(((kh + 1) * (kw * (kw + 1) // 2), cout), dtype=torch.int32,
                          device=w_packed.device)
    else:
        _require(out, torch.int32, "out")
        if out.numel() != size:
            raise ValueError(f"out must hold {size} elements")
    _check(lib().lce_bconv2d_pad_correction(ctypes.byref(desc), w_packed.data_ptr(),
                                            out.data_ptr(), _stream_handle(w_packed)))
    return out


def fold_thresholds(multiplier, bias, c_out: int, k: int,
                    clamp: Optional[Tuple[int, int]] = None):
    """Host-side fold of (multiplier, bias) into (thresholds float32 [c_out],
    flip int32 [ceil(c_out/32)]), both numpy arrays.  multiplier/bias: array-likes
    of c_out floats, or None for 1 / 0."""
    import numpy as np
    lo, hi = (INT32_MIN, INT32_MAX) if clamp is None else clamp
    arrs = []
    for a, name in ((multiplier, "multiplier"), (bias, "bias")):
        if a is None:
            arrs.append(None)
        else:
            a = np.ascontiguousarray(a, dtype=np.float32)
            if a.size != c_out:
                raise ValueError(f"{name} must have {c_out} elements")
            arrs.append(a)
    thr = np.empty(c_out, dtype=np.float32)
    flip = np.empty(max(packed_words(c_out), 0), dtype=np.int32)
    ptr = lambda a: None if a is None else a.ctypes.data
    _check(lib().lce_fold_thresholds(ptr(arrs[0]), ptr(arrs[1]), int(c_out), int(k), int(lo),
                                     int(hi), thr.ctypes.data, flip.ctypes.data))
    return thr, flip


def _epilogue_args(cout, kh, kw, multiplier, bias, thresholds, flip, pad_correction=None):
    """Check the optional per-channel tensors of a convolution; their pointers."""
    import torch
    ptrs = []
    for t, name, dtype, numel in ((multiplier, "multiplier", torch.float32, cout),
                                  (bias, "bias", torch.float32, cout),
                                  (thresholds, "thresholds", torch.float32, cout),
                                  (flip, "flip", torch.int32, packed_words(cout)),
                                  (pad_correction, "pad_correction", torch.int32,
                                   (kh + 1) * (kw * (kw + 1) // 2) * cout)):
        if t is None:
            ptrs.append(None)
        else:
            _require(t, dtype, name)
            if t.numel() != numel:
                raise ValueError(f"{name} must have {numel} elements")
            ptrs.append(t.data_ptr())
    return ptrs


def _conv_out(out, out_type, n, oh, ow, cout, device):
    """Check a caller's output tensor, or allocate one."""
    import torch
    oc = packed_words(cout) if out_type == "bitpacked" else cout
    dt = torch.float32 if out_type == "float" else torch.int32
    if out is None:
        return torch.empty((n, oh, ow, oc), dtype=dt, device=device)
    _require(out, dt, "out")
    if out.numel() != n * oh * ow * oc:
        raise ValueError(f"out must hold {n}x{oh}x{ow}x{oc} elements")
    return out


def bconv2d(x_packed, w_packed, c_in: int, *, stride: Union[int, Sequence[int]] = 1,
            padding: str = "same", pad_value: str = "one",
            clamp: Optional[Tuple[int, int]] = None, out_type: str = "float",
            multiplier=None, bias=None, thresholds=None, flip=None, pad_correction=None,
            out=None):
    """LceBConv2d: x_packed int32 [N,H,W,Cw], w_packed int32 [Cout,KH,KW,Cw].

    out_type "float" -> float32 [N,OH,OW,Cout]; "bitpacked" -> int32
    [N,OH,OW,ceil(Cout/32)]; "int32" -> the clamped accumulator [N,OH,OW,Cout].
    flip: int32 [ceil(Cout/32)] direction bits (bitpacked output).
    pad_correction: the table of pad_correction(w_packed, c_in), needed by
    pad_value "zero" when the geometry pads.
    """
    import torch
    _require(x_packed, torch.int32, "x_packed")
    _require(w_packed, torch.int32, "w_packed")
    n, h, w, cw = x_packed.shape
    cout, kh, kw, cw2 = w_packed.shape
    if cw != packed_words(c_in) or cw2 != cw:
        raise ValueError(f"packed channel words {cw}/{cw2} do not match c_in={c_in}")
    desc = make_desc(n, h, w, c_in, cout, kh, kw, stride, padding, pad_value, clamp, out_type)
    oh, ow = out_shape(desc)
    ptrs = _epilogue_args(cout, kh, kw, multiplier, bias, thresholds, flip, pad_correction)
    out = _conv_out(out, out_type, n, oh, ow, cout, x_packed.device)
    _check(lib().lce_bconv2d(ctypes.byref(desc), x_packed.data_ptr(), w_packed.data_ptr(),
                             *ptrs, out.data_ptr(), _stream_handle(x_packed)))
    return out


def quantize_bconv2d(x, w_packed, *, stride: Union[int, Sequence[int]] = 1,
                     padding: str = "same", clamp: Optional[Tuple[int, int]] = None,
                     out_type: str = "float", multiplier=None, bias=None, thresholds=None,
                     flip=None, out=None):
    """LceQuantize + LceBConv2d in one launch: x float32 [N,H,W,C_in] (C_in a
    multiple of 32, 16-byte aligned), w_packed int32 [Cout,KH,KW,C_in/32].

    The result equals bconv2d(bitpack(x), w_packed, C_in, ...) with one
    padding.  Shapes the fused kernel does not cover raise LceError with
    status LCE_EUNSUPPORTED (nothing is launched); run bitpack and bconv2d.
    """
    import torch
    _require(x, torch.float32, "x")
    _require(w_packed, torch.int32, "w_packed")
    n, h, w, c_in = x.shape
    cout, kh, kw, cw = w_packed.shape
    if cw != packed_words(c_in):
        raise ValueError(f"packed channel words {cw} do not match c_in={c_in}")
    desc = make_desc(n, h, w, c_in, cout, kh, kw, stride, padding, "one", clamp, out_type)
    oh, ow = out_shape(desc)
    ptrs = _epilogue_args(cout, kh, kw, multiplier, bias, thresholds, flip)[:4]
    out = _conv_out(out, out_type, n, oh, ow, cout, x.device)
    _check(lib().lce_quantize_bconv2d(ctypes.byref(desc), x.data_ptr(), w_packed.data_ptr(),
                                      *ptrs, out.data_ptr(), _stream_handle(x)))
    return out


def make_pool_desc(n, h, w, channels, kernel=2, stride=None, padding="valid") -> PoolDesc:
    kh, kw = (kernel, kernel) if isinstance(kernel, int) else tuple(kernel)
    if stride is None:
        stride = (kh, kw)
    sh, sw = (stride, stride) if isinstance(stride, int) else tuple(stride)
    return PoolDesc(n, h, w, channels, kh, kw, sh, sw,
                    PADDING[padding] if isinstance(padding, str) else padding)


def pool_out_shape(desc: PoolDesc) -> Tuple[int, int]:
    oh, ow = ctypes.c_int32(), ctypes.c_int32()
    _check(lib().lce_bmaxpool2d_out_shape(ctypes.byref(desc), ctypes.byref(oh),
                                          ctypes.byref(ow)))
    return oh.value, ow.value


def bmaxpool2d(x_packed, channels: int, kernel=2, stride=None, padding: str = "valid",
               out=None):
    """LceBMaxPool2d on int32 [N,H,W,ceil(C/32)] -> int32 [N,OH,OW,ceil(C/32)]
    (stride defaults to the window size, as in TensorFlow)."""
    import torch
    _require(x_packed, torch.int32, "x_packed")
    n, h, w, cw = x_packed.shape
    if cw != packed_words(channels):
        raise ValueError(f"packed words {cw} do not match channels={channels}")
    desc = make_pool_desc(n, h, w, channels, kernel, stride, padding)
    oh, ow = pool_out_shape(desc)
    if out is None:
        out = torch.empty((n, oh, ow, cw), dtype=torch.int32, device=x_packed.device)
    else:
        _require(out, torch.int32, "out")
        if out.numel() != n * oh * ow * cw:
            raise ValueError(f"out must hold {n}x{oh}x{ow}x{cw} words")
    _check(lib().lce_bmaxpool2d(ctypes.byref(desc), x_packed.data_ptr(), out.data_ptr(),
                                _stream_handle(x_packed)))
    return out


def dequantize(x_packed, channels: int, out=None):
    """LceDequantize: int32 [..., ceil(C/32)] -> float32 [..., C] of +-1.0."""
    import torch
    _require(x_packed, torch.int32, "x_packed")
    cw = x_packed.shape[-1]
    if cw != packed_words(channels):
        raise ValueError(f"packed words {cw} do not match channels={channels}")
    rows = x_packed.numel() // cw if cw else 0
    if out is None:
        out = torch.empty(tuple(x_packed.shape[:-1]) + (channels,), dtype=torch.float32,
                          device=x_packed.device)
    else:
        _require(out, torch.float32, "out")
        if out.numel() != rows * channels:
            raise ValueError("out has the wrong size")
    _check(lib().lce_dequantize(x_packed.data_ptr(), out.data_ptr(), rows, channels,
                                _stream_handle(x_packed)))
    return out


def mfma_weights_size(desc: Desc) -> int:
    """Bytes of the widened filter buffer lce_bconv2d_mfma reads for `desc`."""
    n = ctypes.c_int64()
    _check(lib().lce_bconv2d_mfma_weights_size(ctypes.byref(desc), ctypes.byref(n)))
    return n.value


def mfma_weights(w_packed, c_in: int, out=None):
    """Widened filters for bconv2d_mfma: uint8 device buffer (16-byte aligned)."""
    import torch
    _require(w_packed, torch.int32, "w_packed")
    cout, kh, kw, cw = w_packed.shape
    if cw != packed_words(c_in):
        raise ValueError(f"packed channel words {cw} do not match c_in={c_in}")
    desc = _filter_desc(w_packed, c_in)
    n = ctypes.c_int64()
    _check(lib().lce_bconv2d_mfma_weights_size(ctypes.byref(desc), ctypes.byref(n)))
    if out is None:
        out = torch.empty(n.value, dtype=torch.uint8, device=w_packed.device)
    elif out.numel() * out.element_size() < n.value:
        raise ValueError(f"out must hold {n.value} bytes")
    _check(lib().lce_bconv2d_mfma_weights(ctypes.byref(desc), w_packed.data_ptr(),
                                          out.data_ptr(), _stream_handle(w_packed)))
    return out


def _mfma_conv(fn, x, x_float: bool, w_fp4, c_in: int, c_out: int, kernel, stride, padding,
               pad_value, clamp, out_type, multiplier, bias, thresholds, flip, out):
    """Shared marshalling of the two matrix-core entry points (packed or
    float input); returns the output tensor."""
    import torch
    if x_float:
        _require(x, torch.float32, "x")
        n, h, w, c = x.shape
        if c != c_in:
            raise ValueError(f"x has {c} channels, c_in={c_in}")
    else:
        _require(x, torch.int32, "x_packed")
        n, h, w, cw = x.shape
        if cw != packed_words(c_in):
            raise ValueError(f"packed channel words {cw} do not match c_in={c_in}")
    if not isinstance(w_fp4, torch.Tensor) or w_fp4.device.type != "cuda":
        raise TypeError("w_fp4 must be a device tensor")
    if not w_fp4.is_contiguous():
        raise ValueError("w_fp4 must be contiguous")
    kh, kw = (kernel, kernel) if isinstance(kernel, int) else tuple(kernel)
    desc = make_desc(n, h, w, c_in, c_out, kh, kw, stride, padding, pad_value, clamp, out_type)
    oh, ow = out_shape(desc)
    need = mfma_weights_size(desc)
    if w_fp4.numel() * w_fp4.element_size() < need:
        raise ValueError(f"w_fp4 holds {w_fp4.numel() * w_fp4.element_size()} bytes; these "
                         f"filters widen to {need} (mfma_weights of the same c_in, c_out "
                         f"and kernel)")
    ptrs = []
    for t, name, dtype, numel in ((multiplier, "multiplier", torch.float32, c_out),
                                  (bias, "bias", torch.float32, c_out),
                                  (thresholds, "thresholds", torch.float32, c_out),
                                  (flip, "flip", torch.int32, packed_words(c_out))):
        if t is None:
            ptrs.append(None)
        else:
            _require(t, dtype, name)
            if t.numel() != numel:
                raise ValueError(f"{name} must have {numel} elements")
            ptrs.append(t.data_ptr())
    oc = packed_words(c_out) if out_type == "bitpacked" else c_out
    dt = torch.float32 if out_type == "float" else torch.int32
    if out is None:
        out = torch.empty((n, oh, ow, oc), dtype=dt, device=x.device)
    else:
        _require(out, dt, "out")
        if out.numel() != n * oh * ow * oc:
            raise ValueError(f"out must hold {n}x{oh}x{ow}x{oc} elements")
    _check(fn(ctypes.byref(desc), x.data_ptr(), w_fp4.data_ptr(), *ptrs, out.data_ptr(),
              _stream_handle(x)))
    return out


def bconv2d_mfma(x_packed, w_fp4, c_in: int, c_out: int, kernel, *, stride=1,
                 padding: str = "same", pad_value: str = "one",
                 clamp: Optional[Tuple[int, int]] = None, out_type: str = "float",
                 multiplier=None, bias=None, thresholds=None, flip=None, out=None):
    """LceBConv2d on the matrix cores: x_packed int32 [N,H,W,Cw], w_fp4 from
    mfma_weights(); kernel = (KH, KW) or an int.  Output as bconv2d."""
    return _mfma_conv(lib().lce_bconv2d_mfma, x_packed, False, w_fp4, c_in, c_out, kernel,
                      stride, padding, pad_value, clamp, out_type, multiplier, bias,
                      thresholds, flip, out)


def quantize_bconv2d_mfma(x, w_fp4, c_out: int, kernel, *, stride=1, padding: str = "same",
                          pad_value: str = "one", clamp: Optional[Tuple[int, int]] = None,
                          out_type: str = "float", multiplier=None, bias=None,
                          thresholds=None, flip=None, out=None):
    """LceQuantize + LceBConv2d on the matrix cores in one launch: x float32
    [N,H,W,C_in] (C_in a multiple of 32, 16-byte aligned), w_fp4 from
    mfma_weights().  The result equals bconv2d_mfma(bitpack(x), ...).  Shapes
    the filter-stationary schedule does not take raise LceError with status
    LCE_EUNSUPPORTED (nothing is launched); run bitpack and bconv2d_mfma."""
    return _mfma_conv(lib().lce_quantize_bconv2d_mfma, x, True, w_fp4, x.shape[-1], c_out,
                      kernel, stride, padding, pad_value, clamp, out_type, multiplier, bias,
                      thresholds, flip, out)


class PreparedBConv2dMfma:
    """A bconv2d_mfma call marshalled once (see PreparedBConv2d)."""

    def __init__(self, x_packed, w_fp4, c_in, c_out, kernel, out, *, stride=1, padding="same",
                 pad_value="one", clamp=None, out_type="float", multiplier=None, bias=None,
                 thresholds=None, flip=None):
        bconv2d_mfma(x_packed, w_fp4, c_in, c_out, kernel, stride=stride, padding=padding,
                     pad_value=pad_value, clamp=clamp, out_type=out_type,
                     multiplier=multiplier, bias=bias, thresholds=thresholds, flip=flip,
                     out=out)
        n, h, w, _ = x_packed.shape
        kh, kw = (kernel, kernel) if isinstance(kernel, int) else tuple(kernel)
        self.desc = make_desc(n, h, w, c_in, c_out, kh, kw, stride, padding, pad_value, clamp,
                              out_type)
        self._desc_ref = ctypes.byref(self.desc)
        ptr = lambda t: None if t is None else t.data_ptr()
        self.args = (x_packed.data_ptr(), w_fp4.data_ptr(), ptr(multiplier), ptr(bias),
                     ptr(thresholds), ptr(flip), out.data_ptr())
        self.keep = (x_packed, w_fp4, multiplier, bias, thresholds, flip, out)
        self._fn = lib().lce_bconv2d_mfma

    def __call__(self, stream=None):
        st = self._fn(self._desc_ref, *self.args, _current_stream() if stream is None else stream)
        if st != LCE_OK:
            raise LceError(st, last_error())


def _current_stream():
    import torch
    return torch.cuda.current_stream().cuda_stream


class PreparedBConv2d:
    """A bconv2d call with its descriptor and pointers marshalled once.

    Calling it enqueues the convolution on `stream` (default: torch's current
    stream at call time, so it can be captured in a graph) with no Python-side
    validation; the C ABI still validates.  The tensors must outlive it.
    """

    def __init__(self, x_packed, w_packed, c_in, out, *, stride=1, padding="same",
                 pad_value="one", clamp=None, out_type="float", multiplier=None, bias=None,
                 thresholds=None, flip=None, pad_correction=None):
        # one eager call validates shapes/dtypes and fills `out`
        bconv2d(x_packed, w_packed, c_in, stride=stride, padding=padding, pad_value=pad_value,
                clamp=clamp, out_type=out_type, multiplier=multiplier, bias=bias,
                thresholds=thresholds, flip=flip, pad_correction=pad_correction, out=out)
        n, h, w, _ = x_packed.shape
        cout, kh, kw, _ = w_packed.shape
        self.desc = make_desc(n, h, w, c_in, cout, kh, kw, stride, padding, pad_value, clamp,
                              out_type)
        self._desc_ref = ctypes.byref(self.desc)
        ptr = lambda t: None if t is None else t.data_ptr()
        self.args = (x_packed.data_ptr(), w_packed.data_ptr(), ptr(multiplier), ptr(bias),
                     ptr(thresholds), ptr(flip), ptr(pad_correction), out.data_ptr())
        self.keep = (x_packed, w_packed, multiplier, bias, thresholds, flip, pad_correction, out)
        self._fn = lib().lce_bconv2d

    def __call__(self, stream=None):
        st = self._fn(self._desc_ref, *self.args, _current_stream() if stream is None else stream)
        if st != LCE_OK:
            raise LceError(st, last_error())


class PreparedQuantBConv2dMfma:
    """A quantize_bconv2d_mfma call marshalled once (see PreparedBConv2d)."""

    def __init__(self, x, w_fp4, c_out, kernel, out, *, stride=1, padding="same",
                 pad_value="one", clamp=None, out_type="float", multiplier=None, bias=None,
                 thresholds=None, flip=None):
        quantize_bconv2d_mfma(x, w_fp4, c_out, kernel, stride=stride, padding=padding,
                              pad_value=pad_value, clamp=clamp, out_type=out_type,
                              multiplier=multiplier, bias=bias, thresholds=thresholds,
                              flip=flip, out=out)
        n, h, w, c_in = x.shape
        kh, kw = (kernel, kernel) if isinstance(kernel, int) else tuple(kernel)
        self.desc = make_desc(n, h, w, c_in, c_out, kh, kw, stride, padding, pad_value, clamp,
                              out_type)
        self._desc_ref = ctypes.byref(self.desc)
        ptr = lambda t: None if t is None else t.data_ptr()
        self.args = (x.data_ptr(), w_fp4.data_ptr(), ptr(multiplier), ptr(bias),
                     ptr(thresholds), ptr(flip), out.data_ptr())
        self.keep = (x, w_fp4, multiplier, bias, thresholds, flip, out)
        self._fn = lib().lce_quantize_bconv2d_mfma

    def __call__(self, stream=None):
        st = self._fn(self._desc_ref, *self.args, _current_stream() if stream is None else stream)
        if st != LCE_OK:
            raise LceError(st, last_error())


class PreparedQuantBConv2d:
    """A quantize_bconv2d call marshalled once (see PreparedBConv2d)."""

    def __init__(self, x, w_packed, out, *, stride=1, padding="same", clamp=None,
                 out_type="float", multiplier=None, bias=None, thresholds=None, flip=None):
        quantize_bconv2d(x, w_packed, stride=stride, padding=padding, clamp=clamp,
                         out_type=out_type, multiplier=multiplier, bias=bias,
                         thresholds=thresholds, flip=flip, out=out)
        n, h, w, c_in = x.shape
        cout, kh, kw, _ = w_packed.shape
        self.desc = make_desc(n, h, w, c_in, cout, kh, kw, stride, padding, "one", clamp,
                              out_type)
        self._desc_ref = ctypes.byref(self.desc)
        ptr = lambda t: None if t is None else t.data_ptr()
        self.args = (x.data_ptr(), w_packed.data_ptr(), ptr(multiplier), ptr(bias),
                     ptr(thresholds), ptr(flip), out.data_ptr())
        self.keep = (x, w_packed, multiplier, bias, thresholds, flip, out)
        self._fn = lib().lce_quantize_bconv2d

    def __call__(self, stream=None):
        st = self._fn(self._desc_ref, *self.args, _current_stream() if stream is None else stream)
        if st != LCE_OK:
            raise LceError(st, last_error())


class PreparedBitpack:
    """A bitpack call marshalled once (see PreparedBConv2d)."""

    def __init__(self, x, out):
        bitpack(x, out=out)
        c = x.shape[-1]
        self.args = (x.data_ptr(), out.data_ptr(), x.numel() // c, c)
        self.keep = (x, out)
        self._fn = lib().lce_bitpack

    def __call__(self, stream=None):
        st = self._fn(*self.args, _current_stream() if stream is None else stream)
        if st != LCE_OK:
            raise LceError(st, last_error())
