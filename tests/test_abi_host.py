"""Host side of the C ABI, on the CPU: exports, geometry, validation errors.

Every call here fails validation (or needs no device work), so nothing is
ever launched; fake non-null pointers are plain integers.
"""
import ctypes
import os
import re
import subprocess
from itertools import product

import pytest

import oracle
import paper_2011_09398_amd as lce
from paper_2011_09398_amd import build as lce_build
from tests.conftest import ROOT

HEADER = os.path.join(ROOT, "include", "lce.h")
P = 0x10000          # a fake, suitably aligned device pointer (never dereferenced)


@pytest.fixture(scope="module", autouse=True)
def built():
    if lce_build.is_stale():
        lce_build.build()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lce_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_binding_exports():
    assert declared_functions() == sorted(lce.EXPORTS)


def test_library_exports_every_declared_symbol():
    L = lce.lib()
    for name in declared_functions():
        assert hasattr(L, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", lce_build.LIB], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (lce_\w+)", out))
    assert set(declared_functions()) <= exported


def test_desc_layout_matches_header():
    # 14 int32 fields, no padding
    assert ctypes.sizeof(lce.Desc) == 14 * 4


def test_packed_words():
    assert [lce.packed_words(c) for c in (0, 1, 31, 32, 33, 64, 65, 512)] == \
        [0, 1, 1, 1, 2, 2, 3, 16]
    assert lce.packed_words(-1) == -1


def desc(**kw):
    base = dict(n=1, h=8, w=8, c_in=64, c_out=64, kh=3, kw=3, stride=1, padding="same",
                pad_value="one", clamp=None, out_type="float")
    base.update(kw)
    return lce.make_desc(**base)


def test_out_shape_matches_oracle_geometry():
    for h, k, s, pad in product((1, 2, 5, 7, 8, 28, 56), (1, 2, 3, 5), (1, 2, 3), ("same", "valid")):
        if pad == "valid" and h < k:
            continue
        d = desc(h=h, w=h + 1 if h + 1 >= k else h, kh=k, kw=k, stride=s, padding=pad)
        oh, ow = lce.out_shape(d)
        assert oh == oracle.out_size(h, k, s, pad)[0]
        assert ow == oracle.out_size(d.w, k, s, pad)[0]


def test_out_shape_config_examples():
    assert lce.out_shape(desc(h=56, w=56, stride=2)) == (28, 28)
    assert lce.out_shape(desc(h=7, w=7)) == (7, 7)
    assert lce.out_shape(desc(h=8, w=8, padding="valid")) == (6, 6)
    # geometry does not depend on the pad value
    assert lce.out_shape(desc(pad_value="zero")) == (8, 8)


@pytest.mark.parametrize("field,value", [
    ("n", 0), ("h", 0), ("w", -1), ("c_in", 0), ("c_out", 0), ("kh", 0), ("kw", 0),
    ("stride_h", 0), ("stride_w", -2), ("padding", 7), ("pad_value", 3), ("out_type", 9),
])
def test_out_shape_rejects_bad_field(field, value):
    d = desc()
    setattr(d, field, value)
    with pytest.raises(lce.LceError) as e:
        lce.out_shape(d)
    assert e.value.status == lce.LCE_EINVAL
    assert lce.last_error()


def call_bconv(d, x=P, w=P, m=None, b=None, t=P, flip=None, corr=None, out=P):
    return lce.lib().lce_bconv2d(ctypes.byref(d), x, w, m, b, t, flip, corr, out, None)


def test_bconv2d_validation_errors():
    L = lce.lib()
    assert L.lce_bconv2d(None, P, P, None, None, P, None, None, P, None) == lce.LCE_EINVAL
    assert "desc" in lce.last_error()
    assert call_bconv(desc(clamp=(5, 4))) == lce.LCE_EINVAL
    assert "clamp" in lce.last_error()
    assert call_bconv(desc(h=2, w=2, padding="valid")) == lce.LCE_EINVAL
    assert call_bconv(desc(), x=None) == lce.LCE_EINVAL
    assert call_bconv(desc(), w=None) == lce.LCE_EINVAL
    assert call_bconv(desc(), out=None) == lce.LCE_EINVAL
    assert call_bconv(desc(out_type="bitpacked"), t=None) == lce.LCE_EINVAL
    assert "threshold" in lce.last_error()
    # zero padding on a padded geometry needs the correction table
    assert call_bconv(desc(pad_value="zero")) == lce.LCE_EINVAL
    assert "pad_correction" in lce.last_error()
    assert call_bconv(desc(pad_value="zero"), corr=P + 2) == lce.LCE_EALIGN
    assert call_bconv(desc(out_type="bitpacked"), flip=P + 1) == lce.LCE_EALIGN
    # zero padding K limit (2^29): 3x3 x 2^26 input channels
    assert call_bconv(desc(pad_value="zero", c_in=2 ** 26, c_out=1, h=1, w=1),
                      corr=P) == lce.LCE_EINVAL
    assert call_bconv(desc(), x=P + 2) == lce.LCE_EALIGN
    assert call_bconv(desc(), out=P + 1) == lce.LCE_EALIGN
    assert call_bconv(desc(), m=P + 3) == lce.LCE_EALIGN
    # too large: 2^31 output pixels
    assert call_bconv(desc(n=2 ** 14, h=2 ** 9, w=2 ** 9, c_in=32, c_out=32)) == lce.LCE_EINVAL
    assert call_bconv(desc(c_out=(1 << 20) + 1, c_in=32, h=1, w=1)) == lce.LCE_EINVAL


def call_mfma(d, x=P, w=P, m=None, b=None, t=P, flip=None, out=P):
    return lce.lib().lce_bconv2d_mfma(ctypes.byref(d), x, w, m, b, t, flip, out, None)


def test_bconv2d_mfma_validation_errors():
    """Every refusal comes back before any device call (none is made here)."""
    assert call_mfma(desc(clamp=(5, 4))) == lce.LCE_EINVAL
    assert call_mfma(desc(), x=None) == lce.LCE_EINVAL
    assert call_mfma(desc(), w=None) == lce.LCE_EINVAL
    assert call_mfma(desc(), out=None) == lce.LCE_EINVAL
    assert call_mfma(desc(out_type="bitpacked"), t=None) == lce.LCE_EINVAL
    assert call_mfma(desc(), x=P + 2) == lce.LCE_EALIGN
    assert call_mfma(desc(), w=P + 4) == lce.LCE_EALIGN        # widened filters: 16 bytes
    assert call_mfma(desc(out_type="bitpacked"), flip=P + 1) == lce.LCE_EALIGN
    # exact fp32 dots need K < 2^24
    assert call_mfma(desc(c_in=2 ** 21, c_out=1, h=1, w=1)) == lce.LCE_EUNSUPPORTED
    assert "2^24" in lce.last_error()
    # the input (2^29 words = 2 GiB) and the widened filters are read as
    # buffers with 31-bit byte offsets
    assert call_mfma(desc(n=1, h=2 ** 14, w=2 ** 14, c_in=64, c_out=32,
                          out_type="bitpacked")) == lce.LCE_EUNSUPPORTED
    assert "2 GiB" in lce.last_error()
    assert call_mfma(desc(h=1, w=1, c_in=2 ** 18, c_out=2 ** 14, kh=1, kw=1,
                          out_type="bitpacked")) == lce.LCE_EUNSUPPORTED
    assert "2 GiB" in lce.last_error()


def call_quant_mfma(d, x=P, w=P, m=None, b=None, t=P, flip=None, out=P):
    return lce.lib().lce_quantize_bconv2d_mfma(ctypes.byref(d), x, w, m, b, t, flip, out, None)


def test_quantize_bconv2d_mfma_validation_errors():
    """The float-input matrix-core entry refuses before any device call:
    bad arguments, alignment (x and w_fp4 16 bytes), C_in not a multiple of
    32, K >= 2^24, a float input of 2 GiB or more, and a shape neither the
    filter-stationary nor the K-split schedule takes."""
    L = lce.lib()
    assert L.lce_quantize_bconv2d_mfma(None, P, P, None, None, P, None, P, None) == lce.LCE_EINVAL
    assert call_quant_mfma(desc(clamp=(5, 4))) == lce.LCE_EINVAL
    assert call_quant_mfma(desc(), x=None) == lce.LCE_EINVAL
    assert call_quant_mfma(desc(), w=None) == lce.LCE_EINVAL
    assert call_quant_mfma(desc(), out=None) == lce.LCE_EINVAL
    assert call_quant_mfma(desc(out_type="bitpacked"), t=None) == lce.LCE_EINVAL
    assert call_quant_mfma(desc(), x=P + 4) == lce.LCE_EALIGN      # float input: 16 bytes
    assert call_quant_mfma(desc(), w=P + 4) == lce.LCE_EALIGN
    assert call_quant_mfma(desc(out_type="bitpacked"), flip=P + 1) == lce.LCE_EALIGN
    assert call_quant_mfma(desc(c_in=48)) == lce.LCE_EUNSUPPORTED
    assert "multiple of 32" in lce.last_error()
    assert call_quant_mfma(desc(c_in=2 ** 21, c_out=1, h=1, w=1)) == lce.LCE_EUNSUPPORTED
    assert "2^24" in lce.last_error()
    # 2^24 pixels x 32 channels of float32 = 2 GiB
    assert call_quant_mfma(desc(n=1, h=2 ** 12, w=2 ** 12, c_in=32, c_out=32,
                                out_type="bitpacked")) == lce.LCE_EUNSUPPORTED
    assert "2 GiB" in lce.last_error()
    # 1x1 over 128 channels: 2 K steps, no filter-stationary instance within
    # 1/8 padding and too few for the K split
    assert call_quant_mfma(desc(c_in=128, c_out=32, kh=1, kw=1)) == lce.LCE_EUNSUPPORTED
    assert "filter-stationary" in lce.last_error() and "K-split" in lce.last_error()


def test_quantize_bconv2d_mfma_schedule_key_refusals():
    """The mfma_schedule tuning key restricts the fused entry's choice: the
    pixel split has no fused form, and a filter-stationary restriction
    refuses a shape none of its instances takes (27 K steps) -- both before
    any device call."""
    try:
        lce.set_tuning(mfma_schedule="pixel")
        assert call_quant_mfma(desc()) == lce.LCE_EUNSUPPORTED
        assert "mfma_schedule" in lce.last_error()
        lce.set_tuning(mfma_schedule="fs")
        assert call_quant_mfma(desc(c_in=160, c_out=32)) == lce.LCE_EUNSUPPORTED
        assert "27 K steps" in lce.last_error()
    finally:
        lce.set_tuning(mfma_schedule=0)


def call_quant(d, x=P, w=P, m=None, b=None, t=P, flip=None, out=P):
    return lce.lib().lce_quantize_bconv2d(ctypes.byref(d), x, w, m, b, t, flip, out, None)


def test_quantize_bconv2d_validation_errors():
    L = lce.lib()
    assert L.lce_quantize_bconv2d(None, P, P, None, None, P, None, P, None) == lce.LCE_EINVAL
    assert call_quant(desc(clamp=(5, 4))) == lce.LCE_EINVAL
    # shapes the fused kernel does not cover come back before any pointer check
    assert call_quant(desc(pad_value="zero"), x=None) == lce.LCE_EUNSUPPORTED
    assert "zero padding" in lce.last_error()
    assert call_quant(desc(c_in=40), x=None) == lce.LCE_EUNSUPPORTED
    assert "multiple of 32" in lce.last_error()
    for kh, kw, c_in in ((3, 5, 64), (1, 1, 64), (7, 7, 64), (3, 3, 224), (3, 3, 1024),
                         (5, 5, 512)):
        assert call_quant(desc(kh=kh, kw=kw, c_in=c_in), x=None) == lce.LCE_EUNSUPPORTED, \
            (kh, kw, c_in)
    # a VALID geometry never pads, so zero padding is not a reason to refuse it
    assert call_quant(desc(pad_value="zero", padding="valid"), x=None) == lce.LCE_EINVAL
    assert call_quant(desc(), x=None) == lce.LCE_EINVAL
    assert call_quant(desc(), w=None) == lce.LCE_EINVAL
    assert call_quant(desc(), out=None) == lce.LCE_EINVAL
    assert call_quant(desc(out_type="bitpacked"), t=None) == lce.LCE_EINVAL
    # the float input is read in 16-byte units
    assert call_quant(desc(), x=P + 4) == lce.LCE_EALIGN
    assert "16-byte" in lce.last_error()
    assert call_quant(desc(), x=P + 8) == lce.LCE_EALIGN
    assert call_quant(desc(), out=P + 2) == lce.LCE_EALIGN
    assert call_quant(desc(out_type="bitpacked"), flip=P + 1) == lce.LCE_EALIGN
    # a band too tall for LDS, refused before any launch (and on a GPU too,
    # whose LDS is 160 KiB): with stride 8 a 6-pixel-wide image has one
    # output column, so 64 output pixels span 64 output rows = 507 input rows
    # x 6 pixels x 16 words = 195 KiB, plus 38 KiB of im2col rows
    assert call_quant(desc(h=4096, w=6, c_in=512, stride=8)) == lce.LCE_EUNSUPPORTED
    assert "LDS" in lce.last_error()


def test_bitpack_validation_errors():
    L = lce.lib()
    assert L.lce_bitpack(None, P, 4, 32, None) == lce.LCE_EINVAL
    assert L.lce_bitpack(P, None, 4, 32, None) == lce.LCE_EINVAL
    assert L.lce_bitpack(P, P, -1, 32, None) == lce.LCE_EINVAL
    assert L.lce_bitpack(P, P, 4, 0, None) == lce.LCE_EINVAL
    assert L.lce_bitpack(P + 2, P, 4, 32, None) == lce.LCE_EALIGN
    assert L.lce_bitpack(P, P + 1, 4, 32, None) == lce.LCE_EALIGN
    assert L.lce_bitpack(P, P, 2 ** 62, 64, None) == lce.LCE_EINVAL
    # zero rows is a valid no-op: nothing is launched
    assert L.lce_bitpack(P, P, 0, 32, None) == lce.LCE_OK
    assert L.lce_bitpack(None, None, 0, 32, None) == lce.LCE_OK
    assert lce.last_error() == ""


def test_error_message_is_thread_local():
    import threading
    L = lce.lib()
    assert L.lce_bitpack(None, P, 4, 32, None) == lce.LCE_EINVAL
    seen = []
    th = threading.Thread(target=lambda: seen.append(lce.last_error()))
    th.start()
    th.join()
    assert seen == [""]
    assert lce.last_error() != ""


def test_pad_correction_validation_errors():
    L = lce.lib()
    n = ctypes.c_int64(-1)
    assert L.lce_bconv2d_pad_correction_size(ctypes.byref(desc(kh=3, kw=5, c_out=7)),
                                             ctypes.byref(n)) == lce.LCE_OK
    assert n.value == 4 * 15 * 7        # (KH+1) x KW(KW+1)/2 intervals x C_out
    assert L.lce_bconv2d_pad_correction_size(None, ctypes.byref(n)) == lce.LCE_EINVAL
    assert L.lce_bconv2d_pad_correction_size(ctypes.byref(desc()), None) == lce.LCE_EINVAL
    assert L.lce_bconv2d_pad_correction(ctypes.byref(desc()), None, P, None) == lce.LCE_EINVAL
    assert L.lce_bconv2d_pad_correction(ctypes.byref(desc()), P, None, None) == lce.LCE_EINVAL
    assert L.lce_bconv2d_pad_correction(ctypes.byref(desc()), P + 2, P, None) == lce.LCE_EALIGN
    assert L.lce_bconv2d_pad_correction(ctypes.byref(desc(c_out=0)), P, P, None) == lce.LCE_EINVAL


def test_fold_validation_errors():
    import numpy as np
    L = lce.lib()
    thr = np.zeros(4, np.float32)
    flip = np.zeros(1, np.int32)
    T, F = thr.ctypes.data, flip.ctypes.data
    m = np.ones(4, np.float32)
    assert L.lce_fold_thresholds(None, None, 4, 9, -9, 9, None, F) == lce.LCE_EINVAL
    assert L.lce_fold_thresholds(None, None, 4, 9, -9, 9, T, None) == lce.LCE_EINVAL
    assert L.lce_fold_thresholds(None, None, 0, 9, -9, 9, T, F) == lce.LCE_EINVAL
    assert L.lce_fold_thresholds(None, None, 4, 0, -9, 9, T, F) == lce.LCE_EINVAL
    assert L.lce_fold_thresholds(None, None, 4, 2 ** 24 + 1, -9, 9, T, F) == lce.LCE_EINVAL
    assert L.lce_fold_thresholds(None, None, 4, 9, 9, -9, T, F) == lce.LCE_EINVAL
    for bad in (np.inf, -np.inf, np.nan):
        mm = m.copy()
        mm[2] = bad
        assert L.lce_fold_thresholds(mm.ctypes.data, None, 4, 9, -9, 9, T, F) == lce.LCE_EINVAL
        assert "channel 2" in lce.last_error()
        assert L.lce_fold_thresholds(None, mm.ctypes.data, 4, 9, -9, 9, T, F) == lce.LCE_EINVAL
    assert L.lce_fold_thresholds(m.ctypes.data, None, 4, 9, -9, 9, T, F) == lce.LCE_OK


def test_pool_desc_layout_and_out_shape():
    assert ctypes.sizeof(lce.PoolDesc) == 9 * 4
    for h, k, s, pad in product((1, 2, 5, 7, 28, 56), (1, 2, 3, 5), (1, 2, 3), ("same", "valid")):
        if pad == "valid" and h < k:
            continue
        d = lce.make_pool_desc(2, h, h, 64, k, s, pad)
        assert lce.pool_out_shape(d) == (oracle.out_size(h, k, s, pad)[0],) * 2


def test_pool_validation_errors():
    L = lce.lib()
    oh, ow = ctypes.c_int32(), ctypes.c_int32()
    good = lce.make_pool_desc(2, 8, 8, 64, 2)
    assert L.lce_bmaxpool2d_out_shape(ctypes.byref(good), None, ctypes.byref(ow)) == \
        lce.LCE_EINVAL
    assert L.lce_bmaxpool2d(None, P, P, None) == lce.LCE_EINVAL
    for field, value in (("n", 0), ("h", 0), ("channels", 0), ("kh", 0), ("stride_w", 0),
                         ("padding", 5)):
        d = lce.make_pool_desc(2, 8, 8, 64, 2)
        setattr(d, field, value)
        assert L.lce_bmaxpool2d(ctypes.byref(d), P, P, None) == lce.LCE_EINVAL, field
    assert L.lce_bmaxpool2d(ctypes.byref(lce.make_pool_desc(1, 2, 2, 32, 3)), P, P, None) == \
        lce.LCE_EINVAL                                  # VALID 3x3 on 2x2: no output
    assert L.lce_bmaxpool2d(ctypes.byref(good), None, P, None) == lce.LCE_EINVAL
    assert L.lce_bmaxpool2d(ctypes.byref(good), P, None, None) == lce.LCE_EINVAL
    assert L.lce_bmaxpool2d(ctypes.byref(good), P + 2, P, None) == lce.LCE_EALIGN
    big = lce.make_pool_desc(2 ** 12, 2 ** 10, 2 ** 10, 64, 1)   # 2^33 input words
    assert L.lce_bmaxpool2d(ctypes.byref(big), P, P, None) == lce.LCE_EINVAL


def test_dequantize_validation_errors():
    L = lce.lib()
    assert L.lce_dequantize(None, P, 4, 32, None) == lce.LCE_EINVAL
    assert L.lce_dequantize(P, None, 4, 32, None) == lce.LCE_EINVAL
    assert L.lce_dequantize(P, P, -1, 32, None) == lce.LCE_EINVAL
    assert L.lce_dequantize(P, P, 4, 0, None) == lce.LCE_EINVAL
    assert L.lce_dequantize(P + 1, P, 4, 32, None) == lce.LCE_EALIGN
    assert L.lce_dequantize(P, P, 2 ** 62, 64, None) == lce.LCE_EINVAL
    assert L.lce_dequantize(P, P, 0, 32, None) == lce.LCE_OK
    assert L.lce_dequantize(None, None, 0, 32, None) == lce.LCE_OK     # empty: may be NULL


def test_tuning_overrides_round_trip_and_reset():
    L = lce.lib()
    assert ctypes.sizeof(ctypes.c_int32) == 4
    for name, key in lce.TUNING_KEYS.items():
        assert lce.get_tuning(name) == 0, name          # every override starts automatic
    with lce.tuning(xor_nb=3, mfma_schedule="pixel", mfma_packed=-1):
        assert lce.get_tuning("xor_nb") == 3
        assert lce.get_tuning("mfma_schedule") == lce.MFMA_SCHEDULES["pixel"]
        assert lce.get_tuning("mfma_packed") == -1
    assert all(lce.get_tuning(n) == 0 for n in lce.TUNING_KEYS)
    assert L.lce_set_tuning(len(lce.TUNING_KEYS), 1) == lce.LCE_EINVAL
    assert "tuning key" in lce.last_error()
    assert L.lce_set_tuning(-1, 1) == lce.LCE_EINVAL
    assert L.lce_get_tuning(99) == 0
    with pytest.raises(KeyError):
        lce.set_tuning(no_such_key=1)


def test_tuning_keys_match_header_enum():
    text = open(HEADER).read()
    enum = dict((m.group(1).lower(), int(m.group(2)))
                for m in re.finditer(r"LCE_TUNE_([A-Z0-9_]+)\s*=\s*(\d+)", text))
    count = enum.pop("count")
    assert enum == lce.TUNING_KEYS
    assert count == len(lce.TUNING_KEYS)


def test_tuning_set_from_many_threads():
    """Overrides are atomics: concurrent sets and gets from many threads
    leave one of the written values, never a torn or foreign one."""
    import threading
    L = lce.lib()
    key = lce.TUNING_KEYS["xor_nb"]
    seen = set()

    def work(v):
        for _ in range(2000):
            L.lce_set_tuning(key, v)
            seen.add(L.lce_get_tuning(key))

    threads = [threading.Thread(target=work, args=(v,)) for v in (1, 2, 3, 4)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert seen <= {1, 2, 3, 4}
    assert L.lce_get_tuning(key) in (1, 2, 3, 4)
    lce.set_tuning(xor_nb=0)
