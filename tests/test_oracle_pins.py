"""Pins of the CPU oracle against what the paper and the mathematics fix.

Nothing here compares the oracle with itself: each check is a value the
paper prints, a closed form derived by hand (tests/golden/), a library
routine that computes the same plain definition (numpy sliding windows,
torch's float64 cross-correlation), an exact-arithmetic evaluation
(fractions), or an invariant of the operator.
"""
import json
import os
from fractions import Fraction
from itertools import product

import numpy as np
import pytest

import oracle
from tests.conftest import GOLDEN

RNG = np.random.default_rng(12345)


def golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def rand_signs(shape, rng=RNG):
    return (1 - 2 * rng.integers(0, 2, size=shape)).astype(np.int8)


# ---------------------------------------------------------------- geometry

@pytest.mark.parametrize("h,k,s,padding,expect", [
    (56, 3, 1, "same", (56, 1)),
    (56, 3, 2, "same", (28, 0)),    # total pad 1 -> all of it trailing
    (4, 3, 2, "same", (2, 0)),
    (7, 3, 1, "same", (7, 1)),
    (8, 5, 1, "same", (8, 2)),
    (5, 3, 2, "same", (3, 1)),      # total pad 2 -> 1 + 1
    (6, 1, 2, "same", (3, 0)),
    (8, 3, 1, "valid", (6, 0)),
    (9, 3, 2, "valid", (4, 0)),
    (3, 3, 1, "valid", (1, 0)),
])
def test_out_size_hand(h, k, s, padding, expect):
    assert oracle.out_size(h, k, s, padding) == expect


def test_out_size_same_covers_input_exactly():
    # SAME: ceil(h/s) outputs; the windows cover every input row, the padding
    # is the least that makes the last window fit, and the leading side never
    # gets more than the trailing side.
    for h, k, s in product(range(1, 12), range(1, 7), range(1, 4)):
        oh, pt = oracle.out_size(h, k, s, "same")
        assert oh == -(-h // s)
        pb_needed = max((oh - 1) * s + k - h - pt, 0)
        assert 0 <= pt <= pb_needed <= pt + 1
        rows = set()
        for oy in range(oh):
            rows.update(range(oy * s - pt, oy * s - pt + k))
        if k >= s:   # a kernel narrower than the stride skips rows by design
            assert set(range(h)) <= rows
            assert max(rows) - (h - 1) == pb_needed
        assert min(rows) == -pt


def test_out_size_valid_never_pads():
    for h, k, s in product(range(1, 12), range(1, 7), range(1, 4)):
        if h < k:
            with pytest.raises(ValueError):
                oracle.out_size(h, k, s, "valid")
            continue
        oh, pt = oracle.out_size(h, k, s, "valid")
        assert pt == 0
        assert (oh - 1) * s + k <= h < oh * s + k


# ---------------------------------------------------------------- binarize / pack

def test_binarize_special_values():
    x = np.array([-0.0, 0.0, np.nan, -np.nan, np.inf, -np.inf, 1e-45, -1e-45, -1.0, 2.5],
                 np.float32)
    assert oracle.binarize(x).tolist() == [1, 1, 1, 1, 1, -1, 1, -1, -1, 1]


def test_pack_hand_example():
    g = golden("e5_pack.json")
    s = np.ones((1, g["channels"]), np.int8)
    s[0, g["negative_channels"]] = -1
    assert oracle.pack(s).tolist() == [g["words"]]
    s = np.ones((1, g["channels_ragged"]), np.int8)
    s[0, g["negative_channels_ragged"]] = -1
    assert oracle.pack(s).tolist() == [g["words_ragged"]]


@pytest.mark.parametrize("c", [1, 5, 31, 32, 33, 40, 64, 96, 100])
def test_pack_matches_bit_definition(c):
    s = rand_signs((7, c))
    words = oracle.pack(s)
    assert words.shape == (7, (c + 31) // 32)
    for r in range(7):
        # Independent evaluation: bit j of the little-endian bit string.
        bits = "".join("1" if v == -1 else "0" for v in s[r]) + "0" * (32 * words.shape[1] - c)
        for j in range(words.shape[1]):
            assert int(words[r, j]) == int(bits[32 * j:32 * j + 32][::-1], 2)
    assert np.array_equal(oracle.unpack(words, c), s)


def test_packed_sizes_printed_in_paper():
    g = golden("packed_sizes.json")
    w = g["weights"]
    s = np.ones((w["c_out"], w["kh"], w["kw"], w["c_in"]), np.int8)
    packed = oracle.pack(s)
    assert packed.nbytes == w["kib"] * 1024
    assert (s.size * 4) // packed.nbytes == g["weight_ratio_vs_float32"]
    a = np.ones((1, 8, 8, 64), np.int8)
    pa = oracle.pack(a)
    assert (a.size * 4) // pa.nbytes == g["activation_ratio_vs_float32"]
    assert a.size // pa.nbytes == g["activation_ratio_vs_int8"]
    assert oracle.pack(np.ones((3, 33), np.int8)).shape[-1] * 32 % g["channel_pad_multiple"] == 0


# ---------------------------------------------------------------- identity

def test_xor_popcount_identity_exhaustive_8bit():
    # For every pair of 8-bit patterns: the sum of the +-1 products equals
    # n - 2 * popcount(a XOR w).  Uses the oracle's unpack for the meaning of
    # a bit, so a wrong bit polarity or order fails here.
    a = np.arange(256, dtype=np.uint32)
    sa = oracle.unpack(a.reshape(256, 1), 8).astype(np.int32)   # [256, 8]
    prod_sum = sa @ sa.T                                        # [256, 256]
    pc = np.array([bin(i).count("1") for i in range(256)])
    xor_pc = pc[np.bitwise_xor.outer(np.arange(256), np.arange(256))]
    assert np.array_equal(prod_sum, 8 - 2 * xor_pc)


def test_xor_popcount_identity_random_32bit():
    rng = np.random.default_rng(7)
    a = rng.integers(0, 2 ** 32, size=(500, 1), dtype=np.uint64).astype(np.uint32)
    w = rng.integers(0, 2 ** 32, size=(500, 1), dtype=np.uint64).astype(np.uint32)
    sa = oracle.unpack(a, 32).astype(np.int32)
    sw = oracle.unpack(w, 32).astype(np.int32)
    lhs = (sa * sw).sum(axis=1)
    rhs = np.array([32 - 2 * bin(int(x) ^ int(y)).count("1") for x, y in zip(a[:, 0], w[:, 0])])
    assert np.array_equal(lhs, rhs)


# ---------------------------------------------------------------- convolution

def brute_numpy(a, w, sh, sw, padding):
    """Explicit +1 padding, then numpy sliding windows and tensordot in fp64."""
    n, h, wd, c = a.shape
    cout, kh, kw, _ = w.shape
    if padding == "same":
        oh, ow = -(-h // sh), -(-wd // sw)
        ph = max((oh - 1) * sh + kh - h, 0)
        pw = max((ow - 1) * sw + kw - wd, 0)
        pads = ((0, 0), (ph // 2, ph - ph // 2), (pw // 2, pw - pw // 2), (0, 0))
        a = np.pad(a.astype(np.float64), pads, constant_values=1.0)
    else:
        a = a.astype(np.float64)
    win = np.lib.stride_tricks.sliding_window_view(a, (kh, kw), axis=(1, 2))
    win = win[:, ::sh, ::sw]                         # [n, oh, ow, c, kh, kw]
    return np.tensordot(win, w.astype(np.float64), axes=([3, 4, 5], [3, 1, 2]))


def brute_torch(a, w, sh, sw, padding):
    """torch's float64 cross-correlation on explicitly +1-padded input."""
    import torch
    import torch.nn.functional as F
    n, h, wd, c = a.shape
    cout, kh, kw, _ = w.shape
    x = torch.from_numpy(a.astype(np.float64)).permute(0, 3, 1, 2)
    if padding == "same":
        oh, ow = -(-h // sh), -(-wd // sw)
        ph = max((oh - 1) * sh + kh - h, 0)
        pw = max((ow - 1) * sw + kw - wd, 0)
        x = F.pad(x, (pw // 2, pw - pw // 2, ph // 2, ph - ph // 2), value=1.0)
    wt = torch.from_numpy(w.astype(np.float64)).permute(0, 3, 1, 2)
    y = F.conv2d(x, wt, stride=(sh, sw))
    return y.permute(0, 2, 3, 1).numpy()


TINY = [
    # n, h, w, c, cout, kh, kw, sh, sw, padding
    (1, 1, 1, 32, 3, 1, 1, 1, 1, "same"),
    (2, 5, 6, 32, 4, 3, 3, 1, 1, "same"),
    (1, 6, 5, 33, 5, 3, 3, 2, 2, "same"),
    (2, 4, 4, 1, 2, 3, 3, 1, 1, "same"),
    (1, 6, 6, 64, 3, 5, 5, 1, 1, "same"),
    (1, 6, 6, 40, 2, 5, 5, 2, 2, "same"),
    (1, 5, 6, 7, 3, 3, 2, 1, 2, "same"),
    (2, 6, 5, 32, 3, 3, 3, 1, 1, "valid"),
    (1, 6, 6, 33, 2, 3, 3, 2, 2, "valid"),
    (1, 5, 5, 8, 2, 5, 5, 1, 1, "valid"),
    (1, 3, 6, 16, 2, 2, 4, 1, 2, "valid"),
    (1, 2, 2, 32, 1, 3, 3, 1, 1, "same"),
    (1, 1, 4, 3, 2, 3, 3, 2, 1, "same"),
]


@pytest.mark.parametrize("shape", TINY)
def test_conv_brute_force_numpy(shape):
    n, h, wd, c, cout, kh, kw, sh, sw, padding = shape
    a = rand_signs((n, h, wd, c))
    w = rand_signs((cout, kh, kw, c))
    dot = oracle.conv_dot(a, w, (sh, sw), padding)
    ref = brute_numpy(a, w, sh, sw, padding)
    assert dot.shape == ref.shape
    assert np.array_equal(dot, ref.astype(np.int64))


@pytest.mark.parametrize("shape", TINY[::2])
def test_conv_brute_force_torch(shape):
    n, h, wd, c, cout, kh, kw, sh, sw, padding = shape
    a = rand_signs((n, h, wd, c))
    w = rand_signs((cout, kh, kw, c))
    dot = oracle.conv_dot(a, w, (sh, sw), padding)
    ref = brute_torch(a, w, sh, sw, padding)
    assert np.array_equal(dot, ref.astype(np.int64))


def test_conv_asymmetric_filter_not_transposed():
    # A filter with a single -1 tap at (ky=0, kx=2): the output at (oy, ox)
    # must read the input at (oy-1, ox+1) for a 3x3 SAME stride-1 conv
    # (cross-correlation, no kernel flip, no H/W transpose).
    h, wd, c = 5, 6, 32
    a = rand_signs((1, h, wd, c))
    w = np.ones((1, 3, 3, c), np.int8)
    w[0, 0, 2, :] = -1
    dot = oracle.conv_dot(a, w, 1, "same")
    for oy, ox in product(range(h), range(wd)):
        expect = 0
        for ky, kx in product(range(3), range(3)):
            iy, ix = oy - 1 + ky, ox - 1 + kx
            av = a[0, iy, ix].astype(np.int64) if 0 <= iy < h and 0 <= ix < wd else np.ones(c)
            expect += int((av * w[0, ky, kx]).sum())
        assert dot[0, oy, ox, 0] == expect


@pytest.mark.parametrize("name", ["e1_single_word.json", "e2_one_padding.json",
                                  "e3_same_stride2.json"])
def test_hand_examples(name):
    g = golden(name)
    if "a_word" in g:
        a = oracle.unpack(np.array([[g["a_word"]]], np.uint32), 32).reshape(g["input_shape"])
        w = oracle.unpack(np.array([[g["w_word"]]], np.uint32), 32).reshape(g["filter_shape"])
    else:
        a = np.full(g["input_shape"], g["input_value"], np.int8)
        w = np.full(g["filter_shape"], g["filter_value"], np.int8)
    dot = oracle.conv_dot(a, w, g["stride"], g["padding"])
    assert dot.tolist() == g["dot"]


@pytest.mark.parametrize("s", [1, 2])
def test_all_plus_one_input_gives_filter_sums(s):
    # One-padding is +1, so an all-+1 input makes every output, borders
    # included, the plain sum of the filter's entries.
    a = np.ones((2, 7, 6, 40), np.int8)
    w = rand_signs((5, 3, 3, 40))
    dot = oracle.conv_dot(a, w, s, "same")
    sums = w.astype(np.int64).sum(axis=(1, 2, 3))
    assert np.array_equal(dot, np.broadcast_to(sums, dot.shape))


@pytest.mark.parametrize("h,w_,k,s", [(7, 7, 3, 1), (8, 6, 3, 2), (6, 6, 5, 1), (5, 7, 5, 2)])
def test_one_padding_equals_explicit_padding(h, w_, k, s):
    a = rand_signs((2, h, w_, 33))
    w = rand_signs((3, k, k, 33))
    same = oracle.conv_dot(a, w, s, "same")
    oh, pt = oracle.out_size(h, k, s, "same")
    ow, pl = oracle.out_size(w_, k, s, "same")
    pb = max((oh - 1) * s + k - h - pt, 0)
    pr = max((ow - 1) * s + k - w_ - pl, 0)
    ap = np.pad(a, ((0, 0), (pt, pb), (pl, pr), (0, 0)), constant_values=1)
    valid = oracle.conv_dot(ap, w, s, "valid")
    assert np.array_equal(same, valid)


def test_range_and_parity():
    a = rand_signs((2, 9, 9, 70))
    w = rand_signs((6, 3, 3, 70))
    dot = oracle.conv_dot(a, w, 1, "same")
    k = 3 * 3 * 70
    assert np.abs(dot).max() <= k
    assert np.all((dot - k) % 2 == 0)


def test_negation_and_additivity():
    a = rand_signs((1, 6, 7, 64))
    w = rand_signs((4, 3, 3, 64))
    dot = oracle.conv_dot(a, w, 1, "same")
    assert np.array_equal(oracle.conv_dot(a, -w, 1, "same"), -dot)
    d1 = oracle.conv_dot(np.ascontiguousarray(a[..., :20]), np.ascontiguousarray(w[..., :20]),
                         1, "same")
    d2 = oracle.conv_dot(np.ascontiguousarray(a[..., 20:]), np.ascontiguousarray(w[..., 20:]),
                         1, "same")
    assert np.array_equal(dot, d1 + d2)


def test_single_bit_flip_moves_covering_outputs_by_two():
    a = rand_signs((1, 6, 6, 32))
    w = rand_signs((3, 3, 3, 32))
    dot = oracle.conv_dot(a, w, 1, "same")
    b = a.copy()
    y0, x0, c0 = 2, 4, 17
    b[0, y0, x0, c0] *= -1
    diff = oracle.conv_dot(b, w, 1, "same") - dot
    for oy, ox in product(range(6), range(6)):
        ky, kx = y0 - oy + 1, x0 - ox + 1
        if 0 <= ky < 3 and 0 <= kx < 3:
            expect = -2 * int(a[0, y0, x0, c0]) * w[:, ky, kx, c0].astype(np.int64)
            assert np.array_equal(diff[0, oy, ox], expect)
        else:
            assert not diff[0, oy, ox].any()


# ---------------------------------------------------------------- output transforms

def test_clamp():
    d = np.array([-10, -3, 0, 3, 10], np.int32)
    assert oracle.clamp(d, -3, 4).tolist() == [-3, -3, 0, 3, 4]
    assert oracle.clamp(d, oracle.INT32_MIN, oracle.INT32_MAX).tolist() == d.tolist()


def test_out_float_exact_arithmetic():
    rng = np.random.default_rng(3)
    c = rng.integers(-4608, 4609, size=(50, 6)).astype(np.int32)
    m = rng.normal(1, 0.1, 6).astype(np.float32)
    b = rng.normal(0, 0.1, 6).astype(np.float32)
    y = oracle.out_float(c, m, b)
    for i, j in product(range(50), range(6)):
        exact = Fraction(int(c[i, j])) * Fraction(float(m[j])) + Fraction(float(b[j]))
        # fp64 evaluation of one product (exact) and one sum: one rounding.
        assert abs(Fraction(float(y[i, j])) - exact) <= abs(exact) * Fraction(1, 2 ** 52)
    # multiplier 1 and bias 0 (also the defaults) give the accumulator itself
    assert np.array_equal(oracle.out_float(c, None, None), c.astype(np.float64))
    assert np.array_equal(oracle.out_float(c, np.ones(6, np.float32), np.zeros(6, np.float32)),
                          c.astype(np.float64))


def test_out_bits_hand_cases():
    g = golden("e4_thresholds.json")
    for case in g["cases"]:
        c = np.array([[case["c"]]], np.int32)
        thr = np.array([float(case["thr"])], np.float32)
        assert int(oracle.out_bits(c, thr)[0, 0]) == case["bit"], case


def test_out_bits_exact_comparison_and_packing():
    rng = np.random.default_rng(4)
    cout = 70
    c = rng.integers(-600, 601, size=(20, cout)).astype(np.int32)
    thr = (rng.standard_normal(cout) * 100).astype(np.float32)
    thr[:5] = np.floor(thr[:5])            # thresholds exactly at integers
    words = oracle.out_bits(c, thr)
    assert words.shape == (20, 3)
    for i in range(20):
        signs = np.array([-1 if Fraction(int(c[i, j])) < Fraction(float(thr[j])) else 1
                          for j in range(cout)], np.int8)
        assert np.array_equal(oracle.unpack(words[i:i + 1], cout)[0], signs)
    assert not (words[:, 2] >> (cout - 64)).any()   # pad bits zero


def test_bconv2d_composite_against_torch():
    a = rand_signs((1, 8, 8, 64))
    w = rand_signs((64, 3, 3, 64))
    m = RNG.normal(1, 0.1, 64).astype(np.float32)
    b = RNG.normal(0, 0.1, 64).astype(np.float32)
    y = oracle.bconv2d(a, w, out="float", mult=m, bias=b, clamp_range=(-100, 50))
    ref = np.clip(brute_torch(a, w, 1, 1, "same"), -100, 50) * m.astype(np.float64) + b
    np.testing.assert_allclose(y, ref, rtol=1e-15, atol=1e-12)


# ---------------------------------------------------------------- zero padding (Section 3.2)

def brute_torch_zero(a, w, sh, sw, padding):
    """torch's float64 cross-correlation on explicitly zero-padded input."""
    import torch
    import torch.nn.functional as F
    n, h, wd, c = a.shape
    cout, kh, kw, _ = w.shape
    x = torch.from_numpy(a.astype(np.float64)).permute(0, 3, 1, 2)
    if padding == "same":
        oh, ow = -(-h // sh), -(-wd // sw)
        ph = max((oh - 1) * sh + kh - h, 0)
        pw = max((ow - 1) * sw + kw - wd, 0)
        x = F.pad(x, (pw // 2, pw - pw // 2, ph // 2, ph - ph // 2), value=0.0)
    wt = torch.from_numpy(w.astype(np.float64)).permute(0, 3, 1, 2)
    return F.conv2d(x, wt, stride=(sh, sw)).permute(0, 2, 3, 1).numpy()


@pytest.mark.parametrize("shape", TINY)
def test_zero_padding_against_torch(shape):
    n, h, wd, c, cout, kh, kw, sh, sw, padding = shape
    a = rand_signs((n, h, wd, c))
    w = rand_signs((cout, kh, kw, c))
    dot = oracle.conv_dot(a, w, (sh, sw), padding, pad_value=0)
    assert np.array_equal(dot, brute_torch_zero(a, w, sh, sw, padding).astype(np.int64))


def test_zero_padding_hand_example():
    g = golden("e2_one_padding.json")
    a = np.full(g["input_shape"], g["input_value"], np.int8)
    w = np.full(g["filter_shape"], g["filter_value"], np.int8)
    dot = oracle.conv_dot(a, w, g["stride"], g["padding"], pad_value=0)
    assert (dot == g["dot_if_zero_padded"]).all()


@pytest.mark.parametrize("h,w_,k,s", [(5, 6, 3, 1), (7, 7, 3, 2), (6, 5, 5, 1), (1, 1, 3, 1)])
def test_zero_padding_is_one_padding_minus_padded_tap_sums(h, w_, k, s):
    # The correction step: a padded tap contributes its filter tap's sum of
    # weights under one-padding and nothing under zero-padding.
    a = rand_signs((2, h, w_, 40))
    w = rand_signs((3, k, k, 40))
    one = oracle.conv_dot(a, w, s, "same", pad_value=1)
    zero = oracle.conv_dot(a, w, s, "same", pad_value=0)
    oh, pt = oracle.out_size(h, k, s, "same")
    ow, pl = oracle.out_size(w_, k, s, "same")
    tapsum = w.astype(np.int64).sum(axis=3)                      # [cout, k, k]
    for oy, ox in product(range(oh), range(ow)):
        corr = np.zeros(3, np.int64)
        for ky, kx in product(range(k), range(k)):
            iy, ix = oy * s - pt + ky, ox * s - pl + kx
            if not (0 <= iy < h and 0 <= ix < w_):
                corr += tapsum[:, ky, kx]
        assert np.array_equal(zero[:, oy, ox], one[:, oy, ox] - corr)


# ---------------------------------------------------------------- binarized max pooling (Section 3.2)

@pytest.mark.parametrize("h,w_,k,s,padding", [(6, 6, 2, 2, "valid"), (7, 5, 3, 2, "same"),
                                              (5, 5, 3, 1, "same"), (4, 7, 3, 3, "valid"),
                                              (1, 1, 3, 2, "same")])
def test_bmaxpool_commutes_with_sign(h, w_, k, s, padding):
    # max(sign(X)) = sign(max(X)): binarizing before max pooling gives the
    # same bits as binarizing after it (torch's float max pooling).
    import torch
    import torch.nn.functional as F
    rng = np.random.default_rng(h * 100 + k)
    x = rng.standard_normal((2, h, w_, 37)).astype(np.float32)
    got = oracle.bmaxpool(oracle.binarize(x), k, k, s, padding)
    t = torch.from_numpy(x).permute(0, 3, 1, 2)
    if padding == "same":
        oh, ow = -(-h // s), -(-w_ // s)
        ph = max((oh - 1) * s + k - h, 0)
        pw = max((ow - 1) * s + k - w_, 0)
        t = F.pad(t, (pw // 2, pw - pw // 2, ph // 2, ph - ph // 2), value=float("-inf"))
    ref = F.max_pool2d(t, k, s).permute(0, 2, 3, 1).numpy()
    assert np.array_equal(got, oracle.binarize(ref))


def test_bmaxpool_is_and_of_bits():
    # In bitpacked form the pooled bit is the AND of the window's bits
    # (a 1 bit, -1.0, survives only if every value is -1).
    a = rand_signs((1, 4, 4, 64))
    got = oracle.pack(oracle.bmaxpool(a, 2, 2, 2, "valid"))
    words = oracle.pack(a)
    ref = words[:, 0::2, 0::2] & words[:, 1::2, 0::2] & words[:, 0::2, 1::2] & words[:, 1::2, 1::2]
    assert np.array_equal(got, ref)


# ---------------------------------------------------------------- sign of the float transform (Section 3.1)

def test_sign_of_affine_exact():
    rng = np.random.default_rng(11)
    c = np.arange(-600, 601, dtype=np.int32)
    cases = [(1.0, 0.0), (1.0, -0.5), (-0.75, 3.0), (0.0, -1.0), (0.0, 1.0), (-0.0, 0.0),
             (3.0, -6.0), (0.1, 0.3),
             # near-cancelling: exact c*m + b is a hair below 0 where a float
             # evaluation rounds it to 0 (e.g. c = 3: -7.45e-9)
             (0.1, -0.3), (0.7, -2.1), (1.1, -3.3), (-0.3, 0.9)] + [
             (float(np.float32(m)), float(np.float32(b)))
                                         for m, b in rng.normal(0, 1, (20, 2))]
    for m, b in cases:
        m32, b32 = np.float32(m), np.float32(b)
        bits = oracle.sign_of_affine(c, m32, b32)
        ref = [1 if Fraction(int(ci)) * Fraction(float(m32)) + Fraction(float(b32)) < 0 else 0
               for ci in c]
        assert bits.tolist() == ref, (m, b)


# ---------------------------------------------------------------- per-channel direction (flip)

def test_flip_hand_example():
    """tests/golden/e6_flip.json: four filters with hand-computed dots,
    thresholds on either side of them and a flip word."""
    g = golden("e6_flip.json")
    a = np.ones((1, 1, 1, 8), np.int8)
    w = np.ones((4, 1, 1, 8), np.int8)
    for f, k in enumerate(g["k"]):
        w[f, 0, 0, :k] = -1
    dot = oracle.bconv2d(a, w, out="int32")
    assert dot.reshape(-1).tolist() == g["dot"]
    thr = np.array(g["thresholds"], np.float32)
    plain = oracle.bconv2d(a, w, out="bitpacked", thr=thr)
    assert int(plain.reshape(-1)[0]) == sum(b << i for i, b in enumerate(g["below"]))
    got = oracle.bconv2d(a, w, out="bitpacked", thr=thr, flip=np.array(g["flip"], np.uint8))
    assert got.shape == (1, 1, 1, 1)
    assert int(got.reshape(-1)[0]) == g["word"]


@pytest.mark.parametrize("c_out", [1, 31, 32, 40, 64, 100])
def test_flip_every_channel_complements_valid_bits(c_out):
    """Flipping every channel inverts exactly the C_out valid bits of each
    output word; the pad bits past C_out stay 0.  Flipping none changes
    nothing."""
    rng = np.random.default_rng(c_out)
    a = rand_signs((2, 5, 6, 40), rng)
    w = rand_signs((c_out, 3, 3, 40), rng)
    thr = rng.normal(0.0, 6.0, c_out).astype(np.float32)
    base = oracle.bconv2d(a, w, out="bitpacked", thr=thr)
    none = oracle.bconv2d(a, w, out="bitpacked", thr=thr, flip=np.zeros(c_out, np.uint8))
    assert np.array_equal(none, base)
    allf = oracle.bconv2d(a, w, out="bitpacked", thr=thr, flip=np.ones(c_out, np.uint8))
    cw = (c_out + 31) // 32
    mask = np.array([(1 << min(32, c_out - 32 * j)) - 1 for j in range(cw)], np.uint64)
    assert np.array_equal(allf.astype(np.uint64), (~base.astype(np.uint64)) & mask)


def test_flip_equals_negated_filters_with_mirrored_thresholds():
    """For integer thresholds t: NOT(dot < t) = (-dot < 1 - t), and negating
    the filters negates dot (a +-1 product changes sign).  So flipping a
    channel equals running its negated filter against 1 - t without a flip,
    channel by channel."""
    rng = np.random.default_rng(77)
    a = rand_signs((3, 7, 5, 64), rng)
    w = rand_signs((48, 3, 3, 64), rng)
    thr = rng.integers(-30, 31, 48).astype(np.float32)
    flip = rng.integers(0, 2, 48).astype(np.uint8)
    got = oracle.bconv2d(a, w, out="bitpacked", thr=thr, flip=flip)
    w2 = np.where(flip[:, None, None, None].astype(bool), -w, w).astype(np.int8)
    thr2 = np.where(flip.astype(bool), 1.0 - thr, thr).astype(np.float32)
    want = oracle.bconv2d(a, w2, out="bitpacked", thr=thr2)
    assert np.array_equal(got, want)
