"""GPU parity of the zero-padding correction and of folded thresholds.

Zero padding (Section 3.2 supports TensorFlow's zero padding through a
correction step): lce_bconv2d with pad_value "zero" and the table of
lce_bconv2d_pad_correction must equal the oracle's convolution with 0 at the
padded locations, bit for bit (int32 / bitpacked) or within 1e-6 relative
(float), for every kernel variant and work split.

Threshold fold (Sections 3.1, 3.2): a bitpacked layer run with the
thresholds and flip bits of lce_fold_thresholds must equal the binarization
of the float layer it replaces.
"""
import numpy as np
import pytest

import oracle
from tests.layer_util import (POISON_I32, assert_match, clamp_of, config4_reference, dev,
                              gpu_input, gpu_pack_weights, oracle_signs, poisoned_out)
from workloads import INT32_MAX, INT32_MIN, Layer, config, make_layer_inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2011_09398_amd as lce
    lce.lib()
    yield
    torch.cuda.synchronize()


def sync_np(t):
    import torch
    torch.cuda.synchronize()
    return t.cpu().numpy()


def gpu_run(layer, inp, *, pad_value="zero", x_packed=None, w_packed=None, corr="auto",
            thresholds=None, flip=None, out_type=None):
    import paper_2011_09398_amd as lce
    x_packed = gpu_input(inp) if x_packed is None else x_packed
    w_packed = gpu_pack_weights(inp) if w_packed is None else w_packed
    if isinstance(corr, str):
        corr = lce.pad_correction(w_packed, layer.c_in) if pad_value == "zero" else None
    out_type = layer.out if out_type is None else out_type
    kw = {}
    if out_type == "float":
        kw = dict(multiplier=dev(inp.mult), bias=dev(inp.bias))
    elif out_type == "bitpacked":
        kw = dict(thresholds=dev(inp.thr if thresholds is None else thresholds),
                  flip=None if flip is None else dev(flip))
    return lce.bconv2d(x_packed, w_packed, layer.c_in, stride=layer.strides,
                       padding=layer.padding, pad_value=pad_value, clamp=layer.clamp,
                       out_type=out_type, out=poisoned_out(layer), pad_correction=corr, **kw)


def oracle_run(layer, inp, a_signs, pad_value=0):
    return oracle.bconv2d(a_signs, inp.w_sign, stride=layer.strides, padding=layer.padding,
                          clamp_range=clamp_of(layer), out=layer.out, mult=inp.mult,
                          bias=inp.bias, thr=inp.thr, pad_value=pad_value)


# ---------------------------------------------------------------- correction table

@pytest.mark.parametrize("c_in,c_out,kh,kw", [(64, 40, 3, 3), (33, 13, 5, 3), (512, 8, 1, 1),
                                               (7, 100, 3, 5), (96, 1, 7, 7)])
def test_pad_correction_table_is_prefix_of_interval_sums(c_in, c_out, kh, kw):
    """table[y][I][co] = sum over ky < y and kx in the column interval I of
    the tap sums of the +-1 filter, intervals [x0, x1) numbered by x0 then
    x1 (computed here from the oracle-side signs, not from the GPU)."""
    import paper_2011_09398_amd as lce
    layer = Layer("tab", 1, 4, 4, c_in, c_out, kh=kh, kw=kw, input_kind="bits")
    inp = make_layer_inputs(layer, 3, 70, c_out)
    got = sync_np(lce.pad_correction(gpu_pack_weights(inp), c_in))
    s = inp.w_sign.astype(np.int64).sum(axis=3)                       # [co, ky, kx]
    intervals = [(x0, x1) for x0 in range(kw) for x1 in range(x0 + 1, kw + 1)]
    want = np.zeros((kh + 1, len(intervals), c_out), np.int64)
    for y in range(1, kh + 1):
        for i, (x0, x1) in enumerate(intervals):
            want[y, i] = s[:, :y, x0:x1].sum(axis=(1, 2))
    assert np.array_equal(got.astype(np.int64), want.reshape(-1, c_out))


# ---------------------------------------------------------------- zero-padding parity

def zero_pad_cases():
    rng = np.random.default_rng(4040)
    cases = []
    for i in range(48):
        k = int(rng.choice([1, 2, 3, 3, 3, 5, 7]))
        kw = k if rng.random() < 0.8 else int(rng.choice([1, 3]))
        s = int(rng.choice([1, 1, 2, 3]))
        sw_ = s if rng.random() < 0.8 else int(rng.choice([1, 2]))
        padding = "same" if rng.random() < 0.85 else "valid"
        h = int(rng.integers(1, 11))
        w = int(rng.integers(1, 11))
        if padding == "valid":
            h, w = max(h, k), max(w, kw)
        c_in = int(rng.choice([1, 7, 32, 33, 64, 96, 128, 160, 256, 512]))
        c_out = int(rng.choice([1, 5, 8, 13, 32, 40, 64, 100]))
        n = int(rng.integers(1, 4))
        out = ["float", "bitpacked", "int32"][i % 3]
        kk = k * kw * c_in
        clamp = [None, (-kk, kk), (0, kk), (-3, 3), (0, 0)][int(rng.integers(0, 5))]
        cases.append(Layer(f"zp{i}", n, h, w, c_in, c_out, kh=k, kw=kw, stride=s,
                           stride_w=sw_, padding=padding, out=out, clamp=clamp,
                           input_kind=["float", "bits"][i % 2]))
    return cases


@pytest.mark.parametrize("layer", zero_pad_cases(), ids=lambda l: l.name)
def test_zero_padding_sweep(layer):
    inp = make_layer_inputs(layer, 9, 98, int(layer.name[2:]))
    got = sync_np(gpu_run(layer, inp))
    ref = oracle_run(layer, inp, oracle_signs(inp))
    assert_match(layer, got, ref, layer.name)


STATIC = [(3, cw) for cw in (1, 2, 3, 4, 5, 6, 8, 16)] + [(5, cw) for cw in (1, 2, 3, 4, 5, 6, 8)]


@pytest.mark.parametrize("k,cw", STATIC)
@pytest.mark.parametrize("out", ["float", "bitpacked", "int32"])
def test_zero_padding_every_static_width(k, cw, out):
    """Kernels with a compile-time filter size and word count (3x3, 5x5)
    stage the table in LDS."""
    layer = Layer(f"zs{k}{cw}{out}", 2, 9, 11, 32 * cw, 40, kh=k, kw=k, out=out,
                  input_kind="bits", clamp=(-100, 90) if out != "bitpacked" else None)
    inp = make_layer_inputs(layer, cw + 20 * k, 97, len(out))
    got = sync_np(gpu_run(layer, inp))
    assert_match(layer, got, oracle_run(layer, inp, oracle_signs(inp)), layer.name)


SCHEDULES = [(1, 1), (2, 1), (3, 1), (4, 1), (1, 2), (1, 4)]


@pytest.mark.parametrize("nb,ks", SCHEDULES)
@pytest.mark.parametrize("shape", [
    (2, 9, 7, 64, 40, 1, "bitpacked"),
    (3, 8, 8, 128, 72, 2, "float"),
    (1, 7, 7, 512, 96, 1, "int32"),
    (2, 5, 6, 256, 130, 1, "bitpacked"),
])
def test_zero_padding_every_schedule(nb, ks, shape):
    import paper_2011_09398_amd as lce
    n, h, w, c_in, c_out, s, out = shape
    lce.set_tuning(xor_nb=nb, xor_ks=ks)
    layer = Layer(f"zsched{nb}{ks}", n, h, w, c_in, c_out, stride=s, out=out,
                  clamp=(-50, 60) if out != "bitpacked" else None, input_kind="bits")
    inp = make_layer_inputs(layer, nb * 10 + ks, 61, c_out)
    got = sync_np(gpu_run(layer, inp))
    assert_match(layer, got, oracle_run(layer, inp, oracle_signs(inp)), layer.name)


def test_zero_padding_special_thresholds():
    """Thresholds at the clamp edges, integers, +-inf and NaN under zero padding."""
    layer = Layer("zthr", 2, 9, 7, 64, 40, out="bitpacked", input_kind="bits", clamp=(-20, 30))
    inp = make_layer_inputs(layer, 5, 62, 0)
    thr = inp.thr.copy()
    thr[:10] = [-20.0, -20.5, -19.5, 30.0, 30.5, 31.0, np.inf, -np.inf, np.nan, 0.0]
    thr[10:20] = np.arange(-5, 5, dtype=np.float32)
    inp.thr[:] = thr
    got = sync_np(gpu_run(layer, inp))
    assert_match(layer, got, oracle_run(layer, inp, oracle_signs(inp)), layer.name)


@pytest.mark.parametrize("cfg_layer", [(2, 0), (4, 0), (4, 1), (4, 2), (4, 3)])
def test_zero_padding_config_layers(cfg_layer):
    """The workload layers at full size with zero padding, every output
    (each batch-64 layer on its own input)."""
    cfg, li = cfg_layer
    if cfg == 4:
        layer, inp, ref = config4_reference(chain=False, pad_value=0)[li]
    else:
        layer = config(cfg)[li]
        inp = make_layer_inputs(layer, 0, cfg, li)
        ref = oracle_run(layer, inp, oracle_signs(inp))
    got = sync_np(gpu_run(layer, inp))
    assert_match(layer, got, ref, layer.name)


def test_zero_padding_without_padded_taps_needs_no_table():
    """VALID and 1x1 SAME windows never reach outside the image: the result
    is the one-padded one and no table is needed."""
    for layer in (Layer("zv", 2, 9, 7, 64, 40, out="int32", padding="valid", input_kind="bits"),
                  Layer("z1", 2, 9, 7, 64, 40, kh=1, kw=1, out="int32", input_kind="bits")):
        inp = make_layer_inputs(layer, 1, 63, 0)
        got = sync_np(gpu_run(layer, inp, corr=None))
        assert_match(layer, got, oracle_run(layer, inp, oracle_signs(inp), pad_value=1),
                     layer.name)


def test_zero_padding_all_minus_one_input_hand_example():
    """1x2x2x32 input of -1, all +1 filters, 3x3 SAME: 4 in-image taps of -1
    and 5 padded zeros give -128 at every pixel (one-padding gives +32)."""
    import paper_2011_09398_amd as lce
    import torch
    x = torch.full((1, 2, 2, 1), -1, dtype=torch.int32, device="cuda")      # all bits set
    w = torch.zeros((1, 3, 3, 1), dtype=torch.int32, device="cuda")         # all +1
    corr = lce.pad_correction(w, 32)
    z = sync_np(lce.bconv2d(x, w, 32, pad_value="zero", pad_correction=corr, out_type="int32"))
    o = sync_np(lce.bconv2d(x, w, 32, pad_value="one", out_type="int32"))
    assert z.reshape(-1).tolist() == [-128] * 4
    assert o.reshape(-1).tolist() == [32] * 4


# ---------------------------------------------------------------- flip + fold

def flip_words(bits):
    """Pack a 0/1 per-channel array into int32 words (bit co%32 of word co/32)."""
    bits = np.asarray(bits, np.uint8)
    words = np.zeros((len(bits) + 31) // 32, np.uint32)
    for co, b in enumerate(bits):
        if b:
            words[co // 32] |= np.uint32(1) << np.uint32(co % 32)
    return words.view(np.int32)


@pytest.mark.parametrize("pad_value", ["one", "zero"])
@pytest.mark.parametrize("c_out", [8, 40, 100])
def test_flip_inverts_chosen_channels(pad_value, c_out):
    layer = Layer(f"flip{c_out}", 2, 9, 7, 96, c_out, out="bitpacked", input_kind="bits")
    inp = make_layer_inputs(layer, 2, 64, c_out)
    rng = np.random.default_rng(c_out)
    fbits = rng.integers(0, 2, c_out).astype(np.uint8)
    words = flip_words(fbits)
    # set every pad bit of the flip words: they must be ignored
    if c_out % 32:
        last = words.view(np.uint32)
        last[-1] |= np.uint32(0xFFFFFFFF) << np.uint32(c_out % 32)
    got = sync_np(gpu_run(layer, inp, pad_value=pad_value, flip=words))
    ref = oracle.bconv2d(oracle_signs(inp), inp.w_sign, stride=1, padding="same",
                         out="bitpacked", thr=inp.thr, flip=fbits,
                         pad_value=0 if pad_value == "zero" else 1)
    assert_match(layer, got, ref, layer.name)


@pytest.mark.parametrize("pad_value", ["one", "zero"])
@pytest.mark.parametrize("shape", [
    # (n, h, w, c_in, c_out, k, stride, clamp)
    (2, 9, 7, 64, 40, 3, 1, None),
    (1, 12, 12, 128, 72, 3, 2, (0, 1152)),
    (3, 6, 5, 33, 13, 5, 1, (-40, 40)),
    (1, 8, 8, 256, 256, 3, 1, None),
])
def test_folded_bitpacked_layer_equals_binarized_float_layer(pad_value, shape):
    """lce_bitpack(float layer with m, b) == bitpacked layer with the folded
    thresholds and flip bits == the oracle's exact signs of fmaf(c, m, b)."""
    import paper_2011_09398_amd as lce
    n, h, w, c_in, c_out, k, s, clamp = shape
    layer = Layer("fold", n, h, w, c_in, c_out, kh=k, kw=k, stride=s, out="float",
                  clamp=clamp, input_kind="bits")
    inp = make_layer_inputs(layer, 8, 65, c_out)
    rng = np.random.default_rng(c_out + k)
    # batch-norm-like parameters of both signs, some zero multipliers
    inp.mult[:] = rng.normal(0.0, 1.0, c_out).astype(np.float32)
    inp.mult[rng.integers(0, c_out, 2)] = 0.0
    inp.bias[:] = rng.normal(0.0, 8.0, c_out).astype(np.float32)
    lo, hi = clamp_of(layer)
    thr, fwords = lce.fold_thresholds(inp.mult, inp.bias, c_out, layer.k, (lo, hi))

    xp, wp = gpu_input(inp), gpu_pack_weights(inp)
    yf = gpu_run(layer, inp, pad_value=pad_value, x_packed=xp, w_packed=wp)
    via_float = sync_np(lce.bitpack(yf))
    bits_layer = Layer("foldb", n, h, w, c_in, c_out, kh=k, kw=k, stride=s, out="bitpacked",
                       clamp=clamp, input_kind="bits")
    folded = sync_np(gpu_run(bits_layer, inp, pad_value=pad_value, x_packed=xp, w_packed=wp,
                             thresholds=thr, flip=fwords))
    # the oracle: exact sign of the float transform on its own accumulators
    pv = 0 if pad_value == "zero" else 1
    c = oracle.clamp(oracle.conv_dot(oracle_signs(inp), inp.w_sign, s, "same", pv), lo, hi)
    signs = np.empty(c.shape, np.int8)
    for co in range(c_out):
        signs[..., co] = 1 - 2 * oracle.sign_of_affine(c[..., co], inp.mult[co],
                                                      inp.bias[co]).astype(np.int8)
    want = oracle.pack(signs.reshape(-1, c_out)).reshape(c.shape[:-1] + (-1,))
    assert np.array_equal(folded.view(np.uint32), want.astype(np.uint32))
    assert np.array_equal(via_float.view(np.uint32), want.astype(np.uint32))
