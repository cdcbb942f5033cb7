"""GPU parity of the matrix-core path (lce_bconv2d_mfma) against the oracle.

The MFMA multiplies +-1 values as 4-bit floats and accumulates in fp32, so
its dot is the exact integer the oracle computes: int32 and bitpacked outputs
must match bit for bit, float outputs within 1e-6 relative.  Zero padding
(0.0 at padded locations) is checked against the oracle's pad_value=0.

Every test runs under each schedule of the path, forced through
lce_set_tuning: the filter-stationary one (each wave keeps its filters in
registers and runs through the workgroup's pixel blocks; the default
wherever one of its instances fits), the K-split one (the four waves of a
workgroup share one output tile and divide K; used where its LDS fits) and
the pixel-split one.  A layer no filter-stationary instance fits runs on
one of the other two.  The batch-64 layers are compared over every output.
"""
import numpy as np
import pytest

import oracle
from tests.layer_util import (assert_match, clamp_of, config4_reference, dev, gpu_input,
                              gpu_pack_weights, oracle_signs, poisoned_out)
from workloads import Layer, config, make_layer_inputs

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


SCHEDULE_NAMES = {"fs": "fs", "ks": "ksplit", "pixel": "pixel"}


@pytest.fixture(autouse=True, params=["fs", "ks", "pixel"])
def schedule(request):
    import paper_2011_09398_amd as lce
    lce.set_tuning(**{k: 0 for k in lce.TUNING_KEYS})
    lce.set_tuning(mfma_schedule=SCHEDULE_NAMES[request.param])
    return request.param


def sync_np(t):
    import torch
    torch.cuda.synchronize()
    return t.cpu().numpy()


def mfma_run(layer, inp, *, pad_value="one", x_packed=None, w_packed=None, thresholds=None,
             flip=None):
    import paper_2011_09398_amd as lce
    x_packed = gpu_input(inp) if x_packed is None else x_packed
    w_packed = gpu_pack_weights(inp) if w_packed is None else w_packed
    wf = lce.mfma_weights(w_packed, layer.c_in)
    kw = {}
    if layer.out == "float":
        kw = dict(multiplier=dev(inp.mult), bias=dev(inp.bias))
    elif layer.out == "bitpacked":
        kw = dict(thresholds=dev(inp.thr if thresholds is None else thresholds),
                  flip=None if flip is None else dev(flip))
    return lce.bconv2d_mfma(x_packed, wf, layer.c_in, layer.c_out, (layer.kh, layer.kw),
                            stride=layer.strides, padding=layer.padding, pad_value=pad_value,
                            clamp=layer.clamp, out_type=layer.out, out=poisoned_out(layer), **kw)


def oracle_run(layer, inp, a_signs, pad_value=1):
    return oracle.bconv2d(a_signs, inp.w_sign, stride=layer.strides, padding=layer.padding,
                          clamp_range=clamp_of(layer), out=layer.out, mult=inp.mult,
                          bias=inp.bias, thr=inp.thr, pad_value=pad_value)


def mfma_cases():
    rng = np.random.default_rng(5150)
    cases = []
    for i in range(60):
        k = int(rng.choice([1, 2, 3, 3, 3, 5, 7]))
        kw = k if rng.random() < 0.8 else int(rng.choice([1, 3]))
        s = int(rng.choice([1, 1, 2, 3]))
        sw_ = s if rng.random() < 0.8 else int(rng.choice([1, 2]))
        padding = "same" if rng.random() < 0.75 else "valid"
        h, w = int(rng.integers(1, 13)), int(rng.integers(1, 13))
        if padding == "valid":
            h, w = max(h, k), max(w, kw)
        c_in = int(rng.choice([1, 7, 32, 33, 64, 96, 100, 128, 160, 256, 512]))
        c_out = int(rng.choice([1, 5, 8, 13, 32, 40, 64, 100, 128, 200]))
        n = int(rng.integers(1, 5))
        out = ["float", "bitpacked", "int32"][i % 3]
        kk = k * kw * c_in
        clamp = [None, (-kk, kk), (0, kk), (-3, 3), (0, 0)][int(rng.integers(0, 5))]
        cases.append(Layer(f"mf{i}", n, h, w, c_in, c_out, kh=k, kw=kw, stride=s,
                           stride_w=sw_, padding=padding, out=out, clamp=clamp,
                           input_kind=["float", "bits"][i % 2]))
    return cases


@pytest.mark.parametrize("pad_value", ["one", "zero"])
@pytest.mark.parametrize("layer", mfma_cases(), ids=lambda l: l.name)
def test_mfma_sweep(layer, pad_value):
    inp = make_layer_inputs(layer, 11, 97, int(layer.name[2:]))
    got = sync_np(mfma_run(layer, inp, pad_value=pad_value))
    ref = oracle_run(layer, inp, oracle_signs(inp), 0 if pad_value == "zero" else 1)
    assert_match(layer, got, ref, f"{layer.name} {pad_value}")


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_mfma_config_parity_full(cfg):
    for i, layer in enumerate(config(cfg)):
        inp = make_layer_inputs(layer, 0, cfg, i)
        got = sync_np(mfma_run(layer, inp))
        assert_match(layer, got, oracle_run(layer, inp, oracle_signs(inp)), layer.name)


def test_mfma_config4_full_batch_chained(schedule):
    """Batch 64 as timed, every output of every layer; the stride-2 layer's
    output feeds the 28x28x128 layer on both sides."""
    prev_gpu = None
    for layer, inp, ref in config4_reference(chain=True):
        x = prev_gpu if layer.chained_from is not None else None
        got = mfma_run(layer, inp, x_packed=x)
        assert_match(layer, sync_np(got), ref, f"{layer.name} {schedule}")
        prev_gpu = got


def test_mfma_config4_default_schedule_full(schedule):
    """The library's own schedule choice (no override) on the batch-64
    layers, every output: the configuration the benchmark times."""
    import paper_2011_09398_amd as lce
    if schedule != "fs":
        pytest.skip("one run suffices: the schedule override is cleared here")
    lce.set_tuning(mfma_schedule=0)
    for layer, inp, ref in config4_reference(chain=False):
        assert_match(layer, sync_np(mfma_run(layer, inp)), ref, f"{layer.name} auto")


@pytest.mark.parametrize("nblk", [1, 2, 4])
def test_mfma_config4_every_filter_split(schedule, nblk):
    """The batch-64 layers at full size, every filter-block split, every
    output."""
    import paper_2011_09398_amd as lce
    if schedule == "fs":
        pytest.skip("the filter-stationary schedule has no filter-block split")
    lce.set_tuning(mfma_tile_n=nblk)
    for layer, inp, ref in config4_reference(chain=False):
        got = sync_np(mfma_run(layer, inp))
        assert_match(layer, got, ref, f"{layer.name} nblk={nblk}")


@pytest.mark.parametrize("mbw,nblk", [(4, 2), (2, 4), (2, 2), (4, 1), (1, 4), (2, 1), (1, 2),
                                      (1, 1)])
def test_mfma_every_tile_shape(schedule, mbw, nblk):
    """Every tile of either schedule: the batch-64 7x7x512 layer (every
    output), a ragged float layer and a stride-2 layer with zero padding."""
    import paper_2011_09398_amd as lce
    if schedule == "pixel" and mbw == 4:
        pytest.skip("the pixel-split schedule takes 1 or 2 pixel blocks per wave")
    if schedule == "fs":
        pytest.skip("the filter-stationary schedule has no such tile (its instances are "
                    "covered by test_mfma_fs_every_instance)")
    lce.set_tuning(mfma_tile_m=mbw, mfma_tile_n=nblk)
    layer, inp, ref = config4_reference(chain=False)[3]
    got = sync_np(mfma_run(layer, inp))
    assert_match(layer, got, ref, f"{layer.name} mb={mbw} nblk={nblk}")
    for lay, pv in ((Layer("rag", 3, 11, 9, 100, 200, out="float", clamp=(-60, 90),
                           input_kind="float"), "one"),
                    (Layer("s2z", 2, 13, 10, 96, 72, stride=2, out="bitpacked",
                           input_kind="bits"), "zero")):
        inp = make_layer_inputs(lay, 4, 93, nblk * 10 + mbw)
        got = sync_np(mfma_run(lay, inp, pad_value=pv))
        ref = oracle_run(lay, inp, oracle_signs(inp), 0 if pv == "zero" else 1)
        assert_match(lay, got, ref, f"{lay.name} mb={mbw} nblk={nblk}")


# Filter-stationary instances (K steps per wave, waves per filter block) and,
# for each, layers whose K steps (taps x ceil(Cw/2), Cw rounded up as the
# widened filters are) need every wave of a filter block: ragged sizes,
# stride 2, non-square filters, every output type, zero padding.
FS_INSTANCES = [(9, 1), (18, 1), (5, 2), (9, 2), (18, 2), (18, 4)]


def fs_layers(ks, s):
    """Layers with (s-1)*ks < K steps <= s*ks."""
    out = []
    for kh, kw in ((3, 3), (1, 1), (5, 5), (3, 1), (2, 3), (1, 5), (7, 7)):
        for cw in range(1, 17):
            cwe = (cw + 1) // 2 * 2 if (cw + 1) // 2 * 2 < (cw + 3) // 4 * 4 else (cw + 3) // 4 * 4
            steps = kh * kw * cwe // 2
            if (s - 1) * ks < steps <= s * ks:
                out.append((kh, kw, cw))
    return out


def cwe_of(cw):
    e2, e4 = (cw + 1) // 2 * 2, (cw + 3) // 4 * 4
    return e2 if e2 < e4 else e4


@pytest.mark.parametrize("packed", [True, False], ids=["packed_filters", "widened_filters"])
@pytest.mark.parametrize("ks,s", FS_INSTANCES, ids=lambda v: str(v))
def test_mfma_fs_every_instance(schedule, ks, s, packed):
    """packed: C_in fills every widened word (C_in = 32*Cw'), where the kernel
    loads the packed filter copy and widens it itself; otherwise some
    channels are padding and it loads the widened filters."""
    import paper_2011_09398_amd as lce
    if schedule != "fs":
        pytest.skip("filter-stationary instances")
    lce.set_tuning(mfma_fs_ks=ks, mfma_fs_s=s)
    shapes = fs_layers(ks, s)
    assert shapes, (ks, s)
    rng = np.random.default_rng(ks * 10 + s + (1000 if packed else 0))
    picks = [shapes[0], shapes[-1]] + [shapes[int(i)] for i in rng.integers(0, len(shapes), 2)]
    for j, (kh, kw, cw) in enumerate(picks):
        c_in = 32 * cwe_of(cw) if packed else 32 * cw - int(rng.integers(1, 32))
        c_out = int(rng.choice([13, 32, 64, 100, 128, 200]))
        stride = int(rng.choice([1, 2]))
        out = ["float", "bitpacked", "int32", "bitpacked"][j]
        pv = ["one", "zero"][j % 2]
        k = kh * kw * c_in
        layer = Layer(f"fs{ks}x{s}_{j}", int(rng.integers(1, 4)), int(rng.integers(kh, 15)),
                      int(rng.integers(kw, 15)), c_in, c_out, kh=kh, kw=kw, stride=stride,
                      padding=["same", "valid"][j % 2], out=out,
                      clamp=[None, (-k // 3, k // 2)][j % 2], input_kind="bits")
        inp = make_layer_inputs(layer, 7, 91, ks * 100 + s * 10 + j)
        flip = None
        if out == "bitpacked" and j == 3:
            flip = rng.integers(0, 2**31, (c_out + 31) // 32).astype(np.int32)
        got = sync_np(mfma_run(layer, inp, pad_value=pv, flip=flip))
        if flip is not None:
            fbits = np.array([(int(flip[c // 32]) >> (c % 32)) & 1 for c in range(c_out)],
                             np.uint8)
            ref = oracle.bconv2d(oracle_signs(inp), inp.w_sign, stride=layer.strides,
                                 padding=layer.padding, clamp_range=clamp_of(layer),
                                 out="bitpacked", thr=inp.thr, flip=fbits,
                                 pad_value=0 if pv == "zero" else 1)
        else:
            ref = oracle_run(layer, inp, oracle_signs(inp), 0 if pv == "zero" else 1)
        assert_match(layer, got, ref, f"{layer.name} {kh}x{kw} cw={cw} {pv}")


# Layers whose filter-stationary shares are shorter than an output row, so
# that each workgroup stages only its share's window of padded columns (or
# whole rows over fewer padded rows): stride 1, 2, 3 and (1, 2), one and two
# filter blocks per workgroup, SAME and VALID padding, several images.
WINDOW_LAYERS = [
    Layer("win_s1", 1, 20, 24, 64, 100, out="float", clamp=None),
    Layer("win_s2", 2, 17, 23, 96, 64, stride=2, out="bitpacked"),
    Layer("win_s12", 1, 13, 30, 128, 40, stride=1, stride_w=2, out="int32", clamp=(-200, 300)),
    Layer("win_s3", 1, 11, 40, 64, 200, stride=3, out="bitpacked"),
    Layer("win_valid", 3, 9, 16, 256, 72, padding="valid", out="float", clamp=(-500, 700)),
    Layer("win_c1", 1, 30, 32, 32, 32, padding="valid", out="bitpacked"),
    # a prime output width (no divisor short of the whole row: whole-row
    # shares over fewer rows) and a one-column image (nothing to round)
    Layer("win_prime", 2, 13, 13, 64, 72, out="bitpacked"),
    Layer("win_ow1", 4, 9, 1, 64, 64, out="float", clamp=(-100, 200)),
]


@pytest.mark.parametrize("pad_value", ["one", "zero"])
@pytest.mark.parametrize("layer", WINDOW_LAYERS, ids=lambda l: l.name)
def test_mfma_fs_column_window(schedule, layer, pad_value):
    """Staging each share's window of columns gives the oracle's output, the
    same as staging whole padded rows (tuning key mfma_fs_window = -1)."""
    import paper_2011_09398_amd as lce
    if schedule != "fs":
        pytest.skip("filter-stationary windows")
    inp = make_layer_inputs(layer, 13, 77, WINDOW_LAYERS.index(layer))
    got = sync_np(mfma_run(layer, inp, pad_value=pad_value))
    ref = oracle_run(layer, inp, oracle_signs(inp), 0 if pad_value == "zero" else 1)
    assert_match(layer, got, ref, f"{layer.name} {pad_value}")
    lce.set_tuning(mfma_fs_window=-1)
    rows = sync_np(mfma_run(layer, inp, pad_value=pad_value))
    assert np.array_equal(got.view(np.uint32), rows.view(np.uint32)), layer.name


@pytest.mark.parametrize("ks,s", FS_INSTANCES, ids=lambda v: str(v))
def test_mfma_fs_repeated_launches(schedule, ks, s):
    """Four launches of the same layer, each into a fresh poisoned output,
    all equal to the oracle: layers whose workgroups hold a single pixel
    block, where the waves without a block of their own compute values they
    never store (a kernel once read unassigned registers there and returned
    wrong bits from the second launch on), every output type."""
    import paper_2011_09398_amd as lce
    if schedule != "fs":
        pytest.skip("filter-stationary instances")
    lce.set_tuning(mfma_fs_ks=ks, mfma_fs_s=s)
    shapes = fs_layers(ks, s)
    for j, out in enumerate(["bitpacked", "float", "int32"]):
        kh, kw, cw = shapes[(j * 7) % len(shapes)]
        k = kh * kw * 32 * cwe_of(cw)
        layer = Layer(f"rep{ks}x{s}_{j}", 3, 12, 14, 32 * cwe_of(cw), 200, kh=kh, kw=kw,
                      padding="valid", out=out, clamp=(-k // 3, k // 2), input_kind="bits")
        inp = make_layer_inputs(layer, 8, 94, ks * 10 + s + j)
        ref = oracle_run(layer, inp, oracle_signs(inp))
        x, w = gpu_input(inp), gpu_pack_weights(inp)
        for r in range(4):
            got = sync_np(mfma_run(layer, inp, x_packed=x, w_packed=w))
            assert_match(layer, got, ref, f"{layer.name} launch {r}")


@pytest.mark.parametrize("wpc", ["1", "2"])
@pytest.mark.parametrize("ks,s", [(9, 1), (18, 1), (9, 2)], ids=lambda v: str(v))
def test_mfma_fs_workgroups_per_cu(schedule, ks, s, wpc):
    """One or two workgroups per CU (the grid and the pixel share per
    workgroup change, the result does not): ragged layers, stride 2."""
    import paper_2011_09398_amd as lce
    if schedule != "fs":
        pytest.skip("filter-stationary grids")
    lce.set_tuning(mfma_fs_ks=ks, mfma_fs_s=s, mfma_fs_wpc=int(wpc))
    for j, (kh, kw, cw) in enumerate(fs_layers(ks, s)[:2]):
        layer = Layer(f"wpc{ks}x{s}_{j}", 5, 19 - j, 23, 32 * cwe_of(cw) - 7 * j, 96 + 40 * j,
                      kh=kh, kw=kw, stride=1 + j, out=["bitpacked", "float"][j],
                      input_kind="bits")
        inp = make_layer_inputs(layer, 3, 89, ks * 10 + s + j)
        got = sync_np(mfma_run(layer, inp))
        assert_match(layer, got, oracle_run(layer, inp, oracle_signs(inp)),
                     f"{layer.name} wpc={wpc}")


@pytest.mark.parametrize("packed", ["1", "0"], ids=["packed_filters", "widened_filters"])
def test_mfma_fs_config4_every_instance_that_fits(schedule, packed):
    """The batch-64 layers at full size (every output) on every
    filter-stationary instance whose K steps fit the layer, loading the
    packed filter copy (the default there) or the widened filters."""
    import paper_2011_09398_amd as lce
    if schedule != "fs":
        pytest.skip("filter-stationary instances")
    lce.set_tuning(mfma_packed=1 if packed == "1" else -1)
    for layer, inp, ref in config4_reference(chain=False):
        steps = layer.kh * layer.kw * ((layer.cw + 1) // 2)
        for ks, s in FS_INSTANCES:
            if not ((s - 1) * ks < steps <= s * ks):
                continue
            lce.set_tuning(mfma_fs_ks=ks, mfma_fs_s=s)
            got = sync_np(mfma_run(layer, inp))
            assert_match(layer, got, ref, f"{layer.name} fs {ks}x{s}")


def test_mfma_wide_region_falls_back_to_the_pixel_split():
    """A region too wide for the K-split schedule's LDS (every word of a
    2048-channel, 60-column region) runs on the pixel-split schedule."""
    layer = Layer("wide", 1, 5, 60, 2048, 40, out="int32", input_kind="bits")
    inp = make_layer_inputs(layer, 6, 92, 0)
    got = sync_np(mfma_run(layer, inp))
    assert_match(layer, got, oracle_run(layer, inp, oracle_signs(inp)), layer.name)


def test_mfma_config5_chain_every_layer():
    """The 12-layer batch-16 stack, each layer fed the previous MFMA output."""
    layers = config(5)
    prev_gpu = prev_ref = None
    for i, layer in enumerate(layers):
        inp = make_layer_inputs(layer, 0, 5, i)
        if prev_gpu is None:
            x, a = gpu_input(inp), oracle_signs(inp)
        else:
            x, a = prev_gpu, oracle.unpack(prev_ref, layer.c_in)
        got = mfma_run(layer, inp, x_packed=x)
        ref = oracle_run(layer, inp, a)
        assert_match(layer, sync_np(got), ref, f"stack {layer.name}")
        prev_gpu, prev_ref = got, ref


def test_mfma_matches_xor_path_bit_for_bit():
    """Both implementations of LceBConv2d give identical outputs."""
    from tests.layer_util import gpu_layer
    for layer in (Layer("eqf", 2, 9, 7, 96, 72, out="float", clamp=(-40, 50), input_kind="bits"),
                  Layer("eqb", 3, 14, 14, 256, 256, out="bitpacked", input_kind="bits"),
                  Layer("eqs", 2, 12, 12, 64, 128, stride=2, out="int32", input_kind="bits")):
        inp = make_layer_inputs(layer, 2, 96, layer.c_out)
        xp, wp = gpu_input(inp), gpu_pack_weights(inp)
        a = sync_np(gpu_layer(layer, inp, x_packed=xp, w_packed=wp))
        b = sync_np(mfma_run(layer, inp, x_packed=xp, w_packed=wp))
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), layer.name


def test_mfma_flip_and_special_thresholds():
    layer = Layer("mthr", 2, 9, 7, 64, 72, out="bitpacked", input_kind="bits", clamp=(-20, 30))
    inp = make_layer_inputs(layer, 5, 95, 0)
    inp.thr[:10] = [-20.0, -20.5, -19.5, 30.0, 30.5, 31.0, np.inf, -np.inf, np.nan, 0.0]
    rng = np.random.default_rng(3)
    fbits = rng.integers(0, 2, 72).astype(np.uint8)
    words = np.zeros(3, np.uint32)
    for co, b in enumerate(fbits):
        if b:
            words[co // 32] |= np.uint32(1) << np.uint32(co % 32)
    words[2] |= np.uint32(0xFFFFFF00)                 # pad bits must be ignored
    got = sync_np(mfma_run(layer, inp, flip=words.view(np.int32)))
    ref = oracle.bconv2d(oracle_signs(inp), inp.w_sign, out="bitpacked", thr=inp.thr,
                         clamp_range=(-20, 30), flip=fbits)
    assert_match(layer, got, ref, layer.name)


def test_mfma_weights_are_zero_past_the_real_channels_and_filters():
    """Widened filters: +-1.0 codes for real weights, 0.0 for pad channels,
    pad words and pad filters (checked against the oracle-side signs); the
    packed copy after them: bit 1 = -1, 0 for pad channels, words, filters."""
    import paper_2011_09398_amd as lce
    layer = Layer("wx", 1, 4, 4, 40, 13, kh=3, kw=3, input_kind="bits")
    inp = make_layer_inputs(layer, 1, 94, 0)
    raw = sync_np(lce.mfma_weights(gpu_pack_weights(inp), 40)).view(np.uint32)
    cw, cwe, coutp, taps = 2, 2, 32, 9
    n = taps * cwe * coutp
    assert raw.size == n * 4 + n
    packed = raw[n * 4:].reshape(taps * cwe, coutp)
    codes = np.zeros((taps * cwe, coutp, 32), np.uint8)
    words = raw[:n * 4].reshape(taps * cwe, coutp, 4)
    for j in range(32):                       # channel j: 32-bit word j % 4, nibble j // 4
        codes[..., j] = (words[..., j % 4] >> np.uint32(4 * (j // 4))) & 0xF
    want = np.zeros_like(codes)
    w = inp.w_sign.reshape(13, taps, 40)
    for t in range(taps):
        for c in range(40):
            want[t * cwe + c // 32, :13, c % 32] = np.where(w[:, t, c] > 0, 0x2, 0xA)
    assert np.array_equal(codes, want)
    want_bits = np.zeros((taps * cwe, coutp), np.uint32)
    for t in range(taps):
        for c in range(40):
            want_bits[t * cwe + c // 32, :13] |= (w[:, t, c] < 0).astype(np.uint32) << np.uint32(c % 32)
    assert np.array_equal(packed, want_bits)
