"""GPU parity of the quantize-fused matrix-core convolution
(lce_quantize_bconv2d_mfma).

The float input is binarized while the filter-stationary or the K-split
kernel stages its region.  The output must equal the oracle's binarize + bconv2d (bit for bit
for bitpacked and int32 outputs, within the float tolerance for float
outputs; the dot is the exact integer either way), and equal lce_bitpack +
lce_bconv2d_mfma on the same device buffers bit for bit.  Shapes neither
schedule takes must be refused before anything is launched.  Output buffers are poisoned first.
"""
import numpy as np
import pytest

import oracle
from tests.layer_util import assert_match, clamp_of, dev, gpu_pack_weights, poisoned_out
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


@pytest.fixture(autouse=True)
def automatic_schedule():
    import paper_2011_09398_amd as lce
    lce.set_tuning(**{k: 0 for k in lce.TUNING_KEYS})
    yield
    lce.set_tuning(**{k: 0 for k in lce.TUNING_KEYS})


def sync_np(t):
    import torch
    torch.cuda.synchronize()
    return t.cpu().numpy()


def epilogue_kw(layer, inp, flip=None):
    if layer.out == "float":
        return dict(multiplier=dev(inp.mult), bias=dev(inp.bias))
    if layer.out == "bitpacked":
        return dict(thresholds=dev(inp.thr), flip=None if flip is None else dev(flip))
    return {}


def fused(layer, inp, x, w_fp4, pad_value="one", flip=None, out=None):
    import paper_2011_09398_amd as lce
    return lce.quantize_bconv2d_mfma(x, w_fp4, layer.c_out, (layer.kh, layer.kw),
                                     stride=layer.strides, padding=layer.padding,
                                     pad_value=pad_value, clamp=layer.clamp,
                                     out_type=layer.out,
                                     out=poisoned_out(layer) if out is None else out,
                                     **epilogue_kw(layer, inp, flip))


def unfused(layer, inp, x, w_fp4, pad_value="one", flip=None):
    import paper_2011_09398_amd as lce
    return lce.bconv2d_mfma(lce.bitpack(x), w_fp4, layer.c_in, layer.c_out,
                            (layer.kh, layer.kw), stride=layer.strides, padding=layer.padding,
                            pad_value=pad_value, clamp=layer.clamp, out_type=layer.out,
                            out=poisoned_out(layer), **epilogue_kw(layer, inp, flip))


def reference(layer, inp, x_float, pad_value="one", flip_bits=None):
    return oracle.bconv2d(oracle.binarize(x_float), inp.w_sign, stride=layer.strides,
                          padding=layer.padding, clamp_range=clamp_of(layer), out=layer.out,
                          mult=inp.mult, bias=inp.bias, thr=inp.thr, flip=flip_bits,
                          pad_value=0 if pad_value == "zero" else 1)


def k_steps(layer):
    return layer.kh * layer.kw * ((layer.cw + 1) // 2)


def taken(layer):
    """Filter-stationary where one of its instances takes the layer, else the
    K split from 20 K steps."""
    return fs_takes(layer) or k_steps(layer) >= 20


def fs_takes(layer):
    """Whether a filter-stationary instance (KS K steps per wave, S waves per
    filter block) covers the layer's K steps with every wave busy and at
    most 1/8 of them padding, within the fused plan's 72 K steps."""
    steps = k_steps(layer)
    return steps <= 72 and any(ks * s >= steps > ks * (s - 1) and (ks * s - steps) * 8 <= steps
                               for ks, s in FS_INSTANCES)


def check(layer, inp, what, pad_value="one", x_float=None):
    """Parity with the oracle and with bitpack + bconv2d_mfma; returns False
    (after checking that nothing was written) where the shape is refused."""
    import paper_2011_09398_amd as lce
    x_float = inp.x_float if x_float is None else x_float
    x = dev(x_float)
    w_fp4 = lce.mfma_weights(gpu_pack_weights(inp), layer.c_in)
    out = poisoned_out(layer)
    try:
        got = sync_np(fused(layer, inp, x, w_fp4, pad_value, out=out))
    except lce.LceError as e:
        assert e.status == lce.LCE_EUNSUPPORTED, (what, e)
        assert "filter-stationary" in str(e), (what, e)
        poison = sync_np(poisoned_out(layer))
        assert np.array_equal(sync_np(out).view(np.uint32), poison.view(np.uint32)), what
        return False
    assert_match(layer, got, reference(layer, inp, x_float, pad_value), what)
    assert np.array_equal(got.view(np.uint32),
                          sync_np(unfused(layer, inp, x, w_fp4, pad_value)).view(np.uint32)), what
    return True


# ------------------------------------------------ the float-input layers of the workloads

@pytest.mark.parametrize("cfg,idx", [(1, 0), (2, 0), (3, 0), (3, 1), (3, 2), (3, 3)])
def test_batch1_configs(cfg, idx):
    layer = config(cfg)[idx]
    assert layer.input_kind == "float"
    # every one of them is taken (the 72-K-step 7x7x512 one by the (18, 4)
    # filter-stationary instance)
    assert check(layer, make_layer_inputs(layer, 0, cfg, idx), f"config {cfg} layer {idx}")
    assert taken(layer)


def test_stack_first_layer_full_batch():
    layer = config(5)[0]                     # batch 16, float input, bitpacked output
    assert check(layer, make_layer_inputs(layer, 0, 5, 0), "config 5 L1")


# ------------------------------------------------ geometry, ragged edges, outputs, padding

SHAPES = [
    # n, h, w, c_in, c_out, kh, kw, stride, padding, out
    (1, 9, 13, 64, 40, 3, 3, 1, "same", "float"),
    (2, 7, 7, 96, 33, 3, 3, 1, "same", "bitpacked"),
    (5, 3, 3, 32, 64, 3, 3, 1, "same", "int32"),
    (1, 40, 6, 64, 32, 3, 3, 1, "same", "float"),
    (2, 5, 200, 32, 16, 3, 3, 1, "same", "int32"),
    (1, 17, 11, 128, 128, 3, 3, 2, "valid", "float"),
    (4, 6, 9, 256, 256, 3, 3, 1, "same", "float"),
    (1, 1, 1, 32, 8, 3, 3, 1, "same", "int32"),
    (2, 31, 33, 64, 130, 3, 3, 2, "same", "bitpacked"),
    (2, 7, 9, 512, 100, 1, 1, 1, "same", "int32"),        # 8 K steps
    (2, 10, 8, 192, 64, 3, 1, 2, "same", "bitpacked"),    # 9 K steps
    (1, 12, 12, 128, 40, 1, 5, 1, "same", "float"),       # 10 K steps
    (3, 9, 6, 32, 72, 5, 5, 2, "same", "bitpacked"),      # 25 K steps: K split
    (2, 9, 7, 160, 90, 3, 3, 1, "same", "float"),         # 27 K steps: K split
    (1, 8, 8, 512, 64, 3, 3, 1, "same", "bitpacked"),     # 72 K steps: K split
    (3, 12, 10, 128, 200, 1, 1, 1, "valid", "int32"),     # 2 K steps: refused
]


@pytest.mark.parametrize("pad_value", ["one", "zero"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s[:5])) +
                         f"_k{s[5]}x{s[6]}s{s[7]}{s[8]}_{s[9]}")
def test_shapes(shape, pad_value):
    n, h, w, ci, co, kh, kw, s, pad, out = shape
    k = kh * kw * ci
    clamp = (-k // 3, k // 2) if out != "bitpacked" else None
    layer = Layer("qfm", n, h, w, ci, co, kh=kh, kw=kw, stride=s, padding=pad, out=out,
                  clamp=clamp, input_kind="float")
    was_taken = check(layer, make_layer_inputs(layer, 1, 0, 11), layer.name, pad_value)
    assert was_taken == taken(layer), (layer.name, k_steps(layer))


# ------------------------------------------------ every filter-stationary instance

FS_INSTANCES = [(9, 1), (18, 1), (5, 2), (9, 2), (18, 2), (18, 4)]


def fs_shapes(ks, s):
    """(kh, kw, C_in) whose K steps need every wave of a filter block."""
    out = []
    for kh, kw in ((3, 3), (1, 1), (5, 5), (3, 1), (1, 5)):
        for cw in range(1, 17):
            steps = kh * kw * ((cw + 1) // 2)
            if (s - 1) * ks < steps <= s * ks:
                out.append((kh, kw, 32 * cw))
    return out


@pytest.mark.parametrize("packed", [1, -1], ids=["packed_filters", "widened_filters"])
@pytest.mark.parametrize("ks,s", FS_INSTANCES, ids=lambda v: str(v))
def test_every_instance(ks, s, packed):
    """Each instance forced (tuning keys), loading the packed filter copy or
    the widened filters, on ragged layers of every output kind."""
    import paper_2011_09398_amd as lce
    lce.set_tuning(mfma_fs_ks=ks, mfma_fs_s=s, mfma_packed=packed)
    shapes = fs_shapes(ks, s)
    assert shapes, (ks, s)
    rng = np.random.default_rng(ks * 10 + s + (100 if packed > 0 else 0))
    picks = [shapes[0], shapes[-1], shapes[int(rng.integers(0, len(shapes)))]]
    for j, (kh, kw, ci) in enumerate(picks):
        out = ["float", "bitpacked", "int32"][j]
        k = kh * kw * ci
        layer = Layer(f"inst{ks}x{s}_{j}", int(rng.integers(1, 4)), int(rng.integers(kh, 14)),
                      int(rng.integers(kw, 14)), ci, int(rng.choice([13, 64, 100, 200])),
                      kh=kh, kw=kw, stride=int(rng.choice([1, 2])), out=out,
                      clamp=None if out == "bitpacked" else (-k // 3, k // 2),
                      input_kind="float")
        assert check(layer, make_layer_inputs(layer, 2, 0, ks * 10 + s + j),
                     f"{layer.name} {kh}x{kw} c_in={ci}", ["one", "zero"][j % 2])


@pytest.mark.parametrize("mbw,nblk", [(4, 2), (2, 4), (2, 2), (4, 1), (1, 4), (2, 1), (1, 2),
                                      (1, 1)])
def test_ksplit_every_tile(mbw, nblk):
    """Each K-split tile forced (tuning keys): configuration 3's 7x7x512
    layer and ragged layers with zero padding and a stride."""
    import paper_2011_09398_amd as lce
    lce.set_tuning(mfma_schedule="ksplit", mfma_tile_m=mbw, mfma_tile_n=nblk)
    idx, layer = next((i, l) for i, l in enumerate(config(3)) if l.c_in == 512)
    assert k_steps(layer) == 72
    assert check(layer, make_layer_inputs(layer, 0, 3, idx), f"7x7x512 mb={mbw} nblk={nblk}")
    for j, (lay, pv) in enumerate(((Layer("rk", 3, 11, 9, 160, 200, out="float",
                                          clamp=(-60, 90), input_kind="float"), "one"),
                                   (Layer("s2z", 2, 13, 10, 96, 136, kh=5, kw=5, stride=2,
                                          out="bitpacked", input_kind="float"), "zero"))):
        assert check(lay, make_layer_inputs(lay, 5, 0, 40 + 10 * nblk + mbw + j),
                     f"{lay.name} mb={mbw} nblk={nblk}", pv)


@pytest.mark.parametrize("sched", ["ksplit", "fs"])
def test_schedule_key(sched):
    """The mfma_schedule key restricts the fused entry to one schedule: the K
    split on layers of 9 and 18 K steps (which the default plan gives to the
    filter-stationary schedule), the filter-stationary one on configuration
    3's 7x7x512 layer (72 K steps) and on a 5x5 layer of 50 K steps that no
    instance takes (refused)."""
    import paper_2011_09398_amd as lce
    lce.set_tuning(mfma_schedule=sched)
    if sched == "ksplit":
        for j, layer in enumerate((Layer("k9", 2, 15, 13, 64, 72, out="bitpacked",
                                         input_kind="float"),
                                   Layer("k18", 1, 11, 12, 128, 100, stride=2, out="float",
                                         clamp=(-300, 500), input_kind="float"))):
            assert k_steps(layer) in (9, 18)
            assert check(layer, make_layer_inputs(layer, 6, 0, 50 + j), f"{layer.name} ksplit",
                         ["one", "zero"][j])
    else:
        idx, layer = next((i, l) for i, l in enumerate(config(3)) if l.c_in == 512)
        assert check(layer, make_layer_inputs(layer, 0, 3, idx), "7x7x512 fs")
        lay = Layer("k50", 1, 9, 9, 128, 64, kh=5, kw=5, out="float", input_kind="float")
        assert k_steps(lay) == 50
        assert not check(lay, make_layer_inputs(lay, 6, 0, 60), "k50 fs refused")


@pytest.mark.parametrize("layer", [
    Layer("win_f1", 1, 20, 24, 64, 100, out="float", clamp=None, input_kind="float"),
    Layer("win_f2", 2, 17, 23, 96, 64, stride=2, out="bitpacked", input_kind="float"),
    Layer("win_f12", 1, 13, 30, 128, 40, stride=1, stride_w=2, out="int32", clamp=(-200, 300),
          input_kind="float"),
    Layer("rows_f", 1, 7, 7, 512, 512, out="bitpacked", input_kind="float"),
], ids=lambda l: l.name)
def test_column_windows_and_row_rounding(layer):
    """Shares within one output row stage only their window of columns (or,
    where the window is the whole row, fewer rows): the oracle's output, the
    same as with whole-row shares (tuning key mfma_fs_window = -1), one and
    zero padding."""
    import paper_2011_09398_amd as lce
    for j, pv in enumerate(("one", "zero")):
        inp = make_layer_inputs(layer, 8, 0, 70 + j)
        lce.set_tuning(mfma_fs_window=0)
        assert check(layer, inp, f"{layer.name} {pv}", pv)
        x = dev(inp.x_float)
        w_fp4 = lce.mfma_weights(gpu_pack_weights(inp), layer.c_in)
        win = sync_np(fused(layer, inp, x, w_fp4, pv))
        lce.set_tuning(mfma_fs_window=-1)
        rows = sync_np(fused(layer, inp, x, w_fp4, pv))
        assert np.array_equal(win.view(np.uint32), rows.view(np.uint32)), (layer.name, pv)
    lce.set_tuning(mfma_fs_window=0)


@pytest.mark.parametrize("wpc", [1, 2])
def test_workgroups_per_cu(wpc):
    import paper_2011_09398_amd as lce
    lce.set_tuning(mfma_fs_wpc=wpc)
    for j, layer in enumerate((Layer("w1", 5, 19, 23, 64, 96, out="bitpacked", input_kind="float"),
                               Layer("w2", 3, 18, 17, 128, 136, stride=2, out="float",
                                     input_kind="float"))):
        assert check(layer, make_layer_inputs(layer, 3, 0, 20 + j), f"{layer.name} wpc={wpc}")


def test_repeated_launches_into_fresh_outputs():
    """Four launches, each into a fresh poisoned output, all equal to the
    oracle (layers whose workgroups hold a single pixel block)."""
    import paper_2011_09398_amd as lce
    for j, (ks, s) in enumerate(((9, 1), (18, 2))):
        lce.set_tuning(mfma_fs_ks=ks, mfma_fs_s=s)
        ci = 64 if ks == 9 else 256
        layer = Layer(f"rep{j}", 3, 12, 14, ci, 200, padding="valid", out="bitpacked",
                      input_kind="float")
        inp = make_layer_inputs(layer, 4, 0, 30 + j)
        x = dev(inp.x_float)
        w_fp4 = lce.mfma_weights(gpu_pack_weights(inp), ci)
        ref = reference(layer, inp, inp.x_float)
        for r in range(4):
            assert_match(layer, sync_np(fused(layer, inp, x, w_fp4)), ref, f"{layer.name} {r}")


# ------------------------------------------------ the sign test and the flip mask

def test_sign_test_special_values():
    # -0.0 and NaN are +1 (bit 0), -inf and negative denormals -1, as lce_bitpack
    layer = Layer("special", 1, 6, 6, 64, 32, out="int32", input_kind="float")
    inp = make_layer_inputs(layer, 0, 0, 3)
    x = inp.x_float.copy()
    flat = x.reshape(-1)
    special = np.array([-0.0, 0.0, np.nan, -np.nan, np.inf, -np.inf, 1e-45, -1e-45],
                       np.float32)
    flat[::7] = np.resize(special, flat[::7].size)
    assert check(layer, inp, "special floats", x_float=x)


def test_flip_mask():
    import paper_2011_09398_amd as lce
    layer = Layer("flip", 2, 10, 10, 64, 70, out="bitpacked", input_kind="float")
    inp = make_layer_inputs(layer, 0, 0, 4)
    flip = np.array([0x0F0F00F1, 0x7FFFFFFF, 0xFFFFFFF3], dtype=np.uint32).view(np.int32)
    fbits = (oracle.unpack(flip.view(np.uint32)[None], 70)[0] < 0).astype(np.uint8)
    x = dev(inp.x_float)
    w_fp4 = lce.mfma_weights(gpu_pack_weights(inp), 64)
    got = sync_np(fused(layer, inp, x, w_fp4, flip=flip))
    assert_match(layer, got, reference(layer, inp, inp.x_float, flip_bits=fbits), "flip")
    assert np.array_equal(got, sync_np(unfused(layer, inp, x, w_fp4, flip=flip)))


# ------------------------------------------------ refusals and graph capture

def test_unsupported_requests_raise_before_launch():
    import torch
    import paper_2011_09398_amd as lce
    w_fp4 = torch.zeros(1 << 20, dtype=torch.int32, device="cuda")
    # C_in not a multiple of 32
    x = torch.zeros((1, 8, 8, 40), dtype=torch.float32, device="cuda")
    with pytest.raises(lce.LceError) as e:
        lce.quantize_bconv2d_mfma(x, w_fp4, 8, 3)
    assert e.value.status == lce.LCE_EUNSUPPORTED
    # x off 16-byte alignment
    base = torch.zeros(8 * 8 * 64 + 4, dtype=torch.float32, device="cuda")
    x = base[1:1 + 8 * 8 * 64].view(1, 8, 8, 64)
    with pytest.raises(lce.LceError) as e:
        lce.quantize_bconv2d_mfma(x, w_fp4, 8, 3)
    assert e.value.status == lce.LCE_EALIGN


def test_graph_replay_matches_eager():
    import torch
    import paper_2011_09398_amd as lce
    layer = config(2)[0]
    inp = make_layer_inputs(layer, 0, 2, 0)
    x = dev(inp.x_float)
    w_fp4 = lce.mfma_weights(gpu_pack_weights(inp), layer.c_in)
    out = poisoned_out(layer)
    call = lce.PreparedQuantBConv2dMfma(x, w_fp4, layer.c_out, (layer.kh, layer.kw), out,
                                        stride=layer.strides, padding=layer.padding,
                                        clamp=layer.clamp, out_type=layer.out,
                                        **epilogue_kw(layer, inp))
    eager = sync_np(out).copy()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            call()
    torch.cuda.current_stream().wait_stream(s)
    for _ in range(3):
        out.fill_(float("nan"))
        g.replay()
        assert np.array_equal(sync_np(out).view(np.uint32), eager.view(np.uint32))
