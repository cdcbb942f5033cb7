"""GPU parity of the quantize-fused convolution (lce_quantize_bconv2d).

The float input is binarized inside the convolution's workgroups.  Its
output must equal the oracle's binarize + bconv2d (bit for bit for packed
and int32 outputs, within the float tolerance for float outputs), and equal
lce_bitpack + lce_bconv2d on the same device buffers bit for bit (both apply
the same float output transform).  Output buffers are poisoned first.
"""
import ctypes

import numpy as np
import pytest

import oracle
from tests.layer_util import (POISON_I32, assert_match, dev, gpu_pack_weights, oracle_layer,
                              poisoned_out)
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


def sync_np(t):
    import torch
    torch.cuda.synchronize()
    return t.cpu().numpy()


def epilogue_kw(layer, inp):
    if layer.out == "float":
        return dict(multiplier=dev(inp.mult), bias=dev(inp.bias))
    if layer.out == "bitpacked":
        return dict(thresholds=dev(inp.thr))
    return {}


def fused(layer, inp, x=None, w=None, out=None):
    import paper_2011_09398_amd as lce
    x = dev(inp.x_float) if x is None else x
    w = gpu_pack_weights(inp) if w is None else w
    out = poisoned_out(layer) if out is None else out
    return lce.quantize_bconv2d(x, w, stride=layer.strides, padding=layer.padding,
                                clamp=layer.clamp, out_type=layer.out, out=out,
                                **epilogue_kw(layer, inp))


def unfused(layer, inp, x, w):
    import paper_2011_09398_amd as lce
    return lce.bconv2d(lce.bitpack(x), w, layer.c_in, stride=layer.strides,
                       padding=layer.padding, clamp=layer.clamp, out_type=layer.out,
                       out=poisoned_out(layer), **epilogue_kw(layer, inp))


def check(layer, cfg=0, idx=0, what=""):
    inp = make_layer_inputs(layer, 0, cfg, idx)
    x, w = dev(inp.x_float), gpu_pack_weights(inp)
    got = sync_np(fused(layer, inp, x, w))
    ref = oracle_layer(layer, inp, oracle.binarize(inp.x_float))
    assert_match(layer, got, ref, what or layer.name)
    assert np.array_equal(got.view(np.uint32), sync_np(unfused(layer, inp, x, w)).view(np.uint32))


# ------------------------------------------------ the float-input layers of the workloads

@pytest.mark.parametrize("cfg,idx", [(1, 0), (2, 0), (3, 0), (3, 1), (3, 2), (3, 3)])
def test_batch1_configs(cfg, idx):
    layer = config(cfg)[idx]
    assert layer.input_kind == "float"
    check(layer, cfg, idx, f"config {cfg} layer {idx}")


def test_stack_first_layer_full_batch():
    # configuration 5's first layer: batch 16, float input, bitpacked output
    layer = config(5)[0]
    check(layer, 5, 0, "config 5 L1")


# ------------------------------------------------ geometry, ragged edges, output kinds

SHAPES = [
    # n, h, w, c_in, c_out, k, stride, padding, out
    (1, 9, 13, 64, 40, 3, 1, "same", "float"),
    (2, 7, 7, 96, 33, 3, 1, "same", "bitpacked"),     # 49-pixel images: bands cross images
    (5, 3, 3, 32, 64, 3, 1, "same", "int32"),         # 9-pixel images, several per block
    (1, 40, 6, 64, 32, 3, 1, "same", "float"),        # narrow: a block spans 11 rows
    (2, 5, 200, 32, 16, 3, 1, "same", "int32"),       # wide: a block inside one row
    (1, 21, 37, 64, 48, 5, 3, "same", "bitpacked"),   # stride 3
    (3, 5, 4, 160, 96, 3, 2, "same", "bitpacked"),
    (1, 17, 11, 128, 128, 3, 2, "valid", "float"),
    (2, 12, 12, 192, 64, 3, 1, "valid", "int32"),
    (1, 16, 16, 64, 64, 5, 1, "same", "float"),
    (3, 9, 6, 128, 72, 5, 2, "same", "bitpacked"),
    (1, 8, 8, 512, 512, 3, 1, "same", "bitpacked"),
    (4, 6, 9, 256, 256, 3, 1, "same", "float"),
    (1, 1, 1, 32, 8, 3, 1, "same", "int32"),           # one pixel: every tap but one padded
    (2, 31, 33, 64, 130, 3, 2, "same", "bitpacked"),   # ragged filter tail and tiles
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s[:5])) +
                         f"_k{s[5]}s{s[6]}{s[7]}_{s[8]}")
def test_shapes(shape):
    n, h, w, ci, co, k, s, pad, out = shape
    clamp = (-(k * k * ci) // 3, k * k * ci // 2) if out != "bitpacked" else None
    layer = Layer("fused", n, h, w, ci, co, kh=k, kw=k, stride=s, padding=pad, out=out,
                  clamp=clamp)
    check(layer, 0, 7)


@pytest.mark.parametrize("nb,ks", [(1, 1), (2, 1), (4, 1), (1, 2), (1, 4)])
def test_every_schedule(nb, ks):
    import paper_2011_09398_amd as lce
    with lce.tuning(xor_nb=nb, xor_ks=ks):
        for cfg, idx in ((2, 0), (3, 0), (3, 3)):
            check(config(cfg)[idx], cfg, idx, f"nb={nb} ks={ks} config {cfg} layer {idx}")



def test_sign_test_special_values():
    # -0.0 and NaN are +1 (bit 0), -inf and negative denormals -1, as lce_bitpack
    import torch
    layer = Layer("special", 1, 6, 6, 64, 32, out="int32")
    inp = make_layer_inputs(layer, 0, 0, 3)
    x = inp.x_float.copy()
    flat = x.reshape(-1)
    special = np.array([-0.0, 0.0, np.nan, -np.nan, np.inf, -np.inf, 1e-45, -1e-45],
                       np.float32)
    flat[::7] = np.resize(special, flat[::7].size)
    xd = dev(x)
    w = gpu_pack_weights(inp)
    got = sync_np(fused(layer, inp, xd, w))
    ref = oracle_layer(layer, inp, oracle.binarize(x))
    assert_match(layer, got, ref, "special floats")
    assert np.array_equal(got, sync_np(unfused(layer, inp, xd, w)))


def test_flip_mask():
    import paper_2011_09398_amd as lce
    layer = Layer("flip", 1, 10, 10, 64, 70, out="bitpacked")
    inp = make_layer_inputs(layer, 0, 0, 4)
    flip = np.array([0x0F0F00F1, 0x7FFFFFFF, 0x3], dtype=np.uint32).view(np.int32)
    out = poisoned_out(layer)
    got = sync_np(lce.quantize_bconv2d(dev(inp.x_float), gpu_pack_weights(inp),
                                       out_type="bitpacked", thresholds=dev(inp.thr),
                                       flip=dev(flip), out=out)).view(np.uint32)
    bits = oracle.bconv2d(oracle.binarize(inp.x_float), inp.w_sign, out="bitpacked",
                          thr=inp.thr, flip=oracle.unpack(flip.view(np.uint32)[None], 70)[0] < 0)
    assert np.array_equal(got, bits)


# ------------------------------------------------ refusals (nothing launched)

def test_unsupported_shapes_raise_before_launch():
    import torch
    import paper_2011_09398_amd as lce
    # C_in not a multiple of 32
    x = torch.zeros((1, 8, 8, 40), dtype=torch.float32, device="cuda")
    w = torch.zeros((8, 3, 3, 2), dtype=torch.int32, device="cuda")
    with pytest.raises(lce.LceError) as e:
        lce.quantize_bconv2d(x, w)
    assert e.value.status == lce.LCE_EUNSUPPORTED
    # x off 16-byte alignment
    base = torch.zeros(8 * 8 * 64 + 4, dtype=torch.float32, device="cuda")
    x = base[1:1 + 8 * 8 * 64].view(1, 8, 8, 64)
    w = torch.zeros((8, 3, 3, 2), dtype=torch.int32, device="cuda")
    with pytest.raises(lce.LceError) as e:
        lce.quantize_bconv2d(x, w)
    assert e.value.status == lce.LCE_EALIGN
    # a band too tall for LDS: with stride 8 a 6-pixel-wide image has one
    # output column, so 64 output pixels read 507 input rows x 6 pixels x 16
    # words = 195 KiB of packed band
    x = torch.zeros((1, 4096, 6, 512), dtype=torch.float32, device="cuda")
    w = torch.zeros((32, 3, 3, 16), dtype=torch.int32, device="cuda")
    out = torch.full((1, 512, 1, 32), 7.0, dtype=torch.float32, device="cuda")
    with pytest.raises(lce.LceError) as e:
        lce.quantize_bconv2d(x, w, stride=8, out=out)
    assert e.value.status == lce.LCE_EUNSUPPORTED and "LDS" in str(e.value)
    assert bool((out == 7.0).all())


def test_graph_replay_matches_eager():
    import torch
    import paper_2011_09398_amd as lce
    layer = config(2)[0]
    inp = make_layer_inputs(layer, 0, 2, 0)
    x, w = dev(inp.x_float), gpu_pack_weights(inp)
    out = poisoned_out(layer)
    call = lce.PreparedQuantBConv2d(x, w, out, stride=layer.strides, padding=layer.padding,
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
    for i in range(3):
        out.fill_(float("nan"))
        g.replay()
        assert np.array_equal(sync_np(out).view(np.uint32), eager.view(np.uint32))
