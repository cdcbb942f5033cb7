"""The seeded generators: deterministic, the documented shapes and laws."""
import numpy as np

from workloads import config, make_layer_inputs, sha256


def test_configs_shapes_and_work():
    c4 = config(4)
    assert [l.m for l in c4] == [64 * 28 * 28, 64 * 28 * 28, 64 * 14 * 14, 64 * 7 * 7]
    # binary ops per layer (2 * MACs), counting padded taps
    assert [l.binary_ops for l in c4] == [7_398_752_256, 14_797_504_512,
                                         14_797_504_512, 14_797_504_512]
    c5 = config(5)
    assert len(c5) == 12
    assert sum(l.binary_ops for l in c5) == 40_693_137_408
    assert [l.out for l in c5] == ["bitpacked"] * 11 + ["float"]
    for i, l in enumerate(c5[1:], 1):
        prev = c5[l.chained_from]
        assert l.chained_from == i - 1
        assert (prev.out_hw(), prev.c_out) == ((l.h, l.w), l.c_in)
    s2, l28 = c4[0], c4[1]
    assert l28.chained_from == 0 and (s2.out_hw(), s2.c_out) == ((l28.h, l28.w), l28.c_in)


def test_inputs_deterministic_and_distributed():
    layer = config(1)[0]
    a = make_layer_inputs(layer, seed=0, cfg=1, index=0)
    b = make_layer_inputs(layer, seed=0, cfg=1, index=0)
    for name in ("x_float", "w_sign", "w_float", "mult", "bias", "thr"):
        assert sha256(getattr(a, name)) == sha256(getattr(b, name))
    c = make_layer_inputs(layer, seed=1, cfg=1, index=0)
    assert sha256(a.x_float) != sha256(c.x_float)
    assert a.x_float.dtype == np.float32 and a.x_float.shape == (1, 8, 8, 64)
    assert set(np.unique(a.w_sign)) == {-1, 1}
    assert np.array_equal(a.w_float, a.w_sign.astype(np.float32))
    assert abs(float(a.mult.mean()) - 1.0) < 0.05 and abs(float(a.bias.mean())) < 0.05


def test_random_words_pad_bits_zero():
    from workloads import Layer
    layer = Layer("t", 2, 3, 3, 40, 8, input_kind="bits")
    x = make_layer_inputs(layer).x_words
    assert x.shape == (2, 3, 3, 2) and x.dtype == np.uint32
    assert not (x[..., 1] >> 8).any()
    ones = np.unpackbits(np.ascontiguousarray(x[..., 0]).view(np.uint8)).mean()
    assert 0.4 < ones < 0.6


def test_conv_sweep_shapes():
    """Section 4.1's sweep: 6 channel counts x 4 sizes x 2 kernels = 48
    shape-preserving convolutions, 0.59 M to 6.7 G MACs (the listed
    dimensions; the paper's printed upper bound is garbled)."""
    c6 = config(6)
    assert len(c6) == 48
    assert len({(l.h, l.c_in, l.kh) for l in c6}) == 48
    for l in c6:
        assert l.n == 1 and l.h == l.w and l.c_in == l.c_out and l.kh == l.kw
        assert l.strides == (1, 1) and l.padding == "same" and l.out_hw() == (l.h, l.w)
    macs = sorted(l.macs for l in c6)
    assert macs[0] == 8 * 8 * 32 * 32 * 9 == 589_824
    assert macs[-1] == 64 * 64 * 256 * 256 * 25 == 6_710_886_400
