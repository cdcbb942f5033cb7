"""GPU parity of LceBMaxPool2d and LceDequantize (Section 3.2) against the
oracle.  Binary max pooling is the oracle's max of +-1 values over each
window (locations outside the image ignored), compared word for word with
pad bits; dequantize is the oracle's unpack, compared bit for bit as float.
"""
import numpy as np
import pytest

import oracle
from tests.layer_util import POISON_I32, dev, gpu_input, gpu_pack_weights, oracle_signs
from workloads import Layer, make_layer_inputs
from workloads.gen import random_words

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


def poisoned(shape, dtype):
    import torch
    if dtype == "int32":
        return torch.full(shape, POISON_I32, dtype=torch.int32, device="cuda")
    return torch.full(shape, float("nan"), dtype=torch.float32, device="cuda")


def oracle_pool_words(words, channels, k, s, padding):
    kh, kw = (k, k) if isinstance(k, int) else k
    sh, sw = (s, s) if isinstance(s, int) else s
    signs = oracle.unpack(words, channels)
    pooled = oracle.bmaxpool(signs, kh, kw, (sh, sw), padding)
    return oracle.pack(pooled)


def run_pool(words, channels, k, s, padding, x=None):
    import paper_2011_09398_amd as lce
    x = dev(words.view(np.int32)) if x is None else x
    d = lce.make_pool_desc(*words.shape[:3], channels, k, s, padding)
    oh, ow = lce.pool_out_shape(d)
    out = poisoned((words.shape[0], oh, ow, words.shape[3]), "int32")
    return sync_np(lce.bmaxpool2d(x, channels, k, s, padding, out=out)).view(np.uint32)


def pool_cases():
    rng = np.random.default_rng(77)
    cases = []
    for i in range(40):
        k = [int(rng.choice([1, 2, 2, 3, 3, 5]))] * 2
        if rng.random() < 0.2:
            k[1] = int(rng.choice([1, 2, 3]))
        s = int(rng.choice([1, 2, 2, 3]))
        padding = "same" if rng.random() < 0.6 else "valid"
        h, w = int(rng.integers(1, 12)), int(rng.integers(1, 12))
        if padding == "valid":
            h, w = max(h, k[0]), max(w, k[1])
        c = int(rng.choice([1, 7, 32, 33, 64, 96, 100, 128, 256, 512]))
        n = int(rng.integers(1, 4))
        cases.append((f"p{i}", n, h, w, c, tuple(k), s, padding))
    return cases


@pytest.mark.parametrize("case", pool_cases(), ids=lambda c: c[0])
def test_bmaxpool_sweep(case):
    name, n, h, w, c, k, s, padding = case
    rng = np.random.default_rng(int(name[1:]))
    words = random_words(rng, (n, h, w), c)
    # bias toward -1 so that ANDs of several words are not almost always 0
    words |= random_words(rng, (n, h, w), c)
    got = run_pool(words, c, k, s, padding)
    want = oracle_pool_words(words, c, k, s, padding)
    assert np.array_equal(got, want), name


@pytest.mark.parametrize("cw", [1, 2, 3, 4, 8, 16])
@pytest.mark.parametrize("offset_words", [0, 1, 2])
def test_bmaxpool_vector_widths_and_alignment(cw, offset_words):
    """Word vectors of 4, 2 and 1 words, chosen by word count and alignment."""
    import torch
    rng = np.random.default_rng(cw * 10 + offset_words)
    n, h, w, c = 2, 9, 10, 32 * cw
    words = random_words(rng, (n, h, w), c) | random_words(rng, (n, h, w), c)
    flat = torch.zeros(words.size + 4, dtype=torch.int32, device="cuda")
    x = flat[offset_words:offset_words + words.size].view(n, h, w, cw)
    x.copy_(torch.from_numpy(words.view(np.int32)))
    got = run_pool(words, c, 3, 2, "same", x=x)
    assert np.array_equal(got, oracle_pool_words(words, c, 3, 2, "same"))


def test_bmaxpool_all_minus_one_and_single_plus_one():
    """All -1 pools to all -1; one +1 at (0, 0) makes every window holding it +1."""
    c = 64
    words = np.full((1, 4, 4, 2), 0xFFFFFFFF, np.uint32)
    assert np.array_equal(run_pool(words, c, 2, 2, "valid"),
                          np.full((1, 2, 2, 2), 0xFFFFFFFF, np.uint32))
    words[0, 0, 0, 0] &= ~np.uint32(1)            # channel 0 at (0, 0) becomes +1
    got = run_pool(words, c, 3, 1, "same")
    for oy in range(4):
        for ox in range(4):
            has = oy <= 1 and ox <= 1             # windows containing (0, 0)
            assert (int(got[0, oy, ox, 0]) & 1) == (0 if has else 1), (oy, ox)


@pytest.mark.parametrize("n,h,c,k,s", [(64, 56, 64, 3, 2), (64, 28, 128, 2, 2),
                                      (16, 14, 256, 3, 1)])
def test_bmaxpool_network_sized(n, h, c, k, s):
    rng = np.random.default_rng(n + h + c)
    words = random_words(rng, (n, h, h), c) | random_words(rng, (n, h, h), c)
    got = run_pool(words, c, k, s, "same")
    assert np.array_equal(got, oracle_pool_words(words, c, k, s, "same"))


def test_conv_pool_conv_chain():
    """Binary conv (bitpacked out) -> binary max pool -> binary conv, every
    stage against the oracle running the same chain on its own outputs."""
    import paper_2011_09398_amd as lce
    l1 = Layer("c1", 2, 16, 16, 64, 96, out="bitpacked", input_kind="bits")
    i1 = make_layer_inputs(l1, 1, 90, 0)
    y1 = lce.bconv2d(gpu_input(i1), gpu_pack_weights(i1), 64, out_type="bitpacked",
                     thresholds=dev(i1.thr))
    r1 = oracle.bconv2d(oracle_signs(i1), i1.w_sign, out="bitpacked", thr=i1.thr)
    assert np.array_equal(sync_np(y1).view(np.uint32), r1)
    p1 = lce.bmaxpool2d(y1, 96, 2, 2, "valid")
    rp = oracle_pool_words(r1, 96, 2, 2, "valid")
    assert np.array_equal(sync_np(p1).view(np.uint32), rp)
    l2 = Layer("c2", 2, 8, 8, 96, 40, out="float", input_kind="bits")
    i2 = make_layer_inputs(l2, 1, 90, 1)
    y2 = lce.bconv2d(p1, gpu_pack_weights(i2), 96, out_type="float",
                     multiplier=dev(i2.mult), bias=dev(i2.bias))
    r2 = oracle.bconv2d(oracle.unpack(rp, 96), i2.w_sign, out="float", mult=i2.mult,
                        bias=i2.bias)
    got = sync_np(y2).astype(np.float64)
    assert np.all(np.abs(got - r2) <= 1e-6 * np.abs(r2) + 1e-30)


@pytest.mark.parametrize("rows,c", [(1, 32), (7, 64), (1000, 128), (3, 1), (5, 31), (9, 33),
                                    (4, 100), (0, 64), (333, 512)])
def test_dequantize_parity(rows, c):
    import paper_2011_09398_amd as lce
    rng = np.random.default_rng(rows * 1000 + c)
    words = random_words(rng, (rows,), c)
    out = poisoned((rows, c), "float")
    got = sync_np(lce.dequantize(dev(words.view(np.int32)), c, out=out))
    want = oracle.unpack(words, c).astype(np.float32)
    assert got.dtype == np.float32 and np.array_equal(got.view(np.uint32), want.view(np.uint32))


def test_dequantize_unaligned_output_takes_scalar_path():
    import torch
    import paper_2011_09398_amd as lce
    rng = np.random.default_rng(5)
    words = random_words(rng, (50,), 64)
    flat = torch.full((50 * 64 + 1,), float("nan"), dtype=torch.float32, device="cuda")
    out = flat[1:].view(50, 64)
    lce.dequantize(dev(words.view(np.int32)), 64, out=out)
    want = oracle.unpack(words, 64).astype(np.float32)
    assert np.array_equal(sync_np(out), want)


def test_dequantize_inverts_bitpack_on_signs():
    """dequantize(bitpack(x)) is the sign of x (x < 0 -> -1, else +1)."""
    import paper_2011_09398_amd as lce
    rng = np.random.default_rng(9)
    x = rng.standard_normal((64, 28, 28, 128)).astype(np.float32)
    got = sync_np(lce.dequantize(lce.bitpack(dev(x)), 128))
    assert np.array_equal(got, np.where(x < 0, -1.0, 1.0).astype(np.float32))
