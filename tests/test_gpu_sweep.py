"""GPU parity on the convolution sweep of Section 4.1 (configuration 6).

48 shape-preserving convolutions, one image each: C_in = C_out in
{32, 64, 96, 128, 160, 256} (96 and 160 give odd word counts), H = W in
{8, 16, 32, 64}, 3x3 and 5x5 filters, stride 1, equal padding; bitpacked
input, float output through the fused multiplier and bias.  Every layer runs
on the XOR+POPCOUNT kernel, on the matrix-core kernel with the library's own
schedule choice (what the benchmark times) and with each schedule forced,
each compared with the oracle over the whole output (1e-6 relative).
"""
import functools

import numpy as np
import pytest

from tests.layer_util import (assert_match, dev, gpu_input, gpu_layer, gpu_pack_weights,
                              oracle_layer, oracle_signs, poisoned_out)
from workloads import config, make_layer_inputs

pytestmark = pytest.mark.gpu

LAYERS = config(6)


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2011_09398_amd as lce
    lce.lib()
    yield
    torch.cuda.synchronize()


@functools.lru_cache(maxsize=None)
def case(i):
    layer = LAYERS[i]
    inp = make_layer_inputs(layer, 0, 6, i)
    return layer, inp, oracle_layer(layer, inp, oracle_signs(inp))


def sync_np(t):
    import torch
    torch.cuda.synchronize()
    return t.cpu().numpy()


@pytest.mark.parametrize("kernel", ["xor", "mfma-default", "mfma-fs", "mfma-pixel",
                                    "mfma-ksplit"])
@pytest.mark.parametrize("i", range(len(LAYERS)), ids=[l.name for l in LAYERS])
def test_sweep_layer(i, kernel):
    import paper_2011_09398_amd as lce
    layer, inp, ref = case(i)
    if kernel == "xor":
        got = sync_np(gpu_layer(layer, inp))
    else:
        lce.set_tuning(mfma_schedule={"mfma-default": "auto", "mfma-fs": "fs",
                                      "mfma-pixel": "pixel",
                                      "mfma-ksplit": "ksplit"}[kernel])
        wf = lce.mfma_weights(gpu_pack_weights(inp), layer.c_in)
        got = sync_np(lce.bconv2d_mfma(
            gpu_input(inp), wf, layer.c_in, layer.c_out, (layer.kh, layer.kw),
            stride=layer.strides, padding=layer.padding, clamp=layer.clamp,
            out_type=layer.out, multiplier=dev(inp.mult), bias=dev(inp.bias),
            out=poisoned_out(layer)))
    assert_match(layer, got, ref, f"{layer.name} {kernel}")
    assert np.isfinite(got).all()
