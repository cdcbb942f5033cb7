"""Helpers that run one layer on the HIP path and on the oracle, and compare.

Both sides consume the same seeded inputs (workloads.gen); the oracle never
sees anything the HIP path produced except where a chained layer's input is
the previous layer's output, and then the oracle uses its own previous output.
"""
from __future__ import annotations

import functools
from typing import Optional, Sequence

import numpy as np

import oracle
from workloads import INT32_MAX, INT32_MIN, Layer, LayerInputs, config, make_layer_inputs

POISON_I32 = -1431655766                      # 0xAAAAAAAA
POISON_F32 = np.array([POISON_I32], np.int32).view(np.float32)[0]
FLOAT_RTOL = 1e-6                             # relative tolerance of the float transform


def clamp_of(layer: Layer):
    return layer.clamp if layer.clamp is not None else (INT32_MIN, INT32_MAX)


def dev(a: np.ndarray):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def gpu_pack_weights(inp: LayerInputs):
    import paper_2011_09398_amd as lce
    return lce.bitpack(dev(inp.w_float))


def gpu_input(inp: LayerInputs):
    """Bitpacked input of a layer on the device (bitpacked by lce_bitpack if float)."""
    import paper_2011_09398_amd as lce
    if inp.x_float is not None:
        return lce.bitpack(dev(inp.x_float))
    return dev(inp.x_words.view(np.int32))


def poisoned_out(layer: Layer):
    import torch
    oh, ow = layer.out_hw()
    if layer.out == "float":
        return torch.full((layer.n, oh, ow, layer.c_out), float(POISON_F32),
                          dtype=torch.float32, device="cuda")
    c = layer.cw_out if layer.out == "bitpacked" else layer.c_out
    return torch.full((layer.n, oh, ow, c), POISON_I32, dtype=torch.int32, device="cuda")


def gpu_layer(layer: Layer, inp: LayerInputs, x_packed=None, w_packed=None, out=None):
    import paper_2011_09398_amd as lce
    x_packed = gpu_input(inp) if x_packed is None else x_packed
    w_packed = gpu_pack_weights(inp) if w_packed is None else w_packed
    out = poisoned_out(layer) if out is None else out
    kw = {}
    if layer.out == "float":
        kw = dict(multiplier=dev(inp.mult), bias=dev(inp.bias))
    elif layer.out == "bitpacked":
        kw = dict(thresholds=dev(inp.thr))
    return lce.bconv2d(x_packed, w_packed, layer.c_in, stride=layer.strides,
                       padding=layer.padding, clamp=layer.clamp, out_type=layer.out,
                       out=out, **kw)


def oracle_signs(inp: LayerInputs, images: Optional[Sequence[int]] = None):
    if inp.x_float is not None:
        x = inp.x_float if images is None else inp.x_float[list(images)]
        return oracle.binarize(x)
    words = inp.x_words if images is None else inp.x_words[list(images)]
    return oracle.unpack(words, inp.layer.c_in)


def oracle_layer(layer: Layer, inp: LayerInputs, a_signs: np.ndarray):
    return oracle.bconv2d(a_signs, inp.w_sign, stride=layer.strides, padding=layer.padding,
                          clamp_range=clamp_of(layer), out=layer.out, mult=inp.mult,
                          bias=inp.bias, thr=inp.thr)


def assert_match(layer: Layer, got: np.ndarray, ref: np.ndarray, what: str = ""):
    """Bit-exact for int32/bitpacked outputs; rtol 1e-6 for float outputs."""
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    if layer.out == "float":
        got64 = got.astype(np.float64)
        err = np.abs(got64 - ref)
        bad = ~(err <= FLOAT_RTOL * np.abs(ref) + 1e-30)
        if bad.any():
            idx = np.argwhere(bad)[:5]
            raise AssertionError(f"{what}: {int(bad.sum())} float outputs off, e.g. "
                                 + ", ".join(f"{tuple(i)} got {got64[tuple(i)]!r} "
                                             f"want {ref[tuple(i)]!r}" for i in idx))
    else:
        g = got.view(np.uint32) if got.dtype == np.int32 and layer.out == "bitpacked" else got
        r = ref.astype(g.dtype) if layer.out == "bitpacked" else ref
        if not np.array_equal(g, r):
            diff = np.argwhere(g != r)[:5]
            raise AssertionError(f"{what}: {int((g != r).sum())} mismatches, e.g. "
                                 + ", ".join(f"{tuple(i)} got {g[tuple(i)]} want {r[tuple(i)]}"
                                             for i in diff))


@functools.lru_cache(maxsize=None)
def config4_reference(chain: bool = True, pad_value: int = 1):
    """Oracle outputs of the four batch-64 layers over the whole batch,
    computed once per process: tuple of (layer, inputs, reference).

    chain=True: the 28x28x128 layer takes the oracle's own stride-2 output
    (the chained configuration); chain=False: every layer its own input.
    pad_value: 1 one-padding, 0 zero padding."""
    out, prev = [], None
    for i, layer in enumerate(config(4)):
        inp = make_layer_inputs(layer, 0, 4, i)
        if chain and layer.chained_from is not None:
            a = oracle.unpack(prev, layer.c_in)
        else:
            a = oracle_signs(inp)
        ref = oracle.bconv2d(a, inp.w_sign, stride=layer.strides, padding=layer.padding,
                             clamp_range=clamp_of(layer), out=layer.out, mult=inp.mult,
                             bias=inp.bias, thr=inp.thr, pad_value=pad_value)
        ref.setflags(write=False)
        out.append((layer, inp, ref))
        prev = ref
    return tuple(out)
