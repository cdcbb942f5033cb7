"""Seeded synthetic inputs shared by the oracle side and the HIP side.

Recipe (one numpy PCG64 stream per (seed, config, layer)):
  1. activations: float32 ~N(0,1), NHWC [N,H,W,C_in]
     or, for pre-bitpacked inputs, uint32 words of uniform random bits
     [N,H,W,ceil(C_in/32)] whose bits beyond C_in are zero;
  2. weight signs: Bernoulli(1/2) over {-1,+1}, OHWI [C_out,KH,KW,C_in];
  3. multiplier ~N(1, 0.1), 4. bias ~N(0, 0.1), 5. thresholds ~N(0, 1),
     each float32 [C_out].
All five are always drawn, in this order, so every tensor is reproducible.

Nothing here binarizes, packs or convolves: generating uniform random words
and random signs is input synthesis, not the method.
"""
from __future__ import annotations

import dataclasses
import hashlib
from typing import Optional

import numpy as np

from .configs import Layer


@dataclasses.dataclass
class LayerInputs:
    layer: Layer
    x_float: Optional[np.ndarray]   # float32 [N,H,W,C_in]  (input_kind == "float")
    x_words: Optional[np.ndarray]   # uint32  [N,H,W,Cw]    (input_kind == "bits")
    w_sign: np.ndarray              # int8 +-1 [C_out,KH,KW,C_in]
    w_float: np.ndarray             # float32 +-1, same values
    mult: np.ndarray                # float32 [C_out]
    bias: np.ndarray                # float32 [C_out]
    thr: np.ndarray                 # float32 [C_out]


def rng_for(seed: int, cfg: int, layer: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([seed, cfg, layer]))


def random_words(rng: np.random.Generator, shape_prefix, channels: int) -> np.ndarray:
    """uint32 words of uniform random bits; the bits past `channels` are 0."""
    cw = (channels + 31) // 32
    words = rng.integers(0, 2 ** 32, size=tuple(shape_prefix) + (cw,), dtype=np.uint64)
    words = words.astype(np.uint32)
    rem = channels % 32
    if rem:
        words[..., -1] &= np.uint32((1 << rem) - 1)
    return words


def make_layer_inputs(layer: Layer, seed: int = 0, cfg: int = 0, index: int = 0,
                      input_kind: Optional[str] = None) -> LayerInputs:
    rng = rng_for(seed, cfg, index)
    kind = input_kind or layer.input_kind
    x_float = x_words = None
    if kind == "float":
        x_float = rng.standard_normal((layer.n, layer.h, layer.w, layer.c_in), dtype=np.float32)
    elif kind == "bits":
        x_words = random_words(rng, (layer.n, layer.h, layer.w), layer.c_in)
    else:
        raise ValueError(kind)
    bits = rng.integers(0, 2, size=(layer.c_out, layer.kh, layer.kw, layer.c_in), dtype=np.int8)
    w_sign = (1 - 2 * bits).astype(np.int8)
    w_float = w_sign.astype(np.float32)
    mult = rng.normal(1.0, 0.1, size=layer.c_out).astype(np.float32)
    bias = rng.normal(0.0, 0.1, size=layer.c_out).astype(np.float32)
    thr = rng.standard_normal(layer.c_out, dtype=np.float32)
    return LayerInputs(layer, x_float, x_words, w_sign, w_float, mult, bias, thr)


def sha256(a: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()
