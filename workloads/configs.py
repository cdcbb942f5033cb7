"""The binary-convolution workloads: layer shapes and epilogues.

Shapes come from the paper's workloads: the ResNet18 3x3 convolutions and
the convolution sweep of Section 4.1, and the QuickNet stage widths of
Table 3 (Section 5.1).  Every layer is a binary convolution with one-padding
(Section 3.2, LceBConv2d), 3x3 except the sweep's 5x5 half.

This module holds shapes only; it performs none of the method's arithmetic.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Tuple


@dataclasses.dataclass(frozen=True)
class Layer:
    """One binary convolution.

    input_kind: "float" -> activations ~N(0,1) float32 that the path bitpacks;
                "bits"  -> activations already bitpacked (uniform random bits).
    out: "float" | "bitpacked" | "int32" (raw clamped accumulator).
    clamp: integer (lo, hi) bounds of the fused activation; None = no clamp.
    chained_from: index of the layer (same config) whose bitpacked output is
                  this layer's input; None = the layer gets its own input.
    """

    name: str
    n: int
    h: int
    w: int
    c_in: int
    c_out: int
    kh: int = 3
    kw: int = 3
    stride: int = 1
    padding: str = "same"
    out: str = "bitpacked"
    clamp: Optional[Tuple[int, int]] = None
    input_kind: str = "float"
    chained_from: Optional[int] = None
    stride_w: Optional[int] = None   # None = same as `stride` (the height stride)

    @property
    def strides(self) -> Tuple[int, int]:
        return (self.stride, self.stride if self.stride_w is None else self.stride_w)

    @property
    def cw(self) -> int:
        return (self.c_in + 31) // 32

    @property
    def cw_out(self) -> int:
        return (self.c_out + 31) // 32

    @property
    def k(self) -> int:
        """Number of +-1 products per output value (real channels only)."""
        return self.kh * self.kw * self.c_in

    def out_hw(self) -> Tuple[int, int]:
        sh, sw = self.strides
        if self.padding == "same":
            return (-(-self.h // sh), -(-self.w // sw))
        return ((self.h - self.kh) // sh + 1, (self.w - self.kw) // sw + 1)

    @property
    def m(self) -> int:
        oh, ow = self.out_hw()
        return self.n * oh * ow

    @property
    def macs(self) -> int:
        """Dense algorithmic multiply-accumulates (padded taps included)."""
        return self.m * self.c_out * self.k

    @property
    def binary_ops(self) -> int:
        return 2 * self.macs


INT32_MIN = -(2 ** 31)
INT32_MAX = 2 ** 31 - 1


def _cfg1():
    return [Layer("8x8x64->64", 1, 8, 8, 64, 64, out="float", clamp=None)]


def _cfg2():
    k = 9 * 64
    return [Layer("56x56x64->64", 1, 56, 56, 64, 64, out="float", clamp=(-k, k))]


def _four(n, input_kind, chain):
    # The stride-2 layer comes first so that, at batch 64, its bitpacked
    # 28x28x128 output can feed the 28x28x128 layer.
    return [
        Layer("56x56x64->128/s2", n, 56, 56, 64, 128, stride=2, input_kind=input_kind),
        Layer("28x28x128->128", n, 28, 28, 128, 128, input_kind=input_kind,
              chained_from=0 if chain else None),
        Layer("14x14x256->256", n, 14, 14, 256, 256, input_kind=input_kind),
        Layer("7x7x512->512", n, 7, 7, 512, 512, input_kind=input_kind),
    ]


def _cfg3():
    return _four(1, "float", chain=False)


def _cfg4():
    return _four(64, "bits", chain=True)


def _cfg5():
    n = 16
    layers = []
    for i in range(4):
        layers.append(Layer(f"L{i + 1} 56x56x64->64", n, 56, 56, 64, 64,
                            chained_from=None if i == 0 else i - 1))
    layers.append(Layer("L5 56x56x64->128/s2", n, 56, 56, 64, 128, stride=2, chained_from=3))
    for i in range(5, 8):
        layers.append(Layer(f"L{i + 1} 28x28x128->128", n, 28, 28, 128, 128, chained_from=i - 1))
    layers.append(Layer("L9 28x28x128->256/s2", n, 28, 28, 128, 256, stride=2, chained_from=7))
    for i in range(9, 12):
        last = i == 11
        layers.append(Layer(f"L{i + 1} 14x14x256->256", n, 14, 14, 256, 256,
                            out="float" if last else "bitpacked", chained_from=i - 1))
    return layers


SWEEP_CHANNELS = (32, 64, 96, 128, 160, 256)
SWEEP_SIZES = (8, 16, 32, 64)
SWEEP_KERNELS = (3, 5)


def _cfg6():
    # The convolution sweep of Section 4.1: every combination of channels,
    # square input size and square kernel, stride 1, equal padding, input
    # and output channels equal, one image.  The layer takes bitpacked
    # activations and writes floats through the fused multiplier and bias.
    return [Layer(f"{hw}x{hw}x{c}->{c} k{k}", 1, hw, hw, c, c, kh=k, kw=k, out="float",
                  input_kind="bits")
            for k in SWEEP_KERNELS for hw in SWEEP_SIZES for c in SWEEP_CHANNELS]


CONFIGS = {1: _cfg1, 2: _cfg2, 3: _cfg3, 4: _cfg4, 5: _cfg5, 6: _cfg6}

CONFIG_NAMES = {
    1: "bconv 1x8x8x64->64 3x3 s1 same, float out",
    2: "bconv 1x56x56x64->64 3x3 s1 same, clamp [-K,K], float out",
    3: "QuickNet-shaped bconv sweep, batch 1, bitpacked out",
    4: "QuickNet-shaped bconv sweep, batch 64, pre-bitpacked in, bitpacked out",
    5: "12-layer QuickNet-like stack, batch 16, bitpacked chain, float last",
    6: "conv sweep: C in {32..256}, H=W in {8..64}, 3x3 / 5x5, batch 1, bitpacked in, float out",
}


def config(idx: int):
    return CONFIGS[idx]()
