"""Benchmark of the bitpacked binary convolution on one MI355X.

Default workload (one step): the four batch-64 QuickNet-shaped binary 3x3
convolutions with bitpacked input and output: 56x56x64->128 stride 2, whose
output feeds 28x28x128->128, then 14x14x256->256 and 7x7x512->512.

Each convolution has two implementations with identical results: the XOR +
POPCOUNT kernel of the paper's method (lce_bconv2d, VALU) and the same dot
on the matrix cores (lce_bconv2d_mfma, +-1 widened to 4-bit floats).  Both
are timed per layer; the step uses the faster one for each layer (--kernel
auto, the default) or the one named by --kernel xor|mfma.

Measured on the launch stream with HIP events:
  * the timed region: K steps back to back (events at its two ends, plus
    wall clock around it, synchronized on both sides) -> value, ms_per_step;
  * per launch: each layer launched R times back to back between two events
    -> average launch duration, the figure the roofline uses;
  * batch-1 layers (float input: lce_bitpack timed as its own line, and each
    whole layer as bitpack + either conv, or as one quantize-fused launch)
    the same way, but from a captured HIP graph of the R launches, since
    eager launch cost exceeds their run time;
  * a probe of the achievable xor+popcount VALU rate, next to the spec peak;
  * the same layers with zero padding (the correction-step variant);
  * the memory-bound operators at sizes beyond the 256 MB last-level cache,
    inputs (or outputs) rotated over buffers totalling more than 512 MB:
    bitpack (LceQuantize), binary max pooling (LceBMaxPool2d) and
    dequantize (LceDequantize), in GB/s of algorithmic bytes vs 8 TB/s;
  * the convolution sweep of Section 4.1 (48 batch-1 layers, 3x3 and 5x5,
    bitpacked in, float out), both kernels from captured graphs;
  * configurations 1, 2 and 3 (batch 1) per layer from captured graphs, and
    configuration 5 (the 12-layer batch-16 stack) end to end, from eager
    launches and from one captured graph of the whole pass, with its
    per-layer breakdown;
  * the headline layers on the XOR+POPCOUNT kernel as well, reported against
    the VALU peak (roofline_valu) next to the roofline of the kernel the
    step uses.
Then the CPU oracle, as it stands, on a bounded sample of the same step, on
the whole configuration-5 stack, and on every batch-1 layer with one thread
and with all host threads.

    python bench.py [--steps K] [--warmup W] [--no-cpu] [--workload b64|stack16]
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "binary conv GOPS (2·MACs/s) + µs/layer, batch 1 and 64, vs roofline"

# VALU peak for the XOR+POPCOUNT inner loop: 256 CUs x 64 lanes x 2.4 GHz
# lane-ops/s; one v_xor_b32 plus one v_bcnt_u32_b32 (popcount+accumulate)
# cover 32 binary MACs, i.e. 16 MACs = 32 binary ops per VALU lane-op.
CUS, LANES, CLOCK_HZ = 256, 64, 2.4e9
VALU_LANE_OPS = CUS * LANES * CLOCK_HZ
BINARY_OPS_PER_LANE_OP = 32
PEAK_BINARY_TOPS = VALU_LANE_OPS * BINARY_OPS_PER_LANE_OP / 1e12      # 1258.3
# Dense fp4 MFMA peak (MI355X): one +-1 MAC is one fp4 MAC, 2 ops.
PEAK_FP4_TFLOPS = 10100.0
# The arithmetic each implementation computes in (the bench line's dtype).
DTYPES = {"xor": "u32 xor+popcount (VALU), int32 accumulate",
          "mfma": "fp4 e2m1 MFMA, fp32 accumulate (integer-exact dot)",
          "fused": "fp32 sign test + u32 xor+popcount (VALU), int32 accumulate",
          "fused_mfma": "fp32 sign test + fp4 e2m1 MFMA, fp32 accumulate (integer-exact dot)"}
HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=500)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--reps", type=int, default=100, help="launches per per-kernel timing")
    ap.add_argument("--workload", choices=("b64", "stack16"), default="b64")
    ap.add_argument("--kernel", choices=("auto", "xor", "mfma"), default="auto",
                    help="convolution implementation per layer (auto: the faster)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-batch1", action="store_true", help="skip the batch-1 lines")
    ap.add_argument("--no-stack", action="store_true",
                    help="skip configuration 5 (the 12-layer batch-16 stack)")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the convolution-sweep lines (48 batch-1 layers)")
    ap.add_argument("--sweep-only", action="store_true",
                    help="time only the convolution sweep (for kernel traces); prints the "
                         "sweep lines instead of the benchmark line")
    ap.add_argument("--no-probe", action="store_true", help="skip the VALU rate probe")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the zero-padding and memory-bound operator lines")
    ap.add_argument("--profile-pass", action="store_true",
                    help="short run for counter collection: 512 MiB copies (the byte-counter "
                         "calibration), three launches of each implementation per layer, "
                         "then the VALU probe")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="target wall time of the CPU baseline sample")
    return ap.parse_args()


def ensure_built():
    from paper_2011_09398_amd import build as lb
    if not (os.path.exists(lb.LIB) and os.path.exists(lb.PROBE_LIB)):
        lb.build()


class Step:
    """Device buffers and prepared calls for one configuration's layers."""

    def __init__(self, cfg_idx: int):
        import numpy as np
        import torch
        import paper_2011_09398_amd as lce
        from workloads import config, make_layer_inputs

        self.layers = config(cfg_idx)
        self.inputs = [make_layer_inputs(l, 0, cfg_idx, i) for i, l in enumerate(self.layers)]
        dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
        self.xor_calls, self.mfma_calls, self.fused_calls = [], [], []
        self.fused_mfma_calls = []
        self.packs, self.outs, self.keep = [], [], []
        for i, (layer, inp) in enumerate(zip(self.layers, self.inputs)):
            w_packed = lce.bitpack(dev(inp.w_float))          # 1-bit weight storage
            pack = None
            if layer.chained_from is not None:
                x_packed = self.outs[layer.chained_from]
            elif inp.x_float is not None:
                xf = dev(inp.x_float)
                x_packed = torch.empty(xf.shape[:-1] + (layer.cw,), dtype=torch.int32,
                                       device="cuda")
                pack = lce.PreparedBitpack(xf, x_packed)
            else:
                x_packed = dev(inp.x_words.view(np.int32))
            oh, ow = layer.out_hw()
            if layer.out == "float":
                out = torch.empty((layer.n, oh, ow, layer.c_out), dtype=torch.float32,
                                  device="cuda")
                kw = dict(multiplier=dev(inp.mult), bias=dev(inp.bias))
            else:
                out = torch.empty((layer.n, oh, ow, layer.cw_out), dtype=torch.int32,
                                  device="cuda")
                kw = dict(thresholds=dev(inp.thr))
            self.xor_calls.append(lce.PreparedBConv2d(
                x_packed, w_packed, layer.c_in, out, stride=layer.strides,
                padding=layer.padding, clamp=layer.clamp, out_type=layer.out, **kw))
            w_fp4 = lce.mfma_weights(w_packed, layer.c_in)     # widened once per filter tensor
            m = lce.PreparedBConv2dMfma(
                x_packed, w_fp4, layer.c_in, layer.c_out, (layer.kh, layer.kw), out,
                stride=layer.strides, padding=layer.padding, clamp=layer.clamp,
                out_type=layer.out, **kw)
            m.keep = m.keep + (w_fp4,)
            self.mfma_calls.append(m)
            fused = None
            if pack is not None:      # float input: the quantize-fused launch, where covered
                try:
                    fused = lce.PreparedQuantBConv2d(
                        xf, w_packed, out, stride=layer.strides, padding=layer.padding,
                        clamp=layer.clamp, out_type=layer.out, **kw)
                except lce.LceError as e:
                    if e.status != lce.LCE_EUNSUPPORTED:
                        raise
            self.fused_calls.append(fused)
            fused_mfma = None
            if pack is not None:      # float input: the quantize-fused matrix-core launch
                try:
                    fused_mfma = lce.PreparedQuantBConv2dMfma(
                        xf, w_fp4, layer.c_out, (layer.kh, layer.kw), out,
                        stride=layer.strides, padding=layer.padding, clamp=layer.clamp,
                        out_type=layer.out, **kw)
                except lce.LceError as e:
                    if e.status != lce.LCE_EUNSUPPORTED:
                        raise
            self.fused_mfma_calls.append(fused_mfma)
            self.packs.append(pack)
            self.outs.append(out)
            self.keep.append((w_packed, x_packed, kw))
        self.calls = list(self.xor_calls)
        self.kinds = ["xor"] * len(self.calls)
        self.times = [None] * len(self.calls)

    def kinds_of(self, i):
        """The whole-layer forms layer i has: bitpack (float input) + the XOR
        or the matrix-core convolution, and the quantize-fused launches of
        either kernel where they cover the shape."""
        return (["xor", "mfma"] + (["fused"] if self.fused_calls[i] is not None else [])
                + (["fused_mfma"] if self.fused_mfma_calls[i] is not None else []))

    def layer_call(self, i, kind):
        """Layer i as one callable: bitpack (float input) then the named
        convolution, or a quantize-fused launch."""
        if kind == "fused":
            return self.fused_calls[i]
        if kind == "fused_mfma":
            return self.fused_mfma_calls[i]
        conv = self.mfma_calls[i] if kind == "mfma" else self.xor_calls[i]
        pack = self.packs[i]
        if pack is None:
            return conv

        def both():
            pack()
            conv()
        return both

    def choose(self, mode: str, reps: int, graph: bool = False):
        """Time the implementations of every layer and keep the fastest (auto)
        or the named one for the step: bitpack (float input) + XOR/POPCOUNT
        conv, bitpack + matrix-core conv, or the quantize-fused launch.
        graph: time from captured graphs (layers shorter than an eager
        launch).  times[i] = {form: whole-layer ms}."""
        self.times = []
        for i in range(len(self.layers)):
            kinds = self.kinds_of(i)
            t = {k: time_repeated(self.layer_call(i, k), reps, graph=graph) for k in kinds}
            self.times.append(t)
            kind = mode if mode != "auto" else min(kinds, key=t.__getitem__)
            if kind not in kinds:
                kind = "xor"
            self.kinds[i] = kind
            self.calls[i] = self.layer_call(i, kind)

    def run(self):
        """One pass of the hot path: every layer (bitpack of a float input
        included) with its chosen implementation."""
        for call in self.calls:
            call()


def time_steps(step: Step, steps: int, warmup: int):
    import torch
    for _ in range(warmup):
        step.run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record()
    for _ in range(steps):
        step.run()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return wall, e0.elapsed_time(e1) * 1e-3


def time_graph_steps(step: Step, steps: int) -> float:
    """Seconds per step when one step (every launch of the pass) is replayed
    from a captured HIP graph, `steps` replays back to back between events."""
    import torch
    step.run()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            step.run()
    torch.cuda.current_stream().wait_stream(s)
    for _ in range(3):
        g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e-3 / steps


def time_repeated(fn, reps: int, graph: bool) -> float:
    """Average duration (ms) of `fn` launched `reps` times back to back."""
    import torch
    for _ in range(10):
        fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    if graph:
        g = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            with torch.cuda.graph(g, stream=s):
                for _ in range(reps):
                    fn()
        torch.cuda.current_stream().wait_stream(s)
        g.replay()
        torch.cuda.synchronize()
        e0.record()
        g.replay()
        e1.record()
    else:
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


TRIALS = 7


def time_trials(fn, reps: int, graph: bool, trials: int = TRIALS):
    """`trials` timings of time_repeated (ms each): the per-layer figures
    are their median, with p10 and p90 beside it."""
    return [time_repeated(fn, reps, graph) for _ in range(trials)]


def trial_fields(ts):
    """median (ms) and the record's spread fields of a list of trials."""
    import numpy as np
    a = np.asarray(ts) * 1e3
    return float(np.median(a)) / 1e3, {
        "trials": len(ts), "us_p10": round(float(np.percentile(a, 10)), 3),
        "us_p90": round(float(np.percentile(a, 90)), 3)}


def inputs_digest(inp):
    """The first 16 hex digits of the SHA-256 of each generated tensor of a
    layer (the same buffers the oracle and the GPU consume)."""
    from workloads import sha256
    out = {}
    for name in ("x_float", "x_words", "w_float", "mult", "bias", "thr"):
        a = getattr(inp, name, None)
        if a is not None:
            out[name] = sha256(a)[:16]
    return out


def layer_record(layer, ms, probe_tops=None, kind="xor", times=None):
    """One layer's launch(es): binary GOPS against the roofline of the unit
    that ran it (VALU xor+popcount, or dense fp4 MFMA; "fused" and
    "fused_mfma" are the XOR+POPCOUNT and the matrix-core kernels binarizing
    their float input themselves).  For a float input, `us` covers the whole
    layer: bitpack + conv, or the fused launch.
    times: {form: ms} of the whole-layer forms the choice was made from."""
    ops = layer.binary_ops
    tops = ops / (ms * 1e-3) / 1e12
    r = {"layer": layer.name, "batch": layer.n, "kernel": kind, "us": round(ms * 1e3, 3),
         "binary_gops": round(tops * 1e3, 1), "binary_ops": ops}
    if layer.input_kind == "float" and layer.chained_from is None:
        r["input"] = "float32, binarized in the timed launches"
    if kind in ("xor", "fused"):
        r["valu_frac"] = round(tops / PEAK_BINARY_TOPS, 4)
        if probe_tops:
            r["probe_frac"] = round(tops / probe_tops, 4)
    else:
        r["mfma_fp4_frac"] = round(tops / PEAK_FP4_TFLOPS, 4)
    if times is not None:
        for k, t in times.items():
            r[f"us_{k}"] = round(t * 1e3, 3)
    return r


def bitpack_record(layer, ms):
    n_float = layer.n * layer.h * layer.w * layer.c_in
    nbytes = 4 * n_float + 4 * layer.n * layer.h * layer.w * layer.cw
    gbs = nbytes / (ms * 1e-3) / 1e9
    return {"layer": f"bitpack {layer.n}x{layer.h}x{layer.w}x{layer.c_in}", "batch": layer.n,
            "us": round(ms * 1e3, 3), "bytes": nbytes, "GB/s": round(gbs, 1),
            "hbm_frac": round(gbs / HBM_PEAK_GBS, 4)}


def mem_record(name, nbytes, ms):
    gbs = nbytes / (ms * 1e-3) / 1e9
    return {"op": name, "us": round(ms * 1e3, 3), "bytes": nbytes, "GB/s": round(gbs, 1),
            "hbm_frac": round(gbs / HBM_PEAK_GBS, 4)}


def rotating(calls):
    """One callable that launches calls[0], calls[1], ... in turn."""
    state = {"i": 0}

    def fn():
        calls[state["i"]]()
        state["i"] = (state["i"] + 1) % len(calls)
    return fn


def memory_bound_lines(reps: int):
    """bitpack, binary max pooling and dequantize beyond the last-level cache."""
    import numpy as np
    import torch
    import paper_2011_09398_amd as lce
    from workloads.gen import random_words
    rng = np.random.default_rng(0)
    lines = []
    # reference: a plain device copy of 512 MiB (read + write), the bandwidth
    # a streaming kernel can reach in practice
    src = torch.ones(128 * 2 ** 20, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    lines.append(mem_record("copy 512 MiB (torch)", 2 * 4 * src.numel(),
                            time_repeated(lambda: dst.copy_(src), 20, graph=False)))
    del src, dst
    # LceQuantize: 256x56x56x64 float (205 MB) -> 6.4 MB, 3 rotating inputs
    n, h, c = 256, 56, 64
    xs = [torch.randn((n, h, h, c), dtype=torch.float32, device="cuda") for _ in range(3)]
    outs = [torch.empty((n, h, h, 2), dtype=torch.int32, device="cuda") for _ in range(3)]
    calls = [lce.PreparedBitpack(x, o) for x, o in zip(xs, outs)]
    nbytes = 4 * n * h * h * c + 4 * n * h * h * 2
    lines.append(mem_record(f"bitpack {n}x{h}x{h}x{c}", nbytes,
                            time_repeated(rotating(calls), reps, graph=False)))
    del xs, outs, calls
    # LceBMaxPool2d 3x3 stride 2 SAME: 8192x56x56x64 bits (205 MB) -> 28x28, 3 inputs
    n, h, c = 8192, 56, 64
    words = torch.from_numpy(random_words(rng, (n, h, h), c).view(np.int32)).cuda()
    xs = [words] + [words.clone() for _ in range(2)]
    desc = lce.make_pool_desc(n, h, h, c, 3, 2, "same")
    oh, ow = lce.pool_out_shape(desc)
    outs = [torch.empty((n, oh, ow, 2), dtype=torch.int32, device="cuda") for _ in range(3)]
    L, st = lce.lib(), torch.cuda.current_stream().cuda_stream
    ref = ctypes.byref(desc)
    calls = [(lambda x=x, o=o: L.lce_bmaxpool2d(ref, x.data_ptr(), o.data_ptr(), st))
             for x, o in zip(xs, outs)]
    nbytes = 4 * words.numel() + 4 * outs[0].numel()
    lines.append(mem_record(f"bmaxpool2d 3x3/2 {n}x{h}x{h}x{c}", nbytes,
                            time_repeated(rotating(calls), reps, graph=False)))
    del words, xs, outs, calls
    # LceDequantize: 256x28x28x128 bits (3.2 MB) -> float (103 MB), 3 rotating outputs
    n, h, c = 256, 28, 128
    x = torch.from_numpy(random_words(rng, (n, h, h), c).view(np.int32)).cuda()
    outs = [torch.empty((n, h, h, c), dtype=torch.float32, device="cuda") for _ in range(3)]
    rows = n * h * h
    calls = [(lambda o=o: L.lce_dequantize(x.data_ptr(), o.data_ptr(), rows, c, st))
             for o in outs]
    nbytes = 4 * x.numel() + 4 * outs[0].numel()
    lines.append(mem_record(f"dequantize {n}x{h}x{h}x{c}", nbytes,
                            time_repeated(rotating(calls), reps, graph=False)))
    del x, outs, calls
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return lines


def zero_padding_lines(step, reps: int, probe_tops=None):
    """The step's layers with zero padding: the XOR path with its correction
    table (prepared once), and the matrix-core path (padding widened to 0.0)."""
    import paper_2011_09398_amd as lce
    lines = []
    for m, layer, (w_packed, x_packed, kw), out in zip(step.mfma_calls, step.layers,
                                                       step.keep, step.outs):
        corr = lce.pad_correction(w_packed, layer.c_in)
        z = lce.PreparedBConv2d(x_packed, w_packed, layer.c_in, out, stride=layer.strides,
                                padding=layer.padding, pad_value="zero", clamp=layer.clamp,
                                out_type=layer.out, pad_correction=corr, **kw)
        zm = lce.PreparedBConv2dMfma(x_packed, m.keep[1], layer.c_in, layer.c_out,
                                     (layer.kh, layer.kw), out, stride=layer.strides,
                                     padding=layer.padding, pad_value="zero",
                                     clamp=layer.clamp, out_type=layer.out, **kw)
        for kind, call in (("xor", z), ("mfma", zm)):
            r = layer_record(layer, time_repeated(call, reps, graph=False), probe_tops, kind)
            r["padding"] = "zero"
            lines.append(r)
    return lines


def sweep_lines(args, probe=None):
    """The convolution sweep (48 batch-1 layers): both kernels per layer,
    each from a captured graph of R launches (5 eager warmups first)."""
    s6 = Step(6)
    out = []
    for x, m, layer in zip(s6.xor_calls, s6.mfma_calls, s6.layers):
        tx = time_repeated(x, args.reps, graph=True)
        tm = time_repeated(m, args.reps, graph=True)
        kind = args.kernel if args.kernel != "auto" else ("mfma" if tm < tx else "xor")
        r = layer_record(layer, tm if kind == "mfma" else tx, probe, kind,
                         {"xor": tx, "mfma": tm})
        r["macs"] = layer.macs
        out.append(r)
    return out


def batch1_lines(args, probe=None):
    """Configurations 1, 2 and 3 (batch 1, float input), each timing from a
    captured graph of R launches: per layer, bitpack alone, each convolution
    kernel alone, and the whole layer three ways (bitpack + XOR/POPCOUNT
    conv, bitpack + matrix-core conv, the quantize-fused launch); the layer
    line reports the fastest whole layer."""
    out = []
    for cfg in (1, 2, 3):
        s = Step(cfg)
        for i, (pack, x, m, layer) in enumerate(zip(s.packs, s.xor_calls, s.mfma_calls,
                                                    s.layers)):
            r = bitpack_record(layer, time_repeated(pack, args.reps, graph=True))
            r["config"] = cfg
            out.append(r)
            kinds = s.kinds_of(i)
            whole = {k: time_repeated(s.layer_call(i, k), args.reps, graph=True) for k in kinds}
            kind = args.kernel if args.kernel != "auto" else min(kinds, key=whole.__getitem__)
            r = layer_record(layer, whole[kind], probe, kind, whole)
            r["us_conv_xor"] = round(time_repeated(x, args.reps, graph=True) * 1e3, 3)
            r["us_conv_mfma"] = round(time_repeated(m, args.reps, graph=True) * 1e3, 3)
            r["config"] = cfg
            out.append(r)
    return out


def stack_lines(args, probe=None):
    """Configuration 5, the 12-layer batch-16 stack (bitpack of the float
    input, then the chain): end to end from eager launches and from a
    captured graph, the per-layer breakdown (graph-captured repeats), and
    the oracle's wall time on the same stack."""
    s5 = Step(5)
    s5.choose(args.kernel, max(args.reps // 2, 20), graph=True)
    steps = max(args.steps // 5, 20)
    wall, ev_s = time_steps(s5, steps, max(args.warmup // 5, 5))
    graph_s = time_graph_steps(s5, steps)
    ops = sum(l.binary_ops for l in s5.layers)
    layers = []
    for pack, call, layer, kind, times in zip(s5.packs, s5.calls, s5.layers, s5.kinds,
                                              s5.times):
        if pack is not None:
            layers.append(bitpack_record(layer, time_repeated(pack, args.reps, graph=True)))
        # a float-input layer's line covers bitpack + conv, or the fused launch
        layers.append(layer_record(layer, time_repeated(call, args.reps, graph=True), probe,
                                   kind, times))
    rec = {"workload": "stack16: " + __import__("workloads").CONFIG_NAMES[5],
           "binary_ops": ops, "steps": steps,
           "eager_us": round(wall * 1e6 / steps, 2),
           "eager_event_us": round(ev_s * 1e6 / steps, 2),
           "graph_us": round(graph_s * 1e6, 2),
           "binary_gops_eager": round(ops / (wall / steps) / 1e9, 1),
           "binary_gops_graph": round(ops / graph_s / 1e9, 1),
           "kernels": s5.kinds, "layers": layers}
    if not args.no_cpu:
        import oracle
        t0 = time.perf_counter()
        oracle_pass(5, s5.layers[0].n)
        dt = time.perf_counter() - t0
        rec["cpu_oracle"] = {"us": round(dt * 1e6, 1), "binary_gops": round(ops / dt / 1e9, 3),
                             "cores": oracle.num_threads(), "kind": "oracle",
                             "sample": "the whole stack, all 16 images, once"}
    return rec


def oracle_pass(cfg_idx: int, images: int):
    """One pass of the oracle over a configuration's layers (its first
    `images` images), chained like the device pass; returns binary ops."""
    import oracle
    from workloads import config, make_layer_inputs
    layers = config(cfg_idx)
    ops, prev = 0, None
    for i, layer in enumerate(layers):
        inp = make_layer_inputs(layer, 0, cfg_idx, i)
        if layer.chained_from is not None:
            a = oracle.unpack(prev, layer.c_in)
        elif inp.x_float is not None:
            a = oracle.binarize(inp.x_float[:images])
        else:
            a = oracle.unpack(inp.x_words[:images], layer.c_in)
        prev = oracle.bconv2d(a, inp.w_sign, stride=layer.strides, padding=layer.padding,
                              clamp_range=layer.clamp or (-(2 ** 31), 2 ** 31 - 1),
                              out=layer.out, mult=inp.mult, bias=inp.bias, thr=inp.thr)
        ops += layer.binary_ops // layer.n * images
    return ops


def cpu_batch1_lines():
    """The oracle on every batch-1 layer (configurations 1, 2, 3), with one
    thread and with every host thread: wall time of one pass each."""
    import oracle
    from workloads import config, make_layer_inputs
    full = oracle.num_threads()
    out = []
    try:
        for threads in (1, full):
            oracle.set_num_threads(threads)
            for cfg in (1, 2, 3):
                for i, layer in enumerate(config(cfg)):
                    inp = make_layer_inputs(layer, 0, cfg, i)
                    t0 = time.perf_counter()
                    reps = 0
                    while True:
                        a = oracle.binarize(inp.x_float)
                        oracle.bconv2d(a, inp.w_sign, stride=layer.strides,
                                       padding=layer.padding,
                                       clamp_range=layer.clamp or (-(2 ** 31), 2 ** 31 - 1),
                                       out=layer.out, mult=inp.mult, bias=inp.bias,
                                       thr=inp.thr)
                        reps += 1
                        if time.perf_counter() - t0 > 0.2 or reps >= 50:
                            break
                    dt = (time.perf_counter() - t0) / reps
                    out.append({"config": cfg, "layer": layer.name, "threads": threads,
                                "us": round(dt * 1e6, 1),
                                "binary_gops": round(layer.binary_ops / dt / 1e9, 3),
                                "kind": "oracle"})
    finally:
        oracle.set_num_threads(full)
    return out


def valu_probe():
    """Achievable xor+popcount rate in binary TOP/s (a pair covers 32 MACs = 64 ops)."""
    import torch
    from paper_2011_09398_amd import build as lb
    L = ctypes.CDLL(lb.PROBE_LIB)
    L.lce_probe_xor_popcount.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
                                         ctypes.c_int, ctypes.c_void_p]
    L.lce_probe_pairs.restype = ctypes.c_longlong
    L.lce_probe_pairs.argtypes = [ctypes.c_int, ctypes.c_int]
    blocks, iters = CUS * 8, 2000
    seed = torch.randint(0, 2 ** 31 - 1, (128,), dtype=torch.int32, device="cuda")
    out = torch.empty(blocks * 256, dtype=torch.int32, device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    fn = lambda: L.lce_probe_xor_popcount(seed.data_ptr(), out.data_ptr(), blocks, iters, st)
    ms = time_repeated(fn, 5, graph=False)
    pairs = L.lce_probe_pairs(blocks, iters)   # one v_xor_b32 + one v_bcnt_u32_b32 each
    return pairs * 2 * BINARY_OPS_PER_LANE_OP / (ms * 1e-3) / 1e12


def cpu_baseline(cfg_idx: int, target_s: float):
    """The oracle, as it stands, on a bounded sample of the same step."""
    import oracle
    from workloads import config

    n = config(cfg_idx)[0].n

    def run(images):
        t0 = time.perf_counter()
        ops = oracle_pass(cfg_idx, images)
        return time.perf_counter() - t0, ops

    dt, ops = run(1)
    images = int(max(1, min(n, target_s / max(dt, 1e-6))))
    reps = 1
    if images > 1:
        dt, ops = run(images)
        while images == n and dt < target_s and reps < 20:   # full step, repeated
            dt2, ops2 = run(images)
            dt, ops, reps = dt + dt2, ops + ops2, reps + 1
    return {"value": round(ops / dt / 1e9, 3), "unit": "GOPS", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"the whole step on {images} of {n} images, {reps} pass(es) "
                      f"({ops / 1e9:.2f} G binary ops, {dt:.2f} s wall)",
            "cpu": cpu_model()}


def cpu_model() -> str:
    """The host CPU's model name (/proc/cpuinfo), else the platform's."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def measured_traffic(layer_name, kind):
    """HBM bytes per launch from the committed counter summary, or None when
    the kernel sources have changed since those counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles",
                        "bconv2d_qn-b64_traffic.json" if kind == "xor"
                        else "bconv2d_mfma_qn-b64_traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    h = hashlib.sha256()
    for f in rec["kernel_sources"]:
        h.update(open(os.path.join(ROOT, f), "rb").read())
    if h.hexdigest() != rec["kernel_sources_sha256"]:
        return None
    return rec["per_launch_bytes"].get(layer_name)


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU: the library has no multi-GPU path "
              f"(--gpus {args.gpus} was requested)", file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    ensure_built()
    import paper_2011_09398_amd as lce
    from workloads import CONFIG_NAMES
    lce.lib()

    if args.sweep_only:
        # diagnostic run (kernel traces of the sweep): no step, no contract line
        log("convolution sweep only")
        print(json.dumps({"conv_sweep": sweep_lines(args)}), flush=True)
        return

    cfg_idx = 4 if args.workload == "b64" else 5
    step = Step(cfg_idx)
    if args.profile_pass:
        # Counter runs: the byte-counter calibration copies, then every layer
        # in order, three launches of each implementation (xor, then mfma).
        src = torch.ones(128 * 2 ** 20, dtype=torch.float32, device="cuda")   # 512 MiB
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        for pack, x, m in zip(step.packs, step.xor_calls, step.mfma_calls):
            if pack is not None:
                pack()
            for call in (x, m):
                for _ in range(3):
                    call()
        torch.cuda.synchronize()
        probe = valu_probe()   # 5 warmup + 5 timed launches of the xor+popcount probe
        log("profile pass done: 3 copies of 512 MiB, 3 launches of each implementation "
            f"per layer, 10 launches of the VALU probe ({probe:.1f} binary TOP/s)")
        return
    log(f"choosing the convolution implementation per layer ({args.kernel})")
    step.choose(args.kernel, max(args.reps // 2, 20))
    log(f"timing config {cfg_idx}: {args.warmup} warmup + {args.steps} steps")
    wall, ev_s = time_steps(step, args.steps, args.warmup)
    ms_per_step = wall * 1e3 / args.steps
    total_ops = sum(l.binary_ops for l in step.layers)
    value = total_ops / (ms_per_step * 1e-3) / 1e9

    probe = None
    if not args.no_probe:
        log("VALU xor+popcount probe")
        probe = valu_probe()

    log(f"per-launch timing, {TRIALS} trials of {args.reps} launches each")
    layers = []
    for pack, call, layer, kind, times, inp in zip(step.packs, step.calls, step.layers,
                                                   step.kinds, step.times, step.inputs):
        if pack is not None:   # the layer's line below covers bitpack + conv
            layers.append(bitpack_record(layer, time_repeated(pack, args.reps, graph=False)))
        ms, spread = trial_fields(time_trials(call, args.reps, graph=False))
        r = layer_record(layer, ms, probe, kind, times)
        r.update(spread)
        r["inputs_sha256"] = inputs_digest(inp)
        layers.append(r)
    conv = [r for r in layers if "binary_ops" in r]
    dom = max(conv, key=lambda r: r["us"])
    roofline = roofline_record(dom, dom["kernel"], cfg_idx, probe)
    # The paper's method (XOR + POPCOUNT on the VALU) on the same layers,
    # against the VALU peak, whichever implementation the step uses.
    xor_layers = []
    for call, layer in zip(step.xor_calls, step.layers):
        ms, spread = trial_fields(time_trials(call, args.reps, graph=False))
        r = layer_record(layer, ms, probe, "xor")
        r.update(spread)
        xor_layers.append(r)
    roofline_valu = roofline_record(max(xor_layers, key=lambda r: r["us"]), "xor", cfg_idx,
                                    probe)
    roofline_valu["layers_valu_frac"] = {r["layer"]: r["valu_frac"] for r in xor_layers}

    zero_pad = mem_lines = None
    if not args.no_extra:
        log("zero-padding variant of the step's layers")
        zero_pad = zero_padding_lines(step, args.reps, probe)
        log("memory-bound operators beyond the last-level cache")
        mem_lines = memory_bound_lines(args.reps)

    batch1 = None
    if not args.no_batch1:
        log("batch-1 configurations 1, 2, 3 (graph-captured repeats)")
        batch1 = batch1_lines(args, probe)

    stack = None
    if not args.no_stack:
        log("configuration 5: the 12-layer batch-16 stack, eager and graph")
        stack = stack_lines(args, probe)

    sweep = None
    if not args.no_sweep:
        log("convolution sweep (graph-captured repeats, both kernels)")
        sweep = sweep_lines(args, probe)

    cpu = cpu_b1 = None
    if not args.no_cpu:
        log("CPU oracle sample")
        cpu = cpu_baseline(cfg_idx, args.cpu_seconds)
        log("CPU oracle on the batch-1 layers, one thread and all threads")
        cpu_b1 = cpu_batch1_lines()

    kinds = set(step.kinds)
    dtype = " + ".join(DTYPES[k] for k in sorted(kinds))
    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "GOPS", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": dtype,
        "data": "synthetic",
        "config": {"workload": ("qn-b64: " if cfg_idx == 4 else "stack16: ")
                   + CONFIG_NAMES[cfg_idx],
                   "batch": step.layers[0].n,
                   "layers": [l.name for l in step.layers],
                   "kernels": step.kinds,
                   "binary_ops_per_step": total_ops},
        "event_ms_per_step": round(ev_s * 1e3 / args.steps, 5),
        "roofline": roofline, "roofline_valu": roofline_valu, "cpu_baseline": cpu,
        "layers": layers, "batch1": batch1, "stack16": stack, "cpu_batch1": cpu_b1,
        "zero_padding": zero_pad, "memory_bound": mem_lines, "conv_sweep": sweep,
        "valu_probe": None if probe is None else {
            "binary_tops": round(probe, 1), "spec_binary_tops": round(PEAK_BINARY_TOPS, 1)},
        "device": torch.cuda.get_device_name(0),
    }
    print(json.dumps(line), flush=True)


def roofline_record(rec, kind, cfg_idx, probe):
    """The roofline object of one launch record: binary ops per launch over
    its average duration, against the peak of the unit that ran it."""
    if kind in ("xor", "fused"):
        r = {"bound": "alu", "achieved": round(rec["binary_gops"] / 1e3, 2),
             "peak": round(PEAK_BINARY_TOPS, 1), "unit": "TOP/s", "frac": rec["valu_frac"],
             "traffic": measured_traffic(rec["layer"], "xor") if cfg_idx == 4 else None,
             "kernel": f"bconv2d{' (quantize-fused)' if kind == 'fused' else ''} "
                       f"(xor+popcount, VALU) {rec['layer']} (batch {rec['batch']})",
             "probe_peak": None if probe is None else round(probe, 1),
             "probe_frac": rec.get("probe_frac")}
    else:
        r = {"bound": "mfma", "achieved": round(rec["binary_gops"] / 1e3, 2),
             "peak": PEAK_FP4_TFLOPS, "unit": "TFLOP/s", "frac": rec["mfma_fp4_frac"],
             "traffic": measured_traffic(rec["layer"], "mfma") if cfg_idx == 4 else None,
             "kernel": f"bconv2d_mfma{' (quantize-fused)' if kind == 'fused_mfma' else ''} "
                       f"(fp4 e2m1 MFMA) {rec['layer']} (batch {rec['batch']})"}
    r.update({"per_launch_binary_ops": rec["binary_ops"], "avg_launch_us": rec["us"]})
    return r


if __name__ == "__main__":
    main()
