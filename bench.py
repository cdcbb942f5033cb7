"""Benchmark of the bitpacked binary convolution on one MI355X.

A step is one pass over the batch-64 QuickNet-shaped layers (bitpacked
input, bitpacked output): 56x56x64->128 stride 2, whose output feeds
28x28x128->128, then 14x14x256->256 and 7x7x512->512.  The JSON line also
carries the batch-1 layers (float input through lce_bitpack, timed as its
own line) as per-layer microseconds, the roofline of the dominant kernel,
and the CPU oracle timed on a bounded sample of the same step.

    python bench.py [--steps K] [--warmup W] [--no-cpu] [--workload b64|stack16]
"""
from __future__ import annotations

import argparse
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
HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", choices=("b64", "stack16"), default="b64")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-batch1", action="store_true", help="skip the batch-1 lines")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="target wall time of the CPU baseline sample")
    return ap.parse_args()


def ensure_built():
    from paper_2011_09398_amd import build as lb
    if not os.path.exists(lb.LIB):
        lb.build()


class Step:
    """Device buffers and prepared calls for one config's layers."""

    def __init__(self, cfg_idx: int):
        import numpy as np
        import torch
        import paper_2011_09398_amd as lce
        from workloads import config, make_layer_inputs

        self.layers = config(cfg_idx)
        self.inputs = [make_layer_inputs(l, 0, cfg_idx, i) for i, l in enumerate(self.layers)]
        dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
        self.calls, self.outs, self.keep = [], [], []
        self.x_float = None
        self.pack_call = None
        for i, (layer, inp) in enumerate(zip(self.layers, self.inputs)):
            w_packed = lce.bitpack(dev(inp.w_float))          # 1-bit weight storage
            if layer.chained_from is not None:
                x_packed = self.outs[layer.chained_from]
            elif inp.x_float is not None:
                xf = dev(inp.x_float)
                x_packed = lce.bitpack(xf)
                self.x_float = (xf, x_packed)
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
            self.calls.append(lce.PreparedBConv2d(
                x_packed, w_packed, layer.c_in, out, stride=layer.strides,
                padding=layer.padding, clamp=layer.clamp, out_type=layer.out, **kw))
            self.outs.append(out)
            self.keep.append((w_packed, x_packed, kw))

    def bitpack(self):
        import paper_2011_09398_amd as lce
        xf, xp = self.x_float
        lce.bitpack(xf, out=xp)


def time_step(step: Step, steps: int, warmup: int, with_bitpack: bool):
    """Time `steps` passes; per-launch HIP event durations on the launch stream."""
    import torch
    ncalls = len(step.calls) + (1 if with_bitpack else 0)

    def run(evs=None):
        k = 0
        if evs is not None:
            evs[0].record()
        if with_bitpack:
            step.bitpack()
            if evs is not None:
                evs[1].record()
            k = 1
        for i, call in enumerate(step.calls):
            call()
            if evs is not None:
                evs[k + i + 1].record()

    for _ in range(warmup):
        run()
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(ncalls + 1)]
              for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(steps):
        run(events[s])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per_call_ms = [sum(events[s][i].elapsed_time(events[s][i + 1]) for s in range(steps)) / steps
                   for i in range(ncalls)]
    return wall, per_call_ms


def layer_record(layer, ms):
    ops = layer.binary_ops
    tops = ops / (ms * 1e-3) / 1e12
    return {"layer": layer.name, "batch": layer.n, "us": round(ms * 1e3, 3),
            "binary_gops": round(tops * 1e3, 1),
            "valu_frac": round(tops / PEAK_BINARY_TOPS, 4), "binary_ops": ops}


def bitpack_record(layer, ms):
    n_float = layer.n * layer.h * layer.w * layer.c_in
    nbytes = 4 * n_float + 4 * layer.n * layer.h * layer.w * layer.cw
    gbs = nbytes / (ms * 1e-3) / 1e9
    return {"layer": f"bitpack {layer.n}x{layer.h}x{layer.w}x{layer.c_in}", "batch": layer.n,
            "us": round(ms * 1e3, 3), "bytes": nbytes, "GB/s": round(gbs, 1),
            "hbm_frac": round(gbs / HBM_PEAK_GBS, 4)}


def cpu_baseline(cfg_idx: int, target_s: float):
    """The oracle, as it stands, on a bounded sample of the same step."""
    import numpy as np
    import oracle
    from workloads import config, make_layer_inputs

    layers = config(cfg_idx)
    inputs = [make_layer_inputs(l, 0, cfg_idx, i) for i, l in enumerate(layers)]

    def run(images):
        ops, prev = 0, None
        t0 = time.perf_counter()
        for layer, inp in zip(layers, inputs):
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
        return time.perf_counter() - t0, ops

    n = layers[0].n
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
            "cpu": platform.processor() or platform.machine()}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU: this build has no multi-GPU path "
              f"(--gpus {args.gpus} was requested)", file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    ensure_built()
    import paper_2011_09398_amd as lce
    lce.lib()

    cfg_idx = 4 if args.workload == "b64" else 5
    step = Step(cfg_idx)
    with_bp = step.x_float is not None and cfg_idx == 5
    print(f"[bench] timing config {cfg_idx}: {args.warmup} warmup + {args.steps} steps",
          file=sys.stderr, flush=True)
    wall, per_call = time_step(step, args.steps, args.warmup, with_bp)
    ms_per_step = wall * 1e3 / args.steps
    total_ops = sum(l.binary_ops for l in step.layers)
    value = total_ops / (ms_per_step * 1e-3) / 1e9

    layer_ms = per_call[1:] if with_bp else per_call
    layers = [layer_record(l, ms) for l, ms in zip(step.layers, layer_ms)]
    if with_bp:
        layers.insert(0, bitpack_record(step.layers[0], per_call[0]))
    conv = [r for r in layers if "binary_ops" in r]
    dom = max(conv, key=lambda r: r["us"])
    roofline = {"bound": "alu", "achieved": round(dom["binary_gops"] / 1e3, 2),
                "peak": round(PEAK_BINARY_TOPS, 1), "unit": "TOP/s",
                "frac": dom["valu_frac"], "traffic": None,
                "kernel": f"bconv2d {dom['layer']} (batch {dom['batch']})",
                "per_launch_binary_ops": dom["binary_ops"], "avg_launch_us": dom["us"]}

    batch1 = None
    if not args.no_batch1:
        print("[bench] timing batch-1 layers", file=sys.stderr, flush=True)
        s1 = Step(3)
        recs = []
        import paper_2011_09398_amd as lce  # noqa: F811
        for i, call in enumerate(s1.calls):
            layer, inp = s1.layers[i], s1.inputs[i]
            # bitpack of this layer's float input, then the conv, each timed alone
            xf = torch.from_numpy(inp.x_float).cuda()
            xp = call.keep[0]
            for name, fn in (("bitpack", lambda: lce.bitpack(xf, out=xp)), ("conv", call)):
                for _ in range(20):
                    fn()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                reps = 200
                e0.record()
                for _ in range(reps):
                    fn()
                e1.record()
                torch.cuda.synchronize()
                ms = e0.elapsed_time(e1) / reps
                recs.append(bitpack_record(layer, ms) if name == "bitpack"
                            else layer_record(layer, ms))
        batch1 = recs

    cpu = None
    if not args.no_cpu:
        print("[bench] timing the CPU oracle sample", file=sys.stderr, flush=True)
        cpu = cpu_baseline(cfg_idx, args.cpu_seconds)

    from workloads import CONFIG_NAMES
    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "GOPS", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u32",
        "data": "synthetic",
        "config": {"workload": ("qn-b64: " if cfg_idx == 4 else "stack16: ")
                   + CONFIG_NAMES[cfg_idx],
                   "batch": step.layers[0].n,
                   "layers": [l.name for l in step.layers],
                   "binary_ops_per_step": total_ops},
        "roofline": roofline, "cpu_baseline": cpu, "layers": layers, "batch1": batch1,
        "device": torch.cuda.get_device_name(0),
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
