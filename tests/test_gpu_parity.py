"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Integer and bitpacked outputs must match bit for bit; float outputs within
1e-6 relative.  Output buffers are pre-poisoned (0xAA bytes) so an element
the kernels fail to write, or a dirty pad bit, shows up as a mismatch.
"""
import numpy as np
import pytest

import oracle
from tests.layer_util import (POISON_I32, assert_match, config4_reference, dev, gpu_input,
                              gpu_layer, gpu_pack_weights, oracle_layer, oracle_signs)
from workloads import INT32_MAX, INT32_MIN, Layer, config, make_layer_inputs

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


# ---------------------------------------------------------------- bitpack (LceQuantize)

@pytest.mark.parametrize("rows,c", [(1, 32), (7, 64), (1000, 64), (3, 1), (5, 31), (9, 33),
                                    (11, 40), (6, 100), (4, 256), (257, 96), (33, 512),
                                    (1, 4096)])
def test_bitpack_parity(rows, c):
    import torch
    import paper_2011_09398_amd as lce
    rng = np.random.default_rng(rows * 1000 + c)
    x = rng.standard_normal((rows, c), dtype=np.float32)
    flat = x.reshape(-1)
    special = np.array([-0.0, 0.0, np.nan, -np.nan, np.inf, -np.inf, 1e-45, -1e-45], np.float32)
    flat[: min(flat.size, special.size)] = special[: min(flat.size, special.size)]
    out = torch.full((rows, (c + 31) // 32), POISON_I32, dtype=torch.int32, device="cuda")
    lce.bitpack(dev(x), out=out)
    got = sync_np(out).view(np.uint32)
    assert np.array_equal(got, oracle.pack(oracle.binarize(x)))


@pytest.mark.parametrize("offset_floats", [1, 2, 3])
def test_bitpack_unaligned_input(offset_floats):
    import torch
    import paper_2011_09398_amd as lce
    rng = np.random.default_rng(offset_floats)
    x = rng.standard_normal((50, 64), dtype=np.float32)
    base = torch.zeros(50 * 64 + 8, dtype=torch.float32, device="cuda")
    view = base[offset_floats: offset_floats + 50 * 64].view(50, 64)
    view.copy_(dev(x))
    got = sync_np(lce.bitpack(view)).view(np.uint32)
    assert np.array_equal(got, oracle.pack(oracle.binarize(x)))


def test_bitpack_large_tail():
    # 16x56x56x64 floats: the fast path's grid-stride loop plus a ragged chunk.
    import paper_2011_09398_amd as lce
    rng = np.random.default_rng(5)
    x = rng.standard_normal((16 * 56 * 56 + 3, 64), dtype=np.float32)
    got = sync_np(lce.bitpack(dev(x))).view(np.uint32)
    assert np.array_equal(got, oracle.pack(oracle.binarize(x)))


def test_weight_packing_matches_oracle():
    layer = config(4)[3]
    inp = make_layer_inputs(layer, 0, 4, 3)
    got = sync_np(gpu_pack_weights(inp)).view(np.uint32)
    assert got.shape == (512, 3, 3, 16)
    assert got.nbytes == 512 * 9 * 512 // 8
    assert np.array_equal(got, oracle.pack(inp.w_sign))


# ---------------------------------------------------------------- the five configurations

@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_config_parity_full(cfg):
    for i, layer in enumerate(config(cfg)):
        inp = make_layer_inputs(layer, 0, cfg, i)
        got = sync_np(gpu_layer(layer, inp))
        ref = oracle_layer(layer, inp, oracle_signs(inp))
        assert_match(layer, got, ref, f"config {cfg} layer {layer.name}")


def test_config4_full_batch_chained():
    """Batch 64, launched exactly as timed, every output of every layer
    compared with the oracle.  The stride-2 layer's bitpacked output feeds
    the 28x28x128 layer on both sides (the chain)."""
    prev_gpu = None
    for layer, inp, ref in config4_reference(chain=True):
        if layer.chained_from is not None:
            got = gpu_layer(layer, inp, x_packed=prev_gpu)
        else:
            got = gpu_layer(layer, inp)
        assert_match(layer, sync_np(got), ref, f"config 4 layer {layer.name}")
        prev_gpu = got


def test_config5_chain_every_layer():
    layers = config(5)
    prev_gpu = prev_ref = None
    for i, layer in enumerate(layers):
        inp = make_layer_inputs(layer, 0, 5, i)
        if i == 0:
            got = gpu_layer(layer, inp)
            a = oracle_signs(inp)
        else:
            got = gpu_layer(layer, inp, x_packed=prev_gpu)
            a = oracle.unpack(prev_ref, layer.c_in)
        ref = oracle_layer(layer, inp, a)
        assert_match(layer, sync_np(got), ref, f"config 5 {layer.name}")
        prev_gpu, prev_ref = got, ref


# ---------------------------------------------------------------- property sweep

def sweep_cases():
    rng = np.random.default_rng(2024)
    cases = []
    for i in range(72):
        k = int(rng.choice([1, 2, 3, 3, 3, 5]))
        kw = k if rng.random() < 0.8 else int(rng.choice([1, 3]))
        s = int(rng.choice([1, 1, 2, 3]))
        sw_ = s if rng.random() < 0.8 else int(rng.choice([1, 2]))
        padding = "same" if rng.random() < 0.7 else "valid"
        h = int(rng.integers(max(k, 1), 10))
        w = int(rng.integers(max(kw, 1), 10))
        c_in = int(rng.choice([1, 7, 32, 33, 64, 96, 100, 128, 160, 512]))
        c_out = int(rng.choice([1, 5, 8, 13, 32, 40, 64, 100]))
        n = int(rng.integers(1, 4))
        out = ["float", "bitpacked", "int32"][i % 3]
        kk = k * kw * c_in
        clamp = [None, (-kk, kk), (0, kk), (-3, 3), (0, 0)][int(rng.integers(0, 5))]
        cases.append(Layer(f"sweep{i}", n, h, w, c_in, c_out, kh=k, kw=kw, stride=s,
                           stride_w=sw_, padding=padding, out=out, clamp=clamp,
                           input_kind=["float", "bits"][i % 2]))
    return cases


@pytest.mark.parametrize("layer", sweep_cases(), ids=lambda l: l.name)
def test_property_sweep(layer):
    inp = make_layer_inputs(layer, 7, 99, int(layer.name[5:]))
    run_case(layer, inp)


# ---------------------------------------------------------------- edge cases

def run_case(layer, inp, **override):
    got = sync_np(gpu_layer(layer, inp, **override))
    ref = oracle_layer(layer, inp, oracle_signs(inp))
    assert_match(layer, got, ref, layer.name)
    return got, ref


def test_special_thresholds():
    layer = Layer("thr", 2, 9, 7, 64, 40, out="bitpacked", input_kind="bits")
    inp = make_layer_inputs(layer, 1, 50, 0)
    thr = inp.thr.copy()
    thr[:6] = [np.nan, np.inf, -np.inf, 0.0, -0.0, 3.4e38]
    # thresholds exactly at reachable accumulator values (dot is odd/even like K)
    thr[6:20] = np.arange(-14, 14, 2, dtype=np.float32)
    thr[20:25] = np.array([1.0, -1.0, 2.0, 0.5, -0.5], np.float32)
    inp.thr = thr
    got, ref = run_case(layer, inp)
    assert not (got.view(np.uint32)[..., 1] >> 8).any()   # pad bits of word 1 are zero


@pytest.mark.parametrize("clamp", [(INT32_MIN, INT32_MAX), (0, 0), (-576, 576), (0, 576),
                                   (2 ** 30 + 1, 2 ** 30 + 1), (-(2 ** 31), -(2 ** 30) - 3)])
@pytest.mark.parametrize("out", ["float", "int32", "bitpacked"])
def test_clamp_edges(clamp, out):
    layer = Layer("clamp", 1, 10, 10, 64, 24, out=out, clamp=clamp)
    inp = make_layer_inputs(layer, 2, 51, 0)
    run_case(layer, inp)


def test_float_out_without_multiplier_and_bias_is_the_accumulator():
    import paper_2011_09398_amd as lce
    layer = Layer("nomb", 1, 6, 6, 96, 16, out="float")
    inp = make_layer_inputs(layer, 3, 52, 0)
    got = sync_np(lce.bconv2d(gpu_input(inp), gpu_pack_weights(inp), 96, out_type="float"))
    ref = oracle.bconv2d(oracle_signs(inp), inp.w_sign, out="int32")
    assert np.array_equal(got, ref.astype(np.float32))


@pytest.mark.parametrize("h,w,k,s", [(1, 1, 3, 1), (1, 1, 5, 2), (2, 1, 3, 1), (3, 3, 3, 3)])
def test_tiny_images(h, w, k, s):
    layer = Layer("tiny", 3, h, w, 64, 64, kh=k, kw=k, stride=s, out="int32")
    run_case(layer, make_layer_inputs(layer, 4, 53, 0))


@pytest.mark.parametrize("offset_words", [1, 2])
def test_unaligned_packed_input_takes_narrow_loads(offset_words):
    import torch
    layer = Layer("unal", 2, 14, 14, 128, 64, out="bitpacked", input_kind="bits")
    inp = make_layer_inputs(layer, 5, 54, 0)
    words = inp.x_words.view(np.int32)
    base = torch.zeros(words.size + 8, dtype=torch.int32, device="cuda")
    xp = base[offset_words: offset_words + words.size].view(words.shape)
    xp.copy_(dev(words))
    run_case(layer, inp, x_packed=xp)


def test_ragged_pixels_and_filters():
    # M = 2*13*11 = 286 (not a multiple of 64); 100 filters (not a multiple of 8 or 32)
    for out in ("float", "bitpacked", "int32"):
        layer = Layer("ragged", 2, 13, 11, 160, 100, out=out, input_kind="bits")
        run_case(layer, make_layer_inputs(layer, 6, 55, 0))


def test_all_plus_one_input_gives_filter_sums_on_gpu():
    import torch
    import paper_2011_09398_amd as lce
    layer = Layer("ones", 2, 7, 7, 256, 32, out="int32")
    inp = make_layer_inputs(layer, 8, 56, 0)
    x = torch.zeros((2, 7, 7, 8), dtype=torch.int32, device="cuda")   # all bits 0 = all +1
    got = sync_np(lce.bconv2d(x, gpu_pack_weights(inp), 256, out_type="int32"))
    sums = inp.w_sign.astype(np.int64).sum(axis=(1, 2, 3))
    assert np.array_equal(got, np.broadcast_to(sums, got.shape))


def test_repeated_launches_are_deterministic():
    layer = config(4)[2]
    inp = make_layer_inputs(layer, 0, 4, 2)
    xp, wp = gpu_input(inp), gpu_pack_weights(inp)
    a = sync_np(gpu_layer(layer, inp, x_packed=xp, w_packed=wp))
    for _ in range(3):
        assert np.array_equal(sync_np(gpu_layer(layer, inp, x_packed=xp, w_packed=wp)), a)


def test_graph_replay_matches_eager():
    """A captured graph of the batch-1 step (bitpack + conv per layer) replays
    to the eager result every time, with eager work and syncs in between."""
    import torch
    import bench
    step = bench.Step(3)
    step.run()
    torch.cuda.synchronize()
    ref = [o.clone() for o in step.outs]
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            step.run()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for _ in range(4):
        for o in step.outs:
            o.fill_(POISON_I32)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for o, r in zip(step.outs, ref):
            assert torch.equal(o, r)
        step.run()                     # eager work between replays
        torch.cuda.synchronize()


SCHEDULES = [(1, 1), (2, 1), (3, 1), (4, 1), (1, 2), (1, 4)]


STATIC = [(3, cw) for cw in (1, 2, 3, 4, 5, 6, 8, 16)] + [(5, cw) for cw in (1, 2, 3, 4, 5, 6, 8)]


@pytest.mark.parametrize("k,cw", STATIC)
@pytest.mark.parametrize("out", ["float", "bitpacked", "int32"])
@pytest.mark.parametrize("stride", [1, 2])
def test_every_static_instance(k, cw, out, stride):
    """Every shape-specialized XOR kernel (3x3 and 5x5 filters, each word
    count with a compile-time unrolled k loop) against the oracle, on a
    channel count that leaves pad bits in the last word."""
    layer = Layer(f"st{k}{cw}{out}{stride}", 2, 9, 11, 32 * cw - 7, 45, kh=k, kw=k,
                  stride=stride, out=out, input_kind="bits",
                  clamp=(-150, 120) if out != "bitpacked" else None)
    run_case(layer, make_layer_inputs(layer, 10 * k + cw, 59, stride))


@pytest.mark.parametrize("nb,ks", SCHEDULES)
@pytest.mark.parametrize("shape", [
    # (n, h, w, c_in, c_out, stride, out)
    (2, 9, 7, 64, 40, 1, "bitpacked"),
    (3, 8, 8, 128, 72, 2, "float"),
    (1, 7, 7, 512, 96, 1, "int32"),
    (2, 5, 6, 256, 130, 1, "bitpacked"),
    (1, 6, 6, 32, 100, 1, "float"),
    (2, 7, 9, 160, 70, 1, "bitpacked", 5),
    (1, 8, 8, 96, 64, 1, "float", 5),
    # filters outweigh the input with several pixel blocks: the tiles are
    # renumbered filter-major per XCD (tile counts not a multiple of 8)
    (3, 9, 9, 256, 200, 1, "bitpacked"),
    (5, 7, 7, 512, 72, 2, "float"),
])
def test_every_schedule_matches_oracle(nb, ks, shape):
    """Every work split of the shape-specialized kernel (filter blocks per
    wave, K split across waves) gives the oracle's result."""
    import paper_2011_09398_amd as lce
    n, h, w, c_in, c_out, s, out = shape[:7]
    k = shape[7] if len(shape) > 7 else 3
    lce.set_tuning(xor_nb=nb, xor_ks=ks)
    layer = Layer(f"sched{nb}{ks}", n, h, w, c_in, c_out, kh=k, kw=k, stride=s, out=out,
                  clamp=(-50, 60) if out != "bitpacked" else None, input_kind="bits")
    run_case(layer, make_layer_inputs(layer, nb * 10 + ks, 60, c_out))


@pytest.mark.parametrize("nb,ks", SCHEDULES)
def test_config4_every_schedule_full(nb, ks):
    """The batch-64 layers (each on its own input) under every XOR work
    split, every output compared."""
    import paper_2011_09398_amd as lce
    lce.set_tuning(xor_nb=nb, xor_ks=ks)
    for layer, inp, ref in config4_reference(chain=False):
        got = sync_np(gpu_layer(layer, inp))
        assert_match(layer, got, ref, f"{layer.name} nb={nb} ks={ks}")
