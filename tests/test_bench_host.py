"""Host-side helpers of bench.py: the per-layer trial statistics, the input
digests logged beside each headline layer, and the CPU model reported with
the oracle's timing."""
import math

import bench
from workloads import config, make_layer_inputs, sha256


def test_trial_fields_median_and_spread():
    ms, spread = bench.trial_fields([0.003, 0.001, 0.002, 0.005, 0.004])
    assert math.isclose(ms, 0.003)
    assert spread["trials"] == 5
    # numpy's linear percentiles of 1..5 us: p10 = 1.4, p90 = 4.6
    assert math.isclose(spread["us_p10"], 1.4)
    assert math.isclose(spread["us_p90"], 4.6)


def test_inputs_digest_names_every_generated_tensor():
    layer = config(1)[0]
    inp = make_layer_inputs(layer, 0, 1, 0)
    d = bench.inputs_digest(inp)
    assert set(d) == {n for n in ("x_float", "x_words", "w_float", "mult", "bias", "thr")
                      if getattr(inp, n, None) is not None}
    for name, h in d.items():
        assert h == sha256(getattr(inp, name))[:16]
    # the same seed gives the same digests
    assert bench.inputs_digest(make_layer_inputs(layer, 0, 1, 0)) == d


def test_cpu_model_is_named():
    assert isinstance(bench.cpu_model(), str) and bench.cpu_model()
