"""The oracle's pins must catch plausible mistakes in the oracle.

Each case plants one mistake in a temporary copy of oracle/lce_oracle.c
(on the CPU), builds it, and runs the numpy/fraction pins of
test_oracle_pins.py against it: at least one pin has to fail.
"""
import os
import subprocess
import sys

import pytest

from tests.conftest import ROOT

SRC = os.path.join(ROOT, "oracle", "lce_oracle.c")

MUTANTS = {
    "sign_le_zero": ("(x[i] < 0.0f)", "(x[i] <= 0.0f)"),
    "bit_order_msb_first": ("word |= (uint32_t)1 << b;", "word |= (uint32_t)1 << (31 - b);"),
    "unpack_polarity": ("s[r * channels + c] = bit ? (int8_t)-1 : (int8_t)1;",
                        "s[r * channels + c] = bit ? (int8_t)1 : (int8_t)-1;"),
    "zero_padding": ("int32_t av = inside ? arow[ci] : pad;", "int32_t av = inside ? arow[ci] : 0;"),
    "pad_value_ignored": ("int32_t av = inside ? arow[ci] : pad;", "int32_t av = inside ? arow[ci] : 1;"),
    "maxpool_takes_min": ("if (v > best) best = v;", "if (best == -2 || v < best) best = v;"),
    "maxpool_counts_padding": ("if (iy < 0 || iy >= h || ix < 0 || ix >= w) continue;",
                               "if (iy < 0 || iy >= h || ix < 0 || ix >= w) { best = 1; continue; }"),
    "affine_sign_le": ("bits[i] = (uint8_t)(x < 0.0);", "bits[i] = (uint8_t)(x <= 0.0);"),
    "affine_in_float": ("double x = (double)c[i] * (double)mult + (double)bias;",
                        "double x = (double)((float)c[i] * mult + bias);"),
    "same_pad_leading_heavy": ("*pad_before = total / 2;", "*pad_before = (total + 1) / 2;"),
    "ix_uses_ky": ("int ix = ox * sw - pl + kx;", "int ix = ox * sw - pl + ky;"),
    "iy_plus_pad": ("int iy = oy * sh - pt + ky;", "int iy = oy * sh + pt + ky;"),
    "filter_transposed": ("wt + (((int64_t)co * kh + ky) * kw + kx) * c",
                          "wt + (((int64_t)co * kw + kx) * kh + ky) * c"),
    "stride_h_for_w": ("int ix = ox * sw - pl + kx;", "int ix = ox * sh - pl + kx;"),
    "dropped_last_tap_column": ("for (int kx = 0; kx < kw; ++kx) {",
                                "for (int kx = 0; kx + 1 < kw; ++kx) {"),
    "dropped_upper_clamp": ("if (v > hi) v = hi;", ""),
    "bias_sign": ("* mm + bb;", "* mm - bb;"),
    "threshold_le": ("if ((double)c[i * cout + co] < (double)thr[co])",
                     "if ((double)c[i * cout + co] <= (double)thr[co])"),
    "threshold_in_float": ("if ((double)c[i * cout + co] < (double)thr[co])",
                           "if ((float)c[i * cout + co] < thr[co])"),
    "valid_off_by_one": ("*out = (in - k) / s + 1;", "*out = (in - k) / s;"),
}


def build_mutant(tmp_path, name):
    before, after = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(before) >= 1, f"mutation site for {name} not found"
    mutated = src.replace(before, after, 1)
    cpath = tmp_path / f"{name}.c"
    cpath.write_text(mutated)
    lib = tmp_path / f"{name}.so"
    subprocess.run(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-w",
                    "-o", str(lib), str(cpath)], check=True)
    return lib


def run_pins(lib):
    env = dict(os.environ, LCE_ORACLE_LIB=str(lib), OMP_NUM_THREADS="2")
    cmd = [sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
           os.path.join(ROOT, "tests", "test_oracle_pins.py"),
           "-k", "not torch"]
    return subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True)


def test_unmutated_copy_passes(tmp_path):
    lib = tmp_path / "same.so"
    subprocess.run(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-w",
                    "-o", str(lib), SRC], check=True)
    r = run_pins(lib)
    assert r.returncode == 0, r.stdout[-2000:]


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(tmp_path, name):
    r = run_pins(build_mutant(tmp_path, name))
    assert r.returncode != 0, f"mutant {name} survived the pins:\n{r.stdout[-1500:]}"
