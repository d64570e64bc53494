"""Mutation test of the oracle's pins (CPU only).

Each case plants one plausible mistake in a copy of ``oracle/cd_oracle.c``:
- a flipped comparison;
- a dropped term, factor or token;
- a wrong sign;
- a transposed operand;
- an off-by-one.

The copy is built with the oracle's own compiler line, and the pin tests
(``tests/test_oracle_pins.py``) run against it in a subprocess through
``CD_ORACLE_LIB``. Every mutant must make them fail; the unmodified copy, built
the same way, must pass. The oracle's source itself is never changed.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "cd_oracle.c")
PINS = os.path.join(ROOT, "tests", "test_oracle_pins.py")

# name: (text of the oracle, the mistake put in its place[, occurrences, which one]);
# a text occurs once unless the entry says otherwise
MUTANTS = {
    "threshold >= instead of strict >": (
        "            if (v > thld)\n                keep = 1;",
        "            if (v >= thld)\n                keep = 1;"),
    "SiLU sign for z >= 0": (
        "return z / (1.0 + exp(-z));", "return z / (1.0 + exp(z));"),
    "SiLU numerator for z < 0": (
        "return z * e / (1.0 + e);", "return z / (1.0 + e);"),
    "union over the batch reduced to token 0": (
        "        for (int b = 0; b < B; b++) {\n            double v = c[(int64_t)b * d_ff + i];",
        "        for (int b = 0; b < 1; b++) {\n            double v = c[(int64_t)b * d_ff + i];"),
    "absolute value dropped": (
        "            if (use_abs)\n                v = fabs(v);\n", ""),
    "coefficient s dropped from Eq. 5": (
        "acc += sb[idx[t]] * wide(W_down[(int64_t)idx[t] * d_model + j]);",
        "acc += wide(W_down[(int64_t)idx[t] * d_model + j]);"),
    "quantile position k n instead of k (n - 1)": (
        "double h = k * (double)(n - 1);", "double h = k * (double)n;"),
    "quantile without interpolation": (
        "        q = w[lo] + (h - (double)lo) * (w[lo + 1] - w[lo]);", "        q = w[lo];"),
    "calibration mean over T - 1": (
        "return sum / (double)T;", "return sum / (double)(T > 1 ? T - 1 : 1);"),
    "residual subtracted": ("h[j] += y[j];", "h[j] -= y[j];"),
    "RMSNorm eps outside the root": (
        "sqrt(ss / (double)d_model + eps)", "(sqrt(ss / (double)d_model) + eps)"),
    "last term of x.W dropped": (
        "        for (int64_t j = 0; j < cols; j++)\n            acc += vd[j] * wide(w[j]);",
        "        for (int64_t j = 0; j < cols - 1; j++)\n            acc += vd[j] * wide(w[j]);"),
    "predictor second product transposed": (
        "            acc += v[j] * wide(w[j]);", "            acc += v[j] * wide(W[j * rows + i]);"),
    "ternary weights taken as 0/1": (
        "t += wide(xb[j]) * (double)theta_t[i * d_model + j];",
        "t += wide(xb[j]) * (double)(theta_t[i * d_model + j] != 0);"),
    "gate and up exchanged in s": (
        "= uu[i] * cdo_silu(gg[i]);", "= gg[i] * cdo_silu(uu[i]);"),
    "CATS coefficient without SiLU": (
        "            hb[i] = cdo_silu(hb[i]);", "            hb[i] = hb[i];"),
    "CATS calibration coefficient without SiLU": (
        "            c[i] = cdo_silu(c[i]);", "            c[i] = c[i];"),
    "per-token path: token 0's threshold for every token": (
        "            if (c[(int64_t)b * d_ff + i] > q[b])",
        "            if (c[(int64_t)b * d_ff + i] > q[0])"),
    "per-token path: quantile at 1 - k": (
        "        q[b] = cdo_quantile_linear(k, cb, d_ff);",
        "        q[b] = cdo_quantile_linear(1.0 - k, cb, d_ff);"),
    "dense path: last neuron dropped": (
        "            for (int64_t i = 0; i < d_ff; i++)\n                acc += s[i] * wide(W_down[i * d_model + j]);",
        "            for (int64_t i = 0; i < d_ff - 1; i++)\n                acc += s[i] * wide(W_down[i * d_model + j]);"),
    "dense path: W_down read transposed": (
        "acc += s[i] * wide(W_down[i * d_model + j]);", "acc += s[i] * wide(W_down[j * d_ff + i]);"),
    "index-restricted FFN: gate from W_up": (
        "            double gg = row_dot(xb, W_gate, i, d_model);\n            s[(int64_t)b * d_ff + i] = uu * cdo_silu(gg);",
        "            double gg = row_dot(xb, W_up, i, d_model);\n            s[(int64_t)b * d_ff + i] = uu * cdo_silu(gg);"),
    "index-restricted FFN: compact s of token 0 for every token": (
        "s_c[(int64_t)b * n + t] = s[(int64_t)b * d_ff + idx[t]];",
        "s_c[(int64_t)b * n + t] = s[idx[t]];"),
    # the low-rank predictor's call (the first of two identical lines; the second is the
    # ternary predictor's)
    "low-rank predictor score thresholded as |s_hat|": (
        "    int64_t n = cdo_select(sh, B, d_ff, 0, thld, idx);",
        "    int64_t n = cdo_select(sh, B, d_ff, 1, thld, idx);", 2, 0),
    "ternary predictor score thresholded as |s_hat|": (
        "    int64_t n = cdo_select(sh, B, d_ff, 0, thld, idx);",
        "    int64_t n = cdo_select(sh, B, d_ff, 1, thld, idx);", 2, 1),
}


def build(text, out_dir, name):
    src = os.path.join(out_dir, name + ".c")
    lib = os.path.join(out_dir, name + ".so")
    with open(src, "w") as f:
        f.write(text)
    subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-o", lib, src,
                    "-lm"], check=True, capture_output=True)
    return lib


def run_pins(lib):
    env = dict(os.environ, CD_ORACLE_LIB=lib, OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        PINS], cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    return r.returncode, r.stdout[-2000:]


@pytest.fixture(scope="module")
def source():
    with open(SRC) as f:
        return f.read()


def test_unmodified_copy_passes(source, tmp_path):
    rc, out = run_pins(build(source, str(tmp_path), "control"))
    assert rc == 0, out


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, source, tmp_path):
    old, new, count, nth = (MUTANTS[name] + (1, 0))[:4]
    assert source.count(old) == count, f"mutation target of {name!r} changed"
    at = -1
    for _ in range(nth + 1):
        at = source.index(old, at + 1)
    text = source[:at] + new + source[at + len(old):]
    rc, out = run_pins(build(text, str(tmp_path), "mutant"))
    # 1: tests ran and some failed (not a crash, a collection error or an interrupt)
    assert rc == 1, f"{name}: pins did not catch it (pytest exit {rc})\n{out}"
