"""The pins hold the oracle: a plausible mistake planted in a copy of
oracle.c (a dropped term, a wrong index, sign or bound, a transposed
operand, a wrong rounding rule) must make the pin tests of that function
fail.  Each case rebuilds the mutated copy on the CPU and runs the pin file
in a subprocess against it (KF_ORACLE_SRC); an unmutated copy must pass."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.c")

SOFTMAX = "tests/test_oracle_softmax.py"
CAUSAL = "tests/test_oracle_softmax_causal.py"
GN = "tests/test_oracle_group_norm.py"
LN = "tests/test_oracle_layer_norm.py"
AP = "tests/test_oracle_avgpool.py"
MP = "tests/test_oracle_max_pool.py"
ROUND = "tests/test_oracle_rounding.py"

# (name, text in oracle.c, replacement, occurrences replaced, pin file)
MUTATIONS = [
    ("softmax: no max shift", "double e = exp(xr[j] - m);", "double e = exp(xr[j]);", 1, SOFTMAX),
    ("softmax: sum starts at 0.5", "        double total = 0.0;\n        for (int64_t j = 0; j < len; ++j) {",
     "        double total = 0.5;\n        for (int64_t j = 0; j < len; ++j) {", 1, SOFTMAX),
    ("softmax: row stride off by one", "const double* xr = x + r * len;", "const double* xr = x + r * (len - 1);", 1,
     SOFTMAX),
    ("causal: diagonal masked", "(j <= last)", "(j < last)", 2, CAUSAL),
    ("causal: mask not aligned to the key end", "const int64_t last = i + (k - q);", "const int64_t last = i;", 1,
     CAUSAL),
    ("causal: scale dropped", "scale * xr[j]", "xr[j]", 2, CAUSAL),
    ("group_norm: unbiased variance", "const double var = sq / (double)count;",
     "const double var = sq / (double)(count - 1);", 1, GN),
    ("group_norm: eps outside the root", "1.0 / sqrt(var + eps)", "1.0 / (sqrt(var) + eps)", 1, GN),
    ("group_norm: weight and bias transposed", "(xg[at] - mu) * inv_std * wc + bc", "(xg[at] - mu) * inv_std * bc + wc",
     1, GN),
    ("group_norm: channel index", "const int64_t ch = g * ch_per_group + k;", "const int64_t ch = g + k * groups;", 1,
     GN),
    ("layer_norm: unbiased variance", "sqrt(sq / (double)d + eps)", "sqrt(sq / (double)(d - 1) + eps)", 1, LN),
    ("layer_norm: weight and bias transposed", "(w ? w[j] : 1.0) + (b ? b[j] : 0.0)",
     "(b ? b[j] : 1.0) + (w ? w[j] : 0.0)", 1, LN),
    ("avgpool: window end rounded down", "const int64_t h1 = ((i + 1) * h + oh - 1) / oh;",
     "const int64_t h1 = ((i + 1) * h) / oh + ((i + 1) * h < oh);", 1, AP),
    ("avgpool: column start from the height", "const int64_t w0 = (j * w) / ow;",
     "const int64_t w0 = (j * h) / ow < w ? (j * h) / ow : w - 1;", 1, AP),
    ("avgpool: count off by one", "/ (double)((h1 - h0) * (w1 - w0))", "/ (double)((h1 - h0) * (w1 - w0) + 1)", 1, AP),
    ("max_pool: last position wins a tie", "if (v > best || isnan(v))", "if (v >= best || isnan(v))", 1, MP),
    ("max_pool: padding left out of the row", "const int64_t r = i * sh - ph + a * dh;",
     "const int64_t r = i * sh + a * dh;", 1, MP),
    ("rounding: ties away from zero", "const double units = rint(a / quantum);",
     "const double units = floor(a / quantum + 0.5);", 1, ROUND),
    ("rounding: through float first", "const double units = rint(a / quantum);",
     "const double units = rint((double)(float)a / quantum);", 1, ROUND),
]


def run_pins(tmp_path, source: str, pin_file: str) -> subprocess.CompletedProcess:
    d = tmp_path / "oracle_copy"
    d.mkdir(exist_ok=True)
    (d / "oracle.c").write_text(source)
    env = dict(os.environ, KF_ORACLE_SRC=str(d / "oracle.c"))
    return subprocess.run([sys.executable, "-m", "pytest", pin_file, "-x", "-q", "-m", "not gpu",
                           "-p", "no:cacheprovider"], cwd=ROOT, env=env, capture_output=True, text=True,
                          timeout=600)


def test_unmutated_copy_passes(tmp_path):
    r = run_pins(tmp_path, open(SRC).read(), SOFTMAX)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-2000:]


@pytest.mark.parametrize("name,old,new,times,pin_file", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_mistake_fails_a_pin(tmp_path, name, old, new, times, pin_file):
    source = open(SRC).read()
    assert source.count(old) == times, f"{name}: the text to mutate occurs {source.count(old)} times"
    mutated = source.replace(old, new)
    r = run_pins(tmp_path, mutated, pin_file)
    # 1: tests ran and at least one failed (not a collection or build error).
    assert r.returncode == 1, f"{name}: pins returned {r.returncode}\n" + r.stdout[-2000:] + r.stderr[-2000:]
    assert " failed" in r.stdout, r.stdout[-2000:]
