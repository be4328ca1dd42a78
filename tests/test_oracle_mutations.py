"""The oracle's pins must catch plausible mistakes in the oracle itself.

Each case plants one mistake in a copy of the oracle's C source (the copy
only, never the file), compiles it on the CPU, and runs the oracle's pin
tests against it in a subprocess (SEEDQ_ORACLE_LIB points the loader at the
copy); at least one pin must fail. A control run of the unmodified copy must
pass, so that a failure is the planted mistake's and not the harness's.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "seedq_oracle.c")
PINS = ["tests/test_oracle_lfsr.py", "tests/test_oracle_ls_quant.py",
        "tests/test_oracle_search.py", "tests/test_oracle_stream.py"]

# (name, text in the source, replacement): one plausible mistake each
MUTATIONS = [
    ("lfsr tap bit", "if (x & 1u) return (x >> 1) ^ mask;", "if (x & 2u) return (x >> 1) ^ mask;"),
    ("centring off by one bit", "int32_t half = (int32_t)1 << (K - 1);",
     "int32_t half = (int32_t)1 << K;"),
    ("rounding half away from zero", "nearbyint(", "round("),
    ("mantissa range [-7, 7]", "if (r > 7.0 || r < -8.0) fits = 0;",
     "if (r > 7.0 || r < -7.0) fits = 0;"),
    ("clamp at -7", "if (r < -8.0) r = -8.0;", "if (r < -7.0) r = -7.0;"),
    ("error drops the last weight", "  for (int i = 0; i < OQ_C; i++) {\n    int64_t acc = 0;",
     "  for (int i = 0; i < OQ_C - 1; i++) {\n    int64_t acc = 0;"),
    ("reconstruction scale 2^-(K+e)", "double w_hat = ldexp((double)acc, -(K - 1 + e));",
     "double w_hat = ldexp((double)acc, -(K + e));"),
    ("ties to the larger seed", "if (err < best) {", "if (err <= best) {"),
    ("exponent searched from the coarse end", "for (e = 15; e >= 0; e--) {",
     "for (e = 0; e <= 15; e++) {"),
]


def _build(tmp_path, text):
    src = tmp_path / "oracle_copy.c"
    src.write_text(text)
    lib = tmp_path / "liboq_copy.so"
    subprocess.run(["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-shared",
                    "-fPIC", str(src), "-o", str(lib), "-lm"], check=True)
    return str(lib)


def _run_pins(lib):
    env = dict(os.environ, SEEDQ_ORACLE_LIB=lib)
    return subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                           "-m", "not gpu", *PINS], cwd=ROOT, env=env, capture_output=True,
                          text=True, timeout=600)


def test_pins_pass_on_an_unmodified_copy(tmp_path):
    with open(SRC) as f:
        lib = _build(tmp_path, f.read())
    r = _run_pins(lib)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-2000:]


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_pins_catch_planted_mistake(tmp_path, name, old, new):
    with open(SRC) as f:
        text = f.read()
    assert old in text, f"{name}: the text to mutate is not in the oracle"
    lib = _build(tmp_path, text.replace(old, new))
    r = _run_pins(lib)
    assert r.returncode == 1, f"{name}: no pin failed\n" + r.stdout[-2000:] + r.stderr[-2000:]
