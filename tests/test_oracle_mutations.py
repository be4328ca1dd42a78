"""The oracle's pins must catch plausible mistakes in the oracle itself.

Each case plants one mistake in a copy of the oracle (the copy only, never
the files) and runs the oracle's pin tests against it in a subprocess; at
least one pin must fail. The C half is compiled on the CPU from a mutated
copy of its source (SEEDQ_ORACLE_LIB points the loader at it); the Python
parts (schedule, code stream, importance) run from a copied package with
one mutated module. A control run of each unmodified copy must pass, so that
a failure is the planted mistake's and not the harness's.
"""
import os
import shutil
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


# ---------------------------------------------------------------- Python parts
# (module in oracle/, its pin file, name, text, replacement)
PY_MUTATIONS = [
    ("allocation.py", "test_oracle_schedule.py", "floor as a ceiling",
     "imp = np.maximum(imp, q)", "imp = np.minimum(imp, q)"),
    ("allocation.py", "test_oracle_schedule.py", "ties demoted from the end",
     "tied = np.nonzero(j_lo != j_hi)[0]         # ascending block index",
     "tied = np.nonzero(j_lo != j_hi)[0][::-1]"),
    ("allocation.py", "test_oracle_schedule.py", "rate without the exponent bits",
     "return K + 4 * P + 4", "return K + 4 * P"),
    ("allocation.py", "test_oracle_schedule.py", "collinear hull points kept",
     "if cross <= 0:", "if cross < 0:"),
    ("stream.py", "test_oracle_stream.py", "exponent before seed",
     "        bits += _field(int(seed[b]), K)\n        bits += _field(int(exp[b]), 4)\n",
     "        bits += _field(int(exp[b]), 4)\n        bits += _field(int(seed[b]), K)\n"),
    ("stream.py", "test_oracle_stream.py", "fields most significant bit first",
     "return [(value >> i) & 1 for i in range(width)]",
     "return [(value >> (width - 1 - i)) & 1 for i in range(width)]"),
    ("stream.py", "test_oracle_stream.py", "mantissa -8 read as +8",
     "q[b, j] = v - 16 if v >= 8 else v", "q[b, j] = v - 16 if v > 8 else v"),
    ("importance.py", "test_oracle_importance.py", "E[silu] instead of E[silu^2]",
     "(w * silu(g) ** 2)", "(w * silu(g))"),
    ("importance.py", "test_oracle_importance.py", "Gauss-Hermite nodes not scaled by sqrt(2)",
     "g = np.sqrt(2.0 * var)[..., None] * x", "g = np.sqrt(var)[..., None] * x"),
    ("importance.py", "test_oracle_importance.py", "repeat_kv channel by channel",
     "np.repeat(v.reshape(n_kv_heads, hd), n_heads // n_kv_heads, axis=0)",
     "np.repeat(v.reshape(n_kv_heads, hd), n_heads // n_kv_heads, axis=1)"),
]
PY_PINS = sorted({m[1] for m in PY_MUTATIONS})


def _run_py_pins(tmp_path, module, text, pins):
    # a copy of the package layout the pins import from, with one oracle
    # module replaced; the C half is the repository's own build
    shutil.copytree(os.path.join(ROOT, "oracle"), tmp_path / "oracle",
                    ignore=shutil.ignore_patterns("*.so", "__pycache__"))
    if module is not None:
        (tmp_path / "oracle" / module).write_text(text)
    shutil.copy(os.path.join(ROOT, "synthetic.py"), tmp_path / "synthetic.py")
    shutil.copytree(os.path.join(ROOT, "tests", "golden"), tmp_path / "tests" / "golden")
    for name in ["conftest.py", *pins]:
        shutil.copy(os.path.join(ROOT, "tests", name), tmp_path / "tests" / name)
    env = dict(os.environ, SEEDQ_ORACLE_LIB=os.path.join(ROOT, "oracle", "liboq.so"))
    return subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                           "-m", "not gpu", *["tests/" + p for p in pins]], cwd=tmp_path,
                          env=env, capture_output=True, text=True, timeout=600)


def test_python_pins_pass_on_an_unmodified_copy(tmp_path, oq):
    r = _run_py_pins(tmp_path, None, None, PY_PINS)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-2000:]


@pytest.mark.parametrize("module,pins,name,old,new", PY_MUTATIONS, ids=[m[2] for m in PY_MUTATIONS])
def test_python_pins_catch_planted_mistake(tmp_path, oq, module, pins, name, old, new):
    with open(os.path.join(ROOT, "oracle", module)) as f:
        text = f.read()
    assert old in text, f"{name}: the text to mutate is not in oracle/{module}"
    r = _run_py_pins(tmp_path, module, text.replace(old, new), [pins])
    assert r.returncode == 1, f"{name}: no pin failed\n" + r.stdout[-2000:] + r.stderr[-2000:]
