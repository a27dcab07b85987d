"""Plant plausible mistakes in the oracle -- its C source, and the acceptance
rule in its Python module -- and check that the pin suites reject every one.

Each C mutant is built on the CPU and runs in a child process (a broken index
may read out of bounds).  Each Python mutant is the module's source with one
change, loaded under another name."""
import importlib.util
import json
import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# (name, text in oracle_conv.c, replacement)
MUTANTS = [
    ("filter_flip", "* K + kh) * K + kw]", "* K + (K - 1 - kh)) * K + (K - 1 - kw)]"),
    ("taps_transposed", "* K + kh) * K + kw]", "* K + kw) * K + kh]"),
    ("co_ci_swapped", "(((size_t)co * C_in + ci)", "(((size_t)ci * C_in + co)"),
    ("bias_dropped", "double acc = b ? (double)b[co] : 0.0;", "double acc = 0.0;"),
    ("pad_off_by_one", "long ih = (long)oh * stride - pad + kh;",
     "long ih = (long)oh * stride - pad + kh + 1;"),
    ("stride_ignored_w", "long iw = (long)ow * stride - pad + kw;", "long iw = (long)ow - pad + kw;"),
    ("pad_missing_left_w", "long iw = (long)ow * stride - pad + kw;", "long iw = (long)ow * stride + kw;"),
    ("sumabs_signed", "s += fabs(t);", "s += t;"),
    ("sumabs_with_bias", "double s = 0.0;", "double s = b ? fabs((double)b[co]) : 0.0;"),
    ("last_channel_dropped", "for (int ci = 0; ci < C_in; ++ci)", "for (int ci = 0; ci + 1 < C_in; ++ci)"),
    ("image_transposed", "((size_t)ci * H + ih) * W + iw", "((size_t)ci * W + iw) * H + ih"),
    ("out_size_ceil", "return (int)(span / stride) + 1;", "return (int)((span + stride - 1) / stride) + 1;"),
    ("float_accumulator", "double acc = b ?", "float acc = b ?"),
    ("last_tap_row_dropped", "for (int kh = 0; kh < K; ++kh)", "for (int kh = 0; kh + (K > 1) < K; ++kh)"),
    ("relu_inverted", "y[i] = x[i] > 0.0f ? x[i] : 0.0f;", "y[i] = x[i] < 0.0f ? x[i] : 0.0f;"),
    ("maxpool_min", "if (v > m)", "if (v < m)"),
    ("points_off_by_one", "rem / Wo, rem % Wo, &v, &s);", "rem / Wo, (rem + 1) % Wo, &v, &s);"),
]

_RUNNER = r"""
import json, sys
sys.path[:0] = [{root!r}, {tests!r}]
import oracle
from oracle_pins import ALL_PINS
lib = oracle.load({lib!r})
failed = []
for pin in ALL_PINS:
    try:
        pin(lib)
    except Exception as e:
        failed.append(pin.__name__)
print(json.dumps(failed))
"""


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, name, old, new):
    src = open(oracle.SOURCE).read()
    assert src.count(old) >= 1, f"mutation site for {name} not found"
    mutant_src = tmp_path / f"oracle_{name}.c"
    mutant_src.write_text(src.replace(old, new))
    lib = str(tmp_path / f"liboracle_{name}.so")
    oracle.compile_oracle(str(mutant_src), lib)
    code = _RUNNER.format(root=ROOT, tests=os.path.join(ROOT, "tests"), lib=lib)
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    if r.returncode != 0:
        return  # the mutant crashed the pin run: caught
    failed = json.loads(r.stdout.strip().splitlines()[-1])
    assert failed, f"mutant {name} passed every pin"


# (name, text in oracle/__init__.py, replacement): mistakes in the acceptance
# rule that every parity verdict goes through.
PY_SOURCE = os.path.join(ROOT, "oracle", "__init__.py")
PY_MUTANTS = [
    ("divisor_c_in_only", "float(c_in * k * k)", "float(c_in)"),
    ("divisor_k_squared_only", "float(c_in * k * k)", "float(k * k)"),
    ("absolute_floor_dropped", "1e-4 * (1.0 + np.asarray(sumabs, dtype=np.float64) / float(c_in * k * k))",
     "1e-4 * (np.asarray(sumabs, dtype=np.float64) / float(c_in * k * k))"),
    ("scale_1e-3", "return 1e-4 * (1.0 +", "return 1e-3 * (1.0 +"),
    ("sumabs_ignored", "np.asarray(sumabs, dtype=np.float64) / float", "0.0 * np.asarray(sumabs, dtype=np.float64) / float"),
    ("comparison_inverted", "ratio[i] <= 1.0", "ratio[i] >= 1.0"),
    ("comparison_strict", "ratio[i] <= 1.0", "ratio[i] < 1.0"),
    ("abs_dropped", "ratio = np.abs(r - ref) / tol", "ratio = (r - ref) / tol"),
    ("non_finite_accepted", "return False, float(\"inf\"), i", "return True, float(\"inf\"), i"),
    ("non_finite_guard_dropped", "if bad.any():", "if False:"),
    ("worst_is_best", "i = int(np.argmax(ratio))", "i = int(np.argmin(ratio))"),
    ("shape_check_dropped", "if r.shape != ref.shape:", "if False:"),
]


@pytest.mark.parametrize("name,old,new", PY_MUTANTS, ids=[m[0] for m in PY_MUTANTS])
def test_acceptance_mutant_is_caught(tmp_path, name, old, new):
    from acceptance_pins import ALL_ACCEPTANCE_PINS
    src = open(PY_SOURCE).read()
    assert src.count(old) == 1, f"mutation site for {name} not found exactly once"
    path = tmp_path / f"oracle_{name}.py"
    path.write_text(src.replace(old, new))
    spec = importlib.util.spec_from_file_location(f"oracle_mutant_{name}", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    failed = []
    for pin in ALL_ACCEPTANCE_PINS:
        try:
            pin(mod)
        except Exception:
            failed.append(pin.__name__)
    assert failed, f"acceptance-rule mutant {name} passed every pin"
