"""The oracle's pins must catch plausible mistakes.

Each case plants one mistake into a copy of the oracle (built in a temp
directory, on the CPU), then runs the pin suite against that copy and
expects at least one pin to fail.  The real oracle is never modified.
Mistakes in the C arithmetic are planted in a copy of the C source; mistakes
in the Python-side composition (the routed-expert sum) in a copy of the
oracle package, run from a copy of the pin suite.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "qmlp_oracle.c")
PYSRC = os.path.join(ROOT, "oracle", "__init__.py")

MUTANTS = {
    "round_half_away_from_zero": ("double t = rint((double)w[i] / sd) + (double)z;",
                                  "double t = round((double)w[i] / sd) + (double)z;"),
    "zero_added_before_rounding": ("double t = rint((double)w[i] / sd) + (double)z;",
                                   "double t = rint((double)w[i] / sd + (double)z);"),
    "dropped_zero_point": ("w[row * k + i] = s * ((double)codes[row * k + i] - z);",
                           "w[row * k + i] = s * ((double)codes[row * k + i]);"),
    "transposed_lora_B": ("lr += act_to_f64(Bm[o * rank + c], bf16) * t[m * rank + c];",
                          "lr += act_to_f64(Bm[c * nout + o], bf16) * t[m * rank + c];"),
    "sigmoid_sign": ("h[i] = a / (1.0 + exp(-a)) * uv[i];", "h[i] = a / (1.0 + exp(a)) * uv[i];"),
    "zero_point_sign": ("double zf = rint(-lo / sd);", "double zf = rint(lo / sd);"),
    "range_without_zero": ("double lo = 0.0, hi = 0.0;", "double lo = 1e30, hi = -1e30;"),
    "lora_scale_dropped": ("out[m * nout + o] = acc + lora_scale * lr;", "out[m * nout + o] = acc + lr;"),
    "wrong_group_index": ("double s = orc_f16_to_f64(scale[row * ng + i / g]);",
                          "double s = orc_f16_to_f64(scale[row * ng + i / (2 * g)]);"),
    "scale_via_binary32": ("uint16_t s16 = orc_f64_to_f16(s);",
                           "uint16_t s16 = orc_f64_to_f16((double)(float)s);"),
    "rmsnorm_sum_not_mean": ("double inv = 1.0 / sqrt(ss / (double)d + eps);",
                             "double inv = 1.0 / sqrt(ss + eps);"),
    "rmsnorm_eps_outside_root": ("double inv = 1.0 / sqrt(ss / (double)d + eps);",
                                 "double inv = 1.0 / (sqrt(ss / (double)d) + eps);"),
    "residual_sign": ("out[i] = orc_f64_to_f16(orc_f16_to_f64(x[i]) + orc_f16_to_f64(y[i]));",
                      "out[i] = orc_f64_to_f16(orc_f16_to_f64(x[i]) - orc_f16_to_f64(y[i]));"),
    "down_act_ignores_bf16": ("hd[i] = act_to_f64(h_bits[i], bf16);",
                              "hd[i] = act_to_f64(h_bits[i], 0);"),
    "lora_a_reads_bf16_as_f16": (
        "acc += act_to_f64(A[c * d + i], bf16) * act_to_f64(x[m * d + i], bf16);",
        "acc += act_to_f64(A[c * d + i], 0) * act_to_f64(x[m * d + i], 0);"),
}

PY_MUTANTS = {
    "moe_forward_drops_lora_scale": (
        "ym = ym + w * forward(qg, qu, qd, Ag, Bg, Au, Bu, x[m:m + 1], lora_scale=lora_scale)[0]",
        "ym = ym + w * forward(qg, qu, qd, Ag, Bg, Au, Bu, x[m:m + 1])[0]"),
}


def _run_pins(cwd, env):
    return subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                           os.path.join(cwd, "tests", "test_oracle_pins.py")],
                          env=env, cwd=cwd, capture_output=True, text=True, timeout=600)


def _build(src_text, tmp_path):
    mutant = tmp_path / "mutant.c"
    mutant.write_text(src_text)
    lib = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-O2", "-ffp-contract=off", "-fPIC", "-shared", "-o", str(lib),
                    str(mutant), "-lm"], check=True)
    return lib


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) >= 1, "mutation site moved: " + name
    lib = _build(src.replace(old, new), tmp_path)
    env = dict(os.environ, QMLP_ORACLE_LIB=str(lib))
    r = _run_pins(ROOT, env)
    assert r.returncode != 0, "no pin caught mutant %s:\n%s" % (name, r.stdout[-2000:])


@pytest.mark.parametrize("name", sorted(PY_MUTANTS))
def test_pins_catch_planted_python_mistake(name, tmp_path):
    old, new = PY_MUTANTS[name]
    src = open(PYSRC).read()
    assert src.count(old) == 1, "mutation site moved: " + name
    # a private tree: the mutated oracle package, the workload generator and
    # the pin suite; the C library is the real one, built from the real source
    tree = tmp_path / "tree"
    (tree / "oracle").mkdir(parents=True)
    (tree / "oracle" / "__init__.py").write_text(src.replace(old, new))
    shutil.copy(os.path.join(ROOT, "oracle", "build.py"), tree / "oracle" / "build.py")
    shutil.copy(SRC, tree / "oracle" / "qmlp_oracle.c")
    shutil.copytree(os.path.join(ROOT, "workloads"), tree / "workloads",
                    ignore=shutil.ignore_patterns("__pycache__"))
    (tree / "tests").mkdir()
    for fn in ("conftest.py", "test_oracle_pins.py"):
        shutil.copy(os.path.join(ROOT, "tests", fn), tree / "tests" / fn)
    shutil.copytree(os.path.join(ROOT, "tests", "golden"), tree / "tests" / "golden")
    lib = _build(open(SRC).read(), tmp_path)
    env = dict(os.environ, QMLP_ORACLE_LIB=str(lib))
    # the unmutated copy passes: the tree itself is sound
    if name == sorted(PY_MUTANTS)[0]:
        (tree / "oracle" / "__init__.py").write_text(src)
        ok = _run_pins(str(tree), env)
        assert ok.returncode == 0, ok.stdout[-2000:]
        (tree / "oracle" / "__init__.py").write_text(src.replace(old, new))
    r = _run_pins(str(tree), env)
    assert r.returncode != 0, "no pin caught mutant %s:\n%s" % (name, r.stdout[-2000:])
