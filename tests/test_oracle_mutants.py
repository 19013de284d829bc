"""The oracle's pins must catch plausible mistakes.

Each case plants one mistake into a copy of the C oracle (built in a temp
directory, on the CPU), then runs the pin suite against that copy and
expects at least one pin to fail.  The real oracle is never modified.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "qmlp_oracle.c")

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
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) >= 1, "mutation site moved: " + name
    mutant = tmp_path / "mutant.c"
    mutant.write_text(src.replace(old, new))
    lib = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-O2", "-ffp-contract=off", "-fPIC", "-shared", "-o", str(lib),
                    str(mutant), "-lm"], check=True)
    env = dict(os.environ, QMLP_ORACLE_LIB=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                       env=env, cwd=ROOT, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, "no pin caught mutant %s:\n%s" % (name, r.stdout[-2000:])
