"""The oracle under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

The C oracle is rebuilt in a temp directory with -fsanitize=address,undefined
(no recovery: the first report aborts) and the whole pin suite runs against
it in a subprocess with the ASan runtime preloaded (the interpreter itself is
not instrumented).  A second case plants an out-of-bounds read into a copy of
the oracle and checks that the sanitized run reports it, so the harness is
known to be live.  The real oracle is never modified.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "qmlp_oracle.c")


def _runtime(name):
    r = subprocess.run(["gcc", "-print-file-name=" + name], capture_output=True, text=True)
    path = r.stdout.strip()
    return path if r.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


ASAN = _runtime("libasan.so")
pytestmark = pytest.mark.skipif(ASAN is None or shutil.which("gcc") is None,
                                reason="gcc's ASan runtime is not installed")


def _build(src_text, tmp_path):
    src = tmp_path / "oracle_san.c"
    src.write_text(src_text)
    lib = tmp_path / "liboracle_san.so"
    subprocess.run(["gcc", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    "-fno-omit-frame-pointer", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
                    "-o", str(lib), str(src), "-lm"], check=True)
    return lib


def _run_pins(lib):
    env = dict(os.environ, LD_PRELOAD=ASAN, QMLP_ORACLE_LIB=str(lib),
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    # -s: a sanitizer report goes to stderr as the process stops, past any capture
    return subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-s", "-p", "no:cacheprovider",
                           os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                          env=env, cwd=ROOT, capture_output=True, text=True, timeout=600)


def test_oracle_pins_clean_under_asan_and_ubsan(tmp_path):
    r = _run_pins(_build(open(SRC).read(), tmp_path))
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-3000:]
    assert r.returncode == 0, out[-3000:]


def test_sanitizer_reports_a_planted_out_of_bounds_read(tmp_path):
    src = open(SRC).read()
    old = "            for (long i = 0; i < d; ++i)\n                acc += act_to_f64(A[c * d + i], bf16)"
    assert src.count(old) == 1, "planting site moved"
    lib = _build(src.replace(old, old.replace("i < d", "i <= d")), tmp_path)
    r = _run_pins(lib)
    assert r.returncode != 0
    assert "AddressSanitizer" in r.stdout + r.stderr
