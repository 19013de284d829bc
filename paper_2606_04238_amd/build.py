"""Build ``libqmlp.so`` (the HIP library behind ``include/qmlp.h``) for gfx950.

Each ``csrc/*.hip`` is compiled to an object in parallel with hipcc, then
linked into a shared library next to this file.  Packed-fp32 VALU forms are
disabled (``-packed-fp32-ops``); the compiler still emits ordinary fp32 and
the packed fp16 / dot2 instructions the kernels ask for.

``--host-sanitize`` builds ``_build_san/libqmlp_san.so`` instead: the host
code (argument validation, sizes, dispatch) under AddressSanitizer and
UndefinedBehaviorSanitizer, the device code as usual.  Run the CPU ABI tests
against it with clang's ASan runtime preloaded:
    QMLP_LIB_PATH=paper_2606_04238_amd/_build_san/libqmlp_san.so \
    LD_PRELOAD=$(ls /opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so) \
    ASAN_OPTIONS=detect_leaks=0 UBSAN_OPTIONS=halt_on_error=1 \
    python -m pytest -s tests/test_abi.py tests/test_bench_cli.py
"""
import concurrent.futures
import glob
import os
import subprocess
import sys

_HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(_HERE, "csrc")
BUILD = os.path.join(_HERE, "_build")
LIB = os.path.join(_HERE, "libqmlp.so")
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

COMMON = ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Wall", "-Wno-unused-result", "-I", os.path.join(_HERE, "..", "include")]


# host-only sanitizers (each -fsanitize= right after -Xarch_host: the device
# code is built as usual)
SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer", "-g"]


def _compile(src: str, build_dir: str = BUILD, extra=()) -> str:
    obj = os.path.join(build_dir, os.path.basename(src) + ".o")
    cmd = [HIPCC] + COMMON + list(extra) + ["-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed on %s:\n%s" % (src, r.stderr[-8000:]))
    return obj


def build(jobs: int = 8, host_sanitize: bool = False) -> str:
    build_dir = os.path.join(_HERE, "_build_san") if host_sanitize else BUILD
    lib = os.path.join(build_dir, "libqmlp_san.so") if host_sanitize else LIB
    extra = SANITIZE if host_sanitize else []
    os.makedirs(build_dir, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(jobs, len(srcs))) as ex:
        objs = list(ex.map(lambda s: _compile(s, build_dir, extra), srcs))
    tmp = lib + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC"] + extra + ["-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s" % r.stderr[-8000:])
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    print(build(host_sanitize="--host-sanitize" in sys.argv[1:]), file=sys.stderr)
