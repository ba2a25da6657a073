"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

- The library's host side (argument checks and workspace layouts, csrc/sv_host.cpp) is
  built with g++ on its own and driven over edge and seeded random descriptors
  (tests/sanitize/host_checks_driver.cpp).
- The oracle (oracle/oracle.c) is built as a sanitized shared library and the oracle's
  own test files run against it, with the sanitizer runtime preloaded into Python.
Both builds stop at the first report (-fno-sanitize-recover=all). A third test plants an
out-of-bounds read and a signed overflow in a scratch program built the same way, to
show that these flags do catch them.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]
ENV_SAN = {"ASAN_OPTIONS": "detect_leaks=0:abort_on_error=0:exitcode=23",
           "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1:exitcode=24"}


def _have(tool):
    return shutil.which(tool) is not None


pytestmark = pytest.mark.skipif(not (_have("gcc") and _have("g++")), reason="gcc/g++ not found")


def _run(cmd, env=None, timeout=600):
    e = dict(os.environ)
    e.update(ENV_SAN)
    if env:
        e.update(env)
    return subprocess.run(cmd, capture_output=True, text=True, env=e, timeout=timeout)


def test_sanitizers_catch_planted_errors(tmp_path):
    src = tmp_path / "planted.c"
    src.write_text(
        "#include <stdlib.h>\n#include <limits.h>\n"
        "int main(int argc, char** argv) {\n"
        "  int* a = malloc(4 * sizeof(int));\n"
        "  volatile int big = INT_MAX;\n"
        "  if (argc > 1) { int x = big + argc; return x == 7; }  /* signed overflow */\n"
        "  int v = a[argc + 3];  /* one past the end */\n"
        "  free(a); return v == 12345;\n}\n")
    exe = tmp_path / "planted"
    subprocess.run(["gcc", *SAN, str(src), "-o", str(exe)], check=True)
    r = _run([str(exe)])  # reported by AddressSanitizer or by UBSan's object-size check
    assert r.returncode != 0 and ("heap-buffer-overflow" in r.stderr or "insufficient space" in r.stderr), \
        r.stderr[-2000:]
    r = _run([str(exe), "x", "y"])
    assert r.returncode != 0 and "signed integer overflow" in r.stderr, r.stderr[-2000:]


def test_host_checks_and_layouts_under_sanitizers(tmp_path):
    exe = tmp_path / "host_driver"
    csrc = os.path.join(ROOT, "paper_2607_25852_amd", "csrc")
    subprocess.run(["g++", "-std=c++17", "-Wall", "-Wextra", "-Werror", *SAN, "-I", os.path.join(ROOT, "include"),
                    "-I", csrc, os.path.join(ROOT, "tests", "sanitize", "host_checks_driver.cpp"),
                    os.path.join(csrc, "sv_host.cpp"), "-o", str(exe)], check=True)
    r = _run([str(exe)])
    assert r.returncode == 0, r.stdout[-1000:] + r.stderr[-4000:]
    assert r.stdout.startswith("ok:"), r.stdout
    accepted = int(r.stdout.split()[1])
    assert accepted > 1000, r.stdout  # the layouts of many accepted shapes were checked


def test_oracle_under_sanitizers(tmp_path):
    lib = tmp_path / "liboracle_san.so"
    subprocess.run(["gcc", "-std=gnu11", "-fno-fast-math", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
                    "-Wall", "-Wextra", *SAN, "-o", str(lib), os.path.join(ROOT, "oracle", "oracle.c"), "-lm"],
                   check=True)
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    assert os.path.isabs(asan), "the AddressSanitizer runtime is not installed"
    tests = [os.path.join(ROOT, "tests", f) for f in sorted(os.listdir(os.path.join(ROOT, "tests")))
             if f.startswith("test_oracle_") and f.endswith(".py")]
    env = {"LD_PRELOAD": asan, "SV_ORACLE_LIB": str(lib), "OMP_NUM_THREADS": "4"}
    # the run loads the sanitized build (not the regular liboracle.so) ...
    probe = _run([sys.executable, "-c", "import oracle; oracle._load(); print(oracle._LIB_PATH)"],
                 env=dict(env, PYTHONPATH=ROOT))
    assert probe.returncode == 0 and probe.stdout.strip() == str(lib), probe.stdout + probe.stderr[-2000:]
    # ... and every oracle test passes under it
    r = _run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", *tests],
             env=dict(env, PYTHONPATH=ROOT))
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert " passed" in r.stdout
