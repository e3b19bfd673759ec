"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (no GPU):
the planner of libpgf (pgf_plan.cpp, plain C++) driven over a grid of valid
and invalid arguments by tests/sanitize/plan_driver.cpp, and the C core of
the oracle (pgf_oracle.c) running its pin suite from a Python process that
preloads the ASan runtime."""
import os
import shutil
import subprocess
import sys

import pytest

from oracle import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g"]


def _runtime(name):
    path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


pytestmark = pytest.mark.skipif(shutil.which("g++") is None or _runtime("libasan.so") is None,
                                reason="no g++ with the sanitizer runtimes")


def test_planner_under_sanitizers(tmp_path):
    exe = str(tmp_path / "plan_driver")
    subprocess.run(["g++", "-std=c++17", "-O1", *SAN, "-o", exe,
                    os.path.join(ROOT, "tests", "sanitize", "plan_driver.cpp"),
                    os.path.join(ROOT, "paper_2512_23068_amd", "csrc", "pgf_plan.cpp")], check=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    print(r.stdout, r.stderr)
    assert r.returncode == 0, r.stderr
    assert "0 failures" in r.stdout and "ERROR" not in r.stderr and "runtime error" not in r.stderr


def test_oracle_pins_under_sanitizers(tmp_path):
    lib = str(tmp_path / "liboracle_san.so")
    oracle.build(out=lib, extra=tuple(SAN))
    env = dict(os.environ, PGF_ORACLE_LIB=lib, LD_PRELOAD=_runtime("libasan.so"),
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1",
               PGF_ORACLE_THREADS="4")
    probe = subprocess.run([sys.executable, "-c", "from oracle import oracle; oracle._load(); print(oracle._LIB_PATH)"],
                           cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert probe.stdout.strip().endswith("liboracle_san.so"), probe.stdout + probe.stderr
    pins = sorted(f for f in os.listdir(os.path.join(ROOT, "tests"))
                  if f.startswith("test_oracle") and f.endswith("_pins.py"))
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        *[os.path.join("tests", f) for f in pins]],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=1200)
    tail = "\n".join((r.stdout + r.stderr).splitlines()[-15:])
    print(tail)
    assert r.returncode == 0, tail
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, tail
