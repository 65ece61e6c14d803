"""The oracle under AddressSanitizer and UndefinedBehaviorSanitizer (no GPU):
oracle.c is built with -fsanitize=address,undefined (every report fatal) and
the pin suite runs against that build, so an out-of-bounds access, a signed
overflow, a shift past the width or any other undefined behaviour in the
oracle ends the run instead of going unseen.  The Python interpreter is not
instrumented, so the ASan runtime is preloaded into the child process."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.c")
FLAGS = ["-O1", "-g", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fno-math-errno",
         "-fexcess-precision=standard", "-fPIC", "-shared", "-fno-omit-frame-pointer",
         "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]


def _runtime(name):
    path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def test_pins_pass_against_the_sanitized_oracle(tmp_path):
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    lib = tmp_path / "liboracle_san.so"
    subprocess.run(["gcc", *FLAGS, "-I", os.path.join(ROOT, "oracle"), "-o", str(lib), SRC, "-lm"], check=True)
    env = dict(os.environ, PACT_ORACLE_LIB=str(lib), LD_PRELOAD=asan,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    # the torch comparisons load a large uninstrumented library and add
    # nothing to what the sanitizers check in oracle.c
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        f"--basetemp={tmp_path / 'pins'}", "-k", "not torch", "tests/test_oracle_pins.py"],
                       cwd=ROOT, env=env, capture_output=True, text=True)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-3000:])
    assert "passed" in r.stdout
