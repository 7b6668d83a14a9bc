"""The oracle under AddressSanitizer and UndefinedBehaviorSanitizer (no GPU).

oracle.c is compiled with -fsanitize=address,undefined (gcc, host code only)
and every pin module runs on that copy in a subprocess that loads it through
ORACLE_LIB, with the ASan runtime preloaded into the interpreter.  Any
out-of-bounds access, use after free or undefined operation in the oracle
aborts the run; the pins must still pass.
"""
import os
import subprocess
import sys

import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))
REPO = os.path.dirname(HERE)
PINS = [os.path.join(HERE, f"test_oracle_{m}.py")
        for m in ("schedule", "attention", "accept", "draft", "rnn")]


def _runtime(name):
    path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True,
                          text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def test_pins_pass_on_the_sanitized_oracle(tmp_path):
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    lib = str(tmp_path / "liboracle_san.so")
    subprocess.check_call([
        "gcc", "-O1", "-g", "-std=c11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
        "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
        "-fno-sanitize-recover=undefined", "-shared", "-fPIC", oracle._SRC, "-o", lib, "-lm"])
    logs = str(tmp_path / "san")  # reports go to files: pytest captures stderr
    env = dict(os.environ, ORACLE_LIB=lib, OMP_NUM_THREADS="4", LD_PRELOAD=asan,
               ASAN_OPTIONS=f"detect_leaks=0:abort_on_error=1:log_path={logs}",
               UBSAN_OPTIONS=f"print_stacktrace=1:halt_on_error=1:log_path={logs}")
    r = subprocess.run([sys.executable, "-m", "pytest", *PINS, "-x", "-q", "-m", "not gpu",
                        "-p", "no:cacheprovider", "-p", "no:xdist"],
                       cwd=REPO, env=env, capture_output=True, text=True, timeout=900)
    reports = "".join(open(os.path.join(tmp_path, f)).read() for f in sorted(os.listdir(tmp_path))
                      if f.startswith("san"))
    assert not reports, reports[-4000:]
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
