"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(no GPU).

dspark_api.hip -- argument validation, workspace sizing and dispatch -- is
compiled with the sanitizers on its host pass only (each -fsanitize= behind
-Xarch_host; device code is built as usual) and linked with the library's
other objects.  tests/test_abi.py then runs on that copy (loaded through
DSPARK_LIB) with the sanitizer runtime preloaded: every validation path it
drives must be free of memory errors and undefined behaviour.
"""
import glob
import os
import subprocess
import sys

import pytest

from paper_2607_05147_amd import build

HERE = os.path.dirname(os.path.abspath(__file__))
REPO = os.path.dirname(HERE)


def test_abi_validation_is_clean_under_host_sanitizers(tmp_path):
    rts = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not rts:
        pytest.skip("clang's AddressSanitizer runtime is not installed")
    objs = [os.path.join(build.OBJDIR, os.path.basename(s) + ".o") for s in build.sources()]
    if not all(os.path.exists(o) for o in objs):
        build.build()
    api_src = os.path.join(build.CSRC, "dspark_api.hip")
    api_obj = str(tmp_path / "dspark_api_san.o")
    lib = str(tmp_path / "libdspark_san.so")
    flags = [f for f in build.FLAGS if f != "-O3"] + ["-O1", "-g"]
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-omit-frame-pointer"]
    subprocess.run([build.HIPCC] + flags + san + ["-c", api_src, "-o", api_obj], check=True,
                   capture_output=True)
    others = [o for o in objs if not o.endswith("dspark_api.hip.o")]
    subprocess.run([build.HIPCC, f"--offload-arch={build.ARCH}", "-shared", "-fPIC",
                    "-shared-libsan"] + san[:4] + ["-o", lib, api_obj] + others, check=True,
                   capture_output=True)
    logs = str(tmp_path / "san")  # reports go to files: pytest captures stderr
    env = dict(os.environ, DSPARK_LIB=lib, LD_PRELOAD=rts[-1],
               ASAN_OPTIONS=f"detect_leaks=0:abort_on_error=1:log_path={logs}",
               UBSAN_OPTIONS=f"print_stacktrace=1:halt_on_error=1:log_path={logs}")
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(HERE, "test_abi.py"), "-x",
                        "-q", "-m", "not gpu", "-p", "no:cacheprovider", "-p", "no:xdist"],
                       cwd=REPO, env=env, capture_output=True, text=True, timeout=600)
    reports = "".join(open(os.path.join(tmp_path, f)).read() for f in sorted(os.listdir(tmp_path))
                      if f.startswith("san"))
    assert not reports, reports[-4000:]
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
