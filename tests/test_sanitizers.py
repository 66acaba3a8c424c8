"""The host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

Builds, with clang's sanitizer runtime:
* the oracle's fixed-order C routines (oracle/pinned.c), and
* libincvit.so with the host side of the ABI (incvit_api.hip: config
  validation, layouts and size queries, the overlap and argument checks,
  handle creation) instrumented; the device code is built as usual, and no
  kernel runs here,
then runs the ABI tests and the oracle tests that call the C routines against
those builds in a child process with the runtime preloaded.  Any sanitizer
report aborts the child, which fails this test.
"""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LLVM = "/opt/rocm/llvm"
HIPCC = "/opt/rocm/bin/hipcc"

pytestmark = pytest.mark.slow


def _runtime():
    libs = glob.glob(os.path.join(LLVM, "lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return libs[0] if libs else None


@pytest.mark.skipif(_runtime() is None or not os.path.exists(HIPCC), reason="clang sanitizer runtime not installed")
def test_host_code_is_clean_under_asan_and_ubsan(tmp_path):
    from paper_2607_12287_amd import build as hip_build

    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
           "-shared-libsan", "-g", "-O1"]
    pinned = str(tmp_path / "_pinned_san.so")
    subprocess.check_call([os.path.join(LLVM, "bin/clang"), *san, "-mavx2", "-mfma", "-ffp-contract=off",
                           "-fPIC", "-shared", "-o", pinned, os.path.join(ROOT, "oracle", "pinned.c"), "-lm"])

    # every other object of the library as built (compiled here only if stale);
    # incvit_api.hip with its host pass instrumented (each sanitizer flag
    # applies to the host pass only)
    objs = hip_build.objects([s for s in hip_build.SOURCES if s != "incvit_api.hip"])
    host_san = []
    for f in san:
        host_san += ["-Xarch_host", f]
    api_obj = str(tmp_path / "incvit_api_san.o")
    subprocess.check_call([HIPCC, *hip_build.COMMON, *host_san, "-c",
                           os.path.join(hip_build.CSRC, "incvit_api.hip"), "-o", api_obj])
    lib = str(tmp_path / "libincvit_san.so")
    subprocess.check_call([HIPCC, "--offload-arch=" + hip_build.ARCH, "-shared", "-fPIC", "-shared-libsan",
                           "-fsanitize=address,undefined", api_obj, *objs, "-o", lib])

    env = dict(os.environ)
    env.update(LD_PRELOAD=_runtime(), INCVIT_LIB=lib, ORACLE_PINNED_LIB=pinned,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    tests = ["tests/test_abi.py", "tests/test_oracle_pins.py", "tests/test_oracle_key_score.py",
             "tests/test_oracle_edges.py"]
    res = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu and not slow",
                          "-p", "no:cacheprovider", *tests], cwd=ROOT, env=env, capture_output=True, text=True)
    out = res.stdout[-4000:] + res.stderr[-4000:]
    assert res.returncode == 0, out
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out
    print(res.stdout.strip().splitlines()[-1])
