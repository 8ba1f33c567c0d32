"""CPU runs under AddressSanitizer and UndefinedBehaviorSanitizer.

- The fp64 oracle (oracle/grpo_oracle.c), built with gcc -fsanitize=address,undefined, driven through every one of
  its functions and edge cases by tests/sanitize/oracle_calls.c.
- The host side of libgrpo (argument validation, workspace queries), its HIP sources compiled with the sanitizers on
  the host pass only, driven through every entry point with invalid arguments and every workspace query at extreme
  sizes by tests/sanitize/abi_args.c.  No GPU is involved: nothing gets past validation.

Any out-of-bounds access, use after free, leak (oracle), signed overflow, invalid enum load or similar aborts the
driver with a sanitizer report, and the test fails with it.
"""
import os
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")
CLANG = os.path.join(ROCM, "llvm", "bin", "clang")
# the sanitizers on the host pass only: device code is built as usual
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-Xarch_host",
            "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=all", "-g"]


def _run(cmd, env=None):
    r = subprocess.run(cmd, capture_output=True, text=True, env=env)
    assert r.returncode == 0, f"{' '.join(cmd[:3])} ...: rc {r.returncode}\n{r.stdout[-3000:]}\n{r.stderr[-6000:]}"
    return r


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_calls")
    _run(["gcc", "-std=c11", "-O1", "-g", "-fopenmp", "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
          "-fno-sanitize-recover=all", os.path.join(HERE, "oracle_calls.c"),
          os.path.join(ROOT, "oracle", "grpo_oracle.c"), "-lm", "-o", exe])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = _run([exe], env=env)
    assert "oracle calls ok" in r.stdout


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG)), reason="ROCm compilers not available")
def test_library_host_checks_under_asan_ubsan(tmp_path):
    csrc = os.path.join(ROOT, "paper_2606_05597_amd", "csrc")
    srcs = sorted(f for f in os.listdir(csrc) if f.endswith(".hip"))
    flags = ["--offload-arch=gfx950", "-O1", "-std=c++17", "-fPIC", "-Xclang", "-target-feature", "-Xclang",
             "-packed-fp32-ops", "-I" + os.path.join(ROOT, "include"), "-I" + csrc, *HOST_SAN]

    def obj(f):
        o = str(tmp_path / (f + ".o"))
        _run([HIPCC, *flags, "-c", os.path.join(csrc, f), "-o", o])
        return o

    with ThreadPoolExecutor(8) as ex:
        objs = list(ex.map(obj, srcs))
    lib = str(tmp_path / "libgrpo_san.so")
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *HOST_SAN, *objs, "-o", lib])
    exe = str(tmp_path / "abi_args")
    _run([CLANG, "-std=c11", "-O1", "-g", "-D__HIP_PLATFORM_AMD__", "-I" + os.path.join(ROOT, "include"),
          "-I" + os.path.join(ROCM, "include"), "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
          os.path.join(HERE, "abi_args.c"), lib, "-Wl,-rpath," + str(tmp_path), "-o", exe])
    # the HIP runtime the library loads is not instrumented and keeps allocations for the process lifetime:
    # leak checking is for the oracle, whose code is all ours
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = _run([exe], env=env)
    assert "abi argument checks ok" in r.stdout
