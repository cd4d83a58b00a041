"""AddressSanitizer and UndefinedBehaviorSanitizer builds of the host code,
run on the CPU: the oracle (every entry point on small random inputs) and
the library's C-ABI validation and workspace planning (capi.hip; the kernels
are linked but never launched).  Each driver exits non-zero on an
unexpected status, and a sanitizer finding aborts it."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
HIPCC = "/opt/rocm/bin/hipcc"
ENV = dict(os.environ, UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")


def run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout}\n{r.stderr}"
    return r


@pytest.mark.skipif(shutil.which("gcc") is None, reason="no gcc")
def test_oracle_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    run(["gcc", "-std=c11", "-g", "-O1", "-fno-omit-frame-pointer",
         "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-ffp-contract=off",
         "-I", os.path.join(ROOT, "oracle"), os.path.join(HERE, "oracle_driver.c"),
         os.path.join(ROOT, "oracle", "smallkv_oracle.c"),
         os.path.join(ROOT, "oracle", "match_oracle.c"), "-lm", "-o", exe])
    r = run([exe], env=dict(ENV, ASAN_OPTIONS="detect_leaks=1"))
    assert "oracle driver ok" in r.stdout


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="no hipcc")
def test_library_host_checks_under_asan_and_ubsan(tmp_path):
    from paper_2508_02751_amd import build as B
    others = [os.path.join(B.BUILD, os.path.splitext(s)[0] + ".o") for s in B.SOURCES
              if s != "capi.hip"]
    if not all(os.path.exists(o) for o in others):
        B.build()  # the regular objects of the kernels' sources
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined"]
    capi = str(tmp_path / "capi_san.o")
    run([HIPCC, f"--offload-arch={B.ARCH}", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
         *san, "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", B.INCLUDE, "-I", B.CSRC, "-c", os.path.join(B.CSRC, "capi.hip"), "-o", capi])
    drv = str(tmp_path / "abi_driver.o")
    run([HIPCC, "--offload-host-only", "-std=c++17", "-O1", "-g", *san, "-I", B.INCLUDE, "-c",
         "-x", "c++", os.path.join(HERE, "abi_driver.cpp"), "-o", drv])
    exe = str(tmp_path / "abi_driver")
    run([HIPCC, f"--offload-arch={B.ARCH}", *san, drv, capi, *others, "-o", exe])
    # (the HIP runtime's own allocations outlive main: leak checks off)
    r = run([exe], env=dict(ENV, ASAN_OPTIONS="detect_leaks=0"))
    assert "abi driver ok" in r.stdout
