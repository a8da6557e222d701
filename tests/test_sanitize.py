"""Sanitizer builds on the CPU (no GPU needed): the oracle, and the host side
of the library's C ABI, compiled with AddressSanitizer and
UndefinedBehaviorSanitizer and driven over small and degenerate inputs
(tests/sanitize/). Any out-of-bounds access, use after free, signed overflow
or other undefined behaviour aborts the driver. The device code of the
library is compiled as usual: the sanitizers apply to host code only."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


def _run(exe):
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=ENV)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr
    return r.stdout


def test_oracle_under_asan_ubsan(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("no gcc")
    exe = str(tmp_path / "oracle_san")
    subprocess.run(["gcc", "-std=c11", "-O1", "-g", *SAN, "-fno-fast-math", "-ffp-contract=off",
                    os.path.join(ROOT, "oracle", "oracle.c"),
                    os.path.join(HERE, "oracle_driver.c"), "-lm", "-o", exe], check=True)
    assert "oracle driver ok" in _run(exe)


def test_abi_host_side_under_asan_ubsan(tmp_path):
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    if not os.path.exists(hipcc):
        pytest.skip("no hipcc")
    from paper_2101_11552_amd import build as libbuild
    objs = [os.path.join(libbuild.BUILD, s + ".o") for s in libbuild.SOURCES if s != "api.cpp"]
    if not all(os.path.exists(o) for o in objs):
        libbuild.build()
    # the host-side sanitizer flags, each behind -Xarch_host (device code untouched)
    host_san = [f for flag in SAN for f in ("-Xarch_host", flag)]
    common = [f"--offload-arch={libbuild.ARCH}", "-O1", "-g", "-std=c++17", "-fPIC",
              "-I", os.path.join(ROOT, "include"), *host_san]
    api_o, drv_o, exe = (str(tmp_path / n) for n in ("api.o", "drv.o", "abi_san"))
    subprocess.run([hipcc, *common, "-c", os.path.join(libbuild.CSRC, "api.cpp"), "-o", api_o],
                   check=True, capture_output=True)
    subprocess.run([hipcc, *common, "-c", os.path.join(HERE, "abi_host_driver.cpp"), "-o", drv_o],
                   check=True, capture_output=True)
    subprocess.run([hipcc, f"--offload-arch={libbuild.ARCH}", *host_san, drv_o, api_o, *objs,
                    "-o", exe], check=True, capture_output=True)
    assert "abi host driver ok" in _run(exe)
