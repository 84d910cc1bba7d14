"""Sanitizer builds on the CPU (no GPU): the ABI layer's argument validation
(abi.cpp, host code only, kernel launchers replaced by stubs that must never
be reached) and the oracle's C leg, each built with AddressSanitizer and
UndefinedBehaviorSanitizer and run on inputs that exercise every rejection
path, zero-sized calls and the host-side threshold computation."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = "/opt/rocm/bin/hipcc"
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")

pytestmark = pytest.mark.skipif(os.path.exists("/dev/kfd"), reason="CPU-only sanitizer builds")


def _run(cmd, cwd):
    r = subprocess.run(cmd, cwd=cwd, capture_output=True, text=True)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout}\n{r.stderr}"
    return r


def test_abi_validation_under_sanitizers(tmp_path):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    objs = []
    for src in ("paper_2607_29221_amd/csrc/abi.cpp", "tests/abi_stub_launchers.cpp", "tests/abi_sanitize_driver.cpp"):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        _run([HIPCC, "-x", "hip", "--cuda-host-only", "-std=c++17", "-O1", "-g"] + SAN +
             ["-c", os.path.join(ROOT, src), "-o", obj], str(tmp_path))
        objs.append(obj)
    exe = str(tmp_path / "abi_san")
    _run([HIPCC] + SAN + objs + ["-o", exe], str(tmp_path))
    r = subprocess.run([exe], capture_output=True, text=True, env=ENV)
    assert r.returncode == 0 and "PASS" in r.stdout, r.stdout + r.stderr
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr


def test_oracle_c_under_sanitizers(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    exe = str(tmp_path / "oracle_san")
    _run(["gcc", "-O1", "-g", "-fopenmp", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
          os.path.join(ROOT, "oracle/c/philox_stream.c"), os.path.join(ROOT, "oracle/c/ring_oracle.c"),
          os.path.join(ROOT, "tests/oracle_sanitize_driver.c"), "-o", exe, "-lm"], str(tmp_path))
    r = subprocess.run([exe], capture_output=True, text=True, env=ENV)
    assert r.returncode == 0 and "PASS" in r.stdout, r.stdout + r.stderr
    assert "runtime error" not in r.stderr, r.stderr
