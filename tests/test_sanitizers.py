"""CPU builds of the oracle, the input generator and the C-ABI host layer under
AddressSanitizer and UndefinedBehaviorSanitizer (host code only; no GPU).

* tests/sanitize/oracle_checks.c drives every oracle entry point and every
  generator over small, degenerate and multi-threaded shapes, and the argument
  checks of both.
* tests/sanitize/host_checks.cpp drives the host side of libsom.so
  (som_api.cpp, built for the CPU with the device launches replaced by stubs
  that abort): the CSR validator over valid and broken batches, the workspace
  queries over the whole size range, the schedule, and every argument check
  that must reject a call before it reaches a device.

Each program exits non-zero on a failed check, and any sanitizer report aborts it.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-g", "-O1", "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")


def _run(cmd, cwd):
    r = subprocess.run(cmd, cwd=cwd, capture_output=True, text=True, env=ENV, timeout=600)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout}\n{r.stderr}"
    return r


@pytest.fixture(scope="module")
def outdir(tmp_path_factory):
    return tmp_path_factory.mktemp("sanitize")


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_and_synth_under_sanitizers(outdir):
    exe = str(outdir / "oracle_checks")
    _run(["gcc", "-std=c11", "-Wall", "-Wextra", "-Werror", *SAN, "tests/sanitize/oracle_checks.c", "oracle/oracle.c",
          "synth/synth.c", "-o", exe, "-lm", "-pthread"], ROOT)
    r = _run([exe], ROOT)
    assert "passed" in r.stdout


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.isdir("/opt/rocm/include"),
                    reason="needs g++ and the ROCm headers")
def test_host_layer_under_sanitizers(outdir):
    exe = str(outdir / "host_checks")
    _run(["g++", "-std=c++17", "-Wall", "-Wextra", *SAN, "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
          "-Iinclude", "tests/sanitize/host_checks.cpp", "tests/sanitize/host_stubs.cpp",
          "paper_2608_24067_amd/csrc/som_api.cpp", "-o", exe], ROOT)
    r = _run([exe], ROOT)
    assert "passed" in r.stdout
