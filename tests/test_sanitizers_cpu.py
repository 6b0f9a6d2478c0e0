"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer: the CPU
oracle (every entry point on seeded random operators and meshes) and the
library's host side (argument validation, size queries, error reporting),
each built into a small executable with the sanitizers linked in, with leak
detection on.  No GPU: the library's device calls report TAPS_ERR_DEVICE."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2301_04285_amd", "csrc")
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
           UBSAN_OPTIONS="print_stacktrace=1")


def _run(exe):
    p = subprocess.run([exe], capture_output=True, text=True, timeout=600, env=ENV)
    assert p.returncode == 0, p.stdout + p.stderr
    assert "runtime error" not in p.stderr and "Sanitizer" not in p.stderr, p.stderr
    return p.stdout


def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=undefined", "-o", exe,
                    os.path.join(HERE, "sanitize", "oracle_driver.c"), "-lm"],
                   check=True, capture_output=True, timeout=300)
    assert "entries checked" in _run(exe)


def test_library_host_code_under_sanitizers(tmp_path):
    import torch
    if torch.cuda.is_available():
        pytest.skip("checks the no-device error path; run where no GPU is present")
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    exe = str(tmp_path / "abi_driver")
    # sanitizers on the host code only
    subprocess.run([hipcc, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
                    "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                    "-Xarch_host", "-fno-sanitize-recover=undefined",
                    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
                    os.path.join(CSRC, "taps_api.hip"), os.path.join(CSRC, "taps_kernels.hip"),
                    os.path.join(HERE, "sanitize", "abi_driver.cpp"), "-o", exe],
                   check=True, capture_output=True, timeout=600)
    assert "0 failures" in _run(exe)


def test_batched_alltoall_closed_forms(tmp_path):
    """The edge kernels' closed-form AllToAll costing (byte dot products over
    shard-fraction tables) against axis-by-axis costing from the definitions,
    on every closure of every tops mask (two classes) and on random
    hierarchies of link classes; host build of the device header, under the
    sanitizers."""
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    exe = str(tmp_path / "closed_forms")
    subprocess.run([hipcc, "-x", "hip", "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
                    "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                    "-Xarch_host", "-fno-sanitize-recover=undefined",
                    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
                    os.path.join(HERE, "sanitize", "closed_forms.cpp"), "-o", exe],
                   check=True, capture_output=True, timeout=600)
    out = _run(exe)
    assert " 0 mismatches" in out, out
    assert int(out.split()[0]) > 150_000
