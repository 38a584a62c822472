"""CPU sanitizer runs (no GPU): the oracle under AddressSanitizer +
UndefinedBehaviorSanitizer and under ThreadSanitizer (its pthread pool), and
the host side of the C ABI (descriptor checks, plan, host validation) under
AddressSanitizer + UndefinedBehaviorSanitizer.

Each build links a small driver from tests/sanitize/ that runs the code on
seeded inputs and checks results; a sanitizer report aborts the driver, so
the test only needs its exit status.  The C-ABI layer is linked here with
the GPU launchers replaced by stand-ins that report a
failed launch; no device code runs.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
ORACLE_SRC = os.path.join(ROOT, "oracle", "pda_oracle.c")
HIPCC = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")


def build_and_run(cmd, exe, env_extra=None, timeout=300):
    p = subprocess.run(cmd, capture_output=True, text=True, timeout=timeout)
    noise = "is not a recognized feature for this target"
    assert p.returncode == 0, "build failed:\n" + "\n".join(
        l for l in (p.stdout + p.stderr).splitlines() if noise not in l)
    env = dict(os.environ, **(env_extra or {}))
    r = subprocess.run([exe], capture_output=True, text=True, timeout=timeout, env=env)
    print(r.stdout + r.stderr)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "runtime error" not in r.stderr and "WARNING: ThreadSanitizer" not in r.stderr, r.stderr


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc is not installed")
@pytest.mark.parametrize("kind", ["address,undefined", "thread"])
def test_oracle_under_sanitizer(tmp_path, kind):
    exe = str(tmp_path / "oracle_sanitize")
    cmd = ["gcc", "-O1", "-g", "-std=c11", "-fno-omit-frame-pointer", f"-fsanitize={kind}",
           ORACLE_SRC, os.path.join(SAN, "oracle_sanitize.c"), "-lm", "-lpthread", "-o", exe]
    if kind != "thread":
        cmd.insert(4, "-fno-sanitize-recover=all")
    build_and_run(cmd, exe, {"ASAN_OPTIONS": "detect_leaks=1", "TSAN_OPTIONS": "halt_on_error=1"})


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc is not installed")
def test_host_abi_under_sanitizer(tmp_path):
    exe = str(tmp_path / "api_sanitize")
    # each sanitizer flag applies to the host pass alone (the device code of pda_api.hip, the no-alloc
    # scratch array, is compiled as usual and never runs here)
    cmd = [HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "paper_2405_11143_amd", "csrc"),
           os.path.join(ROOT, "paper_2405_11143_amd", "csrc", "pda_api.hip"),
           os.path.join(SAN, "api_sanitize.cpp"), "-o", exe]
    build_and_run(cmd, exe, {"ASAN_OPTIONS": "detect_leaks=0"})
