"""The host side of the C ABI (paper_2505_17852_amd/csrc/zo_api.hip: config
and shape checks, workspace planning, the allocation-free entry point's size
check, error strings) built with AddressSanitizer and UndefinedBehaviorSanitizer
on its host pass and driven through every entry point
(tests/helpers/api_sanitize_driver.cpp). The kernel launchers are stubbed by
the driver to report a device error, so no kernel runs and no GPU is needed:
every call must return its expected status with no sanitizer report."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2505_17852_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=undefined"]


def run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise AssertionError(" ".join(cmd) + "\n" + r.stdout[-2000:] + r.stderr[-4000:])


def test_api_host_side_under_asan_and_ubsan(tmp_path):
    if not os.path.exists(HIPCC):
        pytest.skip("no hipcc")
    common = ["-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", *SAN]
    hip = ["--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
    objs = []
    for src in ("zo_api.hip", "zo_profile.hip"):
        o = str(tmp_path / (src + ".o"))
        run([HIPCC, *hip, *common, "-c", os.path.join(CSRC, src), "-o", o])
        objs.append(o)
    drv = str(tmp_path / "driver.o")
    run([HIPCC, *common, "-x", "c++", "-I/opt/rocm/include", "-D__HIP_PLATFORM_AMD__", "-c",
         os.path.join(ROOT, "tests", "helpers", "api_sanitize_driver.cpp"), "-o", drv])
    exe = str(tmp_path / "api_sanitize")
    run([HIPCC, "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", *objs, drv,
         "-L/opt/rocm/lib", "-lrocprofiler-sdk-roctx", "-Wl,-rpath,/opt/rocm/lib", "-o", exe])
    # leaks: the HIP runtime keeps allocations of its own until exit
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "api sanitizer driver ok" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr
