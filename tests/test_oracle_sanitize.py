"""The oracle built with AddressSanitizer and UndefinedBehaviorSanitizer
(host C, gcc) and driven through every entry point on small models, error
paths included (tests/helpers/oracle_sanitize_driver.c): no sanitizer report,
every call returning its expected status."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_oracle_under_asan_and_ubsan(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("no C compiler")
    exe = tmp_path / "oracle_sanitize"
    flags = ["-std=c11", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=undefined", "-ffp-contract=off", "-fopenmp"]
    try:
        subprocess.run([gcc, *flags, "-I", os.path.join(ROOT, "oracle"),
                        os.path.join(ROOT, "oracle", "zo_oracle.c"),
                        os.path.join(ROOT, "tests", "helpers", "oracle_sanitize_driver.c"),
                        "-o", str(exe), "-lm"], check=True, capture_output=True, text=True)
    except subprocess.CalledProcessError as e:
        if "asan" in e.stderr.lower() or "sanitize" in e.stderr.lower():
            pytest.skip("sanitizer runtime not available: " + e.stderr[-200:])
        raise
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "oracle sanitizer driver ok" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr
