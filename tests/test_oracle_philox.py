"""Pins the oracle's Philox4x32-10 against two independent implementations
that ship as source in this image (PyTorch's PhiloxRNGEngine.h and rocRAND's
rocrand_philox4x32_10.h), compiled and run live. The generator is the one of
Salmon et al. (SC'11); the paper draws its probes from PyTorch's seeded
generator (Algorithm 2), for which a counter-based Philox stream stands in."""
import os
import shutil
import subprocess

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
TORCH_INC = None
try:
    import torch  # noqa: F401
    TORCH_INC = os.path.join(os.path.dirname(torch.__file__), "include")
except Exception:  # pragma: no cover
    pass


def _inputs(n_random=2000):
    rng = np.random.default_rng(12345)
    fixed = [
        [0, 0, 0, 0, 0, 0],
        [0xFFFFFFFF] * 6,
        [0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344, 0xA4093822, 0x299F31D0],
        [1, 0, 0, 0, 0, 0],
        [0, 0, 7, 1, 3011, 0],
        [0xFFFFFFFF, 0xFFFFFFFF, 5, 2, 0x12345678, 0x9ABCDEF0],
    ]
    rand = rng.integers(0, 2**32, size=(n_random, 6), dtype=np.uint64).tolist()
    return fixed + rand


def _run(exe, rows):
    text = "\n".join(" ".join("%x" % v for v in r) for r in rows) + "\n"
    out = subprocess.run([exe], input=text, capture_output=True, text=True, check=True).stdout
    return [[int(x, 16) for x in line.split()] for line in out.strip().splitlines()]


def _oracle_rows(oracle, rows):
    return [oracle.philox(r[:4], r[4:]).tolist() for r in rows]


@pytest.mark.skipif(TORCH_INC is None or shutil.which("g++") is None, reason="needs torch headers and g++")
def test_philox_matches_torch_engine(oracle, tmp_path):
    exe = str(tmp_path / "xt")
    subprocess.run(["g++", "-std=c++17", "-O1", "-I" + TORCH_INC,
                    os.path.join(HERE, "helpers", "philox_xcheck_torch.cpp"), "-o", exe], check=True)
    rows = _inputs()
    assert _run(exe, rows) == _oracle_rows(oracle, rows)


@pytest.mark.skipif(shutil.which("hipcc") is None, reason="needs hipcc for the rocRAND header")
def test_philox_matches_rocrand_engine(oracle, tmp_path):
    exe = str(tmp_path / "xr")
    subprocess.run(["hipcc", "-std=c++17", "-O1",
                    os.path.join(HERE, "helpers", "philox_xcheck_rocrand.cpp"), "-o", exe], check=True)
    rows = _inputs()
    assert _run(exe, rows) == _oracle_rows(oracle, rows)


def test_philox_counter_and_key_sensitivity(oracle):
    base = oracle.philox([5, 0, 3, 0], [11, 0])
    for ctr, key in [([6, 0, 3, 0], [11, 0]), ([5, 1, 3, 0], [11, 0]), ([5, 0, 4, 0], [11, 0]),
                     ([5, 0, 3, 1], [11, 0]), ([5, 0, 3, 0], [12, 0]), ([5, 0, 3, 0], [11, 1])]:
        other = oracle.philox(ctr, key)
        # every output word changes (avalanche), so no two probes or blocks share bits
        assert np.all(other != base)
