"""Host replay of the bf16 kernels' operand addressing (no GPU): the
activation copies into LDS, the fragment-packed B loads, the sign-probe
cache loads, the gate's cell-state copies and the head's bias copies of
every workgroup, wave, lane, copy and k step of the gate and head launches
stay inside the buffer resources they are issued against, every offset fits
in 32 bits, the copies fill each LDS row and slot exactly once, and the packed
layout and the gate column order are bijections. The replay calls the same
address functions as the kernels (paper_2505_17852_amd/csrc/zo_pack.hpp),
built for the host by tests/helpers/bf16_addresses.cpp."""
import os
import shutil
import subprocess

import pytest

from paper_2505_17852_amd import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.fixture(scope="module")
def replay(tmp_path_factory):
    if not os.path.exists(HIPCC) and shutil.which("hipcc") is None:
        pytest.skip("no hipcc")
    exe = str(tmp_path_factory.mktemp("addr") / "bf16_addresses")
    subprocess.run([HIPCC if os.path.exists(HIPCC) else "hipcc", "-O2", "-std=c++17",
                    os.path.join(ROOT, "tests", "helpers", "bf16_addresses.cpp"), "-o", exe],
                   check=True, capture_output=True)
    return exe


def _shape(name):
    c = wl.CONFIGS[name]
    return (c["n_layers"], c["vocab"], c["embed"], c["hidden"], c["N"], c["B"])


SHAPES = [
    # the workloads with bf16 weights at their full launch configuration, and the
    # same models with other probe counts
    ("c4", _shape("c4")), ("c3", _shape("c3")), ("c3-rad20", (3, 50000, 1024, 1024, 20, 256)),
    ("c4-short", (6, 50000, 4096, 4096, 1, 2)),
    # the shapes of the bf16 GPU tests
    ("ragged", (2, 300, 64, 128, 2, 5)), ("gauss", (2, 200, 128, 64, 3, 3)), ("deep3", (3, 130, 64, 192, 3, 2)),
    ("tiny", (1, 40, 64, 64, 2, 2)), ("v1", (1, 1, 64, 64, 1, 1)), ("wide-batch", (2, 256, 64, 64, 4, 300)),
]


@pytest.mark.parametrize("fd", [0, 1], ids=["central", "forward"])
@pytest.mark.parametrize("name,shape", SHAPES, ids=[s[0] for s in SHAPES])
def test_bf16_addresses_in_bounds(replay, name, shape, fd):
    L, V, E, H, N, B = shape
    r = subprocess.run([replay, str(L), str(V), str(E), str(H), str(N), str(B), str(fd)], capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stdout
