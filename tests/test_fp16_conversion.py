"""The host's fp32 -> fp16 conversion (f16_rne in the device header), used for
the fp16 bits of eps that the bf16-weight kernels add to the weight fragments,
against numpy's float16 conversion (IEEE round to nearest even) bit for bit:
normal values, ties, the subnormal range, overflow to infinity and NaN.
Compiled for the host only with hipcc; no GPU is used."""
import os
import shutil
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

SRC = r'''
#include <cstdio>
#include <cstdint>
#include <cstring>
#include "zo_rng.hpp"
int main() {
  uint32_t bits;
  while (std::scanf("%x", &bits) == 1) {
    float f;
    std::memcpy(&f, &bits, 4);
    std::printf("%04x\n", (unsigned)zo::f16_rne(f));
  }
  return 0;
}
'''


def inputs():
    rng = np.random.default_rng(7)
    vals = [0.0, -0.0, 1e-3, -1e-3, 65504.0, 65519.996, 65520.0, 1e6, np.inf, -np.inf,
            2.0 ** -14, 2.0 ** -24, 2.0 ** -25, 3 * 2.0 ** -26, 2.0 ** -26, 1.0 + 2.0 ** -11,
            1.0 + 3 * 2.0 ** -11, 2.0 ** -15 + 2.0 ** -25]
    f = np.array(vals, np.float32)
    # random fp32 bit patterns over the whole finite range, and ones near fp16 ties:
    # mantissas with the 13 bits below fp16's precision exactly 0x1000
    r = rng.integers(0, 0x7F800000, 20000, dtype=np.uint32)
    r |= (rng.integers(0, 2, 20000, dtype=np.uint32) << 31)
    ties = (rng.integers(0x33000000, 0x47800000, 5000, dtype=np.uint32) & ~np.uint32(0x1FFF)) | 0x1000
    # the subnormal and small-normal fp16 range
    sub = rng.uniform(0, 2.0 ** -13, 5000).astype(np.float32)
    allb = np.concatenate([f.view(np.uint32), r, ties.astype(np.uint32), sub.view(np.uint32)])
    return allb


def test_f16_rne_matches_ieee_rounding(tmp_path):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    src = tmp_path / "f16.cpp"
    src.write_text(SRC)
    exe = tmp_path / "f16"
    subprocess.run([hipcc, "-std=c++17", "-O1", "-x", "hip", "--offload-arch=gfx950", "-I",
                    os.path.join(ROOT, "paper_2505_17852_amd", "csrc"), str(src), "-o", str(exe)],
                   check=True, capture_output=True)
    b = inputs()
    inp = "\n".join(f"{x:08x}" for x in b) + "\n"
    out = subprocess.run([str(exe)], input=inp, check=True, capture_output=True, text=True).stdout.split()
    got = np.array([int(x, 16) for x in out], np.uint16)
    f = b.view(np.float32)
    with np.errstate(over="ignore"):
        ref = f.astype(np.float16).view(np.uint16)
    nan = np.isnan(f)
    assert np.all((got[nan] & 0x7C00) == 0x7C00) and np.all((got[nan] & 0x3FF) != 0)
    bad = np.nonzero((got != ref) & ~nan)[0]
    assert bad.size == 0, [(hex(b[i]), float(f[i]), hex(got[i]), hex(ref[i])) for i in bad[:8]]
