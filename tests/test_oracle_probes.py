"""Pins of the oracle's probe generator (Section 2: Rademacher and N(0,1)
probes with E[p] = 0 and E[p p^T] = I; Algorithm 2: one seeded sign per
parameter) and of the fp32 sub-functions fixed by the Box-Muller contract,
which are checked exhaustively against libm in double."""
import math

import numpy as np
import pytest
from scipy import stats

N24 = 1 << 24


def test_log_f32_exhaustive_against_libm(oracle):
    m = np.arange(N24, dtype=np.uint64)
    u = ((m + 1).astype(np.float64) * 2.0**-24).astype(np.float32)  # every u1 the contract can form
    got = oracle.log_f32(u).astype(np.float64)
    ref = np.log(u.astype(np.float64))
    ulp = np.spacing(np.abs(ref).astype(np.float32)).astype(np.float64)
    ulp[ref == 0] = np.spacing(np.float32(0))
    assert got[-1] == 0.0  # ln 1 == 0 exactly
    assert np.all(np.abs(got - ref) <= 3.0 * ulp)
    assert np.all(got <= 0.0)


def test_sincos_2pi_exhaustive_against_libm(oracle):
    k = np.arange(N24, dtype=np.uint32)
    s, c = oracle.sincos_2pi(k)
    ang = 2.0 * np.pi * k.astype(np.float64) * 2.0**-24
    assert np.max(np.abs(s - np.sin(ang))) <= 1.2e-7
    assert np.max(np.abs(c - np.cos(ang))) <= 1.2e-7
    # exact values on the axes
    for kk, (es, ec) in {0: (0.0, 1.0), 1 << 22: (1.0, 0.0), 1 << 23: (0.0, -1.0), 3 << 22: (-1.0, 0.0)}.items():
        assert abs(s[kk]) == abs(es) and c[kk] == ec or (s[kk] == es and abs(c[kk]) == abs(ec))
    # relative accuracy near the axes where the values are small but not zero
    small = (np.abs(np.sin(ang)) > 1e-7) & (np.abs(np.sin(ang)) < 1e-3)
    rel = np.abs(s[small] - np.sin(ang[small])) / np.abs(np.sin(ang[small]))
    assert rel.max() < 1e-6


def test_gauss_pair_against_double_box_muller(oracle):
    rng = np.random.default_rng(7)
    w = rng.integers(0, 2**32, size=2 * 2_000_000, dtype=np.uint64).astype(np.uint32)
    z = oracle.gauss_pairs(w).astype(np.float64)
    x0, x1 = w[0::2].astype(np.float64), w[1::2].astype(np.float64)
    u1 = (np.floor(x0 / 256) + 1) * 2.0**-24
    u2 = np.floor(x1 / 256) * 2.0**-24
    r = np.sqrt(-2.0 * np.log(u1))
    ref0, ref1 = r * np.cos(2 * np.pi * u2), r * np.sin(2 * np.pi * u2)
    assert np.max(np.abs(z[0::2] - ref0) / np.maximum(1.0, np.abs(ref0))) < 1e-6
    assert np.max(np.abs(z[1::2] - ref1) / np.maximum(1.0, np.abs(ref1))) < 1e-6
    # the extremes of the contract: u1 = 2^-24 gives the largest radius
    zz = oracle.gauss_pairs(np.array([0, 0], np.uint32))
    assert abs(zz[0] - math.sqrt(-2 * math.log(2.0**-24))) < 1e-5 and zz[1] == 0.0
    zz = oracle.gauss_pairs(np.array([0xFFFFFF00, 0x12345600], np.uint32))  # u1 == 1 -> radius 0
    assert zz[0] == 0.0 and zz[1] == 0.0


def test_rademacher_values_norm_and_moments(oracle):
    P = 3_000_017  # not a multiple of the block size: exercises the ragged tail
    z = oracle.probe(0, 99, 3, 0, P)
    assert set(np.unique(z).tolist()) == {-1.0, 1.0}
    assert float(np.dot(z.astype(np.float64), z)) == float(P)  # |p|_2 = sqrt(d) (Section 2)
    assert abs(z.mean()) < 5 / math.sqrt(P)
    # neighbouring elements and neighbouring probes are uncorrelated
    assert abs(np.mean(z[1:] * z[:-1])) < 5 / math.sqrt(P)
    z2 = oracle.probe(0, 99, 4, 0, P)
    assert abs(np.mean(z * z2)) < 5 / math.sqrt(P)
    z3 = oracle.probe(0, 100, 3, 0, P)
    assert abs(np.mean(z * z3)) < 5 / math.sqrt(P)
    # bits at a fixed position inside the 128-element block are balanced
    for pos in (0, 31, 32, 127):
        sel = z[pos::128]
        assert abs(sel.mean()) < 5 / math.sqrt(sel.size)


def test_gaussian_moments_and_ks(oracle):
    n = 8_000_000
    z = oracle.probe(1, 2024, 5, 0, n).astype(np.float64)
    assert abs(z.mean()) < 5 / math.sqrt(n)
    assert abs(z.var() - 1.0) < 5 * math.sqrt(2.0 / n)
    kurt = np.mean(z**4) / z.var() ** 2
    assert abs(kurt - 3.0) < 5 * math.sqrt(24.0 / n)
    assert abs(np.mean(z**3)) < 5 * math.sqrt(15.0 / n)
    ks = stats.kstest(z[:1_000_000], "norm")
    assert ks.pvalue > 1e-4
    # cosine and sine halves are each N(0,1) and uncorrelated with each other
    assert abs(np.mean(z[0::2] * z[1::2])) < 5 / math.sqrt(n / 2)
    z2 = oracle.probe(1, 2024, 6, 0, n // 4).astype(np.float64)
    assert abs(np.mean(z[: n // 4] * z2)) < 5 / math.sqrt(n / 4)


@pytest.mark.parametrize("kind", [0, 1])
def test_probe_range_matches_single_elements(oracle, kind):
    rng = np.random.default_rng(kind)
    for _ in range(20):
        j0 = int(rng.integers(0, 10**9))
        n = int(rng.integers(1, 700))
        i = int(rng.integers(0, 5000))
        seed = int(rng.integers(0, 2**63))
        zr = oracle.probe(kind, seed, i, j0, n)
        for t in rng.integers(0, n, size=10):
            assert zr[t] == oracle.probe_value(kind, seed, i, j0 + int(t))
