"""The fixtures of tests/golden: exact update coefficients (Eq. 7 and Eq. 1)
and the oracle's stored regression losses, checked against the oracle on the
CPU and against the HIP path on the GPU."""
import os

import numpy as np
import pytest

HERE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _coefficients():
    rows = []
    with open(os.path.join(HERE, "update_coefficients.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                k, lr, eps, n, a, b, c = line.split()
                rows.append((k, float(lr), float(eps), int(n), float(a), float(b), float(c)))
    return rows


def _losses():
    import sys
    sys.path.insert(0, HERE)
    from make_golden import CASES
    stored = {}
    with open(os.path.join(HERE, "oracle_losses.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                name, lp, lm, l0 = [x.strip() for x in line.split("|")]
                stored[name] = (np.array([float(x) for x in lp.split()]), np.array([float(x) for x in lm.split()]),
                                float(l0))
    return [(c, stored[c[0]]) for c in CASES]


@pytest.mark.parametrize("row", _coefficients(), ids=lambda r: f"{r[0]}-{r[3]}-{r[4]}-{r[5]}")
def test_update_coefficients_exact(oracle, row):
    kind, lr, eps, n, a, b, c = row
    got = oracle.update_coeff(lr, n, a, b, eps) if kind == "central" else oracle.fd_update_coeff(lr, n, a, b, eps)
    assert got == c


@pytest.mark.parametrize("case", _losses(), ids=lambda c: c[0][0])
def test_oracle_reproduces_stored_losses(oracle, case):
    from paper_2505_17852_amd import workloads as wl
    (name, cfg, si, ss, eps, N, B, C, ts), (lp, lm, l0) = case
    theta = oracle.init(cfg, si)
    tok = wl.uniform_tokens(np.random.default_rng(ts), B, C, cfg["vocab"])
    gp, gm = oracle.perturbed_losses(cfg, theta, ss, eps, N, tok, as_double=True)
    _, g0 = oracle.fd_losses(cfg, theta, ss, eps, N, tok)
    np.testing.assert_allclose(gp, lp, rtol=1e-13)
    np.testing.assert_allclose(gm, lm, rtol=1e-13)
    assert abs(g0 - l0) <= 1e-13 * abs(l0)


@pytest.mark.gpu
@pytest.mark.parametrize("case", _losses(), ids=lambda c: c[0][0])
def test_hip_path_matches_stored_losses(case):
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2505_17852_amd import workloads as wl
    from paper_2505_17852_amd import zo
    (name, cfg, si, ss, eps, N, B, C, ts), (lp, lm, l0) = case
    print(f"stored losses {name}", flush=True)
    theta = zo.new_theta(cfg)
    zo.init(cfg, theta, si)
    tok = torch.from_numpy(wl.uniform_tokens(np.random.default_rng(ts), B, C, cfg["vocab"])).cuda()
    Lp, Lm = zo.perturbed_losses(cfg, theta, ss, eps, N, tok)
    _, L0 = zo.fd_losses(cfg, theta, ss, eps, N, tok)
    tol = 2e-2 if cfg["wdtype"] == wl.BF16 else 1e-5
    assert np.all(np.abs(Lp.cpu().numpy() - lp) <= tol * np.abs(lp))
    assert np.all(np.abs(Lm.cpu().numpy() - lm) <= tol * np.abs(lm))
    assert abs(float(L0.item()) - l0) <= tol * abs(l0)


def _wide():
    import sys
    sys.path.insert(0, HERE)
    from make_golden import WIDE_CASES, wide_key
    stored = {}
    with open(os.path.join(HERE, "oracle_losses_wide.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                key, lp, lm = [x.strip() for x in line.split("|")]
                stored[key] = (np.array([float(x) for x in lp.split()]), np.array([float(x) for x in lm.split()]))
    return WIDE_CASES, stored, wide_key


def test_wide_fixture_is_complete():
    cases, stored, key = _wide()
    for name, _, _, N, _, _, epss in cases:
        for eps in epss:
            lp, lm = stored[key(name, eps)]
            assert lp.size == N and lm.size == N and np.all(np.isfinite(lp)) and np.all(np.isfinite(lm))


@pytest.mark.parametrize("name", ["c4", "c3", "c3-rad"])
def test_oracle_reproduces_stored_wide_losses(oracle, name):
    """The first probe of each wide case at its largest and smallest eps
    (c4: the largest only), recomputed (a probe slice of one gives the same losses as in the full
    set)."""
    import sys
    sys.path.insert(0, HERE)
    from make_golden import wide_inputs
    cases, stored, key = _wide()
    (_, workload, probe, N, B, C, epss), = [c for c in cases if c[0] == name]
    cfg, sd, tok = wide_inputs(name, workload, probe, B, C)
    theta = oracle.init(cfg, sd["init"])
    for eps in ((epss[0],) if name == "c4" else (epss[0], epss[-1])):  # c4: ~10 s per probe
        gp, gm = oracle.perturbed_losses(cfg, theta, sd["step"], eps, 1, tok, as_double=True)
        lp, lm = stored[key(name, eps)]
        np.testing.assert_allclose(gp, lp[:1], rtol=1e-13)
        np.testing.assert_allclose(gm, lm[:1], rtol=1e-13)
