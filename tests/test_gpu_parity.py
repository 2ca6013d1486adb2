"""GPU path vs the CPU oracle, on the same seeded inputs, through the C ABI.

Bars: probe values and initial weights bit-exact; per-pass losses within
1e-5 relative (fp32 path); updated fp32 theta within 1e-5 relative with an
absolute floor of 1e-5 times the mean |theta|.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

from paper_2505_17852_amd import workloads as wl  # noqa: E402

LOSS_RTOL = 1e-5


@pytest.fixture(scope="module")
def zo():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2505_17852_amd import zo as z
    z.lib()
    return z


def say(*a):
    print(*a, flush=True)


def dev_tokens(tokens, mask):
    t = torch.from_numpy(np.ascontiguousarray(tokens)).cuda()
    m = None if mask is None else torch.from_numpy(np.ascontiguousarray(mask)).cuda()
    return t, m


def assert_bits_equal(got, ref, what):
    g, r = got.view(np.uint32), ref.view(np.uint32)
    bad = np.nonzero(g != r)[0]
    if bad.size:
        k = bad[:8]
        raise AssertionError(f"{what}: {bad.size} of {g.size} differ; first at {k.tolist()}: "
                             f"gpu {got[k].tolist()} oracle {ref[k].tolist()}")


def theta_close(got, ref, cfg):
    if cfg["wdtype"] == wl.BF16:
        g = (got.astype(np.uint32) << 16).view(np.float32)
        r = (ref.astype(np.uint32) << 16).view(np.float32)
        ulp = np.abs(r) * 2.0 ** -7 + 1e-30
        return np.all(np.abs(g - r) <= ulp)
    tol = 1e-5 * np.abs(ref) + 1e-5 * np.abs(ref).mean()
    return np.all(np.abs(got.astype(np.float64) - ref) <= tol)


# ---------------------------------------------------------------------------
# probe stream

@pytest.mark.parametrize("kind", [wl.RADEMACHER, wl.GAUSSIAN])
@pytest.mark.parametrize("seed,i,j0,n", [(1, 0, 0, 5000), (0xDEADBEEF12345678, 7, 1 << 33, 3001),
                                         (3003, 1023, 123457, 777)])
def test_probe_bit_exact(zo, oracle, kind, seed, i, j0, n):
    say(f"probe kind={kind} seed={seed} i={i} j0={j0} n={n}")
    got = zo.debug_probe(kind, seed, i, j0, n).cpu().numpy()
    ref = oracle.probe(kind, seed, i, j0, n)
    assert_bits_equal(got, ref, "probe")


def test_gaussian_transform_exhaustive(zo, oracle):
    """Every one of the 2^24 radius inputs and 2^24 angle inputs (the low 8
    bits of each word are ignored by the transform; fill them at random)."""
    say("box-muller over all 2^24 inputs")
    rng = np.random.default_rng(7)
    k = np.arange(1 << 24, dtype=np.uint32)
    words = np.empty(2 << 24, np.uint32)
    words[0::2] = (k << 8) | rng.integers(0, 256, k.size, dtype=np.uint32)
    words[1::2] = (k[::-1] << 8) | rng.integers(0, 256, k.size, dtype=np.uint32)
    got = zo.debug_gauss_pairs(torch.from_numpy(words.view(np.int32)).cuda()).cpu().numpy()
    ref = oracle.gauss_pairs(words)
    assert_bits_equal(got, ref, "box-muller")


# ---------------------------------------------------------------------------
# initialisation

@pytest.mark.parametrize("cfg", [wl.model_cfg("c1"), wl.model_cfg("c2"),
                                 dict(n_layers=2, vocab=300, embed=64, hidden=96, wdtype=wl.BF16, probe=0)])
def test_init_bit_exact(zo, oracle, cfg):
    say(f"init {cfg}")
    theta = zo.new_theta(cfg)
    zo.init(cfg, theta, 2001)
    got = theta.view(torch.int16 if cfg["wdtype"] == wl.BF16 else torch.int32).cpu().numpy()
    ref = oracle.init(cfg, 2001)
    assert np.array_equal(got.view(ref.dtype), ref)


# ---------------------------------------------------------------------------
# update

UPDATE_CASES = [
    ("c1-rad", dict(wl.model_cfg("c1")), 8, 1e-2, 1e-3),
    # sign probes, N <= 16: two 8192-parameter tiles, the second ragged (P = 13325)
    ("tiles-rad16-bf16", dict(n_layers=1, vocab=77, embed=32, hidden=32, wdtype=wl.BF16, probe=0), 16, 1e-3, 1e-3),
    # 23 tiles, 8 < N < 16 (probes 11..15 absent), fp32
    ("tiles-rad11-fp32", dict(n_layers=2, vocab=300, embed=64, hidden=96, wdtype=wl.FP32, probe=0), 11, 1e-2, 1e-2),
    # N <= 8: one table
    ("tiles-rad5-bf16", dict(n_layers=2, vocab=300, embed=64, hidden=96, wdtype=wl.BF16, probe=0), 5, 1e-3, 1e-3),
    ("ragged-rad-bf16", dict(n_layers=1, vocab=77, embed=32, hidden=32, wdtype=wl.BF16, probe=0), 37, 1e-3, 1e-3),
    ("gauss-fp32", dict(n_layers=1, vocab=50, embed=32, hidden=64, wdtype=wl.FP32, probe=1), 19, 1e-2, 1e-2),
    ("gauss-bf16", dict(n_layers=2, vocab=50, embed=32, hidden=32, wdtype=wl.BF16, probe=1), 300, 1e-3, 1e-3),
]


@pytest.mark.parametrize("name,cfg,N,eps,lr", UPDATE_CASES, ids=[c[0] for c in UPDATE_CASES])
def test_update_parity(zo, oracle, name, cfg, N, eps, lr):
    say(f"update {name} P={zo.param_count(cfg)} N={N}")
    rng = np.random.default_rng(11)
    theta = zo.new_theta(cfg)
    zo.init(cfg, theta, 5)
    ref = oracle.init(cfg, 5)
    Lp = (5.0 + rng.standard_normal(N) * 0.01).astype(np.float32)
    Lm = (5.0 + rng.standard_normal(N) * 0.01).astype(np.float32)
    zo.update(cfg, theta, 99, eps, lr, torch.from_numpy(Lp).cuda(), torch.from_numpy(Lm).cuda(), i0=3)
    got = theta.view(torch.int16 if cfg["wdtype"] == wl.BF16 else torch.int32).cpu().numpy().view(ref.dtype)
    assert oracle.update(cfg, ref, 99, eps, lr, Lp, Lm, i0=3) == 0
    assert theta_close(got, ref, cfg)


@pytest.mark.parametrize("wdtype", [wl.FP32, wl.BF16])
@pytest.mark.parametrize("N", [5, 12, 16])
def test_update_small_n_kernel_matches_general(zo, wdtype, N):
    """Sign probes with N <= 16 run their own update kernel; it forms the same
    table sums in the same order as the kernel for any N. With lr = N 2^-10 and
    lr' = 17 2^-10 both calls use the coefficients 2^-10 (L+ - L-)/(2 eps), so
    N probes and 17 probes whose last 17 - N have L+ = L- (coefficient 0) must
    give the same theta (as values: only the sign of a zero may differ)."""
    cfg = dict(n_layers=2, vocab=300, embed=64, hidden=96, wdtype=wdtype, probe=wl.RADEMACHER)
    say(f"update small-N vs general: N={N} wdtype={wdtype} P={zo.param_count(cfg)}")
    rng = np.random.default_rng(N)
    Lp = (5.0 + rng.standard_normal(17) * 0.01).astype(np.float32)
    Lm = (5.0 + rng.standard_normal(17) * 0.01).astype(np.float32)
    Lm[N:] = Lp[N:]
    a = zo.new_theta(cfg)
    zo.init(cfg, a, 7)
    b = a.clone()
    zo.update(cfg, a, 123, 1e-3, N * 2.0 ** -10, torch.from_numpy(Lp[:N]).cuda(),
              torch.from_numpy(Lm[:N]).cuda(), i0=9)
    zo.update(cfg, b, 123, 1e-3, 17 * 2.0 ** -10, torch.from_numpy(Lp).cuda(),
              torch.from_numpy(Lm).cuda(), i0=9)
    if wdtype == wl.BF16:
        fa = (a.view(torch.int16).cpu().numpy().astype(np.uint16).astype(np.uint32) << 16).view(np.float32)
        fb = (b.view(torch.int16).cpu().numpy().astype(np.uint16).astype(np.uint32) << 16).view(np.float32)
    else:
        fa, fb = a.cpu().numpy(), b.cpu().numpy()
    bad = np.nonzero(fa != fb)[0]
    assert bad.size == 0, f"{bad.size} differ, first {bad[:5].tolist()}: {fa[bad[:5]]} vs {fb[bad[:5]]}"


def test_update_equal_losses_leave_theta_unchanged(zo):
    cfg = wl.model_cfg("c1")
    theta = zo.new_theta(cfg)
    zo.init(cfg, theta, 5)
    before = theta.clone()
    L = torch.full((8,), 3.25, device="cuda")
    zo.update(cfg, theta, 1, 1e-2, 1e-3, L, L.clone())
    assert torch.equal(theta.view(torch.int32), before.view(torch.int32))


def test_update_nonfinite_skips(zo):
    cfg = wl.model_cfg("c1")
    theta = zo.new_theta(cfg)
    zo.init(cfg, theta, 5)
    before = theta.clone()
    Lp = torch.full((8,), 3.0, device="cuda")
    Lm = Lp.clone()
    Lm[5] = float("nan")
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    zo.update(cfg, theta, 1, 1e-2, 1e-3, Lp, Lm, skipped=flag)
    assert flag.item() == 1
    assert torch.equal(theta.view(torch.int32), before.view(torch.int32))
    Lm[5] = 3.5
    zo.update(cfg, theta, 1, 1e-2, 1e-3, Lp, Lm, skipped=flag)
    assert flag.item() == 0
    assert not torch.equal(theta.view(torch.int32), before.view(torch.int32))


# ---------------------------------------------------------------------------
# perturbed losses

LOSS_CASES = [
    # name, model cfg, N, B, C, eps, masked
    ("c1", wl.model_cfg("c1"), 8, 4, 32, 1e-2, False),
    # several tiles and ragged tails: 3 unit tiles (H=96, unaligned K), vocab 300 (2 full
    # vocabulary tiles + 44), B=5 (padded rows), C=20 (a full and a partial time chunk)
    ("ragged-rad", dict(n_layers=2, vocab=300, embed=64, hidden=96, wdtype=0, probe=0), 3, 5, 20, 1e-2, True),
    ("ragged-gauss", dict(n_layers=2, vocab=300, embed=32, hidden=128, wdtype=0, probe=1), 2, 3, 18, 1e-2, True),
    ("deep3-gauss", dict(n_layers=3, vocab=130, embed=128, hidden=64, wdtype=0, probe=1), 2, 2, 9, 1e-3, False),
    ("c2-widths", wl.model_cfg("c2"), 2, 3, 12, 1e-3, True),
    ("c5-widths", wl.model_cfg("c5"), 2, 2, 10, 1e-2, False),
    # B = 64 fills 128 rows per probe: the 128-row workgroups of the fp32 gate
    ("wide-rad", dict(n_layers=2, vocab=100, embed=32, hidden=64, wdtype=0, probe=0), 2, 64, 5, 1e-2, True),
    ("wide-gauss", dict(n_layers=2, vocab=100, embed=64, hidden=96, wdtype=0, probe=1), 2, 50, 4, 1e-2, True),
]


def _tokens_for(name, cfg, B, C, masked, seed=4242):
    rng = np.random.default_rng(seed)
    if name.startswith("c2"):
        return wl.reverse_task(rng, B, C, cfg["vocab"])
    tok = wl.uniform_tokens(rng, B, C, cfg["vocab"])
    mask = (rng.random((B, C)) < 0.6).astype(np.uint8) if masked else None
    return tok, mask


@pytest.mark.parametrize("name,cfg,N,B,C,eps,masked", LOSS_CASES, ids=[c[0] for c in LOSS_CASES])
def test_losses_match_oracle(zo, oracle, name, cfg, N, B, C, eps, masked):
    say(f"losses {name} cfg={cfg} N={N} B={B} C={C}")
    tok, mask = _tokens_for(name, cfg, B, C, masked)
    theta = zo.new_theta(cfg)
    zo.init(cfg, theta, 77)
    ref_theta = oracle.init(cfg, 77)
    td, md = dev_tokens(tok, mask)
    Lp, Lm = zo.perturbed_losses(cfg, theta, 12345, eps, N, td, md, i0=4)
    gp, gm = Lp.cpu().numpy(), Lm.cpu().numpy()
    rp, rm = oracle.perturbed_losses(cfg, ref_theta, 12345, eps, N, tok, mask, i0=4, as_double=True)
    say("gpu", gp, gm, "oracle", rp, rm)
    assert np.all(np.abs(gp - rp) <= LOSS_RTOL * np.abs(rp))
    assert np.all(np.abs(gm - rm) <= LOSS_RTOL * np.abs(rm))


def test_losses_slice_and_determinism(zo):
    """Probe slices [i0, i0+n) reproduce the full set's losses bit for bit,
    and two runs are bit-identical."""
    cfg = dict(n_layers=2, vocab=200, embed=64, hidden=64, wdtype=0, probe=0)
    B, C = 6, 17
    tok, _ = _tokens_for("x", cfg, B, C, False)
    theta = zo.new_theta(cfg)
    zo.init(cfg, theta, 3)
    td, _ = dev_tokens(tok, None)
    Lp, Lm = zo.perturbed_losses(cfg, theta, 9, 1e-2, 7, td)
    Lp2, Lm2 = zo.perturbed_losses(cfg, theta, 9, 1e-2, 7, td)
    assert torch.equal(Lp, Lp2) and torch.equal(Lm, Lm2)
    sp, sm = zo.perturbed_losses(cfg, theta, 9, 1e-2, 3, td, i0=2)
    assert torch.equal(sp, Lp[2:5]) and torch.equal(sm, Lm[2:5])


def test_empty_mask_gives_zero_loss(zo):
    cfg = wl.model_cfg("c1")
    theta = zo.new_theta(cfg)
    zo.init(cfg, theta, 3)
    tok, _ = _tokens_for("x", cfg, 2, 5, False)
    td, _ = dev_tokens(tok, None)
    m = torch.zeros((2, 5), dtype=torch.uint8, device="cuda")
    Lp, Lm = zo.perturbed_losses(cfg, theta, 1, 1e-2, 2, td, m)
    assert torch.all(Lp == 0) and torch.all(Lm == 0)


def test_zero_weights_give_ln_v(zo):
    """theta = 0 and eps tiny: every logit is O(eps), so L is ln V to O(eps)."""
    cfg = dict(n_layers=2, vocab=256, embed=32, hidden=64, wdtype=0, probe=0)
    theta = torch.zeros(zo.param_count(cfg), dtype=torch.float32, device="cuda")
    tok, _ = _tokens_for("x", cfg, 3, 6, False)
    td, _ = dev_tokens(tok, None)
    Lp, Lm = zo.perturbed_losses(cfg, theta, 1, 1e-6, 2, td)
    assert torch.allclose(Lp.double(), torch.full_like(Lp.double(), np.log(256)), rtol=1e-5)
    assert torch.allclose(Lm.double(), torch.full_like(Lm.double(), np.log(256)), rtol=1e-5)


# ---------------------------------------------------------------------------
# a full step at a workload's real size, in the launch configuration the
# benchmark times, checked on the first probe's two passes

def test_c2_full_size_first_probe(zo, oracle):
    name = "c2"
    w = wl.CONFIGS[name]
    cfg = wl.model_cfg(name)
    sd = wl.seeds(name)
    tok, mask = wl.batch(name)
    say(f"full-size {name}: N={w['N']} B={w['B']} C={w['C']}")
    theta = zo.new_theta(cfg)
    zo.init(cfg, theta, sd["init"])
    td, md = dev_tokens(tok, mask)
    Lp, Lm = zo.perturbed_losses(cfg, theta, sd["step"], w["eps"], w["N"], td, md)
    gp, gm = Lp.cpu().numpy(), Lm.cpu().numpy()
    ref_theta = oracle.init(cfg, sd["init"])
    rp, rm = oracle.perturbed_losses(cfg, ref_theta, sd["step"], w["eps"], 1, tok, mask, i0=0,
                                     as_double=True)
    say("gpu", gp[0], gm[0], "oracle", rp[0], rm[0])
    assert abs(gp[0] - rp[0]) <= LOSS_RTOL * abs(rp[0])
    assert abs(gm[0] - rm[0]) <= LOSS_RTOL * abs(rm[0])
    assert np.all(np.isfinite(gp)) and np.all(np.isfinite(gm))


# ---------------------------------------------------------------------------
# the estimator's signal: L+ - L- per probe (what the update consumes)

@pytest.mark.parametrize("name,B,C", [("c1", 4, 32), ("c5", 4, 16), ("c2", 4, 140)])
def test_delta_loss_matches_oracle(zo, oracle, name, B, C):
    """L+_n - L-_n agrees with the oracle's to within the fp32 spacing of the
    losses themselves (8 ulp of L) plus 1e-4 relative: the forward loses no
    resolution beyond the fp32 rounding of its outputs."""
    w = wl.CONFIGS[name]
    cfg = wl.model_cfg(name)
    sd = wl.seeds(name)
    tok, mask = wl.batch(name, B=B, C=C)
    N = 8
    theta = zo.new_theta(cfg)
    zo.init(cfg, theta, sd["init"])
    td, md = dev_tokens(tok, mask)
    Lp, Lm = zo.perturbed_losses(cfg, theta, sd["step"], w["eps"], N, td, md)
    gp, gm = Lp.cpu().numpy().astype(np.float64), Lm.cpu().numpy().astype(np.float64)
    rp, rm = oracle.perturbed_losses(cfg, oracle.init(cfg, sd["init"]), sd["step"], w["eps"], N,
                                     tok, mask, as_double=True)
    dg, dr = gp - gm, rp - rm
    say(f"{name}: dL gpu {dg} oracle {dr}")
    assert np.all(np.abs(dr) > 0)
    tol = 8 * 2.0 ** -24 * np.abs(rp) + 1e-4 * np.abs(dr)
    assert np.all(np.abs(dg - dr) <= tol)


@pytest.mark.parametrize("cfg,B", [
    (dict(n_layers=2, vocab=200, embed=32, hidden=64, wdtype=wl.FP32, probe=wl.GAUSSIAN), 5),
    (dict(n_layers=2, vocab=200, embed=32, hidden=64, wdtype=wl.FP32, probe=wl.GAUSSIAN), 64),
    (dict(n_layers=2, vocab=300, embed=64, hidden=128, wdtype=wl.BF16, probe=wl.GAUSSIAN), 5),
], ids=["fp32", "fp32-wide", "bf16"])
def test_probe_cache_is_bit_identical(zo, cfg, B):
    """Normal probes: the losses with the probe cache (default workspace) and
    without it (the smallest workspace: probes regenerated in every tile) are
    bit-identical, for a slice i0 > 0 and a ragged batch; with bf16 weights
    both for the fused products (eps = 1e-2: the cache holds the perturbed
    weights) and the two-stream ones (eps = 1e-4: the cache holds fp16(eps z)),
    over a 13-step head chunk of 3 row blocks per step (the head takes the
    row blocks of a cached probe in pass-block-major order)."""
    N, C = 3, 13
    say(f"probe cache {cfg} N={N} B={B} C={C}")
    rng = np.random.default_rng(23)
    tok = torch.from_numpy(wl.uniform_tokens(rng, B, C, cfg["vocab"])).cuda()
    theta = zo.new_theta(cfg)
    zo.init(cfg, theta, 4)
    assert zo.workspace_bytes(cfg, N, B, C) > zo.workspace_bytes_min(cfg, N, B, C)
    ws_full = zo.new_workspace(cfg, N, B, C)
    ws_min = zo.new_workspace(cfg, N, B, C, probe_cache=False)
    for eps in (1e-2, 1e-4) if cfg["wdtype"] == wl.BF16 else (1e-2,):
        a = zo.perturbed_losses(cfg, theta, 77, eps, N, tok, i0=5, workspace=ws_full)
        b = zo.perturbed_losses(cfg, theta, 77, eps, N, tok, i0=5, workspace=ws_min)
        assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1]), eps


def test_c5_full_size_sampled(zo, oracle):
    """c5 at its full launch configuration (N=1024 normal probes with the
    probe cache, B=32, C=128), scoring only the first positions of two
    sequences so that the oracle can compute the losses on the 2-sequence,
    3-position prefix; probes 0, 511 and 1023 are checked at the fp32 bar."""
    name = "c5"
    w = wl.CONFIGS[name]
    cfg = wl.model_cfg(name)
    sd = wl.seeds(name)
    tok, _ = wl.batch(name)
    B, C = tok.shape[0], tok.shape[1] - 1
    mask = np.zeros((B, C), np.uint8)
    mask[0, :3] = 1
    mask[1, :2] = 1
    say(f"{name} full size N={w['N']} B={B} C={C}, sampled positions")
    theta = zo.new_theta(cfg)
    zo.init(cfg, theta, sd["init"])
    td, md = dev_tokens(tok, mask)
    Lp, Lm = zo.perturbed_losses(cfg, theta, sd["step"], w["eps"], w["N"], td, md)
    gp, gm = Lp.cpu().numpy(), Lm.cpu().numpy()
    ref_theta = oracle.init(cfg, sd["init"])
    ref_tok = np.ascontiguousarray(tok[:2, :4])
    ref_mask = np.ascontiguousarray(mask[:2, :3])
    for i in (0, 511, w["N"] - 1):
        rp, rm = oracle.perturbed_losses(cfg, ref_theta, sd["step"], w["eps"], 1, ref_tok, ref_mask, i0=i)
        say(f"probe {i}: gpu {gp[i]} {gm[i]} oracle {rp[0]} {rm[0]}")
        assert abs(gp[i] - rp[0]) <= LOSS_RTOL * abs(rp[0])
        assert abs(gm[i] - rm[0]) <= LOSS_RTOL * abs(rm[0])


@pytest.mark.parametrize("name,cfg,N,B,C", [
    ("ragged", dict(n_layers=2, vocab=300, embed=64, hidden=96, wdtype=0, probe=0), 3, 5, 12),
    ("wide-gauss", dict(n_layers=2, vocab=100, embed=64, hidden=96, wdtype=0, probe=1), 2, 64, 6),
], ids=["ragged", "wide-gauss"])
def test_fp32_split_form_matches_oracle(zo, oracle, name, cfg, N, B, C):
    """The two-stream form of the fp32 products (zo_perturbed_losses_ex with
    ZO_PRODUCTS_SPLIT: W.h and (s h).(eps z) as two MFMA streams into one
    accumulator, kept for measurement) against the oracle at the fp32 bar, on
    64- and 128-row workgroups."""
    say(f"fp32 split form {name}")
    tok, mask = _tokens_for(name, cfg, B, C, True)
    theta = zo.new_theta(cfg)
    zo.init(cfg, theta, 19)
    td, md = dev_tokens(tok, mask)
    Lp, Lm = zo.perturbed_losses(cfg, theta, 4545, 1e-2, N, td, md, products=zo.PRODUCTS_SPLIT)
    gp, gm = Lp.cpu().numpy(), Lm.cpu().numpy()
    rp, rm = oracle.perturbed_losses(cfg, oracle.init(cfg, 19), 4545, 1e-2, N, tok, mask, as_double=True)
    say("gpu", gp, gm, "oracle", rp, rm)
    assert np.all(np.abs(gp - rp) <= LOSS_RTOL * np.abs(rp))
    assert np.all(np.abs(gm - rm) <= LOSS_RTOL * np.abs(rm))
