"""Degenerate and boundary cases of the step on the GPU, through the C ABI,
against the oracle: the smallest shapes (one probe, one sequence, one
position), a one-word vocabulary, a zero learning rate, probe indices at the
top of the 32-bit range, batches exactly at and one past the row granule,
a large perturbation and a nine-layer stack."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

from paper_2505_17852_amd import workloads as wl  # noqa: E402

RTOL = {wl.FP32: 1e-5, wl.BF16: 2e-2}


@pytest.fixture(scope="module")
def zo():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2505_17852_amd import zo as z
    z.lib()
    return z


def say(*a):
    print(*a, flush=True)


def run_both(zo, oracle, cfg, N, tok, mask, eps, seed=909, init_seed=33, i0=0):
    """GPU central and forward differences and the oracle's, on one theta."""
    theta = zo.new_theta(cfg)
    zo.init(cfg, theta, init_seed)
    td = torch.from_numpy(np.ascontiguousarray(tok)).cuda()
    md = None if mask is None else torch.from_numpy(np.ascontiguousarray(mask)).cuda()
    Lp, Lm = zo.perturbed_losses(cfg, theta, seed, eps, N, td, md, i0=i0)
    L, L0 = zo.fd_losses(cfg, theta, seed, eps, N, td, md, i0=i0)
    gpu = dict(Lp=Lp.cpu().numpy(), Lm=Lm.cpu().numpy(), L=L.cpu().numpy(), L0=L0.cpu().numpy())
    ref_theta = oracle.init(cfg, init_seed)
    rp, rm = oracle.perturbed_losses(cfg, ref_theta, seed, eps, N, tok, mask, i0=i0, as_double=True)
    rl, r0 = oracle.fd_losses(cfg, ref_theta, seed, eps, N, tok, mask, i0=i0)
    ref = dict(Lp=rp, Lm=rm, L=rl, L0=np.array([r0]))
    return gpu, ref


def check(gpu, ref, tol):
    for k in ref:
        g, r = gpu[k].astype(np.float64), ref[k]
        say(f"{k}: gpu {g[:4]} oracle {r[:4]}")
        assert np.all(np.abs(g - r) <= tol * np.abs(r)), k


MINIMAL = [
    ("fp32", dict(n_layers=1, vocab=2, embed=32, hidden=32, wdtype=wl.FP32, probe=wl.RADEMACHER)),
    ("fp32-gauss", dict(n_layers=1, vocab=2, embed=32, hidden=32, wdtype=wl.FP32, probe=wl.GAUSSIAN)),
    ("bf16", dict(n_layers=1, vocab=3, embed=64, hidden=64, wdtype=wl.BF16, probe=wl.RADEMACHER)),
    ("bf16-gauss", dict(n_layers=1, vocab=3, embed=64, hidden=64, wdtype=wl.BF16, probe=wl.GAUSSIAN)),
]


@pytest.mark.parametrize("name,cfg", MINIMAL, ids=[m[0] for m in MINIMAL])
def test_smallest_shapes(zo, oracle, name, cfg):
    """N = 1 probe, B = 1 sequence, C = 1 scored position, the narrowest
    widths each path accepts."""
    say(f"minimal {name}")
    tok = np.array([[1, 0]], np.int32)
    check(*run_both(zo, oracle, cfg, 1, tok, None, 1e-2), RTOL[cfg["wdtype"]])


@pytest.mark.parametrize("wdtype", [wl.FP32, wl.BF16], ids=["fp32", "bf16"])
def test_single_word_vocabulary(zo, wdtype):
    """With V = 1 the target is the only logit: every pass's loss is exactly
    log(1) = 0 (central and forward differences)."""
    E = 32 if wdtype == wl.FP32 else 64
    cfg = dict(n_layers=2, vocab=1, embed=E, hidden=E, wdtype=wdtype, probe=wl.RADEMACHER)
    theta = zo.new_theta(cfg)
    zo.init(cfg, theta, 5)
    tok = torch.zeros((3, 6), dtype=torch.int32, device="cuda")
    Lp, Lm = zo.perturbed_losses(cfg, theta, 1, 1e-2, 2, tok)
    L, L0 = zo.fd_losses(cfg, theta, 1, 1e-2, 2, tok)
    for x in (Lp, Lm, L, L0):
        assert torch.all(x == 0.0), x


@pytest.mark.parametrize("wdtype,probe", [(wl.FP32, wl.RADEMACHER), (wl.FP32, wl.GAUSSIAN),
                                          (wl.BF16, wl.RADEMACHER), (wl.BF16, wl.GAUSSIAN)])
def test_zero_learning_rate_leaves_theta(zo, wdtype, probe):
    cfg = dict(n_layers=1, vocab=77, embed=64, hidden=64, wdtype=wdtype, probe=probe)
    theta = zo.new_theta(cfg)
    zo.init(cfg, theta, 9)
    before = theta.clone()
    L1 = torch.tensor([3.0, 2.0, 2.5], device="cuda")
    L2 = torch.tensor([2.0, 2.5, 2.5], device="cuda")
    zo.update(cfg, theta, 3, 1e-3, 0.0, L1, L2)
    zo.fd_update(cfg, theta, 3, 1e-3, 0.0, L1, L2[:1])
    bits = torch.int16 if wdtype == wl.BF16 else torch.int32
    assert torch.equal(theta.view(bits), before.view(bits))


def test_probe_indices_at_the_top_of_the_range(zo, oracle):
    """i0 = 2^32 - N: the last probe index 2^32 - 1 is valid and matches the
    oracle; the host rejects one more (checked on the CPU)."""
    cfg = dict(n_layers=1, vocab=50, embed=32, hidden=64, wdtype=wl.FP32, probe=wl.GAUSSIAN)
    N = 3
    rng = np.random.default_rng(8)
    tok = wl.uniform_tokens(rng, 2, 5, cfg["vocab"])
    check(*run_both(zo, oracle, cfg, N, tok, None, 1e-2, i0=(1 << 32) - N), 1e-5)


GRANULE = [
    ("fp32-32", dict(n_layers=1, vocab=40, embed=32, hidden=32, wdtype=wl.FP32, probe=wl.RADEMACHER), 32),
    ("fp32-33", dict(n_layers=1, vocab=40, embed=32, hidden=32, wdtype=wl.FP32, probe=wl.RADEMACHER), 33),
    ("bf16-128", dict(n_layers=1, vocab=40, embed=64, hidden=64, wdtype=wl.BF16, probe=wl.GAUSSIAN), 128),
    ("bf16-129", dict(n_layers=1, vocab=40, embed=64, hidden=64, wdtype=wl.BF16, probe=wl.RADEMACHER), 129),
]


@pytest.mark.parametrize("name,cfg,B", GRANULE, ids=[g[0] for g in GRANULE])
def test_batch_at_and_past_the_row_granule(zo, oracle, name, cfg, B):
    """B equal to the rows one sign of a probe occupies (no padding rows)
    and one more (a whole granule of padding but one)."""
    say(f"granule {name} B={B}")
    rng = np.random.default_rng(B)
    tok = wl.uniform_tokens(rng, B, 3, cfg["vocab"])
    mask = (rng.random((B, 3)) < 0.8).astype(np.uint8)
    check(*run_both(zo, oracle, cfg, 2, tok, mask, 1e-2), RTOL[cfg["wdtype"]])


def test_large_perturbation(zo, oracle):
    """eps = 0.5: perturbations as large as the weights themselves."""
    cfg = dict(n_layers=2, vocab=60, embed=32, hidden=64, wdtype=wl.FP32, probe=wl.RADEMACHER)
    rng = np.random.default_rng(12)
    tok = wl.uniform_tokens(rng, 3, 7, cfg["vocab"])
    check(*run_both(zo, oracle, cfg, 2, tok, None, 0.5), 1e-5)


@pytest.mark.parametrize("wdtype", [wl.FP32, wl.BF16], ids=["fp32", "bf16"])
def test_deep_stack(zo, oracle, wdtype):
    """Nine layers and more timesteps than layers: on the fp32 path the
    middle wavefront steps have all nine layers active, more than one launch
    holds (eight), so they are split over two launches."""
    E = 32 if wdtype == wl.FP32 else 64
    cfg = dict(n_layers=9, vocab=20, embed=E, hidden=E, wdtype=wdtype, probe=wl.RADEMACHER)
    rng = np.random.default_rng(19)
    tok = wl.uniform_tokens(rng, 2, 12, cfg["vocab"])
    check(*run_both(zo, oracle, cfg, 1, tok, None, 1e-2), RTOL[wdtype])


BADTOK = [
    ("fp32", dict(n_layers=1, vocab=50, embed=32, hidden=32, wdtype=wl.FP32, probe=wl.RADEMACHER)),
    ("fp32-gauss", dict(n_layers=1, vocab=50, embed=32, hidden=32, wdtype=wl.FP32, probe=wl.GAUSSIAN)),
    ("bf16", dict(n_layers=1, vocab=50, embed=64, hidden=64, wdtype=wl.BF16, probe=wl.RADEMACHER)),
    ("bf16-gauss", dict(n_layers=1, vocab=50, embed=64, hidden=64, wdtype=wl.BF16, probe=wl.GAUSSIAN)),
]


@pytest.mark.parametrize("name,cfg", BADTOK, ids=[g[0] for g in BADTOK])
def test_out_of_range_tokens_poison_losses_and_skip_update(zo, oracle, name, cfg):
    """Token ids outside [0, V) are never read: an input id makes the
    sequence's states NaN from there on, a scored target id makes that
    position's loss NaN, so every loss is non-finite and the update skips
    with theta unchanged; an id used only as an unscored target changes
    nothing; the next call on valid tokens is unaffected."""
    V, B, Cn, N, eps, seed = cfg["vocab"], 3, 6, 2, 1e-2, 77
    rng = np.random.default_rng(5)
    tok = wl.uniform_tokens(rng, B, Cn, V)
    theta = zo.new_theta(cfg)
    zo.init(cfg, theta, 21)
    before = theta.clone()
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    for bad in (V, -1, 2 ** 31 - 1):
        for where in ("input", "target"):
            t = tok.copy()
            if where == "input":
                t[1, 2] = bad  # input at position 2, target of position 1 (scored)
            else:
                t[0, Cn] = bad  # target of the last position only
            say(f"{name}: token {bad} as {where}")
            td = torch.from_numpy(t).cuda()
            Lp, Lm = zo.perturbed_losses(cfg, theta, seed, eps, N, td, None, check_tokens=False)
            L, L0 = zo.fd_losses(cfg, theta, seed, eps, N, td, None, check_tokens=False)
            for x in (Lp, Lm, L, L0):
                assert not torch.isfinite(x).any().item(), (where, x)
            zo.update(cfg, theta, seed, eps, 1e-3, Lp, Lm, skipped=flag)
            assert flag.item() == 1
            assert torch.equal(theta.view(torch.int32), before.view(torch.int32))
    # an out-of-range id only at an unscored target position
    t = tok.copy()
    t[2, Cn] = V + 3
    mask = np.ones((B, Cn), np.uint8)
    mask[2, Cn - 1] = 0
    ok = t.copy()
    ok[2, Cn] = 0
    Lp, Lm = zo.perturbed_losses(cfg, theta, seed, eps, N, torch.from_numpy(t).cuda(),
                                 torch.from_numpy(mask).cuda(), check_tokens=False)
    ref_theta = oracle.init(cfg, 21)
    rp, rm = oracle.perturbed_losses(cfg, ref_theta, seed, eps, N, ok, mask, as_double=True)
    check(dict(Lp=Lp.cpu().numpy(), Lm=Lm.cpu().numpy()), dict(Lp=rp, Lm=rm), RTOL[cfg["wdtype"]])
    # valid tokens afterwards
    Lp, Lm = zo.perturbed_losses(cfg, theta, seed, eps, N, torch.from_numpy(tok).cuda(), None)
    rp, rm = oracle.perturbed_losses(cfg, ref_theta, seed, eps, N, tok, None, as_double=True)
    check(dict(Lp=Lp.cpu().numpy(), Lm=Lm.cpu().numpy()), dict(Lp=rp, Lm=rm), RTOL[cfg["wdtype"]])
