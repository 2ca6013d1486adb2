"""The allocation-free entry point zo_perturbed_losses_noalloc (the library's
fixed device scratch as the workspace) against zo_perturbed_losses with a
caller workspace, through the C ABI: the same kernels on the same inputs, so
the losses must be bit-identical. Calls follow one another on one device and
share the scratch; a later, smaller call must not see the earlier call's
contents."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

from paper_2505_17852_amd import workloads as wl  # noqa: E402


@pytest.fixture(scope="module")
def zo():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2505_17852_amd import zo as z
    z.lib()
    return z


def say(*a):
    print(*a, flush=True)


def both(zo, cfg, N, B, C, seed, eps, masked, i0=0):
    rng = np.random.default_rng(seed)
    if cfg == wl.model_cfg("c2") and B == 64:
        tok, mask = wl.batch("c2")
    else:
        tok = wl.uniform_tokens(rng, B, C, cfg["vocab"])
        mask = (rng.random((B, C)) < 0.7).astype(np.uint8) if masked else None
    theta = zo.new_theta(cfg)
    zo.init(cfg, theta, seed)
    td = torch.from_numpy(tok).cuda()
    md = None if mask is None else torch.from_numpy(mask).cuda()
    say(f"noalloc {cfg} N={N} B={B} C={C} workspace {zo.workspace_bytes_min(cfg, N, B, C)} bytes")
    Lp = torch.full((N,), float("nan"), device="cuda")
    Lm = torch.full((N,), float("nan"), device="cuda")
    zo.perturbed_losses_noalloc(cfg, theta, seed + 1, eps, N, td, md, Lp, Lm, i0=i0)
    rp, rm = zo.perturbed_losses(cfg, theta, seed + 1, eps, N, td, md, i0=i0)
    torch.cuda.synchronize()
    assert torch.equal(Lp.view(torch.int32), rp.view(torch.int32)), (Lp, rp)
    assert torch.equal(Lm.view(torch.int32), rm.view(torch.int32)), (Lm, rm)
    return Lp


SEQUENCE = [
    # the whole c2 workload (113.6 MiB of the 128 MiB scratch), then smaller calls
    ("c2-full", wl.model_cfg("c2"), 32, 64, 256, 1e-3, True),
    ("ragged-fp32", dict(n_layers=2, vocab=300, embed=64, hidden=96, wdtype=wl.FP32, probe=wl.RADEMACHER),
     3, 5, 20, 1e-2, True),
    ("bf16-gauss-cached", dict(n_layers=2, vocab=300, embed=64, hidden=128, wdtype=wl.BF16, probe=wl.GAUSSIAN),
     2, 3, 9, 1e-2, False),
    ("c1", wl.model_cfg("c1"), 8, 4, 32, 1e-2, False),
    ("c1-smaller", wl.model_cfg("c1"), 2, 2, 5, 1e-2, True),
]


def test_noalloc_matches_workspace_path_in_sequence(zo):
    for k, (name, cfg, N, B, C, eps, masked) in enumerate(SEQUENCE):
        L = both(zo, cfg, N, B, C, 40 + k, eps, masked, i0=k)
        assert torch.all(torch.isfinite(L)), name


def test_noalloc_twice_second_smaller(zo):
    """Two calls in a row, the second with a smaller input (fewer probes,
    sequences and positions), each bit-identical to the workspace path."""
    cfg = dict(n_layers=2, vocab=200, embed=64, hidden=64, wdtype=wl.FP32, probe=wl.GAUSSIAN)
    both(zo, cfg, 6, 40, 30, 7, 1e-2, True)
    both(zo, cfg, 2, 3, 4, 8, 1e-2, False)


def test_noalloc_rejects_shapes_beyond_the_scratch(zo):
    """A shape whose workspace exceeds the fixed scratch is ZO_ENOMEM, and the
    output buffers are left untouched."""
    cfg = wl.model_cfg("c1")
    N, B, C = 64, 512, 64
    assert zo.workspace_bytes_min(cfg, N, B, C) > zo.NOALLOC_WORKSPACE_BYTES
    theta = zo.new_theta(cfg)
    zo.init(cfg, theta, 1)
    tok = torch.zeros((B, C + 1), dtype=torch.int32, device="cuda")
    Lp = torch.full((N,), 7.0, device="cuda")
    Lm = torch.full((N,), 7.0, device="cuda")
    with pytest.raises(zo.ZoError) as e:
        zo.perturbed_losses_noalloc(cfg, theta, 1, 1e-3, N, tok, None, Lp, Lm)
    assert e.value.status == zo.ZO_ENOMEM
    torch.cuda.synchronize()
    assert torch.all(Lp == 7.0) and torch.all(Lm == 7.0)
