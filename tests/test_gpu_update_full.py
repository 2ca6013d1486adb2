"""The update (Eq. 7; Algorithm 1's closing loop) at the workloads' real
parameter counts, against the CPU oracle, through the C ABI.

The sign-probe update kernels are persistent: a grid of a few workgroups per
compute unit walks the parameter tiles (8192 parameters each), so at these
sizes every workgroup handles hundreds of tiles and reuses its LDS tables,
rows and prefetched theta across them. Each test takes theta from a real
zo_perturbed_losses + zo_update call at the workload's shape and compares the
updated theta with the oracle (oracle.update_sampled: theta_j minus the sum
of c_n z_n[j] in double, one rounding) at sampled indices: whole tiles at the
start, around multiples of 256 tiles (the tiles a workgroup reaches on its
second and later iterations for any grid of k x 256 workgroups), in the
middle, around 2^30 and at the end (the last tile ragged); the first and
last elements of every tensor of the layout; and 10^4 indices drawn
uniformly. The c2 update (N = 32, the sign-probe kernel for any N) is
compared in full. Where the forward call kept a sign-probe cache (bf16
weights, sign probes), the update reading it (zo_update_cached) must give
the same theta bit for bit.

Bars: bf16 theta within one bf16 ulp of the oracle (the GPU sums the probe
terms in fp32, the oracle in double, before the one rounding) plus 2^-16 of
the mean |theta| (where the step nearly cancels theta_j, the fp32 sum's own
rounding decides the few bits left); fp32 theta within 1e-5 relative plus
1e-5 of the mean |theta|. With bf16 weights the
workload's step (lr = 1e-3) moves most parameters by less than half a bf16
ulp, so those cases use lr x 64, which moves most of them by several ulps.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

from paper_2505_17852_amd import workloads as wl  # noqa: E402

TILE = 8192  # parameters per tile of the sign-probe update kernels


@pytest.fixture(scope="module")
def zo():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2505_17852_amd import zo as z
    z.lib()
    return z


def say(*a):
    print(*a, flush=True)


def as_host(theta, cfg):
    return theta.view(torch.int16 if cfg["wdtype"] == wl.BF16 else torch.int32).cpu().numpy().view(
        np.uint16 if cfg["wdtype"] == wl.BF16 else np.float32)


def as_f64(x, cfg):
    if cfg["wdtype"] == wl.BF16:
        return (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return x.astype(np.float64)


def close(got, ref, cfg, before):
    """Elementwise bar; returns the indices (into got) that fail it. before:
    theta before the update (its mean |theta| sets the absolute floor)."""
    g, r = as_f64(got, cfg), as_f64(ref, cfg)
    mean_abs = np.abs(as_f64(before, cfg)).mean()
    if cfg["wdtype"] == wl.BF16:
        return np.nonzero(np.abs(g - r) > np.abs(r) * 2.0 ** -7 + 2.0 ** -16 * mean_abs)[0]
    return np.nonzero(np.abs(g - r) > 1e-5 * np.abs(r) + 1e-5 * mean_abs)[0]


def sample_indices(zo, cfg, whole_tiles: bool, n_random=10_000, seed=0):
    P = zo.param_count(cfg)
    ntiles = (P + TILE - 1) // TILE
    tiles = {0, 1, 2, ntiles // 2, ntiles - 2, ntiles - 1}
    if whole_tiles:
        for k in (1, 2, 4, 8, 16, 32, 64):
            tiles |= {256 * k - 1, 256 * k, 256 * k + 1}
        if P > (1 << 30):
            tiles |= {(1 << 30) // TILE - 1, (1 << 30) // TILE}
    parts = [np.arange(t * TILE, min(P, (t + 1) * TILE), dtype=np.uint64)
             for t in sorted(tiles) if 0 <= t < ntiles]
    if not whole_tiles:  # a few elements of those tiles only
        parts = [p[[0, 1, 7, 8, p.size // 2, p.size - 2, p.size - 1]] if p.size > 8 else p for p in parts]
    # first and last elements of every tensor of the layout
    L, V, E, H = cfg["n_layers"], cfg["vocab"], cfg["embed"], cfg["hidden"]
    starts, p = [0], V * E
    for l in range(L):
        El = E if l == 0 else H
        for n in (4 * H * El, 4 * H * H, 4 * H):
            starts.append(p)
            p += n
    starts += [p, p + V * H, P]
    edges = [s + d for s in starts for d in (-2, -1, 0, 1) if 0 <= s + d < P]
    if P > (1 << 30):
        edges += [(1 << 30) + d for d in (-3, -1, 0, 1, 5)]
    rng = np.random.default_rng(seed)
    rand = rng.integers(0, P, size=n_random, dtype=np.uint64)
    idx = np.unique(np.concatenate(parts + [np.array(edges, np.uint64), rand]))
    assert idx.max() < P
    return idx


def run_step(zo, name, cfg, N, C=None):
    """theta after init, real losses at the workload's batch shape (C
    positions), and the losses as host arrays."""
    w = wl.CONFIGS[name]
    sd = wl.seeds(name)
    tok, mask = wl.batch(name, C=C)
    theta = zo.new_theta(cfg)
    zo.init(cfg, theta, sd["init"])
    td = torch.from_numpy(tok).cuda()
    md = None if mask is None else torch.from_numpy(mask).cuda()
    ws = zo.new_workspace(cfg, N, tok.shape[0], tok.shape[1] - 1)
    Lp, Lm = zo.perturbed_losses(cfg, theta, sd["step"], w["eps"], N, td, md, workspace=ws)
    torch.cuda.synchronize()
    # the sign-probe cache of this call (bf16 weights, sign probes), kept for zo_update_cached
    pb = zo.probe_bits(cfg, N, tok.shape[0], tok.shape[1] - 1, ws)
    pb = None if pb is None else pb.clone()
    del ws
    torch.cuda.empty_cache()
    lp, lm = Lp.cpu().numpy(), Lm.cpu().numpy()
    assert np.all(np.isfinite(lp)) and np.all(np.isfinite(lm))
    assert np.any(lp != lm)
    return theta, Lp, Lm, lp, lm, pb


# name, workload, probe override, N, C (the update does not depend on C; the
# long-sequence workloads use a short batch of the full width to save time),
# whether whole tiles are sampled (sign probes: the persistent tile walk)
FULL = [
    ("c4-rad16", "c4", None, 16, 16, True),        # N <= 16 sign-probe kernel, bf16, P = 1.2e9
    ("c3-gauss", "c3", None, 64, 16, False),       # normal probes, bf16, P = 1.3e8
    ("c3-rad20", "c3", wl.RADEMACHER, 20, 16, True),  # the sign-probe kernel for any N, bf16
    ("c5-gauss", "c5", None, 1024, None, False),   # normal probes, fp32, N = 1024
]


@pytest.mark.parametrize("case,name,probe,N,C,whole", FULL, ids=[f[0] for f in FULL])
def test_update_full_size_sampled(zo, oracle, case, name, probe, N, C, whole):
    w = wl.CONFIGS[name]
    sd = wl.seeds(name)
    cfg = wl.model_cfg(name) if probe is None else wl.model_cfg(name, probe=probe)
    P = zo.param_count(cfg)
    say(f"full-size update {case}: P={P} N={N} C={C}")
    theta, Lp, Lm, lp, lm, bits = run_step(zo, name, cfg, N, C)
    before = as_host(theta, cfg)
    skipped = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    lr = w["lr"] * (64 if cfg["wdtype"] == wl.BF16 else 1)
    zo.update(cfg, theta, sd["step"], w["eps"], lr, Lp, Lm, skipped=skipped)
    torch.cuda.synchronize()
    assert skipped.item() == 0
    idx = sample_indices(zo, cfg, whole)
    after = as_host(theta, cfg)
    del theta
    torch.cuda.empty_cache()
    got = after[idx]
    say(f"{idx.size} sampled indices; oracle update at them")
    ref = oracle.update_sampled(cfg, before, sd["step"], w["eps"], lr, lp, lm, idx)
    bad = close(got, ref, cfg, before[idx])
    if bad.size:
        k = bad[:8]
        raise AssertionError(f"{case}: {bad.size} of {idx.size} differ; at {idx[k].tolist()}: "
                             f"gpu {got[k].tolist()} oracle {ref[k].tolist()} before {before[idx[k]].tolist()}")
    moved = np.count_nonzero(got != before[idx])
    say(f"{case}: all {idx.size} within the bar; {moved} changed")
    assert moved > idx.size // 2
    if bits is not None:
        # the same update reading the call's sign-probe cache: theta bit for bit
        theta2 = torch.from_numpy(before.view(np.int16)).cuda()
        zo.update_cached(cfg, theta2.view(torch.bfloat16), sd["step"], w["eps"], lr, Lp, Lm, bits)
        assert np.array_equal(theta2.cpu().numpy().view(np.uint16), after)


def test_update_c2_full(zo, oracle):
    """c2: P = 1.0e6, N = 32 sign probes (the kernel for any N), compared at
    every parameter with the oracle's full update."""
    name = "c2"
    w = wl.CONFIGS[name]
    sd = wl.seeds(name)
    cfg = wl.model_cfg(name)
    theta, Lp, Lm, lp, lm, _ = run_step(zo, name, cfg, w["N"])
    ref = as_host(theta, cfg).copy()
    before = ref.copy()
    zo.update(cfg, theta, sd["step"], w["eps"], w["lr"], Lp, Lm)
    got = as_host(theta, cfg)
    assert oracle.update(cfg, ref, sd["step"], w["eps"], w["lr"], lp, lm) == 0
    bad = close(got, ref, cfg, before)
    assert bad.size == 0, f"{bad.size} differ, first {bad[:5].tolist()}"
