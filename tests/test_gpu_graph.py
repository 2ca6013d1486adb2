"""The step captured into a HIP graph (torch.cuda.CUDAGraph over the C ABI
calls on the capturing stream) and replayed: every replay, with eager work
and synchronisations in between, must give bit for bit what the same calls
give eagerly. The library allocates nothing and clears its workspace with
kernels, so a caller can capture a whole step."""
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


CASES = [
    ("fp32-rad", dict(n_layers=2, vocab=300, embed=64, hidden=96, wdtype=wl.FP32, probe=wl.RADEMACHER), 3, 5, 20, "cd"),
    ("bf16-gauss-cached", dict(n_layers=2, vocab=200, embed=128, hidden=64, wdtype=wl.BF16, probe=wl.GAUSSIAN),
     3, 3, 18, "cd"),
    ("bf16-rad-fd", dict(n_layers=2, vocab=300, embed=64, hidden=128, wdtype=wl.BF16, probe=wl.RADEMACHER),
     2, 5, 20, "fd"),
]


def _bits(x):
    return x.view(torch.int32) if x.dtype == torch.float32 else x.view(torch.int16)


@pytest.mark.parametrize("name,cfg,N,B,C,est", CASES, ids=[c[0] for c in CASES])
def test_captured_step_replays_like_eager(zo, name, cfg, N, B, C, est):
    say(f"graph {name} N={N} B={B} C={C} {est}")
    rng = np.random.default_rng(3)
    tok = torch.from_numpy(wl.uniform_tokens(rng, B, C, cfg["vocab"])).cuda()
    mask = torch.from_numpy((rng.random((B, C)) < 0.7).astype(np.uint8)).cuda()
    seed, eps, lr = 4321, 1e-2, 1e-2
    th_g = zo.new_theta(cfg)
    zo.init(cfg, th_g, 17)
    th_e = th_g.clone()
    fd = est == "fd"

    def buffers():
        ws = zo.new_workspace(cfg, N, B, C)
        L1 = torch.empty(N, dtype=torch.float32, device="cuda")
        L2 = torch.empty(1 if fd else N, dtype=torch.float32, device="cuda")
        return ws, L1, L2

    def step(theta, ws, L1, L2, stream=None):
        if fd:
            zo.fd_losses(cfg, theta, seed, eps, N, tok, mask, L=L1, L0=L2, workspace=ws, stream=stream,
                         check_tokens=False)
            zo.fd_update(cfg, theta, seed, eps, lr, L1, L2, stream=stream)
        else:
            zo.perturbed_losses(cfg, theta, seed, eps, N, tok, mask, Lplus=L1, Lminus=L2, workspace=ws,
                                stream=stream, check_tokens=False)
            zo.update(cfg, theta, seed, eps, lr, L1, L2, stream=stream)

    ws_g, L1_g, L2_g = buffers()
    ws_e, L1_e, L2_e = buffers()
    # warm up on a side stream (the library's host-side set-up happens outside the capture)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        scratch = th_g.clone()
        step(scratch, ws_g, L1_g, L2_g, stream=side)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    del scratch

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(th_g, ws_g, L1_g, L2_g, stream=torch.cuda.current_stream())
    torch.cuda.synchronize()

    junk = torch.randn(1 << 20, device="cuda")
    for r in range(3):
        g.replay()
        torch.cuda.synchronize()
        # eager work between replays, on the same device
        junk.mul_(1.0001).add_(0.5)
        step(th_e, ws_e, L1_e, L2_e)
        torch.cuda.synchronize()
        say(f"replay {r}: L1 {L1_g[:2].tolist()} eager {L1_e[:2].tolist()}")
        assert torch.equal(_bits(L1_g), _bits(L1_e)), f"replay {r}: losses differ"
        assert torch.equal(_bits(L2_g), _bits(L2_e)), f"replay {r}: losses differ"
        assert torch.equal(_bits(th_g), _bits(th_e)), f"replay {r}: theta differs"
        # no call may depend on what an earlier call left in its workspace
        ws_e.fill_(0xAB)
        ws_g.fill_(0xCD)
        torch.cuda.synchronize()
