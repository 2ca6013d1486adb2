"""Multi-step CD-RGE training on one GPU.

The host loop of the paper's training algorithm (Algorithm 1): every step
runs the 2N perturbed forward passes of one batch (`zo_perturbed_losses`)
and the update (`zo_update`), with the step's probes drawn from the seed
`seed0 + k`. Argument marshalling only: the forwards and the update run in
the library's HIP kernels, and θ stays on the device for the whole run.

The loss reported per step is the mean over probes of (L⁺ + L⁻)/2, which is
L(θ) + O(ε²) for smooth losses (the central difference's even part), so a
training curve costs no extra forward pass.
"""
from __future__ import annotations

import contextlib

import torch

from . import zo


def train(cfg, theta: torch.Tensor, tokens: torch.Tensor, mask: torch.Tensor | None, *, N: int,
          eps: float, lr: float, steps: int, seed0: int, batches=None, stream=None) -> torch.Tensor:
    """Runs `steps` CD-RGE steps in place on theta and returns the per-step
    loss estimates (a CPU fp32 tensor of `steps` values).

    tokens/mask: the batch used every step (the overfit setting), or the
    first batch when `batches(k) -> (tokens, mask)` supplies step k's batch
    (all of the same shape). A step whose losses are not finite leaves theta
    unchanged (the update's own rule) and reports its NaN/inf estimate."""
    if steps < 1:
        raise ValueError("steps must be >= 1")
    B, C1 = tokens.shape
    dev = theta.device
    ws = zo.new_workspace(cfg, N, B, C1 - 1, device=dev)
    Lp = torch.empty(N, dtype=torch.float32, device=dev)
    Lm = torch.empty(N, dtype=torch.float32, device=dev)
    hist = torch.empty(steps, dtype=torch.float32, device=dev)
    # the loss bookkeeping runs on the same stream as the library calls
    ctx = torch.cuda.stream(stream) if stream is not None else contextlib.nullcontext()
    with ctx:
        for k in range(steps):
            tok, msk = (tokens, mask) if batches is None or k == 0 else batches(k)
            zo.perturbed_losses(cfg, theta, seed0 + k, eps, N, tok, msk, Lplus=Lp, Lminus=Lm,
                                workspace=ws, check_tokens=(k == 0 or batches is not None))
            # step k's estimate: losses at theta before its update
            hist[k] = 0.5 * (Lp.mean() + Lm.mean())
            zo.update(cfg, theta, seed0 + k, eps, lr, Lp, Lm)
        return hist.cpu()
