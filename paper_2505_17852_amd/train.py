"""Multi-step zeroth-order training on one GPU.

The host loop of the paper's training algorithm (Algorithm 1) with either
estimator of Section 2:

* "cd" (default): central differences. Every step runs the 2N perturbed
  forward passes of one batch (`zo_perturbed_losses`) and the update
  (`zo_update`). The loss reported per step is the mean over probes of
  (L⁺ + L⁻)/2, which is L(θ) + O(ε²) for smooth losses (the central
  difference's even part), so a training curve costs no extra pass.
* "fd": forward differences (Eq. 1). Every step runs N perturbed passes and
  one clean pass (`zo_fd_losses`) and the update (`zo_fd_update`); the
  reported loss is the clean pass's L(θ).

The step's probes are drawn from the seed `seed0 + k`. Argument marshalling
only: the forwards and the update run in the library's HIP kernels, and θ
stays on the device for the whole run.
"""
from __future__ import annotations

import contextlib

import torch

from . import zo

ESTIMATORS = ("cd", "fd")


def train(cfg, theta: torch.Tensor, tokens: torch.Tensor, mask: torch.Tensor | None, *, N: int,
          eps: float, lr: float, steps: int, seed0: int, batches=None, stream=None,
          estimator: str = "cd") -> torch.Tensor:
    """Runs `steps` zeroth-order steps in place on theta and returns the
    per-step loss estimates (a CPU fp32 tensor of `steps` values).

    tokens/mask: the batch used every step (the overfit setting), or the
    first batch when `batches(k) -> (tokens, mask)` supplies step k's batch
    (all of the same shape). A step whose losses are not finite leaves theta
    unchanged (the update's own rule) and reports its NaN/inf estimate."""
    if steps < 1:
        raise ValueError("steps must be >= 1")
    if estimator not in ESTIMATORS:
        raise ValueError(f"estimator must be one of {ESTIMATORS}")
    fd = estimator == "fd"
    B, C1 = tokens.shape
    dev = theta.device
    ws = zo.new_workspace(cfg, N, B, C1 - 1, device=dev)
    L1 = torch.empty(N, dtype=torch.float32, device=dev)
    L2 = torch.empty(1 if fd else N, dtype=torch.float32, device=dev)
    hist = torch.empty(steps, dtype=torch.float32, device=dev)
    # the loss bookkeeping runs on the same stream as the library calls
    ctx = torch.cuda.stream(stream) if stream is not None else contextlib.nullcontext()
    with ctx:
        for k in range(steps):
            tok, msk = (tokens, mask) if batches is None or k == 0 else batches(k)
            check = k == 0 or batches is not None
            # step k's estimate: losses at theta before its update
            if fd:
                zo.fd_losses(cfg, theta, seed0 + k, eps, N, tok, msk, L=L1, L0=L2, workspace=ws,
                             check_tokens=check)
                hist[k] = L2[0]
                zo.fd_update(cfg, theta, seed0 + k, eps, lr, L1, L2)
            else:
                zo.perturbed_losses(cfg, theta, seed0 + k, eps, N, tok, msk, Lplus=L1, Lminus=L2,
                                    workspace=ws, check_tokens=check)
                hist[k] = 0.5 * (L1.mean() + L2.mean())
                zo.update(cfg, theta, seed0 + k, eps, lr, L1, L2)
        return hist.cpu()
