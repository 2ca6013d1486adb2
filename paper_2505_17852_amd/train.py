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

As a program it trains one of the seeded workloads and prints its curve,
one JSON line per evaluation:
    python -m paper_2505_17852_amd.train --workload c2 --steps 10000 \
        --eps 3e-2 --lr 3e-2 --fresh-batches --eval-every 1000
Each line holds the mean per-step estimate over the last window and the
clean loss L(θ) (the clean pass of a forward-difference call) on the
training batch and, with --fresh-batches, on a held-out batch of the same
shape.
"""
from __future__ import annotations

import argparse
import contextlib
import json
import sys
import time

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


def clean_loss(cfg, theta: torch.Tensor, tokens: torch.Tensor, mask: torch.Tensor | None) -> float:
    """L(θ) on one batch: the clean pass of zo_fd_losses (with one probe,
    whose perturbed pass is ignored)."""
    _, L0 = zo.fd_losses(cfg, theta, 0, 1e-3, 1, tokens, mask)
    return float(L0.item())


def main(argv=None):
    import numpy as np

    from . import workloads as wl
    ap = argparse.ArgumentParser(description="zeroth-order training of a seeded workload on one GPU")
    ap.add_argument("--workload", default="c2", choices=sorted(wl.CONFIGS))
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--eps", type=float, default=None, help="perturbation size (default: the workload's)")
    ap.add_argument("--lr", type=float, default=None, help="step size (default: the workload's)")
    ap.add_argument("--estimator", default="cd", choices=ESTIMATORS)
    ap.add_argument("--fresh-batches", action="store_true",
                    help="draw a new batch of the workload's distribution every step (seed data + 1 + k) "
                         "and evaluate on a held-out batch; default: one fixed batch")
    ap.add_argument("--eval-every", type=int, default=500)
    ap.add_argument("--reverse-lengths", default=None,
                    help="c2 only: REVERSE payloads of random lengths LO:HI (the paper trains on 1:10) "
                         "instead of the workload's fixed 64")
    args = ap.parse_args(argv)
    name = args.workload
    w, cfg, sd = wl.CONFIGS[name], wl.model_cfg(name), wl.seeds(name)
    eps = w["eps"] if args.eps is None else args.eps
    lr = w["lr"] if args.lr is None else args.lr
    dev = torch.device("cuda:0")

    if args.reverse_lengths and name != "c2":
        raise SystemExit("--reverse-lengths applies to the c2 workload only")

    def host_batch(seed):
        if not args.reverse_lengths:
            return wl.batch(name, seed=seed)
        lo, hi = (int(x) for x in args.reverse_lengths.split(":"))
        rng = np.random.default_rng(sd["data"] if seed is None else seed)
        return wl.reverse_task_varlen(rng, w["B"], w["C"], cfg["vocab"], lo, hi)

    def dev_batch(seed=None):
        tok, mask = host_batch(seed)
        return (torch.from_numpy(tok).to(dev), None if mask is None else torch.from_numpy(mask).to(dev))

    tokens, mask = dev_batch()
    held = dev_batch(seed=sd["data"] + 10_000_000) if args.fresh_batches else None
    batches = (lambda k: dev_batch(seed=sd["data"] + 1 + k)) if args.fresh_batches else None
    theta = zo.new_theta(cfg, dev)
    zo.init(cfg, theta, sd["init"])
    t0 = time.time()

    def report(step, window):
        row = {"workload": name, "reverse_lengths": args.reverse_lengths, "step": step, "eps": eps, "lr": lr,
               "estimator": args.estimator,
               "N": w["N"], "fresh_batches": args.fresh_batches,
               "window_estimate": None if window is None else float(np.mean(window)),
               "clean_loss_train_batch": clean_loss(cfg, theta, tokens, mask),
               "seconds": round(time.time() - t0, 1)}
        if held is not None:
            row["clean_loss_held_out"] = clean_loss(cfg, theta, *held)
        print(json.dumps(row), flush=True)

    report(0, None)
    done = 0
    while done < args.steps:
        n = min(args.eval_every, args.steps - done)
        first = (tokens, mask) if batches is None else batches(done)
        shifted = None if batches is None else (lambda k, d=done: batches(d + k))
        hist = train(cfg, theta, first[0], first[1], N=w["N"], eps=eps, lr=lr, steps=n,
                     seed0=sd["step"] + done, batches=shifted, estimator=args.estimator)
        done += n
        report(done, hist.numpy())
    return 0


if __name__ == "__main__":
    sys.exit(main())
