"""Writes the oracle fixtures of this directory. Calls only the oracle (never
the HIP library):
    python tests/golden/make_golden.py          oracle_losses.txt (small cases)
    python tests/golden/make_golden.py --wide   oracle_losses_wide.txt (the
        billion-parameter and 1024-wide layer shapes at several eps; minutes)"""
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

from oracle import build as ob  # noqa: E402
from paper_2505_17852_amd import workloads as wl  # noqa: E402

CASES = [
    # name, model cfg, init seed, step seed, eps, N, B, C, token seed
    ("c1-rad", dict(n_layers=1, vocab=256, embed=32, hidden=64, wdtype=0, probe=0), 2001, 3001, 1e-2, 4, 2, 8, 11),
    ("gauss-2layer", dict(n_layers=2, vocab=50, embed=32, hidden=32, wdtype=0, probe=1), 2002, 3002, 1e-2, 3, 3, 5, 12),
    ("bf16-rad", dict(n_layers=1, vocab=40, embed=64, hidden=64, wdtype=1, probe=0), 2003, 3003, 1e-3, 2, 2, 4, 13),
]


# The estimator's signal at the real layer widths: the workload's model, init
# and step seeds and a short batch of its token distribution, at several eps.
# name, workload, probe override, N, B, C, eps values
WIDE_CASES = [
    ("c4", "c4", None, 4, 2, 4, (1e-3, 1e-4, 1e-5)),
    ("c3", "c3", None, 8, 2, 4, (1e-3, 3e-4, 1e-4, 3e-5, 1e-5)),
    ("c3-rad", "c3", 0, 8, 2, 4, (1e-3, 1e-4, 1e-5)),
]


def wide_key(name, eps):
    return f"{name}@{eps:g}"


def wide_inputs(name, workload, probe, B, C):
    cfg = wl.model_cfg(workload) if probe is None else wl.model_cfg(workload, probe=probe)
    tok, _ = wl.batch(workload, B=B, C=C)
    return cfg, wl.seeds(workload), tok


def main_wide():
    ob.build()
    from oracle import oracle
    lines = ["# Oracle losses at the real layer widths (written by make_golden.py --wide from the oracle only).",
             "# name@eps | L+ (N, fp64) | L- (N, fp64); repr() of each double"]
    for name, workload, probe, N, B, C, epss in WIDE_CASES:
        cfg, sd, tok = wide_inputs(name, workload, probe, B, C)
        theta = oracle.init(cfg, sd["init"])
        for eps in epss:
            lp, lm = oracle.perturbed_losses(cfg, theta, sd["step"], eps, N, tok, as_double=True)
            lines.append(" | ".join([wide_key(name, eps), " ".join(repr(float(x)) for x in lp),
                                     " ".join(repr(float(x)) for x in lm)]))
            print(lines[-1], flush=True)
        del theta
    with open(os.path.join(HERE, "oracle_losses_wide.txt"), "w") as f:
        f.write("\n".join(lines) + "\n")


def main():
    ob.build()
    from oracle import oracle
    lines = ["# Oracle regression values (written by make_golden.py from the oracle only).",
             "# name | L+ (N, fp64) | L- (N, fp64) | L0 clean loss (fp64); repr() of each double"]
    for name, cfg, si, ss, eps, N, B, C, ts in CASES:
        theta = oracle.init(cfg, si)
        tok = wl.uniform_tokens(np.random.default_rng(ts), B, C, cfg["vocab"])
        lp, lm = oracle.perturbed_losses(cfg, theta, ss, eps, N, tok, as_double=True)
        _, l0 = oracle.fd_losses(cfg, theta, ss, eps, N, tok)
        lines.append(" | ".join([name, " ".join(repr(float(x)) for x in lp), " ".join(repr(float(x)) for x in lm),
                                 repr(float(l0))]))
    with open(os.path.join(HERE, "oracle_losses.txt"), "w") as f:
        f.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    main_wide() if "--wide" in sys.argv else main()
