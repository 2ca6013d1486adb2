"""Writes the oracle regression fixture of this directory. Calls only the
oracle (never the HIP library): python tests/golden/make_golden.py"""
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
    main()
