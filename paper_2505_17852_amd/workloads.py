"""Seeded synthetic workloads shaped like the paper's experiments.

This module only draws inputs (token batches, masks, seeds) and names the
model shapes; it holds none of the method's arithmetic. Both the GPU path's
tests/benchmark and the CPU oracle's checks take their inputs from here.

Workloads (model shape, batch, probes):
  c1  1-layer LSTM, V=256, E=32, H=64, fp32; B=4, C=32 i.i.d. uniform tokens;
      N=8 Rademacher, eps=1e-2, lr=1e-3.                       (parity smoke case)
  c2  2-layer, V=256, E=128, H=256, fp32; B=64, C=256 REVERSE transduction
      (64 payload tokens, a separator, the payload reversed; loss only on the
      reversed part); N=32 Rademacher, eps=lr=1e-3.      (Section 4.2 task shape)
  c3  3-layer, V=50,000, E=H=1024, bf16; B=256, C=1024 Zipf(1.1) tokens;
      N=64 Gaussian, eps=lr=1e-3.                        (language-model shape)
  c4  6-layer, V=50,000, E=H=4096 (~1.2B parameters), bf16; B=256, C=1024
      Zipf(1.1); N=16 Rademacher, eps=lr=1e-3.            (billion-parameter LM)
  c5  2-layer, V=256, E=32, H=512, fp32; one fixed batch B=32, C=128 uniform;
      N=1024 Gaussian, eps=lr=1e-2.                      (overfit-one-batch shape)
The paper trains on Penn Treebank for language modelling; that corpus is not
available here, so Zipf-distributed token ids stand in for it (c3, c4).
"""
from __future__ import annotations

import numpy as np

RADEMACHER = 0
GAUSSIAN = 1
FP32 = 0
BF16 = 1

CONFIGS = {
    "c1": dict(n_layers=1, vocab=256, embed=32, hidden=64, wdtype=FP32, probe=RADEMACHER,
               B=4, C=32, N=8, eps=1e-2, lr=1e-3, data="uniform"),
    "c2": dict(n_layers=2, vocab=256, embed=128, hidden=256, wdtype=FP32, probe=RADEMACHER,
               B=64, C=256, N=32, eps=1e-3, lr=1e-3, data="reverse"),
    "c3": dict(n_layers=3, vocab=50000, embed=1024, hidden=1024, wdtype=BF16, probe=GAUSSIAN,
               B=256, C=1024, N=64, eps=1e-3, lr=1e-3, data="zipf"),
    "c4": dict(n_layers=6, vocab=50000, embed=4096, hidden=4096, wdtype=BF16, probe=RADEMACHER,
               B=256, C=1024, N=16, eps=1e-3, lr=1e-3, data="zipf"),
    "c5": dict(n_layers=2, vocab=256, embed=32, hidden=512, wdtype=FP32, probe=GAUSSIAN,
               B=32, C=128, N=1024, eps=1e-2, lr=1e-2, data="uniform"),
}
CONFIG_ORDER = ["c1", "c2", "c3", "c4", "c5"]

ZIPF_S = 1.1
REVERSE_PAYLOAD = 64


def model_cfg(name_or_cfg, **override) -> dict:
    """The six model fields (n_layers, vocab, embed, hidden, wdtype, probe)."""
    c = dict(CONFIGS[name_or_cfg]) if isinstance(name_or_cfg, str) else dict(name_or_cfg)
    c.update(override)
    return {k: int(c[k]) for k in ("n_layers", "vocab", "embed", "hidden", "wdtype", "probe")}


def seeds(name: str) -> dict:
    k = CONFIG_ORDER.index(name) + 1
    return dict(data=1000 + k, init=2000 + k, step=3000 + k)


def uniform_tokens(rng: np.random.Generator, B: int, C: int, V: int) -> np.ndarray:
    return rng.integers(0, V, size=(B, C + 1), dtype=np.int64).astype(np.int32)


def zipf_tokens(rng: np.random.Generator, B: int, C: int, V: int, s: float = ZIPF_S) -> np.ndarray:
    """i.i.d. ids with P(k) proportional to (k+1)^-s over 0..V-1 (inverse CDF)."""
    p = np.arange(1, V + 1, dtype=np.float64) ** (-s)
    cdf = np.cumsum(p)
    cdf /= cdf[-1]
    u = rng.random(size=(B, C + 1))
    ids = np.searchsorted(cdf, u, side="right")
    return np.minimum(ids, V - 1).astype(np.int32)


def reverse_task(rng: np.random.Generator, B: int, C: int, V: int, payload: int = REVERSE_PAYLOAD):
    """REVERSE transduction rows: [payload, SEP, reversed payload] blocks,
    concatenated and cut to C+1 tokens. Payload ids are uniform over
    0..V-2, SEP = V-1. mask[b][t] = 1 iff the target token t+1 lies in a
    reversed segment."""
    blk = 2 * payload + 1
    nblk = (C + 1 + blk - 1) // blk
    toks = np.empty((B, nblk * blk), np.int32)
    pos_mask = np.zeros(nblk * blk, np.uint8)
    for k in range(nblk):
        pay = rng.integers(0, V - 1, size=(B, payload), dtype=np.int64).astype(np.int32)
        base = k * blk
        toks[:, base:base + payload] = pay
        toks[:, base + payload] = V - 1
        toks[:, base + payload + 1:base + blk] = pay[:, ::-1]
        pos_mask[base + payload + 1:base + blk] = 1
    toks = np.ascontiguousarray(toks[:, :C + 1])
    mask = np.ascontiguousarray(np.broadcast_to(pos_mask[1:C + 1], (B, C)).astype(np.uint8))
    return toks, mask


def reverse_task_varlen(rng: np.random.Generator, B: int, C: int, V: int, lmin: int = 1, lmax: int = 10):
    """REVERSE rows with random payload lengths, as the paper trains its
    transduction models (payloads of 1 to 10 random characters): each row is
    a run of [payload, SEP, payload reversed] blocks, every payload of its
    own length drawn uniformly from lmin..lmax and ids uniform over 0..V-2,
    cut to C+1 tokens. mask[b][t] = 1 iff target t+1 lies in a reversed
    part."""
    toks = np.empty((B, C + 1), np.int32)
    mask = np.zeros((B, C), np.uint8)
    for b in range(B):
        row, m = [], []
        while len(row) < C + 1:
            n = int(rng.integers(lmin, lmax + 1))
            pay = rng.integers(0, V - 1, size=n).tolist()
            row += pay + [V - 1] + pay[::-1]
            m += [0] * (n + 1) + [1] * n
        toks[b] = row[:C + 1]
        mask[b] = np.array(m[1:C + 1], np.uint8)
    return toks, mask


def batch(name: str, B: int | None = None, C: int | None = None, seed: int | None = None):
    """(tokens [B][C+1] int32, mask [B][C] uint8 or None) for workload `name`."""
    c = CONFIGS[name]
    B = c["B"] if B is None else B
    C = c["C"] if C is None else C
    rng = np.random.default_rng(seeds(name)["data"] if seed is None else seed)
    if c["data"] == "uniform":
        return uniform_tokens(rng, B, C, c["vocab"]), None
    if c["data"] == "zipf":
        return zipf_tokens(rng, B, C, c["vocab"]), None
    if c["data"] == "reverse":
        return reverse_task(rng, B, C, c["vocab"])
    raise ValueError(c["data"])


def param_count(cfg: dict) -> int:
    """Closed form of the flat parameter count (layout: EMB, per layer
    W_ih, W_hh, b, then W_out, b_out)."""
    L, V, E, H = cfg["n_layers"], cfg["vocab"], cfg["embed"], cfg["hidden"]
    return V * E + sum(4 * H * ((E if l == 0 else H) + H) + 4 * H for l in range(L)) + V * H + V


def gemm_params(cfg: dict) -> int:
    """Parameters that take part in matrix products per token: sum_l 4H(E_l+H) + V H."""
    L, V, E, H = cfg["n_layers"], cfg["vocab"], cfg["embed"], cfg["hidden"]
    return sum(4 * H * ((E if l == 0 else H) + H) for l in range(L)) + V * H
