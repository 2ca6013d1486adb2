"""A step is a pure function of (theta, seed, eps, N, tokens) for the losses
and of (theta, seed, eps, lr, L+, L-) for the update, so work can be split,
lost, recomputed and replayed. Checked on the oracle (CPU):

- probe slices [i0, i0 + n) give bit for bit the losses of the same probes
  in the full set, so they concatenate to the full-N result;
- a worker's slice that is lost and recomputed by another worker leaves the
  final theta bit-identical;
- a checkpoint (theta, step index, base seed) resumes to the same theta, and
  replaying the per-step log (seed, L+, L-) through the update alone, without
  any forward pass, reconstructs theta from the initial weights."""
import numpy as np

from paper_2505_17852_amd import workloads as wl

CFG = dict(n_layers=2, vocab=24, embed=8, hidden=8, wdtype=0, probe=0)


def _batch(seed=3, B=3, C=6):
    return wl.uniform_tokens(np.random.default_rng(seed), B, C, CFG["vocab"])


def test_slices_concatenate_to_the_full_set(oracle):
    th = oracle.init(CFG, 5)
    tok = _batch()
    lp, lm = oracle.perturbed_losses(CFG, th, 77, 1e-2, 7, tok, as_double=True)
    parts = [(0, 3), (3, 2), (5, 2)]
    sp = np.concatenate([oracle.perturbed_losses(CFG, th, 77, 1e-2, n, tok, i0=i, as_double=True)[0] for i, n in parts])
    sm = np.concatenate([oracle.perturbed_losses(CFG, th, 77, 1e-2, n, tok, i0=i, as_double=True)[1] for i, n in parts])
    assert np.array_equal(sp, lp) and np.array_equal(sm, lm)


def test_lost_worker_slice_recomputed_elsewhere(oracle):
    """Three workers own probe slices of a 6-probe step; worker 1's losses are
    lost and worker 0 recomputes its slice. The update from the reassembled
    losses equals the one from an undisturbed run, bit for bit."""
    th = oracle.init(CFG, 6)
    tok = _batch(4)
    slices = {0: (0, 2), 1: (2, 2), 2: (4, 2)}
    got = {w: oracle.perturbed_losses(CFG, th, 88, 1e-2, n, tok, i0=i) for w, (i, n) in slices.items()}
    del got[1]  # worker 1 fails
    i, n = slices[1]
    got[1] = oracle.perturbed_losses(CFG, th, 88, 1e-2, n, tok, i0=i)  # recomputed by worker 0
    lp = np.concatenate([got[w][0] for w in range(3)])
    lm = np.concatenate([got[w][1] for w in range(3)])
    t_a = th.copy()
    assert oracle.update(CFG, t_a, 88, 1e-2, 1e-2, lp, lm) == 0
    ref_p, ref_m = oracle.perturbed_losses(CFG, th, 88, 1e-2, 6, tok)
    t_b = th.copy()
    assert oracle.update(CFG, t_b, 88, 1e-2, 1e-2, ref_p, ref_m) == 0
    assert np.array_equal(t_a, t_b)


def test_checkpoint_resume_and_log_replay(oracle):
    eps = lr = 1e-2
    N, steps, base = 4, 5, 900
    tok = _batch(5)
    th = oracle.init(CFG, 7)
    th0 = th.copy()
    log, ckpt = [], None
    for k in range(steps):
        lp, lm = oracle.perturbed_losses(CFG, th, base + k, eps, N, tok)
        log.append((base + k, lp.copy(), lm.copy()))
        assert oracle.update(CFG, th, base + k, eps, lr, lp, lm) == 0
        if k == 1:
            ckpt = (th.copy(), k + 1, base)
    # resume from the checkpoint
    t, k0, b = ckpt
    t = t.copy()
    for k in range(k0, steps):
        lp, lm = oracle.perturbed_losses(CFG, t, b + k, eps, N, tok)
        assert oracle.update(CFG, t, b + k, eps, lr, lp, lm) == 0
    assert np.array_equal(t, th)
    # replay the log through the update alone
    r = th0.copy()
    for seed, lp, lm in log:
        assert oracle.update(CFG, r, seed, eps, lr, lp, lm) == 0
    assert np.array_equal(r, th)
    assert not np.array_equal(th, th0)
