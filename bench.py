#!/usr/bin/env python3
"""Throughput of one CD-RGE training step on one MI355X.

A step is the whole hot path: the 2N perturbed forward passes of the
stacked-LSTM language model over one batch (zo_perturbed_losses) and the
parameter update (zo_update), with inputs already resident in device memory.
Prints one JSON line: perturbed-forward tokens per second (2N*B*C / step
time), the roofline position of the dominant kernel (the fused gate kernel,
timed live with HIP events over the timed region) and the CPU oracle timed on
a bounded sample of the same workload.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c4] [--estimator cd]
(default workload c4, the 1.2B-parameter model; c2 is the fp32 transduction shape;
--estimator fd times the forward-difference step instead: N + 1 passes,
zo_fd_losses and zo_fd_update)
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "perturbed-forward tokens/sec per CD-RGE step (2N·B·C/s); % MFMA peak"
METRIC_FD = "forward tokens/sec per FD-RGE step ((N+1)·B·C/s); % MFMA peak"
PEAK_TFLOPS = {"f32": 157.3, "bf16": 2500.0, "fp16": 2500.0}  # dense MFMA peaks of MI355X
HBM_PEAK_GBPS = 8000.0  # HBM3E peak of MI355X
DEFAULTS = {"c1": (3, 20), "c2": (3, 20), "c3": (1, 3), "c4": (1, 3), "c5": (1, 3)}
# Event timing: every launch where kernels are long (an event pair adds a few µs to the
# stream: 0.2% of the c4 step, less for c5's 5 ms launches), every 61st launch of each class where they are short (c2:
# every launch would add ~22% to the step). 61 is prime, so the sample cycles through the
# layers and timesteps.
PROF_EVERY = {"c3": 1, "c4": 1, "c5": 1}
PROF_EVERY_SHORT = 61
DESCRIPTION = {
    "c1": "1-layer LSTM V=256 E=32 H=64 fp32; B=4 C=32 uniform tokens; N=8 Rademacher",
    "c2": "2-layer LSTM V=256 E=128 H=256 fp32; B=64 C=256 REVERSE transduction (loss on "
          "reversed half); N=32 Rademacher, eps=lr=1e-3",
    "c3": "3-layer LSTM V=50000 E=H=1024 bf16; B=256 C=1024 Zipf(1.1); N=64 Gaussian",
    "c4": "6-layer LSTM V=50000 E=H=4096 bf16 (~1.2B params); B=256 C=1024 Zipf(1.1); "
          "N=16 Rademacher",
    "c5": "2-layer LSTM V=256 E=32 H=512 fp32; fixed batch B=32 C=128 uniform; N=1024 Gaussian",
}


def gate_flops(cfg, passes, B):
    """Algorithmic flops of all gate products of one timestep (every layer):
    2 * (passes * B rows) * 4H * (E_l + H) per layer (2N passes for central
    differences, N + 1 for forward differences)."""
    L, E, H = cfg["n_layers"], cfg["embed"], cfg["hidden"]
    rows = passes * B
    return sum(2 * rows * 4 * H * ((E if l == 0 else H) + H) for l in range(L))


def kernel_source_hash(dtype):
    """Hash of the gate kernel's sources, to match the committed counter runs."""
    import hashlib
    src = os.path.join(ROOT, "paper_2505_17852_amd", "csrc")
    files = (["k_forward_bf16.hip", "zo_pack.hpp"] if dtype == "bf16" else ["k_forward.hip"]) + ["zo_rng.hpp", "zo_common.hpp"]
    m = hashlib.sha256()
    for f in files:
        with open(os.path.join(src, f), "rb") as fh:
            m.update(fh.read())
    return m.hexdigest()[:16]


def measured_traffic(name, dtype):
    """HBM bytes (read + write) per gate layer-step from the committed
    rocprofv3 FETCH_SIZE / WRITE_SIZE runs, if they were taken on the current
    kernel sources; None otherwise."""
    path = os.path.join(ROOT, "profiles", "gate_traffic_c4_c2.md")
    if not os.path.exists(path):
        return None
    want = kernel_source_hash(dtype)
    with open(path) as fh:
        for line in fh:
            parts = line.split()
            if len(parts) == 5 and parts[0] == "traffic" and parts[1] == name and parts[2] == want:
                return float(parts[3]) + float(parts[4])
    return None


def library_gemm(name):
    """torch's fp16 GEMM (hipBLASLt) of the bf16 gate's plain product at the
    workload's shape: rows 2 N B (one layer-step of every pass) by K = 2 H
    (the layers above the first; the first has E + H) against the [4H][K]
    weight matrix, as
    torch.nn.functional.linear computes it. Context for the fused gate, which
    also forms fp16(W + s eps z) per fragment and runs the LSTM cell."""
    import torch
    from paper_2505_17852_amd import workloads as wl
    w, cfg = wl.CONFIGS[name], wl.model_cfg(name)
    if cfg["wdtype"] != wl.BF16:
        raise SystemExit("--library-gemm: bf16-weight workloads only")
    H = cfg["hidden"]
    M, K, N = 2 * w["N"] * w["B"], 2 * H, 4 * H
    g = torch.Generator(device="cuda:0").manual_seed(0)
    a = torch.randn(M, K, device="cuda:0", dtype=torch.float16, generator=g)
    wt = torch.randn(N, K, device="cuda:0", dtype=torch.float16, generator=g)
    for _ in range(5):
        torch.nn.functional.linear(a, wt)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = 50
    e0.record()
    for _ in range(reps):
        torch.nn.functional.linear(a, wt)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    tf = 2.0 * M * N * K / (ms * 1e-3) / 1e12
    return {"kernel": "torch fp16 GEMM (hipBLASLt)", "workload": name, "M": M, "N": N, "K": K,
            "ms_per_launch": ms, "TFLOPs": tf, "peak": PEAK_TFLOPS["fp16"], "frac": tf / PEAK_TFLOPS["fp16"]}


def update_hbm(P, w, upd):
    """Algorithmic HBM rate of the update kernel (theta read and written
    once) from its HIP-event time, against the 8 TB/s HBM3E peak."""
    ms, n = upd
    if n == 0 or ms <= 0:
        return None
    t = ms / n * 1e-3
    gbps = 2 * P * w / t / 1e9
    return {"bytes": 2 * P * w, "ms_per_launch": ms / n, "GBps": gbps, "peak_GBps": HBM_PEAK_GBPS,
            "frac": gbps / HBM_PEAK_GBPS}


def embed_hbm(cfg, passes, B, C, w, emb, launches_per_step, fd=False):
    """Algorithmic HBM rate of the perturbed-embedding kernel: per timestep it
    writes the passes*B rows of E activations (w bytes each; padding rows
    included, as written) and reads B rows of EMB; a launch covers one
    timestep (bf16) or a time chunk (fp32)."""
    ms, n = emb
    if n == 0 or ms <= 0 or not launches_per_step:
        return None
    gran = (128 if w == 2 else 32) * (2 if fd else 1)
    Bp = (B + gran - 1) // gran * gran
    E = cfg["embed"]
    byt = C * (passes * Bp * E * w + B * E * w) / launches_per_step
    gbps = byt / (ms / n * 1e-3) / 1e9
    return {"bytes_per_launch": byt, "ms_per_launch": ms / n, "GBps": gbps, "frac": gbps / HBM_PEAK_GBPS}


def stream_limit(name, reps=10):
    """The streaming rate of the update's access pattern without its
    arithmetic: torch's in-place bitwise xor with 0 over the workload's
    theta bytes (read and written once per launch), HIP events over `reps`
    launches after two warm-up launches."""
    import torch
    from paper_2505_17852_amd import workloads as wl
    from paper_2505_17852_amd import zo
    cfg = wl.model_cfg(name)
    w = 2 if cfg["wdtype"] == wl.BF16 else 4
    nbytes = zo.param_count(cfg) * w
    buf = torch.zeros(nbytes // 16, 4, dtype=torch.int32, device="cuda:0")
    for _ in range(2):
        buf.bitwise_xor_(0)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(reps):
        buf.bitwise_xor_(0)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    byt = 2 * buf.numel() * 4
    return {"stream_limit": name, "bytes_per_launch": byt, "ms_per_launch": ms,
            "GBps": byt / (ms * 1e-3) / 1e9, "frac_of_hbm_peak": byt / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS}


def head_hbm(cfg, passes, B, C, w, head, launches_per_step, fd=False):
    """Algorithmic HBM rate of the output head: per step it reads W_out once
    per time chunk, the top layer's states of every timestep once, and writes
    each row's (max, sum of exp) partial of every vocabulary tile (8 bytes)
    and its target logit (4 bytes)."""
    ms, n = head
    if n == 0 or ms <= 0 or not launches_per_step:
        return None
    gran = (128 if w == 2 else 32) * (2 if fd else 1)
    Bp = (B + gran - 1) // gran * gran
    V, H = cfg["vocab"], cfg["hidden"]
    M = passes * Bp
    vt = 256 if w == 2 else 128
    nvt = (V + vt - 1) // vt
    per_step = launches_per_step * V * H * w + C * M * H * w + C * M * (8 * nvt + 4)
    byt = per_step / launches_per_step
    gbps = byt / (ms / n * 1e-3) / 1e9
    return {"bytes_per_launch": byt, "ms_per_launch": ms / n, "GBps": gbps, "frac": gbps / HBM_PEAK_GBPS}


def cpu_baseline(name, budget_s=20.0, fd=False):
    """The oracle on the host cores, on a bounded sample of the workload:
    the full batch with the first N' probes (N' doubling until the budget is
    used), losses and update. Rate = 2 N' B C / time (central differences) or
    (N' + 1) B C / time (forward differences)."""
    import numpy as np  # noqa: F401
    from oracle import oracle as ref
    from paper_2505_17852_amd import workloads as wl
    w = wl.CONFIGS[name]
    cfg = wl.model_cfg(name)
    sd = wl.seeds(name)
    tokens, mask = wl.batch(name)
    B, C = tokens.shape[0], tokens.shape[1] - 1
    if w["embed"] >= 1024:  # billion-parameter shapes: a few sequences, short context
        B, C = 2, 8
        tokens = tokens[:B, :C + 1].copy()
    theta = ref.init(cfg, sd["init"])
    n, spent, rate, sample = 1, 0.0, None, None
    while True:
        th = theta.copy()
        t0 = time.perf_counter()
        if fd:
            L, L0 = ref.fd_losses(cfg, th, sd["step"], w["eps"], n, tokens, mask)
            ref.fd_update(cfg, th, sd["step"], w["eps"], w["lr"], L, L0)
        else:
            lp, lm = ref.perturbed_losses(cfg, th, sd["step"], w["eps"], n, tokens, mask)
            ref.update(cfg, th, sd["step"], w["eps"], w["lr"], lp, lm)
        dt = time.perf_counter() - t0
        spent += dt
        rate = (n + 1 if fd else 2 * n) * B * C / dt
        what = "forward-difference losses + update" if fd else "losses + update"
        sample = f"{name} with the first {n} of {w['N']} probes, B={B} C={C} ({what})"
        if spent + 2.2 * dt > budget_s or n >= w["N"]:
            break
        n *= 2
    return {"value": rate, "unit": "tokens/s", "cores": ref.threads(), "kind": "oracle",
            "sample": sample, "cpu_model": cpu_model(), "host_cpus": host_cpus()}


def cpu_model():
    """The host CPU's model name (from /proc/cpuinfo), or None."""
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def host_cpus():
    """CPUs this process may run on."""
    try:
        return len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        return os.cpu_count()


def start_one_thread(name, fd=False):
    """Starts the same oracle sample on one thread, in a child process with
    OMP_NUM_THREADS=1 (the oracle reads its thread count at load). Called
    before this process touches the GPU, so the child never inherits a GPU
    context; it runs while the GPU steps are timed."""
    import atexit
    import subprocess
    env = dict(os.environ, OMP_NUM_THREADS="1")
    cmd = [sys.executable, os.path.abspath(__file__), "--cpu-baseline-only", "--workload", name,
           "--estimator", "fd" if fd else "cd"]
    proc = subprocess.Popen(cmd, env=env, stdout=subprocess.PIPE, stderr=subprocess.DEVNULL, text=True)
    atexit.register(lambda: proc.poll() is None and proc.kill())  # an early exit ends the child too
    return proc


def finish_one_thread(proc, timeout_s=300):
    """The one-thread figure of start_one_thread's child; None when it fails
    or does not finish within timeout_s more seconds."""
    import subprocess
    try:
        stdout, _ = proc.communicate(timeout=timeout_s)
    except subprocess.TimeoutExpired:
        proc.kill()
        proc.communicate()
        return None
    lines = [l for l in stdout.splitlines() if l.startswith("{")]
    if proc.returncode != 0 or not lines:
        return None
    d = json.loads(lines[-1])
    return {"value": d["value"], "unit": d["unit"], "cores": d["cores"], "sample": d["sample"]}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=None)
    ap.add_argument("--workload", default="c4", choices=sorted(DESCRIPTION))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-baseline-only", action="store_true",
                    help="time only the CPU oracle on the workload's sample and print it as JSON (the "
                         "one-thread figure runs this way, with OMP_NUM_THREADS=1)")
    ap.add_argument("--seq-len", type=int, default=None,
                    help="profiling runs only: score the first C positions of each sequence "
                         "(every gate launch keeps the workload's full shape; the JSON line "
                         "then names the shortened C)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="run one 1 GiB device-to-device copy and exit (the reference kernel "
                         "for scaling the FETCH_SIZE / WRITE_SIZE counters to bytes)")
    ap.add_argument("--calibrate-stream", action="store_true",
                    help="time an in-place read-modify-write of the workload's theta bytes "
                         "(the update's access pattern without its arithmetic) and exit")
    ap.add_argument("--library-gemm", action="store_true",
                    help="bf16-weight workloads: time torch's fp16 GEMM (hipBLASLt) of the "
                         "gate's plain product, the workload's rows times [x; h] against a "
                         "[4H][E + H] weight matrix, for context, and exit")
    ap.add_argument("--prof-every", type=int, default=None,
                    help="time every n-th launch of each kernel class with HIP events "
                         "(default: 1 for c3/c4/c5, 61 otherwise)")
    ap.add_argument("--estimator", default="cd", choices=["cd", "fd"],
                    help="cd: central differences, 2N passes (default); fd: forward "
                         "differences, N perturbed passes and one clean pass")
    args = ap.parse_args()
    if args.cpu_baseline_only:
        print(json.dumps(cpu_baseline(args.workload, budget_s=10.0, fd=args.estimator == "fd")), flush=True)
        return
    if args.gpus != 1:
        print(f"bench.py runs one GPU's share of the step; --gpus {args.gpus} is not supported "
              "(perturbations would be sharded across GPUs with one all-gather of the 2N "
              "losses per step; that path is not built)", file=sys.stderr)
        sys.exit(2)

    special = args.calibrate_copy or args.calibrate_stream or args.library_gemm
    one_thread = None
    if not args.no_cpu_baseline and not special:
        one_thread = start_one_thread(args.workload, fd=args.estimator == "fd")

    import numpy as np
    import torch

    from paper_2505_17852_amd import workloads as wl
    from paper_2505_17852_amd import zo

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    zo.lib()  # fails loudly if the HIP library is not built
    if args.calibrate_copy:
        src = torch.ones(1 << 30, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        print("[bench] copied 1 GiB device to device", file=sys.stderr, flush=True)
        return
    if args.calibrate_stream:
        print(json.dumps(stream_limit(args.workload)), flush=True)
        return
    if args.library_gemm:
        print(json.dumps(library_gemm(args.workload)), flush=True)
        return
    name = args.workload
    W_def, K_def = DEFAULTS[name]
    W = W_def if args.warmup is None else args.warmup
    K = K_def if args.steps is None else args.steps
    w = wl.CONFIGS[name]
    cfg = wl.model_cfg(name)
    sd = wl.seeds(name)
    N, eps, lr = w["N"], w["eps"], w["lr"]
    tokens, mask = wl.batch(name)
    if args.seq_len is not None:
        if not 1 <= args.seq_len <= tokens.shape[1] - 1:
            raise SystemExit(f"--seq-len must lie in [1, {tokens.shape[1] - 1}]")
        tokens = np.ascontiguousarray(tokens[:, :args.seq_len + 1])
        mask = None if mask is None else np.ascontiguousarray(mask[:, :args.seq_len])
    B, C = tokens.shape[0], tokens.shape[1] - 1
    dev = torch.device("cuda:0")
    theta = zo.new_theta(cfg, dev)
    zo.init(cfg, theta, sd["init"])
    td = torch.from_numpy(tokens).to(dev)
    md = None if mask is None else torch.from_numpy(mask).to(dev)
    assert int(td.min()) >= 0 and int(td.max()) < cfg["vocab"]
    ws = zo.new_workspace(cfg, N, B, C, dev)
    fd = args.estimator == "fd"
    passes = N + 1 if fd else 2 * N
    Lp = torch.empty(N, dtype=torch.float32, device=dev)
    Lm = torch.empty(1 if fd else N, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()

    def step(k):
        if fd:
            zo.fd_losses(cfg, theta, sd["step"] + k, eps, N, td, md, L=Lp, L0=Lm, workspace=ws,
                         stream=stream, check_tokens=False)
            zo.fd_update(cfg, theta, sd["step"] + k, eps, lr, Lp, Lm, stream=stream)
        else:
            zo.perturbed_losses(cfg, theta, sd["step"] + k, eps, N, td, md, Lplus=Lp, Lminus=Lm,
                                workspace=ws, stream=stream, check_tokens=False)
            zo.update(cfg, theta, sd["step"] + k, eps, lr, Lp, Lm, stream=stream)

    for k in range(W):
        step(k)
        torch.cuda.synchronize()
        print(f"[bench] warm-up step {k + 1}/{W} done", file=sys.stderr, flush=True)
    every = args.prof_every if args.prof_every is not None else PROF_EVERY.get(name, PROF_EVERY_SHORT)
    zo.profile_enable(every)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(W, W + K):
        step(k)
        if K > 1 and (k - W) % max(1, K // 4) == 0:
            print(f"[bench] timed step {k - W + 1}/{K} enqueued", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    print(f"[bench] {K} timed steps in {dt:.3f} s", file=sys.stderr, flush=True)
    prof = zo.profile_read()
    zo.profile_enable(False)
    losses_ok = bool(torch.isfinite(Lp).all() and torch.isfinite(Lm).all())

    ms_per_step = dt / K * 1e3
    tokens_per_step = passes * B * C
    value = tokens_per_step / (dt / K)
    wdt = "bf16" if cfg["wdtype"] == wl.BF16 else "f32"  # weight storage
    wbytes = 2 if wdt == "bf16" else 4
    # arithmetic of the products: bf16 weights run as fp16 MFMA operands
    # (fp16(W + s eps z) and fp16 activations, fp32 accumulation)
    dtype = "fp16" if wdt == "bf16" else "f32"
    peak = PEAK_TFLOPS[dtype]
    gate_ms, gate_n, gate_all = prof["gate"]
    fl_step = gate_flops(cfg, passes, B) * C  # algorithmic gate flops per step
    # average per launch: C L layer-steps per step, one per launch (bf16) or several
    # layers' steps of one wavefront per launch (fp32)
    fl_launch = fl_step * K / gate_all if gate_all else fl_step / (cfg["n_layers"] * C)
    steps_per_launch = cfg["n_layers"] * C * K / gate_all if gate_all else 1.0  # layer-steps per gate launch
    traffic_step = measured_traffic(name, wdt)
    achieved = (fl_launch * gate_n) / (gate_ms * 1e-3) / 1e12 if gate_ms > 0 else None
    fwd_flops = 2 * wl.gemm_params(cfg) * tokens_per_step
    # per class: the timed launches' mean duration times all launches of the class
    kernels = {k: {"ms_per_step": (v[0] / v[1] * v[2] / K) if v[1] else 0.0, "launches_per_step": v[2] / K,
                   "ms_per_launch": v[0] / v[1] if v[1] else None, "timed_launches": v[1]}
               for k, v in prof.items()}
    out = {
        "metric": METRIC_FD if fd else METRIC,
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype,
        "data": "synthetic",
        "config": {"workload": f"{name}: {DESCRIPTION[name]}", "estimator": args.estimator,
                   "N": N, "B": B, "C": C,
                   "params": zo.param_count(cfg), "eps": eps, "lr": lr},
        "roofline": {"bound": "mfma", "kernel": "gate (fused LSTM layer step)",
                     "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                     "frac": None if achieved is None else achieved / peak,
                     "traffic": None if fd or traffic_step is None else traffic_step * steps_per_launch,
                     "flops_per_launch": fl_launch},
        "step_mfma_frac_algorithmic": fwd_flops / (dt / K) / 1e12 / peak,
        # the parameter update reads and writes theta once: 2 P w bytes
        "update_hbm": update_hbm(zo.param_count(cfg), wbytes, prof["update"][:2]),
        # the perturbed embedding writes 2N*B rows of E activations per timestep
        # (and gathers B rows of EMB): algorithmic bytes over its event time
        "embed_hbm": embed_hbm(cfg, passes, B, C, wbytes, prof["embed"][:2],
                               prof["embed"][2] / K, fd),
        # the head reads W_out once per time chunk and every timestep's top-layer states once
        "head_hbm": head_hbm(cfg, passes, B, C, wbytes, prof["head"][:2],
                             prof["head"][2] / K, fd),
        "kernels": kernels,
        "event_timing": f"every {every}-th launch of each kernel class",
        "losses_finite": losses_ok,
    }
    if not args.no_cpu_baseline:
        # the one-thread child first (it ran beside the GPU steps), so that the
        # multi-thread figure has the host's cores to itself
        print("[bench] waiting for the one-thread CPU oracle sample", file=sys.stderr, flush=True)
        single = finish_one_thread(one_thread)
        print("[bench] timing the CPU oracle on a sample", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(name, fd=fd)
        out["cpu_baseline"]["one_thread"] = single
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
