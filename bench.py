"""Benchmark: fused mini-batch SGD training throughput of the 32-h-1 ReLU/MSE net.

One benchmark step is one full training call (mlp_train_epochs) over the
workload: every epoch, every mini-batch, forward + backward + SGD update, from
the same He-normal initial weights (reset by a 34 KB device copy at the start
of each step). Inputs (X, Y, the per-epoch permutations) are resident in HBM
before the timed region starts.

Prints ONE JSON line. value = samples/s = n * epochs / (seconds per step).
roofline: algorithmic FLOPs of one launch of the training kernel
(134 h FLOP per sample, the five contractions of eqs. 11-18 at 2 FLOP per
multiply-add) divided by that launch's duration, measured with HIP events on
the library's stream, against MI355X's dense fp32 peak (157.3 TFLOP/s).
cpu_baseline: the fp64 oracle on the host cores (oracle_mt.c: each batch cut into
64 fixed row chunks, OpenMP over the chunks, on OMP_NUM_THREADS threads or else
every core the process may use), on a bounded prefix of the same workload (its
first steps, same permutation).
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

FP32_PEAK_TFLOPS = 157.3
HBM_PEAK_GBS = 8000.0
# The trainer, the forward pass and the deep path's 64 x 64 GEMM tiles form fp32
# products on the bf16 matrix cores from three-part operand splits: six bf16
# part products per fp32 product. Against the dense bf16 peak (2.5 PFLOP/s) that
# arithmetic tops out at a sixth of it in fp32 work; the rooflines report the
# fraction of that ceiling beside the fraction of the fp32 peak (the metric's).
BF16_PEAK_TFLOPS = 2500.0
SPLIT_PEAK_TFLOPS = BF16_PEAK_TFLOPS / 6.0


def split_fields(achieved):
    return {"mfma_dtype": "bf16 (three-part splits, six part products per fp32 product)",
            "peak_bf16x3": SPLIT_PEAK_TFLOPS,
            "frac_bf16x3": None if achieved is None else achieved / SPLIT_PEAK_TFLOPS}


# the sources that build and launch the fused trainer (its kernel, its launch
# planning and the headers both include)
TRAINER_SOURCES = ("paper_2606_30497_amd/csrc/train_persistent.hip",
                   "paper_2606_30497_amd/csrc/api.hip",
                   "paper_2606_30497_amd/csrc/lanes.h",
                   "paper_2606_30497_amd/csrc/tags.h",
                   "paper_2606_30497_amd/csrc/mlp_internal.h",
                   "include/mlp.h")


def kernel_source_hash(files=TRAINER_SOURCES):
    h = hashlib.sha256()
    for rel in files:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(rel.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def load_traffic(workload_name):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or None
    when the kernels changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    e = t.get(workload_name)
    if not e or e.get("kernel_source_hash") != kernel_source_hash():
        return None
    return e.get("hbm_bytes_per_launch")


def cpu_baseline(w, data, max_seconds):
    import oracle
    threads = oracle.mt_threads()
    # size the prefix from a one-step probe so the whole leg takes ~max_seconds
    t = time.perf_counter()
    oracle.mt_train(data.X, data.Y, data.W1, data.W2, w.batch, w.lr, w.epochs, perm=data.perm,
                    max_steps=1)
    one = time.perf_counter() - t
    steps = max(1, min(w.steps, int(max_seconds / max(one, 1e-6))))
    t = time.perf_counter()
    oracle.mt_train(data.X, data.Y, data.W1, data.W2, w.batch, w.lr, w.epochs, perm=data.perm,
                    max_steps=steps)
    dt = time.perf_counter() - t
    samples = min(steps * w.batch, w.n * w.epochs)
    try:
        affinity = len(os.sched_getaffinity(0))
    except AttributeError:
        affinity = os.cpu_count()
    return {"value": samples / dt, "unit": "samples/s", "cores": threads, "kind": "oracle",
            "sample": "first %d SGD steps (%d samples, %.1f%% of the run) of the same workload, "
                      "fp64, %d threads (%d cores in the process's affinity mask)"
                      % (steps, samples, 100.0 * samples / (w.n * w.epochs), threads, affinity)}


def copy_calibration(mib):
    """A plain copy of known size: each launch reads and writes mib MiB."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(4):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_per_launch": n * 4, "launches": 4}), flush=True)


def measure(w, args, mlp, torch, np, data=None):
    """Time args.steps full training runs of workload w; return the JSON record."""
    import datagen
    if data is None:
        t0 = time.perf_counter()
        data = datagen.make_workload(w)
        print("# data %s generated in %.1f s" % (w.name, time.perf_counter() - t0),
              file=sys.stderr, flush=True)
    dev = torch.device("cuda:0")
    X = torch.from_numpy(data.X).to(dev)
    Y = torch.from_numpy(data.Y).to(dev)
    perm = None if data.perm is None else torch.from_numpy(data.perm).to(dev)
    W1_0 = torch.from_numpy(data.W1).to(dev)
    W2_0 = torch.from_numpy(data.W2).to(dev)
    W1 = W1_0.clone()
    W2 = W2_0.clone()
    ctx = mlp.mlp_init(W1, W2, w.batch)
    if args.strategy != "fused":
        mlp.mlp_set_strategy(ctx, args.strategy)
    el = torch.zeros(w.epochs, dtype=torch.float32, device=dev)
    mlp.mlp_profile(ctx, True)

    def step():
        W1.copy_(W1_0)
        W2.copy_(W2_0)
        mlp.mlp_train_epochs(ctx, X, Y, w.batch, w.lr, w.epochs, perm=perm, epoch_loss=el)
        return mlp.mlp_last_kernel_ms(ctx)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    mlp.mlp_check_errors(ctx)
    kernel_ms = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        kernel_ms.append(step())
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    mlp.mlp_check_errors(ctx)
    final_loss = el.cpu().numpy().tolist()

    sec = (t1 - t0) / args.steps
    samples = w.n * w.epochs
    value = samples / sec
    flop_launch = float(w.flop_per_sample()) * samples
    wgs, launches = mlp.mlp_launch_info(ctx, w.n, w.batch, w.epochs)
    avg_kernel_s = float(np.mean(kernel_ms)) / 1e3
    # one launch: the trainer's duration; host-loop strategies: the call's span
    # between its two events (every launch of the call)
    achieved = flop_launch / avg_kernel_s / 1e12
    traffic = load_traffic(w.name)
    out = {
        "metric": "training samples/sec (fwd+bwd+SGD) 32-256-1 MLP; % of fp32 peak",
        "value": value,
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": sec * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "d_in": w.d_in, "hidden": w.hidden, "n": w.n,
                   "batch": w.batch, "lr": w.lr, "epochs": w.epochs,
                   "shuffle": "seeded per-epoch permutation" if w.shuffle else "none",
                   "sgd_steps": w.steps, "strategy": args.strategy,
                   "parallelism": "single GPU"},
        "pct_fp32_peak": 100.0 * value * w.flop_per_sample() / (FP32_PEAK_TFLOPS * 1e12),
        "roofline": {
            "bound": "mfma",
            "achieved": achieved,
            "peak": FP32_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": None if achieved is None else achieved / FP32_PEAK_TFLOPS,
            "traffic": traffic,
            "kernel_ms": float(np.mean(kernel_ms)),
            "flop_per_launch": flop_launch,
            **(split_fields(achieved) if args.strategy == "fused" else {}),
        },
        "kernel_launches_per_step": launches,
        "workgroups": wgs,
        "us_per_sgd_step": float(np.mean(kernel_ms)) * 1e3 / w.steps,
        "final_epoch_loss": final_loss,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, data, args.cpu_seconds)
    return out


def measure_phases(w, args, mlp, torch, np):
    """Where a fused-trainer SGD step of workload w spends its cycles: one traced
    call (MLP_TRACE=1) over the first args.phase_steps steps; per phase, the
    median over workgroups of the cycles per step of compute wave 0 and of the
    owner wave (mlp_phase_cycles)."""
    import datagen
    data = datagen.make_workload(w)
    dev = torch.device("cuda:0")
    X = torch.from_numpy(data.X).to(dev)
    Y = torch.from_numpy(data.Y).to(dev)
    perm = None if data.perm is None else torch.from_numpy(data.perm).to(dev)
    W1 = torch.from_numpy(data.W1).to(dev)
    W2 = torch.from_numpy(data.W2).to(dev)
    ctx = mlp.mlp_init(W1, W2, w.batch)
    mlp.mlp_profile(ctx, True)
    steps = min(args.phase_steps, w.steps)
    mlp.mlp_train_epochs(ctx, X, Y, w.batch, w.lr, w.epochs, perm=perm, max_steps=steps)  # warm-up
    W1.copy_(torch.from_numpy(data.W1).to(dev))
    W2.copy_(torch.from_numpy(data.W2).to(dev))
    os.environ["MLP_TRACE"] = "1"
    try:
        mlp.mlp_train_epochs(ctx, X, Y, w.batch, w.lr, w.epochs, perm=perm, max_steps=steps)
        ms = mlp.mlp_last_kernel_ms(ctx)
        ph = mlp.mlp_phase_cycles(ctx)
    finally:
        del os.environ["MLP_TRACE"]
    mlp.mlp_check_errors(ctx)
    ph = ph[ph[:, 0, 0] > 0].astype(np.float64)
    per = ph[:, :, 1:13] / ph[:, :, 0:1]                    # cycles per step
    clock = float(np.median(ph[:, 0, 14] / (ph[:, 0, 13] * 10e-9)))
    table = {}
    for i, name in enumerate(mlp.PHASE_NAMES):
        table[name] = {"wave0_cycles": float(np.median(per[:, 0, i])),
                       "owner_cycles": float(np.median(per[:, 1, i])),
                       "wave0_p90": float(np.percentile(per[:, 0, i], 90))}
    tot = np.median(per.sum(axis=2), axis=0)
    return {"metric": "cycles per SGD step by phase (median over workgroups)",
            "config": {"workload": w.name, "steps_traced": steps, "workgroups": int(ph.shape[0])},
            "clock_hz": clock, "us_per_sgd_step_traced": ms * 1e3 / steps,
            "total_cycles": {"wave0": float(tot[0]), "owner": float(tot[1])},
            "phases": table}


def measure_forward(h, X, args, mlp, torch, np):
    """mlp_forward over every row of X (resident in HBM) with a 32-h-1 net: rows/s
    and the fraction of the fp32 MFMA peak (66 h FLOP per row: 2*32*h of eq. 11 on
    the matrix cores plus 2*h of eq. 13; formed on the bf16 matrix cores from
    three-part splits, so the fraction can pass 1, and the fraction of the
    split arithmetic's ceiling is reported beside it) and of HBM bandwidth
    (132 B per row)."""
    import datagen
    d = datagen.make_data(1, h, seed=2000 + h, with_perm=False)
    dev = X.device
    W1 = torch.from_numpy(d.W1).to(dev)
    W2 = torch.from_numpy(d.W2).to(dev)
    ctx = mlp.mlp_init(W1, W2, 64)
    n = X.shape[0]
    out = torch.empty(n, dtype=torch.float32, device=dev)
    for _ in range(args.warmup):
        mlp.mlp_forward(ctx, X, out=out)
    torch.cuda.synchronize()
    mlp.mlp_check_errors(ctx)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    t0 = time.perf_counter()
    for e0, e1 in ev:
        e0.record()
        mlp.mlp_forward(ctx, X, out=out)
        e1.record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    mlp.mlp_check_errors(ctx)
    ms = float(np.mean([e0.elapsed_time(e1) for e0, e1 in ev]))
    flop = 66.0 * h * n
    achieved = flop / (ms / 1e3) / 1e12
    gbs = 132.0 * n / (ms / 1e3) / 1e9
    # the bound is the side of the ridge the arithmetic intensity (66 h FLOP per
    # 132 bytes) falls on: HBM at h = 32 (16 FLOP/B), the matrix cores above
    if 66.0 * h / 132.0 < FP32_PEAK_TFLOPS * 1e3 / HBM_PEAK_GBS:
        roof = {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": gbs / HBM_PEAK_GBS, "traffic": None,
                "tflops": achieved, "tflops_frac": achieved / FP32_PEAK_TFLOPS}
    else:
        roof = {"bound": "mfma", "achieved": achieved, "peak": FP32_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": achieved / FP32_PEAK_TFLOPS,
                "hbm_gbs": gbs, "hbm_frac": gbs / HBM_PEAK_GBS, **split_fields(achieved)}
    roof.update({"kernel_ms": ms, "flop_per_launch": flop})
    extra = {}
    if not args.no_cpu_baseline:
        import oracle
        threads = oracle.mt_threads()
        Xh = X[:1_000_000].cpu().numpy()
        rows = max(1000, min(Xh.shape[0], int(1e10 / (66.0 * h))))   # about 10 GFLOP of fp64 work
        t = time.perf_counter()
        oracle.mt_forward(Xh[:rows], d.W1, d.W2)
        dt = time.perf_counter() - t
        extra["cpu_baseline"] = {"value": rows / dt, "unit": "rows/s", "cores": threads,
                                 "kind": "oracle",
                                 "sample": "oracle forward over the first %d rows, fp64, %d threads"
                                           % (rows, threads)}
    return dict({
        "metric": "forward rows/sec (eqs. 11-13 over a resident dataset)",
        "value": n / ((t1 - t0) / args.steps),
        "unit": "rows/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": (t1 - t0) / args.steps * 1e3,
        "higher_is_better": True,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "forward_mlp32-%d-1_n%d" % (h, n), "hidden": h, "n": n},
        "roofline": roof,
    }, **extra)


def measure_deep(w, args, mlp, torch, np):
    """mlp_deep_train_epochs over workload w (L hidden layers): samples/s and the
    call's algorithmic FLOP/s (every launch of the call, between two events)."""
    import datagen
    data = datagen.make_workload(w)
    dev = torch.device("cuda:0")
    X = torch.from_numpy(data.X).to(dev)
    Y = torch.from_numpy(data.Y).to(dev)
    perm = None if data.perm is None else torch.from_numpy(data.perm).to(dev)
    P0 = torch.from_numpy(datagen.make_deep_params(w.d_in, w.hidden, w.layers, w.seed)).to(dev)
    P = P0.clone()
    ctx = mlp.mlp_deep_init(P, w.hidden, w.layers, w.batch)
    el = torch.zeros(w.epochs, dtype=torch.float32, device=dev)
    mlp.mlp_deep_profile(ctx, True)

    def step():
        P.copy_(P0)
        mlp.mlp_deep_train_epochs(ctx, X, Y, w.batch, w.lr, w.epochs, perm=perm, epoch_loss=el)
        return mlp.mlp_deep_last_kernel_ms(ctx)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    mlp.mlp_deep_check_errors(ctx)
    t0 = time.perf_counter()
    ms = [step() for _ in range(args.steps)]
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    mlp.mlp_deep_check_errors(ctx)
    samples = w.n * w.epochs
    flop = float(w.flop_per_sample()) * samples
    achieved = flop / (float(np.mean(ms)) / 1e3) / 1e12
    out = {
        "metric": "training samples/sec (fwd+bwd+SGD), %d hidden layers" % w.layers,
        "value": samples / ((t1 - t0) / args.steps),
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": (t1 - t0) / args.steps * 1e3,
        "higher_is_better": True,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "d_in": w.d_in, "hidden": w.hidden, "layers": w.layers,
                   "n": w.n, "batch": w.batch, "lr": w.lr, "epochs": w.epochs,
                   "sgd_steps": w.steps},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": FP32_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / FP32_PEAK_TFLOPS,
                     "kernel_ms": float(np.mean(ms)), "flop_per_launch": flop},
        "us_per_sgd_step": float(np.mean(ms)) * 1e3 / w.steps,
        "final_epoch_loss": el.cpu().numpy().tolist(),
    }
    if not args.no_cpu_baseline:
        import oracle
        n_steps = 1
        t = time.perf_counter()
        oracle.deep_train(data.X, data.Y, P0.cpu().numpy(), w.d_in, w.hidden, w.layers, w.batch,
                          w.lr, w.epochs, perm=data.perm, max_steps=n_steps)
        dt = time.perf_counter() - t
        out["cpu_baseline"] = {"value": n_steps * w.batch / dt, "unit": "samples/s", "cores": 1,
                               "kind": "oracle",
                               "sample": "first SGD step (%d samples), fp64, one thread" % w.batch}
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", type=int, default=4,
                    help="index into datagen.WORKLOADS (default: the 10M-sample 32-256-1 run)")
    ap.add_argument("--suite", choices=("configs", "sweep", "table1", "forward", "deep"),
                    default=None,
                    help="instead of the one headline line, print one line per workload of a "
                         "suite: the five evaluation workloads, the hidden-width sweep "
                         "(Table II sizes), the Table I sizes, mlp_forward over the "
                         "10M-row dataset at every hidden width, or the deeper nets")
    ap.add_argument("--strategy", choices=("fused", "tile", "optimized", "baseline"),
                    default="fused",
                    help="training strategy (the paper's baseline and optimized strategies, "
                         "the per-step fused tile kernel, or the single-launch trainer)")
    ap.add_argument("--phases", action="store_true",
                    help="instead of the headline line: one traced training call of the "
                         "workload, cycles per SGD step by phase (diagnostic)")
    ap.add_argument("--phase-steps", type=int, default=2000)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="CPU seconds spent on the oracle baseline leg")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="run only a plain device copy of MIB MiB (4 launches), the reference "
                         "for scaling the FETCH_SIZE / WRITE_SIZE counters")
    args = ap.parse_args()
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.gpus != 1:
        print("bench.py runs on one GPU only: this path is single-GPU by design "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import datagen
    from paper_2606_30497_amd import mlp

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    mlp.load(require_built=True)
    if args.suite == "forward":
        w = datagen.WORKLOADS[4]
        data = datagen.make_data(w.n, 32, seed=w.seed, with_perm=False)
        X = torch.from_numpy(data.X).to("cuda:0")
        for h in datagen.SWEEP_HIDDEN:
            print(json.dumps(measure_forward(h, X, args, mlp, torch, np)), flush=True)
        return
    if args.suite == "deep":
        for w in datagen.DEEP:
            print(json.dumps(measure_deep(w, args, mlp, torch, np)), flush=True)
        return
    if args.phases:
        print(json.dumps(measure_phases(datagen.WORKLOADS[args.workload], args, mlp, torch, np)),
              flush=True)
        return
    suite = datagen.SUITES[args.suite] if args.suite else [datagen.WORKLOADS[args.workload]]
    for w in suite:
        print(json.dumps(measure(w, args, mlp, torch, np)), flush=True)


if __name__ == "__main__":
    main()
