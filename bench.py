"""Throughput of the fused Non-blocking SGD step on one MI355X.

One "step" is one whole iteration of the hot path: the simulated schedule
(finished-mini-batch mask) and mixing matrix on the host, then the fused
``nbsgd_step`` kernel (accumulate finished gradients, momentum, mix, update)
over replicas, momentum buffers and per-mini-batch gradients resident in HBM.

Prints one JSON line:
  value      learner-parameter updates per second, n * P * steps / wall time
             between two device synchronisations around the timed steps
  roofline   the fused kernel's achieved HBM bandwidth: algorithmic bytes
             4 * P * (sum of finished counts + 4 n) per launch, summed over the
             timed launches, over the summed kernel durations from HIP events
             recorded on the launch stream; against the 8 TB/s HBM3E peak
  cpu_baseline  the CPU oracle (fp64 NumPy, one thread) on a bounded column
             window of the same workload, scaled to the same unit
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
METRIC = "learner-param updates/sec and achieved HBM GB/s (% peak) for fused nbsgd_step"
UNIT = "learner-param updates/s"


def copy_context(nbytes, dev, reps: int = 5):
    """A plain device copy of ``nbytes`` (read ``nbytes``, write ``nbytes``):
    the bandwidth an elementwise kernel reaches at the step's footprint."""
    import torch

    n = max(1, nbytes // 4)
    src = torch.ones(n, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    best = float("inf")
    for _ in range(reps):
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        dst.copy_(src)
        e.record()
        torch.cuda.synchronize()
        best = min(best, s.elapsed_time(e) * 1e-3)
    del src, dst
    torch.cuda.empty_cache()
    return {"kernel": "torch copy_", "bytes_moved": 8 * n, "GBs": 8 * n / best / 1e9,
            "frac": 8 * n / best / 1e9 / PEAK_HBM_GBS}


def kernel_code_sha256(path):
    """sha256 of a source file without its // comments and blank lines: the
    key of a committed counter summary, which stays valid while only
    comments change."""
    import hashlib
    import re

    lines = []
    with open(path) as f:
        for line in f.read().split("\n"):
            line = re.sub(r"//.*$", "", line).rstrip()
            if line:
                lines.append(line)
    return hashlib.sha256("\n".join(lines).encode()).hexdigest()


def measured_traffic(wl):
    """HBM bytes per launch of the fused kernel from the committed rocprofv3
    PMC summary (FETCH_SIZE and WRITE_SIZE, each scaled by what the counter
    reads for a plain 1 GiB copy), or None when there is no summary for this
    workload or the kernel code changed since the counters were taken."""
    import glob

    sha = kernel_code_sha256(os.path.join(ROOT, "paper_2211_00889_amd", "csrc", "step.hip"))
    for path in glob.glob(os.path.join(ROOT, "profiles", "k_step_traffic_*.json")):
        with open(path) as f:
            rec = json.load(f)
        if rec.get("workload") == wl.name and rec.get("kernel_code_sha256") == sha:
            return rec
    return None


def cpu_baseline(wl, budget_s: float = 15.0, cols: int = 1 << 19):
    """The oracle on columns [0, cols) of the workload, one thread, about
    ``budget_s`` seconds; returns learner-param updates per second (the step
    is column-separable, so the cost per column is constant and the rate
    scales to the full P)."""
    from threadpoolctl import threadpool_limits

    import oracle.workload

    cols = min(cols, wl.P)
    X0, G = oracle.workload.window_inputs(wl, np.arange(cols))
    done = []
    with threadpool_limits(limits=1):
        t0 = time.perf_counter()

        def stop(k):
            done.append(k)
            return time.perf_counter() - t0 >= budget_s

        oracle.workload.run(wl, X0, G, 1 << 30, stop=stop)
        el = time.perf_counter() - t0
    steps = len(done)
    return {"value": wl.n * cols * steps / el, "unit": UNIT, "cores": 1, "kind": "oracle",
            "sample": f"{wl.name}: columns [0, {cols}) of P={wl.P}, {steps} steps in {el:.1f} s "
                      f"(fp64 NumPy, 1 thread; the step is column-separable so per-column cost "
                      f"is constant)"}


def cpu_baseline_mlp(wl, A, y, x0, budget_s: float = 15.0):
    """The oracle's MLP iterations (schedule, the bf16-input gradient of every
    finished mini-batch in fp64, the step), one thread, whole iterations until
    ``budget_s`` has passed; returns finished training samples per second.
    The oracle's evaluations of the average replica are left out."""
    from threadpoolctl import threadpool_limits

    import oracle.mlp

    with threadpool_limits(limits=1):
        t0 = time.perf_counter()
        out = oracle.mlp.train(wl, A, y, x0, 1 << 30, evaluate=False,
                               stop=lambda k: time.perf_counter() - t0 >= budget_s)
        el = time.perf_counter() - t0
    finished = int(sum(int(c.sum()) for c in out["counts"]))
    k = out["iterations"]
    return {"value": finished * wl.batch / el, "unit": "samples/s", "cores": 1, "kind": "oracle",
            "sample": f"{wl.name}: iterations 0..{k - 1} ({finished} finished mini-batches) in "
                      f"{el:.1f} s (fp64 NumPy with bf16-rounded GEMM inputs, 1 thread; "
                      f"evaluations not timed)"}


def calibration_copy(dev):
    """One plain 1 GiB device copy (torch's copy kernel), so hardware byte
    counters taken over the run can be scaled against known bytes."""
    import torch

    src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst
    torch.cuda.empty_cache()


def bench_mlp(args):
    """End-to-end MLP workload: per iteration the schedule, the shuffled
    indices, the per-mini-batch gradients on the matrix cores and the fused
    step.  Prints one JSON line with finished training samples per second,
    the algorithmic GEMM work, the device-time split between the gradient
    kernels and the step, the step's roofline figure and the oracle's rate on
    the same workload; per-kernel times come from rocprofv3."""
    import torch

    from paper_2211_00889_amd import runner
    from synth import workloads

    from synth import mlp_data

    wl = workloads.MLP
    dev = torch.device("cuda:0")
    A = mlp_data.inputs(wl.seed, wl.n_samples, wl.d_in)
    y = mlp_data.teacher_labels(wl.seed, A, wl.hidden, wl.classes)
    x0 = mlp_data.student_init(wl.seed, wl.d_in, wl.hidden, wl.classes)
    r = runner.MlpRunner(wl, dev, A, y, x0)
    for k in range(args.warmup):
        r.step(k)
    torch.cuda.synchronize()
    finished = 0
    t0 = time.perf_counter()
    for k in range(args.warmup, args.warmup + args.steps):
        mask, counts, _ = r.step(k)
        finished += int(counts.sum())
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    # the split between the gradient kernels and the step, from device events
    # in a separate pass (events inside the timed loop would slow it)
    stream = torch.cuda.current_stream(dev)
    events, split_finished = [], 0
    k0 = args.warmup + args.steps
    for k in range(k0, k0 + min(args.steps, 20)):
        split_finished += int(r.step(k, stream, events=events)[1].sum())
    torch.cuda.synchronize()
    grad_ms = float(np.mean([a.elapsed_time(b) for a, b, _ in events]))
    step_ms = float(np.mean([b.elapsed_time(c) for _, b, c in events]))
    split_flop = 2 * 2 * wl.batch * wl.d_in * wl.hidden * split_finished / len(events)
    # the fused step's algorithmic bytes (finished G rows once, X and V read
    # and written once) over its event time
    step_bytes = 4 * r.P * (split_finished / len(events) + 4 * wl.n)
    loss = float(r.evaluate().mean().cpu())
    gemm_flop = 2 * 2 * wl.batch * wl.d_in * wl.hidden * finished  # forward and dW1 GEMMs
    step_gbps = step_bytes / (step_ms * 1e-3) / 1e9
    out = {
        "metric": "end-to-end MLP Non-blocking D-PSGD: finished training samples per second",
        "value": finished * wl.batch / wall, "unit": "samples/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": wall * 1e3 / args.steps, "higher_is_better": True,
        "dtype": "bf16 GEMM inputs, fp32 accumulation and step", "data": "synthetic CIFAR-shaped",
        "config": {"workload": wl.name, "n_learners": wl.n, "minibatches": wl.m, "batch": wl.batch,
                   "P": wl.P, "row_stride": r.ld, "mean_finished_per_step": finished / args.steps},
        "layer1_gemm_tflop_per_step": gemm_flop / args.steps / 1e12,
        "split_ms": {"gradients": grad_ms, "step": step_ms, "iterations": len(events)},
        "step_gbps": step_gbps,
        "gradient_tflops": split_flop / (grad_ms * 1e-3) / 1e12,
        "gradient_frac_of_bf16_dense_peak": split_flop / (grad_ms * 1e-3) / 2.5e15,
        "roofline": {"bound": "hbm", "achieved": step_gbps, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": step_gbps / PEAK_HBM_GBS, "traffic": None, "kernel": "k_step",
                     "kernel_ms_mean": step_ms, "alg_bytes_per_launch_mean": step_bytes,
                     "note": "the fused step, the iteration's largest kernel; events around it "
                             "in the split pass"},
        "eval_loss_after": loss}
    tr = measured_traffic(wl)
    if tr is not None:
        out["roofline"]["traffic"] = tr["traffic_bytes_per_launch"]
        out["roofline"]["traffic_over_alg"] = tr["traffic_over_alg"]
        out["roofline"]["traffic_dispatches"] = f"{tr['dispatches']} launches, steps {tr['steps']}"
    del r
    torch.cuda.empty_cache()
    if args.calibration_copy:
        calibration_copy(dev)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_mlp(wl, A, y, x0, args.cpu_budget)
    print(json.dumps(out), flush=True)


def bench_graph(args, wl, r, dev):
    """The timed iterations captured once in a HIP graph and replayed: for
    launch-bound workloads (the 4-learner, 10,000-parameter one), where a
    step's kernel lasts a few microseconds and the launch dominates.  The
    step makes no allocation, copy, memset or synchronisation and carries its
    per-step constants in the kernel arguments, so each captured launch keeps
    its own mask, learning rates and W.  Every replay runs the same K
    iterations' kernels; the time per step is the replay time over K, from
    HIP events on the replay stream."""
    import torch

    K = args.steps
    plans = [r.plan(args.warmup + i) for i in range(K)]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for mask, _, _, W in plans:
            r.launch(mask, W)
    stream = torch.cuda.current_stream(dev)
    for _ in range(3):
        g.replay()
    torch.cuda.synchronize()
    R = args.replays
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(R)]
    t0 = time.perf_counter()
    for a, b in ev:
        a.record(stream)
        g.replay()
        b.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    step_ms = np.array([a.elapsed_time(b) for a, b in ev]) / K
    alg_bytes = float(np.mean([wl.alg_bytes(int(c.sum())) for _, c, _, _ in plans]))
    achieved = alg_bytes / (step_ms.mean() * 1e-3) / 1e9
    return {
        "metric": METRIC,
        "value": wl.n * wl.P * K * R / wall,
        "unit": UNIT,
        "n_gpus": 1,
        "steps": K * R,
        "warmup": args.warmup,
        "ms_per_step": wall * 1e3 / (K * R),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded SplitMix64 Irwin-Hall normals: X ~ N(0, 1), G ~ N(0, 1e-3))",
        "config": {"workload": wl.name, "n_learners": wl.n, "minibatches": wl.m, "P": wl.P,
                   "row_stride": r.ld, "mixing": wl.mixing, "order": wl.order,
                   "delay": wl.delay.kind, "lr": wl.lr, "momentum": wl.momentum,
                   "mean_finished_per_step": float(np.mean([c.sum() for _, c, _, _ in plans])),
                   "launch": f"HIP graph of {K} iterations, replayed {R} times"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM_GBS, "traffic": None, "kernel": "k_step",
                     "kernel_ms_mean": float(step_ms.mean()),
                     "kernel_ms_median": float(np.median(step_ms)),
                     "kernel_ms_of": "graph replay time per iteration (kernel plus the gap to the next)",
                     "alg_bytes_per_launch_mean": alg_bytes},
    }


def bench_unfused(args):
    """The unfused stages on the same workload (nbsgd_accumulate, nbsgd_mix,
    nbsgd_update; mix-then-step composition): per-kernel HIP-event times and
    achieved bandwidth against each kernel's algorithmic bytes.  Contiguous
    rows (these calls take [n][P])."""
    import torch

    from paper_2211_00889_amd import _lib, runner
    from synth import device as synth_device
    from synth import workloads

    wl = workloads.get(args.workload)
    n, m, P = wl.n, wl.m, wl.P
    dev = torch.device("cuda:0")
    X = torch.empty((n, P), dtype=torch.float32, device=dev)
    Y = torch.empty_like(X)
    V = torch.zeros_like(X)
    Gbar = torch.empty_like(X)
    G = torch.empty((n, m, P), dtype=torch.float32, device=dev)
    synth_device.fill_normal(X, wl.seed, workloads.STREAM_X, wl.x_std)
    synth_device.fill_normal(G, wl.seed, workloads.STREAM_G, wl.g_std)
    sched = runner.Schedule(wl)
    mixer = runner.Mixer(wl.mixing, n, wl.seed, wl.matcha_degree, wl.matcha_budget)
    stream = torch.cuda.current_stream(dev)
    names = ("k_accumulate", "k_mix", "k_update")
    ms = {k: [] for k in names}
    nbytes = {k: [] for k in names}
    for k in range(args.warmup + args.steps):
        mask, counts, _, _ = sched.mask(k)
        W = mixer.w(k)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        ev[0].record(stream)
        _lib.accumulate(G, mask, Gbar)
        ev[1].record(stream)
        _lib.mix(X, W, Y)
        ev[2].record(stream)
        _lib.update(Y, V, Gbar, counts, m, wl.lr, wl.momentum)
        ev[3].record(stream)
        torch.cuda.synchronize()
        X, Y = Y, X
        if k >= args.warmup:
            c = int(counts.sum())
            for i, (name, b) in enumerate(zip(names, (4 * P * (c + n), 4 * P * 2 * n, 4 * P * 5 * n))):
                ms[name].append(ev[i].elapsed_time(ev[i + 1]))
                nbytes[name].append(b)
    per = {}
    for name in names:
        t = float(np.mean(ms[name]))
        per[name] = {"ms_mean": t, "alg_bytes_per_launch_mean": float(np.mean(nbytes[name])),
                     "achieved_GBs": float(np.sum(nbytes[name]) / (np.sum(ms[name]) * 1e-3) / 1e9),
                     "frac": float(np.sum(nbytes[name]) / (np.sum(ms[name]) * 1e-3) / 1e9 / PEAK_HBM_GBS)}
    total_ms = float(sum(np.sum(ms[k]) for k in names) / args.steps)
    print(json.dumps({
        "metric": "unfused stages (accumulate, mix, update): per-kernel achieved HBM GB/s",
        "value": n * P / (total_ms * 1e-3), "unit": "learner-param updates/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": total_ms,
        "higher_is_better": True, "dtype": "f32", "data": "synthetic",
        "config": {"workload": wl.name, "n_learners": n, "minibatches": m, "P": P,
                   "mixing": wl.mixing, "composition": "accumulate, mix, update"},
        "kernels": per}), flush=True)


def time_step_workload(wl, args, dev):
    """Times K back-to-back fused steps of a step workload after W warm-up
    steps, on resident buffers; returns the figures of one bench record.
    With ``args.server`` the step is Alg. 3's parameter-server form
    (nbsgd_step_server) on row 0 of X as the server model, V and G."""
    import torch

    from paper_2211_00889_amd import _lib, runner

    ld = _lib.row_stride(wl.P)
    footprint = (2 * wl.n + wl.n * wl.m) * ld * 4
    first_allocation = getattr(args, "first_allocation", False)
    if not first_allocation:
        # On a freshly started device the first allocation of a working set
        # this size (the VGG-16-sized one: 80 GB) streams about 4% slower than
        # any later one, whatever the allocation order or offsets; allocating
        # and freeing the same size once, untouched, first removes that.  The
        # steps, buffers and timed region are unchanged.
        probe = torch.empty(footprint, dtype=torch.uint8, device=dev)
        del probe
        torch.cuda.empty_cache()
    r = runner.StepRunner(wl, dev)
    stream = torch.cuda.current_stream(dev)
    server = getattr(args, "server", False)

    def launch(mask, W):
        if server:
            _lib.step_server(r.Xrows[0], r.Vrows, r.Grows, wl.P, mask, wl.lr, wl.momentum)
        else:
            r.launch(mask, W)

    for k in range(args.warmup):
        mask, counts, _, W = r.plan(k)
        launch(mask, W)
    torch.cuda.synchronize()

    # Two events bracket the K launches on their stream: the launches run back
    # to back, so (end - start) / K is the kernel's mean launch duration.  An
    # event pair around every launch would put two event packets between
    # consecutive kernels (about 10 us per step on a 0.55 ms kernel).
    K = args.steps
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    sum_counts, plan_s = [], []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record(stream)
    for i in range(K):
        t_plan = time.perf_counter()
        mask, counts, _, W = r.plan(args.warmup + i)
        plan_s.append(time.perf_counter() - t_plan)
        launch(mask, W)
        sum_counts.append(int(counts.sum()))
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ld = r.ld
    del r
    torch.cuda.empty_cache()

    kern_ms_mean = start.elapsed_time(end) / K
    if server:  # finished G rows, V read and written, the one server row read and written
        alg_bytes = np.array([4 * wl.P * (c + 2 * wl.n + 2) for c in sum_counts], dtype=np.float64)
    else:
        alg_bytes = np.array([wl.alg_bytes(c) for c in sum_counts], dtype=np.float64)
    achieved = alg_bytes.sum() / (kern_ms_mean * K * 1e-3) / 1e9
    rec = {
        "value": wl.n * wl.P * K / wall,
        "ms_per_step": wall * 1e3 / K,
        "config": {"workload": wl.name, "n_learners": wl.n, "minibatches": wl.m, "P": wl.P,
                   "row_stride": ld, "mixing": wl.mixing, "order": wl.order,
                   "delay": wl.delay.kind, "lr": wl.lr, "momentum": wl.momentum,
                   "mean_finished_per_step": float(np.mean(sum_counts))},
        "host_plan_us": float(np.mean(plan_s) * 1e6),
        "placement": ("first allocation of the working set" if first_allocation else
                      "buffers allocated after one untouched allocation of the same size was freed"),
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM_GBS, "traffic": None,
                     "kernel": "k_step", "kernel_ms_mean": float(kern_ms_mean),
                     "kernel_ms_of": "HIP events around the K back-to-back launches, divided by K",
                     "alg_bytes_per_launch_mean": float(alg_bytes.mean())},
    }
    if server:
        rec["config"]["form"] = "parameter server (nbsgd_step_server, Alg. 3)"
        rec["roofline"]["kernel"] = "k_step<server>"
    tr = None if server else measured_traffic(wl)
    if tr is not None:
        rec["roofline"]["traffic"] = tr["traffic_bytes_per_launch"]
        rec["roofline"]["traffic_over_alg"] = tr["traffic_over_alg"]
        rec["roofline"]["traffic_dispatches"] = f"{tr['dispatches']} launches, steps {tr['steps']}"
    return rec


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="vgg16",
                    help="the headline step workload (default: the VGG-16-sized one, the largest "
                         "that fits one GPU), or mlp for the end-to-end MLP workload")
    ap.add_argument("--also", default=None,
                    help="comma-separated step workloads timed after the headline one in the same "
                         "run and reported under other_configs (default with --workload vgg16: "
                         "resnet18,resnet50; 'none' for none)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--unfused", action="store_true",
                    help="time the three unfused stages instead of the fused step")
    ap.add_argument("--cpu-budget", type=float, default=15.0)
    ap.add_argument("--graph", action="store_true",
                    help="capture the timed steps in a HIP graph and time its replays "
                         "(launch-bound workloads such as --workload tiny)")
    ap.add_argument("--replays", type=int, default=200,
                    help="graph replays timed with --graph")
    ap.add_argument("--server", action="store_true",
                    help="time Alg. 3's parameter-server form of the step (nbsgd_step_server) "
                         "on the workload's shape instead of the replica step")
    ap.add_argument("--first-allocation", action="store_true",
                    help="allocate the step buffers without first allocating and freeing the same "
                         "size (on a fresh device that first allocation of the VGG-16-sized working "
                         "set runs about 4%% slower)")
    ap.add_argument("--calibration-copy", action="store_true",
                    help="after the timed steps, run one plain 1 GiB device copy (torch's copy "
                         "kernel) so hardware byte counters can be scaled against known bytes")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: the simulated learners are replicas in one "
              f"GPU's HBM and there is no multi-GPU path (asked for --gpus {args.gpus})",
              file=sys.stderr)
        sys.exit(2)

    if args.workload == "mlp":
        bench_mlp(args)
        return
    if args.unfused:
        bench_unfused(args)
        return

    import torch

    from synth import workloads

    wl = workloads.get(args.workload)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.graph:
        from paper_2211_00889_amd import runner

        r = runner.StepRunner(wl, dev)
        for k in range(args.warmup):
            mask, counts, _, W = r.plan(k)
            r.launch(mask, W)
        torch.cuda.synchronize()
        out = bench_graph(args, wl, r, dev)
        del r
        torch.cuda.empty_cache()
        if not args.no_cpu_baseline:
            out["cpu_baseline"] = cpu_baseline(wl, args.cpu_budget)
        print(json.dumps(out), flush=True)
        return

    head = time_step_workload(wl, args, dev)
    print(f"[bench] {wl.name}: {head['roofline']['kernel_ms_mean']:.4f} ms per step, "
          f"{head['roofline']['frac']:.3f} of peak", file=sys.stderr, flush=True)
    out = {
        "metric": METRIC,
        "value": head["value"],
        "unit": UNIT,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded SplitMix64 Irwin-Hall normals: X ~ N(0, 1), G ~ N(0, 1e-3))",
        "config": head["config"],
        "host_plan_us": head["host_plan_us"],
        "placement": head["placement"],
        "roofline": head["roofline"],
    }
    out["copy_context"] = copy_context(int(head["roofline"]["alg_bytes_per_launch_mean"]) // 2, dev)
    if args.calibration_copy:
        calibration_copy(dev)
    also = args.also
    if also is None:
        also = "resnet18,resnet50" if wl.name == workloads.VGG16_ALLREDUCE.name else "none"
    others = []
    for name in [a for a in also.split(",") if a and a != "none"]:
        w = workloads.get(name)
        rec = time_step_workload(w, args, dev)
        print(f"[bench] {w.name}: {rec['roofline']['kernel_ms_mean']:.4f} ms per step, "
              f"{rec['roofline']['frac']:.3f} of peak", file=sys.stderr, flush=True)
        rf = rec["roofline"]
        others.append({"workload": w.name, "value": rec["value"], "unit": UNIT,
                       "ms_per_step": rec["ms_per_step"], "kernel": rf["kernel"],
                       "kernel_ms_mean": rf["kernel_ms_mean"],
                       "alg_bytes_per_launch_mean": rf["alg_bytes_per_launch_mean"],
                       "achieved_GBs": rf["achieved"], "frac": rf["frac"],
                       "traffic_over_alg": rf.get("traffic_over_alg"),
                       "mean_finished_per_step": rec["config"]["mean_finished_per_step"],
                       "row_stride": rec["config"]["row_stride"]})
    if others:
        out["other_configs"] = others
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_budget)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
