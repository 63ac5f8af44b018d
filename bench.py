#!/usr/bin/env python3
"""Throughput benchmark of the PNN training path on one MI355X.

A step is one pass of the whole hot path over the workload's synthetic training set: every
child network (CN) trains `epochs` epochs on its own slice (forward, output and hidden
errors, SGD updates), with the scheduled merges (average, and broadcast between epochs).
Inputs are resident in HBM before the timed region; initialisation and evaluation are
outside it (evaluation is timed separately and reported as `eval_ms`).

Printed: one JSON line with samples/s over all CNs (N * epochs / step time), the roofline
position of the dominant kernel (measured with HIP events around every launch in an extra,
untimed step), and the CPU oracle timed on the host cores as a baseline.

Default workload: the largest one, 784-1024-10 sigmoid MLP, K = 256 CNs, mini-batch 128,
600,000 samples, 2 epochs with a merge and broadcast after each (workload index 4).
--workload selects another.

Two further modes (not the default; one JSON line per measurement):
  --sweep-k 1,2,4,...  the time to train the workload's whole training set with K CNs for each
                       K (one epoch + merge), relative to K = 1, on the GPU and for the oracle on
                       the host cores with one thread per CN (the paper's comparison of training
                       time against the number of goroutines, section "Comparing the
                       Performances");
  --compare-cns E      E epochs of the workload; after each, the held-out accuracy and mean cost
                       of every CN and of the network merged from them (the paper's comparison of
                       the CNs' average accuracy with the PNN's, and its cost per epoch).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import pnn_inputs as I  # noqa: E402

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
FP32_PEAK_TFLOPS = 157.3       # MI355X fp32 (vector with packed FMA, and matrix)
BF16_PEAK_TFLOPS = 2500.0      # MI355X bf16 dense matrix
# fp32 products on the bf16 matrix cores (kernels named *_x3): six bf16 part products per fp32
# product, so their compute roof is the bf16 peak over six, in fp32 flops
X3_PEAK_TFLOPS = BF16_PEAK_TFLOPS / 6.0


def method_flops_per_sample(w) -> float:
    """FLOPs of the method for one training sample of one CN: forward 2*sum(W), weight
    gradient and update 2*sum(W) (one multiply-add per weight), hidden errors
    2*sum_{l>=2} W^l, plus the bias terms."""
    s = w.sizes
    fw = sum(s[l] * s[l + 1] for l in range(len(s) - 1))
    back = sum(s[l] * s[l + 1] for l in range(1, len(s) - 1))
    bias = sum(s[1:])
    return 4.0 * fw + 2.0 * back + 4.0 * bias


def kernel_work(w, name: str, launches: int, N: int, epochs_profiled: int, fused_last: bool = False):
    """Algorithmic work of one launch of a library kernel: (flops, bytes), or None.

    psgd_persistent: one launch trains every CN for one epoch (per-sample SGD).  Priced in
      effective HBM bytes: a step of plain per-sample SGD reads and writes every parameter
      once and reads its input row, 8 P + 4 n_in bytes, times the N steps of the launch.
      (The kernel keeps the parameters on chip, so its real traffic is far lower: this is
      the rate at which an HBM-streaming implementation would have to run to match it.)
    mb_persistent: one launch trains every CN for one epoch (mini-batch gradient descent, one
      hidden layer).  Priced like psgd_persistent in effective HBM bytes: a batch step of a
      streaming implementation reads and writes every parameter once, 8 P bytes, and the
      batch's input rows are read once, 4 n_in bytes a row; the flops are the method's per
      sample times the N rows of the launch.
    Mini-batch plan, totals over the profiled step divided by the launches; a layer of `in`
    inputs and `out` neurons, `rows` sample rows over all CNs and epochs, `bsteps` batch steps
    per CN; weight operands are 4 bytes (fp32) or 2 (bf16 shadow), activations and errors 4
    or 2, the fp32 master update reads and writes 8 bytes per weight (+ 2 for the bf16 shadow):
      fwd_gemm (hidden layers):  2 rows out in flops; K bsteps out in w_op + rows (in x + out a)
      bwd_gemm (hidden errors behind a wide layer): 2 rows out in; K bsteps out in w_op +
                                 rows (out a + 2 in a)
      upd_gemm (wide layers):    2 rows out in; K bsteps (out in (8 + shadow) + 8 out) +
                                 rows (out a + in x)
      tail (fused narrow last layer: forward, output error, hidden error, update):
                                 6 rows O H; K bsteps (O H (w_op + 8 + shadow) + 8 O) +
                                 rows (2 H a + 4)
    With the last layer fused into the split-bf16 products (plan "mini-batch fused last
    layer", fused_last): fwd_gemm adds the last layer's forward, 2 rows O H flops and
    K bsteps O H 4 + rows O 4 bytes; out_err (output activation and error) rows O flops and
    rows (8 O + 4) bytes; upd_gemm adds the hidden error and the last layer's update, 4 rows O H
    flops and K bsteps (8 O H + 8 O) + rows O 4 bytes (it reads the activations in place of the
    errors: the same bytes).
    merge: reads K*P floats and writes P (and K*P with broadcast, except in the fused plan, which
      defers the broadcast to the next epoch's first step); broadcast (a deferred copy made on
      demand): reads P, writes K*P.
    """
    if name.endswith("_x3"):
        name = name[:-3]
    s = w.sizes
    K = w.replicas
    L = len(s) - 1
    if name == "psgd_persistent":
        return N * method_flops_per_sample(w), N * (8.0 * w.param_count() + 4.0 * s[0])
    if name == "mb_persistent":
        bsteps_epoch = float(-(-(-(-N // K)) // w.batch))
        return N * method_flops_per_sample(w), K * bsteps_epoch * 8.0 * w.param_count() + N * 4.0 * s[0]
    if name == "merge":
        # (with the last layer fused the broadcast is deferred: the next epoch's first step reads
        # the merged network and writes every CN)
        P = w.param_count()
        return 0.0, (K * P + P + (K * P if w.merge_every_epoch and not fused_last else 0)) * 4.0
    if name == "broadcast":
        P = w.param_count()
        return 0.0, (P + K * P) * 4.0
    bf = w.precision == I.BF16_MIXED
    a = 2.0 if bf else 4.0           # hidden activations and errors
    wop = 2.0 if bf else 4.0         # operand weights
    shadow = 2.0 if bf else 0.0
    rows = float(N * epochs_profiled)
    bsteps = float(-(-(-(-N // K)) // w.batch) * epochs_profiled)

    def x_bytes(l):  # one input value of layer l (1-based): the fp32 data set for layer 1
        return 4.0 if l == 1 else a

    f = b = 0.0
    if name == "fwd_gemm":
        for l in range(1, L):
            f += 2 * rows * s[l] * s[l - 1]
            b += K * bsteps * s[l] * s[l - 1] * wop + rows * (s[l - 1] * x_bytes(l) + s[l] * a)
    elif name == "bwd_gemm":
        for l in range(1, L - 1):  # (the hidden error behind the last layer is in the tail)
            if s[l + 1] > 16:
                f += 2 * rows * s[l + 1] * s[l]
                b += K * bsteps * s[l + 1] * s[l] * wop + rows * (s[l + 1] * a + 2 * s[l] * a)
    elif name == "upd_gemm":
        for l in range(1, L):
            if s[l] > 16:
                f += 2 * rows * s[l] * s[l - 1]
                b += K * bsteps * (s[l] * s[l - 1] * (8 + shadow) + 8 * s[l]) + rows * (s[l] * a + s[l - 1] * x_bytes(l))
    elif name == "tail":
        O, H = s[L], s[L - 1]
        f = 6 * rows * O * H
        b = K * bsteps * (O * H * (wop + 8 + shadow) + 8 * O) + rows * (2 * H * a + 4)
    elif name == "out_err":
        O = s[L]
        f = rows * O
        b = rows * (8 * O + 4)
    else:
        return None
    if fused_last and name in ("fwd_gemm", "upd_gemm"):
        O, H = s[L], s[L - 1]
        if name == "fwd_gemm":
            f += 2 * rows * O * H
            b += K * bsteps * O * H * 4 + rows * O * 4
        else:
            f += 4 * rows * O * H
            b += K * bsteps * (8 * O * H + 8 * O) + rows * O * 4
    return f / launches, b / launches


def source_digest() -> str:
    """sha256 over the library sources (csrc/*.hip, csrc/*.hpp, include/*.h), in name order."""
    import glob
    import hashlib
    h = hashlib.sha256()
    files = sorted(glob.glob(os.path.join(ROOT, "paper_2304_09590_amd", "csrc", "*.hip")) +
                   glob.glob(os.path.join(ROOT, "paper_2304_09590_amd", "csrc", "*.hpp")) +
                   glob.glob(os.path.join(ROOT, "include", "*.h")))
    for f in files:
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` on `workload` from the rocprofv3 counter summaries under
    profiles/ (lines `traffic: kernel=K workload=W source=SHA bytes_per_launch=B`), or None
    when no summary was taken from the current sources."""
    import glob
    src = source_digest()
    for f in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md"))):
        with open(f) as fh:
            for line in fh:
                line = line.strip().strip("`")
                if not line.startswith("traffic:"):
                    continue
                kv = dict(t.split("=", 1) for t in line[len("traffic:"):].split() if "=" in t)
                if kv.get("kernel") == kernel and kv.get("workload") == workload and kv.get("source") == src:
                    return float(kv["bytes_per_launch"])
    return None


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(w, X, y, th0, N):
    """The oracle timed on the host cores: one thread per CN up to the usable cores (the paper
    runs one goroutine per CN), on a bounded sample of the workload (the first rows of every
    CN's slice, one epoch), repeated three times (median), plus one thread on one CN's rows."""
    from oracle import oracle as O
    cores = len(os.sched_getaffinity(0))
    threads = max(1, min(w.replicas, cores))
    o = O.Oracle.from_workload(w)
    per = -(-N // w.replicas)
    # about 6 s of work per repeat at ~2.5 GFLOP/s per thread
    budget = 6.0 * threads * 2.5e9 / method_flops_per_sample(w)
    n_s = int(min(per, max(w.batch, budget // w.replicas)))
    idx = np.concatenate([np.arange(s, s + min(n_s, ln)) for s, ln in
                          (o.shard(N, k) for k in range(w.replicas))])
    Xs, ys = X[idx], y[idx]   # the sample keeps the slicing: each CN gets its own n_s rows
    times = []
    for _ in range(3):
        th = o.replicate(th0)
        t1 = time.time()
        o.train_epoch(th, Xs, ys, threads=threads)
        times.append(time.time() - t1)
    dt = float(np.median(times))
    # one thread, one CN: the first rows of CN 0's slice (about 4 s of work)
    n1 = int(min(per, max(w.batch, 4.0 * 2.5e9 / method_flops_per_sample(w))))
    o1 = O.Oracle.from_workload(w, replicas=1)
    th1 = o1.replicate(th0)
    t1 = time.time()
    o1.train_epoch(th1, X[:n1], y[:n1], threads=1)
    dt1 = time.time() - t1
    return {"value": round(len(idx) / dt, 2), "unit": "samples/s", "cores": cores, "threads": threads,
            "kind": "oracle", "cpu_model": cpu_model(),
            "sample": f"{len(idx)} samples ({min(n_s, per)} per CN x {w.replicas} CNs), 1 epoch, fp64, "
                      f"{threads} threads (one CN per thread at a time), median of 3 repeats "
                      f"{', '.join(f'{t:.2f}' for t in times)} s",
            "one_thread": {"value": round(n1 / dt1, 2), "unit": "samples/s",
                           "sample": f"{n1} samples of one CN, 1 thread, {dt1:.2f} s"}}


def schedule_position(w, N, ms, prof):
    """The whole training schedule against the roofs: the algorithmic flops and HBM bytes of
    every profiled library kernel (kernel_work), summed, over the measured step time."""
    if not prof:
        return None
    fl = by = 0.0
    fused = "out_err" in prof
    for name, (tot, n_l) in prof.items():
        wk = kernel_work(w, name, n_l, N, w.epochs, fused)
        if wk is None:
            continue
        fl += wk[0] * n_l
        by += wk[1] * n_l
    s = ms / 1e3
    mpeak = BF16_PEAK_TFLOPS if w.precision == I.BF16_MIXED else FP32_PEAK_TFLOPS
    return {"flops": fl, "bytes": by, "tflops": round(fl / s / 1e12, 3), "mfma_peak_tflops": mpeak,
            "mfma_frac": round(fl / s / 1e12 / mpeak, 4), "gbs": round(by / s / 1e9, 1),
            "hbm_frac": round(by / s / 1e9 / HBM_PEAK_GBS, 4)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", type=int, default=4)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="first run one device-to-device copy of 1 GiB (reference dispatch for HBM byte counters)")
    ap.add_argument("--sweep-k", type=str, default=None,
                    help="comma-separated CN counts: training time of the whole training set against K")
    ap.add_argument("--sweep-cpu-samples", type=int, default=4096,
                    help="samples the oracle trains in each CPU point of --sweep-k (0: GPU only)")
    ap.add_argument("--compare-cns", type=int, default=0,
                    help="epochs of the CN-versus-merged-network comparison")
    args = ap.parse_args()
    if args.gpus != 1:
        print("the library runs on one GPU only: the CNs of a PNN are independent until the merge, "
              "so a multi-GPU run would only split the CNs across GPUs and all-reduce at the merge; "
              "no multi-GPU path is built", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2304_09590_amd import pnn as B

    if args.calibrate_copy:
        src = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        print("[bench] calibration copy: 1 GiB read + 1 GiB written", file=sys.stderr, flush=True)
        del src, dst

    if args.sweep_k:
        return sweep_k(args, torch, B)
    if args.compare_cns > 0:
        return compare_cns(args, torch, B)

    w = I.WORKLOADS[args.workload]
    N = w.n_train
    t0 = time.time()
    X, y = I.train_set(w)
    Xt, yt = I.test_set(w)
    th0 = I.init_params(w)
    print(f"[bench] workload {w.name}: data ready in {time.time() - t0:.1f}s", file=sys.stderr, flush=True)

    stream = torch.cuda.current_stream()
    xd = torch.from_numpy(X).cuda()
    yd = torch.from_numpy(y).cuda()
    xtd = torch.from_numpy(Xt).cuda()
    ytd = torch.from_numpy(yt).cuda()
    net = B.PNN(B.config_from_workload(w), th0)

    def step():
        for e in range(w.epochs):
            net.train_epoch(xd, yd, stream=stream)
            if w.merge_every_epoch:
                net.merge(broadcast=True, stream=stream)
        if not w.merge_every_epoch:
            net.merge(broadcast=False, stream=stream)

    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        print(f"[bench] warmup step {i} done", file=sys.stderr, flush=True)

    # K steps bracketed by synchronisations; an event pair per step on the launch stream gives
    # the per-step times (their median is reported beside the mean)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    evs[0].record(stream)
    for i in range(args.steps):
        step()
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    per_step = [evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)]
    ms = evs[0].elapsed_time(evs[-1]) / args.steps
    ms_median = float(np.median(per_step))
    samples = N * w.epochs
    value = samples / (ms / 1e3)
    print(f"[bench] timed {args.steps} steps: {ms:.3f} ms/step (median {ms_median:.3f})", file=sys.stderr, flush=True)

    # evaluation (outside the step)
    pred = torch.empty(len(yt), dtype=torch.int32, device="cuda")
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    correct = net.infer(xtd, pred, which=-1, y=ytd, count=True, stream=stream)
    e1.record(stream)
    torch.cuda.synchronize()
    eval_ms = e0.elapsed_time(e1)

    # per-kernel device time in one extra step
    net.profile(True)
    step()
    torch.cuda.synchronize()
    prof = net.profile_read()
    net.profile(False)
    kernels = {k: {"ms_total": round(v[0], 4), "launches": v[1], "avg_us": round(1e3 * v[0] / max(v[1], 1), 3)}
               for k, v in prof.items()}
    dom = max(prof.items(), key=lambda kv: kv[1][0])[0] if prof else None
    roofline = None
    if dom is not None:
        tot, n_l = prof[dom]
        avg_s = tot / 1e3 / n_l
        wk = kernel_work(w, dom, n_l, N, w.epochs, "out_err" in prof)
        if wk is not None:
            flops, byts = wk
            # the bound is the roof the kernel's arithmetic intensity reaches first: the matrix
            # peak of its operand type against HBM (ridge 19.7 flop/B in fp32, 312 in bf16,
            # 52 for fp32 products on the bf16 matrix cores)
            mpeak = BF16_PEAK_TFLOPS if w.precision == I.BF16_MIXED else FP32_PEAK_TFLOPS
            if dom.endswith("_x3"):
                mpeak = X3_PEAK_TFLOPS
            ridge = mpeak * 1e12 / (HBM_PEAK_GBS * 1e9)
            if dom == "psgd_persistent" or flops < ridge * byts:
                bound, ach, peak, unit = "hbm", byts / avg_s / 1e9, HBM_PEAK_GBS, "GB/s"
            else:
                bound, ach, peak, unit = "mfma", flops / avg_s / 1e12, mpeak, "TFLOP/s"
            traffic = measured_traffic(dom, w.name)
            roofline = {"kernel": dom, "bound": bound, "achieved": round(ach, 4), "peak": peak, "unit": unit,
                        "frac": round(ach / peak, 6), "traffic": traffic, "avg_us": round(avg_s * 1e6, 3),
                        "work_per_launch": byts if bound == "hbm" else flops,
                        "flop_per_byte": round(flops / byts, 3) if byts else None}

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, X, y, th0, N)

    out = {
        "metric": "training samples/sec (all K replicas) + % of HBM/MFMA roofline",
        "value": round(value, 2),
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "ms_per_step_median": round(ms_median, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.precision == I.BF16_MIXED else "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "sizes": list(w.sizes), "replicas": w.replicas, "batch": w.batch,
                   "epochs": w.epochs, "n_train": N, "lr": w.lr,
                   "merge": "every epoch" if w.merge_every_epoch else "end"},
        "roofline": roofline,
        "schedule": schedule_position(w, N, ms, prof),
        "cpu_baseline": cpu,
        "eval_ms": round(eval_ms, 3),
        "eval_accuracy": round(correct / len(yt), 4),
        "kernels": kernels,
    }
    print(json.dumps(out), flush=True)
    net.close()


def _plan_of(net, step) -> str:
    """Name of the library kernel that takes the most device time in one step."""
    net.profile(True)
    step()
    prof = net.profile_read()
    net.profile(False)
    return max(prof.items(), key=lambda kv: kv[1][0])[0] if prof else "?"


def sweep_k(args, torch, B):
    base = I.WORKLOADS[args.workload]
    N = base.n_train
    X, y = I.train_set(base)
    th0 = I.init_params(base)
    xd = torch.from_numpy(X).cuda()
    yd = torch.from_numpy(y).cuda()
    stream = torch.cuda.current_stream()
    ks = [int(k) for k in args.sweep_k.split(",") if k.strip()]
    cores = len(os.sched_getaffinity(0))
    ref_gpu = ref_cpu = None
    for K in ks:
        w = base.scaled(replicas=K)
        net = B.PNN(B.config_from_workload(w), th0)

        def step():
            for e in range(w.epochs):
                net.train_epoch(xd, yd, stream=stream)
                if w.merge_every_epoch:
                    net.merge(broadcast=True, stream=stream)
            if not w.merge_every_epoch:
                net.merge(broadcast=False, stream=stream)

        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        ev0.record(stream)
        for _ in range(args.steps):
            step()
        ev1.record(stream)
        torch.cuda.synchronize()
        ms = ev0.elapsed_time(ev1) / args.steps
        plan = _plan_of(net, step)
        torch.cuda.synchronize()
        net.close()
        ref_gpu = ref_gpu or ms
        line = {"mode": "sweep_k", "workload": base.name, "replicas": K, "n_train": N, "epochs": w.epochs,
                "gpu_ms_per_step": round(ms, 4), "gpu_samples_per_s": round(N * w.epochs / (ms / 1e3), 2),
                "gpu_time_vs_k1": round(ms / ref_gpu, 4), "gpu_plan": plan}
        if args.sweep_cpu_samples > 0:
            # the oracle on the host: the same total of samples split over K threads, one per CN
            from oracle import oracle as O
            S = max(K, args.sweep_cpu_samples)
            o = O.Oracle.from_workload(w)
            th = o.replicate(th0)
            threads = min(K, cores)
            t1 = time.time()
            o.train_epoch(th, X[:S], y[:S], threads=threads)
            cpu_s = time.time() - t1
            ref_cpu = ref_cpu or cpu_s
            line.update({"cpu_samples": S, "cpu_threads": threads, "cpu_s": round(cpu_s, 3),
                         "cpu_time_vs_k1": round(cpu_s / ref_cpu, 4)})
        print(json.dumps(line), flush=True)


def compare_cns(args, torch, B):
    w = I.WORKLOADS[args.workload]
    X, y = I.train_set(w)
    Xt, yt = I.test_set(w)
    th0 = I.init_params(w)
    xd, yd = torch.from_numpy(X).cuda(), torch.from_numpy(y).cuda()
    xtd, ytd = torch.from_numpy(Xt).cuda(), torch.from_numpy(yt).cuda()
    net = B.PNN(B.config_from_workload(w), th0)
    K = w.replicas
    for e in range(1, args.compare_cns + 1):
        net.train_epoch(xd, yd)
        # the merged network of this epoch; the CNs go on from their own parameters unless the
        # workload merges every epoch (then they restart from the merged network)
        net.merge(broadcast=False)
        cn = [net.evaluate(xtd, ytd, which=k) for k in range(K)]
        pc, pcost = net.evaluate(xtd, ytd, which=-1)
        acc = np.array([c for c, _ in cn], dtype=np.float64) / len(yt)
        cost = np.array([c for _, c in cn])
        print(json.dumps({"mode": "compare_cns", "workload": w.name, "replicas": K, "epoch": e,
                          "pnn_accuracy": round(pc / len(yt), 5), "pnn_cost": round(pcost, 6),
                          "cn_mean_accuracy": round(float(acc.mean()), 5),
                          "cn_min_accuracy": round(float(acc.min()), 5), "cn_max_accuracy": round(float(acc.max()), 5),
                          "cn_mean_cost": round(float(cost.mean()), 6)}), flush=True)
        if w.merge_every_epoch:
            net.merge(broadcast=True)
    net.close()


if __name__ == "__main__":
    main()
