"""Throughput of mini-batch MLP training on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c2] [--dtype f32]

One step is one pass of the whole training path over the workload's data:
every SGD step of one epoch (forward, back-propagation, batch tendencies,
update) plus, where the workload has a held-out set, batched inference on it.
Inputs are resident in device memory before timing starts.  Prints one JSON
line on stdout; per-kernel timings go to stderr.  `value` is the warm rate
(the K timed steps back to back); `cold_cache` times single steps after a
write larger than the 256 MB memory-side cache, each from the initial
parameters.

--dtype f64 runs the same workload with an fp64 net (the paper's real64 kind):
inputs, targets and parameters in fp64, every kernel in fp64, the roofline
against the fp64 matrix peak.

The default workload is the paper's MNIST network shape (784-30-10, sigmoid,
section 4) on synthetic MNIST-shaped data: 60000 uniform [0,1) 784-vectors
with one-hot labels over 10 classes, batch 1000, eta 3.0, one epoch of 60
steps, then inference on 10000 held-out samples.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
FP32_MFMA_PEAK_TFS = 157.3     # MI355X dense fp32 matrix, TFLOP/s
FP64_MFMA_PEAK_TFS = 78.6      # MI355X dense fp64 matrix, TFLOP/s
PROFILE_REPEATS = 20

METRIC = "training samples/sec (fwd+bwd+SGD) at 784-30-10 and wide MLP; % HBM/MFMA roofline"

DESCRIBE = {
    "c1": "784-30-10 sigmoid fp32, 1000 samples, batch 100, eta 3.0, 10 SGD steps",
    "c2": ("784-30-10 sigmoid fp32, 60000 samples, batch 1000, eta 3.0, one epoch of 60 SGD "
           "steps + inference on 10000 held-out samples"),
    "c3": ("784-100-100-10 tanh/tanh/sigmoid fp32, 60000 samples, batch 10000 as 16 shards "
           "summed in order, eta 1.0, 6 SGD steps"),
    "c4": "784-1024-1024-1024-10 relu/sigmoid fp32, 65536 samples, batch 4096, eta 0.1, 16 SGD steps",
    "c5": "4096-4096-4096-4096-10 relu/sigmoid fp32, 32768 samples, batch 8192, eta 0.01, 4 SGD steps",
}


def kernel_sources_sha() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_1902_06714_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()[:16]


def read_traffic(kernel: str, workload: str, sha: str):
    """HBM bytes per launch of `kernel` from the committed counter summary,
    if it was taken on the current kernel sources; else None."""
    path = os.path.join(ROOT, "profiles", "traffic.txt")
    if not os.path.exists(path):
        return None
    for line in open(path):
        f = dict(kv.split("=", 1) for kv in line.split() if "=" in kv)
        if f.get("kernel") == kernel and f.get("workload") == workload and f.get("sha") == sha:
            try:
                return float(f["bytes_per_launch"])
            except (KeyError, ValueError):
                return None
    return None


def cpu_baseline(w, X, Y, Xh, budget_s: float, precision: str = "f32"):
    """The CPU reference (unchanged) timed on the host cores: whole steps of
    the same workload, repeated until about budget_s seconds have passed."""
    import numpy as np

    from oracle import mlp
    from paper_1902_06714_amd import workloads as W

    try:
        from threadpoolctl import threadpool_info
        cores = max([int(i.get("num_threads", 1)) for i in threadpool_info()] or [1])
    except Exception:
        cores = os.cpu_count() or 1
    theta = W.make_params(w)
    t0, c0 = time.perf_counter(), time.process_time()
    reps, sgd_steps, stop = 0, 0, False
    n_train = w.batch * w.steps
    while not stop:
        for t in range(w.steps):
            sl = slice(t * w.batch, (t + 1) * w.batch)
            theta, _ = mlp.train_batch(theta, w.dims, list(w.acts), X[sl], Y[sl], w.eta, w.shards,
                                       precision=precision)
            sgd_steps += 1
            if time.perf_counter() - t0 > 3 * budget_s:
                stop = True
                break
        else:
            if Xh is not None:
                mlp.output(theta, w.dims, list(w.acts), Xh)
            reps += 1
            stop = time.perf_counter() - t0 >= budget_s
    el = time.perf_counter() - t0
    busy = (time.process_time() - c0) / el   # CPU seconds of all threads per second
    samples = sgd_steps * w.batch
    if reps >= 1 and sgd_steps == reps * w.steps:
        sample = f"{reps} full step(s) of the workload ({reps * n_train} training samples" + (
            f" + {reps} x {Xh.shape[0]} inference samples)" if Xh is not None else ")")
    else:
        sample = f"the first {sgd_steps} SGD steps ({samples} training samples) of the workload"
    return {"value": samples / el, "unit": "samples/s", "cores": cores, "kind": "oracle",
            "sample": sample + f", {el:.1f} s on the host",
            "cpu_seconds_per_second": round(busy, 2)}


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="c2", choices=sorted(DESCRIBE))
    ap.add_argument("--dtype", default="f32", choices=("f32", "f64"),
                    help="element type of the net (f64: the real64 variant)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="budget of the CPU-reference timing (0 skips it)")
    ap.add_argument("--cold-reps", type=int, default=3,
                    help="steps timed one at a time after flushing the memory-side cache")
    ap.add_argument("--flush-mib", type=int, default=512,
                    help="bytes written between cold steps (above the 256 MB memory-side cache)")
    ap.add_argument("--copy-calib-mib", type=int, default=0,
                    help="only run a plain device copy of this size 20 times (counter scale)")
    args = ap.parse_args(argv)

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_1902_06714_amd import nf, workloads as W

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.copy_calib_mib:
        n = args.copy_calib_mib * (1 << 20) // 4
        a = torch.ones(n, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        for _ in range(20):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calib_bytes_each_way": n * 4, "copies": 20}))
        return 0

    w = W.WORKLOADS[args.workload]
    f64 = args.dtype == "f64"
    npt = np.float64 if f64 else np.float32
    tdt = torch.float64 if f64 else torch.float32
    print(f"[bench] generating {w.name} data", file=sys.stderr, flush=True)
    X, Y = W.make_data(w)
    Xh = W.make_data(w, heldout=True)[0] if w.heldout else None
    theta0 = W.make_params(w)
    xd = torch.from_numpy(X.astype(npt)).to(dev)
    yd = torch.from_numpy(Y.astype(npt)).to(dev)
    xhd = torch.from_numpy(Xh.astype(npt)).to(dev) if Xh is not None else None
    outd = torch.empty((Xh.shape[0], w.dims[-1]), dtype=tdt, device=dev) if Xh is not None else None
    n_train = w.batch * w.steps
    train_epoch = nf.nf_train_epoch_f64 if f64 else nf.nf_train_epoch
    forward = nf.nf_forward_f64 if f64 else nf.nf_forward

    net = nf.nf_net_create(w.dims, list(w.acts), dtype=nf.NF_F64 if f64 else nf.NF_F32)
    try:
        if f64:
            nf.nf_set_params_f64(net, theta0.astype(np.float64))
        else:
            nf.nf_set_params(net, theta0)

        def step():
            train_epoch(net, xd[:n_train], yd[:n_train], w.batch, w.eta, w.shards)
            if xhd is not None:
                forward(net, xhd, outd)

        print(f"[bench] warmup {args.warmup}", file=sys.stderr, flush=True)
        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        stream = torch.cuda.current_stream()
        # an event between consecutive steps gives the spread of single steps
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
        ev0, ev1 = evs[0], evs[-1]
        t0 = time.perf_counter()
        ev0.record(stream)
        for i in range(args.steps):
            step()
            evs[i + 1].record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ms = ev0.elapsed_time(ev1)
        per_step = [evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)]
        print(f"[bench] timed {args.steps} steps: {ms:.3f} ms (events), {wall * 1e3:.3f} ms (wall)",
              file=sys.stderr, flush=True)

        # the same step with the data out of the 256 MB memory-side cache (the
        # 188 MB training set of the 784-30-10 workload fits in it): each
        # repetition restarts from the initial parameters, writes a larger
        # buffer, then times one step on its own (all but the step untimed)
        cold = []
        if args.cold_reps > 0:
            flush = torch.empty(args.flush_mib * (1 << 18), dtype=torch.float32, device=dev)
            for r in range(args.cold_reps):
                if f64:
                    nf.nf_set_params_f64(net, theta0.astype(np.float64))
                else:
                    nf.nf_set_params(net, theta0)
                flush.fill_(float(r))
                torch.cuda.synchronize()
                ev0.record(stream)
                step()
                ev1.record(stream)
                torch.cuda.synchronize()
                cold.append(ev0.elapsed_time(ev1))
            del flush
            print(f"[bench] after a {args.flush_mib} MiB flush: "
                  + ", ".join(f"{c:.3f}" for c in cold) + " ms per step", file=sys.stderr,
                  flush=True)

        # per-kernel durations, same workload and launch configuration: every
        # launch runs PROFILE_REPEATS times back to back between two events on
        # the stream it is launched on (kernels never write what they read)
        nf.nf_profile(net, PROFILE_REPEATS)
        step()
        stats = nf.nf_profile_read(net)
        nf.nf_profile(net, 0)
        finite = bool(np.all(np.isfinite(nf.nf_get_params_f64(net) if f64 else nf.nf_get_params(net))))
    finally:
        nf.nf_net_destroy(net)

    for k in stats:
        avg = k["total_ms"] / k["launches"]
        print(f"[kernel] {k['name']:<28} launches {k['launches']:>6}  avg {avg * 1e3:9.2f} us  "
              f"total {k['total_ms']:9.3f} ms  {k['bytes'] / k['launches'] / 1e6:11.6f} MB/launch  "
              f"{k['flops'] / k['launches'] / 1e9:9.4f} GFLOP/launch", file=sys.stderr)
    sha = kernel_sources_sha()
    mfma_peak = FP64_MFMA_PEAK_TFS if f64 else FP32_MFMA_PEAK_TFS
    ridge = mfma_peak * 1e12 / (HBM_PEAK_GBS * 1e9)   # flop per byte

    def roofline(k):
        """Roofline of one timed kernel: algorithmic bytes or flops per launch
        over its average launch time, against the resource that bounds it."""
        avg_s = k["total_ms"] / k["launches"] / 1e3
        bytes_l = k["bytes"] / k["launches"]
        flops_l = k["flops"] / k["launches"]
        if flops_l / bytes_l < ridge:
            achieved = bytes_l / avg_s / 1e9
            r = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                 "frac": achieved / HBM_PEAK_GBS}
        else:
            achieved = flops_l / avg_s / 1e12
            r = {"bound": "mfma", "achieved": achieved, "peak": mfma_peak,
                 "unit": "TFLOP/s", "frac": achieved / mfma_peak}
        r["traffic"] = read_traffic(k["name"], w.name + ("_f64" if f64 else ""), sha)
        r["kernel"] = k["name"]
        r["avg_us"] = avg_s * 1e6
        r["launches_per_step"] = k["launches"]
        r["bytes_per_launch"] = bytes_l
        r["flops_per_launch"] = flops_l
        return r

    # the dominant kernel (most time per step), then every timed kernel
    roof = roofline(stats[0])
    kernels = [roofline(k) for k in stats]

    value = n_train * args.steps / (ms / 1e3)
    line = {
        "metric": METRIC,
        "value": value,
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": args.dtype,
        "data": "synthetic",
        "config": {"workload": DESCRIBE[w.name].replace("fp32", "fp64") if f64 else DESCRIBE[w.name],
                   "dims": list(w.dims), "batch": w.batch,
                   "sgd_steps_per_step": w.steps, "training_samples_per_step": n_train,
                   "heldout_per_step": int(Xh.shape[0]) if Xh is not None else 0,
                   "shards": w.shards, "kernel_sources": sha},
        "roofline": roof,
        "kernels": kernels,
        "params_finite": finite,
    }
    line["per_step_ms"] = {"mean": float(np.mean(per_step)), "std": float(np.std(per_step)),
                           "median": float(np.median(per_step)), "min": float(np.min(per_step)),
                           "max": float(np.max(per_step))}
    if cold:
        med = float(np.median(cold))
        line["cold_cache"] = {"value": n_train / (med / 1e3), "unit": "samples/s",
                              "ms_per_step_median": med, "ms_per_step": cold,
                              "flush_bytes": args.flush_mib << 20}
    if args.cpu_seconds > 0:
        print(f"[bench] timing the CPU reference (~{args.cpu_seconds:.0f} s)", file=sys.stderr,
              flush=True)
        line["cpu_baseline"] = cpu_baseline(w, X, Y, Xh, args.cpu_seconds, args.dtype)
        if w.name in ("c1", "c2"):
            # the same reference on one core, beside the paper's one-core timing
            # of this network shape (section 5); context only
            try:
                from threadpoolctl import threadpool_limits
            except ImportError:
                threadpool_limits = None
            if threadpool_limits is not None:
                with threadpool_limits(limits=1):
                    one = cpu_baseline(w, X, Y, Xh, args.cpu_seconds / 2, args.dtype)
                one["cores"] = 1
                line["cpu_baseline_1core"] = one
    else:
        line["cpu_baseline"] = None
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
