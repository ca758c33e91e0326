"""Throughput of mini-batch MLP training on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c2] [--dtype f32]
                    [--wide c5|none] [--no-peaks]

One step is one pass of the whole training path over the workload's data:
every SGD step of one epoch (forward, back-propagation, batch tendencies,
update) plus, where the workload has a held-out set, batched inference on it.
Inputs are resident in device memory before timing starts.  Prints one JSON
line on stdout; per-kernel timings go to stderr.  `value` is the warm rate
(the K timed steps back to back); `cold_cache` times single steps after a
write larger than the 256 MB memory-side cache, each from the initial
parameters.

Per-kernel durations come from the timed steps run once more (up to five)
with every launch timed by its own start and end (nf_profile with repeats 1:
HIP events bound to the kernel's dispatch on the stream it runs on), behind a
spin kernel that holds the stream while the host enqueues them, so that they
run back to back as in the timed region.  `roofline` is the
kernel with the most time per step, its achieved rate being the compulsory
bytes (inputs, targets and parameters read once, parameters written once:
per sample d_0 + d_L elements, per SGD step twice the parameter count) or
the flops of its launches over its average share of the timed step (its own
duration, run_avg_us, scaled so that the kernels of a step add up to the
measured step time); `step_roofline` does the same for the whole step.  `wide` repeats the measurement on the widest
workload (4096^4-10 by default), the matrix-core half of the metric, with
its own CPU-reference timing.  `peaks_measured` holds the device's streaming
read and copy rates and its matrix-core loop rate, beside the published
peaks the fractions are quoted against.

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
PROFILE_SPIN_US = 60000.0      # stream held while the profiled steps are enqueued

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


def compulsory_bytes(w, esz: int):
    """(bytes of one SGD step, bytes of the held-out inference): every input
    and target read once, the parameters read once and written once per SGD
    step (read once for inference), the outputs of inference written once."""
    P = w.param_count()
    step = esz * (w.batch * (w.dims[0] + w.dims[-1]) + 2 * P)
    infer = esz * (w.heldout * (w.dims[0] + w.dims[-1]) + P) if w.heldout else 0
    return step, infer


def is_inference_kernel(name: str) -> bool:
    return "infer" in name or "fwd_out" in name


def cpu_baseline(w, X, Y, Xh, budget_s: float, precision: str = "f32", max_steps=None):
    """The CPU reference (unchanged) timed on the host cores: whole steps of
    the same workload, repeated until about budget_s seconds have passed (or
    max_steps SGD steps)."""
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
            if time.perf_counter() - t0 > 3 * budget_s or (max_steps and sgd_steps >= max_steps):
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


def measure_peaks(torch, nf, dev):
    """The device's own streaming and matrix-core rates (nf_calib_*)."""
    sink = torch.empty(nf.NF_CALIB_SINK_BYTES // 4, dtype=torch.float32, device=dev)
    out = {}
    big = torch.ones((1 << 30) // 4, dtype=torch.float32, device=dev)     # 1 GiB > the 256 MB cache
    dst = torch.empty_like(big)
    reads = [nf.nf_calib_read(big, sink) for _ in range(3)]
    copies = [nf.nf_calib_copy(dst, big) for _ in range(3)]
    out["hbm_read_GBs"] = big.numel() * 4 / (min(reads) / 1e3) / 1e9
    out["hbm_copy_GBs"] = 2 * big.numel() * 4 / (min(copies) / 1e3) / 1e9
    del dst, big
    # the held-out set's size (31.36 MB of inputs), read back to back: the
    # rate a launch of that size can reach with its data in the caches
    mid = torch.ones(10000 * 784, dtype=torch.float32, device=dev)
    warm = [nf.nf_calib_read(mid, sink) for _ in range(5)]
    out["read_31MB_warm_GBs"] = mid.numel() * 4 / (min(warm[1:]) / 1e3) / 1e9
    del mid
    for dtype, key in ((nf.NF_F32, "mfma_fp32"), (nf.NF_F64, "mfma_fp64")):
        runs = [nf.nf_calib_mfma(dtype, 20000, sink) for _ in range(3)]
        ms, fl, ghz = min(runs)
        out[key + "_TFs"] = fl / (ms / 1e3) / 1e12
        out[key + "_clock_GHz"] = ghz
    out["published"] = {"hbm_GBs": HBM_PEAK_GBS, "mfma_fp32_TFs": FP32_MFMA_PEAK_TFS,
                        "mfma_fp64_TFs": FP64_MFMA_PEAK_TFS}
    out["method"] = ("nf_calib_read / nf_calib_copy over 1 GiB (best of 3; the copy counts its "
                     "reads and writes), nf_calib_read over 31.36 MB back to back (best of 4 "
                     "after one), nf_calib_mfma 8 independent 32x32x2 fp32 / 16x16x4 fp64 chains "
                     "per wave, 8 (fp32) or 16 (fp64) waves per CU (best of 3); kernel timestamps")
    return out


def run_workload(args, w, f64: bool, steps: int, warmup: int, cold_reps: int, log):
    """Time `steps` whole steps of workload w after `warmup`, then profile one
    more step launch by launch.  Returns the fields of the bench line."""
    import numpy as np
    import torch

    from paper_1902_06714_amd import nf, workloads as W

    dev = torch.device("cuda:0")
    npt = np.float64 if f64 else np.float32
    tdt = torch.float64 if f64 else torch.float32
    log(f"generating {w.name} data")
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
    res = {"X": X, "Y": Y, "Xh": Xh}
    try:
        def reset():
            if f64:
                nf.nf_set_params_f64(net, theta0.astype(np.float64))
            else:
                nf.nf_set_params(net, theta0)

        reset()

        def step():
            train_epoch(net, xd[:n_train], yd[:n_train], w.batch, w.eta, w.shards)
            if xhd is not None:
                forward(net, xhd, outd)

        log(f"{w.name}: warmup {warmup}")
        for _ in range(warmup):
            step()
        torch.cuda.synchronize()
        stream = torch.cuda.current_stream()
        # an event between consecutive steps gives the spread of single steps
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        t0 = time.perf_counter()
        evs[0].record(stream)
        for i in range(steps):
            step()
            evs[i + 1].record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ms = evs[0].elapsed_time(evs[-1])
        per_step = [evs[i].elapsed_time(evs[i + 1]) for i in range(steps)]
        log(f"{w.name}: timed {steps} steps: {ms:.3f} ms (events), {wall * 1e3:.3f} ms (wall)")
        res.update(ms=ms, per_step=per_step)

        # the same step with the data out of the 256 MB memory-side cache (the
        # 188 MB training set of the 784-30-10 workload fits in it): each
        # repetition restarts from the initial parameters, writes a larger
        # buffer, then times one step on its own (all but the step untimed)
        cold = []
        if cold_reps > 0:
            flush = torch.empty(args.flush_mib * (1 << 18), dtype=torch.float32, device=dev)
            for r in range(cold_reps):
                reset()
                flush.fill_(float(r))
                torch.cuda.synchronize()
                evs[0].record(stream)
                step()
                evs[1].record(stream)
                torch.cuda.synchronize()
                cold.append(evs[0].elapsed_time(evs[1]))
            del flush
            log(f"{w.name}: after a {args.flush_mib} MiB flush: "
                + ", ".join(f"{c:.3f}" for c in cold) + " ms per step")
        res["cold"] = cold

        # the timed steps once more with every launch timed by its own start
        # and end (events bound to each kernel's dispatch).  Such a launch
        # costs the host more than the kernel runs, so a spin kernel holds the
        # stream while the host enqueues the steps; they then run back to
        # back as in the timed region (whose own time these steps report too)
        psteps = min(steps, 5)
        nf.nf_profile(net, 1)
        nf.nf_calib_spin(PROFILE_SPIN_US)
        evs[0].record(stream)
        for i in range(psteps):
            step()
            evs[i + 1].record(stream)
        stats = nf.nf_profile_read(net)
        nf.nf_profile(net, 0)
        torch.cuda.synchronize()
        res["profiled_ms_per_step"] = evs[0].elapsed_time(evs[psteps]) / psteps
        res["profiled_steps"] = psteps
        res["stats"] = stats
        res["finite"] = bool(np.all(np.isfinite(nf.nf_get_params_f64(net) if f64
                                                else nf.nf_get_params(net))))
    finally:
        nf.nf_net_destroy(net)
    return res


def summarize(w, f64: bool, res, steps: int, sha: str, log):
    """The bench-line fields of one measured workload."""
    import numpy as np

    esz = 8 if f64 else 4
    mfma_peak = FP64_MFMA_PEAK_TFS if f64 else FP32_MFMA_PEAK_TFS
    ridge = mfma_peak * 1e12 / (HBM_PEAK_GBS * 1e9)   # flop per byte
    step_bytes, infer_bytes = compulsory_bytes(w, esz)
    stats = res["stats"]
    for k in stats:
        avg = k["total_ms"] / k["launches"]
        log(f"[kernel] {k['name']:<28} launches {k['launches']:>6}  avg {avg * 1e3:9.2f} us  "
            f"min {k['min_ms'] * 1e3:8.2f}  max {k['max_ms'] * 1e3:8.2f}  "
            f"{k['bytes'] / k['launches'] / 1e6:11.6f} MB/launch  "
            f"{k['flops'] / k['launches'] / 1e9:9.4f} GFLOP/launch")

    # a launch timed by its own dispatch runs from its first wave to its
    # last; in the timed steps the launches also share the gaps between them.
    # Each kernel is charged its own duration scaled so that the kernels of a
    # step add up to the measured step (its share of the step), which is what
    # the roofline divides by; the unscaled duration is reported beside it
    busy_ms = sum(k["total_ms"] for k in stats) / res["profiled_steps"]
    in_step = (res["ms"] / steps) / busy_ms if busy_ms > 0 else 1.0

    def roofline(k):
        """Roofline of one timed kernel over its share of the step: the
        compulsory bytes its launches carry, or its flops above the ridge."""
        run_s = k["total_ms"] / k["launches"] / 1e3
        avg_s = run_s * in_step
        design_b = k["bytes"] / k["launches"]
        flops_l = k["flops"] / k["launches"]
        per_step = k["launches"] / res["profiled_steps"]
        if is_inference_kernel(k["name"]):
            comp = infer_bytes / per_step if infer_bytes else design_b
        else:
            comp = step_bytes * w.steps / per_step
        if flops_l / design_b < ridge:
            achieved = comp / avg_s / 1e9
            r = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                 "frac": achieved / HBM_PEAK_GBS}
        else:
            achieved = flops_l / avg_s / 1e12
            r = {"bound": "mfma", "achieved": achieved, "peak": mfma_peak,
                 "unit": "TFLOP/s", "frac": achieved / mfma_peak}
        r["traffic"] = read_traffic(k["name"], w.name + ("_f64" if f64 else ""), sha)
        r["kernel"] = k["name"]
        r["avg_us"] = avg_s * 1e6
        r["run_avg_us"] = run_s * 1e6
        r["run_min_us"] = k["min_ms"] * 1e3
        r["run_max_us"] = k["max_ms"] * 1e3
        r["launches_per_step"] = per_step
        r["launches_timed"] = k["launches"]
        r["bytes_per_launch"] = comp
        r["design_bytes_per_launch"] = design_b
        r["flops_per_launch"] = flops_l
        return r

    # the dominant kernel (most time per step), then every timed kernel
    kernels = [roofline(k) for k in stats]
    ms = res["ms"]
    ms_step = ms / steps
    n_train = w.batch * w.steps
    step_flops = sum(k["flops"] for k in stats) / res["profiled_steps"]
    whole_bytes = step_bytes * w.steps + infer_bytes
    if kernels[0]["bound"] == "hbm":
        ach = whole_bytes / (ms_step / 1e3) / 1e9
        step_roof = {"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": ach / HBM_PEAK_GBS, "bytes_per_step": whole_bytes}
    else:
        ach = step_flops / (ms_step / 1e3) / 1e12
        step_roof = {"bound": "mfma", "achieved": ach, "peak": mfma_peak, "unit": "TFLOP/s",
                     "frac": ach / mfma_peak, "flops_per_step": step_flops}
    step_roof["kernel_run_ms_per_step"] = busy_ms
    step_roof["in_step_scale"] = in_step
    step_roof["profiled_ms_per_step"] = res["profiled_ms_per_step"]
    per_step = res["per_step"]
    out = {
        "value": n_train * steps / (ms / 1e3),
        "ms_per_step": ms_step,
        "per_step_ms": {"mean": float(np.mean(per_step)), "std": float(np.std(per_step)),
                        "median": float(np.median(per_step)), "min": float(np.min(per_step)),
                        "max": float(np.max(per_step))},
        "roofline": kernels[0],
        "step_roofline": step_roof,
        "kernels": kernels,
        "params_finite": res["finite"],
    }
    if res["cold"]:
        med = float(np.median(res["cold"]))
        out["cold_cache"] = {"value": n_train / (med / 1e3), "unit": "samples/s",
                             "ms_per_step_median": med, "ms_per_step": res["cold"]}
    return out


def config_of(w, f64: bool, sha: str, heldout: int):
    return {"workload": DESCRIBE[w.name].replace("fp32", "fp64") if f64 else DESCRIBE[w.name],
            "dims": list(w.dims), "batch": w.batch,
            "sgd_steps_per_step": w.steps, "training_samples_per_step": w.batch * w.steps,
            "heldout_per_step": heldout, "shards": w.shards, "kernel_sources": sha}


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
    ap.add_argument("--wide", default="c5", choices=sorted(DESCRIBE) + ["none"],
                    help="the wide workload measured beside the main one")
    ap.add_argument("--no-peaks", action="store_true", help="skip the device peak measurements")
    ap.add_argument("--copy-calib-mib", type=int, default=0,
                    help="only run a plain device copy of this size 20 times (counter scale)")
    args = ap.parse_args(argv)

    def log(msg):
        print(f"[bench] {msg}", file=sys.stderr, flush=True)

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        return 2

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

    sha = kernel_sources_sha()
    w = W.WORKLOADS[args.workload]
    f64 = args.dtype == "f64"
    res = run_workload(args, w, f64, args.steps, args.warmup, args.cold_reps, log)
    main_fields = summarize(w, f64, res, args.steps, sha, log)

    line = {
        "metric": METRIC,
        "value": main_fields.pop("value"),
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": main_fields.pop("ms_per_step"),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": args.dtype,
        "data": "synthetic",
        "config": config_of(w, f64, sha, int(res["Xh"].shape[0]) if res["Xh"] is not None else 0),
    }
    line.update(main_fields)
    if args.cpu_seconds > 0:
        log(f"timing the CPU reference (~{args.cpu_seconds:.0f} s)")
        line["cpu_baseline"] = cpu_baseline(w, res["X"], res["Y"], res["Xh"], args.cpu_seconds,
                                            args.dtype)
        if w.name in ("c1", "c2"):
            # the same reference on one core, beside the paper's one-core timing
            # of this network shape (section 5); context only
            try:
                from threadpoolctl import threadpool_limits
            except ImportError:
                threadpool_limits = None
            if threadpool_limits is not None:
                with threadpool_limits(limits=1):
                    one = cpu_baseline(w, res["X"], res["Y"], res["Xh"], args.cpu_seconds / 2,
                                       args.dtype)
                one["cores"] = 1
                line["cpu_baseline_1core"] = one
    else:
        line["cpu_baseline"] = None
    del res

    if args.wide != "none" and args.wide != w.name:
        ww = W.WORKLOADS[args.wide]
        wres = run_workload(args, ww, f64, 2, 1, 0, log)
        wide = summarize(ww, f64, wres, 2, sha, log)
        wide.pop("kernels")
        wide = {"workload": config_of(ww, f64, sha, 0)["workload"], "unit": "samples/s",
                "steps": 2, "warmup": 1, **wide}
        if args.cpu_seconds > 0:
            log("timing the CPU reference on one SGD step of the wide workload")
            wide["cpu_baseline"] = cpu_baseline(ww, wres["X"], wres["Y"], None, 0.0, args.dtype,
                                                max_steps=1)
        else:
            wide["cpu_baseline"] = None
        line["wide"] = wide
        del wres
    if not args.no_peaks:
        log("measuring the device peaks")
        line["peaks_measured"] = measure_peaks(torch, nf, dev)
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
