#!/usr/bin/env python3
"""Throughput of one ARC-Top-K + EF21M compressor step (libarctopk) on one MI355X.

A step is one pass of the whole path over one [N, d] batch of synthetic
gradients already resident in HBM: momentum, residual, per-worker sketch,
worker sum, importance, top-K selection, gather + worker sum + error-feedback
update.  Prints ONE JSON line:

  value        gradient elements per second, N*d / (time per step)
  roofline     the streaming sketch kernel (the dominant one): algorithmic
               bytes per launch / its mean duration (HIP events on the
               library's stream over the timed region) against 8 TB/s
  cpu_baseline the CPU oracle on a bounded prefix of the same workload, with
               the threads it used, the host's core count and free memory
  configs      the same report for further workloads timed in the same run
               (by default GPT-2 small beside the 1.1B headline: the two
               configurations the HBM-bandwidth target covers)

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                       [--also NAME,...]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E, vendor peak
DEFAULT_WORKLOAD = "llama1b"    # the 1.1B-parameter configuration
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "sketch_traffic.json")
KERNEL_SOURCE = os.path.join(ROOT, "paper_2510_26709_amd", "csrc", "arc_sketch.hip")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def algorithmic_bytes(w, K_total, compressor="arc"):
    """Bytes the method must move per step (each array touched once).
    sketch_kernel: the first (streaming) stage of the step."""
    bg = w.bytes_per_grad
    Nd = w.N * w.d
    payload = w.payload_elems()
    if compressor == "randk":
        stream = Nd * (bg + 8)                      # grad + h read/write
        keys = 4 * w.m                              # keys written
        select = 4 * 4 * w.m
        gather = payload * (12 * w.N + 4)
        return {"sketch_kernel": stream, "step": stream + keys + select + gather + 4 * K_total}
    if compressor == "topk":
        stream = Nd * (bg + 12) + 4 * w.N * w.m     # + per-node row norms written
        select = 4 * 4 * w.N * w.m
        gather = payload * w.N * 16                 # h, g read, g written, values written
        return {"sketch_kernel": stream, "step": stream + select + gather + 4 * K_total}
    stream = Nd * (bg + 12)                         # grad + h read/write + g read
    sketch_out = 4 * w.N * w.m * w.r                # per-worker sketch written
    reduce_ = 4 * w.N * w.m * w.r + 4 * w.m         # sketch read, importance written
    select = 4 * 4 * w.m                            # importance read by 4 passes
    gather = payload * (12 * w.N + 4)               # h, g read, g written, agg written
    return {"sketch_kernel": stream + sketch_out, "step": stream + sketch_out + reduce_ +
            select + gather + 4 * K_total}


def table1_communication(w, comp, compressor):
    """Values each node sends per step (Table I's column), from the actual
    row counts: uncompressed 2mn (= 2d), ARC-Top-K 2Kn + 2mr, Rand-K 2Kn,
    Top-K (N - 1)(nK + K) with an All-Gather of values and indices."""
    if compressor == "topk":
        K_node, L = comp.K_total // w.N, comp.payload // w.N
        sent = (w.N - 1) * (L + K_node)
    elif compressor == "randk":
        sent = 2 * comp.payload
    else:
        sent = 2 * comp.payload + 2 * comp.m * w.r
    return {"values": sent, "uncompressed": 2 * w.d, "fraction": sent / (2 * w.d)}


def kernel_source_digest(path=KERNEL_SOURCE):
    """sha256 of the kernel source with comments and whitespace removed, so
    that the recorded counters stay valid across comment-only edits."""
    import re
    with open(path) as f:
        src = f.read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    src = re.sub(r"//[^\n]*", "", src)
    src = re.sub(r"\s+", "", src)
    return hashlib.sha256(src.encode()).hexdigest()


def kernel_traffic(w):
    """HBM bytes per launch of the sketch kernel from committed rocprofv3
    counters (FETCH_SIZE and WRITE_SIZE, each scaled by what the counter reads
    for a plain copy of known size), if they were taken on the current kernel
    source; otherwise None."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
        entry = rec.get("workloads", {}).get(w.name)
        if rec.get("kernel_source_digest") != kernel_source_digest() or entry is None:
            return None
        return float(entry["hbm_bytes_per_launch"])
    except (OSError, ValueError, KeyError):
        return None


def _prefix(w, elems):
    """A prefix of the workload of about `elems` coordinates per worker, as
    (d_s, oracle step keyword arguments, description): whole rows of the
    single view with K scaled to the same ratio, or whole tensors with their
    own K."""
    if not w.per_tensor:
        rows = max(1, min(w.m, elems // w.n))
        K_s = max(1, math.ceil(w.mu * rows))
        return rows * w.n, dict(n=w.n, K=K_s), f"first {rows} of {w.m} rows (n={w.n}, K={K_s})"
    views = w.tensor_views()
    take, d_s = [], 0
    for v in views:
        if take and d_s + v[0] * v[1] > elems:
            break
        take.append(v)
        d_s += v[0] * v[1]
    K_s = sum(min(k, r) for r, _, k in take)
    return d_s, dict(tensors=take), f"first {len(take)} of {len(views)} tensors (K={K_s} rows)"


def cpu_baseline(w, grads_dev, seconds_target=12.0, threads=0):
    """Time the CPU oracle on a prefix of the workload (the first coordinates
    of every worker's vector, whole rows or whole tensors) from h = g = 0, on
    the same synthetic gradients (copied from the device); threads > 0 limits
    the oracle's thread count for this run."""
    import oracle
    all_threads = oracle.num_threads()
    if threads > 0:
        oracle.set_num_threads(threads)
    try:
        return _cpu_baseline(w, grads_dev, seconds_target)
    finally:
        oracle.set_num_threads(all_threads)


def _cpu_baseline(w, grads_dev, seconds_target):
    import numpy as np

    import oracle
    threads = oracle.num_threads()

    def run(elems, steps=None, budget=None):
        """Oracle steps on the first `elems` coordinates: `steps` of them, or
        as many as `budget` seconds take (at least 2, at most 16).  The
        gradients cycle through up to four host copies of the device batches."""
        d_s, kw, desc = _prefix(w, elems)
        h = np.zeros((w.N, d_s), np.float32)
        g = np.zeros((w.N, d_s), np.float32)
        grads = []
        for s in range(min(len(grads_dev), steps or 4)):
            gd = grads_dev[s % len(grads_dev)][:, :d_s].contiguous().cpu().numpy()
            grads.append(gd.view(np.uint16) if w.grad_dtype == "bf16" else gd)
        done, t0 = 0, time.perf_counter()
        while True:
            if w.per_tensor:
                oracle.step_tensors(h, g, grads[done % len(grads)], kw["tensors"], r=w.r,
                                    eta=w.eta, seed=w.sketch_seed, t=done)
            else:
                oracle.step(h, g, grads[done % len(grads)], r=w.r, eta=w.eta,
                            seed=w.sketch_seed, t=done, **kw)
            done += 1
            elapsed = time.perf_counter() - t0
            if steps is not None and done >= steps:
                break
            if budget is not None and ((done >= 2 and elapsed >= budget) or done >= 16):
                break
        return elapsed / done, d_s, desc, done

    # calibrate on a small prefix, then size the sample so that two steps
    # take about the time target, and run steps until it is spent
    t1, d1, _, _ = run(1 << 22, steps=1)
    per_elem = t1 / d1
    elems = int(min(w.d, max(d1, seconds_target / 2 / max(per_elem, 1e-15))))
    t_step, d_s, desc, steps = run(elems, budget=seconds_target)
    return {
        "value": w.N * d_s / t_step,
        "unit": "gradient elements/s",
        "cores": threads,
        "kind": "oracle",
        "sample": (f"{desc} per worker: d={d_s} of {w.d}, N={w.N}; {steps} steps from h=g=0, "
                   f"mean s/step={t_step:.3f}"),
    }


def model_step_timing(torch, arc, w, comp, grads, h, g, stream, nb, t0, steps=5, warmup=2):
    """The full EF21M iteration (11a)-(11c): the compressor step, the payload
    added into G, and an Adam update of x over all d coordinates
    (arc_model_step), timed on the library's stream after the main timed
    region.  Reported beside the compressor-only value."""
    dev = h.device
    need = 4 * 4 * w.d + (1 << 30)  # G, x and Adam's m, v, plus slack
    free, _ = torch.cuda.mem_get_info(dev)
    if free < need:
        return {"skipped": f"needs {need / 1e9:.1f} GB of free device memory, "
                           f"{free / 1e9:.1f} GB free beside the compressor's buffers"}
    G, x, m, v = (torch.zeros(w.d, dtype=torch.float32, device=dev) for _ in range(4))
    mc = arc.make_model_config("adam", lr=1e-3, weight_decay=5e-4)
    for k in range(warmup):
        comp.model_step(t0 + k, grads[(t0 + k) % nb], h, g, G, x, mc, m, v)
    stream.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for k in range(steps):
        t = t0 + warmup + k
        comp.model_step(t, grads[t % nb], h, g, G, x, mc, m, v)
    end.record(stream)
    end.synchronize()
    ms = start.elapsed_time(end) / steps
    del G, x, m, v
    opt_bytes = 28 * w.d  # Adam: read G, x, m, v; write x, m, v
    return {"optimizer": "adam", "ms_per_iteration": ms, "steps": steps,
            "gradient_elements_per_s": w.N * w.d / (ms * 1e-3),
            "adam_update_bytes": opt_bytes}


def time_copy(torch, gib, reps):
    """Plain device-to-device copy of a known size (every launch reads and
    writes `gib` GiB once): (bytes copied, mean ms per copy)."""
    nbytes = int(gib * 2**30) // 16 * 16
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(reps):
        dst.copy_(src)
    end.record()
    end.synchronize()
    ms = start.elapsed_time(end) / reps
    del src, dst
    torch.cuda.empty_cache()
    return nbytes, ms


def copy_calibration(torch, gib, reps):
    nbytes, ms = time_copy(torch, gib, reps)
    print(json.dumps({"copy_bytes_read": nbytes, "copy_bytes_written": nbytes, "reps": reps,
                      "ms_per_copy": ms, "GBps_read_plus_write": 2 * nbytes / (ms * 1e-3) / 1e9}),
          flush=True)


def host_info():
    """Host cores and memory at the time of the CPU baseline."""
    info = {"nproc": os.cpu_count()}
    try:
        info["affinity_cpus"] = len(os.sched_getaffinity(0))
    except AttributeError:
        pass
    try:
        with open("/proc/meminfo") as f:
            mem = {ln.split(":")[0]: int(ln.split()[1]) for ln in f if ln.split()[1].isdigit()}
        info["mem_total_GB"] = round(mem["MemTotal"] * 1024 / 1e9, 1)
        info["mem_available_GB"] = round(mem["MemAvailable"] * 1024 / 1e9, 1)
    except (OSError, KeyError, IndexError, ValueError):
        pass
    return info


def measure(torch, arc, synth, w, args, dev, stream, *, with_model, with_cpu):
    """Time one workload: args.warmup untimed steps, then args.steps timed
    steps (the value), as many with the library's stage events (stage
    breakdown, the streaming kernel's mean launch time) and as many with an
    event after each step (spread).  Returns the workload's report."""
    gen = synth.Generator.for_workload(w)
    gdt = torch.int16 if w.grad_dtype == "bf16" else torch.float32
    nb = max(1, min(args.batches, args.steps + args.warmup))
    log(f"[bench] workload={w.name} d={w.d} N={w.N} n={w.n} r={w.r} grad={w.grad_dtype} "
        f"batches={nb}")
    with torch.cuda.stream(stream):
        grads = []
        for b in range(nb):
            x = torch.empty((w.N, w.d), dtype=gdt, device=dev)
            gen.fill_device(b, x, stream)
            grads.append(x)
        h = torch.zeros((w.N, w.d), dtype=torch.float32, device=dev)
        g = torch.zeros((w.N, w.d), dtype=torch.float32, device=dev)
        comp = arc.Compressor(d=w.d, N=w.N, n=w.n, r=w.r, K=w.K_global(), eta=w.eta,
                              seed=w.sketch_seed, grad_dtype=w.grad_dtype,
                              buckets=w.buckets(),
                              tensors=w.tensor_views() if w.per_tensor else None,
                              compressor=args.compressor, device=dev, stream=stream)
        stream.synchronize()
        log(f"[bench] m={comp.m} K_total={comp.K_total}; {comp.describe()}; warmup {args.warmup}")
        for t in range(args.warmup):
            comp.step(t, grads[t % nb], h, g)
        stream.synchronize()
        # The timed steps run without the library's stage events; the same
        # number of steps follows with them, for the per-stage breakdown and
        # the sketch kernel's mean launch time.
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record(stream)
        for k in range(args.steps):
            t = args.warmup + k
            comp.step(t, grads[t % nb], h, g)
        end.record(stream)
        end.synchronize()
        torch.cuda.synchronize()
        total_ms = start.elapsed_time(end)
        arc.arc_timing_enable(comp.ctx, True)
        arc.arc_timing_read(comp.ctx)  # clear
        for k in range(args.steps):
            t = args.warmup + args.steps + k
            comp.step(t, grads[t % nb], h, g)
        stream.synchronize()
        stage_ms, nsteps = arc.arc_timing_read(comp.ctx)
        arc.arc_timing_enable(comp.ctx, False)
        # The spread of single steps: as many steps again, an event after each.
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
        evs[0].record(stream)
        for k in range(args.steps):
            t = args.warmup + 2 * args.steps + k
            comp.step(t, grads[t % nb], h, g)
            evs[k + 1].record(stream)
        evs[-1].synchronize()
        per_step = sorted(evs[k].elapsed_time(evs[k + 1]) for k in range(args.steps))
        model = None
        if with_model:
            model = model_step_timing(torch, arc, w, comp, grads, h, g, stream, nb,
                                      args.warmup + 3 * args.steps)
    ms_per_step = total_ms / args.steps
    stages = {name: stage_ms[i] / max(nsteps, 1) for i, name in enumerate(arc.STAGE_NAMES)}
    log("[bench] %s ms/step %.4f; stages %s" %
        (w.name, ms_per_step, {k: round(v, 4) for k, v in stages.items()}))

    byt = algorithmic_bytes(w, comp.K_total, args.compressor)
    sk_ms = stages["sketch"]
    achieved = byt["sketch_kernel"] / (sk_ms * 1e-3) / 1e9
    # The committed counters cover the ARC sketch kernel only.
    traffic = kernel_traffic(w) if args.compressor == "arc" else None
    step_gbps = byt["step"] / (ms_per_step * 1e-3) / 1e9
    rep = {
        "value": w.N * w.d / (ms_per_step * 1e-3),
        "unit": "gradient elements/s",
        "ms_per_step": ms_per_step,
        "config": {"workload": w.name, "d": w.d, "N": w.N, "n": w.n, "r": w.r, "m": comp.m,
                   "K_rows": comp.K_total, "grad_dtype": w.grad_dtype, "state_dtype": "f32",
                   "eta": w.eta, "mu": w.mu,
                   "buckets": 0 if w.buckets() is None else len(w.buckets()[1]),
                   "view": "per_tensor" if w.per_tensor else "single",
                   "compressor": args.compressor,
                   "tensors": len(w.views) if w.per_tensor else 0,
                   "payload_elems": comp.payload},
        "step_ms_spread": {"median": per_step[len(per_step) // 2] if len(per_step) % 2
                           else 0.5 * (per_step[len(per_step) // 2 - 1] + per_step[len(per_step) // 2]),
                           "min": per_step[0], "max": per_step[-1], "steps": len(per_step),
                           "how": "a separate pass of as many steps, an event after each"},
        "step_hbm_GBps": step_gbps,
        "step_frac_of_peak": step_gbps / HBM_PEAK_GBPS,
        "stage_ms": stages,
        "path": comp.describe(),
        "roofline": {
            "bound": "hbm",
            "kernel": {"arc": "sketch stage: sketch_per_worker_kernel launches (momentum + "
                              "residual + per-worker sketch), plus the general-row kernel "
                              "where the layout has any",
                       "randk": "momentum_vec_kernel (Eq. (11a) over N*d)",
                       "topk": "row-norm stage: sketch_per_worker_kernel in norm mode "
                               "(momentum + residual + per-node squared row norms)",
                       }[args.compressor],
            "achieved": achieved,
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBPS,
            "traffic": traffic,
            "algorithmic_bytes_per_launch": byt["sketch_kernel"],
            "mean_launch_ms": sk_ms,
        },
        "ef21m_iteration": model,
        "communication_per_node": table1_communication(w, comp, args.compressor),
    }
    cpu = None
    if with_cpu:
        log(f"[bench] {w.name} cpu baseline (oracle) ...")
        host = host_info()
        cpu = cpu_baseline(w, grads)
        cpu.update(host)
        log(f"[bench] cpu baseline {cpu['value']:.3e} elements/s on {cpu['cores']} threads")
        if w.name == "tiny":
            # the smallest workload is also reported on one thread
            one = cpu_baseline(w, grads, seconds_target=6.0, threads=1)
            cpu["single_thread"] = {k: one[k] for k in ("value", "unit", "cores", "sample")}
            log(f"[bench] cpu baseline {one['value']:.3e} elements/s on 1 thread")
    rep["cpu_baseline"] = cpu
    comp.close()
    del grads, h, g
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return rep


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--also", default=None,
                    help="comma-separated further workloads timed in the same run and "
                         "reported under 'configs' (default: gpt2s beside llama1b, the "
                         "two configurations the HBM target names; '' for none)")
    ap.add_argument("--compressor", default="arc", choices=["arc", "randk", "topk"],
                    help="ARC-Top-K, or a comparison compressor of Table I in the same step")
    ap.add_argument("--batches", type=int, default=4,
                    help="distinct gradient batches kept resident and cycled")
    ap.add_argument("--workers", type=int, default=0,
                    help="override the workload's simulated worker count N (1: one "
                         "rank's share of a multi-GPU run, the streaming stage at its "
                         "real shape with nothing to sum over workers)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-model-step", action="store_true",
                    help="skip the extra timing of the full EF21M iteration with Adam")
    ap.add_argument("--print-kernel-digest", action="store_true",
                    help="print the digest of the sketch kernel source and exit")
    ap.add_argument("--copy-calibration", type=float, default=0.0, metavar="GIB",
                    help="instead of the compressor, time a plain device copy of GIB "
                         "gibibytes (empirical bandwidth ceiling; counter calibration)")
    args = ap.parse_args()
    if args.print_kernel_digest:
        print(kernel_source_digest())
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one MI355X: the compressor path here is single-GPU "
              "(workers are simulated on the device); run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    if args.steps < 1 or args.warmup < 0:
        ap.error("--steps must be at least 1 and --warmup at least 0")

    import synth
    if args.workload not in synth.WORKLOADS:
        ap.error(f"unknown workload {args.workload!r}")
    if args.also is None:
        also = ["gpt2s"] if args.workload == "llama1b" and args.compressor == "arc" \
            and args.workers <= 0 else []
    else:
        also = [a for a in args.also.split(",") if a]
    for a in also:
        if a not in synth.WORKLOADS:
            ap.error(f"unknown workload {a!r} in --also")

    import torch

    if args.copy_calibration > 0:
        copy_calibration(torch, args.copy_calibration, max(args.steps, 1))
        return

    import paper_2510_26709_amd as arc

    def sized(name):
        w = synth.WORKLOADS[name]
        if args.workers > 0 and args.workers != w.N:
            import dataclasses
            w = dataclasses.replace(w, name=f"{w.name}_N{args.workers}", N=args.workers)
        return w

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.Stream(dev)
    w = sized(args.workload)
    main_rep = measure(torch, arc, synth, w, args, dev, stream,
                       with_model=not args.no_model_step, with_cpu=not args.no_cpu_baseline)
    others = {}
    for name in also:
        others[name] = measure(torch, arc, synth, sized(name), args, dev, stream,
                               with_model=False, with_cpu=not args.no_cpu_baseline)

    # An empirical ceiling beside the vendor peak: a plain 2 GiB device copy
    # (torch's copy_, the runtime's copy kernel), timed in the same process.
    nbytes, copy_ms = time_copy(torch, 2, 10)
    copy_gbps = 2 * nbytes / (copy_ms * 1e-3) / 1e9
    main_rep["roofline"]["copy_ceiling"] = {
        "GBps": copy_gbps, "bytes_read_plus_written": 2 * nbytes,
        "kernel": "device-to-device copy (torch copy_)",
        "achieved_over_copy": main_rep["roofline"]["achieved"] / copy_gbps}

    out = {
        "metric": "arc_step gradient elements/s and achieved HBM GB/s (% of peak), 1 MI355X",
        "value": main_rep["value"],
        "unit": "gradient elements/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": main_rep["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        # the arithmetic type of every step; the gradients' storage type is
        # config.grad_dtype
        "dtype": "f32",
        "data": "synthetic",
    }
    out.update({k: v for k, v in main_rep.items() if k not in ("value", "unit", "ms_per_step")})
    out["paper_context"] = {
        "what": "mean wall-clock time of a whole LLaMA-1B pre-training iteration with Adam "
                "(Sec. VI, Table 5): 4x NVIDIA A100 40GB, NCCL over shared memory, "
                "NVLink disabled, mu=0.2, r=4; not comparable to this single-GPU "
                "compressor step",
        "s_per_iteration": {"dense": 3.0854, "topk": 2.9628, "randk": 0.9581,
                            "arc_topk": 1.2130},
        "arc_vs_dense": -0.6069,
    }
    if others:
        out["configs"] = others
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
