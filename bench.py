"""Benchmark of the per-sequence sampling step on one MI355X.

One step = one albireo_sample call over one batch: B=256 rows at V=152064 (the Qwen-2.5 vocabulary)
in bf16, with repetition/frequency/presence penalties from 2048-token histories, temperature 0.7,
top_k 40, top_p 0.95 -- the configuration the headline metric is quoted on.  Inputs are synthetic
(workloads.generate(3)) and resident in HBM before the timed region; the call rotates over enough
copies (>= 1 GiB) that every step reads its logits from HBM rather than from the 256 MB MALL.

Timing protocol: REPS (5) repetitions of --steps steps each; before each repetition a spin kernel
holds the stream while the host enqueues the steps, so the HIP events around the steps time the GPU,
not the host's enqueue rate.  The reported step time is the median repetition, with the spread.

Prints one JSON line: rows/s (whole job), ms per step, the roofline entry of the dominant kernel
(algorithmic bytes per launch / its average launch time from HIP events on its stream, against the
8 TB/s HBM peak), the device's clock and memory figures as the runtime reports them, and the CPU
oracle timed on a bounded sample of the same workload (all host threads, and one thread).
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

METRIC = "sampled rows/sec + achieved HBM GB/s (% of peak), B=256 V=152064 bf16"
HBM_PEAK_GBS = 8000.0


def algorithmic_bytes(w) -> int:
    """Bytes the method itself must move per call: logits once, history ids, CSR offsets, the seven
    per-row parameter arrays, the uniforms, and the outputs (ids, logprobs, top-n)."""
    b = w.B * w.V * w.itemsize
    if w.hist_ids is not None:
        b += w.hist_ids.size * 4 + (w.B + 1) * 8
    b += 7 * w.B * 4 + w.B * 4  # parameters + uniforms
    b += w.B * 4 + w.B * 4      # ids + logprobs
    b += w.B * w.n_top * 8      # top-n ids + logprobs
    return int(b)


# per workload, the file tag of its profile summaries; per route, the kernels timed and the sources
# they are compiled from (a summary taken on other sources gives no traffic figure)
PROFILE_TAGS = {1: "C1_B4_V32000_f32", 2: "C2_B64_V128256_bf16", 3: "C3_B256_V152064_bf16",
                4: "C4_B512_V152064_f32", 5: "C5_B1024_V256000_bf16"}
_CSRC = os.path.join(ROOT, "paper_2606_01927_amd", "csrc")
_HDR = os.path.join(ROOT, "include", "albireo.h")
ROUTE_KERNELS = {
    1: ("k_sample", [os.path.join(_CSRC, "albireo.hip"), os.path.join(_CSRC, "common.h"), _HDR]),
    2: ("k_stream_k_resolve", [os.path.join(_CSRC, "stream.hip"), os.path.join(_CSRC, "stream.h"),
                               os.path.join(_CSRC, "common.h"), _HDR]),
}
REPS = 5
# hipDeviceAttribute_t values of this ROCm (hip_runtime_api.h)
HIP_ATTR = {"clock_khz": 5, "memory_bus_bits": 59, "memory_clock_khz": 60, "l2_bytes": 19, "cus": 63}


def device_figures(dev: int = 0) -> dict:
    """What the HIP runtime reports for the device: its name, CU count, peak shader clock, memory clock
    and bus width (and the DRAM bandwidth they imply at two transfers per clock), L2 size."""
    import ctypes

    import torch

    props = torch.cuda.get_device_properties(dev)
    out = {"name": props.name, "gcn_arch": props.gcnArchName, "total_memory_bytes": props.total_memory}
    try:
        hip = ctypes.CDLL("libamdhip64.so")
        for k, attr in HIP_ATTR.items():
            v = ctypes.c_int(0)
            if hip.hipDeviceGetAttribute(ctypes.byref(v), attr, dev) == 0:
                out[k] = v.value
    except OSError:
        pass
    return out


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def kernel_source_hash(route: int) -> str:
    h = hashlib.sha256()
    for p in ROUTE_KERNELS[route][1]:
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def traffic_file(cfg: int, route: int) -> str:
    return os.path.join(ROOT, "profiles", "%s_%s_traffic.txt" % (ROUTE_KERNELS[route][0], PROFILE_TAGS[cfg]))


def measured_traffic(cfg: int, route: int):
    """HBM bytes per step (every launch of the route) from the committed rocprofv3 --pmc summary
    (FETCH_SIZE + WRITE_SIZE, each scaled by what the counter reads for a copy of known size), or
    None when the summary is missing or was taken on different kernel sources."""
    if route not in ROUTE_KERNELS:
        return None
    try:
        with open(traffic_file(cfg, route)) as f:
            kv = dict(line.split(":", 1) for line in f if ":" in line and not line.startswith("#"))
    except OSError:
        return None
    kv = {k.strip(): v.strip() for k, v in kv.items()}
    if kv.get("kernel_source_sha256") != kernel_source_hash(route):
        return None
    try:
        return float(kv["traffic_bytes_per_step"])
    except (KeyError, ValueError):
        return None


def copy_calibration(mib: int):
    """One elementwise copy of a known size (mib MiB read, mib MiB written), launched before the
    timed region so that a counter run of this script can scale FETCH_SIZE / WRITE_SIZE."""
    import torch

    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    torch.mul(src, 1.0, out=dst)
    torch.cuda.synchronize()
    del src, dst


def cpu_baseline(w, seconds_target: float = 15.0, nthreads: int = 0) -> dict:
    """The oracle as it stands, on a bounded sample of rows of the same workload, on nthreads host
    threads (0: all of them)."""
    import numpy as np

    import oracle

    oracle.build(force=False)
    if nthreads <= 0:
        nthreads = oracle.max_threads()
    rows_done = 0
    t0 = time.perf_counter()
    n = max(nthreads, 8)
    lo = 0
    while True:
        hi = min(lo + n, w.B)
        oracle.sample(w.row_slice(lo, hi), nthreads=nthreads)
        rows_done += hi - lo
        lo = hi % w.B
        el = time.perf_counter() - t0
        if el >= seconds_target or rows_done >= 64 * w.B:
            break
        n = min(w.B, n * 2)
    el = time.perf_counter() - t0
    del np
    return {"value": rows_done / el, "unit": "rows/s", "cores": nthreads, "kind": "oracle",
            "sample": "%d rows of the B=256 V=152064 bf16 workload (%.1f s)" % (rows_done, el)}


def step_extras(alb, w, copies, p, ws, stream, reps: int = 50) -> dict:
    """Per-call times (HIP events on the launch stream) of the decoding-step extras on the same
    workload: sampling with device-generated uniforms and the fused backfill (one launch), and the
    standalone generator and scatter kernels for the same B."""
    import torch

    dev = copies[0].device
    B, V = w.B, w.V
    seq = torch.arange(B, dtype=torch.int64, device=dev) * 7919 + 13
    nxt = torch.zeros(B, dtype=torch.int32, device=dev)
    dest = torch.randperm(B, device=dev).to(torch.int32)
    ids = torch.zeros(B, dtype=torch.int32, device=dev)
    outs = (ids, torch.empty(B, dtype=torch.float32, device=dev),
            torch.empty((B, w.n_top), dtype=torch.int32, device=dev),
            torch.empty((B, w.n_top), dtype=torch.float32, device=dev), torch.empty(B, dtype=torch.int32, device=dev))

    def timed(fn):
        for i in range(5):
            fn(i)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for i in range(reps):
            fn(i)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / reps

    t_step = timed(lambda i: alb.sample_step(copies[i % len(copies)], 2026, i, seq, p, n_top=w.n_top, V=V,
                                             next_tokens=nxt, backfill_dest=dest, workspace=ws, stream=stream,
                                             out=outs))
    t_rng = timed(lambda i: alb.philox_uniforms(2026, i, seq, stream=stream))
    t_bf = timed(lambda i: alb.backfill(ids, dest, nxt, stream=stream))
    res = {"sample_step_us": t_step, "philox_uniforms_us": t_rng, "backfill_us": t_bf,
           "note": "sample_step = sampling with device uniforms and the fused backfill, one launch"}
    # the same rows as one worker of t = 8 receives them from the all-to-all: [t][B][V / t] blocks
    t = 8
    L = alb.shard_len_for(V, t, copies[0].dtype)
    if L * t == V and copies[0].stride(0) == V:
        recvs = [c.view(B, t, L).permute(1, 0, 2).contiguous() for c in copies]
        uni = torch.rand(B, device=dev)
        res["sample_sharded_t8_us"] = timed(
            lambda i: alb.sample_sharded(recvs[i % len(recvs)], V=V, uniforms=uni, params=p, n_top=w.n_top,
                                         workspace=ws, stream=stream, out=outs))
        del recvs
    return res


def other_configs(alb, dev, reps: int = 20) -> dict:
    """Per-call time of the sampling step on the four other workloads at their full sizes (HIP events
    over back-to-back calls, logits rotated over copies of at least 512 MiB so that they come from
    HBM), with the algorithmic bytes per call against the 8 TB/s peak."""
    import torch

    import workloads
    from workloads.device import to_device

    res = {}
    stream = torch.cuda.current_stream()
    for cfg in (1, 2, 4, 5):
        w = workloads.generate(cfg)
        logits0, u, p = to_device(w, device=dev)
        nbytes = logits0.numel() * logits0.element_size()
        ncopy = max(2, -(-(1 << 29) // nbytes))
        copies = [logits0] + [logits0.clone() for _ in range(ncopy - 1)]
        ws = alb.Workspace(dev)
        outs = [torch.empty(w.B, dtype=torch.int32, device=dev), torch.empty(w.B, dtype=torch.float32, device=dev),
                torch.empty((w.B, max(w.n_top, 1)), dtype=torch.int32, device=dev),
                torch.empty((w.B, max(w.n_top, 1)), dtype=torch.float32, device=dev),
                torch.empty(w.B, dtype=torch.int32, device=dev)]
        call = alb.PreparedSample(logits0, u, p, w.n_top, w.V, outs, workspace=ws, stream=stream)
        ptrs = [c.data_ptr() for c in copies]
        for i in range(3):
            call(ptrs[i % ncopy])
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        torch.cuda._sleep(int(4e-3 * 2.4e9))  # holds the stream while the calls are enqueued
        e0.record(stream)
        for i in range(reps):
            call(ptrs[i % ncopy])
        e1.record(stream)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / reps
        alg = algorithmic_bytes(w)
        res[w.name] = {"us_per_call": us, "rows_per_s": w.B / (us * 1e-6), "algorithmic_bytes": alg,
                       "hbm_gbs": alg / (us * 1e-6) / 1e9, "frac_of_peak": alg / (us * 1e-6) / 1e9 / HBM_PEAK_GBS}
        print("config %d: %.1f us per call" % (cfg, us), file=sys.stderr, flush=True)
        del copies, logits0, ws, call
        torch.cuda.empty_cache()
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--config", type=int, default=3, help="workload index (3 is the headline one)")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the per-call times of the other four workloads after the main loop")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the timing of the step extras (device uniforms, backfill) after the main loop")
    ap.add_argument("--rows", choices=("as-drawn", "top-p-only", "plain"), default="as-drawn",
                    help="per-row filters: as the workload draws them, top-k and min-p off (the nucleus "
                         "alone), or every filter off (a draw over the whole kept row)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="launch one elementwise copy of this many MiB before the timed region (for "
                         "scaling hardware byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the sampling step of one rank's row-share; --gpus %d is not "
              "supported in this build" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2606_01927_amd as alb
    import workloads
    from workloads.device import to_device

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.calib_copy_mib > 0:
        copy_calibration(args.calib_copy_mib)
    w = workloads.generate(args.config)
    if args.rows != "as-drawn":
        w.top_k = None
        w.min_p = None
        if args.rows == "plain":
            w.top_p = None
        w.name += " [rows: %s]" % args.rows
    logits0, u, p = to_device(w, device=dev)
    nbytes = logits0.numel() * logits0.element_size()
    ncopy = max(2, -(-(1 << 30) // nbytes))
    copies = [logits0] + [logits0.clone() for _ in range(ncopy - 1)]
    ws = alb.Workspace(dev)
    stream = torch.cuda.current_stream()
    B, V = w.B, w.V
    outs = [torch.empty(B, dtype=torch.int32, device=dev), torch.empty(B, dtype=torch.float32, device=dev),
            torch.empty((B, w.n_top), dtype=torch.int32, device=dev),
            torch.empty((B, w.n_top), dtype=torch.float32, device=dev),
            torch.empty(B, dtype=torch.int32, device=dev)]

    call = alb.PreparedSample(logits0, u, p, w.n_top, V, outs, workspace=ws, stream=stream)
    ptrs = [c.data_ptr() for c in copies]

    def step(i):
        call(ptrs[i % ncopy])

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # host enqueue rate, to size the spin that keeps the launch queue ahead of the GPU
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(i)
    host_enqueue_s = time.perf_counter() - t0
    torch.cuda.synchronize()
    spin_cycles = int(max(2e-3, 3.0 * host_enqueue_s) * 2.4e9)

    # REPS repetitions; HIP events on the launch stream bracket the steps of each (the spin kernel ahead
    # of the first event holds the stream while the host enqueues them all)
    reps_ms = []
    wall = 0.0
    for rep in range(REPS):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        torch.cuda._sleep(spin_cycles)
        t0 = time.perf_counter()
        e0.record(stream)
        for i in range(args.steps):
            step(i)
        e1.record(stream)
        enq = time.perf_counter() - t0
        torch.cuda.synchronize()
        wall += enq
        reps_ms.append(e0.elapsed_time(e1) / args.steps)
    order = sorted(reps_ms)
    ms_per_step = order[len(order) // 2]
    launch_us = ms_per_step * 1e3
    alg = algorithmic_bytes(w)
    achieved = alg / (launch_us * 1e-6) / 1e9
    rows_per_s = B / (ms_per_step * 1e-3)
    # the kernels the library routes this shape to (the same host decision the call takes)
    route = alb.sample_route(B, V, logits0.dtype, p)
    kernel = {alb.ROUTE_ONE_WORKGROUP: "k_sample (one launch per step)",
              alb.ROUTE_STREAM: "k_stream, k_resolve, k_gen_a/b/s/c (six launches per step; the time is all)",
              alb.ROUTE_COOPERATIVE: "k_sample_multi (one cooperative launch per step)"}[route]

    res = {
        "metric": METRIC,
        "value": rows_per_s,
        "unit": "rows/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "reps": REPS,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "B": B, "V": V, "n_top": w.n_top,
                   "input_copies": ncopy, "input_bytes_rotated": ncopy * nbytes},
        "hbm_gbs": alg / (ms_per_step * 1e-3) / 1e9,
        "hbm_frac_of_peak": alg / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS,
                     "traffic": measured_traffic(args.config, route) if args.rows == "as-drawn" else None,
                     "kernel": kernel,
                     "algorithmic_bytes": alg,
                     "launch_us_avg": launch_us},
        "timing": {"ms_per_step_reps": reps_ms, "spread_ms": [order[0], order[-1]],
                   "host_enqueue_us_per_step": wall * 1e6 / (REPS * args.steps),
                   "spin_cycles_ahead": spin_cycles},
        "device": device_figures(0),
        "wall_s": wall,
    }
    if not args.no_extras:
        res["step_extras"] = step_extras(alb, w, copies, p, ws, stream)
    if not args.no_configs and args.config == 3:
        res["other_configs"] = other_configs(alb, dev)
    if not args.no_cpu:
        res["cpu_baseline"] = cpu_baseline(w)
        res["cpu_baseline"]["cpu_model"] = cpu_model()
        one = cpu_baseline(w, seconds_target=10.0, nthreads=1)
        res["cpu_baseline"]["one_thread"] = {"value": one["value"], "unit": one["unit"], "sample": one["sample"]}
    print(json.dumps(res))


if __name__ == "__main__":
    main()
