"""Benchmark: simulated request-steps per second of A_min on 4096 instances x
n=1000 (M=16384), one MI355X.

A step is one full simulation of the whole batch (every instance from t=0 to
its last completion) through the C ABI: the per-instance preparation kernel
and the simulation kernel.  Inputs are resident in HBM before timing starts.

Prints one JSON line.  Also reports the roofline of the simulation kernel
(int32 VALU lane-operations: 6 per simulated request-step, the completion
compare, the projected-memory add and the head test's compare, max, end
compare and add for that run)
and the CPU oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# MI355X: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz = int32 VALU lane-operations per second
N_CU = 256
CLOCK_HZ = 2.4e9
PEAK_INT32_LANE_OPS = N_CU * 4 * 16 * CLOCK_HZ
PEAK_LDS_BYTES = 256 * 128 * 2.4e9
# widest LDS access of the simulation kernel: ds_read_b64 over 64 lanes
LDS_BYTES_PER_INST_MAX = 64 * 8
# algorithmic int32 lane-operations per simulated request-step: completion compare,
# projected-memory add, and the head test's planned-end compare, max, end compare, add
OPS_PER_REQUEST_STEP = 6
METRIC = "simulated request-steps/sec (A_min, 4096×n=1000) + % VALU/LDS roofline"
SIM_KERNEL = "k_simulate"


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    # the kernel sources and the build script (its compiler flags shape the code)
    for p in ("paper_2508_14544_amd/csrc/sched_kernels.hip", "paper_2508_14544_amd/csrc/sim_device.hpp",
              "paper_2508_14544_amd/csrc/sched_wide.hip", "paper_2508_14544_amd/csrc/sched_group.hip",
              "paper_2508_14544_amd/csrc/wave.hpp",
              "paper_2508_14544_amd/build.py"):
        h.update(open(os.path.join(ROOT, p), "rb").read())
    return h.hexdigest()[:16]


def load_profile(workload: str, algo: str) -> dict:
    """The machine-readable figures of the committed rocprofv3 summary of this
    kernel and workload, if it is still current (same kernel source); else {}."""
    path = os.path.join(ROOT, "profiles", f"{SIM_KERNEL}_{algo}_{workload}.md")
    if not os.path.exists(path):
        return {}
    text = open(path).read()
    if "```json" not in text:
        return {}
    block = text.split("```json", 1)[1].split("```", 1)[0]
    d = json.loads(block)
    if d.get("kernel_source_hash") != kernel_source_hash():
        return {}
    return d


def load_traffic(workload: str, algo: str):
    """HBM bytes per launch from the committed rocprofv3 --pmc summary (None if
    absent or stale)."""
    return load_profile(workload, algo).get("hbm_bytes_per_launch")


def load_hardware_fraction(workload: str, algo: str, kernel_ms: float = 0.0):
    """The chip's vector lane-cycle fraction over one launch, VALUBusy x
    VALUUtilization from the committed rocprofv3 --pmc summary (None if absent
    or stale): the issued-work counterpart of the algorithmic fraction.  With
    the launch's duration, also an upper bound on its LDS bandwidth: every LDS
    instruction of the kernel (SQ_INSTS_LDS) moves at most 8 B per lane of a
    wave64 (ds_read_b64 is its widest), against the LDS peak."""
    d = load_profile(workload, algo)
    if "valu_busy_pct" not in d:
        return None
    out = {"valu_lane_cycles": d["valu_busy_pct"] * d["valu_utilization_pct"] / 1e4,
           "valu_busy_pct": d["valu_busy_pct"], "valu_utilization_pct": d["valu_utilization_pct"],
           "lds_bank_conflict_pct": d.get("lds_bank_conflict_pct"),
           "source": "rocprofv3 --pmc VALUBusy VALUUtilization (committed summary of this kernel source)"}
    if "salu_insts_per_launch" in d and kernel_ms > 0:
        # a CU issues at most one scalar and one vector instruction per cycle
        cu_cycles = N_CU * CLOCK_HZ * kernel_ms / 1e3
        out["issue_per_cu_cycle"] = {"salu": d["salu_insts_per_launch"] / cu_cycles,
                                     "valu": d["valu_insts_per_launch"] / cu_cycles, "limit": 1.0}
    if "lds_insts_per_launch" in d and kernel_ms > 0:
        lds_bytes = d["lds_insts_per_launch"] * LDS_BYTES_PER_INST_MAX
        out["lds_bytes_per_launch_max"] = lds_bytes
        out["lds_frac_max"] = lds_bytes / (kernel_ms * 1e-3) / PEAK_LDS_BYTES
    return out


def probe_peaks():
    """The int32 VALU and LDS throughput this GPU delivers, from the probe
    kernels of libschedprobe.so (next to the published peaks the roofline
    uses); None if the probe library is not built."""
    import ctypes
    path = os.path.join(ROOT, "paper_2508_14544_amd", "libschedprobe.so")
    if not os.path.exists(path):
        return None
    lib = ctypes.CDLL(path)
    for f in (lib.sched_probe_valu, lib.sched_probe_lds):
        f.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_double)]
        f.restype = ctypes.c_int
    v, l = ctypes.c_double(0), ctypes.c_double(0)
    if lib.sched_probe_valu(4000, ctypes.byref(v)) != 0 or lib.sched_probe_lds(20000, ctypes.byref(l)) != 0:
        return None
    return {"int32_valu_TOPs": v.value / 1e12, "int32_valu_frac_of_published": v.value / PEAK_INT32_LANE_OPS,
            "lds_read_TBs": l.value / 1e12, "lds_frac_of_published": l.value / PEAK_LDS_BYTES}


def pipelined(db, algo, kw, ref_out, steps: int, nstreams: int = 3):
    """Back-to-back batches with `nstreams` in flight (each on its own stream
    with its own output buffers): the tail of one batch, where most SIMDs wait
    for its slowest instances, overlaps the next batch.  Returns the time per
    batch over `steps` batches and whether every stream's outputs equal the
    serial run's."""
    import torch
    from paper_2508_14544_amd import binding as B
    kw = {k: v for k, v in kw.items() if k != "stream"}
    streams = [torch.cuda.Stream() for _ in range(nstreams)]
    outs = [B.alloc_results(db) for _ in range(nstreams)]
    for i in range(nstreams):   # warm-up: one batch per stream
        B.simulate_into(db, algo, outs[i], stream=streams[i], **kw)
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    main = torch.cuda.current_stream()
    start.record(main)
    for st in streams:
        st.wait_event(start)
    for i in range(steps):
        B.simulate_into(db, algo, outs[i % nstreams], stream=streams[i % nstreams], **kw)
    for st in streams:
        main.wait_stream(st)
    end.record(main)
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / steps
    same = all(all(torch.equal(o[k], ref_out[k]) for k in o if o[k] is not None) for o in outs)
    return ms, same


def pinned_transfers(db, out, stream, reps: int = 3):
    """Median milliseconds of copying the batch's inputs from pinned host
    buffers into the resident device tensors, and the outputs back into pinned
    buffers (new pinned tensors; timed with events on the copy stream)."""
    import torch
    srcs = [t for t in (db.offsets, db.arrival, db.prompt, db.output, db.lower, db.upper, db.priority)
            if t is not None]
    outs = [v for v in out.values() if v is not None]
    h_in = [torch.empty(t.shape, dtype=t.dtype, pin_memory=True) for t in srcs]
    for h, t in zip(h_in, srcs):
        h.copy_(t)
    h_out = [torch.empty(v.shape, dtype=v.dtype, pin_memory=True) for v in outs]

    def timed(pairs):
        ms = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record(stream)
            for dst, src in pairs:
                dst.copy_(src, non_blocking=True)
            e1.record(stream)
            torch.cuda.synchronize()
            ms.append(e0.elapsed_time(e1))
        return float(sorted(ms)[len(ms) // 2])

    with torch.cuda.stream(stream):
        return timed(list(zip(srcs, h_in))), timed(list(zip(h_out, outs)))


class HipEvent:
    """A raw hipEvent_t (timing enabled), recorded by the library on its launch stream."""
    _hip = None

    def __init__(self):
        import ctypes
        if HipEvent._hip is None:
            lib = ctypes.CDLL("libamdhip64.so")
            lib.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
            lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
            lib.hipEventDestroy.argtypes = [ctypes.c_void_p]
            HipEvent._hip = lib
        self.h = ctypes.c_void_p()
        if HipEvent._hip.hipEventCreate(ctypes.byref(self.h)) != 0:
            raise RuntimeError("hipEventCreate failed")
        self.cuda_event = self.h.value

    def elapsed_ms(self, end: "HipEvent") -> float:
        import ctypes
        ms = ctypes.c_float()
        if HipEvent._hip.hipEventElapsedTime(ctypes.byref(ms), self.h, end.h) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(ms.value)

    def __del__(self):
        try:
            HipEvent._hip.hipEventDestroy(self.h)
        except Exception:
            pass


def host_cpus():
    """Logical CPUs this process may run on, the oracle pool size (that count,
    capped by OMP_NUM_THREADS where the host sets one: a share of a larger
    machine), and the CPU model from /proc/cpuinfo."""
    avail = len(os.sched_getaffinity(0))
    env = os.environ.get("OMP_NUM_THREADS", "")
    threads = min(avail, int(env)) if env.isdigit() and int(env) > 0 else avail
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return avail, threads, model


def cpu_baseline(batch, algo, g_out, target_s: float, threads: int):
    """Time the oracle on a bounded sample of instances; check parity on it."""
    import numpy as np
    from oracle import oracle as O

    K = batch.num_instances
    probe = list(range(0, K, max(1, K // threads)))[:threads]
    t0 = time.perf_counter()
    O.simulate_batch(batch, algo, instances=probe, threads=threads)
    per = (time.perf_counter() - t0) / max(1, len(probe))  # wall per instance with `threads` in flight
    want = int(max(threads, min(K, target_s / max(per, 1e-6))))
    # evenly spread over the batch (its instances come in blocks of alpha)
    sample = sorted({int(round(i * (K - 1) / max(1, want - 1))) for i in range(want)}) if want < K else list(range(K))
    t0 = time.perf_counter()
    ref = O.simulate_batch(batch, algo, instances=sample, threads=threads)
    wall = time.perf_counter() - t0
    rs = int(ref["request_steps"].sum())
    ok = (g_out["tel"][sample].tolist() == ref["tel"].tolist()
          and g_out["request_steps"][sample].tolist() == ref["request_steps"].tolist()
          and g_out["status"][sample].tolist() == ref["status"].tolist())
    sel = np.concatenate([np.arange(batch.offsets[k], batch.offsets[k + 1]) for k in sample])
    ok = ok and np.array_equal(g_out["completion"][sel], ref["completion"])
    ok = ok and np.array_equal(g_out["evictions"][sel], ref["evictions"])
    # algorithmic work count (untimed pass with the oracle's counters) on part of the sample
    sub = sample[::3]
    st = O.simulate_batch(batch, algo, instances=sub, threads=threads, stats=True)
    work = sum(x["work"] for x in st["stats"])
    w_ratio = work / max(1, int(st["request_steps"].sum()))
    avail, _, model = host_cpus()
    return {
        "value": rs / wall, "unit": "request-steps/s", "cores": threads, "kind": "oracle",
        "threads": threads, "cpus_available": avail, "cpu_model": model,
        "sample": (f"{len(sample)} of {K} instances ("
                   + ("evenly spaced in index order" if len(sample) < K else "all")
                   + f"), {rs} request-steps in {wall:.1f} s on {threads} host threads"),
    }, bool(ok), (w_ratio, len(sub))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="batch4096_n1000_m16384")
    ap.add_argument("--algo", default="amin", choices=["amin", "amax", "hsf", "aell", "adaptive", "arandom"])
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--running-capacity", type=int, default=0)
    ap.add_argument("--workgroup-waves", type=int, default=0,
                    help="2 or 4: every instance simulated by a workgroup of that many waves (A_max, A_min, H-SF)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target CPU time of the oracle sample")
    ap.add_argument("--cpu-threads", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-peak-probe", action="store_true", help="skip the VALU/LDS throughput probes")
    # off by default, so that every launch of the default run is one batch at a
    # time and a kernel trace of it averages the same launches as `roofline`
    ap.add_argument("--pipeline-streams", type=int, default=0,
                    help="batches in flight for the 'pipelined' figure (<= 1: skip it; e.g. 3)")
    ap.add_argument("--instances", default="",
                    help="comma-separated instance ids: simulate only these (critical-path profiling)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after timing, run device copies of this size (for rocprofv3 counter calibration)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only; the instances of a batch are "
                                   "independent, so several GPUs would each simulate a contiguous share "
                                   "of them and gather the per-instance outputs at the end"}))
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2508_14544_amd import binding as B
    from paper_2508_14544_amd import workloads as W

    B.load_library()
    algo = B.ALGOS[args.algo]
    batch = W.generate(args.workload, args.seed)
    subset = [int(x) for x in args.instances.split(",") if x.strip()]
    if subset:
        batch = batch.subset(subset)
    if args.algo == "arandom":   # A_random's random order is an input, drawn by the generator
        batch = W.with_random_order(batch, args.seed)
    dev = torch.device("cuda:0")
    torch.cuda.synchronize()
    h0 = time.perf_counter()
    db = B.to_device(batch, dev)
    torch.cuda.synchronize()
    h2d_ms = (time.perf_counter() - h0) * 1e3
    h2d_bytes = sum(int(t.numel()) * t.element_size() for t in
                    (db.offsets, db.arrival, db.prompt, db.output, db.lower, db.upper, db.priority)
                    if t is not None)
    out = B.alloc_results(db)
    stream = torch.cuda.current_stream(dev)
    kw = dict(stream=stream, running_capacity=args.running_capacity, workgroup_waves=args.workgroup_waves)

    for _ in range(args.warmup):
        B.simulate_into(db, algo, out, **kw)
    torch.cuda.synchronize()

    ev = [(HipEvent(), HipEvent()) for _ in range(args.steps)]
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t_start.record(stream)
    for i in range(args.steps):
        B.simulate_into(db, algo, out, event_before=ev[i][0], event_after=ev[i][1], **kw)
    t_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    step_ms = t_start.elapsed_time(t_end) / args.steps
    sim_ms = [a.elapsed_ms(b) for a, b in ev]
    sim_avg_ms = sum(sim_ms) / len(sim_ms)

    pipe_ms, pipe_same = (pipelined(db, algo, kw, out, args.steps, args.pipeline_streams)
                          if args.pipeline_streams > 1 else (None, None))
    d0 = time.perf_counter()
    g = {k: (None if v is None else v.cpu().numpy()) for k, v in out.items()}
    d2h_ms = (time.perf_counter() - d0) * 1e3
    d2h_bytes = sum(int(v.numel()) * v.element_size() for v in out.values() if v is not None)
    pinned = pinned_transfers(db, out, stream)
    status_ok = bool((g["status"] == 0).all())
    rs = int(g["request_steps"].sum())
    value = rs / (step_ms / 1e3)

    if args.calib_copy_mib > 0:
        nbytes = args.calib_copy_mib << 20
        src = torch.empty(nbytes // 4, dtype=torch.int32, device=dev).fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()

    achieved = OPS_PER_REQUEST_STEP * rs / (sim_avg_ms / 1e3)
    # (the committed profiles are of the default launches, one wave per instance)
    profiled = args.workgroup_waves <= 1 and not args.running_capacity
    traffic = load_traffic(args.workload, args.algo) if profiled else None
    measured_peaks = None if args.no_peak_probe else probe_peaks()
    result = {
        "metric": METRIC,
        "value": value,
        "unit": "request-steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": step_ms,
        # the same step counted in instances advanced by one step (sum of makespans)
        "instance_steps_per_s": int(g["makespan"].astype(np.int64).sum()) / (step_ms / 1e3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic",
        "config": {
            "workload": args.workload,
            "algo": {"amin": "A_min", "amax": "A_max", "hsf": "H-SF", "aell": "A_l",
                     "adaptive": "adaptive A_min/A_l", "arandom": "A_random"}[args.algo],
            "instances": batch.num_instances,
            "requests_per_instance": W.WORKLOADS[args.workload].n,
            "M": batch.M,
            "seed": args.seed,
            "request_steps_per_step": rs,
            "instance_steps_per_step": int(g["makespan"].astype(np.int64).sum()),
            "requests_x_makespan_per_step": int((np.diff(batch.offsets) * g["makespan"].astype(np.int64)).sum()),
            "instances_subset": subset or None,
            "workgroup_waves": args.workgroup_waves or 1,
            "instances_per_policy": ({"A_min": int((g["algo_used"] == B.AMIN).sum()),
                                      "A_l": int((g["algo_used"] == B.AELL).sum())}
                                     if args.algo == "adaptive" else None),
            "all_status_ok": status_ok,
        },
        "roofline": {
            "kernel": SIM_KERNEL,
            "bound": "alu",
            "achieved": achieved / 1e12,
            "peak": PEAK_INT32_LANE_OPS / 1e12,
            "unit": "TOP/s",
            "frac": achieved / PEAK_INT32_LANE_OPS,
            "traffic": traffic,
            "hardware_fraction": load_hardware_fraction(args.workload, args.algo, sim_avg_ms) if profiled else None,
            "kernel_ms": sim_avg_ms,
            "kernel_ms_median": float(np.median(sim_ms)),
            "ops_per_request_step": OPS_PER_REQUEST_STEP,
            "measured_peaks": measured_peaks,
        },
        "transfers": {
            "note": "first copies: torch from/to pageable host memory, allocation included; "
                    "pinned: steady-state copies between pinned host buffers and the resident "
                    "device tensors (HIP events); the PCIe-inclusive rate uses the pinned copies",
            "h2d_ms": h2d_ms, "h2d_bytes": h2d_bytes, "d2h_ms": d2h_ms, "d2h_bytes": d2h_bytes,
            "h2d_pinned_ms": pinned[0], "d2h_pinned_ms": pinned[1],
            "pcie_inclusive_request_steps_per_s": rs / ((step_ms + pinned[0] + pinned[1]) / 1e3),
        },
        "wall_s_timed_region": wall,
        "pipelined": (None if pipe_ms is None else {
            "note": "the same batch simulated back to back with several batches in flight, one stream and "
                    "one output set each: the tail of a batch overlaps the next; value and roofline above "
                    "are one batch at a time",
            "streams": args.pipeline_streams, "ms_per_step": pipe_ms,
            "request_steps_per_s": rs / (pipe_ms / 1e3), "outputs_equal_serial": pipe_same}),
    }
    if not args.no_cpu_baseline:
        threads = args.cpu_threads or host_cpus()[1]
        cb, parity, (w_ratio, w_n) = cpu_baseline(batch, algo, g, args.cpu_seconds, threads)
        result["cpu_baseline"] = cb
        result["parity_on_cpu_sample"] = parity
        result["w_alg"] = {"per_request_step": w_ratio, "per_s": value * w_ratio,
                           "sample": f"oracle work counters on {w_n} sampled instances"}
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
