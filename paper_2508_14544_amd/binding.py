"""ctypes binding of the HIP scheduler-simulator library (libschedsim.so).

Argument marshalling only: every step of the simulation runs in the HIP
kernels behind ``sched_simulate``.  PyTorch provides device memory and
streams.  If the library is missing this module raises; there is no CPU
fallback.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Dict, Optional

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libschedsim.so")

AMAX, AMIN, HSF, AELL, ADAPTIVE, ARANDOM = 0, 1, 2, 3, 4, 5
ALGOS = {"amax": AMAX, "amin": AMIN, "hsf": HSF, "aell": AELL, "adaptive": ADAPTIVE, "arandom": ARANDOM}
OK, E_INVAL, E_INTERVAL, E_TOO_BIG, E_STEP_CAP, E_HIP, E_UNSUPPORTED, E_ARRIVAL, E_SCRATCH = 0, -1, -2, -3, -4, -5, -6, -7, -8

# every symbol include/schedsim.h declares
EXPORTED = ("sched_optimum", "sched_simulate", "sched_simulate_noalloc", "sched_simulate_opts", "sched_strerror",
            "sched_validate", "sched_version")


class SchedInstances(ctypes.Structure):
    _fields_ = [
        ("num_instances", ctypes.c_int32),
        ("max_requests", ctypes.c_int32),
        ("total_requests", ctypes.c_int64),
        ("offsets", ctypes.c_void_p),
        ("arrival", ctypes.c_void_p),
        ("prompt", ctypes.c_void_p),
        ("output", ctypes.c_void_p),
        ("lower", ctypes.c_void_p),
        ("upper", ctypes.c_void_p),
        ("priority", ctypes.c_void_p),
        ("tie_key", ctypes.c_void_p),
    ]


class SchedResults(ctypes.Structure):
    _fields_ = [
        ("completion", ctypes.c_void_p),
        ("evictions", ctypes.c_void_p),
        ("total_latency", ctypes.c_void_p),
        ("makespan", ctypes.c_void_p),
        ("request_steps", ctypes.c_void_p),
        ("total_evictions", ctypes.c_void_p),
        ("status", ctypes.c_void_p),
        ("algo_used", ctypes.c_void_p),
    ]


class SchedOptions(ctypes.Structure):
    _fields_ = [
        ("step_cap", ctypes.c_int64),
        ("running_capacity", ctypes.c_int32),
        ("evicted_capacity", ctypes.c_int32),
        ("event_before", ctypes.c_void_p),
        ("event_after", ctypes.c_void_p),
        ("evicted_lds_limit", ctypes.c_int32),
        ("workgroup_waves", ctypes.c_int32),
    ]


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libschedsim.so (raises OSError if it is not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(path):
            raise OSError(f"{path} is not built; run __graft_entry__.build()")
        # torch first: the library must bind to the HIP runtime that owns the
        # device buffers and streams it is handed, not load a second one
        import torch  # noqa: F401
        lib = ctypes.CDLL(path)
        lib.sched_simulate.restype = ctypes.c_int
        lib.sched_simulate.argtypes = [ctypes.POINTER(SchedInstances), ctypes.c_int, ctypes.c_int64,
                                       ctypes.POINTER(SchedResults), ctypes.c_void_p]
        lib.sched_simulate_opts.restype = ctypes.c_int
        lib.sched_simulate_opts.argtypes = [ctypes.POINTER(SchedInstances), ctypes.c_int, ctypes.c_int64,
                                            ctypes.POINTER(SchedResults), ctypes.c_void_p,
                                            ctypes.POINTER(SchedOptions)]
        lib.sched_simulate_noalloc.restype = ctypes.c_int
        lib.sched_simulate_noalloc.argtypes = lib.sched_simulate_opts.argtypes
        lib.sched_validate.restype = ctypes.c_int
        lib.sched_validate.argtypes = [ctypes.POINTER(SchedInstances), ctypes.c_int, ctypes.c_int64, ctypes.c_void_p,
                                       ctypes.c_void_p]
        lib.sched_strerror.restype = ctypes.c_char_p
        lib.sched_strerror.argtypes = [ctypes.c_int]
        lib.sched_version.restype = ctypes.c_int
        lib.sched_version.argtypes = []
        lib.sched_optimum.restype = ctypes.c_int
        lib.sched_optimum.argtypes = [ctypes.POINTER(SchedInstances), ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                      ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
        _lib = lib
    return _lib


def strerror(code: int) -> str:
    return load_library().sched_strerror(int(code)).decode()


class SchedError(RuntimeError):
    def __init__(self, code: int):
        super().__init__(f"sched_simulate failed: {code} ({strerror(code)})")
        self.code = code


def _ptr(t) -> Optional[int]:
    return None if t is None else int(t.data_ptr())


@dataclass
class DeviceBatch:
    """Device-resident CSR batch (torch tensors on the GPU)."""
    M: int
    max_requests: int
    offsets: object
    arrival: object
    prompt: object
    output: object
    lower: object
    upper: object
    priority: object = None
    tie_key: object = None

    @property
    def num_instances(self) -> int:
        return int(self.offsets.shape[0]) - 1

    @property
    def total_requests(self) -> int:
        return int(self.output.shape[0])


def to_device(batch, device="cuda") -> DeviceBatch:
    """Copy a ``workloads.Instances`` batch to device tensors."""
    import torch

    def t(x, dt):
        return None if x is None else torch.from_numpy(x).to(device=device, dtype=dt).contiguous()

    return DeviceBatch(batch.M, batch.max_requests, t(batch.offsets, torch.int64), t(batch.arrival, torch.int32),
                       t(batch.prompt, torch.int32), t(batch.output, torch.int32), t(batch.lower, torch.int32),
                       t(batch.upper, torch.int32), t(getattr(batch, "priority", None), torch.int32),
                       t(getattr(batch, "tie_key", None), torch.int32))


def alloc_results(db: DeviceBatch, evictions: bool = True):
    import torch
    dev = db.output.device
    K, N = db.num_instances, db.total_requests
    return {
        "completion": torch.empty(N, dtype=torch.int32, device=dev),
        "evictions": torch.empty(N, dtype=torch.int32, device=dev) if evictions else None,
        "tel": torch.empty(K, dtype=torch.int64, device=dev),
        "makespan": torch.empty(K, dtype=torch.int32, device=dev),
        "request_steps": torch.empty(K, dtype=torch.int64, device=dev),
        "total_evictions": torch.empty(K, dtype=torch.int64, device=dev),
        "status": torch.empty(K, dtype=torch.int32, device=dev),
        "algo_used": torch.empty(K, dtype=torch.int32, device=dev),
    }


def _instances(db: DeviceBatch, pass_lower: bool = True, pass_upper: bool = True) -> SchedInstances:
    return SchedInstances(db.num_instances, db.max_requests, db.total_requests, _ptr(db.offsets), _ptr(db.arrival),
                          _ptr(db.prompt), _ptr(db.output), _ptr(db.lower) if pass_lower else None,
                          _ptr(db.upper) if pass_upper else None, _ptr(db.priority), _ptr(db.tie_key))


def simulate_into(db: DeviceBatch, algo: int, out: Dict[str, object], *, M: Optional[int] = None, stream=None,
                  step_cap: int = 0, running_capacity: int = 0, evicted_capacity: int = 0,
                  evicted_lds_limit: int = 0, event_before=None, event_after=None, pass_lower: bool = True,
                  pass_upper: bool = True, no_alloc: bool = False, workgroup_waves: int = 0) -> None:
    """Queue ``sched_simulate_opts`` (``sched_simulate_noalloc`` with no_alloc) on ``stream``
    (default: torch's current stream)."""
    import torch
    lib = load_library()
    if stream is None:
        stream = torch.cuda.current_stream(db.output.device)
    inst = _instances(db, pass_lower, pass_upper)
    res = SchedResults(_ptr(out["completion"]), _ptr(out.get("evictions")), _ptr(out["tel"]),
                       _ptr(out.get("makespan")), _ptr(out.get("request_steps")), _ptr(out.get("total_evictions")),
                       _ptr(out["status"]), _ptr(out.get("algo_used")))
    opts = SchedOptions(int(step_cap), int(running_capacity), int(evicted_capacity),
                        None if event_before is None else int(event_before.cuda_event),
                        None if event_after is None else int(event_after.cuda_event), int(evicted_lds_limit),
                        int(workgroup_waves))
    fn = lib.sched_simulate_noalloc if no_alloc else lib.sched_simulate_opts
    code = fn(ctypes.byref(inst), int(algo), int(db.M if M is None else M), ctypes.byref(res),
              ctypes.c_void_p(stream.cuda_stream), ctypes.byref(opts))
    if code != OK:
        raise SchedError(code)


def validate(db: DeviceBatch, algo: int, *, M: Optional[int] = None, stream=None, pass_lower: bool = True,
             pass_upper: bool = True):
    """Queue ``sched_validate``; returns the int32 device tensor of per-instance statuses (not synchronised)."""
    import torch
    lib = load_library()
    if stream is None:
        stream = torch.cuda.current_stream(db.output.device)
    status = torch.empty(db.num_instances, dtype=torch.int32, device=db.output.device)
    code = lib.sched_validate(ctypes.byref(_instances(db, pass_lower, pass_upper)), int(algo),
                              int(db.M if M is None else M), _ptr(status), ctypes.c_void_p(stream.cuda_stream))
    if code != OK:
        raise SchedError(code)
    return status


def simulate(db: DeviceBatch, algo: int, **kw) -> Dict[str, object]:
    """Allocate outputs, queue the simulation and return the output tensors (not synchronised)."""
    out = alloc_results(db)
    simulate_into(db, algo, out, **kw)
    return out


def optimum(db: DeviceBatch, *, M: Optional[int] = None, node_cap: int = 0, upper_bound=None,
            stream=None) -> Dict[str, object]:
    """Queue ``sched_optimum`` (hindsight optimum, instances of at most 8 requests); returns
    device tensors total_latency, status and nodes (not synchronised).  `upper_bound`: an
    optional int64 device tensor [K] of achievable totals (e.g. a policy's) to prune with."""
    import torch
    lib = load_library()
    if stream is None:
        stream = torch.cuda.current_stream(db.output.device)
    dev = db.output.device
    K = db.num_instances
    out = {"tel": torch.empty(K, dtype=torch.int64, device=dev), "status": torch.empty(K, dtype=torch.int32, device=dev),
           "nodes": torch.empty(K, dtype=torch.int64, device=dev)}
    inst = SchedInstances(K, db.max_requests, db.total_requests, _ptr(db.offsets), _ptr(db.arrival),
                          _ptr(db.prompt), _ptr(db.output), None, None, None, None)
    code = lib.sched_optimum(ctypes.byref(inst), int(db.M if M is None else M), _ptr(upper_bound), _ptr(out["tel"]),
                             _ptr(out["status"]), _ptr(out["nodes"]), int(node_cap),
                             ctypes.c_void_p(stream.cuda_stream))
    if code != OK:
        raise SchedError(code)
    return out
