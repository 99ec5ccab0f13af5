"""The C ABI library loads, exports every declared symbol, and rejects bad
calls before touching a GPU (host-side validation only; no compute here)."""
import ctypes
import os
import re

import pytest

from paper_2508_14544_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    txt = open(os.path.join(ROOT, "include", "schedsim.h")).read()
    return sorted(set(re.findall(r"^(?:int|const char\*)\s+(sched_\w+)\s*\(", txt, re.M)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return B.load_library()


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert names == sorted(B.EXPORTED)
    for nm in names:
        assert hasattr(lib, nm)


def test_probe_library_exports_every_declared_symbol(lib):
    # the throughput probes (include/schedprobe.h) live in their own library
    txt = open(os.path.join(ROOT, "include", "schedprobe.h")).read()
    names = sorted(set(re.findall(r"^int\s+(sched_probe_\w+)\s*\(", txt, re.M)))
    assert names == ["sched_probe_lds", "sched_probe_valu"]
    probe = ctypes.CDLL(os.path.join(ROOT, "paper_2508_14544_amd", "libschedprobe.so"))
    for nm in names:
        assert hasattr(probe, nm)
        f = getattr(probe, nm)
        f.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_double)]
        out = ctypes.c_double(0)
        assert f(0, ctypes.byref(out)) == -1          # rejected before any GPU call
        assert f(10, None) == -1


def test_version_and_strerror(lib):
    assert lib.sched_version() == 131
    for code in (0, -1, -2, -3, -4, -5, -6, -7, -8):
        assert B.strerror(code) and B.strerror(code) != "unknown code"
    assert B.strerror(12345) == "unknown code"


def _inst(K=1, nmax=4, N=4, offsets=1, prompt=1, output=1, lower=1, upper=1, priority=1):
    f = lambda v: None if v is None else 0x1000  # non-null dummies; never dereferenced here
    return B.SchedInstances(K, nmax, N, f(offsets), None, f(prompt), f(output), f(lower), f(upper), f(priority))


def _res(**kw):
    d = dict(completion=0x1000, evictions=None, total_latency=0x1000, makespan=None, request_steps=None,
             total_evictions=None, status=0x1000, algo_used=None)
    d.update(kw)
    return B.SchedResults(*[d[k] for k, _ in B.SchedResults._fields_])


def call(lib, inst, algo=B.AMIN, M=16, res=None, opts=None):
    res = res or _res()
    return lib.sched_simulate_opts(ctypes.byref(inst) if inst is not None else None, algo, M,
                                   ctypes.byref(res), None, ctypes.byref(opts) if opts else None)


def test_host_validation(lib):
    assert lib.sched_simulate(None, B.AMIN, 16, ctypes.byref(_res()), None) == B.E_INVAL
    assert call(lib, _inst(), M=0) == B.E_INVAL
    assert call(lib, _inst(), M=-5) == B.E_INVAL
    assert call(lib, _inst(), M=1 << 30) == B.E_INVAL
    assert call(lib, _inst(), algo=7) == B.E_INVAL
    assert call(lib, _inst(K=-1)) == B.E_INVAL
    assert call(lib, _inst(offsets=None)) == B.E_INVAL
    assert call(lib, _inst(prompt=None)) == B.E_INVAL
    assert call(lib, _inst(output=None)) == B.E_INVAL
    assert call(lib, _inst(lower=None), algo=B.AMIN) == B.E_INVAL
    assert call(lib, _inst(upper=None), algo=B.AMAX) == B.E_INVAL
    for algo in (B.AELL, B.ADAPTIVE):  # both bounds are needed
        assert call(lib, _inst(lower=None), algo=algo) == B.E_INVAL
        assert call(lib, _inst(upper=None), algo=algo) == B.E_INVAL
    assert call(lib, _inst(priority=None), algo=B.ARANDOM) == B.E_INVAL
    assert call(lib, _inst(), algo=6) == B.E_INVAL
    assert call(lib, _inst(), algo=-1) == B.E_INVAL
    assert call(lib, _inst(), res=_res(status=None)) == B.E_INVAL
    assert call(lib, _inst(), res=_res(completion=None)) == B.E_INVAL
    assert call(lib, _inst(), res=_res(total_latency=None)) == B.E_INVAL
    assert call(lib, _inst(nmax=1 << 17)) == B.E_UNSUPPORTED
    assert call(lib, _inst(), opts=B.SchedOptions(1 << 31, 0, 0, None, None)) == B.E_INVAL
    assert call(lib, _inst(), opts=B.SchedOptions(0, 2048, 0, None, None)) == B.E_UNSUPPORTED
    assert call(lib, _inst(), opts=B.SchedOptions(0, -1, 0, None, None)) == B.E_INVAL
    assert call(lib, _inst(), opts=B.SchedOptions(0, 0, -1, None, None)) == B.E_INVAL
    assert call(lib, _inst(), opts=B.SchedOptions(0, 0, 0, None, None, -1)) == B.E_INVAL
    # an empty batch is a no-op
    assert call(lib, _inst(K=0, N=0)) == B.OK


def test_noalloc_host_checks(lib):
    # the no-allocation variant shares the host checks (nothing reaches HIP)
    def na(inst, algo=B.AMIN, M=16, res=None, opts=None):
        res = res or _res()
        return lib.sched_simulate_noalloc(ctypes.byref(inst) if inst is not None else None, algo, M,
                                          ctypes.byref(res), None, ctypes.byref(opts) if opts else None)
    assert na(None) == B.E_INVAL
    assert na(_inst(), M=0) == B.E_INVAL
    assert na(_inst(), algo=7) == B.E_INVAL
    assert na(_inst(output=None)) == B.E_INVAL
    assert na(_inst(), res=_res(status=None)) == B.E_INVAL
    assert na(_inst(nmax=1 << 17)) == B.E_UNSUPPORTED
    assert na(_inst(), opts=B.SchedOptions(0, 2048, 0, None, None)) == B.E_UNSUPPORTED
    assert na(_inst(K=0, N=0)) == B.OK


def test_validate_host_checks(lib):
    # sched_validate rejects the same call-level problems before any HIP call
    def v(inst, algo=B.AMIN, M=16, status=0x1000):
        return lib.sched_validate(ctypes.byref(inst) if inst is not None else None, algo, M, status, None)
    assert v(None) == B.E_INVAL
    assert v(_inst(), M=0) == B.E_INVAL
    assert v(_inst(), M=1 << 30) == B.E_INVAL
    assert v(_inst(), algo=9) == B.E_INVAL
    assert v(_inst(offsets=None)) == B.E_INVAL
    assert v(_inst(lower=None), algo=B.AMIN) == B.E_INVAL
    assert v(_inst(upper=None), algo=B.AMAX) == B.E_INVAL
    assert v(_inst(priority=None), algo=B.ARANDOM) == B.E_INVAL
    assert v(_inst(), status=None) == B.E_INVAL
    assert v(_inst(nmax=1 << 17)) == B.E_UNSUPPORTED
    assert v(_inst(K=0, N=0)) == B.OK
