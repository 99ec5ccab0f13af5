"""CPU oracle for the schedulers of arXiv 2508.14544 (A_max, A_min, H-SF).

TEST INFRASTRUCTURE ONLY.  Only tests, the smoke check and the benchmark's
CPU-baseline leg may import this module.  It shares no code with the HIP path.

Contents
  * ``simulate`` / ``simulate_batch``: ctypes front end of the plain C oracle
    (``sched_oracle.c``), which follows Algorithms 1-4 and equation (2).
  * ``literal_simulate``: a second, independently written step loop in pure
    Python that evaluates equation (2) densely at every step t' in
    [t, t_max(U)] instead of only at planned ends.  Small inputs only.
  * ``opt_tel``: hindsight optimum by exhaustive search over non-preemptive
    schedules (memory constraint of equation (1) at every step).  Tiny inputs.
  * ``audit``: replays an event log and checks the model's invariants.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Optional, Sequence

import numpy as np

AMAX, AMIN, HSF, AELL, ADAPTIVE, ARANDOM = 0, 1, 2, 3, 4, 5
ALGOS = {"amax": AMAX, "amin": AMIN, "hsf": HSF, "aell": AELL, "adaptive": ADAPTIVE, "arandom": ARANDOM}
OK, E_INVAL, E_INTERVAL, E_TOO_BIG, E_STEP_CAP, E_ARRIVAL = 0, -1, -2, -3, -4, -7
EV_START, EV_EVICT, EV_COMPLETE = 0, 1, 2
STAT_NAMES = ["max_running", "max_evicted_waiting", "max_waiting", "steps", "tests", "evict_events", "work"]

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = False) -> str:
    """Compile the C oracle with gcc (a checker, not part of the product)."""
    src = os.path.join(_HERE, "sched_oracle.c")
    if force or not os.path.exists(_SO) or os.path.getmtime(_SO) < os.path.getmtime(src):
        tmp = _SO + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-std=c99", "-Wall", "-Wextra", "-shared", "-fPIC",
                               src, "-o", tmp])
        os.replace(tmp, _SO)
    return _SO


class _Event(ctypes.Structure):
    _fields_ = [("t", ctypes.c_int64), ("kind", ctypes.c_int32), ("req", ctypes.c_int32)]


def _load():
    global _lib
    with _lock:
        if _lib is None:
            build()
            lib = ctypes.CDLL(_SO)
            P32 = ctypes.POINTER(ctypes.c_int32)
            P64 = ctypes.POINTER(ctypes.c_int64)
            lib.orc_simulate.restype = ctypes.c_int
            lib.orc_simulate.argtypes = [ctypes.c_int32, P32, P32, P32, P32, P32, P32, P32, ctypes.c_int32,
                                         ctypes.c_int64, ctypes.c_int64, P32, P32, P64, P64, P64,
                                         P64, P64, ctypes.POINTER(_Event), ctypes.c_int64, P64]
            lib.orc_default_step_cap.restype = ctypes.c_int64
            lib.orc_default_step_cap.argtypes = [ctypes.c_int32, P32, P32]
            lib.orc_adaptive_choice.restype = ctypes.c_int32
            lib.orc_adaptive_choice.argtypes = [ctypes.c_int32, P32, P32]
            _lib = lib
    return _lib


def _p32(x: Optional[np.ndarray]):
    if x is None:
        return ctypes.POINTER(ctypes.c_int32)()
    assert x.dtype == np.int32 and x.flags["C_CONTIGUOUS"]
    return x.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def _c32(x) -> Optional[np.ndarray]:
    return None if x is None else np.ascontiguousarray(np.asarray(x), dtype=np.int32)


def simulate(inst: Dict[str, Sequence[int]], algo: int, M: int, step_cap: int = 0,
             events: bool = False, stats: bool = False) -> Dict[str, object]:
    """Run the C oracle on one instance given as a dict of request fields."""
    lib = _load()
    o = _c32(inst["output"])
    n = int(o.shape[0])
    a = _c32(inst.get("arrival"))
    s = _c32(inst["prompt"])
    lo = _c32(inst.get("lower"))
    up = _c32(inst.get("upper"))
    pr = _c32(inst.get("priority"))
    tk = _c32(inst.get("tie_key"))
    comp = np.empty(n, np.int32)
    ev = np.empty(n, np.int32)
    tel, mk, rs, te, nev = (ctypes.c_int64() for _ in range(5))
    st_arr = np.zeros(8, np.int64)
    cap_ev = 0
    evbuf = None
    if events:
        cap_ev = 1 << 16
        evbuf = (_Event * cap_ev)()
    P64 = ctypes.POINTER(ctypes.c_int64)
    status = lib.orc_simulate(n, _p32(a), _p32(s), _p32(o), _p32(lo), _p32(up), _p32(pr), _p32(tk), int(algo), int(M),
                              int(step_cap), _p32(comp), _p32(ev), ctypes.byref(tel), ctypes.byref(mk),
                              ctypes.byref(rs), ctypes.byref(te), st_arr.ctypes.data_as(P64),
                              evbuf if events else ctypes.POINTER(_Event)(), cap_ev, ctypes.byref(nev))
    if events and nev.value > cap_ev:
        evbuf = (_Event * nev.value)()
        status = lib.orc_simulate(n, _p32(a), _p32(s), _p32(o), _p32(lo), _p32(up), _p32(pr), _p32(tk), int(algo), int(M),
                                  int(step_cap), _p32(comp), _p32(ev), ctypes.byref(tel), ctypes.byref(mk),
                                  ctypes.byref(rs), ctypes.byref(te), st_arr.ctypes.data_as(P64),
                                  evbuf, nev.value, ctypes.byref(nev))
    out: Dict[str, object] = {
        "status": int(status), "completion": comp, "evictions": ev, "tel": int(tel.value),
        "makespan": int(mk.value), "request_steps": int(rs.value), "total_evictions": int(te.value),
    }
    if stats:
        out["stats"] = {k: int(v) for k, v in zip(STAT_NAMES, st_arr[:len(STAT_NAMES)])}
    if events:
        out["events"] = [(int(evbuf[i].t), int(evbuf[i].kind), int(evbuf[i].req)) for i in range(nev.value)]
    return out


def adaptive_choice(inst: Dict[str, Sequence[int]]) -> int:
    """AELL or AMIN: the algorithm ADAPTIVE simulates for this instance."""
    lib = _load()
    lo, up = _c32(inst["lower"]), _c32(inst["upper"])
    return int(lib.orc_adaptive_choice(int(lo.shape[0]), _p32(lo), _p32(up)))


def default_step_cap(inst: Dict[str, Sequence[int]]) -> int:
    lib = _load()
    o = _c32(inst["output"])
    return int(lib.orc_default_step_cap(int(o.shape[0]), _p32(_c32(inst.get("arrival"))), _p32(o)))


def simulate_batch(batch, algo: int, *, instances: Optional[Sequence[int]] = None, threads: int = 0,
                   step_cap: int = 0, stats: bool = False) -> Dict[str, np.ndarray]:
    """Run the C oracle over instances of a CSR batch (``workloads.Instances``) on a thread pool.

    ctypes releases the GIL during the call, so threads run in parallel.
    Returns per-request arrays (for the selected instances, concatenated) and
    per-instance arrays.
    """
    ks = list(range(batch.num_instances)) if instances is None else list(instances)
    if not threads:
        # every CPU this process may use, capped by OMP_NUM_THREADS where the
        # host sets one (a share of a larger machine)
        threads = len(os.sched_getaffinity(0))
        env = os.environ.get("OMP_NUM_THREADS", "")
        if env.isdigit() and int(env) > 0:
            threads = min(threads, int(env))

    def one(k):
        return simulate(batch.instance(k), algo, batch.M, step_cap=step_cap, stats=stats)

    if threads == 1 or len(ks) <= 1:
        res = [one(k) for k in ks]
    else:
        with ThreadPoolExecutor(max_workers=threads) as ex:
            res = list(ex.map(one, ks))
    out = {
        "completion": np.concatenate([r["completion"] for r in res]) if res else np.zeros(0, np.int32),
        "evictions": np.concatenate([r["evictions"] for r in res]) if res else np.zeros(0, np.int32),
    }
    for f in ("status", "tel", "makespan", "request_steps", "total_evictions"):
        out[f] = np.array([r[f] for r in res], dtype=np.int64)
    if stats:
        out["stats"] = [r["stats"] for r in res]
    return out


# ---------------------------------------------------------------------------
# Literal step loop with dense evaluation of equation (2).
# ---------------------------------------------------------------------------

def literal_simulate(inst: Dict[str, Sequence[int]], algo: int, M: int, step_cap: int = 0) -> Dict[str, object]:
    """Pure-Python step loop; equation (2) is checked at every t' in [t, t_max].

    Each step: arrivals join the waiting list; runs reaching p + o complete;
    for A_min the running set's memory at t+1 is projected and runs are removed
    in ascending (o~, index) while it exceeds M, each removed request's o~
    rising to the tokens it had generated; for A_l a run that has generated l
    tokens without finishing is removed, plans with u from then on and goes to
    the back of the queue (fresh requests first, promoted ones in promotion
    order, same step by fresh-queue position) and may restart at once; then
    waiting requests are taken in (planning length, tie key, index) order (A_l:
    queue order) while equation (2) keeps holding.  ADAPTIVE runs the
    algorithm adaptive_choice picks.  Without a tie key, ties go by index.
    """
    if algo == ADAPTIVE:
        algo = adaptive_choice(inst)
    o = [int(x) for x in inst["output"]]
    n = len(o)
    s = [int(x) for x in inst["prompt"]]
    arr = [int(x) for x in inst["arrival"]] if inst.get("arrival") is not None else [0] * n
    if algo == AMAX:
        plan = [int(x) for x in inst["upper"]]
    elif algo in (HSF, ARANDOM):
        plan = list(o)
    else:
        plan = [int(x) for x in inst["lower"]]
    upper = [int(x) for x in inst["upper"]] if inst.get("upper") is not None else None
    cap = step_cap if step_cap > 0 else default_step_cap(inst)
    # equal planning lengths: by the caller's tie key, then by index
    tie = [int(x) for x in inst["tie_key"]] if inst.get("tie_key") is not None else [0] * n
    # A_l order: fresh requests by (arrival, tie, index), then promotion order
    queue_pos = [0] * n
    for pos, i in enumerate(sorted(range(n), key=lambda r: (arr[r], tie[r], r))):
        queue_pos[i] = pos
    promotions = 0

    start = {}                  # request -> current start step (running only)
    waiting: List[int] = []
    eligible_from = [0] * n
    completion = [-1] * n
    evict_count = [0] * n
    rs = 0
    arrived = 0
    t = 0
    status = OK
    while True:
        if t > cap:
            status = E_STEP_CAP
            break
        while arrived < n and arr[arrived] <= t:
            waiting.append(arrived)
            arrived += 1
        finished_now = [i for i in start if start[i] + o[i] == t]
        for i in finished_now:
            completion[i] = t
        for i in finished_now:
            del start[i]
        if all(c >= 0 for c in completion):
            break
        if algo == AMIN:
            proj = sum(s[i] + (t + 1) - start[i] for i in start)
            for i in sorted(start, key=lambda r: (plan[r], tie[r], r)):
                if proj <= M:
                    break
                proj -= s[i] + (t + 1) - start[i]
                plan[i] = max(plan[i], t - start[i])
                evict_count[i] += 1
                del start[i]
                waiting.append(i)
                eligible_from[i] = t + 1
        if algo == AELL:
            # same-step promotions in fresh-queue order (each request is promoted once)
            for i in sorted((r for r in start if start[r] + plan[r] == t), key=lambda r: queue_pos[r]):
                plan[i] = upper[i]
                queue_pos[i] = n + promotions
                promotions += 1
                evict_count[i] += 1
                del start[i]
                waiting.append(i)
                eligible_from[i] = t

        # in-progress runs: (start, prompt, planned length from its start)
        in_progress = [(start[i], s[i], max(plan[i], t + 1 - start[i])) for i in start]
        in_progress += [(t - o[i], s[i], o[i]) for i in finished_now]
        if algo == AELL:
            order_key = lambda r: (queue_pos[r], r)
        elif algo == ARANDOM:
            order_key = lambda r: (int(inst["priority"][r]), tie[r], r)
        else:
            order_key = lambda r: (plan[r], tie[r], r)
        order = sorted((w for w in waiting if eligible_from[w] <= t), key=order_key)
        chosen: List[int] = []
        for w in order:
            trial = chosen + [w]
            t_max = max(t + plan[x] for x in trial)
            for (p0, _, lam) in in_progress:
                t_max = max(t_max, p0 + lam)
            ok = True
            for tp in range(t, t_max + 1):
                tot = 0
                for (p0, sz, lam) in in_progress:
                    if lam >= tp - p0:
                        tot += sz + tp - p0
                for x in trial:
                    if plan[x] >= tp - t:
                        tot += s[x] + tp - t
                if tot > M:
                    ok = False
                    break
            if not ok:
                break
            chosen.append(w)
        for w in chosen:
            waiting.remove(w)
            start[w] = t
        rs += len(start)
        t += 1
    tel = sum(c - a for c, a in zip(completion, arr) if c >= 0)
    return {"status": status, "completion": np.array(completion, np.int32),
            "evictions": np.array(evict_count, np.int32), "tel": tel,
            "makespan": max([c for c in completion if c >= 0], default=0), "request_steps": rs,
            "total_evictions": sum(evict_count)}


# ---------------------------------------------------------------------------
# Hindsight optimum by exhaustive search (tiny instances only).
# ---------------------------------------------------------------------------

def opt_tel(inst: Dict[str, Sequence[int]], M: int, horizon: Optional[int] = None) -> int:
    """Minimum total latency over all non-preemptive schedules with known o.

    A schedule assigns each request a start p_i >= a_i; the run holds
    s_i + (tau - p_i) tokens for tau in [p_i, p_i + o_i] and the sum over runs
    must stay <= M at every tau (equation (1)).  Latency is p_i + o_i - a_i.
    Search: depth-first over steps, choosing at each step any subset of the
    arrived, unstarted requests that keeps the memory feasible; memoised on
    (t, unstarted set, runs still present).
    """
    o = [int(x) for x in inst["output"]]
    n = len(o)
    s = [int(x) for x in inst["prompt"]]
    arr = [int(x) for x in inst["arrival"]] if inst.get("arrival") is not None else [0] * n
    if any(s[i] + o[i] > M for i in range(n)):
        raise ValueError("a request never fits")
    if horizon is None:
        horizon = max(arr, default=0) + sum(x + 1 for x in o) + 1
    from functools import lru_cache

    def mem_ok(runs):
        if not runs:
            return True
        lo = min(p for p, _ in runs)
        hi = max(p + o[i] for p, i in runs)
        for tau in range(lo, hi + 1):
            if sum(s[i] + tau - p for p, i in runs if p <= tau <= p + o[i]) > M:
                return False
        return True

    best = [None]

    @lru_cache(maxsize=None)
    def go(t, unstarted, runs):
        # runs: tuple of (start, request) still present at step t or later
        if not unstarted:
            return 0
        if t > horizon:
            return 10 ** 18
        avail = [i for i in unstarted if arr[i] <= t]
        result = 10 ** 18
        # every subset of the available requests, including the empty one
        for mask in range(1 << len(avail)):
            pick = [avail[b] for b in range(len(avail)) if mask >> b & 1]
            new_runs = tuple(sorted(runs + tuple((t, i) for i in pick)))
            if pick and not mem_ok(new_runs):
                continue
            cost = sum(t + o[i] - arr[i] for i in pick)
            rest = tuple(i for i in unstarted if i not in pick)
            if not rest:
                result = min(result, cost)
                continue
            keep = tuple(r for r in new_runs if r[0] + o[r[1]] >= t + 1)
            # lower bound: each remaining request starts at t+1 or later
            lb = sum(max(t + 1, arr[i]) + o[i] - arr[i] for i in rest)
            if cost + lb >= result:
                continue
            result = min(result, cost + go(t + 1, rest, keep))
        return result

    return int(go(0, tuple(range(n)), ()))


# ---------------------------------------------------------------------------
# Event-log auditor.
# ---------------------------------------------------------------------------

def audit(inst: Dict[str, Sequence[int]], algo: int, M: int, result: Dict[str, object]) -> None:
    """Check a finished run against the model, from its event log alone.

    Raises AssertionError on the first violated property.
    """
    o = [int(x) for x in inst["output"]]
    n = len(o)
    s = [int(x) for x in inst["prompt"]]
    arr = [int(x) for x in inst["arrival"]] if inst.get("arrival") is not None else [0] * n
    if algo == ADAPTIVE:
        algo = adaptive_choice(inst)
    events = result["events"]
    assert result["status"] == OK
    runs = []                # (request, start, end, evicted?)
    open_run = {}
    n_evict = [0] * n
    last_evict = [-1] * n
    final_start = [-1] * n
    for (t, kind, i) in events:
        if kind == EV_START:
            assert i not in open_run, "request started twice"
            assert t >= arr[i], "started before arrival"
            if algo == AMIN:
                assert t > last_evict[i], "restarted in the step it was evicted"
            open_run[i] = t
            final_start[i] = t
        elif kind == EV_EVICT:
            p = open_run.pop(i)
            assert t - p < o[i], "evicted after it should have completed"
            runs.append((i, p, t, True))
            n_evict[i] += 1
            last_evict[i] = t
        else:
            p = open_run.pop(i)
            assert t == p + o[i], "completion is not start + o"
            runs.append((i, p, t, False))
    assert not open_run, "a run never ended"
    comp = [int(x) for x in result["completion"]]
    for i in range(n):
        assert comp[i] == final_start[i] + o[i], "completion mismatch"
        assert comp[i] >= arr[i] + o[i]
        assert int(result["evictions"][i]) == n_evict[i]
    if algo in (AMAX, HSF, ARANDOM):
        assert sum(n_evict) == 0, "A_max, H-SF and A_random never cancel"
    # equation (1) before and after the eviction point of every step
    horizon = max((r[2] for r in runs), default=0)
    for tau in range(0, horizon + 1):
        pre = sum(s[i] + tau - p for (i, p, e, ev) in runs if p < tau <= e)
        post = sum(s[i] + tau - p for (i, p, e, ev) in runs if p <= tau <= e and not (ev and e == tau))
        assert pre <= M and post <= M, f"memory {pre}/{post} > {M} at step {tau}"
    if algo == AELL:
        # promotions: exactly l tokens after the start, only for o > l, once per request
        lo = [int(x) for x in inst["lower"]]
        for (i, p, e, ev) in runs:
            if ev:
                assert e - p == lo[i] and o[i] > lo[i], "promotion not at l tokens"
        assert all(c <= 1 for c in n_evict), "a request was promoted twice"
    # evictions happen only when the projection at tau+1 overflows, and stop once it fits
    ev_steps = sorted({e for (i, p, e, ev) in runs if ev}) if algo == AMIN else []
    for tau in ev_steps:
        # the running set at the eviction point: started before tau, not completing at tau
        before = sum(s[i] + tau + 1 - p for (i, p, e, ev) in runs
                     if p < tau and (e > tau or (ev and e == tau)))
        after = sum(s[i] + tau + 1 - p for (i, p, e, ev) in runs if p < tau and e > tau)
        assert before > M and after <= M, "eviction without overflow, or still overflowing"
    # equation (3): sum of waiting (final start - arrival) plus sum of o
    tel = sum(final_start[i] - arr[i] for i in range(n)) + sum(o)
    assert tel == result["tel"] == sum(c - a for c, a in zip(comp, arr))
    assert result["makespan"] == max(comp, default=0)
    # every run is processed once per step from its start until it ends
    assert result["request_steps"] == sum(e - p for (i, p, e, ev) in runs)
    assert result["total_evictions"] == sum(n_evict)
