"""Locate the first step at which two simulations of one instance disagree.

Both sides simulate with a step cap T (every decision up to step T, then the
partial outputs: completion steps by T, cancellation counts, request-steps
through T, total latency of the completed requests).  The partial outputs at
T are a digest of the state reached at T, so the first divergent step lies at
or before the smallest T whose digests differ: the outputs of a step show a
differing decision no later than the next completion, cancellation or change
in the number of running requests it causes.  The search doubles T until the
digests differ, then bisects between the last agreeing and the first differing
cap (digests that agree again after differing would mislead the bisection;
the returned cap always differs and the one before it always agrees).

Used to bisect a parity failure down to an (instance, step) pair; each side is
a callable run(batch, step_cap) -> outputs dict (tests use the CPU oracle and
the GPU path through the C ABI).
"""
import numpy as np

FIELDS = ("status", "tel", "request_steps", "total_evictions")


def _one(batch, k):
    from paper_2508_14544_amd import workloads as W
    d = batch.instance(k)
    return W.from_lists(batch.M, [{f: d[f] for f in d if d[f] is not None}], name=f"{batch.name}[{k}]")


def _digest(out):
    return tuple(int(out[f][0]) for f in FIELDS) + (tuple(np.asarray(out["completion"]).tolist()),
                                                      tuple(np.asarray(out["evictions"]).tolist()))


def first_divergence(batch, run_a, run_b, instances=None, t_max=1 << 30):
    """[(instance, T)] for every instance whose simulations differ: T is the
    smallest step cap found whose digests differ (the cap T - 1 agrees)."""
    found = []
    ks = range(batch.num_instances) if instances is None else instances
    for k in ks:
        one = _one(batch, k)
        same = lambda T: _digest(run_a(one, T)) == _digest(run_b(one, T))
        if same(t_max):
            continue
        lo, hi = 0, 1      # cap lo agrees (0: taken to), cap hi is tried next (a cap is >= 1)
        while same(hi):
            lo, hi = hi, min(2 * hi, t_max)
        while hi - lo > 1:  # invariant: lo agrees, hi differs
            mid = (lo + hi) // 2
            if same(mid):
                lo = mid
            else:
                hi = mid
        found.append((k, hi))
    return found
