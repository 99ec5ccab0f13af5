"""Digest format of stored oracle outputs (test infrastructure).

A batch's outputs are hashed in blocks of BLOCK consecutive instances.  For each
instance in a block, in order: its five per-instance integers (status, total
latency, makespan, request-steps, total cancellations) as little-endian int64,
then its per-request completion steps and cancellation counts as little-endian
int32.  A block's digest is the first 32 hex digits of SHA-256 over those bytes.

Holds no arithmetic of the schedulers: it only hashes outputs, so the oracle
side (tests/golden/make_oracle_digests.py) and the GPU side (the parity tests)
can compare whole workloads without storing every output.
"""
from __future__ import annotations

import hashlib
from typing import Dict, List

import numpy as np

BLOCK = 64
FIELDS = ("status", "tel", "makespan", "request_steps", "total_evictions")


def inputs_digest(batch) -> str:
    """SHA-256 of a generated batch's arrays: detects a change of the generator."""
    h = hashlib.sha256()
    h.update(np.ascontiguousarray(batch.offsets, dtype="<i8").tobytes())
    for f in ("arrival", "prompt", "output", "lower", "upper", "priority"):
        x = getattr(batch, f, None)
        h.update(f.encode())
        if x is not None:
            h.update(np.ascontiguousarray(x, dtype="<i4").tobytes())
    return h.hexdigest()[:32]


def block_digests(offsets: np.ndarray, out: Dict[str, np.ndarray], first: int = 0) -> List[str]:
    """Digests of consecutive blocks of BLOCK instances.

    ``offsets`` is the CSR offsets of the instances covered by ``out`` (local
    numbering, offsets[0] = 0); ``first`` is the global index of out's first
    instance and must be a multiple of BLOCK.  Per-request arrays in ``out``
    are indexed by the local offsets.
    """
    assert first % BLOCK == 0
    K = len(offsets) - 1
    scal = np.stack([np.asarray(out[f], dtype=np.int64)[:K] for f in FIELDS], axis=1).astype("<i8")
    comp = np.ascontiguousarray(out["completion"], dtype="<i4")
    ev = np.ascontiguousarray(out["evictions"], dtype="<i4")
    res = []
    for b0 in range(0, K, BLOCK):
        h = hashlib.sha256()
        for k in range(b0, min(K, b0 + BLOCK)):
            lo, hi = int(offsets[k]), int(offsets[k + 1])
            h.update(scal[k].tobytes())
            h.update(comp[lo:hi].tobytes())
            h.update(ev[lo:hi].tobytes())
        res.append(h.hexdigest()[:32])
    return res


def totals(out: Dict[str, np.ndarray]) -> Dict[str, object]:
    """Readable per-workload sums stored beside the digests."""
    st = np.asarray(out["status"], dtype=np.int64)
    codes, counts = np.unique(st, return_counts=True)
    return {
        "status_counts": {str(int(c)): int(n) for c, n in zip(codes, counts)},
        "tel": int(np.asarray(out["tel"], dtype=np.int64).sum()),
        "makespan": int(np.asarray(out["makespan"], dtype=np.int64).sum()),
        "request_steps": int(np.asarray(out["request_steps"], dtype=np.int64).sum()),
        "total_evictions": int(np.asarray(out["total_evictions"], dtype=np.int64).sum()),
    }
