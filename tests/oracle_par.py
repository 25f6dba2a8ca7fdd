"""Run the single-threaded oracle on full-size sequential traces in parallel.

The oracle itself stays one plain thread per call; this module only splits
work that is independent by definition and runs the pieces side by side
(ctypes releases the GIL during each call):

* attribution of ONE stream: m(x) is 0 or 1 everywhere, so an interval's
  energy depends on no other interval and any slice of the intervals gives
  the same energies as the whole list;
* grouping: keys are split into ranges by value; a key's rows are taken in
  interval order, so every per-key sum and M2 is computed exactly as in the
  whole-list call, and the ranges concatenate in ascending key order.

Test infrastructure only.
"""
from __future__ import annotations

import concurrent.futures as cf
import os

import numpy as np

import oracle


def workers() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def attribute_one_stream(t, P, s, e, pieces: int | None = None) -> dict:
    """oracle.attribute of a one-stream trace, its intervals split into slices."""
    m = s.shape[0]
    pieces = pieces or workers()
    cuts = np.linspace(0, m, pieces + 1).astype(np.int64)
    energy = np.empty(m, np.float64)
    si = np.empty(m, np.int64)
    ei = np.empty(m, np.int64)

    def run(k):
        a, b = int(cuts[k]), int(cuts[k + 1])
        r = oracle.attribute(t, P, s[a:b], e[a:b], np.array([0, b - a]), equal_split=True)
        energy[a:b] = r["energy"]
        si[a:b] = r["start_idx"]
        ei[a:b] = r["end_idx"]
        return r

    with cf.ThreadPoolExecutor(pieces) as ex:
        parts = list(ex.map(run, range(pieces)))
    # whole-trace energy is the same in every slice; idle = W - attributed
    W = parts[0]["trace_energy"]
    attributed = float(sum(p["attributed_energy"] for p in parts))
    return {"energy": energy, "start_idx": si, "end_idx": ei, "trace_energy": W,
            "attributed_energy": attributed, "idle_energy": W - attributed,
            "n_clipped": int(sum(p["n_clipped"] for p in parts))}


def groupby(keys, energy, pieces: int | None = None) -> dict:
    """oracle.groupby over key-value ranges, concatenated in ascending key order."""
    keys = np.ascontiguousarray(keys, np.uint64)
    pieces = pieces or workers()
    bounds = np.quantile(keys.astype(np.float64), np.linspace(0, 1, pieces + 1)[1:-1])
    edges = np.unique(np.concatenate([[0], bounds.astype(np.uint64)]))
    part = np.searchsorted(edges, keys, side="right") - 1

    def run(k):
        sel = np.nonzero(part == k)[0]  # interval order kept within the range
        if sel.size == 0:
            return None
        return oracle.groupby(keys[sel], energy[sel])

    with cf.ThreadPoolExecutor(pieces) as ex:
        parts = [p for p in ex.map(run, range(edges.shape[0])) if p is not None]
    out = {k: np.concatenate([p[k] for p in parts]) for k in parts[0]}
    assert np.all(out["keys"][1:] > out["keys"][:-1])
    return out
