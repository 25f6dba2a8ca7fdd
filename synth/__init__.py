"""Seeded synthetic inputs shared by the tests, the benchmark and the smoke check.

The heavy workloads are drawn by ``synth.c`` (compiled into ``_synth.so`` next
to this file by :func:`build`); the small randomized edge-case traces are drawn
here with numpy.  Nothing in this module attributes energy: it only produces
timestamps, power samples, readings of a cumulative energy counter (drawn as
running sums of random increments), interval bounds and operator keys.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# MAG_SYNTH_SO: another build of synth.c to load (the sanitizer runs in tests/)
_SO = os.environ.get("MAG_SYNTH_SO") or os.path.join(_HERE, "_synth.so")
_lib = None


def build(out: str | None = None, extra_flags=()) -> str:
    """Compile synth.c into _synth.so (or `out`) with gcc (always recompiles);
    extra_flags: e.g. sanitizer options."""
    src = os.path.join(_HERE, "synth.c")
    so = out or _SO
    tmp = so + ".tmp"
    subprocess.check_call(["gcc", "-O2", "-std=gnu99", "-fopenmp", *extra_flags, "-fPIC", "-shared",
                           "-o", tmp, src, "-lm"])
    os.replace(tmp, so)
    return so


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build()
        lib = ctypes.CDLL(_SO)
        p = ctypes.c_void_p
        lib.synth_shape.argtypes = [ctypes.c_int, p]
        lib.synth_vocab.argtypes = [ctypes.c_int, ctypes.c_uint64, p]
        lib.synth_structure.argtypes = [ctypes.c_int, ctypes.c_uint64, ctypes.c_int, p, p, p, p, p]
        lib.synth_power.argtypes = [ctypes.c_int, ctypes.c_uint64, ctypes.c_int, p, p, p, p, p, p]
        lib.synth_mix64.argtypes = [ctypes.c_uint64]
        lib.synth_mix64.restype = ctypes.c_uint64
        _lib = lib
    return _lib


def _ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data)


def shape(cfg: int) -> dict:
    """Sizes of workload ``cfg`` (1..5) per side."""
    out = np.zeros(4, dtype=np.int64)
    if _load().synth_shape(cfg, _ptr(out)) != 0:
        raise ValueError(f"unknown workload {cfg}")
    return {"n": int(out[0]), "m": int(out[1]), "K": int(out[2]), "streams": int(out[3])}


N_SIDES = {1: 2, 2: 2, 3: 2, 4: 9, 5: 2}


def vocab(cfg: int, seed: int = 0) -> np.ndarray:
    sh = shape(cfg)
    out = np.empty(sh["K"], dtype=np.uint64)
    _load().synth_vocab(cfg, seed, _ptr(out))
    return out


def structure(cfg: int, seed: int = 0, side: int = 0) -> dict:
    """Timestamps, interval bounds, keys and stream offsets of one side."""
    sh = shape(cfg)
    t = np.empty(sh["n"], dtype=np.float64)
    s = np.empty(sh["m"], dtype=np.float64)
    e = np.empty(sh["m"], dtype=np.float64)
    key = np.empty(sh["m"], dtype=np.uint64)
    off = np.empty(sh["streams"] + 1, dtype=np.int64)
    rc = _load().synth_structure(cfg, seed, side, _ptr(t), _ptr(s), _ptr(e), _ptr(key), _ptr(off))
    if rc != 0:
        raise RuntimeError(f"synth_structure({cfg}) failed: {rc}")
    return {"t": t, "s": s, "e": e, "key": key, "offsets": off}


def power(cfg: int, st: dict, seed: int = 0, side: int = 0) -> np.ndarray:
    """fp32 power samples of one side, drawn against the given structure."""
    P = np.empty(st["t"].shape[0], dtype=np.float32)
    rc = _load().synth_power(cfg, seed, side, _ptr(st["t"]), _ptr(st["s"]), _ptr(st["e"]),
                             _ptr(st["key"]), _ptr(st["offsets"]), _ptr(P))
    if rc != 0:
        raise RuntimeError(f"synth_power({cfg}) failed: {rc}")
    return P


def trace(cfg: int, seed: int = 0, side: int = 0) -> dict:
    st = structure(cfg, seed, side)
    st["P"] = power(cfg, st, seed, side)
    return st


def sides(cfg: int, seed: int = 0, which=None) -> list:
    """All sides of a workload; sides that share a structure share its arrays."""
    which = list(range(N_SIDES[cfg])) if which is None else list(which)
    out = []
    base = None
    for side in which:
        if cfg == 5 or base is None:
            st = structure(cfg, seed, side)
            if cfg != 5:
                base = st
        else:
            st = dict(base)
        st = dict(st)
        st["P"] = power(cfg, st, seed, side)
        out.append(st)
    return out


# ----------------------------------------------------------------------------
# small randomized traces for edge cases (numpy)
# ----------------------------------------------------------------------------

def tiny_case(seed: int, n: int = 64, streams: int = 1, per_stream: int = 8,
              snap: float = 0.3, zero_len: float = 0.1, outside: bool = True,
              zero_power: float = 0.1, keys: int = 5, dyadic: bool = False) -> dict:
    """A small random trace with the awkward cases the method has.

    Intervals are sorted and non-overlapping within each stream; some bounds sit
    exactly on sample times, some intervals have zero length, and (when
    ``outside``) some start before the first sample or end after the last.
    """
    rng = np.random.default_rng(seed)
    if dyadic:
        steps = 2 ** rng.integers(0, 3, size=n - 1)  # 1, 2 or 4 ticks of 1/1024 s
        t = np.concatenate([[0], np.cumsum(steps)]).astype(np.float64) / 1024.0
        P = rng.integers(0, 1000, size=n).astype(np.float32)
    else:
        t = np.concatenate([[0.0], np.cumsum(rng.uniform(0.2, 1.8, size=n - 1))])
        t += rng.uniform(-5, 5)
        P = rng.uniform(0.0, 800.0, size=n).astype(np.float32)
        P[rng.random(n) < zero_power] = 0.0
    lo, hi = t[0], t[-1]
    span = hi - lo
    s_all, e_all, off = [], [], [0]
    for _ in range(streams):
        cnt = int(rng.integers(0, per_stream + 1))
        a = lo - (0.1 * span if outside else 0.0)
        b = hi + (0.1 * span if outside else 0.0)
        cuts = np.sort(rng.uniform(a, b, size=2 * cnt))
        if dyadic:
            cuts = np.sort(np.round(cuts * 4096.0) / 4096.0)
        if snap > 0 and cnt:
            m = rng.random(2 * cnt) < snap
            idx = np.clip(np.searchsorted(t, cuts), 0, n - 1)
            cuts = np.where(m, t[idx], cuts)
            cuts = np.sort(cuts)
        s = cuts[0::2].copy()
        e = cuts[1::2].copy()
        if zero_len > 0 and cnt:
            z = rng.random(cnt) < zero_len
            e = np.where(z, s, e)
        s_all.append(s)
        e_all.append(e)
        off.append(off[-1] + cnt)
    s = np.concatenate(s_all) if s_all else np.zeros(0)
    e = np.concatenate(e_all) if e_all else np.zeros(0)
    key_vocab = rng.integers(0, 2**63, size=keys, dtype=np.int64).astype(np.uint64) * np.uint64(2) + \
        rng.integers(0, 2, size=keys).astype(np.uint64)
    key = key_vocab[rng.integers(0, keys, size=s.shape[0])] if s.shape[0] else np.zeros(0, np.uint64)
    return {"t": t.astype(np.float64), "P": P, "s": s.astype(np.float64), "e": e.astype(np.float64),
            "key": key.astype(np.uint64), "offsets": np.array(off, dtype=np.int64)}


def long_trace(seed, n, streams, per_stream, outside=True):
    """A trace of ~1 us steps whose intervals range from sub-sample to many
    thousands of samples, some starting before or ending after the trace."""
    rng = np.random.default_rng(seed)
    t = np.concatenate([[0.0], np.cumsum(rng.uniform(0.5, 1.5, n - 1))]) * 1e-6
    P = rng.uniform(50, 800, n).astype(np.float32)
    s_all, e_all, off = [], [], [0]
    lo, hi = t[0], t[-1]
    for a in range(streams):
        pad = 0.05 * (hi - lo) if outside else 0.0
        cuts = np.sort(rng.uniform(lo - pad, hi + pad, 2 * per_stream))
        s_all.append(cuts[0::2])
        e_all.append(cuts[1::2])
        off.append(off[-1] + per_stream)
    s = np.concatenate(s_all)
    e = np.concatenate(e_all)
    key = rng.integers(0, 40, s.shape[0]).astype(np.uint64) * np.uint64(0x9E3779B97F4A7C15)
    return {"t": t, "P": P, "s": s, "e": e, "key": key, "offsets": np.array(off, np.int64)}


def counter_case(seed: int, n: int = 64, m: int = 8, period: float = 0.02, jitter: float = 0.2,
                 delay: float | None = None, snap: float = 0.3, zero_len: float = 0.1,
                 outside: bool = True, replays: bool = True, keys: int = 5,
                 irregular: bool = False) -> dict:
    """Readings of a cumulative energy counter and a sequence of replay windows.

    Readings come every ``period`` seconds (uniform jitter of ``jitter``
    periods; with ``irregular`` the spacing varies over three decades) and the
    counter never decreases (flat stretches included).  Windows satisfy
    s_0 <= e_0 <= s_1 <= ...; some bounds sit exactly on shifted reading times
    t_j - delay, some windows have zero length, some reach past the readings.
    """
    rng = np.random.default_rng(seed)
    if irregular:
        gaps = period * 10.0 ** rng.uniform(-1.5, 1.5, n - 1)
    else:
        gaps = period * (1.0 + rng.uniform(-jitter, jitter, n - 1))
    t = rng.uniform(-1.0, 1.0) + np.concatenate([[0.0], np.cumsum(gaps)])
    watts = rng.uniform(50.0, 700.0, n - 1)
    watts[rng.random(n - 1) < 0.05] = 0.0
    C = rng.uniform(0.0, 1e4) + np.concatenate([[0.0], np.cumsum(watts * gaps)])
    if delay is None:
        delay = float(rng.choice([0.0, rng.uniform(0.0, 0.3), -rng.uniform(0.0, 0.05)]))
    u = t - delay
    lo, hi = u[0], u[-1]
    pad = 0.1 * (hi - lo) if outside else 0.0
    cuts = np.sort(rng.uniform(lo - pad, hi + pad, 2 * m))
    if snap > 0 and m:
        pick = rng.random(2 * m) < snap
        idx = np.clip(np.searchsorted(u, cuts), 0, n - 1)
        cuts = np.sort(np.where(pick, u[idx], cuts))
    s = cuts[0::2].copy()
    e = cuts[1::2].copy()
    if zero_len > 0 and m:
        e = np.where(rng.random(m) < zero_len, s, e)
    reps = rng.integers(1, 2000, m).astype(np.int32) if replays else None
    vocab = rng.integers(0, 2**63, size=keys, dtype=np.int64).astype(np.uint64) * np.uint64(2) + \
        rng.integers(0, 2, size=keys).astype(np.uint64)
    key = vocab[rng.integers(0, keys, size=m)] if m else np.zeros(0, np.uint64)
    return {"t": t, "C": C, "delay": float(delay), "s": s, "e": e, "reps": reps,
            "key": key.astype(np.uint64)}


def replay_session(seed: int, n_ops: int = 98_304, n_keys: int = 416, rate_hz: float = 50.0,
                   delay: float = 0.1, reps: int = 1000, median_s: float = 20e-6,
                   sigma: float = 1.0) -> dict:
    """A replay profiling session of the energy counter.

    Each of ``n_ops`` operator instances (lognormal duration, keys uniform over
    ``n_keys``) is replayed ``reps`` times back to back; consecutive windows
    are separated by a 10-50 ms pause for setup and settling.  The counter is
    read at ``rate_hz`` (5 % jitter) and lags by ``delay`` seconds; its
    increments follow a power random walk between 100 and 700 W.
    """
    rng = np.random.default_rng(seed)
    dur = np.exp(np.log(median_s) + sigma * rng.standard_normal(n_ops)) * reps
    pause = rng.uniform(0.010, 0.050, n_ops)
    s = np.cumsum(pause + np.concatenate([[0.0], dur[:-1]]))
    e = s + dur
    span = float(e[-1]) + 1.0
    n = int(span * rate_hz) + 2
    t = (np.arange(n) + rng.uniform(-0.05, 0.05, n)) / rate_hz - 0.5 + delay
    t[0] = -0.5 + delay - 1.0 / rate_hz
    watts = np.clip(400.0 + np.cumsum(rng.normal(0.0, 5.0, n - 1)), 100.0, 700.0)
    C = 5e5 + np.concatenate([[0.0], np.cumsum(watts * np.diff(t))])
    vocab = np.array([synth_key(k) for k in range(n_keys)], dtype=np.uint64)
    key = vocab[rng.integers(0, n_keys, n_ops)]
    return {"t": t, "C": C, "delay": float(delay), "s": s, "e": e,
            "reps": np.full(n_ops, reps, np.int32), "key": key}


def synth_key(k: int) -> int:
    """A 64-bit operator key for vocabulary index k (splitmix64 finaliser)."""
    return int(_load().synth_mix64(ctypes.c_uint64(0x4D41474E45544F4E ^ k)))


def graph_pair(seed: int, blocks: int = 8, width: int = 4, decoys: int = 5,
               crossing: int = 0) -> dict:
    """Two computational graphs made of the same sequence of blocks, each block
    built differently in the two graphs (random fan-out width and depth
    between the block's input and output operators), with the block outputs
    declared equivalent, plus decoy pairs between interior operators and
    optionally crossing pairs between block outputs of different positions.
    Node 0 is each graph's input and node n-1 its output."""
    rng = np.random.default_rng(seed)

    def make():
        edges, bounds = [], [0]
        nxt = 1
        interior = []
        for _ in range(blocks):
            a = bounds[-1]
            w = int(rng.integers(1, width + 1))
            tails = []
            for _ in range(w):
                depth = int(rng.integers(1, 4))
                prev = a
                for _ in range(depth):
                    edges.append((prev, nxt))
                    interior.append(nxt)
                    prev = nxt
                    nxt += 1
                tails.append(prev)
            b = nxt
            nxt += 1
            for t in tails:
                edges.append((t, b))
            if rng.random() < 0.3:
                edges.append((a, b))  # a residual edge
            bounds.append(b)
        return nxt, edges, bounds, interior

    n1, e1, b1, i1 = make()
    n2, e2, b2, i2 = make()
    eq = [(x, y) for x, y in zip(b1, b2)]
    for _ in range(decoys):
        eq.append((int(rng.choice(i1)), int(rng.choice(i2))))
    for _ in range(crossing):
        i, j = rng.integers(1, blocks, 2)
        eq.append((b1[int(i)], b2[int(j)]))
    order = rng.permutation(len(eq))
    return {"n1": n1, "edges1": e1, "n2": n2, "edges2": e2,
            "eq": [eq[k] for k in order], "bounds1": b1, "bounds2": b2}
