"""TEST INFRASTRUCTURE ONLY -- the plain CPU oracle for the attribution path.

Only the test suite, the package smoke check and the benchmark's CPU-baseline
leg may import this package.  The library product never does.  The arithmetic
lives in ``oracle.c`` (single-threaded, fp64, no reordering); this module only
compiles it with gcc and marshals numpy arrays.

Pins of the oracle (see tests/test_oracle_pins.py): closed forms for constant,
linear and quadratic power, exact dyadic cases, the equal-split examples,
tiling/additivity/split invariants, brute force on tiny inputs, textbook
lower_bound, M2 closed form and the sign convention of the relative difference
printed in the paper's Table "tab:energy-profiling".  The counter (software
replay) attribution is pinned in tests/test_oracle_counter_pins.py: exact
dyadic closed forms, the delay and replay scenarios worked out by hand,
numpy.interp, exact rational arithmetic and the invariants of a cumulative
quantity.  Per-key latency and the detection rule (flag threshold, waste vs
trade-off) are pinned in tests/test_oracle_detect_pins.py: exactly rounded
sums (math.fsum) by brute force, dyadic closed forms, hand-worked threshold
and tolerance boundaries and a brute-force ranking.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# MAG_ORACLE_SO: another build of oracle.c to load (the sanitizer runs in tests/)
_SO = os.environ.get("MAG_ORACLE_SO") or os.path.join(_HERE, "_oracle.so")
_lib = None


class OracleError(RuntimeError):
    def __init__(self, code: int):
        super().__init__(f"oracle rejected input: status {code}")
        self.code = code


def build(out: str | None = None, extra_flags=()) -> str:
    """Compile oracle.c into _oracle.so (or `out`) with gcc (always recompiles;
    IEEE fp64, no fast-math); extra_flags: e.g. sanitizer options."""
    src = os.path.join(_HERE, "oracle.c")
    so = out or _SO
    tmp = so + ".tmp"
    subprocess.check_call(["gcc", "-O2", "-std=c99", "-fno-fast-math", "-ffp-contract=off",
                           *extra_flags, "-fPIC", "-shared", "-o", tmp, src, "-lm"])
    os.replace(tmp, so)
    return so


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build()
        lib = ctypes.CDLL(_SO)
        p = ctypes.c_void_p
        i64 = ctypes.c_int64
        lib.orc_lower_bound.argtypes = [p, i64, ctypes.c_double]
        lib.orc_lower_bound.restype = i64
        lib.orc_attribute.argtypes = [p, p, i64, p, p, i64, p, ctypes.c_int32, ctypes.c_int32,
                                      p, p, p, p]
        lib.orc_counter_attribute.argtypes = [p, p, i64, ctypes.c_double, p, p, p, i64, p, p, p,
                                              p]
        lib.orc_groupby.argtypes = [p, p, i64, p, p, p, p, p, p]
        lib.orc_key_latency.argtypes = [p, p, p, p, i64, p, p, p]
        lib.orc_diff.argtypes = [p, p, p, i64, p, p, p, i64, i64, p, p, p, p, p, p, p, p]
        lib.orc_ratio.argtypes = [ctypes.c_double, ctypes.c_double]
        lib.orc_ratio.restype = ctypes.c_double
        _lib = lib
    return _lib


def _p(a):
    return ctypes.c_void_p(a.ctypes.data) if a is not None else ctypes.c_void_p(0)


def _c(a, dt):
    return np.ascontiguousarray(a, dtype=dt)


def lower_bound(t, x) -> int:
    t = _c(t, np.float64)
    return int(_load().orc_lower_bound(_p(t), t.shape[0], float(x)))


def ratio(ea: float, eb: float) -> float:
    return float(_load().orc_ratio(ea, eb))


def attribute(t, P, s, e, offsets=None, equal_split: bool = True) -> dict:
    """Per-interval energy (J), lower_bound indices and whole-trace figures."""
    t = _c(t, np.float64)
    P = _c(P, np.float32)
    s = _c(s, np.float64)
    e = _c(e, np.float64)
    m = s.shape[0]
    off = None if offsets is None else _c(offsets, np.int64)
    n_streams = 1 if off is None else off.shape[0] - 1
    energy = np.zeros(m, dtype=np.float64)
    si = np.zeros(m, dtype=np.int64)
    ei = np.zeros(m, dtype=np.int64)
    summ = np.zeros(4, dtype=np.float64)
    rc = _load().orc_attribute(_p(t), _p(P), t.shape[0], _p(s), _p(e), m, _p(off), n_streams,
                               1 if equal_split else 0, _p(energy), _p(si), _p(ei), _p(summ))
    if rc != 0:
        raise OracleError(rc)
    return {"energy": energy, "start_idx": si, "end_idx": ei, "trace_energy": float(summ[0]),
            "idle_energy": float(summ[1]), "attributed_energy": float(summ[2]),
            "n_clipped": int(summ[3])}


def counter_attribute(t, C, s, e, delay: float = 0.0, reps=None) -> dict:
    """Per-window operator energy (J per replay) from a cumulative energy counter.

    Readings C[j] taken at t[j] hold the energy used up to t[j] - delay; the
    counter is interpolated linearly between readings and held outside them;
    window i ran its operator reps[i] times (1 when reps is None).
    """
    t = _c(t, np.float64)
    C = _c(C, np.float64)
    s = _c(s, np.float64)
    e = _c(e, np.float64)
    m = s.shape[0]
    r = None if reps is None else _c(reps, np.int32)
    energy = np.zeros(m, dtype=np.float64)
    si = np.zeros(m, dtype=np.int64)
    ei = np.zeros(m, dtype=np.int64)
    summ = np.zeros(4, dtype=np.float64)
    rc = _load().orc_counter_attribute(_p(t), _p(C), t.shape[0], float(delay), _p(s), _p(e), _p(r),
                                       m, _p(energy), _p(si), _p(ei), _p(summ))
    if rc != 0:
        raise OracleError(rc)
    return {"energy": energy, "start_idx": si, "end_idx": ei, "trace_energy": float(summ[0]),
            "idle_energy": float(summ[1]), "attributed_energy": float(summ[2]),
            "n_clipped": int(summ[3])}


def groupby(keys, energy) -> dict:
    """Per distinct key in ascending order: count, sum, two-pass M2, Welford M2."""
    keys = _c(keys, np.uint64)
    energy = _c(energy, np.float64)
    m = keys.shape[0]
    ok = np.zeros(max(m, 1), np.uint64)
    oc = np.zeros(max(m, 1), np.int64)
    osum = np.zeros(max(m, 1), np.float64)
    om2 = np.zeros(max(m, 1), np.float64)
    omw = np.zeros(max(m, 1), np.float64)
    nk = np.zeros(1, np.int64)
    rc = _load().orc_groupby(_p(keys), _p(energy), m, _p(ok), _p(oc), _p(osum), _p(om2), _p(omw),
                             _p(nk))
    if rc != 0:
        raise OracleError(rc)
    r = int(nk[0])
    return {"keys": ok[:r].copy(), "count": oc[:r].copy(), "sum": osum[:r].copy(),
            "m2": om2[:r].copy(), "m2_welford": omw[:r].copy()}


def key_latency(keys, starts, ends, reps=None) -> dict:
    """Per distinct key in ascending order: the sum of its interval durations
    (end - start, divided by the replay count when reps is given)."""
    keys = _c(keys, np.uint64)
    s = _c(starts, np.float64)
    e = _c(ends, np.float64)
    r = None if reps is None else _c(reps, np.int32)
    m = keys.shape[0]
    ok = np.zeros(max(m, 1), np.uint64)
    ol = np.zeros(max(m, 1), np.float64)
    nk = np.zeros(1, np.int64)
    rc = _load().orc_key_latency(_p(keys), _p(s), _p(e), _p(r), m, _p(ok), _p(ol), _p(nk))
    if rc != 0:
        raise OracleError(rc)
    n = int(nk[0])
    return {"keys": ok[:n].copy(), "latency": ol[:n].copy()}


WASTE = 1
TRADEOFF = 2


def detect(a: dict, b: dict, threshold: float = 0.10, tolerance: float = 0.01) -> dict:
    """Section 6.1's detection rule over two per-key tables (keys ascending,
    with sum, count and latency).

    A key present on both sides is flagged when B's energy exceeds A's by at
    least `threshold` of A's, r = (E_B - E_A)/E_A >= threshold (10 %, or 5 %).
    A flagged key is waste when the efficient side A is not slower than B by
    more than `tolerance` of B's latency, (L_A - L_B) <= tolerance * L_B
    (1 %); otherwise B trades the extra energy for speed.  Rows come in the
    ranking's order (r descending, key ascending).
    """
    full = diff(a, b, len(a["keys"]))  # every joined key, ranked
    flag = full["ratio"] >= threshold
    nf = int(np.count_nonzero(flag))
    assert np.all(flag[:nf]), "flagged keys form a prefix of the ranking"
    ka = _c(a["keys"], np.uint64)
    kb = _c(b["keys"], np.uint64)
    keys = full["key"][:nf]
    la = _c(a["latency"], np.float64)[np.searchsorted(ka, keys)]
    lb = _c(b["latency"], np.float64)[np.searchsorted(kb, keys)]
    verdict = np.where((la - lb) <= tolerance * lb, WASTE, TRADEOFF).astype(np.int32)
    return {"key": keys, "ratio": full["ratio"][:nf], "energy_a": full["energy_a"][:nf],
            "energy_b": full["energy_b"][:nf], "latency_a": la, "latency_b": lb,
            "verdict": verdict, "n_flagged": nf,
            "n_waste": int(np.count_nonzero(verdict == WASTE)),
            "n_tradeoff": int(np.count_nonzero(verdict == TRADEOFF))}


def diff(a: dict, b: dict, k: int) -> dict:
    """Join two key tables (dicts with keys/sum/count) and rank by (E_B - E_A)/E_A."""
    ka, sa, ca = _c(a["keys"], np.uint64), _c(a["sum"], np.float64), _c(a["count"], np.int64)
    kb, sb, cb = _c(b["keys"], np.uint64), _c(b["sum"], np.float64), _c(b["count"], np.int64)
    cap = max(1, min(int(k), ka.shape[0]))
    okey = np.zeros(cap, np.uint64)
    orr = np.zeros(cap, np.float64)
    oea = np.zeros(cap, np.float64)
    oeb = np.zeros(cap, np.float64)
    oca = np.zeros(cap, np.int64)
    ocb = np.zeros(cap, np.int64)
    counts = np.zeros(4, np.int64)
    margin = np.zeros(1, np.float64)
    rc = _load().orc_diff(_p(ka), _p(sa), _p(ca), ka.shape[0], _p(kb), _p(sb), _p(cb), kb.shape[0],
                          int(k), _p(okey), _p(orr), _p(oea), _p(oeb), _p(oca), _p(ocb),
                          _p(counts), _p(margin))
    if rc != 0:
        raise OracleError(rc)
    r = int(counts[0])
    return {"key": okey[:r].copy(), "ratio": orr[:r].copy(), "energy_a": oea[:r].copy(),
            "energy_b": oeb[:r].copy(), "count_a": oca[:r].copy(), "count_b": ocb[:r].copy(),
            "n_only_a": int(counts[1]), "n_only_b": int(counts[2]), "n_join": int(counts[3]),
            "margin": float(margin[0])}
