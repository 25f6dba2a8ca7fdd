"""Pins of the CPU oracle against things other than itself.

Each test fixes the oracle to a closed form, an invariant of the integral, a
textbook routine, a brute-force computation written independently here, or a
number printed in the paper.  Together they are meant to fail on any plausible
slip in the oracle: a dropped 1/2, interpolation replaced by a zero-order hold,
a wrong lower/upper bound, a mis-split of concurrent power, a swapped operand in
the relative difference, a wrong tie order, a wrong M2.
"""
from fractions import Fraction
import os

import math

import numpy as np
import pytest

import oracle
import synth

HERE = os.path.dirname(os.path.abspath(__file__))


# ---------------------------------------------------------------------------
# independent brute force (numpy.interp + midpoint membership)
# ---------------------------------------------------------------------------

def brute_force(t, P, s, e, equal_split=True):
    """Cut [t0, tn] at every sample and every clipped bound; on each piece the
    interpolant is linear, so its trapezoid is exact; the piece's energy goes
    to the intervals that contain the piece's midpoint."""
    t = np.asarray(t, np.float64)
    Pd = np.asarray(P, np.float32).astype(np.float64)
    lo, hi = t[0], t[-1]
    pts = set(t.tolist())
    for x in list(s) + list(e):
        if lo < x < hi:
            pts.add(float(x))
    pts = sorted(pts)
    E = np.zeros(len(s))
    idle = 0.0
    for u, v in zip(pts[:-1], pts[1:]):
        q = 0.5 * (np.interp(u, t, Pd) + np.interp(v, t, Pd)) * (v - u)
        mid = 0.5 * (u + v)
        act = [i for i in range(len(s)) if s[i] <= mid < e[i]]
        if not act:
            idle += q
        for i in act:
            E[i] += q / len(act) if equal_split else q
    return E, idle


def exact_integral(t, P, a, b):
    """Exact rational integral of the piecewise-linear interpolant on [a, b]."""
    t = [Fraction(float(x)) for x in t]
    P = [Fraction(float(x)) for x in np.asarray(P, np.float32)]
    a, b = Fraction(float(a)), Fraction(float(b))
    a, b = max(a, t[0]), min(b, t[-1])
    total = Fraction(0)
    if b <= a:
        return total
    for j in range(len(t) - 1):
        lo, hi = max(a, t[j]), min(b, t[j + 1])
        if hi <= lo:
            continue
        f = lambda x: P[j] + (P[j + 1] - P[j]) * (x - t[j]) / (t[j + 1] - t[j])
        total += (f(lo) + f(hi)) / 2 * (hi - lo)
    return total


def rel_err(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return np.abs(a - b) / np.maximum(np.abs(b), 1e-300)


# ---------------------------------------------------------------------------
# lower_bound
# ---------------------------------------------------------------------------

def test_lower_bound_is_searchsorted_left():
    rng = np.random.default_rng(1)
    t = np.cumsum(rng.uniform(0.1, 1.0, 500))
    xs = np.concatenate([rng.uniform(t[0] - 5, t[-1] + 5, 400), t[::7], [t[0], t[-1]]])
    for x in xs:
        assert oracle.lower_bound(t, x) == int(np.searchsorted(t, x, side="left"))


# ---------------------------------------------------------------------------
# closed forms of the power model
# ---------------------------------------------------------------------------

def test_constant_power_is_power_times_duration():
    rng = np.random.default_rng(2)
    t = np.cumsum(rng.uniform(0.5, 1.5, 300))
    P = np.full(300, 412.5, np.float32)
    a = np.sort(rng.uniform(t[0], t[-1], 60))
    s, e = a[0::2], a[1::2]
    r = oracle.attribute(t, P, s, e)
    assert np.max(rel_err(r["energy"], 412.5 * (e - s))) < 1e-13


def test_linear_power_is_integrated_exactly():
    # P = 100 + 4 t on t_j = j/8: every sample is exact in fp32, so the
    # interpolant IS the line and any interval has a closed-form energy.
    t = np.arange(801, dtype=np.float64) / 8.0
    P = (100.0 + 4.0 * t).astype(np.float32)
    rng = np.random.default_rng(3)
    a = np.sort(rng.uniform(0.0, 100.0, 200))
    s, e = a[0::2], a[1::2]
    # alpha (e - s) + beta (e^2 - s^2) / 2, factored to avoid cancellation
    want = (e - s) * (100.0 + 4.0 * (e + s) / 2.0)
    r = oracle.attribute(t, P, s, e)
    assert np.max(rel_err(r["energy"], want)) < 1e-12


def test_quadratic_power_has_trapezoid_excess():
    # P = t^2 sampled on h = 1/64: the composite trapezoid overestimates the
    # integral of t^2 by exactly h^2 (b - a) / 6 on grid-aligned [a, b].
    h = 1.0 / 64.0
    t = np.arange(641, dtype=np.float64) * h
    P = (t * t).astype(np.float32)
    assert np.array_equal(P.astype(np.float64), t * t)
    s = np.array([0.0, 1.0, 2.5, 0.25])
    e = np.array([10.0, 3.0, 7.75, 0.25 + 64 * h])
    r = oracle.attribute(t, P, s, e, offsets=np.arange(5), equal_split=False)
    want = (e ** 3 - s ** 3) / 3.0 + h * h * (e - s) / 6.0
    assert np.max(rel_err(r["energy"], want)) < 1e-12


def test_interpolation_not_zero_order_hold():
    # one segment rising 0 -> 2 W over 1 s: the first half carries 0.25 J
    # (linear), not 0 J (left hold) or 1 J (right hold)
    r = oracle.attribute(np.array([0.0, 1.0]), np.array([0.0, 2.0], np.float32),
                         np.array([0.0, 0.5]), np.array([0.5, 1.0]))
    assert r["energy"].tolist() == [0.25, 0.75]


def test_dyadic_traces_are_exact():
    # on dyadic grids every partial result is exact in fp64, so the oracle
    # must equal the exact rational integral bit for bit
    for seed in range(40):
        c = synth.tiny_case(seed, n=40, streams=1, per_stream=10, dyadic=True)
        r = oracle.attribute(c["t"], c["P"], c["s"], c["e"], c["offsets"])
        for i in range(c["s"].shape[0]):
            want = exact_integral(c["t"], c["P"], c["s"][i], c["e"][i])
            assert Fraction(r["energy"][i]) == want, (seed, i)


def test_dyadic_two_streams_split_exact():
    # with two streams every concurrency is 1 or 2, so halving stays exact
    for seed in range(20):
        c = synth.tiny_case(100 + seed, n=30, streams=2, per_stream=6, dyadic=True)
        r = oracle.attribute(c["t"], c["P"], c["s"], c["e"], c["offsets"])
        E, _ = brute_force(c["t"], c["P"], c["s"], c["e"])
        assert np.array_equal(r["energy"], E), seed


# ---------------------------------------------------------------------------
# equal split
# ---------------------------------------------------------------------------

def test_equal_split_two_overlapping():
    t = np.linspace(0.0, 4.0, 9)
    P = np.full(9, 10.0, np.float32)
    r = oracle.attribute(t, P, np.array([0.0, 1.0]), np.array([2.0, 3.0]),
                         offsets=np.array([0, 1, 2]))
    # [0,1): alone (10 J), [1,2): shared (5 J each), [2,3): alone
    assert np.allclose(r["energy"], [15.0, 15.0], rtol=0, atol=1e-12)
    assert abs(r["idle_energy"] - 10.0) < 1e-12


def test_equal_split_k_identical():
    t = np.linspace(0.0, 10.0, 101)
    P = np.full(101, 300.0, np.float32)
    k = 3
    r = oracle.attribute(t, P, np.full(k, 2.0), np.full(k, 5.0),
                         offsets=np.arange(k + 1))
    assert np.allclose(r["energy"], 300.0 * 3.0 / k, rtol=1e-13)


def test_one_busy_stream_equals_sequential():
    c = synth.tiny_case(7, n=80, streams=1, per_stream=12)
    empty = np.array([0, 0, c["s"].shape[0], c["s"].shape[0], c["s"].shape[0]])
    r4 = oracle.attribute(c["t"], c["P"], c["s"], c["e"], empty)
    r1 = oracle.attribute(c["t"], c["P"], c["s"], c["e"], c["offsets"], equal_split=False)
    assert np.max(np.abs(r4["energy"] - r1["energy"])) <= 1e-12 * max(1.0, r1["energy"].max())


def test_no_split_gives_each_interval_the_full_power():
    t = np.linspace(0.0, 4.0, 9)
    P = np.full(9, 10.0, np.float32)
    r = oracle.attribute(t, P, np.array([0.0, 1.0]), np.array([2.0, 3.0]),
                         offsets=np.array([0, 1, 2]), equal_split=False)
    assert np.allclose(r["energy"], [20.0, 20.0], rtol=1e-14)


# ---------------------------------------------------------------------------
# invariants
# ---------------------------------------------------------------------------

def test_tiling_intervals_sum_to_trace_energy():
    rng = np.random.default_rng(5)
    t = np.cumsum(rng.uniform(0.1, 1.0, 400))
    P = rng.uniform(50, 700, 400).astype(np.float32)
    cuts = np.concatenate([[t[0]], np.sort(rng.uniform(t[0], t[-1], 99)), [t[-1]]])
    r = oracle.attribute(t, P, cuts[:-1], cuts[1:])
    W = r["trace_energy"]
    assert abs(r["energy"].sum() - W) <= 1e-12 * W
    assert abs(r["idle_energy"]) <= 1e-12 * W
    # trace energy by the plain composite trapezoid rule (numpy)
    assert abs(W - np.trapezoid(P.astype(np.float64), t)) <= 1e-12 * W


def test_additivity_under_splitting():
    rng = np.random.default_rng(6)
    t = np.cumsum(rng.uniform(0.1, 1.0, 300))
    P = rng.uniform(0, 900, 300).astype(np.float32)
    for _ in range(50):
        a, x, b = np.sort(rng.uniform(t[0] - 2, t[-1] + 2, 3))
        whole = oracle.attribute(t, P, np.array([a]), np.array([b]))["energy"][0]
        parts = oracle.attribute(t, P, np.array([a, x]), np.array([x, b]))["energy"].sum()
        assert abs(whole - parts) <= 1e-12 * max(whole, 1e-300)


def test_non_negative_and_idle_plus_attributed_is_trace():
    for seed in range(30):
        c = synth.tiny_case(200 + seed, n=60, streams=1 + seed % 4, per_stream=10)
        r = oracle.attribute(c["t"], c["P"], c["s"], c["e"], c["offsets"])
        assert (r["energy"] >= 0).all()
        W = r["trace_energy"]
        assert abs(r["attributed_energy"] + r["idle_energy"] - W) <= 1e-12 * max(W, 1.0)


def test_split_trace_at_a_sample():
    # attributing the two halves of a trace split at sample k and adding the
    # parts of each interval reproduces the unsplit result
    for seed in range(20):
        c = synth.tiny_case(300 + seed, n=70, streams=1 + seed % 3, per_stream=10)
        k = 20 + seed
        t, P = c["t"], c["P"]
        full = oracle.attribute(t, P, c["s"], c["e"], c["offsets"])["energy"]
        lo = oracle.attribute(t[:k + 1], P[:k + 1], c["s"], c["e"], c["offsets"])["energy"]
        hi = oracle.attribute(t[k:], P[k:], c["s"], c["e"], c["offsets"])["energy"]
        assert np.max(np.abs(lo + hi - full)) <= 1e-12 * max(full.max(), 1.0)


def test_sample_indices_are_unclipped_lower_bounds():
    c = synth.tiny_case(9, n=50, streams=3, per_stream=12)
    r = oracle.attribute(c["t"], c["P"], c["s"], c["e"], c["offsets"])
    assert np.array_equal(r["start_idx"], np.searchsorted(c["t"], c["s"], side="left"))
    assert np.array_equal(r["end_idx"], np.searchsorted(c["t"], c["e"], side="left"))
    clipped = int(((c["s"] < c["t"][0]) | (c["e"] > c["t"][-1])).sum())
    assert r["n_clipped"] == clipped


# ---------------------------------------------------------------------------
# brute force on tiny inputs
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("streams", [1, 2, 3, 4])
def test_brute_force_tiny(streams):
    for seed in range(60):
        c = synth.tiny_case(1000 * streams + seed, n=int(10 + seed % 40), streams=streams,
                            per_stream=int(2 + seed % 9))
        for split in (True, False):
            r = oracle.attribute(c["t"], c["P"], c["s"], c["e"], c["offsets"], equal_split=split)
            E, idle = brute_force(c["t"], c["P"], c["s"], c["e"], equal_split=split)
            scale = max(r["trace_energy"], 1e-300)
            assert np.all(np.abs(r["energy"] - E) <= 1e-12 * np.maximum(E, 1e-3 * scale)), seed
            assert abs(r["idle_energy"] - idle) <= 1e-12 * scale


# ---------------------------------------------------------------------------
# group-by
# ---------------------------------------------------------------------------

def test_m2_closed_form():
    g = oracle.groupby(np.array([7, 7, 7, 7], np.uint64), np.array([1.0, 2.0, 3.0, 4.0]))
    assert g["count"].tolist() == [4]
    assert g["sum"].tolist() == [10.0]
    assert g["m2"].tolist() == [5.0]
    assert g["m2_welford"].tolist() == [5.0]


def test_groupby_matches_dict_and_numpy():
    rng = np.random.default_rng(11)
    vocab = np.array([0, 1, 2**63, 2**64 - 1, 12345678901234567890, 42], np.uint64)
    keys = vocab[rng.integers(0, len(vocab), 5000)]
    E = rng.lognormal(-3, 1.0, 5000)
    g = oracle.groupby(keys, E)
    ref = {}
    for k, x in zip(keys.tolist(), E.tolist()):
        ref.setdefault(k, []).append(x)
    assert g["keys"].tolist() == sorted(ref)  # ascending unsigned
    for k, c, s, m2, m2w in zip(g["keys"].tolist(), g["count"], g["sum"], g["m2"], g["m2_welford"]):
        xs = np.array(ref[k])
        assert c == len(xs)
        assert abs(s - xs.sum()) <= 1e-12 * xs.sum()
        want = np.var(xs) * len(xs)
        assert abs(m2 - want) <= 1e-10 * want
        assert abs(m2w - m2) <= 1e-10 * (m2 + len(xs) * xs.mean() ** 2)


def test_groupby_empty():
    g = oracle.groupby(np.zeros(0, np.uint64), np.zeros(0))
    assert g["keys"].shape == (0,)


# ---------------------------------------------------------------------------
# diff
# ---------------------------------------------------------------------------

def _read_energy_profiling():
    rows = []
    with open(os.path.join(HERE, "golden", "energy_profiling.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            op, phys, zeus, zerr, rep, rerr = line.split()
            rows.append((op, float(phys), float(zeus), float(zerr), float(rep), float(rerr)))
    return rows


def test_relative_difference_matches_paper_table():
    # The printed watts are rounded to 1 W, so the printed error must lie in
    # the range of (value - physical)/physical over values within +-0.5 W.
    rows = _read_energy_profiling()
    keys = np.arange(len(rows), dtype=np.uint64)
    ones = np.ones(len(rows), np.int64)
    phys = np.array([r[1] for r in rows])
    for col_v, col_err in ((2, 3), (4, 5)):
        vals = np.array([r[col_v] for r in rows])
        d = oracle.diff({"keys": keys, "sum": phys, "count": ones},
                        {"keys": keys, "sum": vals, "count": ones}, k=len(rows))
        by_key = dict(zip(d["key"].tolist(), d["ratio"].tolist()))
        for i, r in enumerate(rows):
            printed = r[col_err] / 100.0
            lo = min((r[col_v] + dv - (r[1] + dp)) / (r[1] + dp)
                     for dv in (-0.5, 0.5) for dp in (-0.5, 0.5))
            hi = max((r[col_v] + dv - (r[1] + dp)) / (r[1] + dp)
                     for dv in (-0.5, 0.5) for dp in (-0.5, 0.5))
            assert lo - 0.0005 <= printed <= hi + 0.0005, r[0]
            assert abs(by_key[i] - printed) < 0.001, r[0]


def test_ratio_zero_baseline():
    assert oracle.ratio(0.0, 0.0) == 0.0
    assert oracle.ratio(0.0, 1.0) == float("inf")
    assert oracle.ratio(2.0, 3.0) == 0.5


def test_topk_order_and_join_counts():
    rng = np.random.default_rng(12)
    ka = np.sort(rng.choice(2**40, 300, replace=False)).astype(np.uint64)
    kb = np.sort(np.concatenate([ka[:250], rng.choice(2**40, 30, replace=False).astype(np.uint64)]))
    kb = np.unique(kb)
    sa = rng.uniform(1, 100, ka.shape[0])
    # quantised ratios force exact ties, broken by key ascending
    sb = np.array([sa[np.searchsorted(ka, k)] * (1 + rng.integers(-4, 5) / 8.0)
                   if k in set(ka.tolist()) else rng.uniform(1, 100) for k in kb.tolist()])
    ca = rng.integers(1, 10, ka.shape[0])
    cb = rng.integers(1, 10, kb.shape[0])
    for k in (0, 1, 10, 100, 1000):
        d = oracle.diff({"keys": ka, "sum": sa, "count": ca}, {"keys": kb, "sum": sb, "count": cb}, k)
        ia = {x: i for i, x in enumerate(ka.tolist())}
        ib = {x: i for i, x in enumerate(kb.tolist())}
        common = sorted(set(ia) & set(ib))
        rows = sorted(((sb[ib[x]] - sa[ia[x]]) / sa[ia[x]], x) for x in common)
        rows = sorted(rows, key=lambda p: (-p[0], p[1]))[:k]
        assert d["key"].tolist() == [x for _, x in rows]
        assert np.array_equal(d["ratio"], np.array([r for r, _ in rows]))
        assert d["n_only_a"] == len(set(ia) - set(ib))
        assert d["n_only_b"] == len(set(ib) - set(ia))


def _margin_brute(ka, sa, kb, sb, k):
    """Smallest gap r_p - r_{p+1} between adjacent rows among the first k+1
    rows of the full ranking (by sorting every joined key); a pair of equal
    infinite ratios (both baselines zero) has no numeric gap and is skipped;
    infinity when no pair is compared."""
    ib = {x: i for i, x in enumerate(kb.tolist())}
    rows = []
    for i, x in enumerate(ka.tolist()):
        if x in ib:
            a, b = float(sa[i]), float(sb[ib[x]])
            r = (b - a) / a if a != 0.0 else (math.inf if b > 0.0 else 0.0)
            rows.append((r, x))
    rows.sort(key=lambda q: (-q[0], q[1]))
    gaps = [rows[u][0] - rows[u + 1][0] for u in range(min(k, len(rows) - 1))]
    gaps = [g for g in gaps if not math.isnan(g)]
    return min(gaps) if gaps else math.inf


def test_separation_margin_by_brute_force():
    """The margin guards every top-k parity assertion: it must be the smallest
    adjacent gap over exactly the first k+1 ranked rows."""
    rng = np.random.default_rng(31)
    ka = np.sort(rng.choice(2**40, 400, replace=False)).astype(np.uint64)
    kb = np.unique(np.concatenate([ka[50:], rng.choice(2**40, 40).astype(np.uint64)]))
    sa = rng.uniform(1, 100, ka.shape[0])
    sa[:10] = 0.0  # zero baselines: ratios +inf (or 0) on the joined ones
    sb = rng.uniform(1, 100, kb.shape[0])
    sb[::17] = 0.0
    ca = np.ones(ka.shape[0], np.int64)
    cb = np.ones(kb.shape[0], np.int64)
    nj = len(set(ka.tolist()) & set(kb.tolist()))
    for k in (0, 1, 2, 7, 100, nj - 1, nj, nj + 25):
        d = oracle.diff({"keys": ka, "sum": sa, "count": ca}, {"keys": kb, "sum": sb, "count": cb}, k)
        assert d["margin"] == _margin_brute(ka, sa, kb, sb, k), k
    # quantised ratios give exact ties: a zero margin once a tie is inside
    sbq = np.array([sa[np.searchsorted(ka, x)] * (1 + rng.integers(-3, 4) / 4.0)
                    if x in set(ka.tolist()) and sa[np.searchsorted(ka, x)] > 0 else 5.0
                    for x in kb.tolist()])
    for k in (3, 50, nj + 1):
        d = oracle.diff({"keys": ka, "sum": sa, "count": ca}, {"keys": kb, "sum": sbq, "count": cb},
                        k)
        assert d["margin"] == _margin_brute(ka, sa, kb, sbq, k) == 0.0, k


def test_separation_margin_worked_example():
    """Ratios 3, 2.5, 2.25, 2, 1.999 on five keys (E_A = 1, E_B = 1 + r): the
    gaps are 0.5, 0.25, 0.25, 0.001; only the first k+1 rows count."""
    ka = np.array([10, 20, 30, 40, 50], np.uint64)
    sa = np.ones(5)
    sb = 1.0 + np.array([2.0, 1.999, 3.0, 2.25, 2.5])  # r of keys 10, 20, 30, 40, 50
    c = np.ones(5, np.int64)
    want = {0: math.inf, 1: 0.5, 2: 0.25, 3: 0.25, 4: 1.0 - 0.999, 5: 1.0 - 0.999, 9: 1.0 - 0.999}
    for k, m in want.items():
        d = oracle.diff({"keys": ka, "sum": sa, "count": c}, {"keys": ka, "sum": sb, "count": c}, k)
        assert d["key"].tolist() == [30, 50, 40, 10, 20][:k], k
        assert math.isclose(d["margin"], m, rel_tol=1e-12) or d["margin"] == m, (k, d["margin"])
    # one joined key, or none: no pair, infinite margin
    d = oracle.diff({"keys": ka[:1], "sum": sa[:1], "count": c[:1]},
                    {"keys": ka[:1], "sum": sb[:1], "count": c[:1]}, 10)
    assert d["margin"] == math.inf


# ---------------------------------------------------------------------------
# validation
# ---------------------------------------------------------------------------

def test_oracle_rejects_invalid_inputs():
    t = np.array([0.0, 1.0, 2.0])
    P = np.array([1.0, 2.0, 3.0], np.float32)
    ok_s, ok_e = np.array([0.5]), np.array([1.5])
    cases = [
        (np.array([0.0, 1.0, 1.0]), P, ok_s, ok_e, None, -5),
        (np.array([0.0, np.nan, 2.0]), P, ok_s, ok_e, None, -5),
        (t, np.array([1.0, -1.0, 3.0], np.float32), ok_s, ok_e, None, -6),
        (t, np.array([1.0, np.inf, 3.0], np.float32), ok_s, ok_e, None, -6),
        (t, P, np.array([1.5]), np.array([0.5]), None, -7),
        (t, P, np.array([0.0, 0.5]), np.array([1.0, 1.5]), None, -7),
        (t, P, np.array([0.0, 0.5]), np.array([1.0, 1.5]), np.array([0, 1, 3]), -8),
        (t[:1], P[:1], ok_s, ok_e, None, -2),
    ]
    for tt, pp, s, e, off, code in cases:
        with pytest.raises(oracle.OracleError) as ei:
            oracle.attribute(tt, pp, s, e, off)
        assert ei.value.code == code
