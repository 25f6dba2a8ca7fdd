"""Pins of the oracle's counter (software replay) attribution.

Section 5.2's software mode reads a cumulative energy counter that is refreshed
at 10-50 Hz and lags the device; operators are replayed until the window is
long enough, and the operator's energy is the counter's increase over the
window divided by the number of replays.  The oracle's reading: readings
(t_j - delay, C_j), linear interpolation between them, held constant outside
them.  Each test below fixes that arithmetic to something other than the
oracle's own code: exact closed forms on dyadic grids, the delay and replay
scenarios worked out by hand, numpy.interp, exact rational arithmetic, and the
invariants of a cumulative quantity (additivity, telescoping, monotonicity).
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle

EPS = np.finfo(np.float64).eps


def counter_trace(rng, n, t0=0.0, period=0.02, jitter=0.2, watts=(50.0, 400.0)):
    """Readings at roughly `period` spacing with a non-decreasing counter."""
    t = t0 + period * (np.arange(n) + rng.uniform(-jitter, jitter, n))
    C = 1000.0 + np.concatenate([[0.0], np.cumsum(rng.uniform(*watts, n - 1) * np.diff(t))])
    return t, C


def sequential_windows(rng, lo, hi, m):
    """m windows s_0 <= e_0 <= s_1 <= ... inside [lo, hi] (some of zero length)."""
    x = np.sort(rng.uniform(lo, hi, 2 * m))
    s, e = x[0::2].copy(), x[1::2].copy()
    e[::11] = s[::11]
    return s, e


def exact_increase(u, C, x, y):
    """C^(y) - C^(x) in exact rational arithmetic from the definition: the
    interpolant through (u_j, C_j), held at C_0 before u_0 and C_{n-1} after."""
    U = [Fraction(v) for v in u]
    K = [Fraction(v) for v in C]

    def at(z):
        z = Fraction(z)
        if z <= U[0]:
            return K[0]
        if z >= U[-1]:
            return K[-1]
        j = int(np.searchsorted(u, float(z), side="right")) - 1
        while not (U[j] <= z <= U[j + 1]):
            j += 1 if z > U[j + 1] else -1
        return K[j] + (K[j + 1] - K[j]) * (z - U[j]) / (U[j + 1] - U[j])

    return at(y) - at(x)


# ---------------------------------------------------------------------------
# indices
# ---------------------------------------------------------------------------

def test_indices_are_searchsorted_of_the_shifted_times():
    rng = np.random.default_rng(10)
    t, C = counter_trace(rng, 400)
    delay = 0.137
    u = t - delay
    # bounds drawn at random, plus some exactly on shifted readings
    x = np.sort(np.concatenate([rng.uniform(u[0] - 0.5, u[-1] + 0.5, 150),
                                u[[0, 100, 103, 103, 250, 399]], [u[-1] + 1.0, u[-1] + 2.0]]))
    s, e = x[0::2], x[1::2]
    r = oracle.counter_attribute(t, C, s, e, delay=delay)
    assert np.array_equal(r["start_idx"], np.searchsorted(u, s, side="left"))
    assert np.array_equal(r["end_idx"], np.searchsorted(u, e, side="left"))


# ---------------------------------------------------------------------------
# closed forms
# ---------------------------------------------------------------------------

def test_linear_counter_gives_slope_times_duration_exactly():
    """C_j = 7 + 5 u_j on a dyadic grid: C^(e) - C^(s) = 5 (e - s) with no
    rounding at all, so E_i = 5 (e_i - s_i) / N_i bit for bit."""
    rng = np.random.default_rng(11)
    delay = 0.25
    t = np.arange(400) / 16.0
    u = t - delay
    C = 7.0 + 5.0 * u
    grid = np.sort(rng.choice(np.arange(int(u[0] * 1024), int(u[-1] * 1024) + 1), 120,
                              replace=False)) / 1024.0
    s, e = grid[0::2], grid[1::2]
    reps = rng.integers(1, 2000, s.shape[0]).astype(np.int32)
    reps[:4] = [1, 2, 1000, 3]
    r = oracle.counter_attribute(t, C, s, e, delay=delay, reps=reps)
    want = (5.0 * (e - s)) / reps
    assert np.array_equal(r["energy"], want)
    assert r["trace_energy"] == 5.0 * (u[-1] - u[0])


def test_interpolation_between_readings_not_a_step():
    # readings 0 J at t = 0 and 10 J at t = 1: half way the counter holds 5 J
    r = oracle.counter_attribute([0.0, 1.0], [0.0, 10.0], [0.0, 0.5], [0.5, 1.0])
    assert list(r["energy"]) == [5.0, 5.0]


def test_delay_shift_recovers_the_window():
    """100 W during [1, 2) s, nothing else; readings every 1/8 s that report
    the energy used up to 1/4 s before the reading.  With the right delay the
    window [1, 2] holds all 100 J; ignoring the delay (or doubling it) moves a
    quarter of it out of the window."""
    t = np.arange(33) / 8.0
    true_at = lambda x: 100.0 * np.clip(x - 1.0, 0.0, 1.0)
    C = true_at(t - 0.25)
    for delay, want in [(0.25, 100.0), (0.0, 75.0), (0.5, 75.0)]:
        r = oracle.counter_attribute(t, C, [1.0], [2.0], delay=delay)
        assert r["energy"][0] == want, delay
    r = oracle.counter_attribute(t, C, [1.0], [2.0], delay=0.25)
    assert r["trace_energy"] == 100.0 and r["idle_energy"] == 0.0


def test_replay_average_is_the_per_run_energy():
    """An operator drawing 300 W for 2^-12 s, replayed 1024 times back to back
    over a 90 W idle floor, read at 64 Hz with a 2^-3 s lag.  Window bounds on
    readings: E = 300 * 2^-12 J exactly.  Window bounds between readings: the
    interpolant is off by at most (300 - 90) h / 4 at each bound (the largest
    gap between a kinked line and its chord), divided by the replays."""
    h, d, N, delay = 2.0 ** -6, 2.0 ** -12, 1024, 2.0 ** -3
    t = np.arange(2048) * h

    def run(s0):
        e0 = s0 + N * d
        def true_at(x):
            x = np.asarray(x, np.float64)
            return 90.0 * x + (300.0 - 90.0) * np.clip(x - s0, 0.0, e0 - s0)
        C = true_at(t - delay)
        return oracle.counter_attribute(t, C, [s0], [e0], delay=delay,
                                        reps=np.array([N], np.int32))["energy"][0]

    assert run(4.0) == 300.0 * d
    for s0 in [4.0 + 0.3 * h, 7.0 + 0.77 * h, 9.5 + 0.5 * h]:
        assert abs(run(s0) - 300.0 * d) <= 2 * (300.0 - 90.0) * h / 4 / N + 1e-12


def test_held_outside_the_readings():
    t = np.array([10.0, 11.0, 12.0, 13.0])
    C = np.array([100.0, 150.0, 170.0, 230.0])
    s = np.array([0.0, 5.0, 10.5, 12.5, 20.0])
    e = np.array([4.0, 10.5, 12.5, 20.0, 30.0])
    r = oracle.counter_attribute(t, C, s, e)
    # [0,4]: before the readings; [5,10.5]: only 10..10.5 counts = 25;
    # [10.5,12.5]: 25 + 20 + 30 = 75; [12.5,20]: 30; [20,30]: after the readings
    assert list(r["energy"]) == [0.0, 25.0, 75.0, 30.0, 0.0]
    assert list(r["start_idx"]) == [0, 0, 1, 3, 4]
    assert list(r["end_idx"]) == [0, 1, 3, 4, 4]
    assert r["n_clipped"] == 4
    assert r["trace_energy"] == 130.0 and r["idle_energy"] == 0.0


# ---------------------------------------------------------------------------
# library routine, exact arithmetic
# ---------------------------------------------------------------------------

def test_matches_numpy_interp():
    """numpy.interp holds the end values outside the readings, as the reading
    does; the difference of two interpolated values carries a rounding error of
    a few ulps of the counter's magnitude."""
    rng = np.random.default_rng(12)
    for n, m in [(2, 5), (7, 30), (500, 200), (5000, 3000)]:
        t, C = counter_trace(rng, n)
        delay = rng.uniform(0.0, 0.5)
        u = t - delay
        s, e = sequential_windows(rng, u[0] - 0.1, u[-1] + 0.1, m)
        reps = rng.integers(1, 1500, m).astype(np.int32)
        r = oracle.counter_attribute(t, C, s, e, delay=delay, reps=reps)
        want = (np.interp(e, u, C) - np.interp(s, u, C)) / reps
        tol = 8 * EPS * np.max(np.abs(C)) / reps + 1e-12 * np.abs(want)
        assert np.all(np.abs(r["energy"] - want) <= tol), (n, m)


def test_matches_exact_rational_arithmetic():
    """Exact C^(e) - C^(s), rounded once, against the oracle's sum of three
    rounded parts: a dropped, doubled or mis-bounded part would be off by a
    whole segment's share, far beyond the few ulps allowed."""
    rng = np.random.default_rng(13)
    for n, m in [(2, 6), (3, 10), (25, 40), (120, 60)]:
        t, C = counter_trace(rng, n, period=0.05)
        delay = 0.013
        u = t - delay
        s, e = sequential_windows(rng, u[0] - 0.07, u[-1] + 0.07, m)
        reps = rng.integers(1, 5, m).astype(np.int32)
        r = oracle.counter_attribute(t, C, s, e, delay=delay, reps=reps)
        for i in range(m):
            exact = exact_increase(u, C, s[i], e[i]) / reps[i]
            got = Fraction(r["energy"][i])
            assert abs(got - exact) <= Fraction(16 * EPS) * (abs(exact) + Fraction(C[-1] - C[0])
                                                            * Fraction(EPS)), (n, m, i)


# ---------------------------------------------------------------------------
# invariants of a cumulative quantity
# ---------------------------------------------------------------------------

def test_additive_and_telescoping():
    rng = np.random.default_rng(14)
    t, C = counter_trace(rng, 3000)
    delay = 0.21
    u = t - delay
    a, x, b = np.sort(rng.uniform(u[0], u[-1], 3))
    whole = oracle.counter_attribute(t, C, [a], [b], delay=delay)["energy"][0]
    parts = oracle.counter_attribute(t, C, [a, x], [x, b], delay=delay)["energy"]
    assert abs(parts.sum() - whole) <= 1e-12 * whole
    # windows tiling [u_0, u_{n-1}] take the whole increase; none is idle
    cuts = np.concatenate([[u[0]], np.sort(rng.uniform(u[0], u[-1], 199)), [u[-1]]])
    r = oracle.counter_attribute(t, C, cuts[:-1], cuts[1:], delay=delay)
    assert abs(r["energy"].sum() - (C[-1] - C[0])) <= 1e-12 * (C[-1] - C[0])
    assert abs(r["idle_energy"]) <= 1e-12 * (C[-1] - C[0])
    assert r["n_clipped"] == 0


def test_window_and_idle_energies_add_up_to_the_counter_increase():
    rng = np.random.default_rng(15)
    t, C = counter_trace(rng, 2000)
    u = t - 0.3
    s, e = sequential_windows(rng, u[0] - 1.0, u[-1] + 1.0, 300)
    r = oracle.counter_attribute(t, C, s, e, delay=0.3)
    assert r["trace_energy"] == C[-1] - C[0]
    assert np.all(r["energy"] >= 0.0)
    assert abs(r["attributed_energy"] + r["idle_energy"] - r["trace_energy"]) <= \
        1e-12 * r["trace_energy"]
    assert r["attributed_energy"] == pytest.approx(r["energy"].sum(), rel=1e-14)
    # no windows: everything is idle
    r0 = oracle.counter_attribute(t, C, np.zeros(0), np.zeros(0), delay=0.3)
    assert r0["idle_energy"] == C[-1] - C[0] and r0["attributed_energy"] == 0.0


def test_replays_divide_the_window_increase():
    rng = np.random.default_rng(16)
    t, C = counter_trace(rng, 500)
    s, e = sequential_windows(rng, t[0], t[-1], 50)
    one = oracle.counter_attribute(t, C, s, e)["energy"]
    reps = rng.integers(1, 100000, 50).astype(np.int32)
    many = oracle.counter_attribute(t, C, s, e, reps=reps)["energy"]
    assert np.array_equal(many, one / reps)


# ---------------------------------------------------------------------------
# input validation
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("case,code", [
    ("t_not_increasing", -5), ("t_nan", -5), ("delay_inf", -5), ("shift_collapses", -5),
    ("counter_decreases", -13), ("counter_nan", -13),
    ("start_after_end", -7), ("overlap", -7), ("zero_replays", -7), ("bound_nan", -7),
    ("one_reading", -2),
])
def test_rejects_invalid_input(case, code):
    t = np.array([0.0, 1.0, 2.0, 3.0])
    C = np.array([0.0, 1.0, 2.0, 3.0])
    s = np.array([0.5, 1.5])
    e = np.array([1.0, 2.5])
    reps = np.array([1, 1], np.int32)
    delay = 0.0
    if case == "t_not_increasing":
        t[2] = t[1]
    elif case == "t_nan":
        t[3] = np.nan
    elif case == "delay_inf":
        delay = np.inf
    elif case == "shift_collapses":
        t = np.array([0.0, 1e-300, 1.0, 2.0])
        delay = 1.0
    elif case == "counter_decreases":
        C[2] = 0.5
    elif case == "counter_nan":
        C[0] = np.nan
    elif case == "start_after_end":
        s[1] = 2.6
    elif case == "overlap":
        s[1] = 0.9
    elif case == "zero_replays":
        reps[1] = 0
    elif case == "bound_nan":
        e[0] = np.nan
    elif case == "one_reading":
        t, C = t[:1], C[:1]
    with pytest.raises(oracle.OracleError) as err:
        oracle.counter_attribute(t, C, s, e, delay=delay, reps=reps)
    assert err.value.code == code
