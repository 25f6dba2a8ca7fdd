"""Parity of the counter (software replay) attribution, through the C ABI,
with the CPU oracle.

Sample indices, key grouping and counts are bit-exact; window energies within
1e-9 relative; the summary's totals within 1e-12 of the counter's whole
increase.  Cases span many 64-window chunks and 256-reading blocks with ragged
tails, windows that reach past the readings, bounds exactly on shifted reading
times, zero-length windows, flat counter stretches, delays of either sign,
irregular reading spacing (the chunk-boundary search's fallback), and every
device-detected input error.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import assert_energy_close, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    import paper_2512_08365_amd as mag
    mag.version()
    yield


def _dev(c):
    import torch
    d = {k: torch.from_numpy(np.ascontiguousarray(c[k], np.float64)).cuda()
         for k in ("t", "C", "s", "e")}
    d["key"] = torch.from_numpy(np.ascontiguousarray(c["key"], np.uint64).view(np.int64)).cuda()
    d["reps"] = None if c["reps"] is None else torch.from_numpy(
        np.ascontiguousarray(c["reps"], np.int32)).cuda()
    return d


def compare(c, label, group=True, validate=True):
    import paper_2512_08365_amd as mag
    log(f"[counter] {label}: n={len(c['t'])} m={len(c['s'])} delay={c['delay']}")
    d = _dev(c)
    pi, pk, summ = mag.attribute_counter(d["t"], d["C"], d["s"], d["e"],
                                         d["key"] if group else None, delay=c["delay"],
                                         replays=d["reps"], validate=validate)
    ref = oracle.counter_attribute(c["t"], c["C"], c["s"], c["e"], delay=c["delay"],
                                   reps=c["reps"])
    assert np.array_equal(pi["start_idx"].cpu().numpy(), ref["start_idx"]), label
    assert np.array_equal(pi["end_idx"].cpu().numpy(), ref["end_idx"]), label
    assert_energy_close(pi["energy"].cpu().numpy(), ref["energy"], f"{label} energy")
    scale = abs(ref["trace_energy"]) + 1e-300
    assert summ["trace_energy"] == ref["trace_energy"], label
    assert abs(summ["idle_energy"] - ref["idle_energy"]) <= 1e-12 * scale, label
    assert abs(summ["attributed_energy"] - ref["attributed_energy"]) <= \
        1e-12 * scale + 1e-9 * abs(ref["attributed_energy"]), label
    assert summ["n_clipped"] == ref["n_clipped"], label
    if group and len(c["s"]):
        g = oracle.groupby(c["key"], ref["energy"])
        assert np.array_equal(pk["keys"].cpu().numpy().view(np.uint64), g["keys"]), label
        assert np.array_equal(pk["count"].cpu().numpy(), g["count"]), label
        assert_energy_close(pk["sum"].cpu().numpy(), g["sum"], f"{label} key sums")
        second = g["m2"] + g["sum"] ** 2 / np.maximum(g["count"], 1)
        assert np.all(np.abs(pk["m2"].cpu().numpy() - g["m2"]) <= 1e-9 * second), label
    return pi, pk, summ


def test_tiny_fuzz():
    for seed in range(60):
        n = 2 + (seed * 53) % 400
        m = (seed * 29) % 150
        c = synth.counter_case(7000 + seed, n=n, m=m, replays=bool(seed % 3),
                               outside=bool(seed % 4), zero_len=0.1 * (seed % 2))
        compare(c, f"tiny seed{seed}", group=bool(seed % 5))


@pytest.mark.parametrize("n,m", [(2, 0), (2, 1), (3, 64), (257, 64), (256, 65), (5000, 63),
                                 (20000, 129), (300, 5000), (70000, 6400)])
def test_chunk_and_block_edges(n, m):
    c = synth.counter_case(n * 31 + m, n=n, m=m)
    compare(c, f"edges n={n} m={m}")


def test_dense_windows_in_one_segment():
    # many windows between two readings: every endpoint in the same segment
    c = synth.counter_case(11, n=40, m=3000, outside=False, snap=0.0)
    compare(c, "dense")


def test_sparse_windows_over_long_readings():
    # few windows, each chunk streams tens of thousands of readings
    c = synth.counter_case(12, n=200_000, m=150, period=0.001)
    compare(c, "sparse")


def test_irregular_reading_spacing():
    for seed in range(4):
        c = synth.counter_case(13 + seed, n=50_000, m=4000, irregular=True)
        compare(c, f"irregular seed{seed}")


@pytest.mark.parametrize("delay", [0.0, 0.25, -0.07, 1e6])
def test_delays(delay):
    c = synth.counter_case(21, n=3000, m=700, delay=delay)
    compare(c, f"delay {delay}")


def test_replay_session_full_size():
    c = synth.replay_session(0)
    pi, pk, summ = compare(c, "replay session")
    assert summ["n_keys"] == len(np.unique(c["key"]))


def test_skip_validate_gives_the_same_result():
    c = synth.counter_case(31, n=5000, m=900)
    a = compare(c, "validated")
    b = compare(c, "unvalidated", validate=False)
    assert np.array_equal(a[0]["energy"].cpu().numpy(), b[0]["energy"].cpu().numpy())


@pytest.mark.parametrize("case,code", [
    ("t_not_increasing", -5), ("t_nan", -5), ("shift_collapses", -5), ("delay_inf", -5),
    ("counter_decreases", -13), ("counter_nan", -13),
    ("start_after_end", -7), ("overlap", -7), ("zero_replays", -7), ("bound_nan", -7),
])
def test_device_detected_errors(case, code):
    import torch
    import paper_2512_08365_amd as mag
    rng = np.random.default_rng(5)
    c = synth.counter_case(41, n=3000, m=400, delay=0.0, zero_len=0.0)
    t, C, s, e, reps = (c["t"].copy(), c["C"].copy(), c["s"].copy(), c["e"].copy(),
                        c["reps"].copy())
    delay = 0.0
    j = int(rng.integers(1, 2999))
    i = int(rng.integers(1, 399))
    if case == "t_not_increasing":
        t[j] = t[j - 1]
    elif case == "t_nan":
        t[j] = np.nan
    elif case == "shift_collapses":
        t = np.arange(3000, dtype=np.float64) * 1e-300
        delay = 1.0
    elif case == "delay_inf":
        delay = np.inf
    elif case == "counter_decreases":
        C[j] = C[j - 1] - 1.0
    elif case == "counter_nan":
        C[j] = np.nan
    elif case == "start_after_end":
        s[i] = e[i] + 1e-9
        e[i - 1] = min(e[i - 1], s[i])
    elif case == "overlap":
        s[i] = e[i - 1] - 1e-6
    elif case == "zero_replays":
        reps[i] = 0
    elif case == "bound_nan":
        e[i] = np.nan
    with pytest.raises(oracle.OracleError) as want:
        oracle.counter_attribute(t, C, s, e, delay=delay, reps=reps)
    assert want.value.code == code
    d = {k: torch.from_numpy(v).cuda() for k, v in (("t", t), ("C", C), ("s", s), ("e", e))}
    with pytest.raises(mag.MagnetonError) as got:
        mag.attribute_counter(d["t"], d["C"], d["s"], d["e"], delay=delay,
                              replays=torch.from_numpy(reps).cuda())
    assert got.value.code == code, case


def test_asynchronous_and_timed_calls_equal_the_synchronous_one():
    import paper_2512_08365_amd as mag
    c = synth.counter_case(51, n=20000, m=3000)
    d = _dev(c)
    args = (d["t"], d["C"], d["s"], d["e"], d["key"])
    kw = dict(delay=c["delay"], replays=d["reps"], latency=True)
    ref = mag.attribute_counter(*args, **kw)
    pend = mag.attribute_counter(*args, asynchronous=True, time_kernels=True, **kw)
    got = pend.finish()
    for k in ("energy", "start_idx", "end_idx"):
        assert np.array_equal(got[0][k].cpu().numpy(), ref[0][k].cpu().numpy()), k
    for k in ("keys", "count"):
        assert np.array_equal(got[1][k].cpu().numpy(), ref[1][k].cpu().numpy()), k
    assert_energy_close(got[1]["duration"].cpu().numpy(), ref[1]["duration"].cpu().numpy(),
                        "latency")
    assert got[2]["n_clipped"] == ref[2]["n_clipped"]
    assert got[2]["kernel_ms"] > 0.0 and got[2]["device_ms"] >= got[2]["kernel_ms"]
