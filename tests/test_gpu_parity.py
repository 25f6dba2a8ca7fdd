"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Integer outputs (sample indices, key grouping, counts, top-k order) must be
bit-exact; energies within 1e-9 relative; M2 within 1e-9 of the key's second
moment (sum of E^2).  Sizes span many tiles, ragged tails, endpoint rounds and
the degenerate cases of the method.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import (assert_energy_close, compare_attribution, log, run_gpu, run_oracle,
                      to_gpu)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    import paper_2512_08365_amd as mag
    mag.version()  # loads the HIP library or raises
    yield


# ---------------------------------------------------------------------------
# small randomized cases
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("streams", [1, 2, 3, 4, 7, 12, 20])
def test_tiny_fuzz(streams):
    for seed in range(25):
        c = synth.tiny_case(5000 * streams + seed, n=int(2 + (seed * 37) % 300), streams=streams,
                            per_stream=int(seed % 13))
        for split in (True, False):
            compare_attribution(c, equal_split=split, label=f"tiny s{streams} seed{seed}")


def test_endpoints_shared_by_streams():
    """Streams with identical endpoints (exact ties across streams, many in one
    segment), on a dyadic grid, against the oracle: energies do not depend on
    how equal times are ordered, indices and keys are exact."""
    for streams, per in ((3, 40), (9, 12), (24, 6)):
        base = synth.tiny_case(900 + streams, n=120, streams=1, per_stream=per, dyadic=True)
        m = base["s"].shape[0]
        c = {"t": base["t"], "P": base["P"], "s": np.tile(base["s"], streams),
             "e": np.tile(base["e"], streams), "key": np.tile(base["key"], streams),
             "offsets": np.arange(streams + 1, dtype=np.int64) * m}
        for split in (True, False):
            compare_attribution(c, equal_split=split, label=f"shared s{streams}")


def test_dyadic_bit_exact():
    for seed in range(10):
        c = synth.tiny_case(77 + seed, n=200, streams=2, per_stream=20, dyadic=True)
        o, g = run_oracle(c)
        gi, gk, summ, _ = run_gpu(c)
        assert np.array_equal(gi["energy"], o["energy"]), seed


@pytest.mark.parametrize("streams", [1, 4])
def test_intervals_spanning_many_tiles(streams):
    for seed, (n, per) in enumerate([(20000, 3), (50001, 40), (100000, 400), (4097, 2000)]):
        c = synth.long_trace(seed, n, streams, per)
        compare_attribution(c, label=f"long s{streams} n{n} per{per}")


def test_dense_endpoints_force_rounds():
    # thousands of endpoints inside one tile (and inside single segments)
    rng = np.random.default_rng(3)
    n = 5000
    t = np.arange(n, dtype=np.float64) * 1e-3
    P = rng.uniform(100, 500, n).astype(np.float32)
    for streams in (1, 3, 32):
        s_all, e_all, off = [], [], [0]
        for a in range(streams):
            per = 3000 // streams
            cuts = np.sort(rng.uniform(1.0, 1.3, 2 * per))   # ~300 samples, 6000 endpoints
            s_all.append(cuts[0::2])
            e_all.append(cuts[1::2])
            off.append(off[-1] + per)
        c = {"t": t, "P": P, "s": np.concatenate(s_all), "e": np.concatenate(e_all),
             "key": rng.integers(0, 9, off[-1]).astype(np.uint64), "offsets": np.array(off)}
        compare_attribution(c, label=f"dense s{streams}")
    # all endpoints inside one sample segment
    cuts = np.sort(rng.uniform(2.0001, 2.0009, 4000))
    c = {"t": t, "P": P, "s": cuts[0::2], "e": cuts[1::2], "key": np.zeros(2000, np.uint64),
         "offsets": np.array([0, 2000])}
    compare_attribution(c, label="one segment")


def test_tiny_energies_behind_a_large_tile_prefix():
    # 1 MW for the first samples of every tile, then 1 mW: an interval over
    # whole low-power segments holds ~1e-11 of the tile's prefix energy, far
    # below what a difference of two tile-local prefixes resolves to 1e-9, so
    # the whole segments must be summed directly.  Several streams overlap
    # (equal split), some intervals span tiles, some sit inside one segment.
    rng = np.random.default_rng(11)
    n = 4 * 512 + 37
    t = np.arange(n, dtype=np.float64) * 1e-3
    P = np.where((np.arange(n) % 512) < 300, 1.0e6, 1.0e-3).astype(np.float32)
    P[::97] = 0.0
    for streams in (1, 3):
        s_all, e_all, off = [], [], [0]
        for a in range(streams):
            cuts = np.sort(rng.uniform(0.0, t[-1], 2 * 40))
            s_all.append(cuts[0::2])
            e_all.append(cuts[1::2])
            off.append(off[-1] + 40)
        # intervals wholly inside the low-power stretch of tile 1, over whole segments
        lo = (512 + 310) * 1e-3
        extra_s = lo + np.arange(5) * 0.02 + 0.0003
        extra_e = extra_s + np.array([0.0021, 0.005, 0.0107, 0.0004, 0.0015])
        s_all.append(extra_s)
        e_all.append(extra_e)
        off.append(off[-1] + 5)
        c = {"t": t, "P": P, "s": np.concatenate(s_all), "e": np.concatenate(e_all),
             "key": rng.integers(0, 7, off[-1]).astype(np.uint64), "offsets": np.array(off)}
        for split in (True, False):
            compare_attribution(c, equal_split=split, label=f"tiny energies s{streams + 1}")


def test_degenerate_cases():
    t = np.array([0.0, 1.0])
    P = np.array([3.0, 5.0], np.float32)
    cases = {
        "two samples": (np.array([0.25]), np.array([0.75])),
        "no intervals": (np.zeros(0), np.zeros(0)),
        "zero length": (np.array([0.5, 0.5]), np.array([0.5, 0.7])),
        "all before": (np.array([-3.0, -2.0]), np.array([-2.5, -1.0])),
        "all after": (np.array([2.0, 3.0]), np.array([2.5, 4.0])),
        "covers trace": (np.array([-1.0]), np.array([5.0])),
        "on samples": (np.array([0.0]), np.array([1.0])),
    }
    for name, (s, e) in cases.items():
        c = {"t": t, "P": P, "s": s, "e": e, "key": np.arange(s.shape[0]).astype(np.uint64),
             "offsets": np.array([0, s.shape[0]])}
        compare_attribution(c, label=name)


def test_extreme_keys():
    c = synth.tiny_case(5, n=500, streams=2, per_stream=60)
    m = c["s"].shape[0]
    c["key"] = np.array([0, 2**64 - 1, 2**63, 1, 2**64 - 2] * m, np.uint64)[:m]
    compare_attribution(c, label="extreme keys")


@pytest.mark.parametrize("vocab", [1000, 9000])
def test_keys_first_seen_after_the_insertion_prefix(vocab):
    # more intervals than the key-insertion prefix; some keys, the all-ones key
    # among them, occur only in the tail; a vocabulary that fits the LDS
    # dictionary of the lookup pass and one that does not
    c = synth.long_trace(11, 400000, 2, 160000, outside=False)
    m = c["s"].shape[0]
    rng = np.random.default_rng(vocab)
    key = rng.integers(0, vocab, m).astype(np.uint64) * np.uint64(0x9E3779B97F4A7C15)
    tail = np.arange(m) >= m - 20000
    key[tail] = (rng.integers(0, 300, int(tail.sum())) + 10**6).astype(np.uint64)
    key[m - 5] = np.uint64(2**64 - 1)
    c["key"] = key
    compare_attribution(c, label=f"late keys vocab{vocab}")


def test_rows_not_16_byte_aligned():
    # timestamps and power one element into their allocations: 8- and 4-byte
    # aligned, so the tile kernel reads them without vector loads
    import torch
    c = synth.long_trace(21, 70001, 3, 900)
    d = to_gpu(c)
    for name, dt in (("t", torch.float64), ("P", torch.float32)):
        buf = torch.empty(d[name].numel() + 1, dtype=dt, device=d[name].device)
        buf[1:].copy_(d[name])
        d[name] = buf[1:]
        assert d[name].data_ptr() % 16 != 0
    o, g = run_oracle(c)
    gi, gk, _, _ = run_gpu(c, dev=d)
    assert np.array_equal(gi["start_idx"], o["start_idx"])
    assert np.array_equal(gi["end_idx"], o["end_idx"])
    assert_energy_close(gi["energy"], o["energy"], "unaligned rows")
    assert np.array_equal(gk["count"], g["count"])


def test_key_capacity_error():
    import paper_2512_08365_amd as mag
    c = synth.tiny_case(6, n=300, streams=1, per_stream=40, keys=30)
    nkeys = np.unique(c["key"]).shape[0]
    d = to_gpu(c)
    with pytest.raises(mag.MagnetonError) as ei:
        mag.attribute(d["t"], d["P"], d["s"], d["e"], d["key"], key_capacity=max(1, nkeys - 1))
    assert ei.value.code == -3


def test_device_detected_errors():
    import paper_2512_08365_amd as mag
    import torch
    base = synth.tiny_case(8, n=5000, streams=2, per_stream=50)

    def run(c, off=None):
        d = to_gpu(c)
        off = off or [int(x) for x in c["offsets"]]
        mag.attribute(d["t"], d["P"], d["s"], d["e"], d["key"], n_streams=len(off) - 1,
                      stream_offsets=off)

    bads = []
    c = dict(base); c["t"] = base["t"].copy(); c["t"][3000] = c["t"][2999]; bads.append((c, -5))
    c = dict(base); c["t"] = base["t"].copy(); c["t"][4999] = np.nan; bads.append((c, -5))
    c = dict(base); c["P"] = base["P"].copy(); c["P"][1234] = -1.0; bads.append((c, -6))
    c = dict(base); c["P"] = base["P"].copy(); c["P"][0] = np.inf; bads.append((c, -6))
    c = dict(base); c["s"] = base["s"].copy(); c["s"][10] = c["e"][10] + 1.0; bads.append((c, -7))
    a = int(np.argmax(np.diff(base["offsets"]) >= 2))
    i = int(base["offsets"][a])
    c = dict(base); c["e"] = base["e"].copy(); c["e"][i] = c["s"][i + 1] + 1e-3; bads.append((c, -7))
    c = dict(base); c["s"] = base["s"].copy(); c["s"][0] = np.nan; bads.append((c, -7))
    for i, (c, code) in enumerate(bads):
        log(f"[case] invalid input {i} expects {code}")
        with pytest.raises(mag.MagnetonError) as ei:
            run(c)
        assert ei.value.code == code, i
    # host-detected: bad offsets
    with pytest.raises(mag.MagnetonError) as ei:
        run(base, off=[0, 5, 3, int(base["offsets"][-1])])
    assert ei.value.code == -8
    torch.cuda.synchronize()


def test_asynchronous_pair_equals_synchronous():
    # both sides enqueued back to back, finished afterwards: the same results
    import paper_2512_08365_amd as mag
    A, B = synth.sides(1, 1)
    ref = []
    for c in (A, B):
        gi, gk, summ, _ = run_gpu(c)
        ref.append((gi, gk, summ))
    pend = []
    for c in (A, B):
        d = to_gpu(c)
        off = [int(x) for x in c["offsets"]]
        pend.append(mag.attribute(d["t"], d["P"], d["s"], d["e"], d["key"], n_streams=len(off) - 1,
                                  stream_offsets=off, asynchronous=True))
    for (gi, gk, summ), p in zip(ref, pend):
        pi, pk, ps = p.finish()
        for k in gi:
            assert np.array_equal(pi[k].cpu().numpy(), gi[k]), k
        assert np.array_equal(pk["keys"].cpu().numpy().view(np.uint64), gk["keys"])
        assert np.array_equal(pk["count"].cpu().numpy(), gk["count"])
        assert_energy_close(pk["sum"].cpu().numpy(), gk["sum"], "async key sums")
        assert ps["n_keys"] == summ["n_keys"] and ps["n_clipped"] == summ["n_clipped"]
        assert abs(ps["trace_energy"] - summ["trace_energy"]) <= 1e-12 * summ["trace_energy"]
    # a device-detected error is reported by finish()
    c = synth.tiny_case(8, n=5000, streams=2, per_stream=50)
    c["P"] = c["P"].copy()
    c["P"][77] = -1.0
    d = to_gpu(c)
    off = [int(x) for x in c["offsets"]]
    p = mag.attribute(d["t"], d["P"], d["s"], d["e"], d["key"], n_streams=len(off) - 1,
                      stream_offsets=off, asynchronous=True)
    with pytest.raises(mag.MagnetonError) as ei:
        p.finish()
    assert ei.value.code == -6


def test_deterministic_per_interval():
    c = synth.long_trace(9, 60000, 4, 3000)
    a, ka, _, _ = run_gpu(c)
    b, kb, _, _ = run_gpu(c)
    for k in a:
        assert np.array_equal(a[k], b[k]), k
    assert np.array_equal(ka["keys"], kb["keys"])
    assert np.array_equal(ka["count"], kb["count"])


# ---------------------------------------------------------------------------
# the workloads
# ---------------------------------------------------------------------------

def _diff_and_compare(ga_dev, gb_dev, ga, gb, k, label):
    import paper_2512_08365_amd as mag
    d = mag.diff(ga_dev, gb_dev, k)
    o = oracle.diff(ga, gb, k)
    log(f"[diff] {label}: k={k} joined={o['n_join']} margin={o['margin']:.3g}")
    # the order is only well defined when adjacent ratios are separated by more
    # than the ratios' own error (sums to 1e-9 relative move r by ~2e-9 (1 + |r|))
    assert o["margin"] > 1e-8, f"{label}: workload has near-tied ratios"
    key = d["key"].cpu().numpy().view(np.uint64)
    assert np.array_equal(key, o["key"]), f"{label}: top-k keys/order"
    r = d["ratio"].cpu().numpy()
    assert np.all(np.abs(r - o["ratio"]) <= 3e-9 * (1 + np.abs(o["ratio"]))), label
    assert np.array_equal(d["count_a"].cpu().numpy(), o["count_a"]), label
    assert np.array_equal(d["count_b"].cpu().numpy(), o["count_b"]), label
    assert_energy_close(d["energy_a"].cpu().numpy(), o["energy_a"], label)
    assert_energy_close(d["energy_b"].cpu().numpy(), o["energy_b"], label)
    assert (d["n_only_a"], d["n_only_b"], d["n_join"]) == (o["n_only_a"], o["n_only_b"], o["n_join"])


@pytest.mark.parametrize("cfg,k", [(1, 10), (2, 10)])
def test_workload_ab(cfg, k):
    for seed in range(3):
        A, B = synth.sides(cfg, seed)
        ra = compare_attribution(A, label=f"cfg{cfg} A seed{seed}")
        rb = compare_attribution(B, label=f"cfg{cfg} B seed{seed}")
        _diff_and_compare(ra[5], rb[5], ra[1], rb[1], k, f"cfg{cfg} seed{seed}")


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_workload_multistream_100m(seed):
    A, B = synth.sides(3, seed)
    ra = compare_attribution(A, label=f"cfg3 A seed{seed}")
    rb = compare_attribution(B, label=f"cfg3 B seed{seed}")
    _diff_and_compare(ra[5], rb[5], ra[1], rb[1], 100, f"cfg3 seed{seed}")


def test_workload_batched_sweep():
    """Baseline A against all eight candidates B1..B8: each candidate's
    attribution against the oracle, each pair's top-100 by mag_diff, and the
    eight rankings of one mag_diff_batch call against the oracle's."""
    import paper_2512_08365_amd as mag
    sides = synth.sides(4, 0)
    assert len(sides) == 9
    base = compare_attribution(sides[0], label="cfg4 A")
    dev_tabs, orc_tabs = [], []
    for b in range(1, len(sides)):
        rb = compare_attribution(sides[b], label=f"cfg4 B{b}")
        _diff_and_compare(base[5], rb[5], base[1], rb[1], 100, f"cfg4 B{b}")
        dev_tabs.append(rb[5])
        orc_tabs.append(rb[1])
    got = mag.diff_batch(base[5], dev_tabs, 100)
    assert len(got) == 8
    for b, (d, og) in enumerate(zip(got, orc_tabs), start=1):
        o = oracle.diff(base[1], og, 100)
        label = f"cfg4 batch B{b}"
        assert np.array_equal(d["key"].cpu().numpy().view(np.uint64), o["key"]), label
        r = d["ratio"].cpu().numpy()
        assert np.all(np.abs(r - o["ratio"]) <= 3e-9 * (1 + np.abs(o["ratio"]))), label
        assert np.array_equal(d["count_a"].cpu().numpy(), o["count_a"]), label
        assert np.array_equal(d["count_b"].cpu().numpy(), o["count_b"]), label
        assert_energy_close(d["energy_a"].cpu().numpy(), o["energy_a"], label)
        assert_energy_close(d["energy_b"].cpu().numpy(), o["energy_b"], label)
        assert (d["n_only_a"], d["n_only_b"], d["n_join"]) == (o["n_only_a"], o["n_only_b"],
                                                               o["n_join"]), label


def test_diff_batch_matches_single_diffs():
    """mag_diff_batch over more than one launch group (19 candidates), with
    tables of different sizes, empty tables, k above the join and k = 0,
    equals mag_diff candidate by candidate."""
    import torch
    import paper_2512_08365_amd as mag
    rng = np.random.default_rng(11)

    def table(n, vocab):
        keys = np.sort(rng.choice(vocab, size=n, replace=False)).astype(np.uint64)
        sums = rng.uniform(0.0, 10.0, n)
        sums[rng.random(n) < 0.05] = 0.0
        cnt = rng.integers(1, 50, n)
        return {"keys": torch.from_numpy(keys.view(np.int64)).cuda(),
                "sum": torch.from_numpy(sums).cuda(), "count": torch.from_numpy(cnt).cuda()}

    vocab = np.unique(rng.integers(0, 2**63, 20000, dtype=np.int64).astype(np.uint64)
                      | np.uint64(1 << 63))
    a = table(3000, vocab)
    bs = [table(int(n), vocab) for n in rng.integers(0, 6000, 17)] + [table(0, vocab),
                                                                      table(1, vocab)]
    for k in (0, 1, 37, 5000):
        got = mag.diff_batch(a, bs, k)
        for c, b in enumerate(bs):
            want = mag.diff(a, b, k)
            for f in ("key", "ratio", "energy_a", "energy_b", "count_a", "count_b"):
                assert torch.equal(got[c][f], want[f]), (k, c, f)
            for f in ("n_only_a", "n_only_b", "n_join"):
                assert got[c][f] == want[f], (k, c, f)
    assert mag.diff_batch(a, [], 10) == []
