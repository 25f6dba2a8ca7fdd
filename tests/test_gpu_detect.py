"""Per-key latency and Section 6.1's detection on the GPU, through the C ABI,
against the oracle.

Per-key latency (the sum of interval durations) is compared within 1e-9
relative; keys, counts, flagged sets, order and verdicts bit-exact.  The
detection is run by the oracle on the same per-key tables the GPU produced, so
both take every threshold and tolerance decision on identical fp64 inputs.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import assert_energy_close, log, to_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    import paper_2512_08365_amd as mag
    mag.version()
    yield


def _np(t):
    return {k: v.cpu().numpy() for k, v in t.items()}


def _attribute(c, **kw):
    import paper_2512_08365_amd as mag
    d = to_gpu(c)
    off = [int(x) for x in c["offsets"]]
    return mag.attribute(d["t"], d["P"], d["s"], d["e"], d["key"], n_streams=len(off) - 1,
                         stream_offsets=off, latency=True, **kw)


def _check_latency(pk, c, label, reps=None):
    k = _np(pk)
    want = oracle.key_latency(c["key"], c["s"], c["e"], reps)
    assert np.array_equal(k["keys"].view(np.uint64), want["keys"]), label
    assert_energy_close(k["duration"], want["latency"], f"{label} latency")


def test_latency_tiny_and_workloads():
    for seed in range(20):
        c = synth.tiny_case(900 + seed, n=int(2 + seed * 17 % 300), streams=1 + seed % 4,
                            per_stream=int(seed % 11))
        if c["s"].shape[0] == 0:
            continue
        _, pk, _ = _attribute(c)
        _check_latency(pk, c, f"tiny seed{seed}")
    for cfg in (1, 2):
        A, _ = synth.sides(cfg, 0)
        pi, pk, _ = _attribute(A)
        _check_latency(pk, A, f"cfg{cfg}")
        # the other per-key outputs do not change with the latency pass
        import paper_2512_08365_amd as mag
        d = to_gpu(A)
        _, pk0, _ = mag.attribute(d["t"], d["P"], d["s"], d["e"], d["key"])
        for f in ("keys", "count"):
            assert np.array_equal(pk[f].cpu().numpy(), pk0[f].cpu().numpy())
        assert_energy_close(pk["sum"].cpu().numpy(), pk0["sum"].cpu().numpy(), "sums")


def test_latency_multistream_workload():
    A, _ = synth.sides(3, 0)
    log("[case] multi-stream 100M latency")
    _, pk, _ = _attribute(A)
    _check_latency(pk, A, "cfg3")


def test_latency_chunks_of_several_batches():
    # 4,500,000 intervals: each grouping chunk spans more than one batch of loads
    c = synth.long_trace(77, 9_000_000, 1, 4_500_000)
    log("[case] 4.5M intervals latency")
    _, pk, _ = _attribute(c)
    _check_latency(pk, c, "4.5M")


def test_latency_counter_mode():
    import torch
    import paper_2512_08365_amd as mag
    for seed in range(6):
        c = synth.counter_case(300 + seed, n=5000, m=900 + seed)
        d = {k: torch.from_numpy(np.ascontiguousarray(c[k], np.float64)).cuda()
             for k in ("t", "C", "s", "e")}
        key = torch.from_numpy(c["key"].view(np.int64)).cuda()
        reps = None if c["reps"] is None else torch.from_numpy(c["reps"]).cuda()
        _, pk, _ = mag.attribute_counter(d["t"], d["C"], d["s"], d["e"], key, delay=c["delay"],
                                         replays=reps, latency=True)
        _check_latency(pk, c, f"counter seed{seed}", c["reps"])


def test_latency_streamed_equals_one_shot():
    import paper_2512_08365_amd as mag
    c = synth.long_trace(78, 200_000, 3, 5000)
    d = to_gpu(c)
    off = [int(x) for x in c["offsets"]]
    _, pk1, _ = mag.attribute(d["t"], d["P"], d["s"], d["e"], d["key"], n_streams=3,
                              stream_offsets=off, latency=True)
    st = mag.Stream(200_000, d["s"], d["e"], d["key"], n_streams=3, stream_offsets=off,
                    latency=True)
    for a in range(0, 200_000, 70_001):
        st.push(d["t"][a:a + 70_001], d["P"][a:a + 70_001])
    _, pk2, _ = st.end()
    assert np.array_equal(pk1["keys"].cpu().numpy(), pk2["keys"].cpu().numpy())
    assert_energy_close(pk2["duration"].cpu().numpy(), pk1["duration"].cpu().numpy(), "streamed")


def _compare_detect(ta, tb, threshold, tolerance, rows, label):
    import paper_2512_08365_amd as mag
    got = mag.detect(ta, tb, threshold, tolerance, rows=rows)
    a = _np(ta)
    b = _np(tb)
    for t in (a, b):
        t["keys"] = t["keys"].view(np.uint64)
        t["latency"] = t["duration"]
    want = oracle.detect(a, b, threshold, tolerance)
    nf = want["n_flagged"]
    log(f"[detect] {label}: flagged {nf}, waste {want['n_waste']}, rows {rows}")
    assert got["n_flagged"] == nf and got["n_waste"] == want["n_waste"], label
    assert got["n_tradeoff"] == want["n_tradeoff"], label
    r = min(nf, rows if rows is not None else len(a["keys"]))
    g = _np({k: v for k, v in got.items() if hasattr(v, "cpu")})
    assert len(g["key"]) == r, label
    assert np.array_equal(g["key"].view(np.uint64), want["key"][:r]), label
    assert np.array_equal(g["ratio"], want["ratio"][:r]), label
    assert np.array_equal(g["verdict"], want["verdict"][:r]), label
    assert np.array_equal(g["latency_a"], want["latency_a"][:r]), label
    assert np.array_equal(g["latency_b"], want["latency_b"][:r]), label
    assert np.array_equal(g["energy_a"], want["energy_a"][:r]), label


def _device_table(keys, sums, lat):
    import torch
    return {"keys": torch.from_numpy(keys.view(np.int64)).cuda(),
            "sum": torch.from_numpy(sums).cuda(),
            "count": torch.ones(len(keys), dtype=torch.int64, device="cuda"),
            "duration": torch.from_numpy(lat).cuda()}


@pytest.mark.parametrize("K", [1, 7, 255, 256, 257, 5000, 20000])
def test_detect_synthetic_tables(K):
    rng = np.random.default_rng(K)
    keys = np.unique(rng.integers(0, 2**64, K + 50, dtype=np.uint64))[:K]
    ea = rng.uniform(0.0, 10.0, K)
    ea[rng.random(K) < 0.02] = 0.0
    eb = ea * rng.choice([0.9, 1.0, 1.05, 1.1, 1.3, 2.0], K) * rng.uniform(0.99, 1.01, K)
    la = rng.uniform(1.0, 2.0, K)
    lb = la * rng.choice([0.98, 0.99, 1.0, 1.01, 1.02], K)
    # exact boundaries: r = 0.1 and (la - lb) = 0.01 lb
    if K >= 7:
        ea[:3], eb[:3] = 10.0, 11.0
        la[:3], lb[:3] = 101.0, 100.0
    # B misses some keys of A and has keys of its own
    drop = rng.random(K) < 0.1
    kb = np.concatenate([keys[~drop], np.unique(rng.integers(0, 2**64, 20, dtype=np.uint64))])
    order = np.argsort(kb, kind="stable")
    kb, idx = np.unique(kb[order], return_index=True)
    ebb = np.concatenate([eb[~drop], rng.uniform(0, 10, 20)])[order][idx]
    lbb = np.concatenate([lb[~drop], rng.uniform(1, 2, 20)])[order][idx]
    ta = _device_table(keys, ea, la)
    tb = _device_table(kb, ebb, lbb)
    for th, rows in ((0.10, None), (0.05, None), (0.10, 3), (10.0, None)):
        _compare_detect(ta, tb, th, 0.01, rows, f"K={K} th={th} rows={rows}")


def test_detect_on_attributed_workloads():
    # the tiny A/B pair (B +15 % on three keys) and the batched sweep's candidates
    tabs = []
    for side in synth.sides(1, 0):
        _, pk, _ = _attribute(side)
        tabs.append(pk)
    _compare_detect(tabs[0], tabs[1], 0.10, 0.01, None, "cfg1")
    _compare_detect(tabs[0], tabs[1], 0.05, 0.01, None, "cfg1 5%")
    sides = synth.sides(4, 0, which=range(3))
    base = _attribute(sides[0])[1]
    for b in (1, 2):
        _compare_detect(base, _attribute(sides[b])[1], 0.10, 0.01, 100, f"cfg4 B{b}")
