"""Chunked streaming (through the C ABI): any chunking of the trace gives the
one-shot call's per-interval results bit for bit, and the oracle's within the
parity bar; a checkpoint exported after some chunks and imported into a new
stream resumes to the same result; misuse is rejected with its code."""
import numpy as np
import pytest

import synth
from gpu_util import assert_energy_close, log, run_oracle, to_gpu

pytestmark = pytest.mark.gpu

TILE = 512  # segments per tile of the library; chunk boundaries are probed around it


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    import paper_2512_08365_amd as mag
    mag.version()
    yield


def _one_shot(d, off, equal_split=True):
    import paper_2512_08365_amd as mag
    return mag.attribute(d["t"], d["P"], d["s"], d["e"], d["key"], n_streams=len(off) - 1,
                         stream_offsets=off, equal_split=equal_split)


def _streamed(d, off, sizes, equal_split=True, max_samples=None, checkpoint_after=None):
    import paper_2512_08365_amd as mag
    n = int(d["t"].shape[0])
    assert sum(sizes) == n
    mx = max_samples or n
    kw = dict(n_streams=len(off) - 1, stream_offsets=off, equal_split=equal_split)
    st = mag.Stream(mx, d["s"], d["e"], d["key"], **kw)
    pos = 0
    for i, c in enumerate(sizes):
        st.push(d["t"][pos:pos + c], d["P"][pos:pos + c])
        pos += c
        if checkpoint_after is not None and i == checkpoint_after:
            state = st.export_state()
            st.abort()
            st = mag.Stream(mx, d["s"], d["e"], d["key"], **kw)
            st.import_state(state)
    return st.end()


def _np(res):
    pi, pk, summ = res
    a = {k: v.cpu().numpy() for k, v in pi.items()}
    k = {kk: v.cpu().numpy() for kk, v in pk.items()}
    return a, k, summ


def _assert_same(a, b, label):
    ai, ak, asumm = _np(a)
    bi, bk, bsumm = _np(b)
    assert np.array_equal(ai["energy"], bi["energy"]), f"{label}: energies differ"
    assert np.array_equal(ai["start_idx"], bi["start_idx"]), label
    assert np.array_equal(ai["end_idx"], bi["end_idx"]), label
    assert np.array_equal(ak["keys"], bk["keys"]), label
    assert np.array_equal(ak["count"], bk["count"]), label
    assert_energy_close(ak["sum"], bk["sum"], f"{label}: key sums")
    W = abs(bsumm["trace_energy"])
    for f in ("trace_energy", "idle_energy", "attributed_energy"):
        assert abs(asumm[f] - bsumm[f]) <= 1e-12 * max(W, 1e-300), (label, f)
    assert asumm["n_clipped"] == bsumm["n_clipped"], label
    assert asumm["n_keys"] == bsumm["n_keys"], label


def _chunkings(n, rng):
    T = TILE
    out = [[n]]
    fixed = [1, 2, T - 1, T, T + 1, T + 2, 3 * T + 5, 1, T + 1]
    sz, left = [], n
    for c in fixed:
        if left <= 0:
            break
        c = min(c, left)
        sz.append(c)
        left -= c
    if left > 0:
        sz.append(left)
    out.append(sz)
    # tile-aligned chunks: the staged tile completes exactly at a chunk's end
    sz, left = [], n
    first = True
    while left > 0:
        c = min(T + 1 if first else T, left)
        first = False
        sz.append(c)
        left -= c
    out.append(sz)
    sz, left = [], n
    while left > 0:
        c = int(min(left, rng.integers(1, 3 * T)))
        sz.append(c)
        left -= c
    out.append(sz)
    return out


@pytest.mark.parametrize("streams,split", [(1, True), (3, True), (4, False)])
def test_any_chunking_equals_one_shot(streams, split):
    import torch
    rng = np.random.default_rng(11)
    for seed, (n, per) in enumerate([(3 * TILE + 1, 40), (20000, 300), (4 * TILE + 1, 5),
                                     (TILE + 1, 2000), (777, 30)]):
        c = synth.long_trace(100 + seed, n, streams, per)
        d = to_gpu(c)
        off = [int(x) for x in c["offsets"]]
        ref = _one_shot(d, off, split)
        for sizes in _chunkings(n, rng):
            log(f"[case] stream n={n} streams={streams} split={split} chunks={len(sizes)}")
            got = _streamed(d, off, sizes, split)
            _assert_same(got, ref, f"n={n} chunks={sizes[:6]}")
        # a larger max_samples than pushed (the trace's length is unknown up front)
        got = _streamed(d, off, _chunkings(n, rng)[1], split, max_samples=n + 5 * TILE + 3)
        _assert_same(got, ref, f"n={n} max_samples larger")
        torch.cuda.synchronize()


def test_streamed_matches_oracle():
    for seed in range(6):
        c = synth.tiny_case(900 + seed, n=int(50 + seed * 1500), streams=1 + seed % 4,
                            per_stream=40 + 10 * seed)
        d = to_gpu(c)
        off = [int(x) for x in c["offsets"]]
        n = c["t"].shape[0]
        sizes = []
        left = n
        k = 1
        while left > 0:
            sizes.append(min(left, k))
            left -= sizes[-1]
            k = k * 3 + 1
        o, g = run_oracle(c)
        gi, gk, summ = _np(_streamed(d, off, sizes))
        assert np.array_equal(gi["start_idx"], o["start_idx"]), seed
        assert np.array_equal(gi["end_idx"], o["end_idx"]), seed
        assert_energy_close(gi["energy"], o["energy"], f"seed {seed}")
        assert np.array_equal(gk["keys"].view(np.uint64), g["keys"]), seed
        assert np.array_equal(gk["count"], g["count"]), seed
        assert_energy_close(gk["sum"], g["sum"], f"seed {seed}: key sums")
        assert abs(summ["trace_energy"] - o["trace_energy"]) <= 1e-12 * o["trace_energy"]
        assert summ["n_clipped"] == o["n_clipped"]


def test_checkpoint_resume_equals_uninterrupted():
    c = synth.long_trace(5, 30000, 2, 500)
    d = to_gpu(c)
    off = [int(x) for x in c["offsets"]]
    sizes = [5000, 1, 4095, 7000, 2049, 11855]
    ref = _streamed(d, off, sizes)
    for j in range(len(sizes) - 1):
        log(f"[case] checkpoint after chunk {j}")
        got = _streamed(d, off, sizes, checkpoint_after=j)
        _assert_same(got, ref, f"resume after chunk {j}")


def test_stream_errors():
    import torch
    import paper_2512_08365_amd as mag
    from paper_2512_08365_amd import _native as N
    c = synth.long_trace(6, 10000, 1, 50)
    d = to_gpu(c)
    # more samples than max_samples
    st = mag.Stream(5000, d["s"], d["e"], d["key"])
    st.push(d["t"][:4000], d["P"][:4000])
    with pytest.raises(mag.MagnetonError) as ei:
        st.push(d["t"][4000:6000], d["P"][4000:6000])
    assert ei.value.code == N.MAG_E_SIZE
    st.abort()
    # fewer than two samples
    st = mag.Stream(5000, d["s"], d["e"], d["key"])
    st.push(d["t"][:1], d["P"][:1])
    with pytest.raises(mag.MagnetonError) as ei:
        st.end()
    assert ei.value.code == N.MAG_E_SIZE
    # timestamps that go back across a chunk boundary
    t2 = d["t"].clone()
    t2[3000] = t2[2999] - 1e-9
    st = mag.Stream(10000, d["s"], d["e"], d["key"])
    st.push(t2[:3000], d["P"][:3000])
    st.push(t2[3000:], d["P"][3000:])
    with pytest.raises(mag.MagnetonError) as ei:
        st.end()
    assert ei.value.code == N.MAG_E_TIMESTAMPS
    # a negative power sample at a chunk's first position
    P2 = d["P"].clone()
    P2[TILE * 2] = -1.0
    st = mag.Stream(10000, d["s"], d["e"], d["key"])
    st.push(d["t"][:TILE * 2], P2[:TILE * 2])
    st.push(d["t"][TILE * 2:], P2[TILE * 2:])
    with pytest.raises(mag.MagnetonError) as ei:
        st.end()
    assert ei.value.code == N.MAG_E_POWER
    # unsorted intervals are found at the end
    s2 = d["s"].clone()
    e2 = d["e"].clone()
    s2[10], s2[11] = d["s"][11], d["s"][10]
    e2[10], e2[11] = d["e"][11], d["e"][10]
    st = mag.Stream(10000, s2, e2, d["key"])
    st.push(d["t"][:5000], d["P"][:5000])
    st.push(d["t"][5000:], d["P"][5000:])
    with pytest.raises(mag.MagnetonError) as ei:
        st.end()
    assert ei.value.code == N.MAG_E_INTERVAL
    # a checkpoint imported into a stream begun with other sizes
    st = mag.Stream(10000, d["s"], d["e"], d["key"])
    st.push(d["t"][:3000], d["P"][:3000])
    state = st.export_state()
    st.abort()
    other = mag.Stream(12000, d["s"], d["e"], d["key"])
    with pytest.raises(mag.MagnetonError) as ei:
        other.import_state(state)
    assert ei.value.code == N.MAG_E_STATE
    other.abort()
    # a truncated checkpoint
    st = mag.Stream(10000, d["s"], d["e"], d["key"])
    with pytest.raises(mag.MagnetonError) as ei:
        st.import_state(state[:-8])
    assert ei.value.code == N.MAG_E_SIZE
    st.abort()
    torch.cuda.synchronize()


@pytest.mark.slow
def test_long_run_workload_both_sides_streamed_in_32M_chunks():
    """The hour-long workload (360,000,000 samples at 100 kHz, 50,000,000
    sequential intervals, 20,000 Zipf(1.05) keys), both sides drawn with
    independent seeds.  Side A is pushed from device memory and side B from
    pinned host memory (double-buffered copies on a copy stream), both in
    32,000,000-sample chunks; side A also equals the one-shot call bit for bit.
    Every one of the 50,000,000 energies and sample indices of each side is
    compared with the oracle run on the whole, unchunked trace, the per-key
    rows with the oracle's grouping of the oracle's energies, and the top-100
    diff with the oracle's."""
    import torch
    import oracle
    import oracle_par
    sides = synth.sides(5, 0)
    tables, otables = [], []
    for si, c in enumerate(sides):
        label = "AB"[si]
        n = c["t"].shape[0]
        m = c["s"].shape[0]
        log(f"[case] long-run side {label} n={n} m={m}")
        sizes = [32_000_000] * (n // 32_000_000)
        if n % 32_000_000:
            sizes.append(n % 32_000_000)
        off = [int(x) for x in c["offsets"]]
        if si == 0:
            d = to_gpu(c)
            ref = _one_shot(d, off)
            got = _streamed(d, off, sizes)
            _assert_same(got, ref, "long-run A one-shot vs chunked")
            del ref
        else:
            d = {"s": torch.from_numpy(c["s"]).cuda(), "e": torch.from_numpy(c["e"]).cuda(),
                 "key": torch.from_numpy(c["key"].view(np.int64)).cuda()}
            got = _streamed_host(c, d, off, sizes)
        gi, gk, summ = _np(got)
        tables.append(got[1])
        del d
        torch.cuda.empty_cache()
        log(f"[oracle] long-run side {label}: whole trace, {oracle_par.workers()} interval slices")
        r = oracle_par.attribute_one_stream(c["t"], c["P"], c["s"], c["e"])
        assert np.array_equal(gi["start_idx"], r["start_idx"]), f"{label}: start_idx"
        assert np.array_equal(gi["end_idx"], r["end_idx"]), f"{label}: end_idx"
        assert_energy_close(gi["energy"], r["energy"], f"long-run {label}: energies")
        W = r["trace_energy"]
        assert abs(summ["trace_energy"] - W) <= 1e-12 * W
        assert abs(summ["attributed_energy"] - r["attributed_energy"]) <= 1e-9 * W
        assert abs(summ["idle_energy"] - r["idle_energy"]) <= 1e-9 * W
        assert summ["n_clipped"] == r["n_clipped"]
        g = oracle_par.groupby(c["key"], r["energy"])
        otables.append(g)
        assert np.array_equal(gk["keys"].view(np.uint64), g["keys"]), f"{label}: keys"
        assert np.array_equal(gk["count"], g["count"]), f"{label}: counts"
        assert_energy_close(gk["sum"], g["sum"], f"long-run {label}: key sums")
        second = g["m2"] + g["sum"] ** 2 / np.maximum(g["count"], 1)
        assert np.all(np.abs(gk["m2"] - g["m2"]) <= 1e-9 * second), f"{label}: m2"
        del got, gi, r
    import paper_2512_08365_amd as mag
    d = mag.diff(tables[0], tables[1], 100)
    o = oracle.diff(otables[0], otables[1], 100)
    log(f"[diff] long-run: joined={o['n_join']} margin={o['margin']:.3g}")
    assert o["margin"] > 1e-8, "near-tied ratios in the long-run workload"
    assert np.array_equal(d["key"].cpu().numpy().view(np.uint64), o["key"])
    r_ = d["ratio"].cpu().numpy()
    assert np.all(np.abs(r_ - o["ratio"]) <= 3e-9 * (1 + np.abs(o["ratio"])))
    assert np.array_equal(d["count_a"].cpu().numpy(), o["count_a"])
    assert np.array_equal(d["count_b"].cpu().numpy(), o["count_b"])
    assert (d["n_only_a"], d["n_only_b"], d["n_join"]) == (o["n_only_a"], o["n_only_b"], o["n_join"])


def _streamed_host(c, d, off, sizes):
    """Chunks pushed from pinned host memory through the library's copy stream."""
    import torch
    import paper_2512_08365_amd as mag
    n = c["t"].shape[0]
    t_h = torch.from_numpy(c["t"]).pin_memory()
    P_h = torch.from_numpy(c["P"]).pin_memory()
    st = mag.Stream(n, d["s"], d["e"], d["key"], n_streams=len(off) - 1, stream_offsets=off,
                    host_chunk=max(sizes))
    pos = 0
    for k in sizes:
        st.push_host(t_h[pos:pos + k], P_h[pos:pos + k])
        pos += k
    return st.end()
