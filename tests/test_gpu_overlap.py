"""Two attributions overlapped on two HIP streams through the intervals_ready
event: the second system's attribution starts once the first's per-interval
outputs are complete (the comparison of two systems, Section 3.2).  Results
equal those of the two calls run one after the other, and a consumer on the
second stream that waits for the event sees the first side's final energies.
"""
import numpy as np
import pytest

import synth
from gpu_util import log, to_gpu

pytestmark = pytest.mark.gpu


def test_overlapped_sides_match_serial_and_event_orders_the_outputs():
    import torch
    import paper_2512_08365_amd as mag
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    cases = [synth.long_trace(seed, 300_000, 4, 20_000) for seed in (71, 72)]
    devs = [to_gpu(c) for c in cases]

    def run(d, c, **kw):
        off = [int(x) for x in c["offsets"]]
        return mag.attribute(d["t"], d["P"], d["s"], d["e"], d["key"], n_streams=len(off) - 1,
                             stream_offsets=off, **kw)

    serial = [run(d, c) for d, c in zip(devs, cases)]
    torch.cuda.synchronize()
    s2 = torch.cuda.Stream()
    ready = torch.cuda.Event()
    for rep in range(3):
        log(f"[overlap] repetition {rep}")
        out_a = {"energy": torch.full((cases[0]["s"].shape[0],), float("nan"),
                                      dtype=torch.float64, device="cuda")}
        pend_a = run(devs[0], cases[0], asynchronous=True, intervals_ready=ready, out=out_a)
        s2.wait_event(ready)
        with torch.cuda.stream(s2):
            seen = out_a["energy"].clone()  # ordered after A's per-interval outputs
            pend_b = run(devs[1], cases[1], asynchronous=True)
        res_a = pend_a.finish()
        with torch.cuda.stream(s2):
            res_b = pend_b.finish()
        torch.cuda.synchronize()
        for got, want in ((res_a, serial[0]), (res_b, serial[1])):
            for k in ("energy", "start_idx", "end_idx"):
                assert torch.equal(got[0][k], want[0][k]), k
            for k in ("keys", "count"):
                assert torch.equal(got[1][k], want[1][k]), k
            np.testing.assert_allclose(got[1]["sum"].cpu().numpy(), want[1]["sum"].cpu().numpy(),
                                       rtol=1e-12)
            assert got[2]["n_clipped"] == want[2]["n_clipped"]
        assert torch.equal(seen, serial[0][0]["energy"])


def test_diff_enqueued_before_the_attributions_finish():
    """Key counts left on the device (n_keys_device, n_keys = -1 for the diff):
    A on one stream, B on another from A's intervals_ready event, the diff and
    the detection enqueued right after without a host wait, against the same
    calls made one after the other with host counts."""
    import ctypes
    import torch
    import paper_2512_08365_amd as mag
    from paper_2512_08365_amd import _native as N
    lib = N.load()
    A, B = synth.sides(1, 0)
    cap, k = 64, 10

    class Side:
        def __init__(self, c, ready=None):
            self.d = to_gpu(c)
            self.m = int(c["s"].shape[0])
            self.n = int(c["t"].shape[0])
            self.tab = {"keys": torch.empty(cap, dtype=torch.int64, device="cuda"),
                        "sum": torch.empty(cap, dtype=torch.float64, device="cuda"),
                        "m2": torch.empty(cap, dtype=torch.float64, device="cuda"),
                        "count": torch.empty(cap, dtype=torch.int64, device="cuda"),
                        "duration": torch.empty(cap, dtype=torch.float64, device="cuda")}
            self.nk = torch.full((1,), -7, dtype=torch.int64, device="cuda")
            t = self.tab
            self.ks = N.KeyStats(t["sum"].data_ptr(), t["m2"].data_ptr(), t["count"].data_ptr(),
                                 cap, 0, t["duration"].data_ptr(), self.nk.data_ptr())
            # the diff's view: count on the device
            self.kd = N.KeyStats(t["sum"].data_ptr(), t["m2"].data_ptr(), t["count"].data_ptr(),
                                 cap, -1, t["duration"].data_ptr(), self.nk.data_ptr())
            self.opts = N.AttrOpts(1, N.MAG_EQUAL_SPLIT | N.MAG_ASYNC | N.MAG_KEY_LATENCY, None,
                                   ready)
            b = ctypes.c_size_t(0)
            assert lib.mag_attribute_workspace_size(self.n, self.m, cap, ctypes.byref(self.opts),
                                                    ctypes.byref(b)) == 0
            self.ws = torch.empty(int(b.value), dtype=torch.uint8, device="cuda")
            self.summ = N.Summary()

        def attribute(self, stream):
            d = self.d
            assert lib.mag_attribute(d["t"].data_ptr(), d["P"].data_ptr(), self.n,
                                     d["s"].data_ptr(), d["e"].data_ptr(), d["key"].data_ptr(),
                                     self.m, ctypes.byref(self.opts), None,
                                     self.tab["keys"].data_ptr(), ctypes.byref(self.ks),
                                     ctypes.byref(self.summ), self.ws.data_ptr(),
                                     self.ws.numel(), stream) == 0

        def finish(self, stream):
            assert lib.mag_attribute_finish(self.ws.data_ptr(), ctypes.byref(self.ks),
                                            ctypes.byref(self.summ), stream) == 0

    s1 = torch.cuda.current_stream()
    s2 = torch.cuda.Stream()
    ready = torch.cuda.Event()
    ready.record(s1)
    sa = Side(A, ctypes.c_void_p(ready.cuda_event))
    sb = Side(B)
    h1, h2 = ctypes.c_void_p(s1.cuda_stream), ctypes.c_void_p(s2.cuda_stream)

    def outputs(rows):
        o = {n: torch.empty(rows, dtype=dt, device="cuda") for n, dt in
             (("key", torch.int64), ("ratio", torch.float64), ("ea", torch.float64),
              ("eb", torch.float64), ("ca", torch.int64), ("cb", torch.int64),
              ("la", torch.float64), ("lb", torch.float64), ("v", torch.int32))}
        ro = N.RankOut(o["key"].data_ptr(), o["ratio"].data_ptr(), o["ea"].data_ptr(),
                       o["eb"].data_ptr(), o["ca"].data_ptr(), o["cb"].data_ptr(), rows, 0, 0,
                       0, 0)
        return o, ro

    b = ctypes.c_size_t(0)
    lib.mag_diff_workspace_size(cap, cap, cap, ctypes.byref(b))
    dws = torch.empty(int(b.value), dtype=torch.uint8, device="cuda")
    for rep in range(3):
        log(f"[device counts] repetition {rep}")
        sa.nk.fill_(-7)
        sb.nk.fill_(-7)
        sa.attribute(h1)
        s2.wait_event(ready)
        sb.attribute(h2)
        s1.wait_stream(s2)
        o1, ro1 = outputs(k)
        assert lib.mag_diff(sa.tab["keys"].data_ptr(), ctypes.byref(sa.kd),
                            sb.tab["keys"].data_ptr(), ctypes.byref(sb.kd), k, ctypes.byref(ro1),
                            dws.data_ptr(), dws.numel(), h1) == 0, lib.mag_last_error()
        o2, ro2 = outputs(cap)
        det = N.DetectOut()
        det.rank = ro2
        det.latency_a, det.latency_b, det.verdict = (o2["la"].data_ptr(), o2["lb"].data_ptr(),
                                                     o2["v"].data_ptr())
        opt = N.DetectOpts(0.05, 0.01)
        assert lib.mag_detect(sa.tab["keys"].data_ptr(), ctypes.byref(sa.kd),
                              sb.tab["keys"].data_ptr(), ctypes.byref(sb.kd), ctypes.byref(opt),
                              ctypes.byref(det), dws.data_ptr(), dws.numel(), h1) == 0
        sa.finish(h1)
        sb.finish(h2)
        assert int(sa.nk.item()) == sa.ks.n_keys and int(sb.nk.item()) == sb.ks.n_keys
        # the same comparison with host counts
        ta = {n: v[:sa.ks.n_keys] for n, v in sa.tab.items()}
        tb = {n: v[:sb.ks.n_keys] for n, v in sb.tab.items()}
        ref = mag.diff(ta, tb, k)
        r = int(ro1.n_out)
        assert r == len(ref["key"]) and ro1.n_join == ref["n_join"]
        assert ro1.n_only_a == ref["n_only_a"] and ro1.n_only_b == ref["n_only_b"]
        assert torch.equal(o1["key"][:r], ref["key"]) and torch.equal(o1["ratio"][:r], ref["ratio"])
        dref = mag.detect(ta, tb, 0.05, 0.01)
        assert det.n_flagged == dref["n_flagged"] and det.n_waste == dref["n_waste"]
        nf = int(det.rank.n_out)
        assert torch.equal(o2["key"][:nf], dref["key"])
        assert torch.equal(o2["v"][:nf], dref["verdict"])


def test_tile_events_serialize_the_trace_integrations():
    """tiles_done on A and tiles_wait on B: B's set-up runs at once, its
    trace integration after A's; both results equal the serial calls."""
    import torch
    import paper_2512_08365_amd as mag
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    cases = [synth.long_trace(seed, 300_000, 4, 20_000) for seed in (73, 74)]
    devs = [to_gpu(c) for c in cases]

    def run(d, c, **kw):
        off = [int(x) for x in c["offsets"]]
        return mag.attribute(d["t"], d["P"], d["s"], d["e"], d["key"], n_streams=len(off) - 1,
                             stream_offsets=off, **kw)

    serial = [run(d, c) for d, c in zip(devs, cases)]
    torch.cuda.synchronize()
    s2 = torch.cuda.Stream()
    a_tiles = torch.cuda.Event()
    for rep in range(3):
        log(f"[tile events] repetition {rep}")
        pend_a = run(devs[0], cases[0], asynchronous=True, tiles_done=a_tiles)
        with torch.cuda.stream(s2):
            pend_b = run(devs[1], cases[1], asynchronous=True, tiles_wait=a_tiles)
        res_b = pend_b.finish()
        res_a = pend_a.finish()
        torch.cuda.synchronize()
        for got, want in ((res_a, serial[0]), (res_b, serial[1])):
            for k in ("energy", "start_idx", "end_idx"):
                assert torch.equal(got[0][k], want[0][k]), k
            for k in ("keys", "count"):
                assert torch.equal(got[1][k], want[1][k]), k
            np.testing.assert_allclose(got[1]["sum"].cpu().numpy(), want[1]["sum"].cpu().numpy(),
                                       rtol=1e-12)


def test_group_stream_moves_the_grouping_off_the_tile_stream():
    """mag_attr_opts.group_stream: the fix-ups, grouping and status copy run on
    a second stream after the trace integration; results equal the one-stream
    call's (synchronous and MAG_ASYNC), and the tile stream takes the next
    call's trace integration while the first call still groups."""
    import torch
    import paper_2512_08365_amd as mag
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    cases = [synth.long_trace(seed, 200_000, 3, 15_000) for seed in (81, 82, 83)]
    devs = [to_gpu(c) for c in cases]

    def run(d, c, **kw):
        off = [int(x) for x in c["offsets"]]
        return mag.attribute(d["t"], d["P"], d["s"], d["e"], d["key"], n_streams=len(off) - 1,
                             stream_offsets=off, **kw)

    def same(got, want, label):
        for k in ("energy", "start_idx", "end_idx"):
            assert torch.equal(got[0][k], want[0][k]), (label, k)
        for k in ("keys", "count"):
            assert torch.equal(got[1][k], want[1][k]), (label, k)
        # per-key sums and M2 are added through LDS atomics in no fixed order:
        # equal up to rounding
        for k in ("sum", "m2"):
            np.testing.assert_allclose(got[1][k].cpu().numpy(), want[1][k].cpu().numpy(),
                                       rtol=1e-12, err_msg=f"{label} {k}")
        for k in ("n_keys", "n_clipped"):
            assert got[2][k] == want[2][k], (label, k)
        for k in ("trace_energy", "idle_energy", "attributed_energy"):
            assert abs(got[2][k] - want[2][k]) <= 1e-12 * abs(want[2][k]), (label, k)

    want = [run(d, c) for d, c in zip(devs, cases)]
    torch.cuda.synchronize()
    g = torch.cuda.Stream()
    for rep in range(2):
        log(f"[group stream] repetition {rep}")
        for i, (d, c) in enumerate(zip(devs, cases)):
            same(run(d, c, group_stream=g), want[i], f"synchronous {i}")
        # three asynchronous calls back to back: their trace integrations queue
        # on the current stream, their groupings on the group stream
        pend = [run(d, c, asynchronous=True, group_stream=g) for d, c in zip(devs, cases)]
        for i in reversed(range(3)):
            same(pend[i].finish(), want[i], f"asynchronous {i}, repetition {rep}")
    torch.cuda.synchronize()
