"""Asynchronous attributions (MAG_ASYNC) and their status records.

Each asynchronous call keeps a per-thread record of its workspace: the pinned
buffer its status block is copied into and the stream the copy runs on.  More
unfinished calls than the records kept when idle (16) must each still deliver
their own key count, summary and errors; a call finished while another stream
is current must wait for its own stream; a second call on a workspace whose
asynchronous call is not finished is refused.
"""
import ctypes

import numpy as np
import pytest

import synth
from gpu_util import log, to_gpu

pytestmark = pytest.mark.gpu


def _run(mag, d, c, **kw):
    off = [int(x) for x in c["offsets"]]
    return mag.attribute(d["t"], d["P"], d["s"], d["e"], d["key"], n_streams=len(off) - 1,
                         stream_offsets=off, **kw)


def _same(got, want, label):
    import torch
    for k in ("energy", "start_idx", "end_idx"):
        assert torch.equal(got[0][k], want[0][k]), (label, k)
    for k in ("keys", "count"):
        assert torch.equal(got[1][k], want[1][k]), (label, k)
    np.testing.assert_allclose(got[1]["sum"].cpu().numpy(), want[1]["sum"].cpu().numpy(),
                               rtol=1e-12, err_msg=label)
    for k in ("n_keys", "n_clipped"):
        assert got[2][k] == want[2][k], (label, k)
    assert abs(got[2]["trace_energy"] - want[2]["trace_energy"]) <= 1e-12 * want[2]["trace_energy"]


def test_twenty_outstanding_calls_keep_their_own_status():
    import torch
    import paper_2512_08365_amd as mag
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    # different key counts per case, so a status read from another call's
    # record would show up as a wrong n_keys
    cases = [synth.tiny_case(900 + i, n=4000 + 97 * i, streams=1 + i % 3, per_stream=40 + 7 * i)
             for i in range(20)]
    for i, c in enumerate(cases):
        c["key"] = (c["key"] % np.uint64(3 + i)).astype(np.uint64)
    devs = [to_gpu(c) for c in cases]
    serial = [_run(mag, d, c) for d, c in zip(devs, cases)]
    torch.cuda.synchronize()
    s2 = torch.cuda.Stream()
    for rep in range(2):
        log(f"[async] 20 outstanding calls, repetition {rep}")
        pend = []
        for i, (d, c) in enumerate(zip(devs, cases)):
            if i % 2:
                with torch.cuda.stream(s2):
                    pend.append(_run(mag, d, c, asynchronous=True))
            else:
                pend.append(_run(mag, d, c, asynchronous=True))
            # synchronous calls in between take records of their own
            if i % 5 == 4:
                _ = mag.diff(serial[i][1], serial[i - 1][1], 3)
        # finished in reverse order, each from the default stream
        for i in reversed(range(len(pend))):
            _same(pend[i].finish(), serial[i], f"call {i}")
        torch.cuda.synchronize()


def test_finish_waits_for_the_stream_of_the_call():
    import torch
    import paper_2512_08365_amd as mag
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    c = synth.long_trace(81, 400_000, 4, 30_000)
    d = to_gpu(c)
    want = _run(mag, d, c)
    torch.cuda.synchronize()
    s2 = torch.cuda.Stream()
    for rep in range(3):
        # a long kernel ahead of the call on s2 keeps its status copy pending
        # while the default stream is idle
        with torch.cuda.stream(s2):
            x = torch.randn(4096, 4096, device="cuda", dtype=torch.float32)
            for _ in range(8):
                x = x @ x
                x = x / x.abs().max()
            pend = _run(mag, d, c, asynchronous=True)
        got = pend.finish()  # the default stream is current here
        _same(got, want, f"finished off its stream, repetition {rep}")
    torch.cuda.synchronize()


def test_second_call_on_an_unfinished_workspace_is_refused():
    import torch
    import paper_2512_08365_amd as mag
    from paper_2512_08365_amd import _native as N
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    c = synth.tiny_case(5, n=3000, streams=2, per_stream=30)
    d = to_gpu(c)
    off = [int(x) for x in c["offsets"]]
    ws = torch.empty(mag.workspace_size(3000, c["s"].shape[0], c["s"].shape[0], 2, off),
                     dtype=torch.uint8, device="cuda")
    want = _run(mag, d, c)
    pend = _run(mag, d, c, asynchronous=True, workspace=ws)
    with pytest.raises(mag.MagnetonError) as ei:
        _run(mag, d, c, workspace=ws)
    assert ei.value.code == N.MAG_E_STATE
    _same(pend.finish(), want, "after the refused call")
    # once finished the workspace takes calls again
    _same(_run(mag, d, c, workspace=ws), want, "workspace reused")
    torch.cuda.synchronize()


def _same_rank(got, want, label):
    import torch
    for k in ("key", "ratio", "energy_a", "energy_b", "count_a", "count_b"):
        assert torch.equal(got[k], want[k]), (label, k)
    for k in ("n_only_a", "n_only_b", "n_join"):
        assert got[k] == want[k], (label, k)


def test_asynchronous_diffs_match_synchronous_ones():
    """mag_diff_async / mag_diff_finish: several comparisons in flight on two
    streams, each with its own workspace, give mag_diff's rows and counts; a
    second call on a workspace whose asynchronous comparison is not finished
    is refused, and so is finishing one twice."""
    import torch
    import paper_2512_08365_amd as mag
    from paper_2512_08365_amd import _native as N
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    tabs = []
    for i in range(7):
        c = synth.tiny_case(1300 + i, n=6000, streams=2, per_stream=80)
        c["key"] = (c["key"] % np.uint64(11 + 5 * i)).astype(np.uint64)
        tabs.append(_run(mag, to_gpu(c), c)[1])
    torch.cuda.synchronize()
    want = [mag.diff(tabs[0], tabs[i], 7) for i in range(1, 7)]
    s2 = torch.cuda.Stream()
    for rep in range(2):
        log(f"[async] 6 outstanding comparisons, repetition {rep}")
        pend = []
        for i in range(1, 7):
            if i % 2:
                with torch.cuda.stream(s2):
                    pend.append(mag.diff(tabs[0], tabs[i], 7, asynchronous=True))
            else:
                pend.append(mag.diff(tabs[0], tabs[i], 7, asynchronous=True))
        for i in reversed(range(6)):  # finished in another order than enqueued
            _same_rank(pend[i].result(), want[i], f"comparison {i + 1}, repetition {rep}")
    na, nb = int(tabs[0]["keys"].shape[0]), int(tabs[1]["keys"].shape[0])
    ws = torch.empty(mag.diff_workspace_size(na, nb, 7), dtype=torch.uint8, device="cuda")
    p1 = mag.diff(tabs[0], tabs[1], 7, workspace=ws, asynchronous=True)
    with pytest.raises(mag.MagnetonError) as ei:
        mag.diff(tabs[0], tabs[2], 7, workspace=ws)
    assert ei.value.code == N.MAG_E_STATE
    _same_rank(p1.result(), want[0], "after the refused call")
    lib = mag._lib()
    ro = N.RankOut()
    assert lib.mag_diff_finish(ctypes_ptr(ws), ctypes.byref(ro)) == N.MAG_E_STATE
    _same_rank(mag.diff(tabs[0], tabs[2], 7, workspace=ws), want[1], "workspace reused")
    torch.cuda.synchronize()


def ctypes_ptr(t):
    import ctypes
    return ctypes.c_void_p(t.data_ptr())
