"""Key plans (mag_key_plan_build): the key map of a grouping built from the
operator keys alone, ahead of the attribution or on another stream, gives the
attribution's results exactly; a plan serves several attributions of the same
keys; mismatched sizes and key overflow are reported."""
import numpy as np
import pytest

import synth
from gpu_util import E_RTOL, log, to_gpu

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
    a, b = got[1]["sum"].cpu().numpy(), want[1]["sum"].cpu().numpy()
    assert np.all(np.abs(a - b) <= E_RTOL * np.abs(b)), (label, "sum")
    cnt = want[1]["count"].cpu().numpy()
    second = want[1]["m2"].cpu().numpy() + b ** 2 / np.maximum(cnt, 1)
    assert np.all(np.abs(got[1]["m2"].cpu().numpy() - want[1]["m2"].cpu().numpy())
                  <= E_RTOL * second), (label, "m2")
    for k in ("n_keys", "n_clipped"):
        assert got[2][k] == want[2][k], (label, k)
    W = want[2]["trace_energy"]
    for k in ("trace_energy", "idle_energy", "attributed_energy"):
        assert abs(got[2][k] - want[2][k]) <= 1e-12 * max(abs(W), 1e-300), (label, k)


def test_plan_on_another_stream_equals_the_built_in_map():
    import torch
    import paper_2512_08365_amd as mag
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    cases = [("multi-stream", synth.long_trace(61, 600_000, 4, 40_000), 4096),
             ("decode-shaped A", synth.sides(2, 0)[0], 1024),
             ("tiny", synth.tiny_case(62, n=3000, streams=2, per_stream=80), None)]
    s3 = torch.cuda.Stream()
    for label, c, cap in cases:
        log(f"[case] key plan: {label}")
        d = to_gpu(c)
        want = _run(mag, d, c, key_capacity=cap)
        ready = torch.cuda.Event()
        with torch.cuda.stream(s3):
            plan = mag.KeyPlan(d["key"], cap, ready=ready)
        for rep in range(2):  # the plan serves two attributions
            _same(_run(mag, d, c, key_plan=plan), want, f"{label} rep{rep}")
        # asynchronous use
        pend = _run(mag, d, c, key_plan=plan, asynchronous=True)
        _same(pend.finish(), want, f"{label} async")
    torch.cuda.synchronize()


def test_plan_shared_by_both_sides_of_a_workload():
    import torch
    import paper_2512_08365_amd as mag
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    A, B = synth.sides(1, 0)  # the tiny A/B pair shares its operator keys
    assert np.array_equal(A["key"], B["key"])
    da, db = to_gpu(A), to_gpu(B)
    plan = mag.KeyPlan(da["key"], 64)
    for c, d, label in ((A, da, "A"), (B, db, "B")):
        _same(_run(mag, d, c, key_plan=plan), _run(mag, d, c, key_capacity=64), label)
    torch.cuda.synchronize()


def test_plan_errors():
    import torch
    import paper_2512_08365_amd as mag
    from paper_2512_08365_amd import _native as N
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    c = synth.tiny_case(63, n=2000, streams=1, per_stream=100, keys=40)
    c["key"] = np.arange(c["s"].shape[0], dtype=np.uint64) * np.uint64(7919)  # all distinct
    d = to_gpu(c)
    m = c["s"].shape[0]
    # a plan for fewer intervals is refused before any device work
    short = mag.KeyPlan(d["key"][: max(m - 1, 0)], 256)
    with pytest.raises(mag.MagnetonError) as ei:
        _run(mag, d, c, key_plan=short)
    assert ei.value.code == N.MAG_E_STATE
    # more distinct keys than the plan's capacity: the attribution reports it
    small = mag.KeyPlan(d["key"], max(m // 2, 1))
    with pytest.raises(mag.MagnetonError) as ei:
        _run(mag, d, c, key_plan=small)
    assert ei.value.code == N.MAG_E_CAPACITY
    torch.cuda.synchronize()
