"""The allocation-free attribution (mag_attribute_static, through the C ABI):
its scratch is the library's per-GPU static array instead of a workspace.
Two calls in a row, the second on a smaller input, equal mag_attribute's
results: per-interval energies and indices bit for bit, keys and counts
exactly, key sums and M2 within the parity bar.  Sizes beyond the scratch and
flags that need host resources are refused before any device work."""
import numpy as np
import pytest

import synth
from gpu_util import E_RTOL, log, to_gpu

pytestmark = pytest.mark.gpu


def _both(mag, c, equal_split=True, key_capacity=None):
    d = to_gpu(c)
    off = [int(x) for x in c["offsets"]]
    kw = dict(n_streams=len(off) - 1, stream_offsets=off, equal_split=equal_split,
              key_capacity=key_capacity)
    ref = mag.attribute(d["t"], d["P"], d["s"], d["e"], d["key"], **kw)
    got = mag.attribute_static(d["t"], d["P"], d["s"], d["e"], d["key"], **kw)
    return got, ref


def _same(got, want, label):
    gi, gk, gs = got
    wi, wk, ws = want
    for k in ("energy", "start_idx", "end_idx"):
        assert np.array_equal(gi[k].cpu().numpy(), wi[k].cpu().numpy()), (label, k)
    for k in ("keys", "count"):
        assert np.array_equal(gk[k].cpu().numpy(), wk[k].cpu().numpy()), (label, k)
    a, b = gk["sum"].cpu().numpy(), wk["sum"].cpu().numpy()
    assert np.all(np.abs(a - b) <= E_RTOL * np.abs(b)), (label, "sum")
    cnt = wk["count"].cpu().numpy()
    second = wk["m2"].cpu().numpy() + b ** 2 / np.maximum(cnt, 1)
    assert np.all(np.abs(gk["m2"].cpu().numpy() - wk["m2"].cpu().numpy()) <= E_RTOL * second), \
        (label, "m2")
    assert gs["n_keys"] == ws["n_keys"] and gs["n_clipped"] == ws["n_clipped"], label
    for f in ("trace_energy", "idle_energy", "attributed_energy"):
        assert abs(gs[f] - ws[f]) <= 1e-12 * max(abs(ws["trace_energy"]), 1e-300), (label, f)


def test_static_scratch_equals_workspace_call_on_two_calls():
    import torch
    import paper_2512_08365_amd as mag
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    # first a large input (multi-stream, 2M samples, 400K intervals), then a
    # smaller one on the same scratch (its leftovers must not leak in)
    cases = [("multi-stream 2M", synth.long_trace(41, 2_000_000, 4, 100_000), True, 4096),
             ("decode-shaped", synth.sides(2, 1)[0], True, 1024),
             ("tiny fuzz", synth.tiny_case(42, n=3000, streams=3, per_stream=60), False, None)]
    for label, c, split, cap in cases:
        log(f"[case] static scratch: {label} n={c['t'].shape[0]} m={c['s'].shape[0]}")
        got, ref = _both(mag, c, equal_split=split, key_capacity=cap)
        _same(got, ref, label)
    torch.cuda.synchronize()


def test_static_scratch_refusals():
    import torch
    import paper_2512_08365_amd as mag
    from paper_2512_08365_amd import _native as N
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    c = synth.tiny_case(43, n=2000, streams=1, per_stream=50)
    d = to_gpu(c)
    # a key capacity whose hash table and partial tables exceed the scratch
    with pytest.raises(mag.MagnetonError) as ei:
        mag.attribute_static(d["t"], d["P"], d["s"], d["e"], d["key"], key_capacity=4_000_000)
    assert ei.value.code == N.MAG_E_WORKSPACE
    assert mag.workspace_size(2000, c["s"].shape[0], 4_000_000) > N.MAG_STATIC_SCRATCH_BYTES
    torch.cuda.synchronize()
