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
