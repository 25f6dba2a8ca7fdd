#!/usr/bin/env python3
"""Throughput of operator energy attribution + A/B diff on one MI355X.

Default (the headline): one step = the whole path over one A/B pair of the
multi-stream workload (100,000,000 power samples at 1 MHz, 4 concurrent
streams x 1,000,000 operator intervals, 5,000 Zipf(1.2) keys): attribute side
A, attribute side B (equal split of concurrent power, per-interval energies
and sample indices, per-key count/sum/M2), then join and rank the top-100
excess-energy keys.  Side A runs on the current stream; side B on a second
stream (default priority) whose trace integration waits for A's (the
`tiles_wait` / `tiles_done` events), so the two tile kernels run back to back
while A's per-key grouping overlaps B's tile kernel.  Both attributions and
the diff are enqueued asynchronously (key counts stay on the device) and
collected with one host wait per step, on events of their own.  Two steps are
kept in flight (`--pipeline`), each with its own outputs and workspaces:
step i is enqueued before step i-1 is collected, and A's tile kernel of a
step waits for B's of the step before.  B's key map (distinct keys, ids,
ranks: it depends on the keys only) is built on a third stream while A's
trace is integrated.  The diff runs on A's stream of the step once B's call
is complete (A's two streams alternate, so that stream is idle until the
step after next), so B's next tile kernel does not queue behind it.  Side
A's tile kernel is timed with HIP events carried on its dispatch in every
timed step; side B runs untimed.  Inputs are
synthetic, seeded and resident in HBM before timing.

--workload 1/2/3/4/5 times the other workloads the same way (2 and 4 fit in
or near the 256 MB Infinity Cache and are timed with a 512 MB flush before
each step); workload 5 streams both sides in 32,000,000-sample chunks,
kernel-only (chunks already in HBM) or --end-to-end (from pinned host memory,
PCIe-bound).

Prints ONE JSON line.  `value` is operator intervals attributed per second
(all sides); samples/s and the step's algorithmic HBM GB/s ride along
(`pipeline_roofline`, at 12 B per sample and 48 B per interval).  `roofline`
covers the dominant kernel (the interval-energy tile kernel), timed with HIP
events on the call's stream; `cpu_baseline` is the CPU oracle timed on one
pinned host core over sides of the same workload.  `copy_ceiling` is the
achievable bandwidth of a trivial 1 GiB copy kernel measured in the same run;
both rooflines also give their fraction of it (`frac_of_copy_ceiling`).
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
METRIC = "operator intervals attributed/sec + power samples/sec; achieved HBM GB/s"
WORKLOAD = 3
TOP_K = 100


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def source_hash() -> str:
    h = hashlib.sha256()
    with open(os.path.join(ROOT, "paper_2512_08365_amd", "csrc", "attr_tile.hip"), "rb") as f:
        h.update(f.read())
    return h.hexdigest()[:16]


COUNTERS_JSON = os.path.join(ROOT, "profiles", "tile_kernel_counters.json")
COPY_BYTES = 1 << 30  # calibration copy: 1 GiB read + 1 GiB written


def counters_traffic(algorithmic_bytes):
    """HBM bytes per launch of the tile kernel from the committed counter
    summary, if it was taken on the current kernel source and on a launch of
    the same algorithmic size, i.e. the same workload (else None)."""
    try:
        with open(COUNTERS_JSON) as f:
            d = json.load(f)
    except (OSError, ValueError):
        return None
    if d.get("source_hash") != source_hash():
        return None
    if d.get("algorithmic_bytes_per_launch") != algorithmic_bytes:
        return None
    return d.get("traffic_bytes_per_launch")


def copy_calibration():
    """A plain streaming copy of COPY_BYTES (torch's elementwise kernel computing
    dst = src * 1), run under the same counters as the tile kernel to scale
    FETCH_SIZE / WRITE_SIZE."""
    import torch
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        torch.mul(src, 1.0, out=dst)
    torch.cuda.synchronize()
    log(f"[calibration] copied {COPY_BYTES} bytes 3 times")


# achievable HBM bandwidth on this device, measured once per run (copy_ceiling)
CEILING = {}


def copy_ceiling(torch):
    """The achievable-bandwidth ceiling: a trivial streaming copy kernel
    (torch's vectorized elementwise kernel computing dst = src * 1, the
    calibration copy: COPY_BYTES read and COPY_BYTES written), the median of 10
    launches timed with HIP events after 2 untimed ones.  (torch's copy_ goes
    through the runtime's blit kernel, measured slower: 4.4-5.1 against
    6.1-6.2 TB/s.)"""
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(2):
        torch.mul(src, 1.0, out=dst)
    ev = []
    for _ in range(10):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        torch.mul(src, 1.0, out=dst)
        e1.record()
        ev.append((e0, e1))
    torch.cuda.synchronize()
    ms = sorted(a.elapsed_time(b) for a, b in ev)[len(ev) // 2]
    del src, dst
    torch.cuda.empty_cache()
    CEILING.update({"kernel": "elementwise dst = src * 1 over 1 GiB (1 GiB read + 1 GiB written)",
                    "gbps": 2 * COPY_BYTES / (ms * 1e-3) / 1e9, "ms": ms})
    log(f"[bench] copy ceiling {CEILING['gbps']:.0f} GB/s")


def _counter_rows(path, kernel_substr, counter):
    import csv
    vals = []
    with open(path) as f:
        for row in csv.DictReader(f):
            if kernel_substr in row["Kernel_Name"] and row["Counter_Name"] == counter:
                vals.append(float(row["Counter_Value"]))
    if not vals:
        raise SystemExit(f"no {counter} rows for '{kernel_substr}' in {path}")
    return vals


def summarize_counters(tile_fetch, tile_write, copy_fetch, copy_write, copy_kernel, tile_bytes):
    """FETCH_SIZE / WRITE_SIZE (KiB per dispatch) of the tile kernel, scaled by
    what the same counters read for the calibration copy of known size."""
    f_t = _counter_rows(tile_fetch, "k_tile", "FETCH_SIZE")
    w_t = _counter_rows(tile_write, "k_tile", "WRITE_SIZE")
    f_c = _counter_rows(copy_fetch, copy_kernel, "FETCH_SIZE")
    w_c = _counter_rows(copy_write, copy_kernel, "WRITE_SIZE")
    # the largest dispatches of the copy kernel are the 1 GiB copies
    f_c = max(f_c)
    w_c = max(w_c)
    kf = COPY_BYTES / (f_c * 1024.0)
    kw = COPY_BYTES / (w_c * 1024.0)
    fetch = sum(f_t) / len(f_t) * 1024.0 * kf
    write = sum(w_t) / len(w_t) * 1024.0 * kw
    d = {"source_hash": source_hash(), "kernel": "k_tile",
         "fetch_kib_per_dispatch_raw": sum(f_t) / len(f_t),
         "write_kib_per_dispatch_raw": sum(w_t) / len(w_t),
         "copy_fetch_kib_raw": f_c, "copy_write_kib_raw": w_c,
         "fetch_scale": kf, "write_scale": kw,
         "fetch_bytes_per_launch": fetch, "write_bytes_per_launch": write,
         "traffic_bytes_per_launch": fetch + write,
         "algorithmic_bytes_per_launch": tile_bytes,
         "traffic_over_algorithmic": (fetch + write) / tile_bytes}
    with open(COUNTERS_JSON, "w") as f:
        json.dump(d, f, indent=1)
        f.write("\n")
    print(json.dumps(d, indent=1))


class Side:
    """Device copies of one side plus preallocated outputs and workspace."""

    def __init__(self, c, lib, N, torch, k_cap, timed=True, ready_event=None, tiles_wait=None,
                 tiles_done=None, key_plan=False, inputs=None, group_stream=None,
                 shared_plan=None):
        import numpy as np
        self.n = int(c["t"].shape[0])
        self.m = int(c["s"].shape[0])
        self.off = [int(x) for x in c["offsets"]]
        dev = "cuda"
        if inputs is not None:
            # another Side's device inputs (its own outputs and workspace)
            self.t, self.P, self.s, self.e, self.key = (inputs.t, inputs.P, inputs.s, inputs.e,
                                                        inputs.key)
        else:
            self.t = torch.from_numpy(c["t"]).to(dev)
            self.P = torch.from_numpy(c["P"]).to(dev)
            self.s = torch.from_numpy(c["s"]).to(dev)
            self.e = torch.from_numpy(c["e"]).to(dev)
            self.key = torch.from_numpy(np.ascontiguousarray(c["key"]).view(np.int64)).to(dev)
        self.energy = torch.empty(self.m, dtype=torch.float64, device=dev)
        self.si = torch.empty(self.m, dtype=torch.int64, device=dev)
        self.ei = torch.empty(self.m, dtype=torch.int64, device=dev)
        self.kout = torch.empty(k_cap, dtype=torch.int64, device=dev)
        self.ksum = torch.empty(k_cap, dtype=torch.float64, device=dev)
        self.km2 = torch.empty(k_cap, dtype=torch.float64, device=dev)
        self.kcnt = torch.empty(k_cap, dtype=torch.int64, device=dev)
        self.k_cap = k_cap
        self.offs = (ctypes.c_int64 * len(self.off))(*self.off)
        flags = N.MAG_EQUAL_SPLIT | N.MAG_ASYNC | (N.MAG_TIME_KERNELS if timed else 0)
        self.plan = shared_plan  # a key plan of the same keys, built by the caller
        if key_plan and shared_plan is None:
            # the key map is built on its own stream (build_plan), early in the
            # step, and the grouping waits for it
            b = ctypes.c_size_t(0)
            assert lib.mag_key_plan_size(self.m, k_cap, ctypes.byref(b)) == 0
            self.plan_buf = torch.empty(int(b.value), dtype=torch.uint8, device=dev)
            self.plan_ready = torch.cuda.Event()
            self.plan_ready.record()
            self.plan = N.KeyPlan(self.plan_buf.data_ptr(), self.plan_buf.numel(), 0, 0,
                                  ctypes.c_void_p(self.plan_ready.cuda_event))
        self.opts = N.AttrOpts(len(self.off) - 1, flags, ctypes.cast(self.offs, ctypes.c_void_p),
                               ready_event, ctypes.pointer(self.plan) if self.plan else None,
                               tiles_wait, tiles_done,
                               ctypes.c_void_p(group_stream.cuda_stream) if group_stream else None)
        b = ctypes.c_size_t(0)
        rc = lib.mag_attribute_workspace_size(self.n, self.m, k_cap, ctypes.byref(self.opts),
                                              ctypes.byref(b))
        assert rc == 0
        self.ws = torch.empty(int(b.value), dtype=torch.uint8, device=dev)
        self.pio = N.IntervalOut(self.energy.data_ptr(), self.si.data_ptr(), self.ei.data_ptr())
        # the key-row count is also left on the device, so that the diff can
        # be enqueued behind the attribution without a host wait
        self.nkd = torch.zeros(1, dtype=torch.int64, device=dev)
        self.ks = N.KeyStats(self.ksum.data_ptr(), self.km2.data_ptr(), self.kcnt.data_ptr(), k_cap,
                             0, None, self.nkd.data_ptr())
        self.ks_dev = N.KeyStats(self.ksum.data_ptr(), self.km2.data_ptr(), self.kcnt.data_ptr(),
                                 k_cap, -1, None, self.nkd.data_ptr())
        self.summ = N.Summary()

    def build_plan(self, lib, stream):
        """Enqueue this side's key map (mag_key_plan_build) on `stream`."""
        rc = lib.mag_key_plan_build(self.key.data_ptr(), self.m, self.k_cap,
                                    ctypes.byref(self.plan), stream)
        if rc != 0:
            raise RuntimeError(f"mag_key_plan_build failed {rc}: {lib.mag_last_error().decode()}")

    def attribute(self, lib, stream):
        """Enqueue this side's attribution (MAG_ASYNC: returns at once)."""
        rc = lib.mag_attribute(self.t.data_ptr(), self.P.data_ptr(), self.n, self.s.data_ptr(),
                               self.e.data_ptr(), self.key.data_ptr(), self.m,
                               ctypes.byref(self.opts), ctypes.byref(self.pio), self.kout.data_ptr(),
                               ctypes.byref(self.ks), ctypes.byref(self.summ), self.ws.data_ptr(),
                               self.ws.numel(), stream)
        if rc != 0:
            raise RuntimeError(f"mag_attribute failed {rc}: {lib.mag_last_error().decode()}")

    def finish(self, lib, stream):
        """Wait for the attribution; its key count, errors and tile-kernel time."""
        rc = lib.mag_attribute_finish(self.ws.data_ptr(), ctypes.byref(self.ks),
                                      ctypes.byref(self.summ), stream)
        if rc != 0:
            raise RuntimeError(f"mag_attribute_finish failed {rc}: {lib.mag_last_error().decode()}")
        return self.summ.tile_kernel_ms


def host_description() -> dict:
    """This host's core count and CPU model (recorded with the oracle baseline)."""
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        allowed = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        allowed = None
    return {"nproc": os.cpu_count(), "cpus_allowed": allowed, "cpu_model": model}


class pinned_thread:
    """Pin the calling thread (not the process: the GPU runtime's own threads
    keep their affinity) to one allowed CPU while the oracle is timed."""

    def __enter__(self):
        self.old = None
        self.cpu = None
        try:
            self.old = os.sched_getaffinity(0)
            self.cpu = min(self.old)
            os.sched_setaffinity(0, {self.cpu})
        except (AttributeError, OSError):
            self.old = None
        return self

    def __exit__(self, *exc):
        if self.old is not None:
            os.sched_setaffinity(0, self.old)
        return False


def cpu_baseline(sides, pairs, label):
    """The oracle, as it stands, on the given sides of the workload, pinned to
    one core: attribution and grouping of every side, then the diffs."""
    import oracle
    with pinned_thread() as pin:
        t0 = time.perf_counter()
        tabs = []
        for c in sides:
            r = oracle.attribute(c["t"], c["P"], c["s"], c["e"], c["offsets"])
            tabs.append(oracle.groupby(c["key"], r["energy"]))
        for a, b in pairs:
            oracle.diff(tabs[a], tabs[b], TOP_K)
        dt = time.perf_counter() - t0
    m = sum(c["s"].shape[0] for c in sides)
    n = sum(c["t"].shape[0] for c in sides)
    res = {"value": m / dt, "unit": "intervals/s", "cores": 1, "kind": "oracle",
           "sample": f"{label}: attribution + grouping + top-{TOP_K} diff, {dt:.1f} s",
           "seconds": round(dt, 2), "samples_per_s": n / dt, "pinned_cpu": pin.cpu}
    res.update(host_description())
    return res


def counter_session(args, torch, mag):
    """Counter (software replay) attribution of a replay profiling session:
    98,304 operator windows x 1,000 replays read by a 50 Hz counter with a
    0.1 s lag, with per-key energy and latency; one JSON line."""
    import numpy as np
    import synth
    c = synth.replay_session(args.seed)
    d = {k: torch.from_numpy(np.ascontiguousarray(c[k])).cuda() for k in ("t", "C", "s", "e")}
    key = torch.from_numpy(c["key"].view(np.int64)).cuda()
    reps = torch.from_numpy(c["reps"]).cuda()
    n, m = int(c["t"].shape[0]), int(c["s"].shape[0])
    cap = 1024
    ws = torch.empty(mag.counter_workspace_size(n, m, cap, mag.KEY_LATENCY), dtype=torch.uint8,
                     device="cuda")
    out = {"energy": torch.empty(m, dtype=torch.float64, device="cuda"),
           "start_idx": torch.empty(m, dtype=torch.int64, device="cuda"),
           "end_idx": torch.empty(m, dtype=torch.int64, device="cuda")}

    def call(timed):
        return mag.attribute_counter(d["t"], d["C"], d["s"], d["e"], key, delay=c["delay"],
                                     replays=reps, key_capacity=cap, workspace=ws, out=out,
                                     latency=True, time_kernels=timed)

    for _ in range(args.warmup):
        call(False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        call(False)
    torch.cuda.synchronize()
    sec = (time.perf_counter() - t0) / args.steps
    kms = [call(True)[2]["kernel_ms"] for _ in range(args.steps)]
    kernel_ms = sum(kms) / len(kms)
    res = {"mode": "counter replay session", "n_readings": n, "n_windows": m, "keys": 416,
           "ms_per_call": sec * 1e3, "windows_per_s": m / sec, "readings_per_s": n / sec,
           "window_kernel_ms": kernel_ms,
           "window_kernel_gbps": (16 * n + 44 * m) / (kernel_ms * 1e-3) / 1e9}
    if not args.no_cpu_baseline:
        import oracle
        t0 = time.perf_counter()
        r = oracle.counter_attribute(c["t"], c["C"], c["s"], c["e"], c["delay"], c["reps"])
        oracle.groupby(c["key"], r["energy"])
        oracle.key_latency(c["key"], c["s"], c["e"], c["reps"])
        dt = time.perf_counter() - t0
        res["cpu_baseline"] = {"value": m / dt, "unit": "windows/s", "cores": 1, "kind": "oracle",
                               "sample": "the whole session, attribution + grouping + latency",
                               "seconds": round(dt, 3)}
    print(json.dumps(res), flush=True)


def invariants_bench(args, torch, mag):
    """Multi-mode SVD invariants of a batch of tensors (default: shaped like
    per-layer attention K/V tensors, 64 x fp32 [32 heads, 128 tokens, 128 head
    dims]; --inv-shape / --inv-count for others, e.g. one 4096 x 4096 weight)
    and the all-pairs matching of the batch against a copy with its first two
    modes swapped; one JSON line."""
    import numpy as np
    rng = np.random.default_rng(args.seed)
    shape = tuple(int(x) for x in args.inv_shape.split(","))
    count = args.inv_count
    r = len(shape)
    host = [rng.standard_normal(shape).astype(np.float32) for _ in range(count)]
    A = [torch.from_numpy(h).cuda() for h in host]
    # the other system's layout: the first two modes swapped (NHD for attention K/V)
    perm = (1, 0) + tuple(range(2, r)) if r >= 2 else (0,)
    B = [x.permute(*perm).contiguous() for x in A]
    lay = mag.invariant_layout(A[0])
    # algorithmic work of the Gram products: K (K + 1) L flops per unfolding
    flops = 0
    for g in range(1, (1 << r) - 1, 2):
        M = int(np.prod([shape[i] for i in range(r) if g >> i & 1]))
        N = int(np.prod(shape)) // M
        K, L = min(M, N), max(M, N)
        flops += K * (K + 1) * L
    flops *= count
    ws = torch.empty(1, dtype=torch.uint8, device="cuda")
    for _ in range(max(args.warmup, 1)):
        sa, _ = mag.invariants(A)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        sa, _ = mag.invariants(A)
    torch.cuda.synchronize()
    sec = (time.perf_counter() - t0) / args.steps
    sb, _ = mag.invariants(B)
    m = mag.match(A, sa, B, sb, 1e-5)  # (the first call also allocates)
    torch.cuda.synchronize()
    reps = max(args.steps, 1)
    t1 = time.perf_counter()
    for _ in range(reps):
        m = mag.match(A, sa, B, sb, 1e-5)
    torch.cuda.synchronize()
    msec = (time.perf_counter() - t1) / reps
    matched = int(m.sum().item())
    res = {"mode": "tensor invariants", "tensors": count, "shape": list(shape),
           "spectrum_lengths": lay, "ms_per_batch": sec * 1e3, "tensors_per_s": count / sec,
           "gram_tflops_algorithmic_over_call": flops / sec / 1e12,
           f"match_ms_{count}x{count}": msec * 1e3, "matched_pairs": matched}
    if not args.no_cpu_baseline:
        from threadpoolctl import threadpool_limits
        from oracle import spectra as S
        ns = min(8, count)
        with threadpool_limits(1):
            t0 = time.perf_counter()
            for h in host[:ns]:
                S.invariants(h)
            dt = (time.perf_counter() - t0) / ns
        res["cpu_baseline"] = {"value": 1.0 / dt, "unit": "tensors/s", "cores": 1,
                               "kind": "oracle",
                               "sample": f"{ns} of the {count} tensors, numpy SVD",
                               "seconds_per_tensor": round(dt, 4)}
    print(json.dumps(res), flush=True)


def subgraphs_bench(args):
    """Section 4.2's subgraph matching (host code) on two planted graphs of
    20,000 blocks (about 100,000 operators each); the oracle on 300 blocks."""
    import paper_2512_08365_amd as mag
    import synth
    c = synth.graph_pair(args.seed, blocks=20000, width=4, decoys=2000, crossing=200)
    nodes = c["n1"] + c["n2"]
    t0 = time.perf_counter()
    pairs = mag.match_subgraphs(c["n1"], c["edges1"], c["n2"], c["edges2"], c["eq"])
    dt = time.perf_counter() - t0
    res = {"mode": "subgraph matching (host)", "nodes": nodes,
           "edges": len(c["edges1"]) + len(c["edges2"]), "pairs": len(pairs),
           "seconds": dt, "nodes_per_s": nodes / dt}
    if not args.no_cpu_baseline:
        from oracle import graph_match as G
        s = synth.graph_pair(args.seed, blocks=300, width=4, decoys=30, crossing=3)
        t0 = time.perf_counter()
        G.match(s["n1"], s["edges1"], s["n2"], s["edges2"], s["eq"])
        ot = time.perf_counter() - t0
        res["cpu_baseline"] = {"value": (s["n1"] + s["n2"]) / ot, "unit": "nodes/s", "cores": 1,
                               "kind": "oracle", "sample": "the same generator at 300 blocks",
                               "seconds": round(ot, 3)}
    print(json.dumps(res), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--workload", type=int, default=WORKLOAD, choices=[1, 2, 3, 4, 5],
                    help="workload to time (default 3, the multi-stream 100M-sample trace)")
    ap.add_argument("--pipeline", type=int, default=2,
                    help="A/B workloads: steps in flight, each on its own outputs and "
                         "workspaces (1 = every step collected before the next is enqueued)")
    ap.add_argument("--schedule", choices=["overlap", "plans", "serial", "tilestream"],
                    default="overlap",
                    help="A/B workloads: B's trace integration waits for A's and overlaps A's "
                         "grouping (overlap: B's key map built ahead on a third stream; plans: "
                         "A's too), or waits for A's whole call (serial, both key maps ahead); "
                         "tilestream: both trace integrations on one stream, each side's "
                         "grouping on a stream of its own (group_stream), both key maps ahead")
    ap.add_argument("--timed-side", choices=["a", "b", "none"], default="a",
                    help="which side's tile kernel carries the HIP timing events")
    ap.add_argument("--end-to-end", action="store_true",
                    help="workload 5 only: push the chunks from pinned host memory")
    ap.add_argument("--subgraphs", action="store_true",
                    help="measure the host-side subgraph matching (Section 4.2) instead")
    ap.add_argument("--invariants", action="store_true",
                    help="measure the tensor invariants (Section 4.2) instead")
    ap.add_argument("--inv-shape", default="32,128,128",
                    help="--invariants: tensor shape (comma-separated)")
    ap.add_argument("--inv-count", type=int, default=64, help="--invariants: tensors per batch")
    ap.add_argument("--counter-session", action="store_true",
                    help="measure the counter (software replay) attribution instead")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run the 1 GiB calibration copy (for the HBM counters)")
    ap.add_argument("--summarize-counters", nargs=5,
                    metavar=("TILE_FETCH_CSV", "TILE_WRITE_CSV", "COPY_FETCH_CSV",
                             "COPY_WRITE_CSV", "COPY_KERNEL_SUBSTR"),
                    help="write the tile kernel's scaled HBM traffic from rocprofv3 --pmc CSVs")
    args = ap.parse_args()
    if args.summarize_counters:
        import synth
        sh = synth.shape(WORKLOAD)
        summarize_counters(*args.summarize_counters, tile_bytes=12 * sh["n"] + 48 * sh["m"])
        return
    if args.subgraphs:
        subgraphs_bench(args)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported by this build "
              "(the multi-GPU sharding is design-only).", file=sys.stderr)
        sys.exit(2)

    import numpy as np  # noqa: F401
    import torch

    import paper_2512_08365_amd as mag
    from paper_2512_08365_amd import _native as N
    import synth

    if not torch.cuda.is_available():
        log("bench.py needs a GPU")
        sys.exit(1)
    if args.copy_calibration:
        copy_calibration()
        return
    if args.counter_session:
        counter_session(args, torch, mag)
        return
    if args.invariants:
        invariants_bench(args, torch, mag)
        return
    lib = N.load()
    log(f"[bench] {mag.version()} on {torch.cuda.get_device_name(0)}")
    copy_ceiling(torch)
    if args.workload in (1, 2, 3):
        ab_bench(args, torch, mag, lib, N, synth)
    elif args.workload == 4:
        sweep_bench(args, torch, mag, lib, N, synth)
    else:
        long_bench(args, torch, mag, synth)


WORKLOADS = {
    1: ("tiny A/B pair: 10,000 samples at 1 ms (jittered), 2,000 sequential intervals, "
        "50 Zipf(1.1) keys; A+B attribution + top-10 diff"),
    2: ("decode-shaped trace: 2,000,000 samples at 100 kHz, 32 layers x 12 ops x 256 steps = "
        "98,304 sequential intervals, 416 keys; A+B attribution + top-10 diff"),
    3: ("multi-stream trace: 100,000,000 fp32 power samples at 1 MHz, 4 concurrent streams x "
        "1,000,000 intervals (equal split), 5,000 Zipf(1.2) keys; A+B attribution + top-100 diff"),
    4: ("batched sweep: baseline + 8 candidate traces, each 20,000,000 samples at 200 kHz and "
        "1,000,000 sequential intervals, 2,000 keys; 9 attributions + one batched top-100 diff "
        "of the 8 candidates"),
    5: ("long-run trace: 360,000,000 samples at 100 kHz, 50,000,000 sequential intervals, "
        "20,000 Zipf(1.05) keys, both sides streamed in 32,000,000-sample chunks; "
        "A+B attribution + top-100 diff"),
}
TOPK = {1: 10, 2: 10, 3: 100, 4: 100, 5: 100}
MALL_FLUSH_BYTES = 512 << 20  # larger than the 256 MB Infinity Cache


def result_line(args, cfg, sh, sides, sec_per_step, extra):
    n, m = sh["n"], sh["m"]
    bytes_step = sides * (12 * n + 48 * m)  # algorithmic bytes of a step (12 B/sample + 48 B/interval)
    gbs = bytes_step / sec_per_step / 1e9
    r = {
        "metric": METRIC,
        "value": sides * m / sec_per_step,
        "unit": "intervals/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": sec_per_step * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": WORKLOADS[cfg], "n_samples_per_side": n, "n_intervals_per_side": m,
                   "streams": sh["streams"], "keys": sh["K"], "top_k": TOPK[cfg], "sides": sides,
                   "seed": args.seed},
        "samples_per_s": sides * n / sec_per_step,
        "hbm_gbps_algorithmic": gbs,
        "hbm_frac_algorithmic": gbs / HBM_PEAK_GBS,
        # the whole step (attributions + grouping + diff) against the HBM roofline,
        # at 12 B per sample and 48 B per interval
        "pipeline_roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS,
                              "unit": "GB/s", "frac": gbs / HBM_PEAK_GBS,
                              "algorithmic_bytes_per_step": bytes_step},
    }
    if CEILING:
        r["copy_ceiling"] = dict(CEILING)
        r["pipeline_roofline"]["frac_of_copy_ceiling"] = gbs / CEILING["gbps"]
    r.update(extra)
    if CEILING and "roofline" in r:
        r["roofline"]["frac_of_copy_ceiling"] = r["roofline"]["achieved"] / CEILING["gbps"]
    return r


def tile_roofline(tile_ms, n, m):
    """The dominant kernel (interval energies) against the HBM roofline, timed
    with HIP events carried on its dispatch."""
    avg = sum(tile_ms) / len(tile_ms)
    b48 = 12 * n + 48 * m  # per-unit figures of the method: samples and intervals
    b40 = 12 * n + 40 * m  # what the kernel itself moves (it does not read the keys)
    return {"kernel": "k_tile (interval energies)", "bound": "hbm",
            "achieved": b48 / (avg * 1e-3) / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": b48 / (avg * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "traffic": counters_traffic(b48),
            "traffic_source": ("rocprofv3 FETCH_SIZE + WRITE_SIZE of this kernel source, scaled "
                               "by a 1 GiB copy (profiles/tile_kernel_counters.json); null when "
                               "the source changed since or the counters were taken on another "
                               "workload"),
            "algorithmic_bytes_per_launch": b48, "avg_launch_ms": avg,
            "achieved_at_40B_per_interval": b40 / (avg * 1e-3) / 1e9,
            "frac_at_40B_per_interval": b40 / (avg * 1e-3) / 1e9 / HBM_PEAK_GBS}


def ab_bench(args, torch, mag, lib, N, synth):
    """One step = attribute A, attribute B, top-k diff.  Steps are pipelined
    `--pipeline` deep: step i is enqueued (on its own set of outputs and
    workspaces) before the host collects step i - depth + 1's results, so the
    host's wait and the short kernels at a step's end overlap the next step's
    work.  Every step's results are collected inside the timed region."""
    cfg = args.workload
    t0 = time.perf_counter()
    A, B = synth.sides(cfg, args.seed)
    log(f"[bench] generated workload {cfg} in {time.perf_counter() - t0:.1f} s")
    sh = synth.shape(cfg)
    k_cap = 8192
    top = TOPK[cfg]
    flush = None
    if cfg == 2:
        flush_buf = torch.empty(MALL_FLUSH_BYTES // 4, dtype=torch.float32, device="cuda")
        flush = lambda: flush_buf.fill_(1.0)  # noqa: E731
    # a cache flush before every step leaves nothing to overlap
    depth = 1 if flush is not None else max(1, args.pipeline)
    s1 = torch.cuda.current_stream()
    s2 = torch.cuda.Stream()  # default priority
    s3 = torch.cuda.Stream()  # default priority: B's key map
    serial = args.schedule == "serial"
    # one stream for both sides' trace integrations, the groupings on their own
    tilestream = args.schedule == "tilestream"
    # A's key map built ahead on the third stream
    a_plan = args.schedule in ("serial", "plans", "tilestream")
    g_a = torch.cuda.Stream() if tilestream else None  # default priority: A's grouping
    g_b = s2 if tilestream else None  # B's grouping and the diff
    stream_b = ctypes.c_void_p(s2.cuda_stream)
    stream_k = ctypes.c_void_p(s3.cuda_stream)
    b = ctypes.c_size_t(0)
    lib.mag_diff_workspace_size(k_cap, k_cap, top, ctypes.byref(b))
    d_bytes = int(b.value)

    class Slot:
        """One step's outputs, workspaces, events and A's stream."""

        def __init__(self, sa_stream):
            # A's calls alternate between streams, so that a step's trace
            # integration does not queue behind the previous step's grouping
            # of A (B's next trace integration waits for A's anyway)
            self.s_a = sa_stream
            self.stream_a = ctypes.c_void_p(sa_stream.cuda_stream)
            self.a_tiles = torch.cuda.Event()
            self.a_tiles.record(sa_stream)  # creates the HIP event
            self.a_done = torch.cuda.Event()
            self.a_done.record(sa_stream)
            self.b_tiles = torch.cuda.Event()
            self.b_tiles.record(s2)
            self.b_done = torch.cuda.Event()
            self.d_out = {k: torch.empty(top, dtype=dt, device="cuda") for k, dt in
                          (("key", torch.int64), ("ratio", torch.float64),
                           ("ea", torch.float64), ("eb", torch.float64),
                           ("ca", torch.int64), ("cb", torch.int64))}
            self.d_ws = torch.empty(d_bytes, dtype=torch.uint8, device="cuda")
            d = self.d_out
            self.ro = N.RankOut(d["key"].data_ptr(), d["ratio"].data_ptr(), d["ea"].data_ptr(),
                                d["eb"].data_ptr(), d["ca"].data_ptr(), d["cb"].data_ptr(), top,
                                0, 0, 0, 0)
            self.record = False

        def sides(self, prev, first):
            if tilestream:
                # the trace integrations queue on one stream, in call order
                self.sa = Side(A, lib, N, torch, k_cap, timed=args.timed_side == "a",
                               key_plan=True, inputs=first.sa if first else None,
                               group_stream=g_a)
                self.sb = Side(B, lib, N, torch, k_cap, timed=args.timed_side == "b",
                               key_plan=True, inputs=first.sb if first else None,
                               group_stream=g_b)
                return
            # the trace integrations never overlap: A's waits for the previous
            # step's B, B's for this step's A (serial schedule: A's whole call)
            self.sa = Side(A, lib, N, torch, k_cap, timed=args.timed_side == "a",
                           tiles_wait=ctypes.c_void_p(prev.b_tiles.cuda_event),
                           tiles_done=ctypes.c_void_p(self.a_tiles.cuda_event), key_plan=a_plan,
                           inputs=first.sa if first else None)
            self.sb = Side(B, lib, N, torch, k_cap, timed=args.timed_side == "b",
                           tiles_wait=ctypes.c_void_p(
                               (self.a_done if serial else self.a_tiles).cuda_event),
                           tiles_done=ctypes.c_void_p(self.b_tiles.cuda_event),
                           key_plan=True, inputs=first.sb if first else None)

    a_streams = [s1] + [torch.cuda.Stream() for _ in range(min(depth, 2) - 1 if not tilestream
                                                           else 0)]  # default priority
    slots = [Slot(a_streams[j % len(a_streams)]) for j in range(depth)]
    for j, x in enumerate(slots):
        x.sides(slots[j - 1], slots[0] if j else None)
    torch.cuda.synchronize()
    tile_ms = []

    def enqueue(x, record):
        # B's trace integration starts once A's is done (the two passes run
        # back to back, each with the device to itself), everything else of
        # each side overlaps the other; the diff reads both key counts on the
        # device, behind both attributions
        if a_plan:
            # both key maps on the third stream, A's first, ahead of A's
            # trace integration; each side's call then aggregates only (and
            # with the serial schedule B starts once A's call is complete)
            x.sa.build_plan(lib, stream_k)
        x.sa.attribute(lib, x.stream_a)
        x.a_done.record(g_a if tilestream else x.s_a)
        # B's key map depends on B's keys only: built on a third stream while
        # A's trace is integrated, so B's grouping after its own trace
        # integration only aggregates
        x.sb.build_plan(lib, stream_k)
        x.sb.attribute(lib, x.stream_a if tilestream else stream_b)
        if tilestream:
            s2.wait_event(x.a_done)
            d_stream = stream_b
        else:
            # the diff runs on A's stream of this step (idle until the step
            # after next) once B's call is complete, so that B's next trace
            # integration does not queue behind it on B's stream
            x.b_done.record(s2)
            x.s_a.wait_event(x.b_done)
            d_stream = x.stream_a
        rc = lib.mag_diff_async(x.sa.kout.data_ptr(), ctypes.byref(x.sa.ks_dev),
                                x.sb.kout.data_ptr(), ctypes.byref(x.sb.ks_dev), top,
                                ctypes.byref(x.ro), x.d_ws.data_ptr(), x.d_ws.numel(), d_stream)
        if rc != 0:
            raise RuntimeError(f"mag_diff_async failed {rc}: {lib.mag_last_error().decode()}")
        x.record = record

    def collect(x):
        # the step's results on the host: key counts, errors, the ranking's counts
        rc = lib.mag_diff_finish(x.d_ws.data_ptr(), ctypes.byref(x.ro))
        if rc != 0:
            raise RuntimeError(f"mag_diff_finish failed {rc}: {lib.mag_last_error().decode()}")
        ta = x.sa.finish(lib, x.stream_a)
        tb = x.sb.finish(lib, stream_b)
        if x.record and args.timed_side != "none":
            tile_ms.append(ta if args.timed_side == "a" else tb)

    def run(n_steps, record, depth_):
        inflight = []
        for i in range(n_steps):
            x = slots[i % depth_]
            enqueue(x, record)
            inflight.append(x)
            if len(inflight) == depth_:
                collect(inflight.pop(0))
        while inflight:
            collect(inflight.pop(0))

    run(args.warmup, False, depth)
    torch.cuda.synchronize()
    extra = {"pipeline_depth": depth}
    if flush is None:
        t0 = time.perf_counter()
        run(args.steps, True, depth)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        timing = "wall clock over the timed steps"
        if depth > 1:
            # the same steps one at a time (each collected before the next is enqueued)
            t1 = time.perf_counter()
            run(args.steps, False, 1)
            torch.cuda.synchronize()
            extra["ms_per_step_unpipelined"] = (time.perf_counter() - t1) / args.steps * 1e3
    else:
        # the cache is flushed before every step, outside the timed region
        evs = []
        x = slots[0]
        for _ in range(args.steps):
            flush()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(s1)
            s2.wait_stream(s1)
            s3.wait_stream(s1)
            enqueue(x, True)
            s1.wait_stream(s2)
            e1.record(s1)
            collect(x)
            evs.append((e0, e1))
        torch.cuda.synchronize()
        dt = sum(a.elapsed_time(b_) for a, b_ in evs) * 1e-3
        timing = "HIP events around each step; a 512 MB write flushes the Infinity Cache before it"
    sec_per_step = dt / args.steps
    x = slots[0]
    log(f"[bench] {args.steps} steps in {dt:.4f} s -> {sec_per_step * 1e3:.4f} ms/step "
        f"(pipeline depth {depth}); keys A={x.sa.ks.n_keys} B={x.sb.ks.n_keys} "
        f"joined={x.ro.n_join}" + (f"; one step at a time {extra['ms_per_step_unpipelined']:.4f} ms"
                                   if "ms_per_step_unpipelined" in extra else ""))
    extra["timing"] = timing
    if tile_ms:
        extra["roofline"] = tile_roofline(tile_ms, sh["n"], sh["m"])
    res = result_line(args, cfg, sh, 2, sec_per_step, extra)
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on both sides ...")
        res["cpu_baseline"] = cpu_baseline([A, B], [(0, 1)], "both sides of the same workload")
    print(json.dumps(res), flush=True)


def sweep_bench(args, torch, mag, lib, N, synth):
    """One step = 9 attributions (baseline + 8 candidates, alternating two
    streams, each trace integration behind the previous side's) and one
    batched top-100 diff of the 8 candidates against the baseline.  The
    candidates share the baseline's intervals and operator keys, so the step
    builds one key map (a key plan, on a third stream) for all nine
    groupings."""
    import numpy as np
    cfg = 4
    t0 = time.perf_counter()
    sides_h = synth.sides(cfg, args.seed)
    log(f"[bench] generated workload {cfg} in {time.perf_counter() - t0:.1f} s")
    sh = synth.shape(cfg)
    k_cap = 4096
    top = TOPK[cfg]
    s = [torch.cuda.current_stream(), torch.cuda.Stream()]
    # the candidates share the baseline's intervals and keys: one key map per
    # step (mag_key_plan_build, on a third stream while the first trace is
    # integrated) serves all nine groupings
    shared = all(np.array_equal(c["key"], sides_h[0]["key"]) for c in sides_h[1:])
    plan = None
    if shared:
        b = ctypes.c_size_t(0)
        m0 = int(sides_h[0]["s"].shape[0])
        assert lib.mag_key_plan_size(m0, k_cap, ctypes.byref(b)) == 0
        plan_buf = torch.empty(int(b.value), dtype=torch.uint8, device="cuda")
        plan_ready = torch.cuda.Event()
        plan_ready.record()  # creates the HIP event
        plan = N.KeyPlan(plan_buf.data_ptr(), plan_buf.numel(), 0, 0,
                         ctypes.c_void_p(plan_ready.cuda_event))
        s_k = torch.cuda.Stream()  # default priority
        handle_k = ctypes.c_void_p(s_k.cuda_stream)
    tiles = [torch.cuda.Event() for _ in sides_h]
    for ev in tiles:
        ev.record(s[0])  # creates the HIP events
    last = torch.cuda.Event()
    # each side's trace integration waits for the previous side's: the
    # bandwidth-bound passes run back to back, the rest overlaps them
    sides = [Side(c, lib, N, torch, k_cap, timed=(i == 0),
                  tiles_wait=ctypes.c_void_p(tiles[i - 1].cuda_event) if i > 0 else None,
                  tiles_done=ctypes.c_void_p(tiles[i].cuda_event), shared_plan=plan)
             for i, c in enumerate(sides_h)]
    torch.cuda.synchronize()
    handles = [ctypes.c_void_p(x.cuda_stream) for x in s]
    nb = len(sides) - 1
    b = ctypes.c_size_t(0)
    lib.mag_diff_batch_workspace_size(k_cap, nb, top, ctypes.byref(b))
    d_ws = torch.empty(int(b.value), dtype=torch.uint8, device="cuda")
    outs = (N.RankOut * nb)()
    keep = []
    for c in range(nb):
        t = [torch.empty(top, dtype=dt, device="cuda") for dt in
             (torch.int64, torch.float64, torch.float64, torch.float64, torch.int64, torch.int64)]
        keep.append(t)
        outs[c] = N.RankOut(*[x.data_ptr() for x in t], top, 0, 0, 0, 0)
    keys_b = (ctypes.c_void_p * nb)(*[x.kout.data_ptr() for x in sides[1:]])
    stats_b = (N.KeyStats * nb)(*[x.ks_dev for x in sides[1:]])
    tile_ms = []

    def step(record):
        if plan is not None:
            # the previous step is collected: the plan buffer is free again
            s_k.wait_stream(s[0])
            rc = lib.mag_key_plan_build(sides[0].key.data_ptr(), sides[0].m, k_cap,
                                        ctypes.byref(plan), handle_k)
            if rc != 0:
                raise RuntimeError(f"mag_key_plan_build failed {rc}: {lib.mag_last_error().decode()}")
        for i, side in enumerate(sides):
            side.attribute(lib, handles[i % 2])
        # the diff waits for every side's grouping: the sides on the second
        # stream are all behind this event
        last.record(s[1])
        s[0].wait_event(last)
        rc = lib.mag_diff_batch(sides[0].kout.data_ptr(), ctypes.byref(sides[0].ks_dev), nb,
                                keys_b, stats_b, top, outs, d_ws.data_ptr(), d_ws.numel(),
                                handles[0])
        if rc != 0:
            raise RuntimeError(f"mag_diff_batch failed {rc}: {lib.mag_last_error().decode()}")
        for i, side in enumerate(sides):
            t = side.finish(lib, handles[i % 2])
            if i == 0 and record:
                tile_ms.append(t)

    flush_buf = torch.empty(MALL_FLUSH_BYTES // 4, dtype=torch.float32, device="cuda")
    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    evs = []
    for _ in range(args.steps):
        flush_buf.fill_(1.0)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(s[0])
        step(True)
        e1.record(s[0])
        evs.append((e0, e1))
    torch.cuda.synchronize()
    dt = sum(a.elapsed_time(b_) for a, b_ in evs) * 1e-3
    sec_per_step = dt / args.steps
    log(f"[bench] {args.steps} steps in {dt:.4f} s -> {sec_per_step * 1e3:.4f} ms/step; "
        f"joined={[int(o.n_join) for o in outs]}")
    extra = {"timing": ("HIP events around each step; a 512 MB write flushes the Infinity Cache "
                        "before it"),
             "key_map": ("one key plan per step shared by the 9 traces (identical key arrays)"
                         if plan is not None else "one key map per trace"),
             "roofline": tile_roofline(tile_ms, sh["n"], sh["m"])}
    res = result_line(args, cfg, sh, len(sides), sec_per_step, extra)
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on the baseline and one candidate ...")
        res["cpu_baseline"] = cpu_baseline(sides_h[:2], [(0, 1)],
                                           "the baseline and candidate B1 (2 of the 9 traces)")
    print(json.dumps(res), flush=True)


def long_bench(args, torch, mag, synth):
    """Both sides of the long-run workload streamed in 32,000,000-sample
    chunks, then the top-100 diff.  Kernel-only: chunks already in HBM
    (mag_stream_push); end to end (--end-to-end): chunks in pinned host memory,
    copied over PCIe on a copy stream, double-buffered (mag_stream_push_host)."""
    import numpy as np
    cfg = 5
    t0 = time.perf_counter()
    sides_h = synth.sides(cfg, args.seed)
    log(f"[bench] generated workload {cfg} in {time.perf_counter() - t0:.1f} s")
    sh = synth.shape(cfg)
    n = sh["n"]
    chunk = 32_000_000
    sizes = [chunk] * (n // chunk) + ([n % chunk] if n % chunk else [])
    s_ = [torch.cuda.current_stream(), torch.cuda.Stream()]
    dev = []
    for c in sides_h:
        d = {"s": torch.from_numpy(c["s"]).cuda(), "e": torch.from_numpy(c["e"]).cuda(),
             "key": torch.from_numpy(np.ascontiguousarray(c["key"]).view(np.int64)).cuda()}
        if args.end_to_end:
            d["t"] = torch.from_numpy(c["t"]).pin_memory()
            d["P"] = torch.from_numpy(c["P"]).pin_memory()
        else:
            d["t"] = torch.from_numpy(c["t"]).cuda()
            d["P"] = torch.from_numpy(c["P"]).cuda()
        dev.append(d)
    torch.cuda.synchronize()

    def step():
        streams = []
        for i, d in enumerate(dev):
            with torch.cuda.stream(s_[i]):
                st = mag.Stream(n, d["s"], d["e"], d["key"], key_capacity=32768,
                                host_chunk=chunk if args.end_to_end else 0)
                pos = 0
                for k in sizes:
                    if args.end_to_end:
                        st.push_host(d["t"][pos:pos + k], d["P"][pos:pos + k])
                    else:
                        st.push(d["t"][pos:pos + k], d["P"][pos:pos + k])
                    pos += k
                streams.append(st)
        tabs = []
        for i, st in enumerate(streams):
            with torch.cuda.stream(s_[i]):
                tabs.append(st.end()[1])
        return mag.diff(tabs[0], tabs[1], TOPK[cfg])

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        d = step()
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    sec_per_step = dt / args.steps
    log(f"[bench] {args.steps} steps in {dt:.3f} s -> {sec_per_step * 1e3:.2f} ms/step; "
        f"joined={d['n_join']}")
    if args.end_to_end:
        timing = ("end to end: wall clock from pinned host chunks (PCIe H2D included, "
                  "bound by the link, not by HBM)")
        extra = {"timing": timing,
                 "h2d_gbps": 2 * 12 * n / sec_per_step / 1e9}
    else:
        extra = {"timing": "kernel-only: chunks resident in HBM, wall clock over the timed steps"}
    res = result_line(args, cfg, sh, 2, sec_per_step, extra)
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on side A ...")
        res["cpu_baseline"] = cpu_baseline(sides_h[:1], [], "side A (one of the two traces), "
                                           "unchunked")
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
