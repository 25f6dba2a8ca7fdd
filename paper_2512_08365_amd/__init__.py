"""MI355X operator energy attribution and A/B energy comparison.

Thin Python binding over libmagneton.so (C ABI in include/magneton.h).  Torch
is used only to allocate device memory and to name the current HIP stream;
every step of the computation runs in the library's HIP kernels.  There is no
CPU fallback: if the library is missing, or the device is not a GPU, the calls
raise.
"""
from __future__ import annotations

import ctypes
import functools

import torch

from . import _native as N

__all__ = ["MagnetonError", "KeyPlan", "attribute", "attribute_static", "attribute_counter", "diff", "diff_batch", "detect", "invariants",
           "match", "match_subgraphs", "Stream", "workspace_size",
           "stream_workspace_size", "diff_workspace_size", "counter_workspace_size", "version", "EQUAL_SPLIT",
           "SKIP_VALIDATE"]

EQUAL_SPLIT = N.MAG_EQUAL_SPLIT
SKIP_VALIDATE = N.MAG_SKIP_VALIDATE
ASYNC = N.MAG_ASYNC
KEY_LATENCY = N.MAG_KEY_LATENCY
WASTE = N.MAG_WASTE
TRADEOFF = N.MAG_TRADEOFF


class MagnetonError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"[{code}] {msg}")
        self.code = code


def _lib():
    return N.load()


def _check(rc: int):
    if rc != N.MAG_OK:
        lib = _lib()
        detail = lib.mag_last_error().decode() or lib.mag_strerror(rc).decode()
        raise MagnetonError(rc, detail)


def version() -> str:
    return _lib().mag_version().decode()


def _event_handle(ev):
    """Raw HIP event of a torch.cuda.Event (created by a first record if needed)."""
    if ev is None:
        return None
    if not ev.cuda_event:
        ev.record()
    return ctypes.c_void_p(ev.cuda_event)


def _opts(n_streams: int, stream_offsets, flags: int, intervals_ready=None, key_plan=None,
          tiles_wait=None, tiles_done=None, group_stream=None):
    o = N.AttrOpts()
    if group_stream is not None:
        o.group_stream = ctypes.c_void_p(group_stream.cuda_stream)
    o.n_streams = int(n_streams)
    o.flags = int(flags)
    o.intervals_ready = _event_handle(intervals_ready)
    o.tiles_wait = _event_handle(tiles_wait)
    o.tiles_done = _event_handle(tiles_done)
    if key_plan is not None:
        o.key_plan = ctypes.pointer(key_plan._kp)
    keep = None
    if stream_offsets is not None:
        keep = (ctypes.c_int64 * len(stream_offsets))(*[int(x) for x in stream_offsets])
        o.stream_offsets = ctypes.cast(keep, ctypes.c_void_p)
    return o, keep


def _dev_ptr(x, dtype, name):
    if x is None:
        return None
    if not isinstance(x, torch.Tensor) or not x.is_cuda:
        raise MagnetonError(N.MAG_E_NULL, f"{name} must be a GPU tensor")
    if x.dtype != dtype:
        raise MagnetonError(N.MAG_E_SIZE, f"{name} must be {dtype}, got {x.dtype}")
    if not x.is_contiguous():
        raise MagnetonError(N.MAG_E_SIZE, f"{name} must be contiguous")
    return x.data_ptr()


def workspace_size(n_samples: int, n_intervals: int, key_capacity: int = 0, n_streams: int = 1,
                   stream_offsets=None, flags: int = EQUAL_SPLIT, key_plan=None) -> int:
    o, keep = _opts(n_streams, stream_offsets, flags, key_plan=key_plan)
    b = ctypes.c_size_t(0)
    _check(_lib().mag_attribute_workspace_size(n_samples, n_intervals, key_capacity,
                                                ctypes.byref(o), ctypes.byref(b)))
    return int(b.value)


def diff_workspace_size(n_keys_a: int, n_keys_b: int, k: int) -> int:
    b = ctypes.c_size_t(0)
    _check(_lib().mag_diff_workspace_size(n_keys_a, n_keys_b, k, ctypes.byref(b)))
    return int(b.value)


def _key_outputs(cap: int, dev, latency: bool):
    """Device arrays of a per-key table and the KeyStats struct naming them."""
    t = {"keys": torch.empty(cap, dtype=torch.int64, device=dev),
         "sum": torch.empty(cap, dtype=torch.float64, device=dev),
         "m2": torch.empty(cap, dtype=torch.float64, device=dev),
         "count": torch.empty(cap, dtype=torch.int64, device=dev)}
    if latency:
        t["duration"] = torch.empty(cap, dtype=torch.float64, device=dev)
    ks = N.KeyStats(t["sum"].data_ptr(), t["m2"].data_ptr(), t["count"].data_ptr(), cap, 0,
                    t["duration"].data_ptr() if latency else None)
    return t, ks


def _key_rows(t: dict, ks) -> dict:
    nk = int(ks.n_keys)
    return {k: v[:nk] for k, v in t.items()}


def _stream_handle(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


class Pending:
    """An attribution enqueued with asynchronous=True; finish() waits for it and
    returns what attribute() returns (raising its errors).  The stream current
    when the call was made is the one waited for, whatever stream is current
    when finish() runs."""

    def __init__(self, workspace, ks, summ, build, keep, stream):
        self._workspace, self._ks, self._summ, self._build, self._keep = (
            workspace, ks, summ, build, keep)
        self._stream = stream
        self._result = None

    def finish(self):
        if self._result is None:
            rc = _lib().mag_attribute_finish(
                self._workspace.data_ptr(), ctypes.byref(self._ks) if self._ks else None,
                ctypes.byref(self._summ), self._stream)
            _check(rc)
            self._result = self._build()
        return self._result


def attribute(t, P, s, e, keys=None, *, n_streams: int = 1, stream_offsets=None,
              equal_split: bool = True, validate: bool = True, key_capacity: int | None = None,
              indices: bool = True, workspace=None, out=None, asynchronous: bool = False,
              intervals_ready=None, latency: bool = False, key_plan=None, tiles_wait=None,
              tiles_done=None, group_stream=None):
    """Attribute the energy of a power trace to intervals and group it by key.

    t: float64 [n] timestamps (s), P: float32 [n] power (W), s/e: float64 [m]
    interval bounds, keys: int64 [m] (bits read as uint64) or None.
    intervals_ready: a torch.cuda.Event recorded on the current stream once the
    per-interval outputs are complete (before the grouping), or None.
    key_plan: a KeyPlan of these keys (its key map is used instead of building
    one; its capacity is the key capacity).  tiles_wait / tiles_done: events
    waited for before / recorded after the trace integration.  group_stream: a
    torch.cuda.Stream that runs the fix-ups and grouping after the trace
    integration (the current stream is then free for the next call's).
    latency: also sum each key's interval durations (per_key["duration"]).
    Returns (per_interval, per_key, summary): dicts of tensors / numbers; with
    asynchronous=True a Pending whose finish() returns them once the work ran.
    """
    lib = _lib()
    n = int(t.shape[0])
    m = int(s.shape[0])
    dev = t.device
    flags = ((EQUAL_SPLIT if equal_split else 0) | (0 if validate else SKIP_VALIDATE) |
             (ASYNC if asynchronous else 0) | (KEY_LATENCY if latency and keys is not None else 0))
    o, keep = _opts(n_streams, stream_offsets, flags, intervals_ready, key_plan, tiles_wait,
                    tiles_done, group_stream)
    group = keys is not None
    cap = int(key_capacity) if key_capacity is not None else max(1, m)
    if key_plan is not None:
        cap = key_plan.key_capacity
    ws_bytes = workspace_size(n, m, cap if group else 0, n_streams, stream_offsets, flags,
                              key_plan)
    if workspace is None or workspace.numel() < ws_bytes:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    out = out or {}
    energy = out.get("energy")
    if energy is None:
        energy = torch.empty(m, dtype=torch.float64, device=dev)
    si = ei = None
    if indices:
        si = out.get("start_idx")
        ei = out.get("end_idx")
        if si is None:
            si = torch.empty(m, dtype=torch.int64, device=dev)
        if ei is None:
            ei = torch.empty(m, dtype=torch.int64, device=dev)
    pio = N.IntervalOut(_dev_ptr(energy, torch.float64, "energy"),
                        _dev_ptr(si, torch.int64, "start_idx"), _dev_ptr(ei, torch.int64, "end_idx"))
    ks = tab = None
    if group:
        tab, ks = _key_outputs(cap, dev, latency)
    summ = N.Summary()
    sh = _stream_handle(dev)
    rc = lib.mag_attribute(
        _dev_ptr(t, torch.float64, "t"), _dev_ptr(P, torch.float32, "P"), n,
        _dev_ptr(s, torch.float64, "s"), _dev_ptr(e, torch.float64, "e"),
        _dev_ptr(keys, torch.int64, "keys") if group else None, m, ctypes.byref(o),
        ctypes.byref(pio), tab["keys"].data_ptr() if group else None,
        ctypes.byref(ks) if group else None, ctypes.byref(summ), workspace.data_ptr(),
        workspace.numel(), sh)
    _check(rc)

    def build():
        per_interval = {"energy": energy}
        if indices:
            per_interval["start_idx"] = si
            per_interval["end_idx"] = ei
        per_key = _key_rows(tab, ks) if group else None
        summary = {"trace_energy": summ.trace_energy, "idle_energy": summ.idle_energy,
                   "attributed_energy": summ.attributed_energy, "n_clipped": int(summ.n_clipped),
                   "n_keys": int(summ.n_keys)}
        return per_interval, per_key, summary

    if asynchronous:
        # the inputs and the options stay referenced until finish()
        return Pending(workspace, ks, summ, build,
                       (keep, o, t, P, s, e, keys, key_plan, group_stream), sh)
    return build()


def counter_workspace_size(n_samples: int, n_intervals: int, key_capacity: int = 0,
                           flags: int = 0) -> int:
    b = ctypes.c_size_t(0)
    _check(_lib().mag_counter_workspace_size(n_samples, n_intervals, key_capacity, flags,
                                             ctypes.byref(b)))
    return int(b.value)


class KeyPlan:
    """The key map of a grouping (mag_key_plan_build): built from the
    operator keys alone, on the current stream, so it can be made while the
    power trace is integrated on another stream, or reused by several
    attributions of the same keys.  `ready`: a torch.cuda.Event recorded when
    the map is complete (attributions using the plan wait for it)."""

    def __init__(self, keys, key_capacity: int | None = None, ready=None):
        lib = _lib()
        m = int(keys.shape[0])
        cap = int(key_capacity) if key_capacity is not None else max(1, m)
        b = ctypes.c_size_t(0)
        _check(lib.mag_key_plan_size(m, cap, ctypes.byref(b)))
        self.buffer = torch.empty(int(b.value), dtype=torch.uint8, device=keys.device)
        self.keys = keys
        self.ready = ready
        self.key_capacity = cap
        self._kp = N.KeyPlan(self.buffer.data_ptr(), self.buffer.numel(), 0, 0,
                             _event_handle(ready) if ready is not None else None)
        self.rebuild()

    def rebuild(self):
        """(Re)build the map from self.keys on the current stream."""
        k = self.keys
        if self.ready is not None:
            self._kp.ready = _event_handle(self.ready)
        _check(_lib().mag_key_plan_build(_dev_ptr(k, torch.int64, "keys"), int(k.shape[0]),
                                         self.key_capacity, ctypes.byref(self._kp),
                                         _stream_handle(k.device)))


def attribute_static(t, P, s, e, keys=None, *, n_streams: int = 1, stream_offsets=None,
                     equal_split: bool = True, validate: bool = True,
                     key_capacity: int | None = None, out=None, key_out=None):
    """attribute() through mag_attribute_static: the library's own scratch
    array (MAG_STATIC_SCRATCH_BYTES per GPU) replaces the workspace and the
    call allocates nothing.  `out` / `key_out` may hold preallocated result
    tensors (energy, start_idx, end_idx / keys, sum, m2, count) so that this
    function allocates nothing either; missing ones are allocated here."""
    lib = _lib()
    n = int(t.shape[0])
    m = int(s.shape[0])
    dev = t.device
    flags = (EQUAL_SPLIT if equal_split else 0) | (0 if validate else SKIP_VALIDATE)
    o, keep = _opts(n_streams, stream_offsets, flags)
    group = keys is not None
    cap = int(key_capacity) if key_capacity is not None else max(1, m)
    out = dict(out or {})
    for name, dt in (("energy", torch.float64), ("start_idx", torch.int64),
                     ("end_idx", torch.int64)):
        if out.get(name) is None:
            out[name] = torch.empty(m, dtype=dt, device=dev)
    pio = N.IntervalOut(_dev_ptr(out["energy"], torch.float64, "energy"),
                        _dev_ptr(out["start_idx"], torch.int64, "start_idx"),
                        _dev_ptr(out["end_idx"], torch.int64, "end_idx"))
    tab = ks = None
    if group:
        tab = dict(key_out or {})
        for name, dt in (("keys", torch.int64), ("sum", torch.float64), ("m2", torch.float64),
                         ("count", torch.int64)):
            if tab.get(name) is None:
                tab[name] = torch.empty(cap, dtype=dt, device=dev)
        ks = N.KeyStats(tab["sum"].data_ptr(), tab["m2"].data_ptr(), tab["count"].data_ptr(), cap,
                        0, None)
    summ = N.Summary()
    _check(lib.mag_attribute_static(
        _dev_ptr(t, torch.float64, "t"), _dev_ptr(P, torch.float32, "P"), n,
        _dev_ptr(s, torch.float64, "s"), _dev_ptr(e, torch.float64, "e"),
        _dev_ptr(keys, torch.int64, "keys") if group else None, m, ctypes.byref(o),
        ctypes.byref(pio), tab["keys"].data_ptr() if group else None,
        ctypes.byref(ks) if group else None, ctypes.byref(summ), _stream_handle(dev)))
    per_key = _key_rows(tab, ks) if group else None
    summary = {"trace_energy": summ.trace_energy, "idle_energy": summ.idle_energy,
               "attributed_energy": summ.attributed_energy, "n_clipped": int(summ.n_clipped),
               "n_keys": int(summ.n_keys)}
    return out, per_key, summary


def attribute_counter(t, C, s, e, keys=None, *, delay: float = 0.0, replays=None,
                      validate: bool = True, key_capacity: int | None = None,
                      indices: bool = True, workspace=None, out=None, time_kernels: bool = False,
                      latency: bool = False, asynchronous: bool = False):
    """Per-operator energy from a cumulative energy counter (software replay mode).

    t: float64 [n] reading times (s), C: float64 [n] cumulative energy (J),
    delay: seconds by which the counter lags (a reading at t holds the energy
    used up to t - delay), s/e: float64 [m] replay windows (one sequence),
    replays: int32 [m] runs per window or None, keys: int64 [m] or None.
    Returns (per_interval, per_key, summary) as attribute() does; the energies
    are per run (the window's counter increase over its replay count).  With
    asynchronous=True a Pending whose finish() returns them once the work ran.
    """
    lib = _lib()
    n = int(t.shape[0])
    m = int(s.shape[0])
    dev = t.device
    group = keys is not None
    flags = ((0 if validate else SKIP_VALIDATE) | (N.MAG_TIME_KERNELS if time_kernels else 0) |
             (KEY_LATENCY if latency and group else 0) | (ASYNC if asynchronous else 0))
    cap = int(key_capacity) if key_capacity is not None else max(1, m)
    ws_bytes = counter_workspace_size(n, m, cap if group else 0, flags)
    if workspace is None or workspace.numel() < ws_bytes:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    out = out or {}
    energy = out.get("energy")
    if energy is None:
        energy = torch.empty(m, dtype=torch.float64, device=dev)
    si = ei = None
    if indices:
        si = out.get("start_idx")
        ei = out.get("end_idx")
        if si is None:
            si = torch.empty(m, dtype=torch.int64, device=dev)
        if ei is None:
            ei = torch.empty(m, dtype=torch.int64, device=dev)
    pio = N.IntervalOut(_dev_ptr(energy, torch.float64, "energy"),
                        _dev_ptr(si, torch.int64, "start_idx"), _dev_ptr(ei, torch.int64, "end_idx"))
    ks = tab = None
    if group:
        tab, ks = _key_outputs(cap, dev, latency)
    summ = N.Summary()
    sh = _stream_handle(dev)
    rc = lib.mag_attribute_counter(
        _dev_ptr(t, torch.float64, "t"), _dev_ptr(C, torch.float64, "C"), n, float(delay),
        _dev_ptr(s, torch.float64, "s"), _dev_ptr(e, torch.float64, "e"),
        _dev_ptr(replays, torch.int32, "replays"),
        _dev_ptr(keys, torch.int64, "keys") if group else None, m, flags, ctypes.byref(pio),
        tab["keys"].data_ptr() if group else None, ctypes.byref(ks) if group else None,
        ctypes.byref(summ), workspace.data_ptr(), workspace.numel(), sh)
    _check(rc)

    def build():
        per_interval = {"energy": energy}
        if indices:
            per_interval["start_idx"] = si
            per_interval["end_idx"] = ei
        per_key = _key_rows(tab, ks) if group else None
        summary = {"trace_energy": summ.trace_energy, "idle_energy": summ.idle_energy,
                   "attributed_energy": summ.attributed_energy, "n_clipped": int(summ.n_clipped),
                   "n_keys": int(summ.n_keys), "kernel_ms": summ.tile_kernel_ms,
                   "device_ms": summ.device_ms}
        return per_interval, per_key, summary

    if asynchronous:
        return Pending(workspace, ks, summ, build, (t, C, s, e, keys, replays), sh)
    return build()


def diff(a: dict, b: dict, k: int, workspace=None, asynchronous: bool = False):
    """Rank keys present in both per-key tables by (E_B - E_A)/E_A (descending,
    ties by ascending key).  a/b: per-key dicts as returned by attribute().
    asynchronous: enqueue only (mag_diff_async) and return a PendingDiff whose
    result() waits (mag_diff_finish) and returns what diff() returns."""
    lib = _lib()
    dev = a["keys"].device
    na, nb = int(a["keys"].shape[0]), int(b["keys"].shape[0])
    ws_bytes = diff_workspace_size(na, nb, k)
    if workspace is None or workspace.numel() < ws_bytes:
        workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    cap = max(1, min(int(k), na))
    key = torch.empty(cap, dtype=torch.int64, device=dev)
    ratio = torch.empty(cap, dtype=torch.float64, device=dev)
    ea = torch.empty(cap, dtype=torch.float64, device=dev)
    eb = torch.empty(cap, dtype=torch.float64, device=dev)
    ca = torch.empty(cap, dtype=torch.int64, device=dev)
    cb = torch.empty(cap, dtype=torch.int64, device=dev)
    sa = N.KeyStats(_dev_ptr(a["sum"], torch.float64, "a.sum"), a["m2"].data_ptr() if "m2" in a else None,
                    _dev_ptr(a["count"], torch.int64, "a.count"), na, na)
    sb = N.KeyStats(_dev_ptr(b["sum"], torch.float64, "b.sum"), b["m2"].data_ptr() if "m2" in b else None,
                    _dev_ptr(b["count"], torch.int64, "b.count"), nb, nb)
    ro = N.RankOut(key.data_ptr(), ratio.data_ptr(), ea.data_ptr(), eb.data_ptr(), ca.data_ptr(),
                   cb.data_ptr(), cap, 0, 0, 0, 0)
    call = lib.mag_diff_async if asynchronous else lib.mag_diff
    rc = call(_dev_ptr(a["keys"], torch.int64, "a.keys"), ctypes.byref(sa),
              _dev_ptr(b["keys"], torch.int64, "b.keys"), ctypes.byref(sb), int(k),
              ctypes.byref(ro), workspace.data_ptr(), workspace.numel(), _stream_handle(dev))
    _check(rc)

    def collect():
        r = int(ro.n_out)
        return {"key": key[:r], "ratio": ratio[:r], "energy_a": ea[:r], "energy_b": eb[:r],
                "count_a": ca[:r], "count_b": cb[:r], "n_only_a": int(ro.n_only_a),
                "n_only_b": int(ro.n_only_b), "n_join": int(ro.n_join)}

    if not asynchronous:
        return collect()
    # the input tables stay referenced until result()
    return PendingDiff(lib, workspace, ro, collect, (a, b))


class PendingDiff:
    """An enqueued comparison (diff(..., asynchronous=True)); result() waits
    for it once (mag_diff_finish) and returns the ranking."""

    def __init__(self, lib, workspace, ro, collect, keep=None):
        self._lib, self._ws, self._ro, self._collect = lib, workspace, ro, collect
        self._keep = keep
        self._done = None

    def result(self) -> dict:
        if self._done is None:
            _check(self._lib.mag_diff_finish(self._ws.data_ptr(), ctypes.byref(self._ro)))
            self._done = self._collect()
            self._keep = None
        return self._done


def diff_batch(a: dict, bs: list, k: int, workspace=None) -> list:
    """diff(a, b, k) for every per-key table b in bs, in one library call
    (mag_diff_batch: a fixed number of launches per 8 candidates, one
    synchronization)."""
    lib = _lib()
    dev = a["keys"].device
    n = len(bs)
    na = int(a["keys"].shape[0])
    b_ws = ctypes.c_size_t(0)
    _check(lib.mag_diff_batch_workspace_size(na, n, int(k), ctypes.byref(b_ws)))
    if workspace is None or workspace.numel() < int(b_ws.value):
        workspace = torch.empty(max(1, int(b_ws.value)), dtype=torch.uint8, device=dev)
    cap = max(1, min(int(k), na))
    sa = N.KeyStats(_dev_ptr(a["sum"], torch.float64, "a.sum"), None,
                    _dev_ptr(a["count"], torch.int64, "a.count"), na, na)
    keys_b = (ctypes.c_void_p * max(n, 1))()
    stats_b = (N.KeyStats * max(n, 1))()
    outs = (N.RankOut * max(n, 1))()
    tens = []
    for c, b in enumerate(bs):
        nb = int(b["keys"].shape[0])
        keys_b[c] = _dev_ptr(b["keys"], torch.int64, "b.keys")
        stats_b[c] = N.KeyStats(_dev_ptr(b["sum"], torch.float64, "b.sum"), None,
                                _dev_ptr(b["count"], torch.int64, "b.count"), nb, nb)
        t = {"key": torch.empty(cap, dtype=torch.int64, device=dev),
             "ratio": torch.empty(cap, dtype=torch.float64, device=dev),
             "energy_a": torch.empty(cap, dtype=torch.float64, device=dev),
             "energy_b": torch.empty(cap, dtype=torch.float64, device=dev),
             "count_a": torch.empty(cap, dtype=torch.int64, device=dev),
             "count_b": torch.empty(cap, dtype=torch.int64, device=dev)}
        outs[c] = N.RankOut(t["key"].data_ptr(), t["ratio"].data_ptr(), t["energy_a"].data_ptr(),
                            t["energy_b"].data_ptr(), t["count_a"].data_ptr(),
                            t["count_b"].data_ptr(), cap, 0, 0, 0, 0)
        tens.append(t)
    _check(lib.mag_diff_batch(_dev_ptr(a["keys"], torch.int64, "a.keys"), ctypes.byref(sa), n,
                              keys_b, stats_b, int(k), outs, workspace.data_ptr(),
                              workspace.numel(), _stream_handle(dev)))
    res = []
    for c, t in enumerate(tens):
        r = int(outs[c].n_out)
        d = {kk: v[:r] for kk, v in t.items()}
        d.update(n_only_a=int(outs[c].n_only_a), n_only_b=int(outs[c].n_only_b),
                 n_join=int(outs[c].n_join))
        res.append(d)
    return res


def detect(a: dict, b: dict, threshold: float = 0.10, tolerance: float = 0.01,
           rows: int | None = None, workspace=None):
    """Section 6.1's detection over two per-key tables from attribute(...,
    latency=True): keys with (E_B - E_A)/E_A >= threshold, in ranking order,
    with their latencies and a verdict (WASTE when A is at most `tolerance`
    slower than B, else TRADEOFF).  rows: how many flagged keys to return
    (default: all keys of A)."""
    lib = _lib()
    dev = a["keys"].device
    na, nb = int(a["keys"].shape[0]), int(b["keys"].shape[0])
    cap = max(1, int(rows) if rows is not None else na)
    b_ws = ctypes.c_size_t(0)
    _check(lib.mag_detect_workspace_size(na, nb, cap, ctypes.byref(b_ws)))
    if workspace is None or workspace.numel() < int(b_ws.value):
        workspace = torch.empty(int(b_ws.value), dtype=torch.uint8, device=dev)
    o = {k: torch.empty(cap, dtype=dt, device=dev) for k, dt in
         (("key", torch.int64), ("ratio", torch.float64), ("energy_a", torch.float64),
          ("energy_b", torch.float64), ("count_a", torch.int64), ("count_b", torch.int64),
          ("latency_a", torch.float64), ("latency_b", torch.float64), ("verdict", torch.int32))}

    def stats(t, n, name):
        return N.KeyStats(_dev_ptr(t["sum"], torch.float64, f"{name}.sum"),
                          t["m2"].data_ptr() if "m2" in t else None,
                          _dev_ptr(t["count"], torch.int64, f"{name}.count"), n, n,
                          _dev_ptr(t.get("duration"), torch.float64, f"{name}.duration"))

    sa, sb = stats(a, na, "a"), stats(b, nb, "b")
    out = N.DetectOut()
    out.rank = N.RankOut(o["key"].data_ptr(), o["ratio"].data_ptr(), o["energy_a"].data_ptr(),
                         o["energy_b"].data_ptr(), o["count_a"].data_ptr(),
                         o["count_b"].data_ptr(), cap, 0, 0, 0, 0)
    out.latency_a = o["latency_a"].data_ptr()
    out.latency_b = o["latency_b"].data_ptr()
    out.verdict = o["verdict"].data_ptr()
    opts = N.DetectOpts(float(threshold), float(tolerance))
    _check(lib.mag_detect(_dev_ptr(a["keys"], torch.int64, "a.keys"), ctypes.byref(sa),
                          _dev_ptr(b["keys"], torch.int64, "b.keys"), ctypes.byref(sb),
                          ctypes.byref(opts), ctypes.byref(out), workspace.data_ptr(),
                          workspace.numel(), _stream_handle(dev)))
    r = int(out.rank.n_out)
    res = {k: v[:r] for k, v in o.items()}
    res.update(n_flagged=int(out.n_flagged), n_waste=int(out.n_waste),
               n_tradeoff=int(out.n_tradeoff), n_join=int(out.rank.n_join))
    return res


def _tensor_descs(tensors):
    arr = (N.Tensor * max(1, len(tensors)))()
    for i, x in enumerate(tensors):
        shape = tuple(x.shape)
        if len(shape) < 1 or len(shape) > N.MAG_SVD_MAX_RANK:
            raise MagnetonError(N.MAG_E_SIZE, f"tensor {i}: rank {len(shape)} out of range")
        arr[i].data = _dev_ptr(x, torch.float32, f"tensor {i}")
        arr[i].rank = len(shape)
        arr[i].dims[:len(shape)] = shape
    return arr


@functools.lru_cache(maxsize=4096)
def _layout_of_shape(shape: tuple) -> tuple:
    r = len(shape)
    out = []
    for g in range(1, (1 << r) - 1, 2):
        M = N_ = 1
        for i, n in enumerate(shape):
            if g >> i & 1:
                M *= int(n)
            else:
                N_ *= int(n)
        out.append(min(M, N_))
    return tuple(out)


def invariant_layout(tensor) -> list:
    """Lengths of a tensor's spectra, in the order invariants() writes them."""
    return list(_layout_of_shape(tuple(tensor.shape)))


def invariants(tensors, workspace=None):
    """Multi-mode SVD invariants (Section 4.2) of fp32 GPU tensors (rank 1-5):
    one fp64 tensor holding each tensor's spectra back to back (unfoldings in
    increasing bit-mask order of G, mode 0 always in G, values descending),
    and per tensor the list of spectrum lengths."""
    lib = _lib()
    tensors = list(tensors)
    descs = _tensor_descs(tensors)
    n = len(tensors)
    dev = tensors[0].device if n else torch.device("cuda")
    # (the library checks every tensor again while planning the workspace)
    layouts = [_layout_of_shape(tuple(x.shape)) for x in tensors]
    total = sum(sum(lay) for lay in layouts)
    b = ctypes.c_size_t(0)
    _check(lib.mag_invariants_workspace_size(descs, n, ctypes.byref(b)))
    if workspace is None or workspace.numel() < int(b.value):
        workspace = torch.empty(int(b.value), dtype=torch.uint8, device=dev)
    spectra = torch.empty(max(total, 1), dtype=torch.float64, device=dev)
    _check(lib.mag_invariants(descs, n, spectra.data_ptr(), workspace.data_ptr(), workspace.numel(),
                              _stream_handle(dev)))
    return spectra[:total], [list(lay) for lay in layouts]


def match(tensors_a, spectra_a, tensors_b, spectra_b, eps: float = 1e-5):
    """Which tensors of A are equivalent to which of B: a uint8 [len(A), len(B)]
    GPU tensor, 1 where the invariant lists pair up within eps x the leading
    singular value."""
    lib = _lib()
    ta, tb = list(tensors_a), list(tensors_b)
    da, db = _tensor_descs(ta), _tensor_descs(tb)
    dev = spectra_a.device
    out = torch.zeros((len(ta), len(tb)), dtype=torch.uint8, device=dev)
    b = ctypes.c_size_t(0)
    _check(lib.mag_match_workspace_size(len(ta), len(tb), ctypes.byref(b)))
    ws = torch.empty(max(int(b.value), 1), dtype=torch.uint8, device=dev)
    _check(lib.mag_match(da, len(ta), _dev_ptr(spectra_a, torch.float64, "spectra_a"), db, len(tb),
                         _dev_ptr(spectra_b, torch.float64, "spectra_b"), float(eps),
                         out.data_ptr(), ws.data_ptr(), ws.numel(), _stream_handle(dev)))
    return out


def match_subgraphs(n1: int, edges1, n2: int, edges2, eq):
    """Section 4.2's topology-aware matching of two computational graphs (host
    code): edges as (src, dst) node pairs, node 0 the input and node n-1 the
    output of each graph; eq: (node of graph 1, node of graph 2) pairs with
    equivalent outputs.  Returns the finest matched pairs as ((entry1, exit1),
    (entry2, exit2)), in path order."""
    import numpy as np
    lib = _lib()
    e1 = np.ascontiguousarray(np.asarray(edges1, np.int32).reshape(-1, 2))
    e2 = np.ascontiguousarray(np.asarray(edges2, np.int32).reshape(-1, 2))
    q = np.ascontiguousarray(np.asarray(eq, np.int32).reshape(-1, 2))
    s1, d1 = np.ascontiguousarray(e1[:, 0]), np.ascontiguousarray(e1[:, 1])
    s2, d2 = np.ascontiguousarray(e2[:, 0]), np.ascontiguousarray(e2[:, 1])
    g1 = N.GraphDesc(int(n1), len(e1), s1.ctypes.data, d1.ctypes.data)
    g2 = N.GraphDesc(int(n2), len(e2), s2.ctypes.data, d2.ctypes.data)
    cap = max(n1, n2)
    out = np.zeros(4 * cap, np.int32)
    n_out = ctypes.c_int32(0)
    _check(lib.mag_match_subgraphs(ctypes.byref(g1), ctypes.byref(g2), q.ctypes.data, len(q),
                                   out.ctypes.data, cap, ctypes.byref(n_out)))
    r = out[:4 * n_out.value].reshape(-1, 4)
    return [((int(a), int(b)), (int(c), int(d))) for a, b, c, d in r]


def stream_workspace_size(max_samples: int, n_intervals: int, key_capacity: int = 0,
                          n_streams: int = 1, stream_offsets=None, flags: int = EQUAL_SPLIT) -> int:
    o, keep = _opts(n_streams, stream_offsets, flags)
    b = ctypes.c_size_t(0)
    _check(_lib().mag_stream_workspace_size(max_samples, n_intervals, key_capacity,
                                             ctypes.byref(o), ctypes.byref(b)))
    return int(b.value)


class Stream:
    """Chunked attribution of a trace that arrives in pieces.

    The intervals (and keys) are given up front; push() hands over the next
    chunk of samples; end() returns what attribute() returns for the whole
    trace.  Chunks are read asynchronously on the current stream: keep them
    alive and unchanged until later work on that stream (this object keeps a
    reference to each chunk until end()).
    """

    def __init__(self, max_samples: int, s, e, keys=None, *, n_streams: int = 1,
                 stream_offsets=None, equal_split: bool = True, validate: bool = True,
                 key_capacity: int | None = None, indices: bool = True, latency: bool = False,
                 host_chunk: int = 0):
        lib = _lib()
        m = int(s.shape[0])
        dev = s.device
        self._dev = dev
        self._lat = latency and keys is not None
        flags = ((EQUAL_SPLIT if equal_split else 0) | (0 if validate else SKIP_VALIDATE) |
                 (KEY_LATENCY if self._lat else 0))
        self._o, self._keep = _opts(n_streams, stream_offsets, flags)
        self._group = keys is not None
        self._cap = (int(key_capacity) if key_capacity is not None else max(1, m)) if self._group else 0
        ws = stream_workspace_size(max_samples, m, self._cap, n_streams, stream_offsets, flags)
        self._ws = torch.empty(ws, dtype=torch.uint8, device=dev)
        self.energy = torch.empty(m, dtype=torch.float64, device=dev)
        self.start_idx = torch.empty(m, dtype=torch.int64, device=dev) if indices else None
        self.end_idx = torch.empty(m, dtype=torch.int64, device=dev) if indices else None
        self._pio = N.IntervalOut(self.energy.data_ptr(),
                                  self.start_idx.data_ptr() if indices else None,
                                  self.end_idx.data_ptr() if indices else None)
        self._inputs = (s, e, keys)
        self._chunks = []
        h = ctypes.c_void_p(None)
        _check(lib.mag_stream_begin(
            ctypes.byref(h), int(max_samples), _dev_ptr(s, torch.float64, "s"),
            _dev_ptr(e, torch.float64, "e"),
            _dev_ptr(keys, torch.int64, "keys") if self._group else None, m, ctypes.byref(self._o),
            ctypes.byref(self._pio), self._cap, self._ws.data_ptr(), self._ws.numel(),
            _stream_handle(dev)))
        self._h = h
        self._staging = self._copy_stream = None
        if host_chunk:
            # two device halves filled from host memory on a copy stream of
            # the default priority, while the compute stream runs the tiles
            b = ctypes.c_size_t(0)
            _check(lib.mag_stream_host_staging_size(int(host_chunk), ctypes.byref(b)))
            self._staging = torch.empty(int(b.value), dtype=torch.uint8, device=dev)
            self._copy_stream = torch.cuda.Stream(dev)
            rc = lib.mag_stream_set_host_staging(
                h, int(host_chunk), self._staging.data_ptr(), self._staging.numel(),
                ctypes.c_void_p(self._copy_stream.cuda_stream))
            if rc != N.MAG_OK:
                self.abort()
                _check(rc)

    def _handle(self):
        if self._h is None or not self._h.value:
            raise MagnetonError(N.MAG_E_STATE, "stream already ended")
        return self._h

    def push(self, t, P):
        h = self._handle()
        n = int(t.shape[0])
        if int(P.shape[0]) != n:
            raise MagnetonError(N.MAG_E_SIZE, "t and P differ in length")
        self._chunks.append((t, P))
        _check(_lib().mag_stream_push(h, _dev_ptr(t, torch.float64, "t"),
                                      _dev_ptr(P, torch.float32, "P"), n))

    def push_host(self, t, P):
        """The next chunk from host memory (CPU tensors, pinned for asynchronous
        copies): float64 t and float32 P, at most host_chunk samples."""
        h = self._handle()
        n = int(t.shape[0])
        if int(P.shape[0]) != n:
            raise MagnetonError(N.MAG_E_SIZE, "t and P differ in length")
        for x, dt, name in ((t, torch.float64, "t"), (P, torch.float32, "P")):
            if not isinstance(x, torch.Tensor) or x.is_cuda:
                raise MagnetonError(N.MAG_E_NULL, f"{name} must be a CPU tensor")
            if x.dtype != dt or not x.is_contiguous():
                raise MagnetonError(N.MAG_E_SIZE, f"{name} must be contiguous {dt}")
        self._chunks.append((t, P))
        _check(_lib().mag_stream_push_host(h, t.data_ptr(), P.data_ptr(), n))

    def export_state(self) -> bytes:
        h = self._handle()
        lib = _lib()
        b = ctypes.c_size_t(0)
        _check(lib.mag_stream_state_export(h, None, ctypes.byref(b)))
        buf = ctypes.create_string_buffer(int(b.value))
        _check(lib.mag_stream_state_export(h, buf, ctypes.byref(b)))
        return buf.raw[:int(b.value)]

    def import_state(self, state: bytes):
        h = self._handle()
        buf = ctypes.create_string_buffer(state, len(state))
        _check(_lib().mag_stream_state_import(h, buf, len(state)))

    def abort(self):
        if self._h is not None and self._h.value:
            _lib().mag_stream_abort(self._h)
        self._h = None
        if getattr(self, "_copy_stream", None) is not None:
            # copies may still be landing in the staging buffer
            self._copy_stream.synchronize()
        self._chunks = []

    def end(self):
        h = self._handle()
        self._h = None
        dev = self._dev
        cap = self._cap
        ks = tab = None
        if self._group:
            tab, ks = _key_outputs(cap, dev, self._lat)
        summ = N.Summary()
        rc = _lib().mag_stream_end(h, tab["keys"].data_ptr() if self._group else None,
                                   ctypes.byref(ks) if self._group else None, ctypes.byref(summ))
        self._chunks = []
        _check(rc)
        per_interval = {"energy": self.energy}
        if self.start_idx is not None:
            per_interval["start_idx"] = self.start_idx
            per_interval["end_idx"] = self.end_idx
        per_key = _key_rows(tab, ks) if self._group else None
        summary = {"trace_energy": summ.trace_energy, "idle_energy": summ.idle_energy,
                   "attributed_energy": summ.attributed_energy, "n_clipped": int(summ.n_clipped),
                   "n_keys": int(summ.n_keys)}
        return per_interval, per_key, summary

    def __del__(self):
        try:
            self.abort()
        except Exception:
            pass
