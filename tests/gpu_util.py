"""Shared helpers of the GPU parity tests: run the HIP path and the oracle on
the same seeded inputs and compare them to the stated bar."""
from __future__ import annotations

import sys

import numpy as np

import oracle

# energies: relative 1e-9 (fp64); see the design notes for the derivation of
# the M2 and ratio bounds
E_RTOL = 1e-9


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def to_gpu(c: dict):
    import torch
    d = {}
    d["t"] = torch.from_numpy(np.ascontiguousarray(c["t"], np.float64)).cuda()
    d["P"] = torch.from_numpy(np.ascontiguousarray(c["P"], np.float32)).cuda()
    d["s"] = torch.from_numpy(np.ascontiguousarray(c["s"], np.float64)).cuda()
    d["e"] = torch.from_numpy(np.ascontiguousarray(c["e"], np.float64)).cuda()
    d["key"] = torch.from_numpy(np.ascontiguousarray(c["key"], np.uint64).view(np.int64)).cuda()
    return d


def run_gpu(c: dict, equal_split=True, key_capacity=None, dev=None):
    import paper_2512_08365_amd as mag
    d = dev or to_gpu(c)
    off = [int(x) for x in c["offsets"]]
    pi, pk, summ = mag.attribute(d["t"], d["P"], d["s"], d["e"], d["key"], n_streams=len(off) - 1,
                                 stream_offsets=off, equal_split=equal_split,
                                 key_capacity=key_capacity)
    out = {k: v.cpu().numpy() for k, v in pi.items()}
    keys = {k: v.cpu().numpy() for k, v in pk.items()}
    keys["keys"] = keys["keys"].view(np.uint64)
    return out, keys, summ, pk


def run_oracle(c: dict, equal_split=True):
    r = oracle.attribute(c["t"], c["P"], c["s"], c["e"], c["offsets"], equal_split=equal_split)
    g = oracle.groupby(c["key"], r["energy"])
    return r, g


def log_error_distribution(err, want, what):
    """The relative-error distribution of one comparison (max, 99th percentile,
    median over the nonzero expected values; the largest absolute error where
    the expected value is zero), logged as an [err] line."""
    nz = want != 0
    rel = err[nz] / np.abs(want[nz])
    zmax = float(err[~nz].max()) if (~nz).any() else 0.0
    if rel.size:
        log(f"[err] {what}: n={want.size} max_rel={rel.max():.3e} "
            f"p99_rel={np.quantile(rel, 0.99):.3e} median_rel={np.median(rel):.3e} "
            f"zero_expected={int((~nz).sum())} max_abs_there={zmax:.3e}")


def assert_energy_close(got, want, what="energy"):
    got = np.asarray(got)
    want = np.asarray(want)
    assert got.shape == want.shape, what
    err = np.abs(got - want)
    bound = E_RTOL * np.abs(want)
    log_error_distribution(err, want, what)
    bad = np.nonzero(err > bound)[0]
    assert bad.size == 0, (f"{what}: {bad.size} mismatches, first {bad[:5]}: got {got[bad[:5]]} "
                           f"want {want[bad[:5]]}")


def compare_attribution(c, equal_split=True, key_capacity=None, label=""):
    log(f"[case] {label} n={c['t'].shape[0]} m={c['s'].shape[0]} streams={len(c['offsets']) - 1} "
        f"split={equal_split}")
    o, g = run_oracle(c, equal_split)
    gi, gk, summ, pk = run_gpu(c, equal_split, key_capacity)
    assert np.array_equal(gi["start_idx"], o["start_idx"]), f"{label}: start_idx"
    assert np.array_equal(gi["end_idx"], o["end_idx"]), f"{label}: end_idx"
    assert_energy_close(gi["energy"], o["energy"], f"{label}: energy")
    W = o["trace_energy"]
    assert abs(summ["trace_energy"] - W) <= 1e-12 * W, label
    assert abs(summ["idle_energy"] - o["idle_energy"]) <= E_RTOL * W, label
    assert abs(summ["attributed_energy"] - o["attributed_energy"]) <= E_RTOL * W, label
    assert summ["n_clipped"] == o["n_clipped"], label
    # per key
    assert np.array_equal(gk["keys"], g["keys"]), f"{label}: keys"
    assert np.array_equal(gk["count"], g["count"]), f"{label}: counts"
    assert_energy_close(gk["sum"], g["sum"], f"{label}: key sums")
    second = g["m2"] + g["count"] * (g["sum"] / np.maximum(g["count"], 1)) ** 2
    assert np.all(np.abs(gk["m2"] - g["m2"]) <= E_RTOL * second), f"{label}: m2"
    return o, g, gi, gk, summ, pk
