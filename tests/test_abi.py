"""The C-ABI library: it loads, exports every symbol include/*.h declares, and
rejects bad arguments on the host before any device work (no GPU needed)."""
import ctypes
import glob
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        text = open(h).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        for mt in re.finditer(r"^[A-Za-z_][\w\s\*]*?\b(mag_\w+)\s*\(", text, flags=re.M):
            names.add(mt.group(1))
    return names


def test_header_declares_the_entry_points():
    names = _declared()
    assert {"mag_attribute", "mag_diff", "mag_attribute_workspace_size",
            "mag_diff_workspace_size", "mag_stream_workspace_size", "mag_stream_begin",
            "mag_stream_push", "mag_stream_end", "mag_stream_abort", "mag_stream_state_export",
            "mag_stream_state_import", "mag_strerror", "mag_last_error"} <= names


def test_library_exports_every_declared_symbol():
    from paper_2512_08365_amd import _native
    lib = _native.load()
    for name in _declared():
        assert hasattr(lib, name), name
    assert set(_native.EXPORTED) == _declared()


def test_host_side_errors_without_gpu():
    from paper_2512_08365_amd import _native as N
    lib = N.load()
    b = ctypes.c_size_t(0)
    assert lib.mag_attribute_workspace_size(1, 0, 0, None, ctypes.byref(b)) == N.MAG_E_SIZE
    assert lib.mag_attribute_workspace_size(10, -1, 0, None, ctypes.byref(b)) == N.MAG_E_SIZE
    assert lib.mag_attribute_workspace_size(10, 5, 0, None, None) == N.MAG_E_NULL
    assert lib.mag_attribute_workspace_size((1 << 40) + 1, 0, 0, None, ctypes.byref(b)) == N.MAG_E_SIZE
    o = N.AttrOpts(2, N.MAG_EQUAL_SPLIT, None)
    assert lib.mag_attribute_workspace_size(10, 5, 0, ctypes.byref(o), ctypes.byref(b)) == N.MAG_E_STREAMS
    offs = (ctypes.c_int64 * 3)(0, 4, 3)
    o = N.AttrOpts(2, N.MAG_EQUAL_SPLIT, ctypes.cast(offs, ctypes.c_void_p))
    assert lib.mag_attribute_workspace_size(10, 3, 0, ctypes.byref(o), ctypes.byref(b)) == N.MAG_E_STREAMS
    o = N.AttrOpts(33, N.MAG_EQUAL_SPLIT, None)
    assert lib.mag_attribute_workspace_size(10, 3, 0, ctypes.byref(o), ctypes.byref(b)) == N.MAG_E_STREAMS
    assert lib.mag_attribute_workspace_size(10, 3, 8, None, ctypes.byref(b)) == N.MAG_OK
    assert b.value > 0
    # NULL inputs and bad sizes are rejected before any HIP call
    assert lib.mag_attribute(None, None, 10, None, None, None, 0, None, None, None, None, None,
                             None, 0, None) == N.MAG_E_NULL
    fake = ctypes.c_void_p(256)
    assert lib.mag_attribute(fake, fake, 1, None, None, None, 0, None, None, None, None, None,
                             fake, 0, None) == N.MAG_E_SIZE
    assert lib.mag_attribute(fake, fake, 10, None, None, None, 3, None, None, None, None, None,
                             fake, 0, None) == N.MAG_E_NULL
    assert lib.mag_attribute(fake, fake, 10, fake, fake, None, 3, None, None, None, None, None,
                             fake, 0, None) == N.MAG_E_WORKSPACE
    assert b"workspace" in lib.mag_last_error()
    ks = N.KeyStats(None, None, None, 0, 0)
    assert lib.mag_attribute(fake, fake, 10, fake, fake, fake, 3, None, None, None,
                             ctypes.byref(ks), None, fake, 1 << 30, None) == N.MAG_E_SIZE
    assert lib.mag_diff(None, None, None, None, 3, None, None, 0, None) == N.MAG_E_NULL
    sa = N.KeyStats(None, None, None, 0, 0)
    ro = N.RankOut()
    assert lib.mag_diff(None, ctypes.byref(sa), None, ctypes.byref(sa), -1, ctypes.byref(ro),
                        None, 0, None) == N.MAG_E_SIZE
    assert lib.mag_diff_workspace_size(5, 5, -1, ctypes.byref(b)) == N.MAG_E_SIZE
    for code in range(-13, 1):
        assert b"unknown" not in lib.mag_strerror(code)


def test_counter_host_side_errors_without_gpu():
    from paper_2512_08365_amd import _native as N
    lib = N.load()
    b = ctypes.c_size_t(0)
    assert lib.mag_counter_workspace_size(1, 0, 0, 0, ctypes.byref(b)) == N.MAG_E_SIZE
    assert lib.mag_counter_workspace_size(10, -1, 0, 0, ctypes.byref(b)) == N.MAG_E_SIZE
    assert lib.mag_counter_workspace_size(10, 5, -1, 0, ctypes.byref(b)) == N.MAG_E_SIZE
    assert lib.mag_counter_workspace_size(10, 5, 0, 0, None) == N.MAG_E_NULL
    assert lib.mag_counter_workspace_size(10, 500, 0, 0, ctypes.byref(b)) == N.MAG_OK
    plain = b.value
    assert lib.mag_counter_workspace_size(10, 500, 64, 0, ctypes.byref(b)) == N.MAG_OK
    grouped = b.value
    assert grouped > plain  # the group-by state
    assert lib.mag_counter_workspace_size(10, 500, 64, N.MAG_KEY_LATENCY, ctypes.byref(b)) == 0
    assert b.value > grouped  # the per-chunk latency rows
    fake = ctypes.c_void_p(256)
    big = 1 << 30

    def call(t=fake, C=fake, n=10, delay=0.0, s=fake, e=fake, reps=None, keys=None, m=3,
             ws=fake, ws_bytes=big):
        return lib.mag_attribute_counter(t, C, n, delay, s, e, reps, keys, m, 0, None, None,
                                         None, None, ws, ws_bytes, None)

    assert call(t=None) == N.MAG_E_NULL
    assert call(C=None) == N.MAG_E_NULL
    assert call(delay=float("inf")) == N.MAG_E_TIMESTAMPS
    assert call(delay=float("nan")) == N.MAG_E_TIMESTAMPS
    assert call(n=1) == N.MAG_E_SIZE
    assert call(m=-1) == N.MAG_E_SIZE
    assert call(s=None) == N.MAG_E_NULL
    assert call(ws=None) == N.MAG_E_NULL
    assert call(ws=ctypes.c_void_p(264)) == N.MAG_E_WORKSPACE
    assert call(t=ctypes.c_void_p(260)) == N.MAG_E_ALIGN
    assert call(reps=ctypes.c_void_p(258)) == N.MAG_E_ALIGN
    assert call(ws_bytes=16) == N.MAG_E_WORKSPACE
    assert b"workspace" in lib.mag_last_error()


def test_latency_and_detect_host_side_errors_without_gpu():
    from paper_2512_08365_amd import _native as N
    lib = N.load()
    b = ctypes.c_size_t(0)
    assert lib.mag_attribute_workspace_size(10_000, 3, 8, None, ctypes.byref(b)) == N.MAG_OK
    plain = b.value
    o = N.AttrOpts(1, N.MAG_EQUAL_SPLIT | N.MAG_KEY_LATENCY, None)
    assert lib.mag_attribute_workspace_size(10_000, 3, 8, ctypes.byref(o), ctypes.byref(b)) == 0
    assert b.value > plain
    fake = ctypes.c_void_p(256)
    # MAG_KEY_LATENCY needs the per-key duration array
    ks = N.KeyStats(fake, fake, fake, 8, 0, None)
    assert lib.mag_attribute(fake, fake, 10, fake, fake, fake, 3, ctypes.byref(o), None, fake,
                             ctypes.byref(ks), None, fake, 1 << 30, None) == N.MAG_E_NULL
    assert b"duration" in lib.mag_last_error()
    ks.duration = ctypes.c_void_p(260)
    assert lib.mag_attribute(fake, fake, 10, fake, fake, fake, 3, ctypes.byref(o), None, fake,
                             ctypes.byref(ks), None, fake, 1 << 30, None) == N.MAG_E_ALIGN
    # detect: durations required on both sides, thresholds must be numbers
    sa = N.KeyStats(fake, None, fake, 5, 5, None)
    sb = N.KeyStats(fake, None, fake, 5, 5, fake)
    out = N.DetectOut()
    out.rank = N.RankOut(fake, fake, fake, fake, fake, fake, 5, 0, 0, 0, 0)
    out.latency_a = out.latency_b = out.verdict = fake
    assert lib.mag_detect(fake, ctypes.byref(sa), fake, ctypes.byref(sb), None, ctypes.byref(out),
                          fake, 1 << 20, None) == N.MAG_E_NULL
    sa.duration = fake
    nan = N.DetectOpts(float("nan"), 0.01)
    assert lib.mag_detect(fake, ctypes.byref(sa), fake, ctypes.byref(sb), ctypes.byref(nan),
                          ctypes.byref(out), fake, 1 << 20, None) == N.MAG_E_SIZE
    out.verdict = None
    assert lib.mag_detect(fake, ctypes.byref(sa), fake, ctypes.byref(sb), None, ctypes.byref(out),
                          fake, 1 << 20, None) == N.MAG_E_NULL
    assert lib.mag_detect(None, None, None, None, None, None, None, 0, None) == N.MAG_E_NULL
    assert lib.mag_detect_workspace_size(5, 5, -1, ctypes.byref(b)) == N.MAG_E_SIZE


def test_stream_host_side_errors_without_gpu():
    from paper_2512_08365_amd import _native as N
    lib = N.load()
    b = ctypes.c_size_t(0)
    assert lib.mag_stream_workspace_size(1, 0, 0, None, ctypes.byref(b)) == N.MAG_E_SIZE
    assert lib.mag_stream_workspace_size(10, 0, 0, None, None) == N.MAG_E_NULL
    assert lib.mag_stream_workspace_size(10, 3, -1, None, ctypes.byref(b)) == N.MAG_E_SIZE
    assert lib.mag_stream_workspace_size(10_000, 3, 8, None, ctypes.byref(b)) == N.MAG_OK
    one = b.value
    assert lib.mag_attribute_workspace_size(10_000, 3, 8, None, ctypes.byref(b)) == N.MAG_OK
    assert one > b.value  # the staging buffer of the tile spanning two chunks
    h = ctypes.c_void_p(1234)
    fake = ctypes.c_void_p(256)
    assert lib.mag_stream_begin(None, 10, None, None, None, 0, None, None, 0, fake, 1 << 20,
                                None) == N.MAG_E_NULL
    assert lib.mag_stream_begin(ctypes.byref(h), 1, None, None, None, 0, None, None, 0, fake,
                                1 << 20, None) == N.MAG_E_SIZE
    assert h.value is None  # no handle on failure
    assert lib.mag_stream_begin(ctypes.byref(h), 10, fake, fake, None, 3, None, None, 4, fake,
                                1 << 20, None) == N.MAG_E_NULL  # keys needed for grouping
    assert lib.mag_stream_begin(ctypes.byref(h), 10, fake, fake, None, 3, None, None, 0, fake,
                                16, None) == N.MAG_E_WORKSPACE
    assert lib.mag_stream_push(None, fake, fake, 10) == N.MAG_E_NULL
    assert lib.mag_stream_end(None, None, None, None) == N.MAG_E_NULL
    assert lib.mag_stream_state_export(None, None, ctypes.byref(b)) == N.MAG_E_NULL
    assert lib.mag_stream_state_import(None, None, 0) == N.MAG_E_NULL
    lib.mag_stream_abort(None)


def test_product_has_no_cpu_fallback():
    # the binding refuses CPU tensors instead of computing on the host
    torch = pytest.importorskip("torch")
    import paper_2512_08365_amd as mag
    t = torch.linspace(0, 1, 10, dtype=torch.float64)
    P = torch.ones(10, dtype=torch.float32)
    s = torch.zeros(1, dtype=torch.float64)
    with pytest.raises(mag.MagnetonError):
        mag.attribute(t, P, s, s + 0.5)


def test_product_does_not_import_the_oracle():
    pkg = os.path.join(ROOT, "paper_2512_08365_amd")
    for path in glob.glob(os.path.join(pkg, "**", "*"), recursive=True):
        if os.path.isfile(path) and path.endswith((".py", ".hip", ".hpp", ".h", ".cpp")):
            text = open(path).read()
            assert "oracle" not in text.lower().replace("oracle-free", ""), path


def test_invariants_host_side_errors_without_gpu():
    from paper_2512_08365_amd import _native as N
    lib = N.load()
    u, v = ctypes.c_int32(0), ctypes.c_int64(0)
    t = N.Tensor(ctypes.c_void_p(256), 3, 0, (ctypes.c_int64 * 5)(4, 6, 5, 0, 0))
    assert lib.mag_invariant_count(ctypes.byref(t), ctypes.byref(u), ctypes.byref(v)) == 0
    # masks {0}, {0,1}, {0,2}: min(4, 30) + min(24, 5) + min(20, 6)
    assert u.value == 3 and v.value == 4 + 5 + 6
    t.rank = 6
    assert lib.mag_invariant_count(ctypes.byref(t), ctypes.byref(u), ctypes.byref(v)) == N.MAG_E_SIZE
    t.rank, t.dims[1] = 3, 0
    assert lib.mag_invariant_count(ctypes.byref(t), ctypes.byref(u), ctypes.byref(v)) == N.MAG_E_SIZE
    # a Gram side above 512 takes the many-workgroup path; above MAG_SVD_MAX_K it is refused
    mid = N.Tensor(ctypes.c_void_p(256), 2, 0, (ctypes.c_int64 * 5)(600, 700, 0, 0, 0))
    assert lib.mag_invariant_count(ctypes.byref(mid), ctypes.byref(u), ctypes.byref(v)) == 0
    assert (u.value, v.value) == (1, 600)
    big = N.Tensor(ctypes.c_void_p(256), 2, 0,
                   (ctypes.c_int64 * 5)(N.MAG_SVD_MAX_K + 1, N.MAG_SVD_MAX_K + 2, 0, 0, 0))
    assert lib.mag_invariant_count(ctypes.byref(big), ctypes.byref(u), ctypes.byref(v)) == N.MAG_E_SIZE
    assert str(N.MAG_SVD_MAX_K).encode() in lib.mag_last_error()
    assert lib.mag_invariant_count(None, ctypes.byref(u), ctypes.byref(v)) == N.MAG_E_NULL
    b = ctypes.c_size_t(0)
    ok = N.Tensor(ctypes.c_void_p(256), 2, 0, (ctypes.c_int64 * 5)(30, 40, 0, 0, 0))
    assert lib.mag_invariants_workspace_size(ctypes.byref(ok), 1, ctypes.byref(b)) == 0
    assert b.value >= 30 * 30 * 8
    assert lib.mag_invariants(ctypes.byref(ok), 1, None, ctypes.c_void_p(256), b.value,
                              None) == N.MAG_E_NULL
    assert lib.mag_invariants(ctypes.byref(ok), 1, ctypes.c_void_p(256), ctypes.c_void_p(256),
                              16, None) == N.MAG_E_WORKSPACE
    assert lib.mag_match(None, 1, None, None, 1, None, float("nan"), None, None, 0,
                         None) == N.MAG_E_SIZE
    assert lib.mag_match(None, 1, None, None, 1, None, 1e-5, None, None, 0, None) == N.MAG_E_NULL
    assert lib.mag_match_workspace_size(-1, 2, ctypes.byref(b)) == N.MAG_E_SIZE
