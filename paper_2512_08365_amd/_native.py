"""ctypes view of libmagneton.so (declarations mirror include/magneton.h)."""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
# MAG_LIBRARY_SO: another build of the library to load (the host-sanitizer run
# of the CPU tests); the default is the in-tree build
LIB_PATH = os.environ.get("MAG_LIBRARY_SO") or os.path.join(HERE, "libmagneton.so")

c_i64 = ctypes.c_int64
c_vp = ctypes.c_void_p

MAG_OK = 0
MAG_E_NULL = -1
MAG_E_SIZE = -2
MAG_E_CAPACITY = -3
MAG_E_WORKSPACE = -4
MAG_E_TIMESTAMPS = -5
MAG_E_POWER = -6
MAG_E_INTERVAL = -7
MAG_E_STREAMS = -8
MAG_E_STATE = -9
MAG_E_HIP = -10
MAG_E_ALIGN = -11
MAG_E_KEYS = -12
MAG_E_COUNTER = -13
MAG_E_GRAPH = -14

MAG_EQUAL_SPLIT = 0x1
MAG_SKIP_VALIDATE = 0x2
MAG_TIME_KERNELS = 0x4
MAG_ASYNC = 0x8
MAG_KEY_LATENCY = 0x10
MAG_WASTE = 1
MAG_TRADEOFF = 2
MAG_MAX_STREAMS = 32
MAG_STATIC_SCRATCH_BYTES = 64 << 20

# every symbol include/magneton.h declares
EXPORTED = (
    "mag_attribute_workspace_size", "mag_attribute", "mag_attribute_static",
    "mag_key_plan_size", "mag_key_plan_build",
    "mag_attribute_finish",
    "mag_counter_workspace_size", "mag_attribute_counter",
    "mag_diff_workspace_size", "mag_diff", "mag_diff_async", "mag_diff_finish",
    "mag_diff_batch_workspace_size", "mag_diff_batch",
    "mag_detect_workspace_size", "mag_detect",
    "mag_invariant_count", "mag_invariants_workspace_size", "mag_invariants",
    "mag_match_workspace_size", "mag_match", "mag_match_subgraphs",
    "mag_stream_workspace_size", "mag_stream_begin", "mag_stream_push", "mag_stream_end",
    "mag_stream_abort", "mag_stream_state_export", "mag_stream_state_import",
    "mag_stream_host_staging_size", "mag_stream_set_host_staging", "mag_stream_push_host",
    "mag_strerror", "mag_last_error", "mag_version",
)


class KeyPlan(ctypes.Structure):
    _fields_ = [("buffer", c_vp), ("bytes", ctypes.c_size_t), ("n_intervals", c_i64),
                ("key_capacity", c_i64), ("ready", c_vp)]


class AttrOpts(ctypes.Structure):
    _fields_ = [("n_streams", ctypes.c_int32), ("flags", ctypes.c_uint32),
                ("stream_offsets", c_vp), ("intervals_ready", c_vp),
                ("key_plan", ctypes.POINTER(KeyPlan)), ("tiles_wait", c_vp), ("tiles_done", c_vp),
                ("group_stream", c_vp)]


class IntervalOut(ctypes.Structure):
    _fields_ = [("energy", c_vp), ("start_idx", c_vp), ("end_idx", c_vp)]


class KeyStats(ctypes.Structure):
    _fields_ = [("sum", c_vp), ("m2", c_vp), ("count", c_vp), ("capacity", c_i64),
                ("n_keys", c_i64), ("duration", c_vp), ("n_keys_device", c_vp)]


class Summary(ctypes.Structure):
    _fields_ = [("trace_energy", ctypes.c_double), ("idle_energy", ctypes.c_double),
                ("attributed_energy", ctypes.c_double), ("n_clipped", c_i64), ("n_keys", c_i64),
                ("tile_kernel_ms", ctypes.c_double), ("device_ms", ctypes.c_double)]


class RankOut(ctypes.Structure):
    _fields_ = [("key", c_vp), ("ratio", c_vp), ("energy_a", c_vp), ("energy_b", c_vp),
                ("count_a", c_vp), ("count_b", c_vp), ("capacity", c_i64), ("n_out", c_i64),
                ("n_only_a", c_i64), ("n_only_b", c_i64), ("n_join", c_i64)]


MAG_SVD_MAX_RANK = 5
MAG_SVD_MAX_K = 8192


class Tensor(ctypes.Structure):
    _fields_ = [("data", c_vp), ("rank", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("dims", c_i64 * MAG_SVD_MAX_RANK)]


class GraphDesc(ctypes.Structure):
    _fields_ = [("n_nodes", ctypes.c_int32), ("n_edges", ctypes.c_int32), ("src", c_vp),
                ("dst", c_vp)]


class DetectOpts(ctypes.Structure):
    _fields_ = [("threshold", ctypes.c_double), ("tolerance", ctypes.c_double)]


class DetectOut(ctypes.Structure):
    _fields_ = [("rank", RankOut), ("latency_a", c_vp), ("latency_b", c_vp), ("verdict", c_vp),
                ("n_flagged", c_i64), ("n_waste", c_i64), ("n_tradeoff", c_i64)]


_lib = None


def load(path: str = LIB_PATH):
    """Load the HIP library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(
            f"{path} is missing: build the HIP library first (python -c 'import __graft_entry__ as g; g.build()')")
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER
    lib.mag_attribute_workspace_size.argtypes = [c_i64, c_i64, c_i64, P(AttrOpts), P(ctypes.c_size_t)]
    lib.mag_attribute_workspace_size.restype = ctypes.c_int
    lib.mag_attribute.argtypes = [c_vp, c_vp, c_i64, c_vp, c_vp, c_vp, c_i64, P(AttrOpts),
                                  P(IntervalOut), c_vp, P(KeyStats), P(Summary), c_vp,
                                  ctypes.c_size_t, c_vp]
    lib.mag_attribute.restype = ctypes.c_int
    lib.mag_attribute_static.argtypes = [c_vp, c_vp, c_i64, c_vp, c_vp, c_vp, c_i64, P(AttrOpts),
                                         P(IntervalOut), c_vp, P(KeyStats), P(Summary), c_vp]
    lib.mag_attribute_static.restype = ctypes.c_int
    lib.mag_key_plan_size.argtypes = [c_i64, c_i64, P(ctypes.c_size_t)]
    lib.mag_key_plan_size.restype = ctypes.c_int
    lib.mag_key_plan_build.argtypes = [c_vp, c_i64, c_i64, P(KeyPlan), c_vp]
    lib.mag_key_plan_build.restype = ctypes.c_int
    lib.mag_attribute_finish.argtypes = [c_vp, P(KeyStats), P(Summary), c_vp]
    lib.mag_attribute_finish.restype = ctypes.c_int
    lib.mag_counter_workspace_size.argtypes = [c_i64, c_i64, c_i64, ctypes.c_uint32,
                                               P(ctypes.c_size_t)]
    lib.mag_counter_workspace_size.restype = ctypes.c_int
    lib.mag_attribute_counter.argtypes = [c_vp, c_vp, c_i64, ctypes.c_double, c_vp, c_vp, c_vp,
                                          c_vp, c_i64, ctypes.c_uint32, P(IntervalOut), c_vp,
                                          P(KeyStats), P(Summary), c_vp, ctypes.c_size_t, c_vp]
    lib.mag_attribute_counter.restype = ctypes.c_int
    lib.mag_diff_workspace_size.argtypes = [c_i64, c_i64, c_i64, P(ctypes.c_size_t)]
    lib.mag_diff_workspace_size.restype = ctypes.c_int
    lib.mag_diff.argtypes = [c_vp, P(KeyStats), c_vp, P(KeyStats), c_i64, P(RankOut), c_vp,
                             ctypes.c_size_t, c_vp]
    lib.mag_diff.restype = ctypes.c_int
    lib.mag_diff_async.argtypes = lib.mag_diff.argtypes
    lib.mag_diff_async.restype = ctypes.c_int
    lib.mag_diff_finish.argtypes = [c_vp, P(RankOut)]
    lib.mag_diff_finish.restype = ctypes.c_int
    lib.mag_diff_batch_workspace_size.argtypes = [c_i64, ctypes.c_int32, c_i64,
                                                  P(ctypes.c_size_t)]
    lib.mag_diff_batch_workspace_size.restype = ctypes.c_int
    # keysB: host array of device pointers; statsB / out: host arrays of structs
    lib.mag_diff_batch.argtypes = [c_vp, P(KeyStats), ctypes.c_int32, c_vp, c_vp, c_i64, c_vp,
                                   c_vp, ctypes.c_size_t, c_vp]
    lib.mag_diff_batch.restype = ctypes.c_int
    lib.mag_detect_workspace_size.argtypes = [c_i64, c_i64, c_i64, P(ctypes.c_size_t)]
    lib.mag_detect_workspace_size.restype = ctypes.c_int
    lib.mag_detect.argtypes = [c_vp, P(KeyStats), c_vp, P(KeyStats), P(DetectOpts), P(DetectOut),
                               c_vp, ctypes.c_size_t, c_vp]
    lib.mag_detect.restype = ctypes.c_int
    i32 = ctypes.c_int32
    lib.mag_invariant_count.argtypes = [P(Tensor), P(i32), P(c_i64)]
    lib.mag_invariant_count.restype = ctypes.c_int
    lib.mag_invariants_workspace_size.argtypes = [P(Tensor), i32, P(ctypes.c_size_t)]
    lib.mag_invariants_workspace_size.restype = ctypes.c_int
    lib.mag_invariants.argtypes = [P(Tensor), i32, c_vp, c_vp, ctypes.c_size_t, c_vp]
    lib.mag_invariants.restype = ctypes.c_int
    lib.mag_match_workspace_size.argtypes = [i32, i32, P(ctypes.c_size_t)]
    lib.mag_match_workspace_size.restype = ctypes.c_int
    lib.mag_match.argtypes = [P(Tensor), i32, c_vp, P(Tensor), i32, c_vp, ctypes.c_double, c_vp,
                              c_vp, ctypes.c_size_t, c_vp]
    lib.mag_match.restype = ctypes.c_int
    lib.mag_match_subgraphs.argtypes = [P(GraphDesc), P(GraphDesc), c_vp, i32, c_vp, i32, P(i32)]
    lib.mag_match_subgraphs.restype = ctypes.c_int
    lib.mag_stream_workspace_size.argtypes = [c_i64, c_i64, c_i64, P(AttrOpts), P(ctypes.c_size_t)]
    lib.mag_stream_workspace_size.restype = ctypes.c_int
    lib.mag_stream_begin.argtypes = [P(c_vp), c_i64, c_vp, c_vp, c_vp, c_i64, P(AttrOpts),
                                     P(IntervalOut), c_i64, c_vp, ctypes.c_size_t, c_vp]
    lib.mag_stream_begin.restype = ctypes.c_int
    lib.mag_stream_push.argtypes = [c_vp, c_vp, c_vp, c_i64]
    lib.mag_stream_push.restype = ctypes.c_int
    lib.mag_stream_end.argtypes = [c_vp, c_vp, P(KeyStats), P(Summary)]
    lib.mag_stream_end.restype = ctypes.c_int
    lib.mag_stream_abort.argtypes = [c_vp]
    lib.mag_stream_abort.restype = None
    lib.mag_stream_state_export.argtypes = [c_vp, c_vp, P(ctypes.c_size_t)]
    lib.mag_stream_state_export.restype = ctypes.c_int
    lib.mag_stream_state_import.argtypes = [c_vp, c_vp, ctypes.c_size_t]
    lib.mag_stream_state_import.restype = ctypes.c_int
    lib.mag_stream_host_staging_size.argtypes = [c_i64, P(ctypes.c_size_t)]
    lib.mag_stream_host_staging_size.restype = ctypes.c_int
    lib.mag_stream_set_host_staging.argtypes = [c_vp, c_i64, c_vp, ctypes.c_size_t, c_vp]
    lib.mag_stream_set_host_staging.restype = ctypes.c_int
    lib.mag_stream_push_host.argtypes = [c_vp, c_vp, c_vp, c_i64]
    lib.mag_stream_push_host.restype = ctypes.c_int
    lib.mag_strerror.argtypes = [ctypes.c_int]
    lib.mag_strerror.restype = ctypes.c_char_p
    lib.mag_last_error.argtypes = []
    lib.mag_last_error.restype = ctypes.c_char_p
    lib.mag_version.argtypes = []
    lib.mag_version.restype = ctypes.c_char_p
    _lib = lib
    return lib
