// api.hip -- host side of the C ABI: argument checks, workspace carving,
// launch sequence and status read-back.  See include/magneton.h.

#include <stdio.h>
#include <string.h>

#include <algorithm>

#include "mag_internal.hpp"

namespace {

thread_local char g_last_error[512] = "";

int fail(int code, const char* msg)
{
    snprintf(g_last_error, sizeof(g_last_error), "%s", msg);
    return code;
}

int hip_fail(hipError_t e, const char* where)
{
    snprintf(g_last_error, sizeof(g_last_error), "%s: %s", where, hipGetErrorString(e));
    return MAG_E_HIP;
}

constexpr size_t ALIGN = 256;

size_t align_up(size_t x) { return (x + ALIGN - 1) / ALIGN * ALIGN; }

// sequential carving of one workspace
struct Carver {
    size_t off = 0;
    char* base = nullptr;
    template <class T>
    T* take(size_t count)
    {
        T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
        off = align_up(off + count * sizeof(T));
        return p;
    }
};

uint32_t hash_slots(int64_t cap)
{
    uint64_t want = (uint64_t)std::max<int64_t>(2 * cap + 2, 1024);
    uint64_t h = 1;
    while (h < want) h <<= 1;
    return (uint32_t)h;
}

struct Plan {
    int64_t n, m, NT, cap;
    int S;
    uint32_t H;
    int nchunks;
    int64_t chunk;
};

struct AttrWorkspace {
    mag::Status* status;
    int64_t* cnt;
    int64_t* cnt_fin;
    double* head;
    double* tail;
    double* tileW;
    double* tileIdle;
    double* energy;
    unsigned long long* table;
    uint32_t* slot;
    uint32_t* slot2id;
    uint64_t* ukey;
    uint32_t* uslot;
    uint32_t* urank;
    double* mean;
    uint32_t* pcnt;
    double* psum;
    double* pm2;
};

void plan_groupby(Plan& pl)
{
    pl.H = hash_slots(pl.cap);
    int64_t nc = (pl.m + 4095) / 4096;
    nc = std::max<int64_t>(1, std::min<int64_t>(nc, mag::AGG_MAX_CHUNKS));
    pl.nchunks = (int)nc;
    pl.chunk = (pl.m + nc - 1) / nc;
}

size_t carve(const Plan& pl, void* ws, AttrWorkspace& w)
{
    Carver c;
    c.base = static_cast<char*>(ws);
    w.status = c.take<mag::Status>(1);
    w.cnt = c.take<int64_t>((size_t)pl.S * (pl.NT + 1));
    w.cnt_fin = c.take<int64_t>((size_t)pl.S * (pl.NT + 1));
    w.head = c.take<double>((size_t)pl.S * pl.NT);
    w.tail = c.take<double>((size_t)pl.S * pl.NT);
    w.tileW = c.take<double>((size_t)pl.NT);
    w.tileIdle = c.take<double>((size_t)pl.NT);
    w.energy = c.take<double>((size_t)std::max<int64_t>(pl.m, 1));
    if (pl.H > 0) {
        w.table = c.take<unsigned long long>(pl.H);
        w.slot = c.take<uint32_t>((size_t)std::max<int64_t>(pl.m, 1));
        w.slot2id = c.take<uint32_t>((size_t)pl.H + 1);
        w.ukey = c.take<uint64_t>((size_t)pl.H + 1);
        w.uslot = c.take<uint32_t>((size_t)pl.H + 1);
        w.urank = c.take<uint32_t>((size_t)pl.H + 1);
        w.mean = c.take<double>((size_t)std::max<int64_t>(pl.cap, 1));
        w.pcnt = c.take<uint32_t>((size_t)pl.nchunks * std::max<int64_t>(pl.cap, 1));
        w.psum = c.take<double>((size_t)pl.nchunks * std::max<int64_t>(pl.cap, 1));
        w.pm2 = c.take<double>((size_t)pl.nchunks * std::max<int64_t>(pl.cap, 1));
    }
    return c.off;
}

int check_opts(const mag_attr_opts* opts, int64_t m, int* S, uint32_t* flags, mag::StreamSet* ss)
{
    *S = opts ? opts->n_streams : 1;
    *flags = opts ? opts->flags : MAG_EQUAL_SPLIT;
    if (*S < 1 || *S > MAG_MAX_STREAMS) {
        snprintf(g_last_error, sizeof(g_last_error), "n_streams must be in [1, %d], got %d",
                 MAG_MAX_STREAMS, *S);
        return MAG_E_STREAMS;
    }
    const int64_t* offs = opts ? opts->stream_offsets : nullptr;
    if (!offs && *S != 1) return fail(MAG_E_STREAMS, "stream_offsets is NULL with n_streams > 1");
    if (ss) {
        memset(ss, 0, sizeof(*ss));
        ss->S = *S;
    }
    if (offs) {
        if (offs[0] != 0 || offs[*S] != m)
            return fail(MAG_E_STREAMS, "stream_offsets must start at 0 and end at n_intervals");
        for (int a = 0; a < *S; ++a)
            if (offs[a + 1] < offs[a]) return fail(MAG_E_STREAMS, "stream_offsets must not decrease");
        if (ss)
            for (int a = 0; a <= *S; ++a) ss->off[a] = offs[a];
    } else if (ss) {
        ss->off[0] = 0;
        ss->off[1] = m;
    }
    return MAG_OK;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// optional HIP-event timing of a call's device work on its stream
struct EventTimer {
    bool on = false;
    hipStream_t stream;
    hipEvent_t ev[4] = {nullptr, nullptr, nullptr, nullptr};
    EventTimer(bool enable, hipStream_t s) : on(enable), stream(s)
    {
        if (!on) return;
        for (auto& x : ev)
            if (hipEventCreate(&x) != hipSuccess) on = false;
    }
    ~EventTimer()
    {
        for (auto& x : ev)
            if (x) (void)hipEventDestroy(x);
    }
    void mark(int i)
    {
        if (on) (void)hipEventRecord(ev[i], stream);
    }
    double ms(int a, int b) const
    {
        float v = 0.0f;
        if (!on || hipEventElapsedTime(&v, ev[a], ev[b]) != hipSuccess) return 0.0;
        return (double)v;
    }
};

}  // namespace

namespace mag {

int device_cu_count()
{
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
        return 256;
    return cus;
}

}  // namespace mag

extern "C" {

const char* mag_version(void) { return "magneton-mi355x 0.1"; }

const char* mag_last_error(void) { return g_last_error; }

const char* mag_strerror(int status)
{
    switch (status) {
    case MAG_OK: return "ok";
    case MAG_E_NULL: return "a required pointer is NULL";
    case MAG_E_SIZE: return "invalid size";
    case MAG_E_CAPACITY: return "output capacity too small";
    case MAG_E_WORKSPACE: return "workspace too small or misaligned";
    case MAG_E_TIMESTAMPS: return "timestamps not finite or not strictly increasing";
    case MAG_E_POWER: return "power sample negative or not finite";
    case MAG_E_INTERVAL: return "interval bounds invalid, unsorted or overlapping within a stream";
    case MAG_E_STREAMS: return "invalid stream description";
    case MAG_E_STATE: return "invalid handle state";
    case MAG_E_HIP: return "HIP runtime error";
    case MAG_E_ALIGN: return "device array misaligned";
    case MAG_E_KEYS: return "key table not strictly ascending";
    default: return "unknown status";
    }
}

int mag_attribute_workspace_size(int64_t n_samples, int64_t n_intervals, int64_t key_capacity,
                                 const mag_attr_opts* opts, size_t* bytes)
{
    g_last_error[0] = 0;
    if (!bytes) return fail(MAG_E_NULL, "bytes is NULL");
    if (n_samples < 2) return fail(MAG_E_SIZE, "n_samples must be >= 2");
    if (n_intervals < 0 || key_capacity < 0) return fail(MAG_E_SIZE, "negative size");
    int S;
    uint32_t flags;
    int rc = check_opts(opts, n_intervals, &S, &flags, nullptr);
    if (rc) return rc;
    Plan pl{};
    pl.n = n_samples;
    pl.m = n_intervals;
    pl.S = S;
    pl.NT = (n_samples - 1 + mag::TILE - 1) / mag::TILE;
    pl.cap = key_capacity;
    pl.H = 0;
    if (key_capacity > 0) plan_groupby(pl);
    AttrWorkspace w{};
    *bytes = carve(pl, nullptr, w);
    return MAG_OK;
}

int mag_attribute(const double* timestamps, const float* power, int64_t n_samples,
                  const double* starts, const double* ends, const uint64_t* op_keys,
                  int64_t n_intervals, const mag_attr_opts* opts, mag_interval_out* per_interval,
                  uint64_t* keys_out, mag_key_stats* per_key, mag_summary* summary, void* workspace,
                  size_t workspace_bytes, hipStream_t stream)
{
    g_last_error[0] = 0;
    if (!timestamps || !power) return fail(MAG_E_NULL, "timestamps/power is NULL");
    if (n_samples < 2) return fail(MAG_E_SIZE, "n_samples must be >= 2");
    if (n_intervals < 0) return fail(MAG_E_SIZE, "n_intervals must be >= 0");
    if (n_intervals > 0 && (!starts || !ends)) return fail(MAG_E_NULL, "starts/ends is NULL");
    if (per_key) {
        if (per_key->capacity < 1) return fail(MAG_E_SIZE, "per_key->capacity must be >= 1");
        if (!keys_out || !per_key->sum || !per_key->m2 || !per_key->count)
            return fail(MAG_E_NULL, "per-key output array is NULL");
        if (n_intervals > 0 && !op_keys) return fail(MAG_E_NULL, "op_keys is NULL");
    }
    if (!workspace) return fail(MAG_E_NULL, "workspace is NULL");
    if (!aligned(workspace, 256)) return fail(MAG_E_WORKSPACE, "workspace must be 256-byte aligned");
    if (!aligned(timestamps, 8) || !aligned(power, 4) || (starts && !aligned(starts, 8)) ||
        (ends && !aligned(ends, 8)) || (op_keys && !aligned(op_keys, 8)))
        return fail(MAG_E_ALIGN, "input array not aligned to its element size");

    int S;
    uint32_t flags;
    mag::StreamSet ss;
    int rc = check_opts(opts, n_intervals, &S, &flags, &ss);
    if (rc) return rc;

    const bool group = per_key != nullptr;
    Plan pl{};
    pl.n = n_samples;
    pl.m = n_intervals;
    pl.S = S;
    pl.NT = (n_samples - 1 + mag::TILE - 1) / mag::TILE;
    pl.cap = group ? per_key->capacity : 0;
    pl.H = 0;
    if (group) plan_groupby(pl);
    AttrWorkspace w{};
    const size_t need = carve(pl, nullptr, w);
    if (workspace_bytes < need) {
        snprintf(g_last_error, sizeof(g_last_error), "workspace needs %zu bytes, got %zu", need,
                 workspace_bytes);
        return MAG_E_WORKSPACE;
    }
    carve(pl, workspace, w);

    double* energy = (per_interval && per_interval->energy) ? per_interval->energy : w.energy;
    hipError_t e;
    EventTimer timer((flags & MAG_TIME_KERNELS) != 0, stream);
    timer.mark(0);
    if ((e = mag::launch_init_status(w.status, timestamps, n_samples, stream)) != hipSuccess)
        return hip_fail(e, "init");

    // --- attribution
    mag::TileParams tp{};
    tp.t = timestamps;
    tp.P = power;
    tp.base = 0;
    tp.nseg = n_samples - 1;
    tp.n_total = n_samples;
    tp.NT = pl.NT;
    tp.tile_begin = 0;
    tp.tile_end = pl.NT;
    const int64_t wgs = (int64_t)mag::device_cu_count() * mag::TILE_WGS_PER_CU;
    tp.tiles_per_wg = std::max<int64_t>(1, (pl.NT + wgs - 1) / wgs);
    const int grid = (int)((pl.NT + tp.tiles_per_wg - 1) / tp.tiles_per_wg);
    tp.s = starts;
    tp.e = ends;
    tp.ss = ss;
    tp.energy = energy;
    tp.start_idx = per_interval ? per_interval->start_idx : nullptr;
    tp.end_idx = per_interval ? per_interval->end_idx : nullptr;
    tp.cnt = w.cnt;
    tp.cnt_fin = w.cnt_fin;
    tp.head = w.head;
    tp.tail = w.tail;
    tp.tileW = w.tileW;
    tp.tileIdle = w.tileIdle;
    tp.status = w.status;
    tp.split = (flags & MAG_EQUAL_SPLIT) ? 1 : 0;
    tp.validate = (flags & MAG_SKIP_VALIDATE) ? 0 : 1;
    tp.aligned16 = (aligned(timestamps, 16) && aligned(power, 16)) ? 1 : 0;
    timer.mark(1);
    e = mag::launch_tile(tp, grid, stream);
    if (e != hipSuccess) return hip_fail(e, "tile kernel");
    timer.mark(2);

    mag::FixParams fp{};
    fp.s = starts;
    fp.e = ends;
    fp.ss = ss;
    fp.NT = pl.NT;
    fp.n_total = n_samples;
    fp.cnt = w.cnt;
    fp.cnt_fin = w.cnt_fin;
    fp.tile_begin = tp.tile_begin;
    fp.tiles_per_wg = tp.tiles_per_wg;
    fp.head = w.head;
    fp.tail = w.tail;
    fp.energy = energy;
    fp.start_idx = tp.start_idx;
    fp.end_idx = tp.end_idx;
    fp.status = w.status;
    fp.validate = tp.validate;
    if ((e = mag::launch_cross(fp, stream)) != hipSuccess) return hip_fail(e, "cross kernel");
    if ((e = mag::launch_outside(fp, stream)) != hipSuccess) return hip_fail(e, "outside kernel");
    if ((e = mag::launch_summary(w.tileW, w.tileIdle, pl.NT, w.status, stream)) != hipSuccess)
        return hip_fail(e, "summary kernel");

    // --- grouping
    if (group && n_intervals > 0) {
        mag::GroupParams gp{};
        gp.keys = op_keys;
        gp.energy = energy;
        gp.m = n_intervals;
        gp.H = pl.H;
        gp.cap = pl.cap;
        gp.nchunks = pl.nchunks;
        gp.chunk = pl.chunk;
        gp.table = w.table;
        gp.slot = w.slot;
        gp.slot2id = w.slot2id;
        gp.ukey = w.ukey;
        gp.uslot = w.uslot;
        gp.urank = w.urank;
        gp.mean = w.mean;
        gp.pcnt = w.pcnt;
        gp.psum = w.psum;
        gp.pm2 = w.pm2;
        gp.keys_out = keys_out;
        gp.sum_out = per_key->sum;
        gp.m2_out = per_key->m2;
        gp.count_out = per_key->count;
        gp.status = w.status;
        if ((e = mag::launch_groupby(gp, stream)) != hipSuccess) return hip_fail(e, "group-by");
    } else if (n_intervals > 0) {
        if ((e = mag::launch_energy_total(energy, n_intervals, w.status, stream)) != hipSuccess)
            return hip_fail(e, "energy total");
    }

    timer.mark(3);
    mag::Status st;
    if ((e = hipMemcpyAsync(&st, w.status, sizeof(st), hipMemcpyDeviceToHost, stream)) != hipSuccess)
        return hip_fail(e, "status copy");
    if ((e = hipStreamSynchronize(stream)) != hipSuccess) return hip_fail(e, "synchronize");

    const int64_t n_keys = (int64_t)st.n_unique;
    if (summary) {
        summary->tile_kernel_ms = timer.ms(1, 2);
        summary->device_ms = timer.ms(0, 3);
    }
    if (per_key) per_key->n_keys = std::min<int64_t>(n_keys, per_key->capacity);
    if (summary) {
        summary->trace_energy = st.trace_energy;
        summary->idle_energy = st.idle_energy;
        summary->attributed_energy = st.attributed_energy;
        summary->n_clipped = (int64_t)st.n_clipped;
        summary->n_keys = n_keys;
    }
    if (st.err & mag::ERR_TIMESTAMPS)
        return fail(MAG_E_TIMESTAMPS, "timestamps not finite or not strictly increasing");
    if (st.err & mag::ERR_POWER) return fail(MAG_E_POWER, "power sample negative or not finite");
    if (st.err & mag::ERR_INTERVAL)
        return fail(MAG_E_INTERVAL, "interval bound not finite, start > end, or a stream unsorted/overlapping");
    if (group && (st.overflow || n_keys > per_key->capacity)) {
        per_key->n_keys = n_keys;
        snprintf(g_last_error, sizeof(g_last_error),
                 "%lld distinct keys%s exceed the key capacity %lld", (long long)n_keys,
                 st.overflow ? " (at least)" : "", (long long)per_key->capacity);
        return MAG_E_CAPACITY;
    }
    return MAG_OK;
}

int mag_diff_workspace_size(int64_t n_keys_a, int64_t n_keys_b, int64_t k, size_t* bytes)
{
    g_last_error[0] = 0;
    if (!bytes) return fail(MAG_E_NULL, "bytes is NULL");
    if (n_keys_a < 0 || n_keys_b < 0 || k < 0) return fail(MAG_E_SIZE, "negative size");
    Carver c;
    c.take<mag::Status>(1);
    const size_t na = (size_t)std::max<int64_t>(n_keys_a, 1);
    c.take<double>(na);
    c.take<uint64_t>(na);
    c.take<int32_t>(na);
    c.take<int32_t>(na);
    *bytes = c.off;
    return MAG_OK;
}

int mag_diff(const uint64_t* keysA, const mag_key_stats* statsA, const uint64_t* keysB,
             const mag_key_stats* statsB, int64_t k, mag_rank_out* out, void* workspace,
             size_t workspace_bytes, hipStream_t stream)
{
    g_last_error[0] = 0;
    if (!statsA || !statsB || !out) return fail(MAG_E_NULL, "statsA/statsB/out is NULL");
    if (k < 0 || statsA->n_keys < 0 || statsB->n_keys < 0) return fail(MAG_E_SIZE, "negative size");
    const int64_t na = statsA->n_keys, nb = statsB->n_keys;
    if ((na > 0 && (!keysA || !statsA->sum || !statsA->count)) ||
        (nb > 0 && (!keysB || !statsB->sum || !statsB->count)))
        return fail(MAG_E_NULL, "key table array is NULL");
    if (na > INT32_MAX || nb > INT32_MAX) return fail(MAG_E_SIZE, "key table too large");
    const int64_t need_rows = std::min(k, na);
    if (out->capacity < need_rows) return fail(MAG_E_CAPACITY, "out->capacity < min(k, n_keys_a)");
    if (need_rows > 0 && (!out->key || !out->ratio || !out->energy_a || !out->energy_b ||
                          !out->count_a || !out->count_b))
        return fail(MAG_E_NULL, "output array is NULL");
    if (!workspace) return fail(MAG_E_NULL, "workspace is NULL");
    if (!aligned(workspace, 256)) return fail(MAG_E_WORKSPACE, "workspace must be 256-byte aligned");
    size_t need = 0;
    mag_diff_workspace_size(na, nb, k, &need);
    if (workspace_bytes < need) return fail(MAG_E_WORKSPACE, "workspace too small");

    Carver c;
    c.base = static_cast<char*>(workspace);
    const size_t nas = (size_t)std::max<int64_t>(na, 1);
    mag::DiffParams p{};
    p.status = c.take<mag::Status>(1);
    p.cand_r = c.take<double>(nas);
    p.cand_key = c.take<uint64_t>(nas);
    p.cand_ia = c.take<int32_t>(nas);
    p.cand_ib = c.take<int32_t>(nas);
    p.ka = keysA;
    p.sa = statsA->sum;
    p.ca = statsA->count;
    p.na = na;
    p.kb = keysB;
    p.sb = statsB->sum;
    p.cb = statsB->count;
    p.nb = nb;
    p.k = k;
    p.out_key = out->key;
    p.out_ratio = out->ratio;
    p.out_ea = out->energy_a;
    p.out_eb = out->energy_b;
    p.out_ca = out->count_a;
    p.out_cb = out->count_b;
    hipError_t e;
    if ((e = mag::launch_init_status(p.status, nullptr, 0, stream)) != hipSuccess)
        return hip_fail(e, "init");
    if ((e = mag::launch_diff(p, stream)) != hipSuccess) return hip_fail(e, "diff kernels");
    mag::Status st;
    if ((e = hipMemcpyAsync(&st, p.status, sizeof(st), hipMemcpyDeviceToHost, stream)) != hipSuccess)
        return hip_fail(e, "status copy");
    if ((e = hipStreamSynchronize(stream)) != hipSuccess) return hip_fail(e, "synchronize");
    if (st.err & mag::ERR_KEYS) return fail(MAG_E_KEYS, "key table not strictly ascending");
    out->n_join = st.n_join;
    out->n_out = std::min<int64_t>(k, st.n_join);
    out->n_only_a = na - st.n_join;
    out->n_only_b = nb - st.n_join;
    return MAG_OK;
}

}  // extern "C"
