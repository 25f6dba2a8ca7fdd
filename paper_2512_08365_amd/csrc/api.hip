// api.hip -- host side of the C ABI: argument checks, workspace carving,
// launch sequence and status read-back.  See include/magneton.h.

#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <memory>
#include <mutex>
#include <new>
#include <vector>

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
    bool staging;
    bool lat;  // per-key latency sums (MAG_KEY_LATENCY)
    bool ext_keys;  // the key map comes from a key plan built beforehand
};

struct AttrWorkspace {
    mag::Status* status;
    mag::Status* kstat;  // key state: status, or the key plan's header
    int64_t* cnt;
    int64_t* cnt_fin;
    double* head;
    double* tail;
    double2* part;
    double* energy;
    unsigned long long* table;
    uint32_t* slot;
    uint64_t* ukey;
    uint32_t* urank;
    double* mean;
    uint32_t* pcnt;
    double* psum;
    double* pm2;
    double* pdur;
    double* ctot;    // per-chunk energy totals (the aggregation's)
    double2* fold;   // k_fix's partial sums of the per-run trace and idle energies
    double* stage_t;
    float* stage_P;
};

void plan_groupby(Plan& pl)
{
    pl.H = hash_slots(pl.cap);
    int64_t nc = (pl.m + 4095) / 4096;
    nc = std::max<int64_t>(1, std::min<int64_t>(nc, mag::AGG_MAX_CHUNKS));
    pl.nchunks = (int)nc;
    pl.chunk = (pl.m + nc - 1) / nc;
}

void carve_groupby(Carver& c, const Plan& pl, AttrWorkspace& w);

size_t carve(const Plan& pl, void* ws, AttrWorkspace& w)
{
    Carver c;
    c.base = static_cast<char*>(ws);
    w.status = c.take<mag::Status>(1);
    w.kstat = w.status;
    w.cnt = c.take<int64_t>((size_t)pl.S * (pl.NT + 1));
    w.cnt_fin = c.take<int64_t>((size_t)pl.S * (pl.NT + 1));
    w.head = c.take<double>((size_t)pl.S * pl.NT);
    w.tail = c.take<double>((size_t)pl.S * pl.NT);
    w.part = c.take<double2>((size_t)pl.NT);
    w.fold = c.take<double2>((size_t)mag::FOLD_BLOCKS);
    w.energy = c.take<double>((size_t)std::max<int64_t>(pl.m, 1));
    if (pl.staging) {
        w.stage_t = c.take<double>((size_t)mag::TILE + 1);
        w.stage_P = c.take<float>((size_t)mag::TILE + 1);
    }
    carve_groupby(c, pl, w);
    return c.off;
}

// the counter mode: status, per-chunk figures, energies, group-by state
size_t carve_counter(const Plan& pl, void* ws, AttrWorkspace& w)
{
    Carver c;
    c.base = static_cast<char*>(ws);
    w.status = c.take<mag::Status>(1);
    w.kstat = w.status;
    w.part = c.take<double2>((size_t)pl.NT);
    w.energy = c.take<double>((size_t)std::max<int64_t>(pl.m, 1));
    carve_groupby(c, pl, w);
    return c.off;
}

void carve_groupby(Carver& c, const Plan& pl, AttrWorkspace& w)
{
    if (pl.H > 0) {
        if (!pl.ext_keys) {
            w.table = c.take<unsigned long long>(2 * ((size_t)pl.H + 1));
            w.slot = c.take<uint32_t>((size_t)std::max<int64_t>(pl.m, 1));
            w.ukey = c.take<uint64_t>((size_t)pl.H + 1);
            w.urank = c.take<uint32_t>((size_t)pl.H + 1);
        }
        w.mean = c.take<double>((size_t)std::max<int64_t>(pl.cap, 1));
        w.pcnt = c.take<uint32_t>((size_t)pl.nchunks * std::max<int64_t>(pl.cap, 1));
        w.psum = c.take<double>((size_t)pl.nchunks * std::max<int64_t>(pl.cap, 1));
        w.pm2 = c.take<double>((size_t)pl.nchunks * std::max<int64_t>(pl.cap, 1));
        if (pl.lat) w.pdur = c.take<double>((size_t)pl.nchunks * std::max<int64_t>(pl.cap, 1));
        w.ctot = c.take<double>((size_t)pl.nchunks);
    }
}

// a key plan's buffer: header (a status block holding the key state), then
// the key map of a grouping
size_t carve_key_plan(int64_t m, int64_t cap, void* buf, AttrWorkspace& w)
{
    Carver c;
    c.base = static_cast<char*>(buf);
    const uint32_t H = hash_slots(cap);
    w.kstat = c.take<mag::Status>(1);
    w.table = c.take<unsigned long long>(2 * ((size_t)H + 1));
    w.slot = c.take<uint32_t>((size_t)std::max<int64_t>(m, 1));
    w.ukey = c.take<uint64_t>((size_t)H + 1);
    w.urank = c.take<uint32_t>((size_t)H + 1);
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

// Per-thread records of a call's timing events and of the pinned host buffer
// its status block is copied into, one per (device, workspace).  A record
// whose asynchronous call is not finished yet (events recorded but not read,
// or a status copy in flight) is never handed to another workspace: idle
// records are recycled, least recently used first, once TIMER_KEEP of them
// exist, and the table grows when every record is busy (up to TIMER_MAX
// unfinished asynchronous calls per thread).
struct TimerSlot {
    int dev = -1;
    const void* ws = nullptr;
    hipEvent_t ev[4] = {nullptr, nullptr, nullptr, nullptr};
    bool pending = false;          // events recorded by an asynchronous call, not read yet
    bool status_pending = false;   // an asynchronous call copied its status here
    hipStream_t stream = nullptr;  // the stream that call was enqueued on
    // recorded right after that call's status copy: finishing waits for this
    // call alone, not for later work on its stream (the next call of a
    // caller that keeps several in flight)
    hipEvent_t done = nullptr;
    // a call with a group stream: recorded after its trace integration, waited
    // for by the group stream
    hipEvent_t split = nullptr;
    mag::Status* host_status = nullptr;  // pinned host copy of the status block
    // an asynchronous mag_diff on this workspace: what its conclusion needs
    // besides the status block (table sizes or bounds, rows asked for, whether
    // a size is read on the device)
    bool diff = false, diff_dev = false;
    int64_t diff_na = 0, diff_nb = 0, diff_k = 0;
    uint64_t used = 0;             // last use, for the recycling order
    bool busy() const { return pending || status_pending; }
};
constexpr size_t TIMER_KEEP = 16;
constexpr size_t TIMER_MAX = 4096;
thread_local std::vector<std::unique_ptr<TimerSlot>> g_timers;
thread_local uint64_t g_timer_clock = 0;

TimerSlot* timer_slot(const void* ws, bool create)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return nullptr;
    for (auto& t : g_timers)
        if (t->dev == dev && t->ws == ws) {
            t->used = ++g_timer_clock;
            return t.get();
        }
    if (!create) return nullptr;
    TimerSlot* t = nullptr;
    if (g_timers.size() >= TIMER_KEEP)
        for (auto& x : g_timers)
            if (!x->busy() && (!t || x->used < t->used)) t = x.get();
    if (!t) {
        if (g_timers.size() >= TIMER_MAX) return nullptr;
        std::unique_ptr<TimerSlot> fresh(new (std::nothrow) TimerSlot());
        if (!fresh) return nullptr;
        t = fresh.get();
        g_timers.push_back(std::move(fresh));
    }
    for (auto& x : t->ev)
        if (x) (void)hipEventDestroy(x);
    mag::Status* keep = t->host_status;  // the pinned buffer and the event are reused
    hipEvent_t keep_done = t->done, keep_split = t->split;
    *t = TimerSlot{};
    t->host_status = keep;
    t->done = keep_done;
    t->split = keep_split;
    t->used = ++g_timer_clock;
    for (auto& x : t->ev)
        if (hipEventCreate(&x) != hipSuccess) {
            x = nullptr;
            return nullptr;
        }
    if (!t->host_status) {
        void* h = nullptr;
        if (hipHostMalloc(&h, sizeof(mag::Status), hipHostMallocDefault) != hipSuccess)
            return nullptr;
        t->host_status = static_cast<mag::Status*>(h);
    }
    if (!t->done && hipEventCreateWithFlags(&t->done, hipEventDisableTiming) != hipSuccess) {
        t->done = nullptr;
        return nullptr;
    }
    if (!t->split && hipEventCreateWithFlags(&t->split, hipEventDisableTiming) != hipSuccess) {
        t->split = nullptr;
        return nullptr;
    }
    t->dev = dev;
    t->ws = ws;
    return t;
}

// an asynchronous call on `ws` whose result has not been collected yet
bool unfinished(const void* ws)
{
    const TimerSlot* t = timer_slot(ws, false);
    return t && t->busy();
}

struct EventTimer {
    bool on;
    hipStream_t stream;
    TimerSlot* slot = nullptr;
    EventTimer(bool enable, hipStream_t s, const void* ws) : on(enable), stream(s)
    {
        if (!on) return;
        slot = timer_slot(ws, true);
        on = slot != nullptr;
    }
    // timing is best effort: a failed event call reads as zero time, and its
    // error is cleared so that it is not reported by a later launch check
    void mark(int i)
    {
        if (on && hipEventRecord(slot->ev[i], stream) != hipSuccess) (void)hipGetLastError();
    }
    double ms(int a, int b) const
    {
        float v = 0.0f;
        if (!on) return 0.0;
        if (hipEventElapsedTime(&v, slot->ev[a], slot->ev[b]) != hipSuccess) {
            (void)hipGetLastError();
            return 0.0;
        }
        return (double)v;
    }
};

}  // namespace

namespace mag {

int device_cu_count()
{
    static int cached[16] = {};  // per device, queried once
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    if (dev >= 0 && dev < 16 && cached[dev] > 0) return cached[dev];
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
        return 256;
    if (dev >= 0 && dev < 16) cached[dev] = cus;
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
    case MAG_E_COUNTER: return "energy-counter reading not finite or decreasing";
    default: return "unknown status";
    }
}

int mag_attribute_workspace_size(int64_t n_samples, int64_t n_intervals, int64_t key_capacity,
                                 const mag_attr_opts* opts, size_t* bytes);

}  // extern "C"

namespace {

int plan_attribution(Plan& pl, int64_t n_samples, int64_t n_intervals, int64_t key_capacity,
                     const mag_attr_opts* opts, bool streaming, uint32_t* flags,
                     mag::StreamSet* ss)
{
    if (n_samples < 2) return fail(MAG_E_SIZE, "n_samples must be >= 2");
    if (n_samples > MAG_MAX_SAMPLES) return fail(MAG_E_SIZE, "n_samples exceeds MAG_MAX_SAMPLES");
    if (n_intervals < 0 || key_capacity < 0) return fail(MAG_E_SIZE, "negative size");
    if (key_capacity > MAG_MAX_KEYS) return fail(MAG_E_SIZE, "key_capacity exceeds MAG_MAX_KEYS");
    int S;
    int rc = check_opts(opts, n_intervals, &S, flags, ss);
    if (rc) return rc;
    pl = Plan{};
    pl.n = n_samples;
    pl.m = n_intervals;
    pl.S = S;
    pl.NT = (n_samples - 1 + mag::TILE - 1) / mag::TILE;
    pl.cap = key_capacity;
    pl.H = 0;
    pl.staging = streaming;
    pl.lat = key_capacity > 0 && (*flags & MAG_KEY_LATENCY) != 0;
    pl.ext_keys = key_capacity > 0 && opts && opts->key_plan && !streaming;
    if (key_capacity > 0) plan_groupby(pl);
    return MAG_OK;
}

// One attribution job: plan, carved workspace and launch parameters, shared
// by the one-shot call and the chunked streaming calls.  pl.NT is the number
// of tiles the workspace holds (the row stride of the per-tile arrays).
// read a call's status block back (synchronizing its stream) and turn it into
// the call's result
int interpret_status(const mag::Status& st, mag_key_stats* per_key, mag_summary* summary)
{
    const int64_t n_keys = (int64_t)st.n_unique;
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
    if (st.err & mag::ERR_COUNTER)
        return fail(MAG_E_COUNTER, "energy-counter reading not finite or decreasing");
    if (st.err & mag::ERR_POWER) return fail(MAG_E_POWER, "power sample negative or not finite");
    if (st.err & mag::ERR_INTERVAL)
        return fail(MAG_E_INTERVAL,
                    "interval bound not finite, start > end, or a stream unsorted/overlapping");
    if (per_key && (st.overflow || n_keys > per_key->capacity)) {
        per_key->n_keys = n_keys;
        snprintf(g_last_error, sizeof(g_last_error),
                 "%lld distinct keys%s exceed the key capacity %lld", (long long)n_keys,
                 st.overflow ? " (at least)" : "", (long long)per_key->capacity);
        return MAG_E_CAPACITY;
    }
    return MAG_OK;
}

// copy a device status block to the host (through the workspace's pinned
// buffer) and synchronize `stream`
int read_status(const mag::Status* status, hipStream_t stream, mag::Status* out)
{
    TimerSlot* t = timer_slot(status, true);
    mag::Status* dst = (t && t->host_status) ? t->host_status : out;
    hipError_t e2;
    if ((e2 = hipMemcpyAsync(dst, status, sizeof(mag::Status), hipMemcpyDeviceToHost, stream)) !=
        hipSuccess)
        return hip_fail(e2, "status copy");
    if ((e2 = hipStreamSynchronize(stream)) != hipSuccess) return hip_fail(e2, "synchronize");
    if (dst != out) *out = *dst;
    return MAG_OK;
}

int finish_status(const mag::Status* status, mag_key_stats* per_key, mag_summary* summary,
                  hipStream_t stream)
{
    mag::Status st;
    const int rc = read_status(status, stream, &st);
    if (rc != MAG_OK) return rc;
    return interpret_status(st, per_key, summary);
}

// the end of an asynchronous call: its status block is copied to the pinned
// buffer of the workspace's record on `stream`, and the record keeps that
// stream (and the timing events, when timed) for mag_attribute_finish.
// Without a record, finishing reads the status block from the device.
int async_status(const void* workspace, const mag::Status* status, hipStream_t stream, bool timed)
{
    TimerSlot* t = timer_slot(workspace, true);
    if (!t) return MAG_OK;
    t->pending = timed;
    t->stream = stream;
    if (t->host_status) {
        hipError_t e = hipMemcpyAsync(t->host_status, status, sizeof(mag::Status),
                                      hipMemcpyDeviceToHost, stream);
        if (e != hipSuccess) return hip_fail(e, "status copy");
        if ((e = hipEventRecord(t->done, stream)) != hipSuccess) return hip_fail(e, "event record");
        t->status_pending = true;
    }
    return MAG_OK;
}

struct Job {
    Plan pl{};
    AttrWorkspace w{};
    mag::StreamSet ss{};
    uint32_t flags = 0;
    const double* s = nullptr;
    const double* e = nullptr;
    const uint64_t* keys = nullptr;
    const int32_t* reps = nullptr;  // counter mode: replays per window
    hipEvent_t keys_ready = nullptr;  // a key plan's completion event (external key map)
    double* energy = nullptr;
    int64_t* start_idx = nullptr;
    int64_t* end_idx = nullptr;
    hipStream_t stream = nullptr;

    bool validate() const { return (flags & MAG_SKIP_VALIDATE) == 0; }

    // Tiles [b_begin, b_end) of a trace with `nseg` segments and `NT` tiles
    // (any larger value while the trace's end is unknown); sample g of the
    // trace is t[g - base], P[g - base].
    hipError_t run_tiles(const double* t, const float* P, int64_t base, int64_t b_begin,
                         int64_t b_end, int64_t nseg, int64_t NT, hipEvent_t ev_start = nullptr,
                         hipEvent_t ev_stop = nullptr)
    {
        if (b_end <= b_begin) return hipSuccess;
        mag::TileParams tp{};
        tp.t = t;
        tp.P = P;
        tp.base = base;
        tp.nseg = nseg;
        tp.n_total = nseg + 1;
        tp.tile_begin = b_begin;
        tp.tile_end = b_end;
        tp.NT = NT;
        tp.ld = pl.NT;
        tp.s = s;
        tp.e = e;
        tp.ss = ss;
        tp.energy = energy;
        tp.start_idx = start_idx;
        tp.end_idx = end_idx;
        tp.cnt = w.cnt;
        tp.cnt_fin = w.cnt_fin;
        tp.head = w.head;
        tp.tail = w.tail;
        tp.status = w.status;
        tp.part = w.part;
        tp.split = (flags & MAG_EQUAL_SPLIT) ? 1 : 0;
        tp.validate = validate() ? 1 : 0;
        // vector loads need 16-byte aligned rows: aligned arrays and a base at a
        // multiple of 4 samples (every tile starts at a multiple of TILE)
        tp.aligned16 = (aligned(t, 16) && aligned(P, 16) && (base % 4) == 0) ? 1 : 0;
        return mag::launch_tile(tp, stream, ev_start, ev_stop);
    }

    // cross-tile intervals, endpoints outside the trace; the group-by state is
    // cleared in the same launch when a grouping follows
    hipError_t fixups(int64_t n_samples, int64_t NT, bool grouping)
    {
        mag::FixParams fp{};
        fp.s = s;
        fp.e = e;
        fp.ss = ss;
        fp.NT = NT;
        fp.ld = pl.NT;
        fp.n_total = n_samples;
        fp.cnt = w.cnt;
        fp.cnt_fin = w.cnt_fin;
        fp.head = w.head;
        fp.tail = w.tail;
        fp.energy = energy;
        fp.start_idx = start_idx;
        fp.end_idx = end_idx;
        fp.status = w.status;
        fp.part = w.part;
        fp.fold = w.fold;
        fp.validate = validate() ? 1 : 0;
        if (grouping && pl.m > 0 && pl.H > 0 && !pl.ext_keys) {
            fp.table = w.table;
            fp.H = pl.H;
            fp.urank = w.urank;
        }
        return mag::launch_fix(fp, stream);
    }

    hipError_t grouping(uint64_t* keys_out, mag_key_stats* per_key)
    {
        if (pl.m == 0 || !per_key) {
            // no aggregation: one workgroup adds up the energies and the fold
            const hipError_t e2 = mag::launch_energy_total(energy, pl.m, w.fold, w.status, stream);
            if (e2 != hipSuccess || pl.m > 0) return e2;
            return (per_key && per_key->n_keys_device)
                       ? mag::launch_set_i64(per_key->n_keys_device, 0, stream)
                       : hipSuccess;
        }
        mag::GroupParams gp{};
        gp.keys = keys;
        gp.energy = energy;
        gp.m = pl.m;
        gp.H = pl.H;
        gp.cap = pl.cap;
        gp.nchunks = pl.nchunks;
        gp.chunk = pl.chunk;
        gp.table = w.table;
        gp.slot = w.slot;
        gp.ukey = w.ukey;
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
        gp.kstat = w.kstat;
        gp.ctot = w.ctot;
        gp.fold = w.fold;  // NULL in the counter mode: its fold kernel sets those totals
        gp.n_keys_out = per_key->n_keys_device;
        if (pl.lat) {
            gp.s = s;
            gp.e = e;
            gp.reps = reps;
            gp.dur_out = per_key->duration;
            gp.pdur = w.pdur;
        }
        if (!pl.ext_keys) return mag::launch_groupby(gp, stream);
        if (keys_ready) {
            const hipError_t e2 = hipStreamWaitEvent(stream, keys_ready, 0);
            if (e2 != hipSuccess) return e2;
        }
        return mag::launch_aggregate(gp, stream);
    }

    // read the status block back and turn it into the call's result
    int conclude(mag_key_stats* per_key, mag_summary* summary)
    {
        return finish_status(w.status, per_key, summary, stream);
    }
};

int check_key_outputs(const uint64_t* keys_out, const mag_key_stats* per_key, uint32_t flags)
{
    if (per_key->capacity < 1) return fail(MAG_E_SIZE, "per_key->capacity must be >= 1");
    if (!keys_out || !per_key->sum || !per_key->m2 || !per_key->count)
        return fail(MAG_E_NULL, "per-key output array is NULL");
    if ((flags & MAG_KEY_LATENCY) && !per_key->duration)
        return fail(MAG_E_NULL, "per_key->duration is NULL with MAG_KEY_LATENCY");
    if (!aligned(keys_out, 8) || !aligned(per_key->sum, 8) || !aligned(per_key->m2, 8) ||
        !aligned(per_key->count, 8) || !aligned(per_key->duration, 8) ||
        !aligned(per_key->n_keys_device, 8))
        return fail(MAG_E_ALIGN, "per-key output array not aligned to its element size");
    return MAG_OK;
}

// checks, planning and carving shared by mag_attribute and mag_stream_begin
int prepare(Job& job, int64_t n_samples, const double* starts, const double* ends,
            const uint64_t* op_keys, int64_t n_intervals, const mag_attr_opts* opts,
            mag_interval_out* per_interval, int64_t key_capacity, void* workspace,
            size_t workspace_bytes, hipStream_t stream, bool streaming)
{
    int rc = plan_attribution(job.pl, n_samples, n_intervals, key_capacity, opts, streaming,
                              &job.flags, &job.ss);
    if (rc) return rc;
    if (n_intervals > 0 && (!starts || !ends)) return fail(MAG_E_NULL, "starts/ends is NULL");
    if (key_capacity > 0 && n_intervals > 0 && !op_keys) return fail(MAG_E_NULL, "op_keys is NULL");
    if (!workspace) return fail(MAG_E_NULL, "workspace is NULL");
    if (!aligned(workspace, 256)) return fail(MAG_E_WORKSPACE, "workspace must be 256-byte aligned");
    if ((starts && !aligned(starts, 8)) || (ends && !aligned(ends, 8)) ||
        (op_keys && !aligned(op_keys, 8)))
        return fail(MAG_E_ALIGN, "interval array not aligned to its element size");
    if (per_interval && ((per_interval->energy && !aligned(per_interval->energy, 8)) ||
                         (per_interval->start_idx && !aligned(per_interval->start_idx, 8)) ||
                         (per_interval->end_idx && !aligned(per_interval->end_idx, 8))))
        return fail(MAG_E_ALIGN, "per-interval output not aligned to its element size");
    const size_t need = carve(job.pl, nullptr, job.w);
    if (workspace_bytes < need) {
        snprintf(g_last_error, sizeof(g_last_error), "workspace needs %zu bytes, got %zu", need,
                 workspace_bytes);
        return MAG_E_WORKSPACE;
    }
    carve(job.pl, workspace, job.w);
    if (job.pl.ext_keys) {
        // the key map of a plan built beforehand for these keys and capacity
        const mag_key_plan* kp = opts->key_plan;
        if (!kp->buffer) return fail(MAG_E_NULL, "key_plan->buffer is NULL");
        if (!aligned(kp->buffer, 256))
            return fail(MAG_E_WORKSPACE, "key_plan->buffer must be 256-byte aligned");
        if (kp->n_intervals != n_intervals || kp->key_capacity != key_capacity)
            return fail(MAG_E_STATE, "key plan built for another interval count or key capacity");
        AttrWorkspace pw{};
        if (kp->bytes < carve_key_plan(n_intervals, key_capacity, nullptr, pw))
            return fail(MAG_E_WORKSPACE, "key plan buffer too small");
        carve_key_plan(n_intervals, key_capacity, kp->buffer, job.w);
        job.keys_ready = kp->ready;
    }
    job.s = starts;
    job.e = ends;
    job.keys = op_keys;
    job.energy = (per_interval && per_interval->energy) ? per_interval->energy : job.w.energy;
    job.start_idx = per_interval ? per_interval->start_idx : nullptr;
    job.end_idx = per_interval ? per_interval->end_idx : nullptr;
    job.stream = stream;
    return MAG_OK;
}

}  // namespace

namespace {

int plan_counter(Plan& pl, int64_t n_samples, int64_t n_intervals, int64_t key_capacity,
                 uint32_t flags)
{
    if (n_samples < 2) return fail(MAG_E_SIZE, "n_samples must be >= 2");
    if (n_samples > MAG_MAX_SAMPLES) return fail(MAG_E_SIZE, "n_samples exceeds MAG_MAX_SAMPLES");
    if (n_intervals < 0 || key_capacity < 0) return fail(MAG_E_SIZE, "negative size");
    if (key_capacity > MAG_MAX_KEYS) return fail(MAG_E_SIZE, "key_capacity exceeds MAG_MAX_KEYS");
    pl = Plan{};
    pl.n = n_samples;
    pl.m = n_intervals;
    pl.S = 1;
    // NT: chunks of windows, one wave each (at least one, which checks the readings)
    pl.NT = std::max<int64_t>(1, (n_intervals + mag::CNT_CHUNK - 1) / mag::CNT_CHUNK);
    pl.cap = key_capacity;
    pl.H = 0;
    pl.staging = false;
    pl.lat = key_capacity > 0 && (flags & MAG_KEY_LATENCY) != 0;
    if (key_capacity > 0) plan_groupby(pl);
    return MAG_OK;
}

}  // namespace

extern "C" {

int mag_attribute_workspace_size(int64_t n_samples, int64_t n_intervals, int64_t key_capacity,
                                 const mag_attr_opts* opts, size_t* bytes)
{
    g_last_error[0] = 0;
    if (!bytes) return fail(MAG_E_NULL, "bytes is NULL");
    Plan pl;
    uint32_t flags;
    int rc = plan_attribution(pl, n_samples, n_intervals, key_capacity, opts, false, &flags,
                              nullptr);
    if (rc) return rc;
    AttrWorkspace w{};
    *bytes = carve(pl, nullptr, w);
    return MAG_OK;
}

}  // extern "C"

namespace {

// mag_attribute and its allocation-free variant: with no_alloc the status
// block is read back through a plain host copy (no pinned buffer, no events)
int attribute_impl(const double* timestamps, const float* power, int64_t n_samples,
                   const double* starts, const double* ends, const uint64_t* op_keys,
                   int64_t n_intervals, const mag_attr_opts* opts, mag_interval_out* per_interval,
                   uint64_t* keys_out, mag_key_stats* per_key, mag_summary* summary,
                   void* workspace, size_t workspace_bytes, hipStream_t stream, bool no_alloc)
{
    int rc;
    if (per_key && (rc = check_key_outputs(keys_out, per_key, opts ? opts->flags : 0u)) != MAG_OK)
        return rc;
    Job job;
    rc = prepare(job, n_samples, starts, ends, op_keys, n_intervals, opts, per_interval,
                 per_key ? per_key->capacity : 0, workspace, workspace_bytes, stream, false);
    if (rc) return rc;

    hipError_t e;
    const int64_t NT = job.pl.NT;
    // timing (MAG_TIME_KERNELS): events 1 and 2 travel with the tile kernel's
    // dispatch, event 3 follows the call's last kernel
    EventTimer timer(!no_alloc && (job.flags & MAG_TIME_KERNELS) != 0, stream, workspace);
    if ((e = mag::launch_init(job.w.status, job.w.cnt_fin, (int64_t)job.pl.S * (NT + 1),
                              timestamps, n_samples, stream)) != hipSuccess)
        return hip_fail(e, "init");
    if (opts && opts->tiles_wait && (e = hipStreamWaitEvent(stream, opts->tiles_wait, 0)) != hipSuccess)
        return hip_fail(e, "tiles_wait event");
    if ((e = job.run_tiles(timestamps, power, 0, 0, NT, n_samples - 1, NT,
                           timer.on ? timer.slot->ev[1] : nullptr,
                           timer.on ? timer.slot->ev[2] : nullptr)) != hipSuccess)
        return hip_fail(e, "tile kernel");
    if (opts && opts->tiles_done && (e = hipEventRecord(opts->tiles_done, stream)) != hipSuccess)
        return hip_fail(e, "tiles_done event");
    if (opts && opts->group_stream && opts->group_stream != stream) {
        // everything after the trace integration moves to the group stream,
        // which first waits for the integration
        TimerSlot* ts = timer_slot(workspace, true);
        if (!ts || !ts->split) return fail(MAG_E_HIP, "no event for the group stream");
        if ((e = hipEventRecord(ts->split, stream)) != hipSuccess ||
            (e = hipStreamWaitEvent(opts->group_stream, ts->split, 0)) != hipSuccess)
            return hip_fail(e, "group stream event");
        stream = opts->group_stream;
        job.stream = stream;
        timer.stream = stream;
    }
    if ((e = job.fixups(n_samples, NT, per_key != nullptr)) != hipSuccess)
        return hip_fail(e, "fix-up kernels");
    if (opts && opts->intervals_ready &&
        (e = hipEventRecord(opts->intervals_ready, stream)) != hipSuccess)
        return hip_fail(e, "intervals_ready event");
    if ((e = job.grouping(keys_out, per_key)) != hipSuccess) return hip_fail(e, "group-by");
    timer.mark(3);
    if (no_alloc) {
        mag::Status st;
        if ((e = hipMemcpyAsync(&st, job.w.status, sizeof(mag::Status), hipMemcpyDeviceToHost,
                                stream)) != hipSuccess)
            return hip_fail(e, "status copy");
        if ((e = hipStreamSynchronize(stream)) != hipSuccess) return hip_fail(e, "synchronize");
        rc = interpret_status(st, per_key, summary);
        if (summary) summary->tile_kernel_ms = summary->device_ms = 0.0;
        return rc;
    }
    if (job.flags & MAG_ASYNC)
        // results, errors and timings come from mag_attribute_finish; the status
        // block is copied to pinned host memory now, so that finishing needs
        // no further device work
        return async_status(workspace, job.w.status, stream, timer.on);
    rc = job.conclude(per_key, summary);
    if (summary) {
        summary->tile_kernel_ms = timer.ms(1, 2);
        summary->device_ms = timer.ms(1, 3);
    }
    return rc;
}

// The allocation-free entry point's scratch memory: one copy per GPU, in the
// library's code object, held until the process ends.  Host code never passes
// this symbol itself to a kernel (in host code it names a host-side stand-in):
// the device address of each GPU's copy is looked up once per device with
// that device current, and only that address is used.
constexpr size_t STATIC_SCRATCH_BYTES = (size_t)MAG_STATIC_SCRATCH_BYTES;
__device__ __align__(256) unsigned char scratch[STATIC_SCRATCH_BYTES];

constexpr int SCRATCH_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[SCRATCH_DEVICES] = {};

int scratch_address(void** out)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= SCRATCH_DEVICES) return fail(MAG_E_STATE, "device index out of range");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_addr[dev]) {
        void* p = nullptr;
        if ((e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) != hipSuccess)
            return hip_fail(e, "scratch address");
        if (!p || !aligned(p, 256)) return fail(MAG_E_STATE, "scratch address not 256-byte aligned");
        g_scratch_addr[dev] = p;
    }
    *out = g_scratch_addr[dev];
    return MAG_OK;
}

}  // namespace

extern "C" {

int mag_attribute(const double* timestamps, const float* power, int64_t n_samples,
                  const double* starts, const double* ends, const uint64_t* op_keys,
                  int64_t n_intervals, const mag_attr_opts* opts, mag_interval_out* per_interval,
                  uint64_t* keys_out, mag_key_stats* per_key, mag_summary* summary, void* workspace,
                  size_t workspace_bytes, hipStream_t stream)
{
    g_last_error[0] = 0;
    if (!timestamps || !power) return fail(MAG_E_NULL, "timestamps/power is NULL");
    if (!aligned(timestamps, 8) || !aligned(power, 4))
        return fail(MAG_E_ALIGN, "input array not aligned to its element size");
    if (unfinished(workspace))
        return fail(MAG_E_STATE, "an asynchronous call on this workspace is not finished");
    return attribute_impl(timestamps, power, n_samples, starts, ends, op_keys, n_intervals, opts,
                          per_interval, keys_out, per_key, summary, workspace, workspace_bytes,
                          stream, false);
}

int mag_attribute_static(const double* timestamps, const float* power, int64_t n_samples,
                         const double* starts, const double* ends, const uint64_t* op_keys,
                         int64_t n_intervals, const mag_attr_opts* opts,
                         mag_interval_out* per_interval, uint64_t* keys_out,
                         mag_key_stats* per_key, mag_summary* summary, hipStream_t stream)
{
    g_last_error[0] = 0;
    if (!timestamps || !power) return fail(MAG_E_NULL, "timestamps/power is NULL");
    if (!aligned(timestamps, 8) || !aligned(power, 4))
        return fail(MAG_E_ALIGN, "input array not aligned to its element size");
    if (opts && ((opts->flags & (MAG_ASYNC | MAG_TIME_KERNELS)) || opts->group_stream))
        return fail(MAG_E_STATE, "MAG_ASYNC, MAG_TIME_KERNELS and group_stream need host "
                                 "resources: not accepted by the allocation-free entry point");
    size_t need = 0;
    int rc = mag_attribute_workspace_size(n_samples, n_intervals,
                                          per_key ? per_key->capacity : 0, opts, &need);
    if (rc != MAG_OK) return rc;
    if (need > STATIC_SCRATCH_BYTES) {
        snprintf(g_last_error, sizeof(g_last_error),
                 "these sizes need %zu bytes of scratch; the allocation-free entry point has %zu",
                 need, STATIC_SCRATCH_BYTES);
        return MAG_E_WORKSPACE;
    }
    void* ws = nullptr;
    if ((rc = scratch_address(&ws)) != MAG_OK) return rc;
    return attribute_impl(timestamps, power, n_samples, starts, ends, op_keys, n_intervals, opts,
                          per_interval, keys_out, per_key, summary, ws, STATIC_SCRATCH_BYTES,
                          stream, true);
}

int mag_key_plan_size(int64_t n_intervals, int64_t key_capacity, size_t* bytes)
{
    g_last_error[0] = 0;
    if (!bytes) return fail(MAG_E_NULL, "bytes is NULL");
    if (n_intervals < 0 || key_capacity < 1) return fail(MAG_E_SIZE, "n_intervals < 0 or key_capacity < 1");
    if (key_capacity > MAG_MAX_KEYS) return fail(MAG_E_SIZE, "key_capacity exceeds MAG_MAX_KEYS");
    AttrWorkspace w{};
    *bytes = carve_key_plan(n_intervals, key_capacity, nullptr, w);
    return MAG_OK;
}

int mag_key_plan_build(const uint64_t* op_keys, int64_t n_intervals, int64_t key_capacity,
                       mag_key_plan* plan, hipStream_t stream)
{
    g_last_error[0] = 0;
    if (!plan || !plan->buffer) return fail(MAG_E_NULL, "plan/plan->buffer is NULL");
    if (n_intervals > 0 && !op_keys) return fail(MAG_E_NULL, "op_keys is NULL");
    if (op_keys && !aligned(op_keys, 8)) return fail(MAG_E_ALIGN, "op_keys not 8-byte aligned");
    if (!aligned(plan->buffer, 256))
        return fail(MAG_E_WORKSPACE, "plan->buffer must be 256-byte aligned");
    size_t need = 0;
    int rc = mag_key_plan_size(n_intervals, key_capacity, &need);
    if (rc) return rc;
    if (plan->bytes < need) {
        snprintf(g_last_error, sizeof(g_last_error), "key plan needs %zu bytes, got %zu", need,
                 plan->bytes);
        return MAG_E_WORKSPACE;
    }
    AttrWorkspace w{};
    carve_key_plan(n_intervals, key_capacity, plan->buffer, w);
    mag::GroupParams gp{};
    gp.keys = op_keys;
    gp.m = n_intervals;
    gp.H = hash_slots(key_capacity);
    gp.cap = key_capacity;
    gp.table = w.table;
    gp.slot = w.slot;
    gp.ukey = w.ukey;
    gp.urank = w.urank;
    gp.status = w.kstat;
    gp.kstat = w.kstat;
    hipError_t e;
    if ((e = mag::launch_key_map(gp, true, stream)) != hipSuccess) return hip_fail(e, "key map");
    if (plan->ready && (e = hipEventRecord(plan->ready, stream)) != hipSuccess)
        return hip_fail(e, "key plan event");
    plan->n_intervals = n_intervals;
    plan->key_capacity = key_capacity;
    return MAG_OK;
}

int mag_counter_workspace_size(int64_t n_samples, int64_t n_intervals, int64_t key_capacity,
                               uint32_t flags, size_t* bytes)
{
    g_last_error[0] = 0;
    if (!bytes) return fail(MAG_E_NULL, "bytes is NULL");
    Plan pl;
    int rc = plan_counter(pl, n_samples, n_intervals, key_capacity, flags);
    if (rc) return rc;
    AttrWorkspace w{};
    *bytes = carve_counter(pl, nullptr, w);
    return MAG_OK;
}

int mag_attribute_counter(const double* timestamps, const double* counter, int64_t n_samples,
                          double delay, const double* starts, const double* ends,
                          const int32_t* replays, const uint64_t* op_keys, int64_t n_intervals,
                          uint32_t flags, mag_interval_out* per_interval, uint64_t* keys_out,
                          mag_key_stats* per_key, mag_summary* summary, void* workspace,
                          size_t workspace_bytes, hipStream_t stream)
{
    g_last_error[0] = 0;
    if (!timestamps || !counter) return fail(MAG_E_NULL, "timestamps/counter is NULL");
    if (!aligned(timestamps, 8) || !aligned(counter, 8))
        return fail(MAG_E_ALIGN, "input array not aligned to its element size");
    if (!(delay - delay == 0.0)) return fail(MAG_E_TIMESTAMPS, "delay is not finite");
    if (unfinished(workspace))
        return fail(MAG_E_STATE, "an asynchronous call on this workspace is not finished");
    int rc;
    if (per_key && (rc = check_key_outputs(keys_out, per_key, flags)) != MAG_OK) return rc;
    Job job;
    const int64_t cap = per_key ? per_key->capacity : 0;
    if ((rc = plan_counter(job.pl, n_samples, n_intervals, cap, flags)) != MAG_OK) return rc;
    if (n_intervals > 0 && (!starts || !ends)) return fail(MAG_E_NULL, "starts/ends is NULL");
    if (cap > 0 && n_intervals > 0 && !op_keys) return fail(MAG_E_NULL, "op_keys is NULL");
    if (!workspace) return fail(MAG_E_NULL, "workspace is NULL");
    if (!aligned(workspace, 256)) return fail(MAG_E_WORKSPACE, "workspace must be 256-byte aligned");
    if ((starts && !aligned(starts, 8)) || (ends && !aligned(ends, 8)) ||
        (op_keys && !aligned(op_keys, 8)) || (replays && !aligned(replays, 4)))
        return fail(MAG_E_ALIGN, "window array not aligned to its element size");
    if (per_interval && ((per_interval->energy && !aligned(per_interval->energy, 8)) ||
                         (per_interval->start_idx && !aligned(per_interval->start_idx, 8)) ||
                         (per_interval->end_idx && !aligned(per_interval->end_idx, 8))))
        return fail(MAG_E_ALIGN, "per-interval output not aligned to its element size");
    const size_t need = carve_counter(job.pl, nullptr, job.w);
    if (workspace_bytes < need) {
        snprintf(g_last_error, sizeof(g_last_error), "workspace needs %zu bytes, got %zu", need,
                 workspace_bytes);
        return MAG_E_WORKSPACE;
    }
    carve_counter(job.pl, workspace, job.w);
    job.flags = flags;
    job.s = starts;
    job.e = ends;
    job.keys = op_keys;
    job.reps = replays;
    job.energy = (per_interval && per_interval->energy) ? per_interval->energy : job.w.energy;
    job.start_idx = per_interval ? per_interval->start_idx : nullptr;
    job.end_idx = per_interval ? per_interval->end_idx : nullptr;
    job.stream = stream;

    mag::CounterParams cp{};
    cp.t = timestamps;
    cp.C = counter;
    cp.n = n_samples;
    cp.delay = delay;
    cp.s = starts;
    cp.e = ends;
    cp.reps = replays;
    cp.m = n_intervals;
    cp.nchunks = job.pl.NT;
    cp.energy = job.energy;
    cp.start_idx = job.start_idx;
    cp.end_idx = job.end_idx;
    cp.part = job.w.part;
    cp.status = job.w.status;
    cp.validate = job.validate() ? 1 : 0;
    if (per_key && n_intervals > 0 && job.pl.H > 0) {
        cp.table = job.w.table;
        cp.H = job.pl.H;
        cp.urank = job.w.urank;
    }

    hipError_t e;
    EventTimer timer((flags & MAG_TIME_KERNELS) != 0, stream, workspace);
    if ((e = mag::launch_init_status(job.w.status, nullptr, 0, stream)) != hipSuccess)
        return hip_fail(e, "init");
    if ((e = mag::launch_counter(cp, stream, timer.on ? timer.slot->ev[1] : nullptr,
                                 timer.on ? timer.slot->ev[2] : nullptr)) != hipSuccess)
        return hip_fail(e, "counter kernel");
    if ((e = mag::launch_counter_fold(cp, stream)) != hipSuccess) return hip_fail(e, "fold kernel");
    if ((e = job.grouping(keys_out, per_key)) != hipSuccess) return hip_fail(e, "group-by");
    timer.mark(3);
    if (flags & MAG_ASYNC) return async_status(workspace, job.w.status, stream, timer.on);
    rc = job.conclude(per_key, summary);
    if (summary) {
        summary->tile_kernel_ms = timer.ms(1, 2);
        summary->device_ms = timer.ms(1, 3);
    }
    return rc;
}

int mag_attribute_finish(const void* workspace, mag_key_stats* per_key, mag_summary* summary,
                         hipStream_t stream)
{
    g_last_error[0] = 0;
    if (!workspace) return fail(MAG_E_NULL, "workspace is NULL");
    if (!aligned(workspace, 256)) return fail(MAG_E_WORKSPACE, "workspace must be 256-byte aligned");
    // the status block is the first piece of every attribution workspace
    TimerSlot* t = timer_slot(workspace, false);
    int rc;
    if (t && t->status_pending && t->host_status) {
        // the call already copied its status to pinned memory on its own
        // stream (which may differ from `stream`) and recorded an event
        // after the copy: that event is waited for, not later work
        t->status_pending = false;
        hipError_t e2;
        if ((e2 = hipEventSynchronize(t->done)) != hipSuccess) {
            t->pending = false;
            return hip_fail(e2, "synchronize");
        }
        rc = interpret_status(*t->host_status, per_key, summary);
    } else {
        rc = finish_status(static_cast<const mag::Status*>(workspace), per_key, summary, stream);
        t = timer_slot(workspace, false);
    }
    if (summary) {
        summary->tile_kernel_ms = 0.0;
        summary->device_ms = 0.0;
    }
    if (t && t->pending) {
        t->pending = false;
        float v = 0.0f;
        // best effort, as in EventTimer: a failure reads as zero and is cleared
        if (summary) {
            if (hipEventElapsedTime(&v, t->ev[1], t->ev[2]) == hipSuccess)
                summary->tile_kernel_ms = (double)v;
            else
                (void)hipGetLastError();
            if (hipEventElapsedTime(&v, t->ev[1], t->ev[3]) == hipSuccess)
                summary->device_ms = (double)v;
            else
                (void)hipGetLastError();
        }
    }
    return rc;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// chunked streaming
//
// The trace arrives as consecutive chunks.  Tiles are the same as in the
// one-shot call (tile b covers samples b*TILE .. b*TILE + TILE); a tile whose
// samples all lie in one chunk runs in place, a tile spanning two or more
// chunks is assembled in a staging buffer first.  A tile runs only once a
// sample beyond it has arrived, so the trace's last tile (the only one that
// may be short, and the one that records the final cursors) runs at the end.
// Everything carried from chunk to chunk lives in the workspace: per-tile
// cursors and partial energies, the staging buffer and the status block.
// ---------------------------------------------------------------------------

struct mag_stream {
    Job job;
    int64_t received = 0;  // samples pushed so far
    int64_t b_next = 0;    // first tile not yet run
    int64_t n_stage = 0;   // samples held in staging, from sample b_next * TILE on
    int failed = 0;        // a launch failed: the handle only accepts end/abort
    // chunks pushed from host memory: two device halves of the caller's
    // staging buffer, filled in turn on the copy stream
    struct HostHalf {
        double* t = nullptr;
        float* P = nullptr;
        hipEvent_t copied = nullptr;  // the half's copy is complete (copy stream)
        hipEvent_t freed = nullptr;   // the half's samples are consumed (compute stream)
        bool copied_rec = false;      // the events have been recorded at least once
        bool freed_rec = false;
    } half[2];
    int64_t host_chunk = 0;   // most samples one host chunk may hold (0: no staging)
    int next_half = 0;
    hipStream_t copy_stream = nullptr;
    ~mag_stream()
    {
        for (auto& x : half) {
            if (x.copied) (void)hipEventDestroy(x.copied);
            if (x.freed) (void)hipEventDestroy(x.freed);
        }
    }
};

namespace {

constexpr uint64_t STATE_MAGIC = 0x314554415453474dull;  // "MGSTATE1"

struct StateHeader {
    uint64_t magic;
    int64_t max_samples, n_intervals, key_capacity;
    int32_t n_streams;
    uint32_t flags;
    int64_t received, b_next, n_stage;
    uint32_t has_energy, has_start, has_end, pad;
    uint64_t bytes_total;
};

// device regions of the carried state, in checkpoint order
struct Region {
    void* ptr;
    size_t bytes;
};

int state_regions(const mag_stream* h, Region* r)
{
    const Job& j = h->job;
    const size_t S = (size_t)j.pl.S, ld = (size_t)j.pl.NT, m = (size_t)j.pl.m;
    int k = 0;
    r[k++] = {j.w.status, sizeof(mag::Status)};
    r[k++] = {j.w.cnt, sizeof(int64_t) * S * (ld + 1)};
    r[k++] = {j.w.cnt_fin, sizeof(int64_t) * S * (ld + 1)};
    r[k++] = {j.w.head, sizeof(double) * S * ld};
    r[k++] = {j.w.tail, sizeof(double) * S * ld};
    r[k++] = {j.w.part, sizeof(double2) * ld};
    r[k++] = {j.w.stage_t, sizeof(double) * (mag::TILE + 1)};
    r[k++] = {j.w.stage_P, sizeof(float) * (mag::TILE + 1)};
    r[k++] = {j.energy, sizeof(double) * m};
    if (j.start_idx) r[k++] = {j.start_idx, sizeof(int64_t) * m};
    if (j.end_idx) r[k++] = {j.end_idx, sizeof(int64_t) * m};
    return k;
}

size_t state_bytes(const mag_stream* h)
{
    Region r[16];
    const int k = state_regions(h, r);
    size_t b = sizeof(StateHeader);
    for (int i = 0; i < k; ++i) b += r[i].bytes;
    return b;
}

}  // namespace

namespace {

// the candidate slots and per-workgroup counts of one comparison
void carve_candidates(Carver& c, int64_t na, int64_t k, mag::DiffParams* p)
{
    const int64_t groups = mag::diff_groups(na);
    const int64_t slots = mag::diff_max_candidates(na, k);
    const size_t nc = (size_t)std::max<int64_t>(slots, 1);
    double* r = c.take<double>(nc);
    uint64_t* key = c.take<uint64_t>(nc);
    int32_t* ia = c.take<int32_t>(nc);
    int32_t* ib = c.take<int32_t>(nc);
    uint32_t* rank = c.take<uint32_t>(nc);
    uint32_t* blk = c.take<uint32_t>(8 * (size_t)groups);
    if (p) {
        p->cand_r = r;
        p->cand_key = key;
        p->cand_ia = ia;
        p->cand_ib = ib;
        p->cand_rank = rank;
        p->blk = blk;
        p->n_groups = groups;
        p->n_slots = slots;
    }
}

}  // namespace

extern "C" {

int mag_stream_workspace_size(int64_t max_samples, int64_t n_intervals, int64_t key_capacity,
                              const mag_attr_opts* opts, size_t* bytes)
{
    g_last_error[0] = 0;
    if (!bytes) return fail(MAG_E_NULL, "bytes is NULL");
    Plan pl;
    uint32_t flags;
    int rc = plan_attribution(pl, max_samples, n_intervals, key_capacity, opts, true, &flags,
                              nullptr);
    if (rc) return rc;
    AttrWorkspace w{};
    *bytes = carve(pl, nullptr, w);
    return MAG_OK;
}

int mag_stream_begin(mag_stream** handle, int64_t max_samples, const double* starts,
                     const double* ends, const uint64_t* op_keys, int64_t n_intervals,
                     const mag_attr_opts* opts, mag_interval_out* per_interval,
                     int64_t key_capacity, void* workspace, size_t workspace_bytes,
                     hipStream_t stream)
{
    g_last_error[0] = 0;
    if (!handle) return fail(MAG_E_NULL, "handle is NULL");
    *handle = nullptr;
    mag_stream* h = new (std::nothrow) mag_stream();
    if (!h) return fail(MAG_E_STATE, "out of host memory");
    int rc = prepare(h->job, max_samples, starts, ends, op_keys, n_intervals, opts, per_interval,
                     key_capacity, workspace, workspace_bytes, stream, true);
    if (rc) {
        delete h;
        return rc;
    }
    const hipError_t e = mag::launch_init(h->job.w.status, h->job.w.cnt_fin,
                                          (int64_t)h->job.pl.S * (h->job.pl.NT + 1), nullptr, 0,
                                          stream);
    if (e != hipSuccess) {
        delete h;
        return hip_fail(e, "init");
    }
    *handle = h;
    return MAG_OK;
}

int mag_stream_push(mag_stream* h, const double* t_chunk, const float* p_chunk, int64_t n_chunk)
{
    g_last_error[0] = 0;
    if (!h) return fail(MAG_E_NULL, "handle is NULL");
    if (h->failed) return fail(MAG_E_STATE, "a previous call on this stream failed");
    if (n_chunk < 0) return fail(MAG_E_SIZE, "n_chunk must be >= 0");
    if (n_chunk == 0) return MAG_OK;
    if (!t_chunk || !p_chunk) return fail(MAG_E_NULL, "chunk pointer is NULL");
    if (!aligned(t_chunk, 8) || !aligned(p_chunk, 4))
        return fail(MAG_E_ALIGN, "chunk not aligned to its element size");
    Job& job = h->job;
    const int64_t T = mag::TILE;
    const int64_t g0 = h->received, g1 = g0 + n_chunk;
    if (g1 > job.pl.n) return fail(MAG_E_SIZE, "more samples pushed than max_samples");
    const hipStream_t st = job.stream;
    const int64_t unknown_end = job.pl.NT + 1;  // tile count while the end is unknown
    const int64_t full = (int64_t)1 << 62;       // segment count while the end is unknown
    hipError_t e = hipSuccess;
    auto bad = [&](const char* where) {
        h->failed = 1;
        return hip_fail(e, where);
    };
    auto stage = [&](int64_t at, int64_t from, int64_t count) {
        // chunk samples [from, from + count) into staging slots [at, at + count)
        return mag::launch_stage_copy(job.w.stage_t + at, t_chunk + (from - g0),
                                      job.w.stage_P + at, p_chunk + (from - g0), count, st);
    };
    if (g0 == 0 &&
        (e = hipMemcpyAsync(&job.w.status->bounds[0], t_chunk, sizeof(double),
                            hipMemcpyDeviceToDevice, st)) != hipSuccess)
        return bad("bounds copy");

    int64_t pos = g0;  // first sample of this chunk not yet consumed
    while (h->n_stage > 0) {
        // complete the staged tile b_next
        const int64_t take = std::min<int64_t>(T + 1 - h->n_stage, g1 - pos);
        if (take > 0) {
            if ((e = stage(h->n_stage, pos, take)) != hipSuccess) return bad("staging copy");
            h->n_stage += take;
            pos += take;
        }
        if (h->n_stage < T + 1 || pos >= g1) {
            h->received = g1;  // wait for more samples
            return MAG_OK;
        }
        const int64_t b = h->b_next;
        if ((e = job.run_tiles(job.w.stage_t, job.w.stage_P, b * T, b, b + 1, full,
                               unknown_end)) != hipSuccess)
            return bad("tile kernel");
        h->b_next = b + 1;
        if (pos - 1 >= g0) {
            // the next tile starts inside this chunk
            h->n_stage = 0;
            pos -= 1;
        } else {
            // its first sample is the staged tile's last one
            if ((e = mag::launch_stage_copy(job.w.stage_t, job.w.stage_t + T, job.w.stage_P,
                                            job.w.stage_P + T, 1, st)) != hipSuccess)
                return bad("staging copy");
            h->n_stage = 1;
        }
    }
    // pos == b_next * TILE lies in this chunk: run in place every tile with a
    // sample after it in this chunk (tile b needs b*T + T + 1 <= g1 - 1)
    const int64_t b0 = h->b_next;
    int64_t b1 = b0;
    if (g1 - 2 - T >= 0) b1 = std::max<int64_t>(b0, (g1 - 2 - T) / T + 1);
    if (b1 > b0) {
        if ((e = job.run_tiles(t_chunk, p_chunk, g0, b0, b1, full, unknown_end)) != hipSuccess)
            return bad("tile kernel");
        h->b_next = b1;
    }
    const int64_t first = h->b_next * T;
    if ((e = stage(0, first, g1 - first)) != hipSuccess) return bad("staging copy");
    h->n_stage = g1 - first;
    h->received = g1;
    return MAG_OK;
}

int mag_stream_host_staging_size(int64_t max_chunk, size_t* bytes)
{
    g_last_error[0] = 0;
    if (!bytes) return fail(MAG_E_NULL, "bytes is NULL");
    if (max_chunk < 1) return fail(MAG_E_SIZE, "max_chunk must be >= 1");
    if (max_chunk > MAG_MAX_SAMPLES) return fail(MAG_E_SIZE, "max_chunk exceeds MAG_MAX_SAMPLES");
    Carver c;
    for (int i = 0; i < 2; ++i) {
        c.take<double>((size_t)max_chunk);
        c.take<float>((size_t)max_chunk);
    }
    *bytes = c.off;
    return MAG_OK;
}

int mag_stream_set_host_staging(mag_stream* h, int64_t max_chunk, void* staging,
                                size_t staging_bytes, hipStream_t copy_stream)
{
    g_last_error[0] = 0;
    if (!h || !staging) return fail(MAG_E_NULL, "handle/staging is NULL");
    if (h->failed) return fail(MAG_E_STATE, "a previous call on this stream failed");
    if (h->host_chunk > 0) return fail(MAG_E_STATE, "host staging is already set");
    if (copy_stream == h->job.stream)
        return fail(MAG_E_STATE, "the copy stream must differ from the stream's compute stream");
    size_t need = 0;
    int rc = mag_stream_host_staging_size(max_chunk, &need);
    if (rc) return rc;
    if (!aligned(staging, 256)) return fail(MAG_E_WORKSPACE, "staging must be 256-byte aligned");
    if (staging_bytes < need) {
        snprintf(g_last_error, sizeof(g_last_error), "staging needs %zu bytes, got %zu", need,
                 staging_bytes);
        return MAG_E_WORKSPACE;
    }
    Carver c;
    c.base = static_cast<char*>(staging);
    for (auto& x : h->half) {
        x.t = c.take<double>((size_t)max_chunk);
        x.P = c.take<float>((size_t)max_chunk);
        hipError_t e;
        if ((e = hipEventCreateWithFlags(&x.copied, hipEventDisableTiming)) != hipSuccess ||
            (e = hipEventCreateWithFlags(&x.freed, hipEventDisableTiming)) != hipSuccess)
            return hip_fail(e, "staging events");
        x.copied_rec = x.freed_rec = false;
    }
    h->host_chunk = max_chunk;
    h->next_half = 0;
    h->copy_stream = copy_stream;
    return MAG_OK;
}

int mag_stream_push_host(mag_stream* h, const double* t_host, const float* p_host, int64_t n_chunk)
{
    g_last_error[0] = 0;
    if (!h) return fail(MAG_E_NULL, "handle is NULL");
    if (h->failed) return fail(MAG_E_STATE, "a previous call on this stream failed");
    if (h->host_chunk == 0) return fail(MAG_E_STATE, "no host staging set on this stream");
    if (n_chunk < 0) return fail(MAG_E_SIZE, "n_chunk must be >= 0");
    if (n_chunk > h->host_chunk) return fail(MAG_E_SIZE, "chunk larger than the staging holds");
    if (n_chunk == 0) return MAG_OK;
    if (!t_host || !p_host) return fail(MAG_E_NULL, "chunk pointer is NULL");
    if (h->received + n_chunk > h->job.pl.n)
        return fail(MAG_E_SIZE, "more samples pushed than max_samples");
    auto& x = h->half[h->next_half];
    hipError_t e;
    auto bad = [&](const char* where) {
        h->failed = 1;
        return hip_fail(e, where);
    };
    // the host chunk copied into this half two pushes ago is complete, so the
    // caller may reuse its memory once this call returns
    if (x.copied_rec && (e = hipEventSynchronize(x.copied)) != hipSuccess)
        return bad("staging wait");
    // the half's previous samples have been consumed by the compute stream
    if ((x.freed_rec && (e = hipStreamWaitEvent(h->copy_stream, x.freed, 0)) != hipSuccess) ||
        (e = hipMemcpyAsync(x.t, t_host, sizeof(double) * (size_t)n_chunk, hipMemcpyHostToDevice,
                            h->copy_stream)) != hipSuccess ||
        (e = hipMemcpyAsync(x.P, p_host, sizeof(float) * (size_t)n_chunk, hipMemcpyHostToDevice,
                            h->copy_stream)) != hipSuccess ||
        (e = hipEventRecord(x.copied, h->copy_stream)) != hipSuccess)
        return bad("staging copy");
    x.copied_rec = true;
    if ((e = hipStreamWaitEvent(h->job.stream, x.copied, 0)) != hipSuccess)
        return bad("staging wait");
    const int rc = mag_stream_push(h, x.t, x.P, n_chunk);
    if (rc != MAG_OK) return rc;
    if ((e = hipEventRecord(x.freed, h->job.stream)) != hipSuccess) return bad("staging event");
    x.freed_rec = true;
    h->next_half ^= 1;
    return MAG_OK;
}

int mag_stream_end(mag_stream* h, uint64_t* keys_out, mag_key_stats* per_key, mag_summary* summary)
{
    g_last_error[0] = 0;
    if (!h) return fail(MAG_E_NULL, "handle is NULL");
    Job& job = h->job;
    int rc = MAG_OK;
    hipError_t e;
    const int64_t n = h->received;
    const int64_t NT = (n - 1 + mag::TILE - 1) / mag::TILE;
    if (h->failed) {
        rc = fail(MAG_E_STATE, "a previous call on this stream failed");
    } else if (n < 2) {
        rc = fail(MAG_E_SIZE, "fewer than 2 samples pushed");
    } else if (per_key && job.pl.cap == 0) {
        rc = fail(MAG_E_STATE, "per-key outputs requested but key_capacity was 0 at begin");
    } else if (per_key && per_key->capacity != job.pl.cap) {
        rc = fail(MAG_E_SIZE, "per_key->capacity differs from the key_capacity given at begin");
    } else if (per_key && (rc = check_key_outputs(keys_out, per_key, job.flags)) != MAG_OK) {
        // rc set
    } else if ((e = hipMemcpyAsync(&job.w.status->bounds[1], job.w.stage_t + (h->n_stage - 1),
                                   sizeof(double), hipMemcpyDeviceToDevice, job.stream)) !=
               hipSuccess) {
        rc = hip_fail(e, "bounds copy");
    } else if ((e = job.run_tiles(job.w.stage_t, job.w.stage_P, h->b_next * mag::TILE, h->b_next,
                                  NT, n - 1, NT)) != hipSuccess) {
        rc = hip_fail(e, "tile kernel");
    } else if ((e = job.fixups(n, NT, per_key != nullptr)) != hipSuccess) {
        rc = hip_fail(e, "fix-up kernels");
    } else if ((e = job.grouping(keys_out, per_key)) != hipSuccess) {
        rc = hip_fail(e, "group-by");
    } else {
        rc = job.conclude(per_key, summary);
    }
    delete h;
    return rc;
}

void mag_stream_abort(mag_stream* h) { delete h; }

int mag_stream_state_export(const mag_stream* h, void* host_buf, size_t* bytes)
{
    g_last_error[0] = 0;
    if (!h || !bytes) return fail(MAG_E_NULL, "handle/bytes is NULL");
    if (h->failed) return fail(MAG_E_STATE, "a previous call on this stream failed");
    const size_t need = state_bytes(h);
    if (!host_buf) {
        *bytes = need;
        return MAG_OK;
    }
    if (*bytes < need) {
        *bytes = need;
        return fail(MAG_E_SIZE, "state buffer too small");
    }
    const Job& j = h->job;
    StateHeader hd{};
    hd.magic = STATE_MAGIC;
    hd.max_samples = j.pl.n;
    hd.n_intervals = j.pl.m;
    hd.key_capacity = j.pl.cap;
    hd.n_streams = j.pl.S;
    hd.flags = j.flags;
    hd.received = h->received;
    hd.b_next = h->b_next;
    hd.n_stage = h->n_stage;
    hd.has_energy = 1;
    hd.has_start = j.start_idx ? 1 : 0;
    hd.has_end = j.end_idx ? 1 : 0;
    hd.bytes_total = need;
    char* out = static_cast<char*>(host_buf);
    memcpy(out, &hd, sizeof(hd));
    size_t off = sizeof(hd);
    Region r[16];
    const int k = state_regions(h, r);
    hipError_t e;
    for (int i = 0; i < k; ++i) {
        if (r[i].bytes &&
            (e = hipMemcpyAsync(out + off, r[i].ptr, r[i].bytes, hipMemcpyDeviceToHost, j.stream)) !=
                hipSuccess)
            return hip_fail(e, "state copy");
        off += r[i].bytes;
    }
    if ((e = hipStreamSynchronize(j.stream)) != hipSuccess) return hip_fail(e, "synchronize");
    *bytes = need;
    return MAG_OK;
}

int mag_stream_state_import(mag_stream* h, const void* host_buf, size_t bytes)
{
    g_last_error[0] = 0;
    if (!h || !host_buf) return fail(MAG_E_NULL, "handle/host_buf is NULL");
    if (h->failed || h->received != 0)
        return fail(MAG_E_STATE, "state can only be imported into a freshly begun stream");
    StateHeader hd;
    if (bytes < sizeof(hd)) return fail(MAG_E_SIZE, "state buffer too small");
    memcpy(&hd, host_buf, sizeof(hd));
    const Job& j = h->job;
    if (hd.magic != STATE_MAGIC) return fail(MAG_E_STATE, "not a stream state");
    if (hd.max_samples != j.pl.n || hd.n_intervals != j.pl.m || hd.key_capacity != j.pl.cap ||
        hd.n_streams != j.pl.S || hd.flags != j.flags || hd.has_start != (j.start_idx ? 1u : 0u) ||
        hd.has_end != (j.end_idx ? 1u : 0u))
        return fail(MAG_E_STATE, "state was exported from a stream begun with other arguments");
    const size_t need = state_bytes(h);
    if (hd.bytes_total != need || bytes < need) return fail(MAG_E_SIZE, "state buffer size mismatch");
    if (hd.received < 0 || hd.received > j.pl.n || hd.b_next < 0 || hd.n_stage < 0 ||
        hd.n_stage > mag::TILE + 1)
        return fail(MAG_E_STATE, "corrupt stream state");
    const char* in = static_cast<const char*>(host_buf);
    size_t off = sizeof(hd);
    Region r[16];
    const int k = state_regions(h, r);
    hipError_t e;
    for (int i = 0; i < k; ++i) {
        if (r[i].bytes &&
            (e = hipMemcpyAsync(r[i].ptr, in + off, r[i].bytes, hipMemcpyHostToDevice, j.stream)) !=
                hipSuccess)
            return hip_fail(e, "state copy");
        off += r[i].bytes;
    }
    if ((e = hipStreamSynchronize(j.stream)) != hipSuccess) return hip_fail(e, "synchronize");
    h->received = hd.received;
    h->b_next = hd.b_next;
    h->n_stage = hd.n_stage;
    return MAG_OK;
}

int mag_diff_workspace_size(int64_t n_keys_a, int64_t n_keys_b, int64_t k, size_t* bytes)
{
    g_last_error[0] = 0;
    if (!bytes) return fail(MAG_E_NULL, "bytes is NULL");
    if (n_keys_a < 0 || n_keys_b < 0 || k < 0) return fail(MAG_E_SIZE, "negative size");
    Carver c;
    c.take<mag::Status>(1);
    carve_candidates(c, n_keys_a, k, nullptr);
    *bytes = c.off;
    return MAG_OK;
}

}  // extern "C"

namespace {

// the checks of one comparison and the parameters that do not depend on the
// workspace; *na / *nb are the table sizes (upper bounds for device counts)
int diff_params(const uint64_t* keysA, const mag_key_stats* statsA, const uint64_t* keysB,
                const mag_key_stats* statsB, int64_t k, mag_rank_out* out, mag::DiffParams& p)
{
    if (!statsA || !statsB || !out) return fail(MAG_E_NULL, "statsA/statsB/out is NULL");
    // a negative n_keys: the count is read on the device, bounded by the capacity
    const bool devA = statsA->n_keys < 0, devB = statsB->n_keys < 0;
    if (k < 0 || (devA && (!statsA->n_keys_device || statsA->capacity < 0)) ||
        (devB && (!statsB->n_keys_device || statsB->capacity < 0)))
        return fail(MAG_E_SIZE, "negative size (or n_keys < 0 without n_keys_device)");
    const int64_t na = devA ? statsA->capacity : statsA->n_keys;
    const int64_t nb = devB ? statsB->capacity : statsB->n_keys;
    if ((na > 0 && (!keysA || !statsA->sum || !statsA->count)) ||
        (nb > 0 && (!keysB || !statsB->sum || !statsB->count)))
        return fail(MAG_E_NULL, "key table array is NULL");
    if (p.detect && ((na > 0 && !statsA->duration) || (nb > 0 && !statsB->duration)))
        return fail(MAG_E_NULL, "per-key duration array is NULL");
    if (na > INT32_MAX || nb > INT32_MAX) return fail(MAG_E_SIZE, "key table too large");
    const int64_t need_rows = std::min(k, na);
    if (out->capacity < need_rows) return fail(MAG_E_CAPACITY, "out->capacity < min(k, n_keys_a)");
    if (need_rows > 0 && (!out->key || !out->ratio || !out->energy_a || !out->energy_b ||
                          !out->count_a || !out->count_b ||
                          (p.detect && (!p.out_la || !p.out_lb || !p.out_verdict))))
        return fail(MAG_E_NULL, "output array is NULL");
    p.ka = keysA;
    p.sa = statsA->sum;
    p.ca = statsA->count;
    p.na = na;
    p.kb = keysB;
    p.sb = statsB->sum;
    p.cb = statsB->count;
    p.nb = nb;
    p.na_dev = devA ? statsA->n_keys_device : nullptr;
    p.nb_dev = devB ? statsB->n_keys_device : nullptr;
    p.k = k;
    p.out_key = out->key;
    p.out_ratio = out->ratio;
    p.out_ea = out->energy_a;
    p.out_eb = out->energy_b;
    p.out_ca = out->count_a;
    p.out_cb = out->count_b;
    if (p.detect) {
        p.la = statsA->duration;
        p.lb = statsB->duration;
    }
    return MAG_OK;
}


// a comparison's result from its status block: na, nb the table sizes (or
// their bounds when dev: sizes read on the device), k the rows asked for
int conclude_diff(int64_t na, int64_t nb, int64_t k, bool dev, const mag::Status& st,
                  mag_rank_out* out)
{
    if (st.err & mag::ERR_KEYS) return fail(MAG_E_KEYS, "key table not strictly ascending");
    const int64_t ra = dev ? (int64_t)st.diff_na : na;
    const int64_t rb = dev ? (int64_t)st.diff_nb : nb;
    out->n_join = st.n_join;
    out->n_out = std::min<int64_t>(k, st.n_join);
    out->n_only_a = ra - st.n_join;
    out->n_only_b = rb - st.n_join;
    return MAG_OK;
}
int conclude_diff(const mag::DiffParams& p, const mag::Status& st, mag_rank_out* out)
{
    return conclude_diff(p.na, p.nb, p.k, p.na_dev || p.nb_dev, st, out);
}

// the checks and kernels of one comparison (mag_diff, mag_diff_async,
// mag_detect; p's detection fields are set by the caller)
int enqueue_diff(const uint64_t* keysA, const mag_key_stats* statsA, const uint64_t* keysB,
                 const mag_key_stats* statsB, int64_t k, mag_rank_out* out, mag::DiffParams& p,
                 void* workspace, size_t workspace_bytes, hipStream_t stream)
{
    int rc = diff_params(keysA, statsA, keysB, statsB, k, out, p);
    if (rc != MAG_OK) return rc;
    if (!workspace) return fail(MAG_E_NULL, "workspace is NULL");
    if (!aligned(workspace, 256)) return fail(MAG_E_WORKSPACE, "workspace must be 256-byte aligned");
    if (unfinished(workspace))
        return fail(MAG_E_STATE, "an asynchronous call on this workspace is not finished");
    size_t need = 0;
    mag_diff_workspace_size(p.na, p.nb, k, &need);
    if (workspace_bytes < need) return fail(MAG_E_WORKSPACE, "workspace too small");
    Carver c;
    c.base = static_cast<char*>(workspace);
    p.status = c.take<mag::Status>(1);
    carve_candidates(c, p.na, k, &p);
    hipError_t e;
    // every field of the status block the call reads is written by its kernels
    if ((e = mag::launch_diff(p, stream)) != hipSuccess) return hip_fail(e, "diff kernels");
    return MAG_OK;
}

// the join and ranking, waited for; the status block is returned in *st
int run_diff(const uint64_t* keysA, const mag_key_stats* statsA, const uint64_t* keysB,
             const mag_key_stats* statsB, int64_t k, mag_rank_out* out, mag::DiffParams& p,
             void* workspace, size_t workspace_bytes, hipStream_t stream, mag::Status* st)
{
    int rc = enqueue_diff(keysA, statsA, keysB, statsB, k, out, p, workspace, workspace_bytes,
                          stream);
    if (rc != MAG_OK) return rc;
    rc = read_status(p.status, stream, st);
    if (rc != MAG_OK) return rc;
    return conclude_diff(p, *st, out);
}

size_t diff_batch_bytes(int64_t na, int32_t n, int64_t k)
{
    Carver c;
    c.take<mag::Status>((size_t)std::max(n, 1));
    for (int32_t i = 0; i < n; ++i) carve_candidates(c, na, k, nullptr);
    return c.off;
}

}  // namespace

extern "C" {

int mag_diff(const uint64_t* keysA, const mag_key_stats* statsA, const uint64_t* keysB,
             const mag_key_stats* statsB, int64_t k, mag_rank_out* out, void* workspace,
             size_t workspace_bytes, hipStream_t stream)
{
    g_last_error[0] = 0;
    mag::DiffParams p{};
    mag::Status st;
    return run_diff(keysA, statsA, keysB, statsB, k, out, p, workspace, workspace_bytes, stream,
                    &st);
}

int mag_diff_async(const uint64_t* keysA, const mag_key_stats* statsA, const uint64_t* keysB,
                   const mag_key_stats* statsB, int64_t k, mag_rank_out* out, void* workspace,
                   size_t workspace_bytes, hipStream_t stream)
{
    g_last_error[0] = 0;
    mag::DiffParams p{};
    int rc = enqueue_diff(keysA, statsA, keysB, statsB, k, out, p, workspace, workspace_bytes,
                          stream);
    if (rc != MAG_OK) return rc;
    // the status block (first in the workspace) goes to the pinned buffer of
    // the workspace's record, in stream order
    TimerSlot* t = timer_slot(workspace, true);
    if (!t || !t->host_status)
        return fail(MAG_E_HIP, "no host buffer for the status of an asynchronous call");
    hipError_t e =
        hipMemcpyAsync(t->host_status, p.status, sizeof(mag::Status), hipMemcpyDeviceToHost, stream);
    if (e != hipSuccess) return hip_fail(e, "status copy");
    if ((e = hipEventRecord(t->done, stream)) != hipSuccess) return hip_fail(e, "event record");
    t->status_pending = true;
    t->stream = stream;
    t->diff = true;
    t->diff_dev = p.na_dev || p.nb_dev;
    t->diff_na = p.na;
    t->diff_nb = p.nb;
    t->diff_k = k;
    return MAG_OK;
}

int mag_diff_finish(const void* workspace, mag_rank_out* out)
{
    g_last_error[0] = 0;
    if (!workspace || !out) return fail(MAG_E_NULL, "workspace/out is NULL");
    TimerSlot* t = timer_slot(workspace, false);
    if (!t || !t->status_pending || !t->diff || !t->host_status)
        return fail(MAG_E_STATE, "no unfinished mag_diff_async call on this workspace");
    t->status_pending = false;
    t->diff = false;
    hipError_t e;
    if ((e = hipEventSynchronize(t->done)) != hipSuccess) return hip_fail(e, "synchronize");
    return conclude_diff(t->diff_na, t->diff_nb, t->diff_k, t->diff_dev, *t->host_status, out);
}

int mag_diff_batch_workspace_size(int64_t n_keys_a, int32_t n_candidates, int64_t k,
                                  size_t* bytes)
{
    g_last_error[0] = 0;
    if (!bytes) return fail(MAG_E_NULL, "bytes is NULL");
    if (n_keys_a < 0 || k < 0 || n_candidates < 0 || n_candidates > MAG_DIFF_BATCH_MAX)
        return fail(MAG_E_SIZE, "negative size or too many candidates");
    *bytes = diff_batch_bytes(n_keys_a, n_candidates, k);
    return MAG_OK;
}

int mag_diff_batch(const uint64_t* keysA, const mag_key_stats* statsA, int32_t n_candidates,
                   const uint64_t* const* keysB, const mag_key_stats* statsB, int64_t k,
                   mag_rank_out* out, void* workspace, size_t workspace_bytes, hipStream_t stream)
{
    g_last_error[0] = 0;
    if (n_candidates < 0 || n_candidates > MAG_DIFF_BATCH_MAX)
        return fail(MAG_E_SIZE, "n_candidates must be in [0, MAG_DIFF_BATCH_MAX]");
    if (n_candidates == 0) return MAG_OK;
    if (!keysB || !statsB || !out) return fail(MAG_E_NULL, "keysB/statsB/out is NULL");
    std::vector<mag::DiffParams> ps((size_t)n_candidates);
    for (int32_t c = 0; c < n_candidates; ++c) {
        ps[c] = mag::DiffParams{};
        const int rc = diff_params(keysA, statsA, keysB[c], &statsB[c], k, &out[c], ps[c]);
        if (rc != MAG_OK) return rc;
    }
    if (!workspace) return fail(MAG_E_NULL, "workspace is NULL");
    if (!aligned(workspace, 256)) return fail(MAG_E_WORKSPACE, "workspace must be 256-byte aligned");
    const int64_t na = ps[0].na;
    if (workspace_bytes < diff_batch_bytes(na, n_candidates, k))
        return fail(MAG_E_WORKSPACE, "workspace too small");
    Carver c;
    c.base = static_cast<char*>(workspace);
    mag::Status* status = c.take<mag::Status>((size_t)n_candidates);
    for (int32_t i = 0; i < n_candidates; ++i) {
        ps[i].status = status + i;
        carve_candidates(c, na, k, &ps[i]);
    }
    hipError_t e;
    if ((e = mag::launch_diff_batch(ps.data(), n_candidates, stream)) != hipSuccess)
        return hip_fail(e, "diff kernels");
    std::vector<mag::Status> st((size_t)n_candidates);
    if ((e = hipMemcpyAsync(st.data(), status, sizeof(mag::Status) * (size_t)n_candidates,
                            hipMemcpyDeviceToHost, stream)) != hipSuccess)
        return hip_fail(e, "status copy");
    if ((e = hipStreamSynchronize(stream)) != hipSuccess) return hip_fail(e, "synchronize");
    for (int32_t i = 0; i < n_candidates; ++i) {
        const int rc = conclude_diff(ps[i], st[i], &out[i]);
        if (rc != MAG_OK) return rc;
    }
    return MAG_OK;
}

int mag_detect_workspace_size(int64_t n_keys_a, int64_t n_keys_b, int64_t rows, size_t* bytes)
{
    return mag_diff_workspace_size(n_keys_a, n_keys_b, rows, bytes);
}

int mag_detect(const uint64_t* keysA, const mag_key_stats* statsA, const uint64_t* keysB,
               const mag_key_stats* statsB, const mag_detect_opts* opts, mag_detect_out* out,
               void* workspace, size_t workspace_bytes, hipStream_t stream)
{
    g_last_error[0] = 0;
    if (!out) return fail(MAG_E_NULL, "out is NULL");
    mag::DiffParams p{};
    p.detect = 1;
    p.threshold = opts ? opts->threshold : 0.10;
    p.tolerance = opts ? opts->tolerance : 0.01;
    if (p.threshold != p.threshold || p.tolerance != p.tolerance)
        return fail(MAG_E_SIZE, "threshold or tolerance is NaN");
    p.out_la = out->latency_a;
    p.out_lb = out->latency_b;
    p.out_verdict = out->verdict;
    mag::Status st;
    // the flagged keys are a prefix of the ranking: rank as many rows as fit
    const int rc = run_diff(keysA, statsA, keysB, statsB, out->rank.capacity, &out->rank, p,
                            workspace, workspace_bytes, stream, &st);
    if (rc != MAG_OK) return rc;
    out->n_flagged = st.n_flag;
    out->n_waste = st.n_waste;
    out->n_tradeoff = (int64_t)st.n_flag - (int64_t)st.n_waste;
    out->rank.n_out = std::min<int64_t>(out->rank.n_out, out->n_flagged);
    return MAG_OK;
}

}  // extern "C"

// ------------------------------------------------------ tensor matching (4.2)

namespace {

int check_tensor(const mag_tensor* t)
{
    if (!t) return fail(MAG_E_NULL, "tensor descriptor is NULL");
    if (t->rank < 1 || t->rank > MAG_SVD_MAX_RANK) return fail(MAG_E_SIZE, "tensor rank out of range");
    int64_t total = 1;
    for (int i = 0; i < t->rank; ++i) {
        if (t->dims[i] < 1) return fail(MAG_E_SIZE, "tensor dimension < 1");
        total *= t->dims[i];
        if (total >= ((int64_t)1 << 31)) return fail(MAG_E_SIZE, "tensor has 2^31 elements or more");
    }
    return MAG_OK;
}

// Gram sides whose product one workgroup makes whole
bool gram_whole(int64_t K) { return K > 64 && K <= mag::GRAM_WHOLE; }

// the unfolding of mask g as a Gram task (K side = the shorter side)
void unfolding_task(const mag_tensor* t, int g, mag::SvdTask& task)
{
    const int r = t->rank;
    int64_t str[MAG_SVD_MAX_RANK];
    str[r - 1] = 1;
    for (int i = r - 2; i >= 0; --i) str[i] = str[i + 1] * t->dims[i + 1];
    int64_t M = 1, N = 1;
    for (int i = 0; i < r; ++i) ((g >> i) & 1 ? M : N) *= t->dims[i];
    const bool rows_k = M <= N;
    task = mag::SvdTask{};
    task.data = t->data;
    task.K = rows_k ? M : N;
    task.L = rows_k ? N : M;
    for (int i = 0; i < r; ++i) {
        const bool in_g = (g >> i) & 1;
        if (in_g == rows_k) {
            task.kdim[task.nk] = t->dims[i];
            task.kstr[task.nk++] = str[i];
        } else {
            task.ldim[task.nl] = t->dims[i];
            task.lstr[task.nl++] = str[i];
        }
    }
    // work items of the Gram product: one 32-side block for a short side, the
    // whole triangle for a side in (64, GRAM_WHOLE], else pairs of 64-side blocks
    const int64_t gb = task.K <= mag::GRAM_NARROW ? 32 : 64;
    task.nt = gram_whole(task.K) ? 1 : (int32_t)((task.K + gb - 1) / gb);
    const int64_t ch = task.K <= mag::GRAM_NARROW ? mag::GRAM_CHUNK_NARROW
                     : gram_whole(task.K)         ? mag::GRAM_CHUNK_WHOLE
                                                  : mag::GRAM_CHUNK;
    task.nchunk = (int32_t)((task.L + ch - 1) / ch);
}

int count_invariants(const mag_tensor* t, int32_t* n_unf, int64_t* n_values)
{
    int rc = check_tensor(t);
    if (rc) return rc;
    int32_t u = 0;
    int64_t v = 0;
    for (int g = 1; g < (1 << t->rank) - 1; g += 2) {  // masks containing mode 0
        mag::SvdTask task;
        unfolding_task(t, g, task);
        if (task.K > MAG_SVD_MAX_K) {
            snprintf(g_last_error, sizeof(g_last_error),
                     "an unfolding has min(M, N) = %lld > %d", (long long)task.K, MAG_SVD_MAX_K);
            return MAG_E_SIZE;
        }
        ++u;
        v += task.K;
    }
    *n_unf = u;
    *n_values = v;
    return MAG_OK;
}

struct InvPlan {
    // tasks with K <= mag::GRAM_NARROW first (n_narrow of them, n_items_narrow
    // work items), then those made whole (n_whole, n_items_whole), then the
    // others (n_items work items); spec_off: each task's offset in the spectra
    // array (the tensors' and unfoldings' order)
    std::vector<mag::SvdTask> tasks;
    std::vector<int64_t> spec_off;
    int n_narrow = 0, n_whole = 0;
    int64_t gram_len = 0, n_items = 0, n_items_narrow = 0, n_items_whole = 0;
    // eigenvalue work items (tasks with K <= mag::SVD_SMALL_K, in task order)
    // and the doubles of their tridiagonal forms (2 K + 3 each)
    int64_t n_eig_items = 0, tri_len = 0;
    int large_k = 0;  // largest Gram side above mag::SVD_SMALL_K (0: none)
};

int plan_invariants(const mag_tensor* ts, int32_t n, InvPlan& pl)
{
    if (n < 0) return fail(MAG_E_SIZE, "n_tensors < 0");
    if (n > 0 && !ts) return fail(MAG_E_NULL, "tensors is NULL");
    pl = InvPlan{};
    std::vector<mag::SvdTask> whole, wide;
    std::vector<int64_t> whole_off, wide_off;
    int64_t so = 0;
    for (int32_t i = 0; i < n; ++i) {
        int32_t u;
        int64_t v;
        int rc = count_invariants(&ts[i], &u, &v);
        if (rc) return rc;
        for (int g = 1; g < (1 << ts[i].rank) - 1; g += 2) {
            mag::SvdTask task;
            unfolding_task(&ts[i], g, task);
            const int64_t items = (int64_t)task.nt * (task.nt + 1) / 2 * task.nchunk;
            pl.gram_len += task.K * task.K;
            if (task.K > mag::SVD_SMALL_K) pl.large_k = std::max(pl.large_k, (int)task.K);
            if (task.K <= mag::GRAM_NARROW) {
                task.item0 = pl.n_items_narrow;
                pl.n_items_narrow += items;
                pl.tasks.push_back(task);
                pl.spec_off.push_back(so);
            } else if (gram_whole(task.K)) {
                task.item0 = pl.n_items_whole;
                pl.n_items_whole += items;
                whole.push_back(task);
                whole_off.push_back(so);
            } else {
                task.item0 = pl.n_items;
                pl.n_items += items;
                wide.push_back(task);
                wide_off.push_back(so);
            }
            so += task.K;
        }
    }
    pl.n_narrow = (int)pl.tasks.size();
    pl.n_whole = (int)whole.size();
    pl.tasks.insert(pl.tasks.end(), whole.begin(), whole.end());
    pl.spec_off.insert(pl.spec_off.end(), whole_off.begin(), whole_off.end());
    pl.tasks.insert(pl.tasks.end(), wide.begin(), wide.end());
    pl.spec_off.insert(pl.spec_off.end(), wide_off.begin(), wide_off.end());
    for (auto& t : pl.tasks) {
        t.eig0 = pl.n_eig_items;
        if (t.K <= mag::SVD_SMALL_K) {
            pl.n_eig_items += (t.K + mag::EIG_PER_ITEM - 1) / mag::EIG_PER_ITEM;
            pl.tri_len += 2 * t.K + 3;
        }
    }
    return MAG_OK;
}

size_t carve_invariants(const InvPlan& pl, void* ws, mag::SvdTask** tasks, double** gram,
                        double** tri, double** large)
{
    Carver c;
    c.base = static_cast<char*>(ws);
    *tasks = c.take<mag::SvdTask>(std::max<size_t>(pl.tasks.size(), 1));
    *gram = c.take<double>((size_t)std::max<int64_t>(pl.gram_len, 1));
    *tri = c.take<double>((size_t)std::max<int64_t>(pl.tri_len, 1));
    // scratch of the many-workgroup reduction, shared by the large unfoldings
    // (they run one after another)
    *large = pl.large_k ? c.take<double>((size_t)mag::svd_large_scratch(pl.large_k)) : nullptr;
    return c.off;
}

// spectra descriptors of a tensor set: offsets in the order mag_invariants writes
int spec_descs(const mag_tensor* ts, int32_t n, std::vector<mag::SpecDesc>& out)
{
    out.assign((size_t)std::max(n, 0), mag::SpecDesc{});
    int64_t off = 0;
    for (int32_t i = 0; i < n; ++i) {
        int32_t u;
        int64_t v;
        int rc = count_invariants(&ts[i], &u, &v);
        if (rc) return rc;
        mag::SpecDesc& d = out[i];
        for (int g = 1; g < (1 << ts[i].rank) - 1; g += 2) {
            mag::SvdTask task;
            unfolding_task(&ts[i], g, task);
            d.off[d.n] = off;
            d.len[d.n++] = task.K;
            off += task.K;
        }
    }
    return MAG_OK;
}

}  // namespace

extern "C" {

int mag_invariant_count(const mag_tensor* tensor, int32_t* n_unfoldings, int64_t* n_values)
{
    g_last_error[0] = 0;
    if (!n_unfoldings || !n_values) return fail(MAG_E_NULL, "output pointer is NULL");
    return count_invariants(tensor, n_unfoldings, n_values);
}

int mag_invariants_workspace_size(const mag_tensor* tensors, int32_t n_tensors, size_t* bytes)
{
    g_last_error[0] = 0;
    if (!bytes) return fail(MAG_E_NULL, "bytes is NULL");
    InvPlan pl;
    int rc = plan_invariants(tensors, n_tensors, pl);
    if (rc) return rc;
    mag::SvdTask* t;
    double *g, *tr, *lg;
    *bytes = carve_invariants(pl, nullptr, &t, &g, &tr, &lg);
    return MAG_OK;
}

int mag_invariants(const mag_tensor* tensors, int32_t n_tensors, double* spectra, void* workspace,
                   size_t workspace_bytes, hipStream_t stream)
{
    g_last_error[0] = 0;
    InvPlan pl;
    int rc = plan_invariants(tensors, n_tensors, pl);
    if (rc) return rc;
    if (pl.tasks.empty()) return MAG_OK;
    for (int32_t i = 0; i < n_tensors; ++i) {
        if (!tensors[i].data) return fail(MAG_E_NULL, "tensor data is NULL");
        if (!aligned(tensors[i].data, 4)) return fail(MAG_E_ALIGN, "tensor data not 4-byte aligned");
    }
    if (!spectra) return fail(MAG_E_NULL, "spectra is NULL");
    if (!aligned(spectra, 8)) return fail(MAG_E_ALIGN, "spectra not 8-byte aligned");
    if (!workspace) return fail(MAG_E_NULL, "workspace is NULL");
    if (!aligned(workspace, 256)) return fail(MAG_E_WORKSPACE, "workspace must be 256-byte aligned");
    mag::SvdTask* dtasks;
    double *gram, *tri, *large;
    const size_t need = carve_invariants(pl, nullptr, &dtasks, &gram, &tri, &large);
    if (workspace_bytes < need) return fail(MAG_E_WORKSPACE, "workspace too small");
    carve_invariants(pl, workspace, &dtasks, &gram, &tri, &large);
    int64_t go = 0, to = 0;
    for (size_t i = 0; i < pl.tasks.size(); ++i) {
        mag::SvdTask& t = pl.tasks[i];
        t.gram = gram + go;
        t.out = spectra + pl.spec_off[i];
        go += t.K * t.K;
        t.tri = nullptr;
        if (t.K <= mag::SVD_SMALL_K) {
            t.tri = tri + to;
            to += 2 * t.K + 3;
        }
    }
    hipError_t e;
    if ((e = hipMemcpyAsync(dtasks, pl.tasks.data(), sizeof(mag::SvdTask) * pl.tasks.size(),
                            hipMemcpyHostToDevice, stream)) != hipSuccess)
        return hip_fail(e, "task copy");
    if ((e = mag::launch_svd(dtasks, (int)pl.tasks.size(), pl.n_narrow, pl.n_items_narrow,
                             pl.n_whole, pl.n_items_whole, pl.n_items, pl.n_eig_items, gram,
                             pl.gram_len, stream)) != hipSuccess)
        return hip_fail(e, "invariant kernels");
    for (const auto& t : pl.tasks)
        if (t.K > mag::SVD_SMALL_K &&
            (e = mag::launch_svd_large(t.gram, (int)t.K, large, t.out, stream)) != hipSuccess)
            return hip_fail(e, "large unfolding kernels");
    // (the task table on the host stays alive until the copy is done)
    if ((e = hipStreamSynchronize(stream)) != hipSuccess) return hip_fail(e, "synchronize");
    return MAG_OK;
}

int mag_match_workspace_size(int32_t na, int32_t nb, size_t* bytes)
{
    g_last_error[0] = 0;
    if (!bytes) return fail(MAG_E_NULL, "bytes is NULL");
    if (na < 0 || nb < 0) return fail(MAG_E_SIZE, "negative count");
    Carver c;
    c.take<mag::SpecDesc>((size_t)std::max(na + nb, 1));
    *bytes = c.off;
    return MAG_OK;
}

int mag_match(const mag_tensor* ta, int32_t na, const double* spectra_a, const mag_tensor* tb,
              int32_t nb, const double* spectra_b, double eps, uint8_t* match, void* workspace,
              size_t workspace_bytes, hipStream_t stream)
{
    g_last_error[0] = 0;
    if (na < 0 || nb < 0) return fail(MAG_E_SIZE, "negative count");
    if (!(eps >= 0.0)) return fail(MAG_E_SIZE, "eps must be >= 0");
    if ((int64_t)na * nb == 0) return MAG_OK;
    if (!ta || !tb || !spectra_a || !spectra_b || !match || !workspace)
        return fail(MAG_E_NULL, "NULL argument");
    if (!aligned(workspace, 256)) return fail(MAG_E_WORKSPACE, "workspace must be 256-byte aligned");
    if ((int64_t)na * nb > 0x7fffffffLL) return fail(MAG_E_SIZE, "too many pairs");
    std::vector<mag::SpecDesc> da, db;
    int rc = spec_descs(ta, na, da);
    if (rc == MAG_OK) rc = spec_descs(tb, nb, db);
    if (rc) return rc;
    size_t need = 0;
    mag_match_workspace_size(na, nb, &need);
    if (workspace_bytes < need) return fail(MAG_E_WORKSPACE, "workspace too small");
    auto* dd = static_cast<mag::SpecDesc*>(workspace);
    da.insert(da.end(), db.begin(), db.end());
    hipError_t e;
    if ((e = hipMemcpyAsync(dd, da.data(), sizeof(mag::SpecDesc) * da.size(), hipMemcpyHostToDevice,
                            stream)) != hipSuccess)
        return hip_fail(e, "descriptor copy");
    if ((e = mag::launch_svd_match(dd, na, spectra_a, dd + na, nb, spectra_b, eps, match,
                                   stream)) != hipSuccess)
        return hip_fail(e, "match kernel");
    if ((e = hipStreamSynchronize(stream)) != hipSuccess) return hip_fail(e, "synchronize");
    return MAG_OK;
}

}  // extern "C"

// ------------------------------------------------------ subgraph matching

namespace {

int check_graph(const mag_graph* g)
{
    if (!g) return fail(MAG_E_NULL, "graph is NULL");
    if (g->n_nodes < 2) return fail(MAG_E_SIZE, "a graph needs at least 2 nodes");
    if (g->n_edges < 0) return fail(MAG_E_SIZE, "n_edges < 0");
    if (g->n_edges > 0 && (!g->src || !g->dst)) return fail(MAG_E_NULL, "edge arrays are NULL");
    for (int32_t e = 0; e < g->n_edges; ++e)
        if (g->src[e] < 0 || g->src[e] >= g->n_nodes || g->dst[e] < 0 || g->dst[e] >= g->n_nodes)
            return fail(MAG_E_SIZE, "edge endpoint out of range");
    return MAG_OK;
}

}  // namespace

extern "C" int mag_match_subgraphs(const mag_graph* g1, const mag_graph* g2, const int32_t* eq,
                                   int32_t n_eq, int32_t* out, int32_t capacity, int32_t* n_out)
{
    g_last_error[0] = 0;
    int rc;
    if ((rc = check_graph(g1)) != MAG_OK || (rc = check_graph(g2)) != MAG_OK) return rc;
    if (!n_out) return fail(MAG_E_NULL, "n_out is NULL");
    if (n_eq < 0 || capacity < 0) return fail(MAG_E_SIZE, "negative count");
    if (n_eq > 0 && !eq) return fail(MAG_E_NULL, "eq is NULL");
    for (int32_t p = 0; p < n_eq; ++p)
        if (eq[2 * p] < 0 || eq[2 * p] >= g1->n_nodes || eq[2 * p + 1] < 0 ||
            eq[2 * p + 1] >= g2->n_nodes)
            return fail(MAG_E_SIZE, "eq node out of range");
    std::vector<int32_t> pairs;
    try {
        rc = mag::match_subgraphs(*g1, *g2, eq, n_eq, pairs);
    } catch (const std::bad_alloc&) {
        return fail(MAG_E_SIZE, "out of host memory");
    }
    if (rc == MAG_E_GRAPH)
        return fail(MAG_E_GRAPH, "a graph has a cycle or a node off every input-to-output path");
    const int32_t np = (int32_t)(pairs.size() / 4);
    *n_out = np;
    if (np > capacity) return fail(MAG_E_CAPACITY, "more matched pairs than capacity");
    if (np > 0 && !out) return fail(MAG_E_NULL, "out is NULL");
    std::copy(pairs.begin(), pairs.end(), out);
    return MAG_OK;
}
