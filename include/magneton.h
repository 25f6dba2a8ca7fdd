/*
 * magneton.h -- C ABI of the MI355X operator energy attribution library.
 *
 * The library implements the data-parallel core of differential energy
 * debugging (Magneton, arXiv 2512.08365): a sampled power trace is integrated
 * over operator/kernel execution intervals (Section 5.2, which asks for energy
 * attributed to individual kernels lasting tens to hundreds of microseconds),
 * the interval energies are aggregated per operator key (Section 4.1 makes
 * the operator the unit of comparison; Section 2.1 ranks operators by energy),
 * and the per-key energies of two systems running the same workload are
 * joined and ranked by their relative difference (Section 6.1 flags operators
 * whose energy differs by more than a threshold; Table "tab:energy-profiling"
 * fixes the sign convention (value - reference) / reference).
 *
 * Conventions for every entry point:
 *   - All array arguments are DEVICE pointers to caller-owned memory (for
 *     example torch tensors on the current HIP device), unless documented as
 *     host.  The library never allocates device memory and keeps no pointer
 *     after a call returns.  Scratch memory is the caller's `workspace`.
 *   - Work is enqueued on `stream`.  Entry points that return data-dependent
 *     sizes or device-detected errors synchronize `stream` before returning.
 *   - Return value: MAG_OK (0) or a negative MAG_E_* code.  No exception
 *     crosses the ABI.  On error, device outputs are unspecified;
 *     mag_last_error() gives a human-readable detail (thread-local).
 *   - Energies are joules (fp64) when timestamps are seconds and power watts.
 */
#ifndef MAGNETON_H
#define MAGNETON_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---------------------------------------------------------------- status */
#define MAG_OK 0
#define MAG_E_NULL (-1)       /* a required pointer is NULL                          */
#define MAG_E_SIZE (-2)       /* n_samples < 2 or > MAG_MAX_SAMPLES, a negative count, */
                              /* a key capacity above MAG_MAX_KEYS                     */
#define MAG_E_CAPACITY (-3)   /* more distinct keys than the key table capacity       */
#define MAG_E_WORKSPACE (-4)  /* workspace too small (or misaligned: 256 B required)  */
#define MAG_E_TIMESTAMPS (-5) /* timestamps not finite or not strictly increasing     */
#define MAG_E_POWER (-6)      /* a power sample is NaN, infinite or negative          */
#define MAG_E_INTERVAL (-7)   /* start > end, non-finite bound, or a stream whose     */
                              /* intervals are unsorted or overlap                    */
#define MAG_E_STREAMS (-8)    /* bad n_streams or stream_offsets                      */
#define MAG_E_STATE (-9)      /* streaming handle used out of order                   */
#define MAG_E_HIP (-10)       /* a HIP runtime call failed                            */
#define MAG_E_ALIGN (-11)     /* a device array is not aligned to its element size    */
#define MAG_E_KEYS (-12)      /* a key table passed to mag_diff is not strictly       */
                              /* ascending                                            */
#define MAG_E_COUNTER (-13)   /* an energy-counter reading is not finite or decreases */
#define MAG_E_GRAPH (-14)     /* a graph is not a DAG from node 0 to node n-1 through  */
                              /* every node                                           */

/* ----------------------------------------------------------------- flags */
/* Split the power at each instant equally among the intervals active at that
   instant (several concurrent streams).  Without it every interval receives
   the full power over its span. */
#define MAG_EQUAL_SPLIT 0x1u
/* Skip the device-side input checks (sortedness, finiteness, signs). */
#define MAG_SKIP_VALIDATE 0x2u
/* Time the call on `stream` with HIP events and report it in mag_summary. */
#define MAG_TIME_KERNELS 0x4u
/* mag_attribute returns once its work is enqueued; mag_attribute_finish
   delivers n_keys, the summary and device-detected errors.  A workspace holds
   at most one unfinished asynchronous call: any attribution on it before
   mag_attribute_finish returns MAG_E_STATE.  One thread may have up to 4096
   unfinished asynchronous calls (on as many workspaces); beyond that the
   status is read back by mag_attribute_finish from the device instead. */
#define MAG_ASYNC 0x8u
/* Also sum each key's interval durations (end - start; per replay run in the
   counter mode) into per_key->duration, which must then be non-NULL: the
   latency side of Section 6.1's comparison. */
#define MAG_KEY_LATENCY 0x10u

/* Verdicts of mag_detect (Section 6.1). */
#define MAG_WASTE 1    /* the efficient side is at most `tolerance` slower     */
#define MAG_TRADEOFF 2 /* the extra energy buys more speed than that           */

/* Most concurrent streams one call accepts. */
#define MAG_MAX_STREAMS 32
/* Longest trace one call (or one stream) accepts, in samples. */
#define MAG_MAX_SAMPLES (1LL << 40)
/* Largest key-table capacity (rows of per-key statistics) one call accepts. */
#define MAG_MAX_KEYS (1LL << 28)

typedef struct mag_attr_opts {
    int32_t n_streams;              /* >= 1; intervals are concatenated by stream   */
    uint32_t flags;                 /* MAG_EQUAL_SPLIT | MAG_SKIP_VALIDATE |          */
                                    /* MAG_TIME_KERNELS | MAG_ASYNC | MAG_KEY_LATENCY */
    const int64_t* stream_offsets;  /* HOST int64[n_streams + 1]: stream a owns       */
                                    /* intervals [offs[a], offs[a+1]); offs[0] = 0,   */
                                    /* offs[n_streams] = n_intervals; NULL allowed    */
                                    /* only when n_streams == 1                       */
    hipEvent_t intervals_ready;     /* mag_attribute only, may be NULL: recorded on   */
                                    /* `stream` once the per-interval outputs are     */
                                    /* complete, before the per-key grouping, so that */
                                    /* work on another stream (the other system's     */
                                    /* attribution, Section 3.2) can start while the  */
                                    /* grouping runs; the caller owns the event       */
    const struct mag_key_plan* key_plan; /* mag_attribute only, may be NULL: host     */
                                    /* struct of a key plan built by                  */
                                    /* mag_key_plan_build for these op_keys (same     */
                                    /* n_intervals and key capacity); the call then   */
                                    /* groups with its key map instead of building    */
                                    /* one, after waiting for key_plan->ready         */
    hipEvent_t tiles_wait;          /* mag_attribute only, may be NULL: waited for on */
                                    /* `stream` right before the power trace is       */
                                    /* integrated (after the call's own set-up)       */
    hipEvent_t tiles_done;          /* mag_attribute only, may be NULL: recorded on   */
                                    /* `stream` right after the trace integration,    */
                                    /* before the fix-ups and the grouping; with      */
                                    /* tiles_wait it lets the bandwidth-bound passes  */
                                    /* of two attributions run back to back while     */
                                    /* the rest of each overlaps the other            */
    hipStream_t group_stream;       /* mag_attribute only, may be NULL: the fix-ups,  */
                                    /* grouping and status copy run on this stream,   */
                                    /* which first waits for the trace integration    */
                                    /* on `stream`; `stream` is then free for the next */
                                    /* call's integration (a synchronous call waits   */
                                    /* for group_stream; MAG_ASYNC finishes as usual) */
} mag_attr_opts;

/*
 * A key plan: the key map of a per-key grouping (the distinct operator keys,
 * a dense id per key, each key's rank in ascending order, and every
 * interval's id), which depends on the operator keys only, not on the power
 * trace.  Built on its own (mag_key_plan_build) it can be made on another
 * stream while the power trace is integrated, or once for several
 * attributions of the same operator trace (Section 3.2 compares systems that
 * run the same workload; Section 4.1 makes the operator the unit).
 *   buffer        device memory, >= mag_key_plan_size(...) bytes, 256-byte
 *                 aligned, caller-owned; holds the map until rebuilt
 *   bytes         size of buffer
 *   n_intervals, key_capacity   written by mag_key_plan_build; an attribution
 *                 using the plan must pass the same values (else MAG_E_STATE)
 *   ready         optional HIP event (caller-owned): recorded on the build's
 *                 stream once the map is complete; an attribution using the
 *                 plan waits for it on its own stream before grouping
 */
typedef struct mag_key_plan {
    void* buffer;
    size_t bytes;
    int64_t n_intervals;
    int64_t key_capacity;
    hipEvent_t ready;
} mag_key_plan;

/* Per-interval outputs (device arrays of n_intervals entries; any may be NULL). */
typedef struct mag_interval_out {
    double* energy;     /* E_i, J                                                  */
    int64_t* start_idx; /* lower_bound(timestamps, starts[i]) in [0, n_samples]     */
    int64_t* end_idx;   /* lower_bound(timestamps, ends[i])   in [0, n_samples]     */
} mag_interval_out;

/* Per-key statistics (device arrays of `capacity` rows, ascending key order). */
typedef struct mag_key_stats {
    double* sum;      /* sum of E_i over the key's intervals                      */
    double* m2;       /* sum of (E_i - mean)^2 over the key's intervals            */
    int64_t* count;   /* number of intervals carrying the key                      */
    int64_t capacity; /* rows available in each array (host value)                 */
    int64_t n_keys;   /* rows filled (host value): output of mag_attribute, input  */
                      /* of mag_diff                                               */
    double* duration; /* with MAG_KEY_LATENCY: sum of the key's interval durations */
                      /* (s); read by mag_detect; may be NULL otherwise           */
    int64_t* n_keys_device; /* device int64, may be NULL: the attribution writes   */
                      /* the number of rows filled there, in stream order; mag_diff */
                      /* and mag_detect read the count there when n_keys < 0, so  */
                      /* that the comparison can be enqueued before the           */
                      /* attributions have finished (capacity then bounds it)     */
} mag_key_stats;

/* Whole-trace figures (host struct). */
typedef struct mag_summary {
    double trace_energy;      /* integral of the power over [t_0, t_{n-1}]          */
    double idle_energy;       /* energy at instants where no interval is active     */
    double attributed_energy; /* sum of all E_i                                     */
    int64_t n_clipped;        /* intervals with start < t_0 or end > t_{n-1}        */
    int64_t n_keys;           /* distinct keys (also when over capacity)            */
    double tile_kernel_ms;    /* MAG_TIME_KERNELS: duration of the interval-energy  */
                              /* kernel (HIP events on `stream`), else 0            */
    double device_ms;         /* MAG_TIME_KERNELS: device time from the start of    */
                              /* that kernel to the end of the call's work          */
} mag_summary;

/* Ranked join of two key tables (device arrays of `capacity` rows). */
typedef struct mag_rank_out {
    uint64_t* key;
    double* ratio;    /* (E_B - E_A) / E_A; +inf when E_A = 0 < E_B; 0 when both 0  */
    double* energy_a;
    double* energy_b;
    int64_t* count_a;
    int64_t* count_b;
    int64_t capacity; /* rows available (host), must be >= min(k, keys joined)      */
    int64_t n_out;    /* rows written (host output)                                  */
    int64_t n_only_a; /* keys present only in A (host output)                        */
    int64_t n_only_b; /* keys present only in B (host output)                        */
    int64_t n_join;   /* keys present in both (host output)                          */
} mag_rank_out;

/* Options of mag_detect (Section 6.1's values: 0.10, or 0.05; and 0.01). */
typedef struct mag_detect_opts {
    double threshold; /* flag a joined key when (E_B - E_A) / E_A >= threshold    */
    double tolerance; /* waste when (L_A - L_B) <= tolerance * L_B, else trade-off */
} mag_detect_opts;

/* Flagged keys of mag_detect (device arrays of `rank.capacity` rows). */
typedef struct mag_detect_out {
    mag_rank_out rank;  /* the flagged keys in ranking order (rank.n_out rows)   */
    double* latency_a;  /* L_A: statsA->duration of the row's key                */
    double* latency_b;  /* L_B                                                   */
    int32_t* verdict;   /* MAG_WASTE or MAG_TRADEOFF                             */
    int64_t n_flagged;  /* host output: joined keys with r >= threshold (all of  */
                        /* them, also beyond the rows written)                   */
    int64_t n_waste;    /* host output: flagged keys judged waste                */
    int64_t n_tradeoff; /* host output: flagged keys judged a trade-off          */
} mag_detect_out;

/*
 * mag_attribute_workspace_size -- bytes of device workspace mag_attribute needs
 * for the given sizes, key-table capacity (0 when no per-key output is asked
 * for) and options.  Host only; no device work.  Returns MAG_OK or
 * MAG_E_SIZE / MAG_E_STREAMS / MAG_E_NULL.
 */
int mag_attribute_workspace_size(int64_t n_samples, int64_t n_intervals, int64_t key_capacity,
                                 const mag_attr_opts* opts, size_t* bytes);

/*
 * mag_attribute -- attribute the energy of a sampled power trace to operator
 * intervals, and aggregate it per operator key.
 *
 * The paper asks for per-kernel energy from a microsecond-resolution power
 * source (Section 5.2) and compares operators (Section 4.1); it does not give
 * the integration rule.  This library's definition:
 *   P^(x)  = piecewise-linear interpolant of (timestamps[j], power[j]) on
 *            [t_0, t_{n-1}], zero outside;
 *   m(x)   = number of intervals i with starts[i] <= x < ends[i];
 *   E_i    = integral over [starts[i], ends[i]] of P^(x) / m(x)  (MAG_EQUAL_SPLIT)
 *          = integral over [starts[i], ends[i]] of P^(x)          (otherwise).
 * Per key: count, sum of E_i and M2 = sum of (E_i - mean)^2; rows ascending by
 * unsigned key; with MAG_KEY_LATENCY also the sum of (ends[i] - starts[i]),
 * the operator's latency (Section 6.1).  Every energy is computed in fp64 as a sum of non-negative
 * pieces; no energy is a difference of whole-trace running totals (the whole
 * sample segments between two endpoints are a difference of two prefixes
 * local to a 512-segment tile only where that difference keeps 6e-11
 * relative accuracy, and a direct sum otherwise).
 *
 * Arguments (device arrays unless noted):
 *   timestamps[n_samples] fp64, strictly increasing, finite (seconds)
 *   power[n_samples]      fp32, finite, >= 0 (watts)
 *   starts/ends[n_intervals] fp64, starts <= ends; within each stream sorted
 *                          and non-overlapping (ends[i] <= starts[i+1])
 *   op_keys[n_intervals]  uint64 operator key (any value); may be NULL when
 *                          per_key is NULL
 *   opts                  host; NULL means one stream with MAG_EQUAL_SPLIT
 *   per_interval          host struct of device pointers; may be NULL
 *   keys_out[capacity]    device uint64, ascending distinct keys; NULL iff
 *                          per_key is NULL
 *   per_key               host struct of device arrays; may be NULL to skip
 *                          the grouping; n_keys is written back
 *   summary               host struct; may be NULL
 *   workspace             device, >= mag_attribute_workspace_size(...,
 *                          per_key ? per_key->capacity : 0, opts) bytes,
 *                          256-byte aligned; its contents are scratch
 * Synchronizes `stream` (with MAG_ASYNC: returns once the work is enqueued,
 * see mag_attribute_finish).  Errors: MAG_E_NULL, MAG_E_SIZE, MAG_E_STREAMS,
 * MAG_E_WORKSPACE, MAG_E_ALIGN (host-detected, before any device work);
 * MAG_E_TIMESTAMPS, MAG_E_POWER, MAG_E_INTERVAL (device-detected, unless
 * MAG_SKIP_VALIDATE); MAG_E_CAPACITY (n_keys and summary->n_keys still report
 * the number of distinct keys; the key rows are unspecified); MAG_E_HIP.
 */
int mag_attribute(const double* timestamps, const float* power, int64_t n_samples,
                  const double* starts, const double* ends, const uint64_t* op_keys,
                  int64_t n_intervals, const mag_attr_opts* opts, mag_interval_out* per_interval,
                  uint64_t* keys_out, mag_key_stats* per_key, mag_summary* summary, void* workspace,
                  size_t workspace_bytes, hipStream_t stream);

/*
 * mag_attribute_static -- mag_attribute for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation): the same computation and results, with the
 * workspace replaced by a scratch array that the library holds in device
 * memory, MAG_STATIC_SCRATCH_BYTES (64 MiB) per GPU, for the life of the
 * process.  The call allocates nothing: no hipMalloc / hipFree, no pinned
 * host buffer, no events; the caller still provides every input and output.
 *   Sizes: those whose mag_attribute_workspace_size exceeds
 *   MAG_STATIC_SCRATCH_BYTES are rejected with MAG_E_WORKSPACE before any
 *   device work (for example 20,000,000 samples with 1,000,000 intervals and
 *   2,048 keys need 23 MiB and fit).
 *   opts->flags must not contain MAG_ASYNC or MAG_TIME_KERNELS, and
 *   opts->group_stream must be NULL (MAG_E_STATE).
 *   Every call on one GPU shares that GPU's scratch and leaves its contents
 *   behind (every call initializes what it reads): calls that overlap on one
 *   GPU (other host threads, or work still running on another stream) race
 *   and give unspecified results.
 * Synchronizes `stream`; returns what mag_attribute returns.
 */
#define MAG_STATIC_SCRATCH_BYTES (64LL << 20)
int mag_attribute_static(const double* timestamps, const float* power, int64_t n_samples,
                         const double* starts, const double* ends, const uint64_t* op_keys,
                         int64_t n_intervals, const mag_attr_opts* opts,
                         mag_interval_out* per_interval, uint64_t* keys_out,
                         mag_key_stats* per_key, mag_summary* summary, hipStream_t stream);

/*
 * mag_key_plan_size -- device bytes of a key plan for n_intervals keys and a
 * key capacity (>= 1).  Host only.  MAG_E_SIZE for a negative count or a
 * capacity out of [1, MAG_MAX_KEYS].
 * mag_key_plan_build -- build the key map of op_keys[n_intervals] (device,
 * any uint64) into plan->buffer on `stream` (asynchronous; records
 * plan->ready when given).  Distinct keys beyond the capacity are reported
 * by the attribution that uses the plan (MAG_E_CAPACITY).  Errors:
 * MAG_E_NULL, MAG_E_ALIGN, MAG_E_SIZE, MAG_E_WORKSPACE, MAG_E_HIP.
 */
int mag_key_plan_size(int64_t n_intervals, int64_t key_capacity, size_t* bytes);
int mag_key_plan_build(const uint64_t* op_keys, int64_t n_intervals, int64_t key_capacity,
                       mag_key_plan* plan, hipStream_t stream);

/*
 * mag_attribute_finish -- complete a mag_attribute (or mag_attribute_counter)
 * call made with MAG_ASYNC.
 * The paper's comparison is between two systems running the same workload
 * (Section 3.2); attributing both traces back to back, and waiting once, keeps
 * the device busy while the host enqueues the second.
 *   workspace  the call's workspace (its status block sits at its head); it
 *              must not be reused before this call
 *   per_key    host struct of the call (same capacity), or NULL if the call
 *              had none: n_keys is written
 *   summary    host struct, may be NULL: filled as by a synchronous call
 *              (tile_kernel_ms and device_ms when the call had MAG_TIME_KERNELS
 *              and is finished on the thread that made it)
 * Waits for the call itself when it was made on this thread (an event
 * recorded after its status copy: work enqueued on its stream after the call
 * is not waited for, so several calls can be kept in flight), otherwise
 * synchronizes `stream`, which must then be the call's stream; returns what
 * the synchronous call would have
 * returned for its device work: MAG_OK, MAG_E_TIMESTAMPS, MAG_E_POWER,
 * MAG_E_INTERVAL, MAG_E_CAPACITY or MAG_E_HIP; MAG_E_NULL or MAG_E_WORKSPACE
 * for a NULL or misaligned workspace.  A workspace that no asynchronous call
 * used gives unspecified results.
 */
int mag_attribute_finish(const void* workspace, mag_key_stats* per_key, mag_summary* summary,
                         hipStream_t stream);

/*
 * mag_counter_workspace_size -- bytes of device workspace mag_attribute_counter
 * needs for the given sizes, key-table capacity (0 when no per-key output is
 * asked for) and flags (MAG_KEY_LATENCY needs more).  Host only.  Returns
 * MAG_OK, MAG_E_SIZE or MAG_E_NULL.
 */
int mag_counter_workspace_size(int64_t n_samples, int64_t n_intervals, int64_t key_capacity,
                               uint32_t flags, size_t* bytes);

/*
 * mag_attribute_counter -- per-operator energy from a cumulative energy
 * counter, the software mode of Section 5.2: vendor energy interfaces refresh
 * at 10-50 Hz and lag the device, so each operator is replayed back to back
 * until its window is long enough, and its energy is the counter's increase
 * over the window divided by the number of replays.  This library's reading:
 *   u_j    = timestamps[j] - delay (fp64): a reading taken at t_j holds the
 *            energy used up to t_j - delay;
 *   C^(x)  = linear interpolant of (u_j, counter[j]); C^(x) = counter[0] for
 *            x <= u_0 and counter[n-1] for x >= u_{n-1};
 *   E_i    = (C^(ends[i]) - C^(starts[i])) / replays[i].
 * The increase is computed as the part of the start's segment after the
 * start, plus the difference of the two readings that bound the whole
 * segments in between, plus the part of the end's segment before the end; it
 * is never a difference of two interpolated values.
 * Per key: count, sum of E_i and M2, as mag_attribute.
 *
 * Arguments (device arrays unless noted):
 *   timestamps[n_samples] fp64 reading times (s); timestamps - delay strictly
 *                          increasing and finite
 *   counter[n_samples]    fp64 cumulative energy (J), finite, non-decreasing
 *   delay                 host fp64, seconds (finite; may be 0 or negative)
 *   starts/ends[n_intervals] fp64 replay windows, one sequence:
 *                          starts[i] <= ends[i] <= starts[i+1]
 *   replays[n_intervals]  int32 >= 1, or NULL for one run per window
 *   op_keys[n_intervals]  uint64 operator key; may be NULL when per_key is NULL
 *   flags                 MAG_SKIP_VALIDATE | MAG_TIME_KERNELS | MAG_ASYNC |
 *                          MAG_KEY_LATENCY (per-key sum of (ends - starts) /
 *                          replays); other bits are ignored
 *   per_interval          energy = E_i (J per run), start_idx / end_idx =
 *                          lower_bound of starts[i] / ends[i] among u; may be
 *                          NULL
 *   keys_out, per_key     as mag_attribute
 *   summary               host, may be NULL: trace_energy = counter[n-1] -
 *                          counter[0]; idle_energy = counter increase outside
 *                          every window; attributed_energy = sum of E_i;
 *                          n_clipped = windows with start < u_0 or end >
 *                          u_{n-1}; tile_kernel_ms = duration of the window
 *                          kernel
 *   workspace             device, >= mag_counter_workspace_size(...) bytes,
 *                          256-byte aligned
 * Synchronizes `stream` (with MAG_ASYNC: returns once the work is enqueued;
 * mag_attribute_finish completes it).  Errors: MAG_E_NULL, MAG_E_SIZE,
 * MAG_E_WORKSPACE, MAG_E_ALIGN, MAG_E_TIMESTAMPS (also for a non-finite delay)
 * (host-detected); MAG_E_TIMESTAMPS, MAG_E_COUNTER, MAG_E_INTERVAL (also for
 * replays < 1) (device-detected unless MAG_SKIP_VALIDATE); MAG_E_CAPACITY;
 * MAG_E_HIP.
 */
int mag_attribute_counter(const double* timestamps, const double* counter, int64_t n_samples,
                          double delay, const double* starts, const double* ends,
                          const int32_t* replays, const uint64_t* op_keys, int64_t n_intervals,
                          uint32_t flags, mag_interval_out* per_interval, uint64_t* keys_out,
                          mag_key_stats* per_key, mag_summary* summary, void* workspace,
                          size_t workspace_bytes, hipStream_t stream);

/*
 * mag_diff_workspace_size -- device workspace bytes for mag_diff.  Host only.
 */
int mag_diff_workspace_size(int64_t n_keys_a, int64_t n_keys_b, int64_t k, size_t* bytes);

/*
 * mag_diff -- join two per-key tables and rank the keys by relative energy
 * difference (Section 6.1 compares the energy of matched operators; Table
 * "tab:energy-profiling" uses (value - reference) / reference).
 *   keysA[statsA->n_keys], keysB[statsB->n_keys]: strictly ascending uint64
 *   (as produced by mag_attribute); statsA/statsB: host structs of device
 *   arrays (sum and count are read).  Rows are the keys present in both
 *   tables, r = (sum_B - sum_A) / sum_A (+inf if sum_A = 0 < sum_B, 0 if both
 *   are 0), ordered by r descending then key ascending (unsigned); the first
 *   min(k, joined) rows are written to out (device arrays, host counts).
 * Synchronizes `stream`.  Errors: MAG_E_NULL, MAG_E_SIZE (k < 0 or a negative
 * n_keys), MAG_E_CAPACITY (out->capacity < min(k, joined) possible rows, i.e.
 * < min(k, n_keys_a)), MAG_E_WORKSPACE, MAG_E_KEYS, MAG_E_HIP.
 */
int mag_diff(const uint64_t* keysA, const mag_key_stats* statsA, const uint64_t* keysB,
             const mag_key_stats* statsB, int64_t k, mag_rank_out* out, void* workspace,
             size_t workspace_bytes, hipStream_t stream);

/*
 * mag_diff_async -- mag_diff without the wait (Section 6.1's comparison, for
 * callers that keep several comparisons in flight): the arguments, checks and
 * device outputs are mag_diff's, written in `stream` order; the call returns
 * once the kernels and a copy of the call's status block are enqueued.  The
 * host counts of *out (n_out, n_only_a, n_only_b, n_join) are filled by
 * mag_diff_finish, which must be called before the workspace is used again
 * (one unfinished call per workspace; another call on it returns
 * MAG_E_STATE).  A device-detected error (MAG_E_KEYS) is returned by
 * mag_diff_finish.  Errors: as mag_diff, and MAG_E_STATE.
 */
int mag_diff_async(const uint64_t* keysA, const mag_key_stats* statsA, const uint64_t* keysB,
                   const mag_key_stats* statsB, int64_t k, mag_rank_out* out, void* workspace,
                   size_t workspace_bytes, hipStream_t stream);

/*
 * mag_diff_finish -- waits for the mag_diff_async call on `workspace` (an
 * event recorded after the call's status copy; later work on its stream is
 * not waited for) and fills the host counts of *out.  Must run on the host
 * thread that made the call.  Errors: MAG_E_NULL,
 * MAG_E_STATE (no unfinished mag_diff_async call on this workspace), MAG_E_KEYS,
 * MAG_E_HIP.
 */
int mag_diff_finish(const void* workspace, mag_rank_out* out);

/*
 * mag_diff_batch -- one baseline table A ranked against several candidate
 * tables B_0 .. B_{n-1} (Section 6.1 evaluates each case by comparing a
 * system against its more efficient counterparts, Table
 * "tab:known-issues-diagnosis"): for every candidate c exactly what
 * mag_diff(keysA, statsA, keysB[c], &statsB[c], k, &out[c]) computes, in a
 * fixed number of launches per 8 candidates (the candidates' parameters
 * travel as kernel arguments, one candidate per grid z index).
 *   n_candidates  0 .. MAG_DIFF_BATCH_MAX (0: nothing is done)
 *   keysB         HOST array of n_candidates device pointers
 *   statsB, out   HOST arrays of n_candidates structs (as in mag_diff)
 *   workspace     device, >= mag_diff_batch_workspace_size(n_keys_a,
 *                 n_candidates, k) bytes (n_keys_a: statsA's n_keys, or its
 *                 capacity when counted on the device)
 * Synchronizes `stream` once.  Errors as mag_diff (the first failing
 * candidate's), and MAG_E_SIZE for n_candidates out of range.
 */
#define MAG_DIFF_BATCH_MAX 1024
int mag_diff_batch_workspace_size(int64_t n_keys_a, int32_t n_candidates, int64_t k,
                                  size_t* bytes);
int mag_diff_batch(const uint64_t* keysA, const mag_key_stats* statsA, int32_t n_candidates,
                   const uint64_t* const* keysB, const mag_key_stats* statsB, int64_t k,
                   mag_rank_out* out, void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------ tensor matching (4.2) */
#define MAG_SVD_MAX_RANK 5
#define MAG_SVD_MAX_K 8192 /* largest min(M, N) of an unfolding this library handles */

/* A dense tensor: fp32, row-major (the last mode fastest), on the device. */
typedef struct mag_tensor {
    const float* data;
    int32_t rank;  /* 1 .. MAG_SVD_MAX_RANK */
    int32_t reserved;
    int64_t dims[MAG_SVD_MAX_RANK]; /* each >= 1; the product below 2^31 */
} mag_tensor;

/*
 * mag_invariant_count -- size of a tensor's multi-mode SVD invariant list
 * (Section 4.2): the unfoldings T_(G) over the non-empty proper mode subsets G
 * that contain mode 0 (T_(G^c) is the transpose of T_(G) and has the same
 * singular values), 2^(rank-1) - 1 of them, and the total number of singular
 * values, the sum of min(M_G, N_G).  Host only.  MAG_E_NULL, MAG_E_SIZE
 * (a rank or size out of range, or an unfolding with min(M, N) above
 * MAG_SVD_MAX_K).
 */
int mag_invariant_count(const mag_tensor* tensor, int32_t* n_unfoldings, int64_t* n_values);

/*
 * mag_invariants_workspace_size / mag_invariants -- the invariant lists of
 * n_tensors tensors (host array of descriptors).  spectra (device fp64)
 * receives the lists one after the other in tensor order; inside a list the
 * unfoldings come in increasing order of the bit mask of G (bit i = mode i),
 * each as its min(M, N) singular values in descending order.  The unfolding
 * has the modes of G as rows and the others as columns, both in increasing
 * mode order.  Singular values are the square roots of the eigenvalues of the
 * fp64 Gram matrix of the unfolding's shorter side (fp32 data widened
 * exactly; MFMA products), reduced to tridiagonal form and bisected; an
 * eigenvalue is within about 1e-13 of the largest (relative), so a singular
 * value far below the largest carries an absolute error near 3e-7 of it.
 * Gram sides up to 512 are reduced by one workgroup each, all unfoldings side
 * by side, and their eigenvalues then bisected by waves spread over the whole
 * device (the workspace holds each tridiagonal form between the two); larger
 * ones (up to MAG_SVD_MAX_K) one after another, each
 * Householder step spread over the whole device (about 4 launches per row of
 * the Gram matrix, so a side of n costs some 4 n launches; the workspace then
 * also holds about (n / 256 + 4) n doubles of scratch).
 * Synchronizes `stream`.  Errors: MAG_E_NULL, MAG_E_SIZE, MAG_E_ALIGN,
 * MAG_E_WORKSPACE, MAG_E_HIP.
 */
int mag_invariants_workspace_size(const mag_tensor* tensors, int32_t n_tensors, size_t* bytes);
int mag_invariants(const mag_tensor* tensors, int32_t n_tensors, double* spectra, void* workspace,
                   size_t workspace_bytes, hipStream_t stream);

/*
 * mag_match_workspace_size / mag_match -- which tensors of set A are
 * equivalent to which tensors of set B (Section 4.2: equivalent when their
 * invariant sets match under a tolerance).  spectra_a / spectra_b are
 * mag_invariants outputs for the same descriptors.  Tensors a and b match when
 * their lists can be paired one to one so that paired spectra have the same
 * length and differ by at most eps x (the larger of the two leading singular
 * values) at every position.  match[i * nb + j] (device uint8) = 1 or 0.
 * Synchronizes `stream`.  Errors: MAG_E_NULL, MAG_E_SIZE (also eps negative or
 * NaN), MAG_E_WORKSPACE, MAG_E_HIP.
 */
int mag_match_workspace_size(int32_t na, int32_t nb, size_t* bytes);
int mag_match(const mag_tensor* ta, int32_t na, const double* spectra_a, const mag_tensor* tb,
              int32_t nb, const double* spectra_b, double eps, uint8_t* match, void* workspace,
              size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------- subgraph matching (4.2) */
/* A computational graph on the host: operators 0..n_nodes-1, edge e (a tensor)
   from src[e] to dst[e]; node 0 is the input, node n_nodes-1 the output. */
typedef struct mag_graph {
    int32_t n_nodes;
    int32_t n_edges;
    const int32_t* src;
    const int32_t* dst;
} mag_graph;

/*
 * mag_match_subgraphs -- Section 4.2's topology-aware matching of two
 * computational graphs (host only; no device work).  eq[2 p], eq[2 p + 1]:
 * node of g1 and node of g2 whose output tensors are equivalent (as found by
 * mag_match).  Readings of the printed algorithm: the dominator path of a
 * graph is the chain of its output's dominators, input first; the cut points
 * are the eq pairs on both dominator paths plus the inputs and the outputs,
 * reduced to the longest chain rising in both paths (ties: the chain whose
 * sequence of path positions is lexicographically smallest); the region
 * between consecutive cuts c and c' is every node c dominates minus those c'
 * strictly dominates; region pairs are matched again recursively with eq
 * restricted to them, and a pair without an interior cut is a finest match.
 * out[4 q .. 4 q + 3] = entry and exit node of the q-th finest pair in g1,
 * then in g2, in path order; *n_out = the number of pairs.
 * Errors: MAG_E_NULL, MAG_E_SIZE (fewer than 2 nodes, a node index out of
 * range), MAG_E_GRAPH (a cycle, or a node off every input-to-output path),
 * MAG_E_CAPACITY (*n_out still reports the count).
 */
int mag_match_subgraphs(const mag_graph* g1, const mag_graph* g2, const int32_t* eq,
                        int32_t n_eq, int32_t* out, int32_t capacity, int32_t* n_out);

/*
 * mag_detect_workspace_size -- device workspace bytes for mag_detect with
 * `rows` output rows.  Host only.
 */
int mag_detect_workspace_size(int64_t n_keys_a, int64_t n_keys_b, int64_t rows, size_t* bytes);

/*
 * mag_detect -- Section 6.1's detection of energy inefficiencies over two
 * per-key tables: a key present on both sides is flagged when B's energy
 * exceeds A's by at least the threshold, r = (E_B - E_A) / E_A >= threshold
 * (the paper uses 10 % and finds 5 % free of false positives); a flagged key
 * is software energy waste when the efficient side A is not slower than B by
 * more than the tolerance, (L_A - L_B) <= tolerance * L_B with L the per-key
 * latency (the paper allows 1 %), and a performance-energy trade-off
 * otherwise.  (The paper's second condition, outputs within 1 %, concerns the
 * operators' results, which this library does not see.)  Swap A and B to
 * examine the other direction.
 *   keysA/statsA, keysB/statsB as for mag_diff, and both duration arrays
 *   (mag_attribute with MAG_KEY_LATENCY) must be given.
 *   out->rank.capacity rows are available; the first
 *   min(capacity, n_flagged) flagged keys, in the ranking's order (r
 *   descending, key ascending), are written with their energies, counts,
 *   latencies and verdicts; out->rank.n_out receives that number, and
 *   n_flagged / n_waste / n_tradeoff count every flagged key.
 *   opts: NULL for threshold 0.10 and tolerance 0.01.
 * Synchronizes `stream`.  Errors: as mag_diff, plus MAG_E_NULL for a missing
 * duration array and MAG_E_SIZE for a threshold or tolerance that is NaN.
 */
int mag_detect(const uint64_t* keysA, const mag_key_stats* statsA, const uint64_t* keysB,
               const mag_key_stats* statsB, const mag_detect_opts* opts, mag_detect_out* out,
               void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Chunked streaming.  A long trace (for example an hour of samples at
 * 100 kHz, Section 5.2's continuous power source) can be attributed while it
 * arrives, chunk by chunk, with the intervals already resident on the device.
 * The result is the one mag_attribute would give for the concatenated trace,
 * bit for bit: the same tiles run the same kernels, whatever the chunking.
 * Carried from chunk to chunk, inside the caller's workspace: the per-tile
 * stream cursors and partial energies of intervals still open, the samples of
 * the tile that straddles the chunk boundary, and the status block.
 *
 *   mag_stream_workspace_size(max_samples, n_intervals, key_capacity, opts,
 *                             &bytes)
 *       workspace for a trace of at most max_samples samples (host only).
 *   mag_stream_begin(&h, max_samples, starts, ends, op_keys, n_intervals,
 *                    opts, per_interval, key_capacity, workspace, bytes,
 *                    stream)
 *       intervals, keys, options and per-interval outputs as for
 *       mag_attribute (they must stay valid and unchanged until
 *       mag_stream_end); key_capacity > 0 reserves the per-key table
 *       (op_keys required), 0 skips grouping.  Host checks only; *h is a
 *       host object owned by the caller until mag_stream_end or
 *       mag_stream_abort.
 *   mag_stream_push(h, t_chunk, p_chunk, n_chunk)
 *       the next n_chunk samples (device arrays, same layout and rules as
 *       mag_attribute's timestamps/power; n_chunk may be 0).  Asynchronous on
 *       the stream given at begin: the chunk must stay unchanged until the
 *       work enqueued by this call has run (reusing it from later work on the
 *       same stream is safe).  Errors: MAG_E_SIZE (more than max_samples in
 *       total), MAG_E_NULL, MAG_E_ALIGN, MAG_E_STATE, MAG_E_HIP.
 *       Device-detected input errors are reported by mag_stream_end.
 *   mag_stream_end(h, keys_out, per_key, summary)
 *       runs the last tile, the cross-tile fix-ups and the grouping, and
 *       synchronizes; per_key (capacity equal to key_capacity) may be NULL.
 *       Returns what mag_attribute would return for the whole trace, or
 *       MAG_E_STATE (a failed push), MAG_E_SIZE (fewer than 2 samples).
 *       Always releases h.
 *   mag_stream_abort(h)
 *       releases h without finishing (no device work).
 *   mag_stream_state_export(h, host_buf, &bytes)
 *       checkpoint: copies the carried state, and the per-interval outputs
 *       written so far, to host memory (host_buf NULL: *bytes = size needed).
 *       Synchronizes the stream.
 *   mag_stream_state_import(h, host_buf, bytes)
 *       resume: h must be freshly begun with the same sizes, options and
 *       output set as the exported stream (other device addresses are fine);
 *       the next push continues after the last exported sample.  MAG_E_STATE
 *       for a mismatch, MAG_E_SIZE for a short buffer.
 */
typedef struct mag_stream mag_stream;

int mag_stream_workspace_size(int64_t max_samples, int64_t n_intervals, int64_t key_capacity,
                              const mag_attr_opts* opts, size_t* bytes);
int mag_stream_begin(mag_stream** handle, int64_t max_samples, const double* starts,
                     const double* ends, const uint64_t* op_keys, int64_t n_intervals,
                     const mag_attr_opts* opts, mag_interval_out* per_interval,
                     int64_t key_capacity, void* workspace, size_t workspace_bytes,
                     hipStream_t stream);
int mag_stream_push(mag_stream* handle, const double* t_chunk, const float* p_chunk,
                    int64_t n_chunk);
int mag_stream_end(mag_stream* handle, uint64_t* keys_out, mag_key_stats* per_key,
                   mag_summary* summary);
void mag_stream_abort(mag_stream* handle);
int mag_stream_state_export(const mag_stream* handle, void* host_buf, size_t* bytes);
int mag_stream_state_import(mag_stream* handle, const void* host_buf, size_t bytes);

/*
 * Chunks pushed from HOST memory (the long-run case of a trace that arrives
 * over time, Section 5.2's continuous microsecond-resolution power source,
 * reaching the GPU over PCIe).  The chunk is copied into one of two device
 * halves of a caller-owned staging buffer on a caller-owned copy stream while
 * the previous chunk's tiles run on the compute stream, so copy and compute
 * overlap (pinned host memory is needed for the copies to be asynchronous;
 * pageable memory works, with copies that block the calling thread).
 *   mag_stream_host_staging_size(max_chunk, &bytes)
 *       device bytes of a staging buffer for chunks of up to max_chunk
 *       samples (two halves of 12 B per sample).  MAG_E_SIZE for
 *       max_chunk < 1 or > MAG_MAX_SAMPLES.
 *   mag_stream_set_host_staging(h, max_chunk, staging, staging_bytes, copy_stream)
 *       once per handle, before the first mag_stream_push_host: staging is
 *       device memory (256-byte aligned, >= the size above) that must stay
 *       allocated until mag_stream_end / mag_stream_abort; copy_stream must
 *       differ from the stream given at begin.  Creates two pairs of HIP
 *       events, released with the handle.  MAG_E_STATE if staging is already
 *       set, MAG_E_WORKSPACE, MAG_E_NULL, MAG_E_HIP.
 *   mag_stream_push_host(h, t_host, p_host, n_chunk)
 *       the next n_chunk <= max_chunk samples from host memory, same rules as
 *       mag_stream_push otherwise.  The host chunk must stay unchanged until
 *       the second later mag_stream_push_host call returns, or until
 *       mag_stream_end / mag_stream_abort (the call waits on the host for the
 *       copy of the chunk pushed two calls earlier, whose half it reuses).
 *       Chunks from device memory (mag_stream_push) and from host memory may
 *       be mixed.  Errors as mag_stream_push, and MAG_E_STATE without staging.
 */
int mag_stream_host_staging_size(int64_t max_chunk, size_t* bytes);
int mag_stream_set_host_staging(mag_stream* handle, int64_t max_chunk, void* staging,
                                size_t staging_bytes, hipStream_t copy_stream);
int mag_stream_push_host(mag_stream* handle, const double* t_host, const float* p_host,
                         int64_t n_chunk);

/* Static description of a status code. */
const char* mag_strerror(int status);
/* Detail of the last error on the calling thread ("" if none). */
const char* mag_last_error(void);
/* Library version string. */
const char* mag_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MAGNETON_H */
