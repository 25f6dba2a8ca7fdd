// mag_internal.hpp -- shared definitions of the HIP kernels and the host
// orchestration of the attribution library (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "magneton.h"

namespace mag {

// ---------------------------------------------------------------- tiling
// A tile is TILE consecutive sample segments [t_j, t_{j+1}] (TILE + 1 samples,
// the last one shared with the next tile), processed by one 64-lane wave whose
// lanes each own SEG_PER_THREAD consecutive segments.  Interval endpoints
// inside a tile are processed in rounds of at most ROUND_EVENTS endpoints.
constexpr int SEG_PER_THREAD = 8;
constexpr int TILE = 64 * SEG_PER_THREAD;  // 512
constexpr int ROUND_EVENTS = 64;
constexpr int MAX_STREAMS = MAG_MAX_STREAMS;

// group-by
constexpr int AGG_THREADS = 1024;
constexpr int AGG_IDS = 8192;       // key ids per LDS table (count u32 + sum f64)
constexpr int AGG_MAX_CHUNKS = 256; // interval chunks (partial tables)

// workgroups of k_fix that add up the per-run trace and idle energies; each
// leaves its partial sum in a fold array that the call's last kernel adds up
constexpr int FOLD_BLOCKS = 256;

// cnt_fin entry that no workgroup wrote (no workgroup of any launch ended there)
constexpr int64_t CNT_UNSET = -1;

// device-side error bits
enum : uint32_t {
    ERR_TIMESTAMPS = 1u,
    ERR_POWER = 2u,
    ERR_INTERVAL = 4u,
    ERR_KEYS = 8u,
    ERR_COUNTER = 16u,
};

// small device status block at the head of every workspace
struct Status {
    uint32_t err;
    uint32_t n_flag;      // detect: joined keys at or above the threshold
    uint32_t special;     // the all-ones key was seen (stored out of band)
    uint32_t overflow;    // a key found no free slot
    unsigned long long n_clipped;
    uint32_t n_unique;    // rows of the compacted distinct-key list
    uint32_t n_cand;      // diff: surviving candidates
    uint32_t n_join;      // diff: keys present on both sides
    uint32_t n_waste;     // detect: flagged keys judged waste
    double trace_energy;
    double idle_energy;
    double attributed_energy;
    double bounds[2];     // t_0 and t_{n-1}
    uint32_t diff_na;     // diff: key-table rows read on the device
    uint32_t diff_nb;
};
static_assert(sizeof(Status) <= 256, "status block");

struct StreamSet {
    int32_t S;
    int32_t pad;
    int64_t off[MAX_STREAMS + 1];
};

struct TileParams {
    const double* t;    // sample g (global index) is t[g - base]
    const float* P;
    int64_t base;
    int64_t nseg;       // segments of the whole trace (n_samples - 1)
    int64_t n_total;    // samples of the whole trace
    int64_t tile_begin; // global tile range of this launch
    int64_t tile_end;
    int64_t tiles_per_wg; // set by launch_tile
    int64_t NT;         // tiles of the whole trace (any larger value when not yet known)
    int64_t ld;         // row stride of cnt/cnt_fin (ld + 1) and head/tail (ld), ld >= tiles
    const double* s;
    const double* e;
    StreamSet ss;
    double* energy;
    int64_t* start_idx;
    int64_t* end_idx;
    int64_t* cnt;       // [S][ld+1] endpoints <= tile start time, per stream
    int64_t* cnt_fin;   // [S][ld+1] cursor of a workgroup after its last tile, at the index of
                        // the tile after it (CNT_UNSET where no workgroup ended)
    double* head;       // [S][ld] in-tile energy of the interval active at tile start
    double* tail;       // [S][ld] in-tile energy of the interval started in the tile, active at its end
    Status* status;
    double2* part;      // [ld] {trace, idle} energy of the wave whose run of tiles starts at b
    int split;
    int validate;
    int aligned16;      // t and P are 16-byte aligned (vector loads)
};

struct FixParams {
    const double* s;
    const double* e;
    StreamSet ss;
    int64_t NT;
    int64_t ld;           // row strides as in TileParams
    int64_t n_total;
    const int64_t* cnt;
    const int64_t* cnt_fin;
    const double* head;
    const double* tail;
    double* energy;
    int64_t* start_idx;
    int64_t* end_idx;
    Status* status;
    const double2* part;  // per-run {trace, idle} energies (TileParams::part), added up here
    double2* fold;        // [FOLD_BLOCKS] partial sums of part, one per fold workgroup
    int validate;
    // group-by state cleared for the grouping that follows (table NULL: none)
    unsigned long long* table;     // [2 (H+1)] {key, id} slots: all ones = empty / no id
    uint32_t H;
    uint32_t* urank;               // [H+1] rank counters
};

struct GroupParams {
    const uint64_t* keys;
    const double* energy;
    int64_t m;
    uint32_t H;           // hash slots (power of two); slot H holds the all-ones key
    int64_t cap;          // key rows available
    int nchunks;
    int64_t chunk;        // intervals per chunk
    unsigned long long* table;  // [2 (H+1)] slot h = {key, id}; slot H: the all-ones key
    uint32_t* slot;       // [m] id of each interval's key, or MISS | slot (k_keymap)
    uint64_t* ukey;       // [H+1] distinct keys, by dense id
    uint32_t* urank;      // [H+1] rank of each distinct key (zeroed, then counted)
    double* mean;         // [cap]
    uint32_t* pcnt;       // [nchunks][cap]
    double* psum;         // [nchunks][cap]
    double* pm2;          // [nchunks][cap]
    uint64_t* keys_out;   // [cap]
    double* sum_out;
    double* m2_out;
    int64_t* count_out;
    Status* status;
    // per-key latency (dur_out NULL: none): sum of (e - s) / reps (reps NULL: 1)
    const double* s;
    const double* e;
    const int32_t* reps;
    double* dur_out;      // [cap]
    double* pdur;         // [nchunks][cap]
    int64_t* n_keys_out;  // device copy of the number of rows filled, or NULL
    // the key state (distinct-key count, all-ones key seen, table overflow):
    // the call's own status block when the call builds its key map, the
    // header of a key plan built beforehand otherwise (the aggregation then
    // copies the count and the overflow flag into the call's status)
    Status* kstat;
    // the call's totals, written by its last kernel with plain stores:
    // attributed energy = sum of ctot (one entry per interval chunk, written
    // by the aggregation); trace and idle energy = sum of fold (NULL: set
    // elsewhere)
    double* ctot;         // [nchunks]
    const double2* fold;  // [FOLD_BLOCKS] or NULL
};

// per-operator energy from a delayed cumulative energy counter
constexpr int CNT_CHUNK = 64;   // windows per wave (one per lane)
constexpr int CNT_BLOCK = 256;  // readings streamed through LDS at a time (4 per lane)
constexpr int CNT_WAVES = 4;    // waves (independent chunks) per workgroup

struct CounterParams {
    const double* t;      // [n] reading times
    const double* C;      // [n] cumulative energy
    int64_t n;
    double delay;         // u_j = t_j - delay
    const double* s;      // [m] window starts
    const double* e;      // [m] window ends
    const int32_t* reps;  // [m] replays per window, NULL: 1
    int64_t m;
    int64_t nchunks;      // ceil(m / CNT_CHUNK), at least 1
    double* energy;       // [m]
    int64_t* start_idx;   // [m] or NULL
    int64_t* end_idx;     // [m] or NULL
    double2* part;        // [nchunks] {sum of window increases, windows clipped}
    Status* status;
    int validate;
    // group-by state cleared by the fold kernel (table NULL: none)
    unsigned long long* table;
    uint32_t H;
    uint32_t* urank;
};

struct DiffParams {
    const uint64_t* ka;
    const double* sa;
    const int64_t* ca;
    int64_t na;
    const uint64_t* kb;
    const double* sb;
    const int64_t* cb;
    int64_t nb;
    int64_t k;
    double* cand_r;
    uint64_t* cand_key;
    int32_t* cand_ia;
    int32_t* cand_ib;
    uint32_t* cand_rank;  // global rank of each candidate (counted by k_diff_rank)
    uint32_t* blk;        // [n_groups][8] per join workgroup: joined, candidates, flagged,
                          // waste, error bits
    int64_t n_groups;     // join workgroups (diff_groups(na))
    int64_t n_slots;      // candidate slots (diff_max_candidates(na, k))
    uint64_t* out_key;
    double* out_ratio;
    double* out_ea;
    double* out_eb;
    int64_t* out_ca;
    int64_t* out_cb;
    Status* status;
    // detection (detect != 0): flag r >= threshold; waste when
    // (la - lb) <= tolerance * lb
    // key-table rows on the device (NULL: na / nb are the counts; otherwise
    // na / nb are upper bounds and the counts are read here)
    const int64_t* na_dev;
    const int64_t* nb_dev;
    int detect;
    double threshold;
    double tolerance;
    const double* la;     // [na] per-key latency of A
    const double* lb;     // [nb]
    double* out_la;
    double* out_lb;
    int32_t* out_verdict;
};

// Workgroup barrier for LDS traffic only: waits for this wave's LDS operations
// and meets the other waves, without the global-memory fence that
// __syncthreads() implies (which would also wait for every in-flight global
// load and store, prefetches included).  Kernels use it wherever the waves
// only communicate through LDS.
__device__ __forceinline__ void lds_barrier()
{
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// launchers (return hipError_t of the launch)
// status block reset (bounds from t[0], t[n-1] when t is given) and cnt_fin := CNT_UNSET
hipError_t launch_init(Status* st, int64_t* cnt_fin, int64_t n_fin, const double* t, int64_t n,
                       hipStream_t stream);
hipError_t launch_init_status(Status* st, const double* t, int64_t n, hipStream_t stream);
// n samples (time and power) copied in one launch: the staging of a streamed
// tile that spans two chunks
hipError_t launch_stage_copy(double* dst_t, const double* src_t, float* dst_P, const float* src_P,
                             int64_t n, hipStream_t stream);
// tiles [p.tile_begin, p.tile_end) on persistent waves (sets the launch shape);
// ev_start / ev_stop (may be NULL) are recorded by the launch itself
hipError_t launch_tile(const TileParams& p, hipStream_t stream, hipEvent_t ev_start = nullptr,
                       hipEvent_t ev_stop = nullptr);
// intervals spanning tiles, endpoints outside the trace, clearing of the group-by state
hipError_t launch_fix(const FixParams& p, hipStream_t stream);
// the key map of a grouping (distinct keys, their ids and ranks, every
// interval's id): built into p.table / p.slot / p.ukey / p.urank / p.kstat;
// clear: the table, ranks and key state are cleared first (else k_fix did)
hipError_t launch_key_map(const GroupParams& p, bool clear, hipStream_t stream);
// the per-key aggregation over a built key map (count, sum, M2, latency, rows
// in key order)
hipError_t launch_aggregate(const GroupParams& p, hipStream_t stream);
// multi-mode SVD invariants (Section 4.2): one task per (tensor, unfolding)
constexpr int SVD_MAX_RANK = 5;
constexpr int SVD_MAX_K = 8192;       // largest Gram side (min(M, N) of an unfolding)
constexpr int SVD_SMALL_K = 512;      // Gram sides reduced by one workgroup (larger: many)
constexpr int SVD_MAX_UNF = 15;       // unfoldings of a rank-5 tensor, complements folded
constexpr int64_t GRAM_CHUNK = 2048;  // unfolding columns per Gram work item
constexpr int64_t GRAM_CHUNK_NARROW = 1024;  // the same for K <= GRAM_NARROW (one 32-side block)
constexpr int GRAM_NARROW = 32;       // Gram sides up to this use 32-side blocks (else 64)
constexpr int EIG_PER_ITEM = 16;      // eigenvalues per work item of the Sturm counts
constexpr int GRAM_WHOLE = 128;       // sides in (64, GRAM_WHOLE]: the whole triangle per item
constexpr int64_t GRAM_CHUNK_WHOLE = 1024;  // unfolding columns per item for those sides

struct SvdTask {
    const float* data;
    int64_t K, L;  // the Gram matrix X X^T is K x K, X the unfolding's shorter-side view
    int32_t nk, nl;  // modes on the K side and on the L side
    int64_t kdim[SVD_MAX_RANK], kstr[SVD_MAX_RANK];  // sizes and element strides, last fastest
    int64_t ldim[SVD_MAX_RANK], lstr[SVD_MAX_RANK];
    double* gram;    // [K][K]
    double* out;     // [K] singular values, descending
    int64_t item0;   // first Gram work item of this task (within its block size's launch)
    double* tri;     // (K <= SVD_SMALL_K) the tridiagonal form: d[K], e2[K], glo, ghi, pivmin
    int64_t eig0;    // (K <= SVD_SMALL_K) first eigenvalue work item, EIG_PER_ITEM values each
    int32_t nt;      // row blocks: 1 when K <= GRAM_NARROW or 64 < K <= GRAM_WHOLE, else ceil(K / 64)
    int32_t nchunk;  // column chunks of L: GRAM_CHUNK_NARROW, GRAM_CHUNK_WHOLE or GRAM_CHUNK columns
};

// a tensor's invariant list inside a spectra array
struct SpecDesc {
    int32_t n;  // unfoldings
    int32_t pad;
    int64_t off[SVD_MAX_UNF];
    int64_t len[SVD_MAX_UNF];
};

// Gram matrices (zeroed, then accumulated), then the spectra of the tasks
// with K <= SVD_SMALL_K; the first n_narrow tasks (K <= GRAM_NARROW) are
// numbered by their own n_items_narrow work items, the next n_whole (64 < K <=
// GRAM_WHOLE) by n_items_whole, the others by n_items; the eigenvalue counts
// by n_eig_items (each task's from its eig0, in task order)
hipError_t launch_svd(const SvdTask* tasks, int n_tasks, int n_narrow, int64_t n_items_narrow,
                      int n_whole, int64_t n_items_whole, int64_t n_items, int64_t n_eig_items,
                      double* gram, int64_t gram_len, hipStream_t stream);
// the spectrum of one n x n Gram matrix with n > SVD_SMALL_K (overwritten):
// a Householder step is four launches over the whole device, then
// multisection on Sturm counts; scratch of svd_large_scratch(n) doubles
int64_t svd_large_scratch(int n);
hipError_t launch_svd_large(double* gram, int n, double* scratch, double* out,
                            hipStream_t stream);
// match[i * nb + j] = 1 when tensor i of A and tensor j of B have matching invariants
hipError_t launch_svd_match(const SpecDesc* da, int na, const double* sa, const SpecDesc* db,
                            int nb, const double* sb, double eps, uint8_t* match,
                            hipStream_t stream);

// Section 4.2's subgraph matching (host): finest pairs as (entry1, exit1,
// entry2, exit2) quadruples appended to out; MAG_OK or MAG_E_GRAPH
int match_subgraphs(const mag_graph& a, const mag_graph& b, const int32_t* eq, int32_t n_eq,
                    std::vector<int32_t>& out);

hipError_t launch_groupby(const GroupParams& p, hipStream_t stream);
// *dst = v, in stream order (a kernel, so the write can sit in a captured graph)
hipError_t launch_set_i64(int64_t* dst, int64_t v, hipStream_t stream);
// window energies of the counter mode (ev_start / ev_stop may be NULL), then the
// fold of the per-chunk figures into the status block and the group-by clearing
hipError_t launch_counter(const CounterParams& p, hipStream_t stream, hipEvent_t ev_start = nullptr,
                          hipEvent_t ev_stop = nullptr);
hipError_t launch_counter_fold(const CounterParams& p, hipStream_t stream);
// attributed energy = sum of energy[m]; trace and idle energy from the fold
// partials (fold NULL: left alone)
hipError_t launch_energy_total(const double* energy, int64_t m, const double2* fold, Status* st,
                               hipStream_t stream);
hipError_t launch_diff(const DiffParams& p, hipStream_t stream);
// comparisons per launch of a batch (their parameters travel as kernel arguments)
constexpr int DIFF_BATCH = 8;
// n comparisons sharing table A (p[c].ka/sa/ca/na/na_dev and k equal for all c)
hipError_t launch_diff_batch(const DiffParams* p, int n, hipStream_t stream);
// the diff's join workgroups for n_keys_a rows (at least one), and their
// candidate slots for top k
int64_t diff_groups(int64_t na);
int64_t diff_max_candidates(int64_t na, int64_t k);

int device_cu_count();

}  // namespace mag
