// groupby.hip -- per-operator-key count, sum and M2 of the interval energies.
//
// The key table (keys and ids) and the rank counters are cleared by k_fix,
// the launch before.
//
// 1. k_key_insert: the distinct keys of a prefix of the intervals go into an
//    open-addressing hash table (linear probing, 64-bit compare-and-swap; the
//    all-ones key is kept out of band in slot H so any uint64 is a legal key).
//    A slot is 16 bytes, {key, id}, so a lookup reads both from one line.
//    Each workgroup de-duplicates its part of the prefix in LDS first.
// 2. k_compact: every occupied slot without an id takes the next dense id (its
//    place in the distinct-key list).
// 3. k_keymap: the id of every interval's key, found with plain cached loads
//    (the table and the ids come from earlier launches).  A key first seen
//    after the prefix is inserted and recorded as MISS | slot; k_compact, run
//    again, gives it an id, which the aggregation passes look up.
// 4. k_rank: rank of each key = number of smaller keys (its row in the output,
//    ascending by key).
// 5. k_agg_sum / k_fin_sum: each workgroup aggregates one chunk of intervals
//    into an LDS table indexed by id (count, sum); the partial tables are
//    reduced per key in chunk order, and the key, count and sum written to the
//    key's row.  Per-workgroup atomics add the rows into the attributed energy.
// 6. k_agg_m2 / k_fin_m2: second pass over the chunk for sum (E - mean)^2
//    (the two-pass definition of M2).
// When a chunk fits one batch of loads per thread (up to AGG_THREADS *
// AGG_BATCH intervals), steps 5 and 6 are one pass instead: k_agg_one keeps
// the chunk's ids and energies in registers, takes count and sum, then the
// chunk's own M2 about the chunk mean; k_fin_one merges the chunk rows per key
// by Chan, Golub and LeVeque's pairwise update, M2 = sum_c M2_c +
// sum_c n_c (mean_c - mean)^2 (every term non-negative).
// Plain stores carry every partial result: device-scope atomics, which are
// slow on this part, are used only for counters, inserts and one add per
// workgroup.  Every thread requests all the loads of a batch before it uses
// any of them, so a pass costs about one memory latency per batch.

#include "mag_internal.hpp"

namespace mag {

namespace {

constexpr unsigned long long EMPTY_KEY = ~0ull;
constexpr uint32_t NO_ID = 0xffffffffu;  // no id (also: table full)
constexpr uint32_t MISS = 0x80000000u;   // MISS | slot: id assigned after the lookup pass

// 64-bit finalizer of MurmurHash3 (Appleby): spreads keys over the table
__device__ __forceinline__ uint64_t fmix64(uint64_t k)
{
    k ^= k >> 33;
    k *= 0xff51afd7ed558ccdull;
    k ^= k >> 33;
    k *= 0xc4ceb9fe1a85ec53ull;
    k ^= k >> 33;
    return k;
}

// slot h of the table: {key, id}
__device__ __forceinline__ unsigned long long* slot_key(const GroupParams& p, uint32_t h)
{
    return p.table + 2 * (size_t)h;
}
__device__ __forceinline__ ulonglong2 slot_load(const GroupParams& p, uint32_t h)
{
    return reinterpret_cast<const ulonglong2*>(p.table)[h];
}

// the id of an interval's key from what the lookup pass recorded (NO_ID: none)
__device__ __forceinline__ uint32_t resolve_id(const GroupParams& p, uint32_t r)
{
    if (r == NO_ID || !(r & MISS)) return r;
    const uint32_t h = r & ~MISS;
    return (h <= p.H) ? (uint32_t)p.table[2 * (size_t)h + 1] : NO_ID;
}

// an interval's duration, per replay run when replay counts are given
__device__ __forceinline__ double interval_duration(const GroupParams& p, int64_t i)
{
    const double d = p.e[i] - p.s[i];
    return p.reps ? d / (double)p.reps[i] : d;
}

}  // namespace

// sum of v over a workgroup of nthreads (a multiple of 64) into thread 0's
// return value; red holds one value per wave
__device__ __forceinline__ double block_sum(double v, double* red, int nthreads)
{
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    double t = 0.0;
    if (threadIdx.x == 0)
        for (int w = 0; w < nthreads / 64; ++w) t += red[w];
    return t;
}

// the call's totals, by the first workgroup of its last kernel: attributed
// energy from the chunk totals, trace and idle energy from k_fix's fold
// partials (plain stores; no workgroup adds into a shared address)
__device__ void write_totals(const GroupParams& p, double* red, int nthreads)
{
    double a = 0.0, w = 0.0, i = 0.0;
    for (int c = threadIdx.x; c < p.nchunks; c += nthreads) a += p.ctot[c];
    if (p.fold)
        for (int b = threadIdx.x; b < FOLD_BLOCKS; b += nthreads) {
            w += p.fold[b].x;
            i += p.fold[b].y;
        }
    // the three sums reduced together: one pass over the waves
    for (int off = 32; off > 0; off >>= 1) {
        a += __shfl_xor(a, off);
        w += __shfl_xor(w, off);
        i += __shfl_xor(i, off);
    }
    if ((threadIdx.x & 63) == 0) {
        red[3 * (threadIdx.x >> 6)] = a;
        red[3 * (threadIdx.x >> 6) + 1] = w;
        red[3 * (threadIdx.x >> 6) + 2] = i;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        a = w = i = 0.0;
        for (int v = 0; v < nthreads / 64; ++v) {
            a += red[3 * v];
            w += red[3 * v + 1];
            i += red[3 * v + 2];
        }
        p.status->attributed_energy = a;
        if (p.fold) {
            p.status->trace_energy = w;
            p.status->idle_energy = i;
        }
    }
}

// Insert the distinct keys of a prefix of the intervals.  Each workgroup first
// de-duplicates its chunk in an LDS table; then every thread takes a few LDS
// slots and inserts their keys into the global table, all of them side by side
// (one probe round of every key per memory round trip).
constexpr int INS_THREADS = 512;
constexpr int INS_CHUNK = 2048;
constexpr int INS_SLOTS = 4096;
constexpr int INS_GROUPS = 128;  // the lookup pass inserts keys first seen later
constexpr int INS_PER = INS_CHUNK / INS_THREADS;
constexpr int INS_SPT = INS_SLOTS / INS_THREADS;

__global__ __launch_bounds__(INS_THREADS) void k_key_insert(const GroupParams p, int64_t n_insert)
{
    __shared__ unsigned long long lt[INS_SLOTS];
    const int tid = threadIdx.x;
    const int64_t lo = (int64_t)blockIdx.x * INS_CHUNK;
    unsigned long long kv[INS_PER];
#pragma unroll
    for (int u = 0; u < INS_PER; ++u) {
        const int64_t i = lo + tid + (int64_t)u * INS_THREADS;
        kv[u] = (i < n_insert) ? p.keys[i] : EMPTY_KEY;
    }
    for (int v = tid; v < INS_SLOTS; v += INS_THREADS) lt[v] = EMPTY_KEY;
    __syncthreads();
    bool special = false;
#pragma unroll
    for (int u = 0; u < INS_PER; ++u) {
        const int64_t i = lo + tid + (int64_t)u * INS_THREADS;
        const unsigned long long k = kv[u];
        if (i >= n_insert) continue;
        if (k == EMPTY_KEY) {
            special = true;
            continue;
        }
        uint32_t h = (uint32_t)fmix64(k) & (INS_SLOTS - 1);
        for (int probe = 0; probe < INS_SLOTS; ++probe) {
            const unsigned long long old = atomicCAS(&lt[h], EMPTY_KEY, k);
            if (old == EMPTY_KEY || old == k) break;
            h = (h + 1u) & (INS_SLOTS - 1);
        }
    }
    if (special) atomicOr(&p.kstat->special, 1u);
    __syncthreads();

    const uint32_t mask = p.H - 1u;
    unsigned long long key[INS_SPT];
    uint32_t h[INS_SPT];
    uint32_t pending = 0u;
#pragma unroll
    for (int u = 0; u < INS_SPT; ++u) {
        key[u] = lt[tid + u * INS_THREADS];
        h[u] = (uint32_t)fmix64(key[u]) & mask;
        if (key[u] != EMPTY_KEY) pending |= 1u << u;
    }
    for (uint32_t probe = 0; pending != 0u && probe < p.H; ++probe) {
        // device-coherent loads (the level-2 caches of the XCDs are not
        // coherent with each other, so a plain load could keep returning a
        // stale empty slot and force a swap per probe); a slot only ever
        // changes from empty to its final key, so a non-empty value is final
        unsigned long long cur[INS_SPT];
#pragma unroll
        for (int u = 0; u < INS_SPT; ++u)
            cur[u] = ((pending >> u) & 1u)
                         ? __hip_atomic_load(slot_key(p, h[u]), __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT)
                         : 0ull;
        unsigned long long old[INS_SPT];
#pragma unroll
        for (int u = 0; u < INS_SPT; ++u)
            old[u] = (((pending >> u) & 1u) && cur[u] == EMPTY_KEY)
                         ? atomicCAS(slot_key(p, h[u]), EMPTY_KEY, key[u])
                         : cur[u];
#pragma unroll
        for (int u = 0; u < INS_SPT; ++u) {
            if (!((pending >> u) & 1u)) continue;
            if (old[u] == key[u] || (cur[u] == EMPTY_KEY && old[u] == EMPTY_KEY))
                pending &= ~(1u << u);
            else
                h[u] = (h[u] + 1u) & mask;
        }
    }
    if (pending) atomicOr(&p.kstat->overflow, 1u);
}

// ids for the occupied slots that have none yet (slot H: the all-ones key);
// each workgroup counts its new ids, takes a range of them with one atomic,
// and hands them out in slot order within the workgroup
constexpr int CMP_THREADS = 1024;
constexpr int CMP_PER = 8;  // slots per thread

__global__ __launch_bounds__(CMP_THREADS) void k_compact(const GroupParams p)
{
    __shared__ uint32_t wtot[CMP_THREADS / 64];
    __shared__ uint32_t wbase[CMP_THREADS / 64];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t b0 = (int64_t)blockIdx.x * CMP_THREADS * CMP_PER;
    const bool special = p.kstat->special != 0u;
    unsigned long long key[CMP_PER];
    uint32_t cur[CMP_PER];
#pragma unroll
    for (int u = 0; u < CMP_PER; ++u) {
        const int64_t h = b0 + (int64_t)u * CMP_THREADS + tid;
        const ulonglong2 e = (h <= (int64_t)p.H) ? slot_load(p, (uint32_t)h)
                                                 : make_ulonglong2(EMPTY_KEY, 0ull);
        key[u] = e.x;
        cur[u] = (uint32_t)e.y;
    }
    uint32_t mine = 0u;  // bit u: slot u of this thread takes a new id
#pragma unroll
    for (int u = 0; u < CMP_PER; ++u) {
        const int64_t h = b0 + (int64_t)u * CMP_THREADS + tid;
        const bool occ = (h < (int64_t)p.H) ? (key[u] != EMPTY_KEY)
                                            : (h == (int64_t)p.H && special);
        if (occ && cur[u] == NO_ID) mine |= 1u << u;
    }
    // exclusive prefix of the counts over the workgroup
    const uint32_t c = (uint32_t)__popc(mine);
    uint32_t incl = c;
    for (int off = 1; off < 64; off <<= 1) {
        const uint32_t v = __shfl_up(incl, off);
        if (lane >= off) incl += v;
    }
    if (lane == 63) wtot[wave] = incl;
    __syncthreads();
    if (tid == 0) {
        uint32_t t = 0u;
        for (int w = 0; w < CMP_THREADS / 64; ++w) {
            wbase[w] = t;
            t += wtot[w];
        }
        const uint32_t base = t ? atomicAdd(&p.kstat->n_unique, t) : 0u;
        for (int w = 0; w < CMP_THREADS / 64; ++w) wbase[w] += base;
    }
    __syncthreads();
    uint32_t id = wbase[wave] + incl - c;
#pragma unroll
    for (int u = 0; u < CMP_PER; ++u) {
        if (!((mine >> u) & 1u)) continue;
        const int64_t h = b0 + (int64_t)u * CMP_THREADS + tid;
        p.ukey[id] = (h < (int64_t)p.H) ? key[u] : EMPTY_KEY;
        p.table[2 * h + 1] = id;
        ++id;
    }
}

// the id of every interval's key (plain cached probes: the table and the ids
// were written by earlier launches); keys missing from the table are inserted
// and recorded as MISS | slot.  A thread looks up KM_BATCH intervals, spaced
// a grid apart, with all their first probes in flight together.
constexpr int KM_THREADS = 256;
constexpr int KM_BATCH = 4;

__device__ __noinline__ uint32_t keymap_probe(const GroupParams& p, unsigned long long k,
                                              uint32_t h, bool& over)
{
    // the first probe missed: walk the chain, inserting the key if absent
    const uint32_t mask = p.H - 1u;
    for (uint32_t probe = 0; probe < p.H; ++probe) {
        const ulonglong2 e = slot_load(p, h);
        if (e.x == k) return ((uint32_t)e.y != NO_ID) ? (uint32_t)e.y : (MISS | h);
        if (e.x == EMPTY_KEY) {
            // a stale empty read is settled by the swap
            const unsigned long long old = atomicCAS(slot_key(p, h), EMPTY_KEY, k);
            if (old == EMPTY_KEY || old == k) return MISS | h;
        }
        h = (h + 1u) & mask;
    }
    over = true;
    return NO_ID;
}

__global__ __launch_bounds__(KM_THREADS) void k_keymap(const GroupParams p)
{
    const uint32_t H = p.H;
    const uint32_t mask = H - 1u;
    const int64_t T = (int64_t)gridDim.x * KM_THREADS;
    bool special = false, over = false;
    for (int64_t i0 = (int64_t)blockIdx.x * KM_THREADS + threadIdx.x; i0 < p.m;
         i0 += T * KM_BATCH) {
        unsigned long long k[KM_BATCH];
#pragma unroll
        for (int u = 0; u < KM_BATCH; ++u) {
            const int64_t i = min(i0 + u * T, p.m - 1);  // in bounds; extra lanes repeat the last
            k[u] = p.keys[i];
        }
        uint32_t h[KM_BATCH];
#pragma unroll
        for (int u = 0; u < KM_BATCH; ++u) h[u] = (uint32_t)fmix64(k[u]) & mask;
        // every first probe is issued before the first one is used
        asm volatile("" ::: "memory");
        ulonglong2 e[KM_BATCH];
#pragma unroll
        for (int u = 0; u < KM_BATCH; ++u) e[u] = slot_load(p, h[u]);
        asm volatile("" ::: "memory");
#pragma unroll
        for (int u = 0; u < KM_BATCH; ++u) {
            uint32_t id = (uint32_t)e[u].y;
            if (k[u] == EMPTY_KEY) {
                special = true;
                id = MISS | H;
            } else if (e[u].x != k[u] || id == NO_ID) {
                id = keymap_probe(p, k[u], h[u], over);
            }
            const int64_t i = i0 + u * T;
            if (i < p.m) p.slot[i] = id;
        }
    }
    if (special && p.kstat->special == 0u) atomicOr(&p.kstat->special, 1u);
    if (over) atomicOr(&p.kstat->overflow, 1u);
}

// rank = number of distinct keys smaller than this one: the pairs (x, y) of key
// tiles are spread over the workgroups; pair (x, y) compares keys
// [256 x, 256 x + 256) against keys [256 y, 256 y + 256)
constexpr uint32_t RANK_TILE = 256u;

__global__ __launch_bounds__(RANK_TILE) void k_rank(const GroupParams p)
{
    __shared__ uint64_t tile[RANK_TILE];
    const uint32_t nu = p.kstat->n_unique;
    const uint32_t nt = (nu + RANK_TILE - 1) / RANK_TILE;
    const uint64_t pairs = (uint64_t)nt * nt;
    for (uint64_t pr = blockIdx.x; pr < pairs; pr += gridDim.x) {
        const uint32_t bx = (uint32_t)(pr % nt), by = (uint32_t)(pr / nt);
        const uint32_t base = by * RANK_TILE;
        const uint32_t cnt = min(RANK_TILE, nu - base);
        __syncthreads();  // the previous pair's reads of the tile are done
        for (uint32_t v = threadIdx.x; v < cnt; v += RANK_TILE) tile[v] = p.ukey[base + v];
        __syncthreads();
        const uint32_t u = bx * RANK_TILE + threadIdx.x;
        if (u < nu) {
            const uint64_t mine = p.ukey[u];
            uint32_t rank = 0;
            uint32_t v = 0;
            for (; v + 16 <= cnt; v += 16) {
#pragma unroll
                for (int w = 0; w < 16; ++w) rank += (tile[v + w] < mine) ? 1u : 0u;
            }
            for (; v < cnt; ++v) rank += (tile[v] < mine) ? 1u : 0u;
            if (rank) atomicAdd(&p.urank[u], rank);
        }
    }
}

// intervals per thread whose loads are requested together
constexpr int AGG_BATCH = 16;

// chunk of intervals -> LDS table over ids [r0, r0 + SUM_IDS) -> partial table
// row.  Its 12 bytes per id fit 12,288 ids in 144 KiB of LDS, so a chunk is
// read once per 12,288 keys (the M2 pass, at 16 bytes per id, per 8,192)
constexpr int SUM_IDS = 12288;
__global__ __launch_bounds__(AGG_THREADS) void k_agg_sum(const GroupParams p)
{
    __shared__ uint32_t lcnt[SUM_IDS];
    __shared__ double lsum[SUM_IDS];
    const int c = blockIdx.x;
    const int64_t r0 = (int64_t)blockIdx.y * SUM_IDS;
    const int64_t nk = min((int64_t)p.kstat->n_unique, p.cap);
    if (r0 >= nk) return;  // uniform
    const int nid = (int)min((int64_t)SUM_IDS, nk - r0);
    for (int v = threadIdx.x; v < nid; v += AGG_THREADS) {
        lcnt[v] = 0u;
        lsum[v] = 0.0;
    }
    __syncthreads();
    const int64_t lo = (int64_t)c * p.chunk, hi = min(lo + p.chunk, p.m);
    double ctot = 0.0;  // the chunk's total energy (all its intervals)
    for (int64_t i0 = lo + threadIdx.x; i0 < hi; i0 += (int64_t)AGG_BATCH * AGG_THREADS) {
        uint32_t sl[AGG_BATCH];
        double en[AGG_BATCH];
#pragma unroll
        for (int k = 0; k < AGG_BATCH; ++k) {
            const int64_t i = i0 + (int64_t)k * AGG_THREADS;
            sl[k] = (i < hi) ? p.slot[i] : NO_ID;
            en[k] = (i < hi) ? p.energy[i] : 0.0;
        }
#pragma unroll
        for (int k = 0; k < AGG_BATCH; ++k) {
            ctot += en[k];
            const uint32_t id = resolve_id(p, sl[k]);
            const int64_t d = (id == NO_ID) ? -1 : (int64_t)id - r0;
            if (d < 0 || d >= nid) continue;
            atomicAdd(&lcnt[d], 1u);
            atomicAdd(&lsum[d], en[k]);
        }
    }
    __syncthreads();
    if (blockIdx.y == 0) {
        __shared__ double red[AGG_THREADS / 64];
        ctot = block_sum(ctot, red, AGG_THREADS);
        if (threadIdx.x == 0) p.ctot[c] = ctot;
    }
    for (int v = threadIdx.x; v < nid; v += AGG_THREADS) {
        p.pcnt[(int64_t)c * p.cap + r0 + v] = lcnt[v];
        p.psum[(int64_t)c * p.cap + r0 + v] = lsum[v];
    }
}

// per key, the chunk rows are added in FIN_GROUPS interleaved groups (each in
// chunk order), and the groups are combined in order: a fixed summation order
constexpr int FIN_KEYS = 64;
constexpr int FIN_GROUPS = 16;

__global__ __launch_bounds__(FIN_KEYS * FIN_GROUPS) void k_fin_sum(const GroupParams p)
{
    if (blockIdx.x == 0) {
        __shared__ double red[3 * FIN_KEYS * FIN_GROUPS / 64];
        write_totals(p, red, FIN_KEYS * FIN_GROUPS);
    }
    if (p.kstat != p.status && blockIdx.x == 0 && threadIdx.x == 0) {
        // a key plan built beforehand: its counts become the call's
        p.status->n_unique = p.kstat->n_unique;
        if (p.kstat->overflow) p.status->overflow = 1u;
    }
    __shared__ uint64_t qc[FIN_GROUPS][FIN_KEYS];
    __shared__ double qs[FIN_GROUPS][FIN_KEYS];
    const int kl = threadIdx.x % FIN_KEYS, grp = threadIdx.x / FIN_KEYS;
    const int64_t id = (int64_t)blockIdx.x * FIN_KEYS + kl;
    // every load is requested before the key count is read (rows up to the
    // capacity exist; those past the count are ignored)
    uint64_t cnt = 0;
    double sum = 0.0;
    if (id < p.cap) {
#pragma unroll 16
        for (int c = grp; c < p.nchunks; c += FIN_GROUPS) {
            cnt += p.pcnt[(int64_t)c * p.cap + id];
            sum += p.psum[(int64_t)c * p.cap + id];
        }
    }
    uint32_t r = 0xffffffffu;
    uint64_t key = 0;
    if (grp == 0 && id < p.cap) {
        r = p.urank[id];
        key = p.ukey[id];
    }
    const int64_t nk = min((int64_t)p.kstat->n_unique, p.cap);
    if (p.n_keys_out && blockIdx.x == 0 && threadIdx.x == 0) *p.n_keys_out = nk;
    if ((int64_t)blockIdx.x * FIN_KEYS >= nk) return;  // uniform
    qc[grp][kl] = cnt;
    qs[grp][kl] = sum;
    __syncthreads();
    if (grp == 0 && id < nk) {
        cnt = 0;
        sum = 0.0;
        for (int g = 0; g < FIN_GROUPS; ++g) {
            cnt += qc[g][kl];
            sum += qs[g][kl];
        }
        if ((int64_t)r < p.cap) {
            p.keys_out[r] = key;
            p.count_out[r] = (int64_t)cnt;
            p.sum_out[r] = sum;
        }
        p.mean[id] = cnt ? sum / (double)cnt : 0.0;
    }
}

__global__ __launch_bounds__(AGG_THREADS) void k_agg_m2(const GroupParams p)
{
    __shared__ double lm2[AGG_IDS];
    __shared__ double lmean[AGG_IDS];
    const int c = blockIdx.x;
    const int64_t r0 = (int64_t)blockIdx.y * AGG_IDS;
    const int64_t nk = min((int64_t)p.kstat->n_unique, p.cap);
    if (r0 >= nk) return;
    const int nid = (int)min((int64_t)AGG_IDS, nk - r0);
    for (int v = threadIdx.x; v < nid; v += AGG_THREADS) {
        lm2[v] = 0.0;
        lmean[v] = p.mean[r0 + v];
    }
    __syncthreads();
    const int64_t lo = (int64_t)c * p.chunk, hi = min(lo + p.chunk, p.m);
    for (int64_t i0 = lo + threadIdx.x; i0 < hi; i0 += (int64_t)AGG_BATCH * AGG_THREADS) {
        uint32_t sl[AGG_BATCH];
        double en[AGG_BATCH];
#pragma unroll
        for (int k = 0; k < AGG_BATCH; ++k) {
            const int64_t i = i0 + (int64_t)k * AGG_THREADS;
            sl[k] = (i < hi) ? p.slot[i] : NO_ID;
            en[k] = (i < hi) ? p.energy[i] : 0.0;
        }
#pragma unroll
        for (int k = 0; k < AGG_BATCH; ++k) {
            const uint32_t id = resolve_id(p, sl[k]);
            const int64_t d = (id == NO_ID) ? -1 : (int64_t)id - r0;
            if (d < 0 || d >= nid) continue;
            const double x = en[k] - lmean[d];
            atomicAdd(&lm2[d], x * x);
        }
    }
    __syncthreads();
    for (int v = threadIdx.x; v < nid; v += AGG_THREADS) p.pm2[(int64_t)c * p.cap + r0 + v] = lm2[v];
}

__global__ __launch_bounds__(FIN_KEYS * FIN_GROUPS) void k_fin_m2(const GroupParams p)
{
    __shared__ double qs[FIN_GROUPS][FIN_KEYS];
    __shared__ double qd[FIN_GROUPS][FIN_KEYS];
    const int kl = threadIdx.x % FIN_KEYS, grp = threadIdx.x / FIN_KEYS;
    const int64_t id = (int64_t)blockIdx.x * FIN_KEYS + kl;
    // loads requested before the key count is read, as in k_fin_sum
    double m2 = 0.0, du = 0.0;
    if (id < p.cap)
#pragma unroll 16
        for (int c = grp; c < p.nchunks; c += FIN_GROUPS) m2 += p.pm2[(int64_t)c * p.cap + id];
    if (p.dur_out && id < p.cap)
#pragma unroll 16
        for (int c = grp; c < p.nchunks; c += FIN_GROUPS) du += p.pdur[(int64_t)c * p.cap + id];
    const uint32_t r = (grp == 0 && id < p.cap) ? p.urank[id] : 0xffffffffu;
    const int64_t nk = min((int64_t)p.kstat->n_unique, p.cap);
    if ((int64_t)blockIdx.x * FIN_KEYS >= nk) return;  // uniform
    qs[grp][kl] = m2;
    qd[grp][kl] = du;
    __syncthreads();
    if (grp == 0 && id < nk) {
        m2 = 0.0;
        du = 0.0;
        for (int g = 0; g < FIN_GROUPS; ++g) {
            m2 += qs[g][kl];
            du += qd[g][kl];
        }
        if ((int64_t)r < p.cap) {
            p.m2_out[r] = m2;
            if (p.dur_out) p.dur_out[r] = du;
        }
    }
}

// count, sum and M2 about the chunk's own mean, per id of one chunk held in
// registers (the chunk is at most AGG_THREADS * AGG_BATCH intervals)
__global__ __launch_bounds__(AGG_THREADS) void k_agg_one(const GroupParams p)
{
    __shared__ uint32_t lcnt[AGG_IDS];
    __shared__ double lsum[AGG_IDS];
    const int c = blockIdx.x;
    const int64_t r0 = (int64_t)blockIdx.y * AGG_IDS;
    const int64_t lo = (int64_t)c * p.chunk, hi = min(lo + p.chunk, p.m);
    uint32_t sl[AGG_BATCH];
    double en[AGG_BATCH];
    // the loads are requested before the key count is read
#pragma unroll
    for (int k = 0; k < AGG_BATCH; ++k) {
        const int64_t i = lo + threadIdx.x + (int64_t)k * AGG_THREADS;
        sl[k] = (i < hi) ? p.slot[i] : NO_ID;
        en[k] = (i < hi) ? p.energy[i] : 0.0;
    }
    if (blockIdx.y == 0) {
        // the chunk's total energy (all its intervals, whatever their key)
        __shared__ double red[AGG_THREADS / 64];
        double v = 0.0;
#pragma unroll
        for (int k = 0; k < AGG_BATCH; ++k) v += en[k];
        v = block_sum(v, red, AGG_THREADS);
        if (threadIdx.x == 0) p.ctot[c] = v;
    }
    const int64_t nk = min((int64_t)p.kstat->n_unique, p.cap);
    if (r0 >= nk) return;  // uniform
    const int nid = (int)min((int64_t)AGG_IDS, nk - r0);
    for (int v = threadIdx.x; v < nid; v += AGG_THREADS) {
        lcnt[v] = 0u;
        lsum[v] = 0.0;
    }
    int d[AGG_BATCH];
#pragma unroll
    for (int k = 0; k < AGG_BATCH; ++k) {
        const uint32_t id = resolve_id(p, sl[k]);
        const int64_t x = (id == NO_ID) ? -1 : (int64_t)id - r0;
        d[k] = (x < 0 || x >= nid) ? -1 : (int)x;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < AGG_BATCH; ++k) {
        if (d[k] < 0) continue;
        atomicAdd(&lcnt[d[k]], 1u);
        atomicAdd(&lsum[d[k]], en[k]);
    }
    __syncthreads();
    // the chunk rows out; the table then holds each key's chunk mean, once
    for (int v = threadIdx.x; v < nid; v += AGG_THREADS) {
        const uint32_t n = lcnt[v];
        const double sm = lsum[v];
        p.pcnt[(int64_t)c * p.cap + r0 + v] = n;
        p.psum[(int64_t)c * p.cap + r0 + v] = sm;
        lsum[v] = n ? sm / (double)n : 0.0;
    }
    __syncthreads();
    // each interval's deviation from its key's chunk mean
#pragma unroll
    for (int k = 0; k < AGG_BATCH; ++k)
        if (d[k] >= 0) en[k] -= lsum[d[k]];
    __syncthreads();
    for (int v = threadIdx.x; v < nid; v += AGG_THREADS) lsum[v] = 0.0;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < AGG_BATCH; ++k)
        if (d[k] >= 0) atomicAdd(&lsum[d[k]], en[k] * en[k]);
    __syncthreads();
    for (int v = threadIdx.x; v < nid; v += AGG_THREADS) p.pm2[(int64_t)c * p.cap + r0 + v] = lsum[v];
    if (!p.dur_out) return;  // uniform
    // per-key latency: the same table once more, over the interval durations
#pragma unroll
    for (int k = 0; k < AGG_BATCH; ++k)
        en[k] = (d[k] >= 0) ? interval_duration(p, lo + threadIdx.x + (int64_t)k * AGG_THREADS) : 0.0;
    __syncthreads();
    for (int v = threadIdx.x; v < nid; v += AGG_THREADS) lsum[v] = 0.0;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < AGG_BATCH; ++k)
        if (d[k] >= 0) atomicAdd(&lsum[d[k]], en[k]);
    __syncthreads();
    for (int v = threadIdx.x; v < nid; v += AGG_THREADS) p.pdur[(int64_t)c * p.cap + r0 + v] = lsum[v];
}

// per-key latency when a chunk spans several batches: one more pass
__global__ __launch_bounds__(AGG_THREADS) void k_agg_dur(const GroupParams p)
{
    __shared__ double ldur[AGG_IDS];
    const int c = blockIdx.x;
    const int64_t r0 = (int64_t)blockIdx.y * AGG_IDS;
    const int64_t nk = min((int64_t)p.kstat->n_unique, p.cap);
    if (r0 >= nk) return;
    const int nid = (int)min((int64_t)AGG_IDS, nk - r0);
    for (int v = threadIdx.x; v < nid; v += AGG_THREADS) ldur[v] = 0.0;
    __syncthreads();
    const int64_t lo = (int64_t)c * p.chunk, hi = min(lo + p.chunk, p.m);
    for (int64_t i0 = lo + threadIdx.x; i0 < hi; i0 += (int64_t)AGG_BATCH * AGG_THREADS) {
        uint32_t sl[AGG_BATCH];
        double du[AGG_BATCH];
#pragma unroll
        for (int k = 0; k < AGG_BATCH; ++k) {
            const int64_t i = i0 + (int64_t)k * AGG_THREADS;
            sl[k] = (i < hi) ? p.slot[i] : NO_ID;
            du[k] = (i < hi) ? interval_duration(p, i) : 0.0;
        }
#pragma unroll
        for (int k = 0; k < AGG_BATCH; ++k) {
            const uint32_t id = resolve_id(p, sl[k]);
            const int64_t d = (id == NO_ID) ? -1 : (int64_t)id - r0;
            if (d < 0 || d >= nid) continue;
            atomicAdd(&ldur[d], du[k]);
        }
    }
    __syncthreads();
    for (int v = threadIdx.x; v < nid; v += AGG_THREADS) p.pdur[(int64_t)c * p.cap + r0 + v] = ldur[v];
}

// per key: count and sum over the chunk rows (as k_fin_sum), then
// M2 = sum_c (M2_c + n_c (mean_c - mean)^2) over the same rows; 32 keys per
// workgroup, each key's rows split over 32 interleaved groups
constexpr int FO_KEYS = 32;
constexpr int FO_GROUPS = 32;
__global__ __launch_bounds__(FO_KEYS * FO_GROUPS) void k_fin_one(const GroupParams p)
{
    if (blockIdx.x == 0) {
        __shared__ double red[3 * FO_KEYS * FO_GROUPS / 64];
        write_totals(p, red, FO_KEYS * FO_GROUPS);
    }
    if (p.kstat != p.status && blockIdx.x == 0 && threadIdx.x == 0) {
        // a key plan built beforehand: its counts become the call's
        p.status->n_unique = p.kstat->n_unique;
        if (p.kstat->overflow) p.status->overflow = 1u;
    }
    __shared__ uint64_t qc[FO_GROUPS][FO_KEYS];
    __shared__ double qs[FO_GROUPS][FO_KEYS];
    __shared__ double qmean[FO_KEYS];
    __shared__ double qdu[FO_GROUPS][FO_KEYS];
    const int kl = threadIdx.x % FO_KEYS, grp = threadIdx.x / FO_KEYS;
    const int64_t id = (int64_t)blockIdx.x * FO_KEYS + kl;
    uint64_t cnt = 0;
    double sum = 0.0, du = 0.0;
    if (id < p.cap) {
#pragma unroll 8
        for (int c = grp; c < p.nchunks; c += FO_GROUPS) {
            cnt += p.pcnt[(int64_t)c * p.cap + id];
            sum += p.psum[(int64_t)c * p.cap + id];
        }
    }
    if (p.dur_out && id < p.cap) {
#pragma unroll 8
        for (int c = grp; c < p.nchunks; c += FO_GROUPS) du += p.pdur[(int64_t)c * p.cap + id];
    }
    uint32_t r = 0xffffffffu;
    uint64_t key = 0;
    if (grp == 0 && id < p.cap) {
        r = p.urank[id];
        key = p.ukey[id];
    }
    const int64_t nk = min((int64_t)p.kstat->n_unique, p.cap);
    if (p.n_keys_out && blockIdx.x == 0 && threadIdx.x == 0) *p.n_keys_out = nk;
    if ((int64_t)blockIdx.x * FO_KEYS >= nk) return;  // uniform
    qc[grp][kl] = cnt;
    qs[grp][kl] = sum;
    qdu[grp][kl] = du;
    __syncthreads();
    if (grp == 0) {
        cnt = 0;
        sum = 0.0;
        du = 0.0;
        for (int g = 0; g < FO_GROUPS; ++g) {
            cnt += qc[g][kl];
            sum += qs[g][kl];
            du += qdu[g][kl];
        }
        qmean[kl] = cnt ? sum / (double)cnt : 0.0;
        if (id < nk) {
            if ((int64_t)r < p.cap) {
                p.keys_out[r] = key;
                p.count_out[r] = (int64_t)cnt;
                p.sum_out[r] = sum;
                if (p.dur_out) p.dur_out[r] = du;
            }
        }
    }
    __syncthreads();
    double m2 = 0.0;
    if (id < nk) {
        // branch-free, so that the loads of many chunk rows are in flight together
        const double mean = qmean[kl];
#pragma unroll 8
        for (int c = grp; c < p.nchunks; c += FO_GROUPS) {
            const uint32_t nc = p.pcnt[(int64_t)c * p.cap + id];
            const double sc = p.psum[(int64_t)c * p.cap + id];
            const double mc = p.pm2[(int64_t)c * p.cap + id];
            const double dn = (double)nc;
            const double dm = (nc ? sc / dn : mean) - mean;
            m2 += mc + dn * dm * dm;
        }
    }
    __syncthreads();
    qs[grp][kl] = m2;
    __syncthreads();
    if (grp == 0 && id < nk) {
        m2 = 0.0;
        for (int g = 0; g < FO_GROUPS; ++g) m2 += qs[g][kl];
        if ((int64_t)r < p.cap) p.m2_out[r] = m2;
    }
}

__global__ void k_set_i64(int64_t* dst, int64_t v) { *dst = v; }

hipError_t launch_set_i64(int64_t* dst, int64_t v, hipStream_t stream)
{
    hipLaunchKernelGGL(k_set_i64, dim3(1), dim3(1), 0, stream, dst, v);
    return hipGetLastError();
}

// clears the table, the rank counters and the key state (a key plan built
// on its own; inside an attribution k_fix does this)
__global__ __launch_bounds__(256) void k_plan_clear(const GroupParams p)
{
    for (int64_t h = (int64_t)blockIdx.x * 256 + threadIdx.x; h <= (int64_t)p.H;
         h += (int64_t)gridDim.x * 256) {
        reinterpret_cast<ulonglong2*>(p.table)[h] = make_ulonglong2(~0ull, ~0ull);  // empty, no id
        p.urank[h] = 0u;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        p.kstat->n_unique = 0u;
        p.kstat->special = 0u;
        p.kstat->overflow = 0u;
        p.kstat->err = 0u;
    }
}

hipError_t launch_key_map(const GroupParams& p, bool clear, hipStream_t stream)
{
    if (clear) {
        const unsigned cb = (unsigned)min(((int64_t)p.H + 256) / 256, (int64_t)2048);
        hipLaunchKernelGGL(k_plan_clear, dim3(cb), dim3(256), 0, stream, p);
    }
    if (p.m <= 0) return hipGetLastError();
    const int64_t n_ins = min(p.m, (int64_t)INS_CHUNK * INS_GROUPS);
    hipLaunchKernelGGL(k_key_insert, dim3((unsigned)((n_ins + INS_CHUNK - 1) / INS_CHUNK)),
                       dim3(INS_THREADS), 0, stream, p, n_ins);
    const unsigned hb =
        (unsigned)(((int64_t)p.H + 1 + CMP_THREADS * CMP_PER - 1) / (CMP_THREADS * CMP_PER));
    hipLaunchKernelGGL(k_compact, dim3(hb), dim3(CMP_THREADS), 0, stream, p);
    const int64_t mb =
        min((p.m + KM_THREADS * KM_BATCH - 1) / (KM_THREADS * KM_BATCH), (int64_t)8192);
    hipLaunchKernelGGL(k_keymap, dim3((unsigned)max(mb, (int64_t)1)), dim3(KM_THREADS), 0, stream,
                       p);
    // ids for the keys the lookup pass inserted
    hipLaunchKernelGGL(k_compact, dim3(hb), dim3(CMP_THREADS), 0, stream, p);
    // the distinct keys that can get a row are at most min(H + 1, cap + 1)
    // (more only on overflow, which is reported and ranked partially)
    const int64_t nmax = min((int64_t)p.H + 1, p.cap + 1);
    const int64_t ntile = (nmax + RANK_TILE - 1) / RANK_TILE;
    hipLaunchKernelGGL(k_rank, dim3((unsigned)min(ntile * ntile, (int64_t)4096)), dim3(RANK_TILE),
                       0, stream, p);
    return hipGetLastError();
}

hipError_t launch_aggregate(const GroupParams& p, hipStream_t stream)
{
    if (p.m <= 0) return p.n_keys_out ? launch_set_i64(p.n_keys_out, 0, stream) : hipSuccess;
    const unsigned ranges = (unsigned)((p.cap + AGG_IDS - 1) / AGG_IDS);
    const unsigned kb = (unsigned)max((int64_t)1, (p.cap + FIN_KEYS - 1) / FIN_KEYS);
    if (ranges > 0 && p.chunk <= (int64_t)AGG_THREADS * AGG_BATCH) {
        hipLaunchKernelGGL(k_agg_one, dim3((unsigned)p.nchunks, ranges), dim3(AGG_THREADS), 0,
                           stream, p);
        const unsigned kb1 = (unsigned)max((int64_t)1, (p.cap + FO_KEYS - 1) / FO_KEYS);
        hipLaunchKernelGGL(k_fin_one, dim3(kb1), dim3(FO_KEYS * FO_GROUPS), 0, stream, p);
    } else if (ranges > 0) {
        const unsigned ranges_sum = (unsigned)((p.cap + SUM_IDS - 1) / SUM_IDS);
        hipLaunchKernelGGL(k_agg_sum, dim3((unsigned)p.nchunks, ranges_sum), dim3(AGG_THREADS), 0,
                           stream, p);
        hipLaunchKernelGGL(k_fin_sum, dim3(kb), dim3(FIN_KEYS * FIN_GROUPS), 0, stream, p);
        hipLaunchKernelGGL(k_agg_m2, dim3((unsigned)p.nchunks, ranges), dim3(AGG_THREADS), 0,
                           stream, p);
        if (p.dur_out)
            hipLaunchKernelGGL(k_agg_dur, dim3((unsigned)p.nchunks, ranges), dim3(AGG_THREADS),
                               0, stream, p);
        hipLaunchKernelGGL(k_fin_m2, dim3(kb), dim3(FIN_KEYS * FIN_GROUPS), 0, stream, p);
    }
    return hipGetLastError();
}

hipError_t launch_groupby(const GroupParams& p, hipStream_t stream)
{
    if (p.m <= 0) return p.n_keys_out ? launch_set_i64(p.n_keys_out, 0, stream) : hipSuccess;
    const hipError_t e = launch_key_map(p, false, stream);
    if (e != hipSuccess) return e;
    return launch_aggregate(p, stream);
}

}  // namespace mag
