// groupby.hip -- per-operator-key count, sum and M2 of the interval energies.
//
// The key table and the rank counters are cleared by k_fix, the launch before.
//
// 1. k_key_insert + k_keymap: the 64-bit keys go into an open-addressing hash
//    table (linear probing, 64-bit compare-and-swap; the all-ones key is kept
//    out of band so any uint64 is a legal key).  Insertion (of the keys of a
//    prefix of the intervals) de-duplicates in LDS first; the lookup pass then
//    finds almost every key with a plain, cached load (a separate launch, so
//    no cached line predates an insert) and inserts the rest.
// 2. k_compact: the distinct keys are listed; a key's place in the list is its
//    dense id.  k_rank: rank of each key = number of smaller keys (its row in
//    the output, ascending by key).
// 3. k_agg_sum / k_fin_sum: each workgroup aggregates one chunk of intervals
//    into an LDS table indexed by dense id (count, sum); the partial tables are
//    reduced per key in chunk order, and the key, count and sum written to the
//    key's row.  Per-workgroup atomics add the rows into the attributed energy.
// 4. k_agg_m2 / k_fin_m2: second pass over the chunk for sum (E - mean)^2
//    (the two-pass definition of M2).
// Plain stores carry every partial result: device-scope atomics, which are
// slow on this part, are used only for counters and one add per workgroup.

#include "mag_internal.hpp"

namespace mag {

namespace {

constexpr unsigned long long EMPTY_KEY = ~0ull;

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

}  // namespace

// Insert the distinct keys of a prefix of the intervals.  Each workgroup first
// de-duplicates its chunk in an LDS table; then every thread takes a few LDS
// slots and inserts their keys into the global table, so a key costs one global
// probe per workgroup and the probe chains of a workgroup run in parallel.
constexpr int INS_THREADS = 512;
constexpr int INS_CHUNK = 4096;
constexpr int INS_SLOTS = 8192;
constexpr int INS_GROUPS = 64;  // the lookup pass inserts keys first seen later

__device__ __forceinline__ void global_insert(const GroupParams& p, unsigned long long k)
{
    const uint32_t mask = p.H - 1u;
    uint32_t h = (uint32_t)fmix64(k) & mask;
    for (uint32_t probe = 0; probe < p.H; ++probe) {
        // a device-coherent load first (the level-2 caches of the XCDs are not
        // coherent with each other, so a plain load could keep returning a stale
        // empty slot and force a swap per probe); a slot only ever changes from
        // empty to its final key, so a non-empty value read here is final
        const unsigned long long cur =
            __hip_atomic_load(&p.table[h], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (cur == k) return;
        if (cur == EMPTY_KEY) {
            const unsigned long long old = atomicCAS(&p.table[h], EMPTY_KEY, k);
            if (old == EMPTY_KEY || old == k) return;
        }
        h = (h + 1u) & mask;
    }
    atomicOr(&p.status->overflow, 1u);
}

__global__ __launch_bounds__(INS_THREADS) void k_key_insert(const GroupParams p, int64_t n_insert)
{
    __shared__ unsigned long long lt[INS_SLOTS];
    for (int v = threadIdx.x; v < INS_SLOTS; v += blockDim.x) lt[v] = EMPTY_KEY;
    __syncthreads();
    const int64_t lo = (int64_t)blockIdx.x * INS_CHUNK, hi = min(lo + INS_CHUNK, n_insert);
    for (int64_t i = lo + threadIdx.x; i < hi; i += blockDim.x) {
        const unsigned long long k = p.keys[i];
        if (k == EMPTY_KEY) {
            atomicOr(&p.status->special, 1u);
            continue;
        }
        uint32_t h = (uint32_t)fmix64(k) & (INS_SLOTS - 1);
        for (int probe = 0; probe < INS_SLOTS; ++probe) {
            const unsigned long long old = atomicCAS(&lt[h], EMPTY_KEY, k);
            if (old == EMPTY_KEY || old == k) break;
            h = (h + 1u) & (INS_SLOTS - 1);
        }
    }
    __syncthreads();
    for (int v = threadIdx.x; v < INS_SLOTS; v += blockDim.x) {
        const unsigned long long k = lt[v];
        if (k != EMPTY_KEY) global_insert(p, k);
    }
}

// slot of every interval's key (the table holds most keys already, so this is
// normally a plain cached probe)
__global__ __launch_bounds__(256) void k_keymap(const GroupParams p)
{
    const uint32_t H = p.H;
    const uint32_t mask = H - 1u;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < p.m;
         i += (int64_t)gridDim.x * blockDim.x) {
        const unsigned long long k = p.keys[i];
        uint32_t slot = H + 1u;  // invalid
        if (k == EMPTY_KEY) {
            slot = H;
            if (p.status->special == 0u) atomicOr(&p.status->special, 1u);
        } else {
            uint32_t h = (uint32_t)fmix64(k) & mask;
            for (uint32_t probe = 0; probe < H; ++probe) {
                // plain (cached) load: a slot only ever changes from empty to its
                // final key, and the compare-and-swap below settles a stale read
                unsigned long long cur = p.table[h];
                if (cur == k) {
                    slot = h;
                    break;
                }
                if (cur == EMPTY_KEY) {
                    const unsigned long long old = atomicCAS(&p.table[h], EMPTY_KEY, k);
                    if (old == EMPTY_KEY || old == k) {
                        slot = h;
                        break;
                    }
                }
                h = (h + 1u) & mask;
            }
            if (slot > H) atomicOr(&p.status->overflow, 1u);
        }
        p.slot[i] = slot;
    }
}

// list the occupied slots (order irrelevant: ranks come from key comparisons)
__global__ __launch_bounds__(256) void k_compact(const GroupParams p)
{
    const int lane = threadIdx.x & 63;
    // whole waves iterate together (the ballot below needs every lane)
    const uint32_t span = ((p.H + 1u + 63u) / 64u) * 64u;
    for (uint32_t h = blockIdx.x * blockDim.x + threadIdx.x; h < span; h += gridDim.x * blockDim.x) {
        unsigned long long k = EMPTY_KEY;
        bool occ = false;
        if (h < p.H) {
            k = p.table[h];
            occ = (k != EMPTY_KEY);
        } else if (h == p.H) {
            occ = p.status->special != 0u;
        }
        // one counter update per wave: occupied slots take consecutive rows
        const uint64_t ob = __ballot(occ);
        uint32_t base = 0u;
        if (lane == 0 && ob) base = atomicAdd(&p.status->n_unique, (uint32_t)__popcll(ob));
        base = __shfl(base, 0);
        if (occ) {
            const uint32_t u = base + (uint32_t)__popcll(ob & ((1ull << lane) - 1ull));
            p.ukey[u] = k;
            p.uslot[u] = h;
            p.slot2id[h] = u;
        }
    }
}

// rank = number of distinct keys smaller than this one: the pairs (x, y) of key
// tiles are spread over the workgroups; pair (x, y) compares keys
// [256 x, 256 x + 256) against keys [256 y, 256 y + 256)
constexpr uint32_t RANK_TILE = 256u;

__global__ __launch_bounds__(RANK_TILE) void k_rank(const GroupParams p)
{
    __shared__ uint64_t tile[RANK_TILE];
    const uint32_t nu = p.status->n_unique;
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

// chunk of intervals -> LDS table over ids [r0, r0 + AGG_IDS) -> partial table row
__global__ __launch_bounds__(AGG_THREADS) void k_agg_sum(const GroupParams p)
{
    __shared__ uint32_t lcnt[AGG_IDS];
    __shared__ double lsum[AGG_IDS];
    const int c = blockIdx.x;
    const int64_t r0 = (int64_t)blockIdx.y * AGG_IDS;
    const int64_t nk = min((int64_t)p.status->n_unique, p.cap);
    if (r0 >= nk) return;  // uniform
    const int nid = (int)min((int64_t)AGG_IDS, nk - r0);
    for (int v = threadIdx.x; v < nid; v += AGG_THREADS) {
        lcnt[v] = 0u;
        lsum[v] = 0.0;
    }
    __syncthreads();
    const int64_t lo = (int64_t)c * p.chunk, hi = min(lo + p.chunk, p.m);
    constexpr int U = 4;  // independent loads in flight per thread
    for (int64_t i0 = lo + threadIdx.x; i0 < hi; i0 += (int64_t)U * AGG_THREADS) {
        uint32_t sl[U];
        double en[U];
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const int64_t i = i0 + (int64_t)k * AGG_THREADS;
            sl[k] = (i < hi) ? p.slot[i] : 0xffffffffu;
            en[k] = (i < hi) ? p.energy[i] : 0.0;
        }
        int64_t id[U];
#pragma unroll
        for (int k = 0; k < U; ++k) id[k] = (sl[k] <= p.H) ? (int64_t)p.slot2id[sl[k]] - r0 : -1;
#pragma unroll
        for (int k = 0; k < U; ++k) {
            if (id[k] < 0 || id[k] >= nid) continue;
            atomicAdd(&lcnt[id[k]], 1u);
            atomicAdd(&lsum[id[k]], en[k]);
        }
    }
    __syncthreads();
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
    __shared__ uint64_t qc[FIN_GROUPS][FIN_KEYS];
    __shared__ double qs[FIN_GROUPS][FIN_KEYS];
    const int64_t nk = min((int64_t)p.status->n_unique, p.cap);
    const int kl = threadIdx.x % FIN_KEYS, grp = threadIdx.x / FIN_KEYS;
    const int64_t id = (int64_t)blockIdx.x * FIN_KEYS + kl;
    if ((int64_t)blockIdx.x * FIN_KEYS >= nk) return;  // uniform
    uint64_t cnt = 0;
    double sum = 0.0;
    if (id < nk) {
        for (int c = grp; c < p.nchunks; c += FIN_GROUPS) {
            cnt += p.pcnt[(int64_t)c * p.cap + id];
            sum += p.psum[(int64_t)c * p.cap + id];
        }
    }
    qc[grp][kl] = cnt;
    qs[grp][kl] = sum;
    __syncthreads();
    double tot = 0.0;
    if (grp == 0 && id < nk) {
        cnt = 0;
        sum = 0.0;
        for (int g = 0; g < FIN_GROUPS; ++g) {
            cnt += qc[g][kl];
            sum += qs[g][kl];
        }
        const uint32_t r = p.urank[id];
        if ((int64_t)r < p.cap) {
            p.keys_out[r] = p.ukey[id];
            p.count_out[r] = (int64_t)cnt;
            p.sum_out[r] = sum;
        }
        p.mean[id] = cnt ? sum / (double)cnt : 0.0;
        tot = sum;
    }
    if (grp == 0) {
        // this workgroup's rows, once into the attributed energy
        for (int off = 32; off > 0; off >>= 1) tot += __shfl_xor(tot, off);
        if (kl == 0 && tot != 0.0) atomicAdd(&p.status->attributed_energy, tot);
    }
}

__global__ __launch_bounds__(AGG_THREADS) void k_agg_m2(const GroupParams p)
{
    __shared__ double lm2[AGG_IDS];
    __shared__ double lmean[AGG_IDS];
    const int c = blockIdx.x;
    const int64_t r0 = (int64_t)blockIdx.y * AGG_IDS;
    const int64_t nk = min((int64_t)p.status->n_unique, p.cap);
    if (r0 >= nk) return;
    const int nid = (int)min((int64_t)AGG_IDS, nk - r0);
    for (int v = threadIdx.x; v < nid; v += AGG_THREADS) {
        lm2[v] = 0.0;
        lmean[v] = p.mean[r0 + v];
    }
    __syncthreads();
    const int64_t lo = (int64_t)c * p.chunk, hi = min(lo + p.chunk, p.m);
    constexpr int U = 4;
    for (int64_t i0 = lo + threadIdx.x; i0 < hi; i0 += (int64_t)U * AGG_THREADS) {
        uint32_t sl[U];
        double en[U];
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const int64_t i = i0 + (int64_t)k * AGG_THREADS;
            sl[k] = (i < hi) ? p.slot[i] : 0xffffffffu;
            en[k] = (i < hi) ? p.energy[i] : 0.0;
        }
        int64_t id[U];
#pragma unroll
        for (int k = 0; k < U; ++k) id[k] = (sl[k] <= p.H) ? (int64_t)p.slot2id[sl[k]] - r0 : -1;
#pragma unroll
        for (int k = 0; k < U; ++k) {
            if (id[k] < 0 || id[k] >= nid) continue;
            const double d = en[k] - lmean[id[k]];
            atomicAdd(&lm2[id[k]], d * d);
        }
    }
    __syncthreads();
    for (int v = threadIdx.x; v < nid; v += AGG_THREADS) p.pm2[(int64_t)c * p.cap + r0 + v] = lm2[v];
}

__global__ __launch_bounds__(FIN_KEYS * FIN_GROUPS) void k_fin_m2(const GroupParams p)
{
    __shared__ double qs[FIN_GROUPS][FIN_KEYS];
    const int64_t nk = min((int64_t)p.status->n_unique, p.cap);
    const int kl = threadIdx.x % FIN_KEYS, grp = threadIdx.x / FIN_KEYS;
    const int64_t id = (int64_t)blockIdx.x * FIN_KEYS + kl;
    if ((int64_t)blockIdx.x * FIN_KEYS >= nk) return;  // uniform
    double m2 = 0.0;
    if (id < nk)
        for (int c = grp; c < p.nchunks; c += FIN_GROUPS) m2 += p.pm2[(int64_t)c * p.cap + id];
    qs[grp][kl] = m2;
    __syncthreads();
    if (grp == 0 && id < nk) {
        m2 = 0.0;
        for (int g = 0; g < FIN_GROUPS; ++g) m2 += qs[g][kl];
        const uint32_t r = p.urank[id];
        if ((int64_t)r < p.cap) p.m2_out[r] = m2;
    }
}

hipError_t launch_groupby(const GroupParams& p, hipStream_t stream)
{
    if (p.m <= 0) return hipSuccess;
    const int64_t n_ins = min(p.m, (int64_t)INS_CHUNK * INS_GROUPS);
    hipLaunchKernelGGL(k_key_insert, dim3((unsigned)((n_ins + INS_CHUNK - 1) / INS_CHUNK)),
                       dim3(INS_THREADS), 0, stream, p, n_ins);
    const int64_t mb = min((p.m + 255) / 256, (int64_t)16384);
    hipLaunchKernelGGL(k_keymap, dim3((unsigned)max(mb, (int64_t)1)), dim3(256), 0, stream, p);
    const unsigned hb = (unsigned)min((int64_t)(p.H + 1 + 255) / 256, (int64_t)4096);
    hipLaunchKernelGGL(k_compact, dim3(hb), dim3(256), 0, stream, p);
    // the distinct keys that can get a row are at most min(H + 1, cap + 1)
    // (more only on overflow, which is reported and ranked partially)
    const int64_t nmax = min((int64_t)p.H + 1, p.cap + 1);
    const int64_t ntile = (nmax + RANK_TILE - 1) / RANK_TILE;
    hipLaunchKernelGGL(k_rank, dim3((unsigned)min(ntile * ntile, (int64_t)4096)), dim3(RANK_TILE),
                       0, stream, p);
    const unsigned ranges = (unsigned)((p.cap + AGG_IDS - 1) / AGG_IDS);
    if (ranges > 0) {
        hipLaunchKernelGGL(k_agg_sum, dim3((unsigned)p.nchunks, ranges), dim3(AGG_THREADS), 0,
                           stream, p);
        const unsigned kb = (unsigned)max((int64_t)1, (p.cap + FIN_KEYS - 1) / FIN_KEYS);
        hipLaunchKernelGGL(k_fin_sum, dim3(kb), dim3(FIN_KEYS * FIN_GROUPS), 0, stream, p);
        hipLaunchKernelGGL(k_agg_m2, dim3((unsigned)p.nchunks, ranges), dim3(AGG_THREADS), 0,
                           stream, p);
        hipLaunchKernelGGL(k_fin_m2, dim3(kb), dim3(FIN_KEYS * FIN_GROUPS), 0, stream, p);
    }
    return hipGetLastError();
}

}  // namespace mag
