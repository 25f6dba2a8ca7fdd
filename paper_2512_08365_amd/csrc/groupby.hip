// groupby.hip -- per-operator-key count, sum and M2 of the interval energies.
//
// 1. k_keymap: every interval's 64-bit key is inserted into an open-addressing
//    hash table (linear probing, 64-bit compare-and-swap; the all-ones key is
//    kept out of band so any uint64 is a legal key).  Repeated keys are found
//    with a plain load, so hot keys cost no atomics.
// 2. k_compact + k_rank: the distinct keys are listed and ranked (rank = number
//    of smaller keys), which gives dense ids in ascending key order.
// 3. k_agg_sum / k_fin_sum: each workgroup aggregates one chunk of intervals
//    into an LDS table indexed by dense id (count, sum); the partial tables are
//    reduced per key in chunk order.
// 4. k_agg_m2 / k_fin_m2: second pass over the chunk for sum (E - mean)^2
//    (the two-pass definition of M2).

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

__global__ __launch_bounds__(256) void k_table_fill(unsigned long long* table, uint32_t H)
{
    for (uint32_t h = blockIdx.x * blockDim.x + threadIdx.x; h < H; h += gridDim.x * blockDim.x)
        table[h] = EMPTY_KEY;
}

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
            if (__hip_atomic_load(&p.status->special, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0u)
                atomicOr(&p.status->special, 1u);
        } else {
            uint32_t h = (uint32_t)fmix64(k) & mask;
            for (uint32_t probe = 0; probe < H; ++probe) {
                unsigned long long cur =
                    __hip_atomic_load(&p.table[h], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (cur == k) {
                    slot = h;
                    break;
                }
                if (cur == EMPTY_KEY) {
                    const unsigned long long old = atomicCAS(&p.table[h], EMPTY_KEY, k);
                    if (old == EMPTY_KEY) {
                        atomicAdd(&p.status->n_inserted, 1u);
                        slot = h;
                        break;
                    }
                    if (old == k) {
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
    for (uint32_t h = blockIdx.x * blockDim.x + threadIdx.x; h <= p.H; h += gridDim.x * blockDim.x) {
        unsigned long long k;
        bool occ;
        if (h < p.H) {
            k = p.table[h];
            occ = (k != EMPTY_KEY);
        } else {
            k = EMPTY_KEY;
            occ = p.status->special != 0u;
        }
        if (occ) {
            const uint32_t u = atomicAdd(&p.status->n_unique, 1u);
            p.ukey[u] = k;
            p.uslot[u] = h;
        }
    }
}

// dense id = number of distinct keys smaller than this one
__global__ __launch_bounds__(256) void k_rank(const GroupParams p)
{
    __shared__ uint64_t tile[1024];
    const uint32_t nu = p.status->n_unique;
    const uint32_t u = blockIdx.x * blockDim.x + threadIdx.x;
    if (blockIdx.x * blockDim.x >= nu) return;  // uniform over the block
    const uint64_t mine = (u < nu) ? p.ukey[u] : 0ull;
    uint32_t rank = 0;
    for (uint32_t base = 0; base < nu; base += 1024) {
        const uint32_t cnt = min(1024u, nu - base);
        __syncthreads();
        for (uint32_t v = threadIdx.x; v < cnt; v += blockDim.x) tile[v] = p.ukey[base + v];
        __syncthreads();
        for (uint32_t v = 0; v < cnt; ++v) rank += (tile[v] < mine) ? 1u : 0u;
    }
    if (u < nu) {
        p.slot2id[p.uslot[u]] = rank;
        if ((int64_t)rank < p.cap) p.keys_out[rank] = mine;
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
    for (int64_t i = lo + threadIdx.x; i < hi; i += AGG_THREADS) {
        const uint32_t sl = p.slot[i];
        if (sl > p.H) continue;
        const int64_t id = (int64_t)p.slot2id[sl] - r0;
        if (id < 0 || id >= nid) continue;
        atomicAdd(&lcnt[id], 1u);
        atomicAdd(&lsum[id], p.energy[i]);
    }
    __syncthreads();
    for (int v = threadIdx.x; v < nid; v += AGG_THREADS) {
        p.pcnt[(int64_t)c * p.cap + r0 + v] = lcnt[v];
        p.psum[(int64_t)c * p.cap + r0 + v] = lsum[v];
    }
}

__global__ __launch_bounds__(256) void k_fin_sum(const GroupParams p)
{
    const int64_t nk = min((int64_t)p.status->n_unique, p.cap);
    for (int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; id < nk;
         id += (int64_t)gridDim.x * blockDim.x) {
        uint64_t cnt = 0;
        double sum = 0.0;
        for (int c = 0; c < p.nchunks; ++c) {
            cnt += p.pcnt[(int64_t)c * p.cap + id];
            sum += p.psum[(int64_t)c * p.cap + id];
        }
        p.count_out[id] = (int64_t)cnt;
        p.sum_out[id] = sum;
        p.mean[id] = cnt ? sum / (double)cnt : 0.0;
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
    for (int64_t i = lo + threadIdx.x; i < hi; i += AGG_THREADS) {
        const uint32_t sl = p.slot[i];
        if (sl > p.H) continue;
        const int64_t id = (int64_t)p.slot2id[sl] - r0;
        if (id < 0 || id >= nid) continue;
        const double d = p.energy[i] - lmean[id];
        atomicAdd(&lm2[id], d * d);
    }
    __syncthreads();
    for (int v = threadIdx.x; v < nid; v += AGG_THREADS) p.pm2[(int64_t)c * p.cap + r0 + v] = lm2[v];
}

__global__ __launch_bounds__(256) void k_fin_m2(const GroupParams p)
{
    const int64_t nk = min((int64_t)p.status->n_unique, p.cap);
    for (int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; id < nk;
         id += (int64_t)gridDim.x * blockDim.x) {
        double m2 = 0.0;
        for (int c = 0; c < p.nchunks; ++c) m2 += p.pm2[(int64_t)c * p.cap + id];
        p.m2_out[id] = m2;
    }
}

// sum of the per-key sums (attributed energy), in key order
__global__ __launch_bounds__(1024) void k_key_total(const GroupParams p)
{
    __shared__ double red[16];
    const int tid = threadIdx.x;
    const int64_t nk = min((int64_t)p.status->n_unique, p.cap);
    const int64_t per = (nk + 1023) / 1024;
    const int64_t lo = (int64_t)tid * per, hi = min(lo + per, nk);
    double v = 0.0;
    for (int64_t i = lo; i < hi; ++i) v += p.sum_out[i];
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    if ((tid & 63) == 0) red[tid >> 6] = v;
    __syncthreads();
    if (tid == 0) {
        double s = 0.0;
        for (int u = 0; u < 16; ++u) s += red[u];
        p.status->attributed_energy = s;
    }
}

hipError_t launch_groupby(const GroupParams& p, hipStream_t stream)
{
    const unsigned fill_blocks = (unsigned)min((p.H + 255u) / 256u, 4096u);
    hipLaunchKernelGGL(k_table_fill, dim3(fill_blocks), dim3(256), 0, stream, p.table, p.H);
    const int64_t mb = min((p.m + 255) / 256, (int64_t)16384);
    hipLaunchKernelGGL(k_keymap, dim3((unsigned)max(mb, (int64_t)1)), dim3(256), 0, stream, p);
    const unsigned hb = (unsigned)min((int64_t)(p.H + 1 + 255) / 256, (int64_t)4096);
    hipLaunchKernelGGL(k_compact, dim3(hb), dim3(256), 0, stream, p);
    const unsigned rb = (unsigned)(((int64_t)p.H + 1 + 255) / 256);
    hipLaunchKernelGGL(k_rank, dim3(rb), dim3(256), 0, stream, p);
    const unsigned ranges = (unsigned)((p.cap + AGG_IDS - 1) / AGG_IDS);
    if (ranges > 0) {
        hipLaunchKernelGGL(k_agg_sum, dim3((unsigned)p.nchunks, ranges), dim3(AGG_THREADS), 0,
                           stream, p);
        const unsigned kb = (unsigned)max((int64_t)1, min((p.cap + 255) / 256, (int64_t)4096));
        hipLaunchKernelGGL(k_fin_sum, dim3(kb), dim3(256), 0, stream, p);
        hipLaunchKernelGGL(k_agg_m2, dim3((unsigned)p.nchunks, ranges), dim3(AGG_THREADS), 0,
                           stream, p);
        hipLaunchKernelGGL(k_fin_m2, dim3(kb), dim3(256), 0, stream, p);
        hipLaunchKernelGGL(k_key_total, dim3(1), dim3(1024), 0, stream, p);
    }
    return hipGetLastError();
}

}  // namespace mag
