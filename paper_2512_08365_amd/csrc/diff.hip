// diff.hip -- join two per-key energy tables and rank the keys by
// r = (E_B - E_A) / E_A, descending, ties by ascending key.
//
// Stage 1 (k_diff_join): each workgroup takes 256 consecutive rows of table A,
// finds each key in table B by binary search (both tables are ascending), and
// ranks its joined rows inside the workgroup; only rows whose local rank is
// below k can be in the global top k, so only those become candidates.
// Stage 2 (k_diff_rank): every candidate's global rank is the number of
// candidates ordered before it; ranks below k are written out.

#include "mag_internal.hpp"

namespace mag {

namespace {

__device__ __forceinline__ double rel_diff(double ea, double eb)
{
    if (ea == 0.0) return eb > 0.0 ? INFINITY : 0.0;
    return (eb - ea) / ea;
}

// total order of the ranking: larger r first, then smaller key
__device__ __forceinline__ bool before(double rq, uint64_t kq, double rp, uint64_t kp)
{
    return rq > rp || (rq == rp && kq < kp);
}

}  // namespace

__global__ __launch_bounds__(256) void k_diff_check(const DiffParams p)
{
    unsigned bad = 0u;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i + 1 < max(p.na, p.nb);
         i += (int64_t)gridDim.x * blockDim.x) {
        if (i + 1 < p.na && !(p.ka[i] < p.ka[i + 1])) bad = 1u;
        if (i + 1 < p.nb && !(p.kb[i] < p.kb[i + 1])) bad = 1u;
    }
    if (bad) atomicOr(&p.status->err, ERR_KEYS);
}

__global__ __launch_bounds__(256) void k_diff_join(const DiffParams p)
{
    __shared__ double lr[256];
    __shared__ uint64_t lk[256];
    __shared__ int lv[256];
    const int tid = threadIdx.x;
    const int64_t row = (int64_t)blockIdx.x * 256 + tid;
    double r = 0.0;
    uint64_t key = 0;
    int valid = 0;
    int64_t ib = -1;
    if (row < p.na) {
        key = p.ka[row];
        int64_t lo = 0, hi = p.nb;
        while (lo < hi) {
            const int64_t mid = (lo + hi) >> 1;
            if (p.kb[mid] < key) lo = mid + 1; else hi = mid;
        }
        if (lo < p.nb && p.kb[lo] == key) {
            valid = 1;
            ib = lo;
            r = rel_diff(p.sa[row], p.sb[lo]);
        }
    }
    lr[tid] = r;
    lk[tid] = key;
    lv[tid] = valid;
    __syncthreads();
    if (valid) {
        int64_t rank = 0;
#pragma unroll 16
        for (int q = 0; q < 256; ++q)
            if (lv[q] && before(lr[q], lk[q], r, key)) ++rank;
        if (rank < p.k) {
            const uint32_t c = atomicAdd(&p.status->n_cand, 1u);
            p.cand_r[c] = r;
            p.cand_key[c] = key;
            p.cand_ia[c] = (int32_t)row;
            p.cand_ib[c] = (int32_t)ib;
        }
    }
    const unsigned long long nvalid = __popcll(__ballot(valid != 0));
    if ((tid & 63) == 0 && nvalid) atomicAdd(&p.status->n_join, (uint32_t)nvalid);
}

__global__ __launch_bounds__(256) void k_diff_rank(const DiffParams p)
{
    __shared__ double tr[1024];
    __shared__ uint64_t tk[1024];
    const uint32_t nc = p.status->n_cand;
    const uint32_t c = blockIdx.x * blockDim.x + threadIdx.x;
    if (blockIdx.x * blockDim.x >= nc) return;  // uniform
    const double r = (c < nc) ? p.cand_r[c] : 0.0;
    const uint64_t key = (c < nc) ? p.cand_key[c] : 0ull;
    int64_t rank = 0;
    for (uint32_t base = 0; base < nc; base += 1024) {
        const uint32_t cnt = min(1024u, nc - base);
        __syncthreads();
        for (uint32_t v = threadIdx.x; v < cnt; v += blockDim.x) {
            tr[v] = p.cand_r[base + v];
            tk[v] = p.cand_key[base + v];
        }
        __syncthreads();
        uint32_t v = 0;
        for (; v + 16 <= cnt; v += 16) {
#pragma unroll
            for (int w = 0; w < 16; ++w) rank += before(tr[v + w], tk[v + w], r, key) ? 1 : 0;
        }
        for (; v < cnt; ++v) rank += before(tr[v], tk[v], r, key) ? 1 : 0;
    }
    if (c < nc && rank < p.k) {
        const int32_t ia = p.cand_ia[c], ib = p.cand_ib[c];
        p.out_key[rank] = key;
        p.out_ratio[rank] = r;
        p.out_ea[rank] = p.sa[ia];
        p.out_eb[rank] = p.sb[ib];
        p.out_ca[rank] = p.ca[ia];
        p.out_cb[rank] = p.cb[ib];
    }
}

hipError_t launch_diff(const DiffParams& p, hipStream_t stream)
{
    const int64_t mx = max(p.na, p.nb);
    const unsigned cb = (unsigned)max((int64_t)1, min((mx + 255) / 256, (int64_t)1024));
    hipLaunchKernelGGL(k_diff_check, dim3(cb), dim3(256), 0, stream, p);
    if (p.na > 0 && p.nb > 0) {
        const unsigned jb = (unsigned)((p.na + 255) / 256);
        hipLaunchKernelGGL(k_diff_join, dim3(jb), dim3(256), 0, stream, p);
        if (p.k > 0) hipLaunchKernelGGL(k_diff_rank, dim3(jb), dim3(256), 0, stream, p);
    }
    return hipGetLastError();
}

}  // namespace mag
