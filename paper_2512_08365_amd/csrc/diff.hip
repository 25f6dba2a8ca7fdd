// diff.hip -- join two per-key energy tables and rank the keys by
// r = (E_B - E_A) / E_A, descending, ties by ascending key.
//
// Stage 1 (k_diff_join): each workgroup takes 256 consecutive rows of table A.
// Both tables are ascending, so those rows can only match a contiguous range of
// table B; one wave finds the range (64-ary search), the workgroup stages it in
// LDS and every row finds its partner there.  Joined rows are ranked inside
// the workgroup; only rows whose local rank is below k can be in the global
// top k, so only those become candidates, stored at the workgroup's own slots
// in local rank order, with the workgroup's counts beside them (no counter
// shared between workgroups).
// Stage 2 (k_diff_rank): every candidate's global rank is the number of
// candidates ordered before it, counted in 256-slot slices by many small
// workgroups; stage 3 (k_diff_write) writes ranks below k out, and its first
// workgroup adds the per-workgroup counts into the status block.
// A batch (mag_diff_batch: one baseline against several candidates, the
// sweep of Section 6.1's per-case comparisons) runs the same stages for up to
// DIFF_BATCH candidates per launch, one candidate per blockIdx.z, with the
// candidates' parameters in the kernel-argument segment.
// Detection (Section 6.1) runs the same stages with k = the rows wanted: the
// flagged keys (r >= threshold) are a prefix of the ranking, so the first
// rows are the flagged ones; stage 1 also counts every flagged key and the
// waste among them, and stage 3 writes each row's latencies and verdict.

#include "mag_internal.hpp"

namespace mag {

namespace {

constexpr int JOIN_ROWS = 256;
constexpr int B_TILE = 2048;  // B keys staged per join workgroup

__device__ __forceinline__ double rel_diff(double ea, double eb)
{
    if (ea == 0.0) return eb > 0.0 ? INFINITY : 0.0;
    return (eb - ea) / ea;
}

// a flagged key is waste when the efficient side A is at most `tolerance`
// slower than B
__device__ __forceinline__ bool is_waste(double la, double lb, double tolerance)
{
    return (la - lb) <= tolerance * lb;
}

// total order of the ranking: larger r first, then smaller key (evaluated
// without short-circuit branches, so loops over it stay straight-line code)
__device__ __forceinline__ bool before(double rq, uint64_t kq, double rp, uint64_t kp)
{
    return (rq > rp) | ((rq == rp) & (kq < kp));
}

// entries of the ascending array a[0, n) below v (or at most v), found by the
// 64 lanes of one wave together: a 64-ary search, a few dependent loads
__device__ int64_t wave_count_below(const uint64_t* a, int64_t n, uint64_t v, bool inclusive)
{
    const int lane = threadIdx.x & 63;
    int64_t lo = 0, hi = n;
    while (hi - lo > 64) {
        const int64_t step = (hi - lo + 63) / 64;
        const int64_t pr = lo + (int64_t)(lane + 1) * step - 1;
        bool ok = false;
        if (pr < hi) ok = inclusive ? (a[pr] <= v) : (a[pr] < v);
        const int c = __popcll(__ballot(ok));
        const int64_t nlo = lo + (int64_t)c * step;
        const int64_t nhi = min(hi, lo + (int64_t)(c + 1) * step - 1);
        lo = min(nlo, hi);
        hi = max(nhi, lo);
    }
    const int64_t pr = lo + lane;
    bool ok = false;
    if (pr < hi) ok = inclusive ? (a[pr] <= v) : (a[pr] < v);
    return lo + __popcll(__ballot(ok));
}

}  // namespace

// the key-table sizes: host values, or counts the attributions left on the
// device (never above the host bound)
__device__ __forceinline__ int64_t rows_a(const DiffParams& p)
{
    return p.na_dev ? min(max(*p.na_dev, (int64_t)0), p.na) : p.na;
}
__device__ __forceinline__ int64_t rows_b(const DiffParams& p)
{
    return p.nb_dev ? min(max(*p.nb_dev, (int64_t)0), p.nb) : p.nb;
}

// both key tables strictly ascending (the grid strides over the rows): whether
// this thread's stripe breaks the order
__device__ __forceinline__ bool unordered(const DiffParams& p, int64_t na, int64_t nb)
{
    bool bad = false;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i + 1 < max(na, nb);
         i += (int64_t)gridDim.x * blockDim.x) {
        if (i + 1 < na && !(p.ka[i] < p.ka[i + 1])) bad = true;
        if (i + 1 < nb && !(p.kb[i] < p.kb[i + 1])) bad = true;
    }
    return bad;
}

// candidate slots per join workgroup
__device__ __forceinline__ int64_t slots_per_group(const DiffParams& p)
{
    return min(p.k, (int64_t)JOIN_ROWS);
}

// the parameters of one comparison (blockIdx.z = 0), or of the candidate
// blockIdx.z of a batch
struct OneDiff {
    DiffParams p;
    __device__ __forceinline__ const DiffParams& get() const { return p; }
    __host__ const DiffParams& get_host(int) const { return p; }
};
struct BatchDiff {
    DiffParams p[DIFF_BATCH];
    __device__ __forceinline__ const DiffParams& get() const { return p[blockIdx.z]; }
    __host__ const DiffParams& get_host(int c) const { return p[c]; }
};

template <class A>
__global__ __launch_bounds__(JOIN_ROWS) void k_diff_join(const A a)
{
    const DiffParams& p = a.get();
    __shared__ uint64_t bk[B_TILE];
    __shared__ double lr[JOIN_ROWS];
    __shared__ uint64_t lk[JOIN_ROWS];
    __shared__ int lv[JOIN_ROWS];
    __shared__ int64_t sh_range[2];
    __shared__ uint32_t wstat[JOIN_ROWS / 64][4];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t na = rows_a(p), nb = rows_b(p);
    if (blockIdx.x == 0 && tid == 0) {
        p.status->diff_na = (uint32_t)na;
        p.status->diff_nb = (uint32_t)nb;
    }
    const bool bad = unordered(p, na, nb);  // a failed check voids the result anyway
    const int64_t row0 = (int64_t)blockIdx.x * JOIN_ROWS;
    const int64_t rows = min((int64_t)JOIN_ROWS, na - row0);
    double r = 0.0;
    uint64_t key = 0;
    int valid = 0;
    int64_t ib = -1;
    bool cand = false;
    int64_t rank = 0;
    if (rows > 0) {  // uniform: rows past a count read on the device have none
        if (tid < 128) {
            // B rows that can match: keys in [A[row0], A[row0 + rows - 1]]; the
            // two bounds searched by two waves side by side
            const bool upper = tid >= 64;
            const int64_t b = wave_count_below(p.kb, nb, p.ka[upper ? row0 + rows - 1 : row0], upper);
            if ((tid & 63) == 0) sh_range[upper ? 1 : 0] = b;
        }
        __syncthreads();
        const int64_t blo = sh_range[0], bn = max(sh_range[1], sh_range[0]) - sh_range[0];
        const bool staged = bn <= B_TILE;
        if (staged)
            for (int64_t v = tid; v < bn; v += JOIN_ROWS) bk[v] = p.kb[blo + v];
        __syncthreads();
        if (tid < rows) {
            const int64_t row = row0 + tid;
            key = p.ka[row];
            int64_t lo = 0, hi = bn;
            while (lo < hi) {
                const int64_t mid = (lo + hi) >> 1;
                const uint64_t y = staged ? bk[mid] : p.kb[blo + mid];
                if (y < key) lo = mid + 1; else hi = mid;
            }
            if (lo < bn && (staged ? bk[lo] : p.kb[blo + lo]) == key) {
                valid = 1;
                ib = blo + lo;
                r = rel_diff(p.sa[row], p.sb[ib]);
            }
        }
        lr[tid] = r;
        lk[tid] = key;
        lv[tid] = valid;
        __syncthreads();
        if (valid) {
#pragma unroll 16
            for (int q = 0; q < JOIN_ROWS; ++q) rank += (lv[q] != 0) & before(lr[q], lk[q], r, key);
            cand = rank < slots_per_group(p);
        }
    }
    bool flag = false, waste = false;
    if (p.detect && valid) {
        flag = r >= p.threshold;
        waste = flag && is_waste(p.la[row0 + tid], p.lb[ib], p.tolerance);
    }
    if (cand) {
        // the workgroup's candidates sit at its slots in local rank order
        const int64_t c = (int64_t)blockIdx.x * slots_per_group(p) + rank;
        p.cand_r[c] = r;
        p.cand_key[c] = key;
        p.cand_ia[c] = (int32_t)(row0 + tid);
        p.cand_ib[c] = (int32_t)ib;
        p.cand_rank[c] = (uint32_t)rank;  // the candidates of this workgroup before it
    }
    // the workgroup's counts, with plain stores: joined keys, candidates,
    // flagged keys, waste among them, and the order check
    const uint32_t nv = (uint32_t)__popcll(__ballot(valid != 0));
    const uint32_t nf = (uint32_t)__popcll(__ballot(flag));
    const uint32_t nw = (uint32_t)__popcll(__ballot(waste));
    const uint32_t nbad = (uint32_t)__popcll(__ballot(bad));
    if (lane == 0) {
        wstat[wave][0] = nv;
        wstat[wave][1] = nf;
        wstat[wave][2] = nw;
        wstat[wave][3] = nbad;
    }
    __syncthreads();
    if (tid == 0) {
        uint32_t t[4] = {0u, 0u, 0u, 0u};
        for (int w = 0; w < JOIN_ROWS / 64; ++w)
            for (int u = 0; u < 4; ++u) t[u] += wstat[w][u];
        uint32_t* g = p.blk + 8 * (int64_t)blockIdx.x;
        g[0] = t[0];
        g[1] = (uint32_t)min((int64_t)t[0], slots_per_group(p));
        g[2] = t[1];
        g[3] = t[2];
        g[4] = t[3] ? ERR_KEYS : 0u;
    }
}

// groups of candidates staged per rank workgroup
constexpr int RANK_GROUPS = 8;

// the candidates of join workgroup g (one per thread) counted against those of
// workgroups [RANK_GROUPS by, RANK_GROUPS by + RANK_GROUPS) other than g: each
// of those lists is in ranking order, so the number of its candidates ordered
// before a given one is found by binary search
template <class A>
__global__ __launch_bounds__(JOIN_ROWS) void k_diff_rank(const A a)
{
    const DiffParams& p = a.get();
    __shared__ double tr[RANK_GROUPS][JOIN_ROWS];
    __shared__ uint64_t tk[RANK_GROUPS][JOIN_ROWS];
    __shared__ int tn[RANK_GROUPS];
    const int64_t spg = slots_per_group(p);
    const int64_t g = blockIdx.x;
    const int64_t h0 = (int64_t)blockIdx.y * RANK_GROUPS;
    const int ncand = (int)p.blk[8 * g + 1];
    if (ncand == 0) return;  // uniform
    for (int u = 0; u < RANK_GROUPS; ++u) {
        const int64_t h = h0 + u;
        const int nh = (h < p.n_groups && h != g) ? (int)p.blk[8 * h + 1] : 0;
        if (threadIdx.x == 0) tn[u] = nh;
        for (int v = threadIdx.x; v < nh; v += JOIN_ROWS) {
            tr[u][v] = p.cand_r[h * spg + v];
            tk[u][v] = p.cand_key[h * spg + v];
        }
    }
    __syncthreads();
    const int i = threadIdx.x;
    if (i >= ncand) return;
    const int64_t c = g * spg + i;
    const double r = p.cand_r[c];
    const uint64_t key = p.cand_key[c];
    uint32_t rank = 0;
    for (int u = 0; u < RANK_GROUPS; ++u) {
        int lo = 0, hi = tn[u];
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if (before(tr[u][mid], tk[u][mid], r, key)) lo = mid + 1; else hi = mid;
        }
        rank += (uint32_t)lo;
    }
    if (rank) atomicAdd(&p.cand_rank[c], rank);
}

// candidates of join workgroup g (one per thread) whose rank is below k go
// out; workgroup 0 also adds the per-workgroup counts into the status block
template <class A>
__global__ __launch_bounds__(JOIN_ROWS) void k_diff_write(const A a)
{
    const DiffParams& p = a.get();
    const int64_t spg = slots_per_group(p);
    const int64_t g = blockIdx.x;
    if (g == 0) {
        __shared__ uint32_t red[5][JOIN_ROWS / 64];
        uint32_t t[5] = {0u, 0u, 0u, 0u, 0u};
        for (int64_t h = threadIdx.x; h < p.n_groups; h += JOIN_ROWS) {
            const uint32_t* b = p.blk + 8 * h;
            t[0] += b[0];
            t[1] += b[1];
            t[2] += b[2];
            t[3] += b[3];
            t[4] |= b[4];
        }
        for (int off = 32; off > 0; off >>= 1) {
            for (int u = 0; u < 4; ++u) t[u] += __shfl_xor(t[u], off);
            t[4] |= __shfl_xor(t[4], off);
        }
        if ((threadIdx.x & 63) == 0)
            for (int u = 0; u < 5; ++u) red[u][threadIdx.x >> 6] = t[u];
        __syncthreads();
        if (threadIdx.x == 0) {
            uint32_t s_[5] = {0u, 0u, 0u, 0u, 0u};
            for (int w = 0; w < JOIN_ROWS / 64; ++w) {
                for (int u = 0; u < 4; ++u) s_[u] += red[u][w];
                s_[4] |= red[4][w];
            }
            p.status->n_join = s_[0];
            p.status->n_cand = s_[1];
            p.status->n_flag = s_[2];
            p.status->n_waste = s_[3];
            p.status->err = s_[4];
        }
    }
    const int i = threadIdx.x;
    if (i >= (int)p.blk[8 * g + 1]) return;
    const int64_t c = g * spg + i;
    const uint32_t rank = p.cand_rank[c];
    if ((int64_t)rank >= p.k) return;
    const int32_t ia = p.cand_ia[c], ib = p.cand_ib[c];
    p.out_key[rank] = p.cand_key[c];
    p.out_ratio[rank] = p.cand_r[c];
    p.out_ea[rank] = p.sa[ia];
    p.out_eb[rank] = p.sb[ib];
    p.out_ca[rank] = p.ca[ia];
    p.out_cb[rank] = p.cb[ib];
    if (p.detect) {
        const double la = p.la[ia], lb = p.lb[ib];
        p.out_la[rank] = la;
        p.out_lb[rank] = lb;
        p.out_verdict[rank] = is_waste(la, lb, p.tolerance) ? MAG_WASTE : MAG_TRADEOFF;
    }
}

int64_t diff_groups(int64_t na) { return max((na + JOIN_ROWS - 1) / JOIN_ROWS, (int64_t)1); }

int64_t diff_max_candidates(int64_t na, int64_t k)
{
    return diff_groups(na) * min(k, (int64_t)JOIN_ROWS);
}

namespace {

// the stages of `n` comparisons that share table A (the single call: n = 1);
// p0.n_groups join workgroups (at least one: it also checks the order of B)
template <class A>
void launch_stages(const A& a, const DiffParams& p0, int n, hipStream_t stream)
{
    const unsigned jb = (unsigned)p0.n_groups;
    hipLaunchKernelGGL(k_diff_join<A>, dim3(jb, 1, n), dim3(JOIN_ROWS), 0, stream, a);
    if (p0.n_slots > 0) {
        const dim3 rg(jb, (unsigned)((p0.n_groups + RANK_GROUPS - 1) / RANK_GROUPS), n);
        hipLaunchKernelGGL(k_diff_rank<A>, rg, dim3(JOIN_ROWS), 0, stream, a);
    }
    hipLaunchKernelGGL(k_diff_write<A>, dim3(jb, 1, n), dim3(JOIN_ROWS), 0, stream, a);
}

}  // namespace

hipError_t launch_diff(const DiffParams& p, hipStream_t stream)
{
    OneDiff a{p};
    launch_stages(a, p, 1, stream);
    return hipGetLastError();
}

hipError_t launch_diff_batch(const DiffParams* p, int n, hipStream_t stream)
{
    for (int c0 = 0; c0 < n; c0 += DIFF_BATCH) {
        const int cnt = min(DIFF_BATCH, n - c0);
        BatchDiff b{};
        for (int c = 0; c < cnt; ++c) b.p[c] = p[c0 + c];
        launch_stages(b, p[c0], cnt, stream);
    }
    return hipGetLastError();
}

}  // namespace mag
