// diff.hip -- join two per-key energy tables and rank the keys by
// r = (E_B - E_A) / E_A, descending, ties by ascending key.
//
// Stage 1 (k_diff_join): each workgroup takes 256 consecutive rows of table A.
// Both tables are ascending, so those rows can only match a contiguous range of
// table B; one wave finds the range (64-ary search), the workgroup stages it in
// LDS and every row finds its partner there.  Joined rows are ranked inside
// the workgroup; only rows whose local rank is below k can be in the global
// top k, so only those become candidates.
// Stage 2 (k_diff_rank): every candidate's global rank is the number of
// candidates ordered before it, counted in 256-candidate slices by many small
// workgroups; ranks below k are written out (k_diff_write).
// A batch (mag_diff_batch: one baseline against several candidates, the
// sweep of Section 6.1's per-case comparisons) runs the same stages for up to
// DIFF_BATCH candidates per launch, one candidate per blockIdx.z, with the
// candidates' parameters in the kernel-argument segment.
// Detection (Section 6.1) runs the same stages with k = the rows wanted: the
// flagged keys (r >= threshold) are a prefix of the ranking, so the first
// rows are the flagged ones; stage 1 also counts every flagged key and the
// waste among them, and stage 2 writes each row's latencies and verdict.

#include "mag_internal.hpp"

namespace mag {

namespace {

constexpr int JOIN_ROWS = 256;
constexpr int B_TILE = 2048;  // B keys staged per join workgroup
constexpr int RANK_SLICE = 256;

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

// both key tables strictly ascending (the grid strides over the rows)
__device__ __forceinline__ void check_ascending(const DiffParams& p, int64_t na, int64_t nb)
{
    unsigned bad = 0u;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i + 1 < max(na, nb);
         i += (int64_t)gridDim.x * blockDim.x) {
        if (i + 1 < na && !(p.ka[i] < p.ka[i + 1])) bad = 1u;
        if (i + 1 < nb && !(p.kb[i] < p.kb[i + 1])) bad = 1u;
    }
    if (bad) atomicOr(&p.status->err, ERR_KEYS);
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

// counters of each candidate's status block cleared (batches only: a single
// comparison clears its status with the attribution's init kernel)
__global__ __launch_bounds__(64) void k_diff_init(const BatchDiff b, int n)
{
    const int c = threadIdx.x;
    if (c < n) {
        Status* st = b.p[c].status;
        st->err = 0u;
        st->n_cand = 0u;
        st->n_join = 0u;
        st->n_flag = 0u;
        st->n_waste = 0u;
        st->diff_na = 0u;
        st->diff_nb = 0u;
    }
}

template <class A>
__global__ __launch_bounds__(256) void k_diff_check(const A a)
{
    const DiffParams& p = a.get();
    check_ascending(p, rows_a(p), rows_b(p));
}

template <class A>
__global__ __launch_bounds__(JOIN_ROWS) void k_diff_join(const A a)
{
    const DiffParams& p = a.get();
    __shared__ uint64_t bk[B_TILE];
    __shared__ double lr[JOIN_ROWS];
    __shared__ uint64_t lk[JOIN_ROWS];
    __shared__ int lv[JOIN_ROWS];
    __shared__ int64_t sh_range[2];
    const int tid = threadIdx.x;
    const int64_t na = rows_a(p), nb = rows_b(p);
    if (blockIdx.x == 0 && tid == 0) {
        p.status->diff_na = (uint32_t)na;
        p.status->diff_nb = (uint32_t)nb;
    }
    check_ascending(p, na, nb);  // (in the same launch: a failed check voids the result anyway)
    const int64_t row0 = (int64_t)blockIdx.x * JOIN_ROWS;
    const int64_t rows = min((int64_t)JOIN_ROWS, na - row0);
    if (rows <= 0) return;  // uniform: rows past a count read on the device
    if (tid < 64) {
        // B rows that can match: keys in [A[row0], A[row0 + rows - 1]]
        const int64_t lo = wave_count_below(p.kb, nb, p.ka[row0], false);
        const int64_t hi = wave_count_below(p.kb, nb, p.ka[row0 + rows - 1], true);
        if (tid == 0) {
            sh_range[0] = lo;
            sh_range[1] = max(hi, lo);
        }
    }
    __syncthreads();
    const int64_t blo = sh_range[0], bn = sh_range[1] - sh_range[0];
    const bool staged = bn <= B_TILE;
    if (staged)
        for (int64_t v = tid; v < bn; v += JOIN_ROWS) bk[v] = p.kb[blo + v];
    __syncthreads();

    double r = 0.0;
    uint64_t key = 0;
    int valid = 0;
    int64_t ib = -1;
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
    bool cand = false;
    if (valid) {
        int64_t rank = 0;
#pragma unroll 16
        for (int q = 0; q < JOIN_ROWS; ++q) rank += (lv[q] != 0) & before(lr[q], lk[q], r, key);
        cand = rank < p.k;
    }
    // one counter update per wave: candidates take consecutive slots
    const int lane = tid & 63;
    const uint64_t cb = __ballot(cand);
    const unsigned long long nvalid = __popcll(__ballot(valid != 0));
    bool flag = false, waste = false;
    if (p.detect && valid) {
        flag = r >= p.threshold;
        waste = flag && is_waste(p.la[row0 + tid], p.lb[ib], p.tolerance);
    }
    const unsigned long long nflag = __popcll(__ballot(flag));
    const unsigned long long nwaste = __popcll(__ballot(waste));
    uint32_t base = 0u;
    if (lane == 0) {
        if (cb) base = atomicAdd(&p.status->n_cand, (uint32_t)__popcll(cb));
        if (nvalid) atomicAdd(&p.status->n_join, (uint32_t)nvalid);
        if (nflag) atomicAdd(&p.status->n_flag, (uint32_t)nflag);
        if (nwaste) atomicAdd(&p.status->n_waste, (uint32_t)nwaste);
    }
    base = __shfl(base, 0);
    if (cand) {
        const uint32_t c = base + (uint32_t)__popcll(cb & ((1ull << lane) - 1ull));
        p.cand_r[c] = r;
        p.cand_key[c] = key;
        p.cand_ia[c] = (int32_t)(row0 + tid);
        p.cand_ib[c] = (int32_t)ib;
        p.cand_rank[c] = 0u;
    }
}

// candidates [64 bx, 64 bx + 64) counted against the slice [256 by, 256 by + 256)
template <class A>
__global__ __launch_bounds__(64) void k_diff_rank(const A a)
{
    const DiffParams& p = a.get();
    __shared__ double tr[RANK_SLICE];
    __shared__ uint64_t tk[RANK_SLICE];
    const uint32_t nc = p.status->n_cand;
    const uint32_t c0 = blockIdx.x * 64u, s0 = blockIdx.y * (uint32_t)RANK_SLICE;
    if (c0 >= nc || s0 >= nc) return;  // uniform
    const uint32_t cnt = min((uint32_t)RANK_SLICE, nc - s0);
    for (uint32_t v = threadIdx.x; v < cnt; v += 64) {
        tr[v] = p.cand_r[s0 + v];
        tk[v] = p.cand_key[s0 + v];
    }
    __syncthreads();
    const uint32_t c = c0 + threadIdx.x;
    if (c >= nc) return;
    const double r = p.cand_r[c];
    const uint64_t key = p.cand_key[c];
    uint32_t rank = 0;
    uint32_t v = 0;
    for (; v + 8 <= cnt; v += 8) {
#pragma unroll
        for (int w = 0; w < 8; ++w) rank += before(tr[v + w], tk[v + w], r, key) ? 1u : 0u;
    }
    for (; v < cnt; ++v) rank += before(tr[v], tk[v], r, key) ? 1u : 0u;
    if (rank) atomicAdd(&p.cand_rank[c], rank);
}

template <class A>
__global__ __launch_bounds__(256) void k_diff_write(const A a)
{
    const DiffParams& p = a.get();
    const uint32_t nc = p.status->n_cand;
    const uint32_t c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= nc) return;
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

int64_t diff_max_candidates(int64_t na, int64_t k)
{
    const int64_t groups = (na + JOIN_ROWS - 1) / JOIN_ROWS;
    return min(na, groups * min(k, (int64_t)JOIN_ROWS));
}

namespace {

// the stages of `n` comparisons that share table A (the single call: n = 1)
template <class A>
void launch_stages(const A& a, const DiffParams& p0, int n, hipStream_t stream)
{
    bool on_device = false;  // some sizes known on the device only
    bool any_empty_b = false;
    for (int c = 0; c < n; ++c) {
        on_device |= a.get_host(c).na_dev || a.get_host(c).nb_dev;
        any_empty_b |= (a.get_host(c).nb == 0);
    }
    if (!on_device && (p0.na == 0 || any_empty_b)) {
        int64_t mx = p0.na;
        for (int c = 0; c < n; ++c) mx = max(mx, a.get_host(c).nb);
        const unsigned cb = (unsigned)max((int64_t)1, min((mx + 255) / 256, (int64_t)1024));
        hipLaunchKernelGGL(k_diff_check<A>, dim3(cb, 1, n), dim3(256), 0, stream, a);
    }
    // an empty table B (known on the host) leaves no joined row: the join
    // kernel then finds no partner for any row of A
    if (p0.na > 0 && (on_device || n > 1 || p0.nb > 0)) {
        const unsigned jb = (unsigned)((p0.na + JOIN_ROWS - 1) / JOIN_ROWS);
        hipLaunchKernelGGL(k_diff_join<A>, dim3(jb, 1, n), dim3(JOIN_ROWS), 0, stream, a);
        const int64_t mc = diff_max_candidates(p0.na, p0.k);
        if (p0.k > 0 && mc > 0) {
            const dim3 rg((unsigned)((mc + 63) / 64), (unsigned)((mc + RANK_SLICE - 1) / RANK_SLICE),
                          n);
            hipLaunchKernelGGL(k_diff_rank<A>, rg, dim3(64), 0, stream, a);
            hipLaunchKernelGGL(k_diff_write<A>, dim3((unsigned)((mc + 255) / 256), 1, n), dim3(256),
                               0, stream, a);
        }
    }
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
        hipLaunchKernelGGL(k_diff_init, dim3(1), dim3(64), 0, stream, b, cnt);
        launch_stages(b, p[c0], cnt, stream);
    }
    return hipGetLastError();
}

}  // namespace mag
