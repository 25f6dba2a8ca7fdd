// attr_fix.hip -- the small kernels around the tile kernel: intervals whose
// endpoints lie in different tiles, endpoints outside [t_0, t_{n-1}], the
// status block, and the clearing of the group-by state.

#include <algorithm>

#include "mag_internal.hpp"

namespace mag {

namespace {

__device__ __forceinline__ double endpoint_x(const double* s, const double* e, int64_t off,
                                             int64_t q)
{
    // endpoint q of a stream: even q = start of interval q/2, odd q = its end
    const int64_t i = off + (q >> 1);
    return (q & 1) ? e[i] : s[i];
}

}  // namespace

// ---------------------------------------------------------------------------
// one launch after the tiles: three kinds of workgroups
//   [0, nb_cross)               intervals whose endpoints lie in different tiles
//   [nb_cross, + 32 S)          endpoints before t_0 or after t_{n-1}
//   [.., + FOLD_BLOCKS)         the trace and idle energies of the tile waves
//   [.., + nb_clear)            the group-by state, cleared for the grouping
// ---------------------------------------------------------------------------
namespace {

__device__ void fix_cross(const FixParams& p, int64_t idx)
{
    const int64_t NT = p.NT, LD = p.ld;
    const int a = (int)(idx / (NT + 1));
    const int64_t b = idx - (int64_t)a * (NT + 1);
    const int64_t* c = p.cnt + (int64_t)a * (LD + 1);
    // the three loads requested together
    const int64_t c0 = c[b];
    const int64_t cprev = (b > 0) ? c[b - 1] : -1;
    const int64_t fin = p.cnt_fin[(int64_t)a * (LD + 1) + b];
    const int64_t len = 2 * (p.ss.off[a + 1] - p.ss.off[a]);
    if (p.validate && b > 0 && b < NT && fin != CNT_UNSET && fin != c0) {
        // a wave stopped at tile b with a cursor other than the one the next
        // wave searched for: some stream is unsorted
        atomicOr(&p.status->err, ERR_INTERVAL);
    }
    if (!(c0 & 1) || c0 > len) return;         // no interval active at tile start
    if (cprev == c0) return;                   // not the first tile it is active at
    const int64_t gid = p.ss.off[a] + (c0 >> 1);
    double E = (b > 0) ? p.tail[(int64_t)a * LD + b - 1] : 0.0;
    for (int64_t bb = b; bb < NT && c[bb] == c0; ++bb) E += p.head[(int64_t)a * LD + bb];
    p.energy[gid] = E;
}

// endpoints of stream a before t_0 / after t_{n-1}: thread r of nthreads
__device__ void fix_outside(const FixParams& p, int a, int64_t r, int64_t nthreads)
{
    const int64_t NT = p.NT;
    const int64_t off = p.ss.off[a];
    const int64_t len = 2 * (p.ss.off[a + 1] - off);
    const int64_t* c = p.cnt + (int64_t)a * (p.ld + 1);
    const int64_t c0 = min(max(c[0], (int64_t)0), len);
    const int64_t cN = min(max(c[NT], c0), len);
    const int64_t nbefore = c0, nafter = len - cN;
    const double t0 = p.status->bounds[0], tn = p.status->bounds[1];
    unsigned err = 0u;
    unsigned long long clipped = 0;
    for (int64_t qq = r; qq < nbefore + nafter; qq += nthreads) {
        const int64_t q = (qq < nbefore) ? qq : cN + (qq - nbefore);
        const int64_t gid = off + (q >> 1);
        const double x = endpoint_x(p.s, p.e, off, q);
        const int64_t sidx = (q < c0) ? 0 : p.n_total;
        if (q & 1) {
            if (p.end_idx) p.end_idx[gid] = sidx;
        } else {
            if (p.start_idx) p.start_idx[gid] = sidx;
        }
        if (p.validate) {
            bool bad = !(fabs(x) < INFINITY);
            if (q + 1 < len && !(x <= endpoint_x(p.s, p.e, off, q + 1))) bad = true;
            if (bad) err |= ERR_INTERVAL;
        }
        if (!(q & 1)) {
            if (q + 1 < c0 || q >= cN) p.energy[gid] = 0.0;  // wholly before or after
            if (x < t0) ++clipped;
        } else if (q >= cN && x > tn) {
            if (!(p.s[gid] < t0)) ++clipped;
        }
    }
    if (err) atomicOr(&p.status->err, err);
    if (clipped) atomicAdd(&p.status->n_clipped, clipped);
}

constexpr int FIX_THREADS = 256;
constexpr int OUT_BLOCKS = 32;  // workgroups per stream for the outside endpoints

// the {trace, idle} energies the tile waves left at the first tile of their
// runs; a run starts at tile 0 and at every tile where a wave stopped (its
// cnt_fin entry is set)
__device__ void fold_parts(const FixParams& p, int blk)
{
    __shared__ double2 red[FIX_THREADS / 64];
    const int64_t NT = p.NT;
    const int64_t per = (NT + FOLD_BLOCKS - 1) / FOLD_BLOCKS;
    const int64_t lo = (int64_t)blk * per, hi = min(lo + per, NT);
    double w = 0.0, idle = 0.0;
    for (int64_t b = lo + threadIdx.x; b < hi; b += FIX_THREADS) {
        // both loads issued together; other tiles' entries are never written
        const int64_t f = p.cnt_fin[b];
        const double2 v = p.part[b];
        const bool start = (b == 0) || (f != CNT_UNSET);
        w += start ? v.x : 0.0;
        idle += start ? v.y : 0.0;
    }
    for (int off = 32; off > 0; off >>= 1) {
        w += __shfl_xor(w, off);
        idle += __shfl_xor(idle, off);
    }
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = make_double2(w, idle);
    __syncthreads();
    if (threadIdx.x == 0) {
        double2 t = red[0];
        for (int u = 1; u < FIX_THREADS / 64; ++u) {
            t.x += red[u].x;
            t.y += red[u].y;
        }
        // a plain store: the call's last kernel adds the partial sums up (a
        // same-address atomic from every workgroup would queue for microseconds)
        p.fold[blk] = t;
    }
}

}  // namespace

__global__ __launch_bounds__(FIX_THREADS) void k_fix(const FixParams p, int64_t nb_cross,
                                                    int64_t nb_clear)
{
    const int64_t blk = blockIdx.x;
    if (blk < nb_cross) {
        const int64_t idx = blk * FIX_THREADS + threadIdx.x;
        if (idx < (int64_t)p.ss.S * (p.NT + 1)) fix_cross(p, idx);
        return;
    }
    const int64_t bo = blk - nb_cross;
    if (bo < (int64_t)OUT_BLOCKS * p.ss.S) {
        const int a = (int)(bo / OUT_BLOCKS);
        fix_outside(p, a, (bo % OUT_BLOCKS) * FIX_THREADS + threadIdx.x,
                    (int64_t)OUT_BLOCKS * FIX_THREADS);
        return;
    }
    const int64_t bf = bo - (int64_t)OUT_BLOCKS * p.ss.S;
    if (bf < FOLD_BLOCKS) {
        fold_parts(p, (int)bf);
        return;
    }
    const int64_t bc = bf - FOLD_BLOCKS;
    for (int64_t h = bc * FIX_THREADS + threadIdx.x; h <= (int64_t)p.H;
         h += nb_clear * FIX_THREADS) {
        reinterpret_cast<ulonglong2*>(p.table)[h] = make_ulonglong2(~0ull, ~0ull);  // empty, no id
        p.urank[h] = 0u;
    }
}

// ---------------------------------------------------------------------------
// small kernels
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_init(Status* st, int64_t* cnt_fin, int64_t n_fin,
                                              const double* t, int64_t n)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_fin;
         i += (int64_t)gridDim.x * blockDim.x)
        cnt_fin[i] = CNT_UNSET;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        st->err = 0u;
        st->special = 0u;
        st->overflow = 0u;
        st->n_clipped = 0ull;
        st->n_unique = 0u;
        st->n_cand = 0u;
        st->n_join = 0u;
        st->n_flag = 0u;
        st->n_waste = 0u;
        st->trace_energy = 0.0;
        st->idle_energy = 0.0;
        st->attributed_energy = 0.0;
        if (t) {
            st->bounds[0] = t[0];
            st->bounds[1] = t[n - 1];
        }
    }
}

__global__ __launch_bounds__(1024) void k_energy_total(const double* energy, int64_t m,
                                                      const double2* fold, Status* st)
{
    __shared__ double red[16];
    __shared__ double2 redf[16];
    const int tid = threadIdx.x;
    double v = 0.0;
    for (int64_t i = tid; i < m; i += 1024) v += energy[i];
    double2 f = make_double2(0.0, 0.0);
    if (fold)
        for (int b = tid; b < FOLD_BLOCKS; b += 1024) {
            f.x += fold[b].x;
            f.y += fold[b].y;
        }
    for (int off = 32; off > 0; off >>= 1) {
        v += __shfl_xor(v, off);
        f.x += __shfl_xor(f.x, off);
        f.y += __shfl_xor(f.y, off);
    }
    if ((tid & 63) == 0) {
        red[tid >> 6] = v;
        redf[tid >> 6] = f;
    }
    lds_barrier();
    if (tid == 0) {
        double s = 0.0;
        double2 t = make_double2(0.0, 0.0);
        for (int u = 0; u < 16; ++u) {
            s += red[u];
            t.x += redf[u].x;
            t.y += redf[u].y;
        }
        st->attributed_energy = s;
        if (fold) {
            st->trace_energy = t.x;
            st->idle_energy = t.y;
        }
    }
}

// samples [0, n) of a time and a power array copied together (one launch
// instead of two runtime copies, each of which costs a blit kernel)
__global__ __launch_bounds__(256) void k_stage_copy(double* dst_t, const double* src_t,
                                                    float* dst_P, const float* src_P, int64_t n)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        dst_t[i] = src_t[i];
        dst_P[i] = src_P[i];
    }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
hipError_t launch_stage_copy(double* dst_t, const double* src_t, float* dst_P, const float* src_P,
                             int64_t n, hipStream_t stream)
{
    if (n <= 0) return hipSuccess;
    const int64_t blocks = std::min<int64_t>((n + 255) / 256, 64);
    hipLaunchKernelGGL(k_stage_copy, dim3((unsigned)blocks), dim3(256), 0, stream, dst_t, src_t,
                       dst_P, src_P, n);
    return hipGetLastError();
}

hipError_t launch_init(Status* st, int64_t* cnt_fin, int64_t n_fin, const double* t, int64_t n,
                       hipStream_t stream)
{
    const int64_t blocks = max((int64_t)1, min((n_fin + 255) / 256, (int64_t)1024));
    hipLaunchKernelGGL(k_init, dim3((unsigned)blocks), dim3(256), 0, stream, st, cnt_fin, n_fin, t,
                       n);
    return hipGetLastError();
}

hipError_t launch_init_status(Status* st, const double* t, int64_t n, hipStream_t stream)
{
    return launch_init(st, nullptr, 0, t, n, stream);
}

hipError_t launch_fix(const FixParams& p, hipStream_t stream)
{
    const int64_t total = (int64_t)p.ss.S * (p.NT + 1);
    const int64_t nb_cross = (total + FIX_THREADS - 1) / FIX_THREADS;
    const int64_t nb_clear =
        p.table ? std::min<int64_t>(((int64_t)p.H + FIX_THREADS) / FIX_THREADS, 2048) : 0;
    const int64_t blocks = nb_cross + (int64_t)OUT_BLOCKS * p.ss.S + FOLD_BLOCKS + nb_clear;
    hipLaunchKernelGGL(k_fix, dim3((unsigned)blocks), dim3(FIX_THREADS), 0, stream, p, nb_cross,
                       nb_clear);
    return hipGetLastError();
}

hipError_t launch_energy_total(const double* energy, int64_t m, const double2* fold, Status* st,
                               hipStream_t stream)
{
    hipLaunchKernelGGL(k_energy_total, dim3(1), dim3(1024), 0, stream, energy, m, fold, st);
    return hipGetLastError();
}

}  // namespace mag
