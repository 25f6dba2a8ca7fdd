// attr_fix.hip -- the small kernels around the tile kernel: intervals whose
// endpoints lie in different tiles, endpoints outside [t_0, t_{n-1}], the
// status block, and the fixed-order reductions of the per-tile totals.

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
// intervals whose endpoints lie in different tiles
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_cross(const FixParams p)
{
    const int64_t NT = p.NT, LD = p.ld;
    const int64_t total = (int64_t)p.ss.S * (NT + 1);
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int a = (int)(idx / (NT + 1));
        const int64_t b = idx - (int64_t)a * (NT + 1);
        const int64_t* c = p.cnt + (int64_t)a * (LD + 1);
        const int64_t c0 = c[b];
        const int64_t len = 2 * (p.ss.off[a + 1] - p.ss.off[a]);
        const int64_t fin = p.cnt_fin[(int64_t)a * (LD + 1) + b];
        if (p.validate && b > 0 && b < NT && fin != CNT_UNSET && fin != c0) {
            // a workgroup stopped at tile b with a cursor other than the one the
            // next workgroup searched for: some stream is unsorted
            atomicOr(&p.status->err, ERR_INTERVAL);
        }
        if (!(c0 & 1) || c0 > len) continue;            // no interval active at tile start
        if (b > 0 && c[b - 1] == c0) continue;         // not the first tile it is active at
        const int64_t gid = p.ss.off[a] + (c0 >> 1);
        double E = (b > 0) ? p.tail[(int64_t)a * LD + b - 1] : 0.0;
        for (int64_t bb = b; bb < NT && c[bb] == c0; ++bb) E += p.head[(int64_t)a * LD + bb];
        p.energy[gid] = E;
    }
}

// ---------------------------------------------------------------------------
// endpoints before t_0 or after t_{n-1}
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_outside(const FixParams p)
{
    const int a = blockIdx.y;
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
    for (int64_t qq = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; qq < nbefore + nafter;
         qq += (int64_t)gridDim.x * blockDim.x) {
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
        st->trace_energy = 0.0;
        st->idle_energy = 0.0;
        st->attributed_energy = 0.0;
        if (t) {
            st->bounds[0] = t[0];
            st->bounds[1] = t[n - 1];
        }
    }
}

// whole-trace and idle energy: fixed-order reduction of the per-tile sums,
// first over slices of SUM_SLICE tiles (one workgroup each), then over slices
__global__ __launch_bounds__(1024) void k_summary_part(const double* tileW, const double* tileIdle,
                                                        int64_t NT, double* part)
{
    __shared__ double red[2][16];
    const int tid = threadIdx.x;
    const int64_t lo = (int64_t)blockIdx.x * SUM_SLICE, hi = min(lo + SUM_SLICE, NT);
    double w = 0.0, z = 0.0;
    for (int64_t b = lo + tid; b < hi; b += 1024) {
        w += tileW[b];
        z += tileIdle[b];
    }
    for (int off = 32; off > 0; off >>= 1) {
        w += __shfl_xor(w, off);
        z += __shfl_xor(z, off);
    }
    if ((tid & 63) == 0) {
        red[0][tid >> 6] = w;
        red[1][tid >> 6] = z;
    }
    lds_barrier();
    if (tid == 0) {
        double W = 0.0, I = 0.0;
        for (int u = 0; u < 16; ++u) {
            W += red[0][u];
            I += red[1][u];
        }
        part[2 * blockIdx.x] = W;
        part[2 * blockIdx.x + 1] = I;
    }
}

__global__ __launch_bounds__(64) void k_summary_final(const double* part, int64_t nparts, Status* st)
{
    if (threadIdx.x == 0) {
        double W = 0.0, I = 0.0;
        for (int64_t k = 0; k < nparts; ++k) {
            W += part[2 * k];
            I += part[2 * k + 1];
        }
        st->trace_energy = W;
        st->idle_energy = I;
    }
}

__global__ __launch_bounds__(1024) void k_energy_total(const double* energy, int64_t m, Status* st)
{
    __shared__ double red[16];
    const int tid = threadIdx.x;
    double v = 0.0;
    for (int64_t i = tid; i < m; i += 1024) v += energy[i];
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    if ((tid & 63) == 0) red[tid >> 6] = v;
    lds_barrier();
    if (tid == 0) {
        double s = 0.0;
        for (int u = 0; u < 16; ++u) s += red[u];
        st->attributed_energy = s;
    }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
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

hipError_t launch_cross(const FixParams& p, hipStream_t stream)
{
    const int64_t total = (int64_t)p.ss.S * (p.NT + 1);
    const int64_t blocks = min((total + 255) / 256, (int64_t)65536);
    hipLaunchKernelGGL(k_cross, dim3((unsigned)blocks), dim3(256), 0, stream, p);
    return hipGetLastError();
}

hipError_t launch_outside(const FixParams& p, hipStream_t stream)
{
    hipLaunchKernelGGL(k_outside, dim3(32, (unsigned)p.ss.S), dim3(256), 0, stream, p);
    return hipGetLastError();
}

hipError_t launch_summary(const double* tileW, const double* tileIdle, int64_t NT, double* part,
                          Status* st, hipStream_t stream)
{
    const int64_t nparts = (NT + SUM_SLICE - 1) / SUM_SLICE;
    if (nparts > 0)
        hipLaunchKernelGGL(k_summary_part, dim3((unsigned)nparts), dim3(1024), 0, stream, tileW,
                           tileIdle, NT, part);
    hipLaunchKernelGGL(k_summary_final, dim3(1), dim3(64), 0, stream, part, nparts, st);
    return hipGetLastError();
}

hipError_t launch_energy_total(const double* energy, int64_t m, Status* st, hipStream_t stream)
{
    hipLaunchKernelGGL(k_energy_total, dim3(1), dim3(1024), 0, stream, energy, m, st);
    return hipGetLastError();
}

}  // namespace mag
