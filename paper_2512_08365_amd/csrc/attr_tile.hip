// attr_tile.hip -- per-interval energy attribution on gfx950.
//
// The power trace is cut into tiles of TILE sample segments.  A persistent
// workgroup walks a contiguous run of tiles; for each tile it stages the
// samples in LDS, builds positive partial sums of the segment energies
// (per thread: 8 segments; per 8 threads: 64 segments), and consumes the
// interval endpoints of every stream that fall in the tile, in time order.
// The endpoints cut the tile into "gaps" with a constant set of active
// intervals; each gap's energy (trapezoid pieces at its ends plus whole
// segments in between) is divided by the number of active intervals (equal
// split) and added to each of them.  Every energy is a sum of non-negative
// terms, so no result is a difference of large running totals.
//
// Intervals whose endpoints lie in different tiles leave partial energies
// (head: the piece of the interval active at a tile's start; tail: the piece
// of the interval started in a tile and still active at its end), which
// k_cross adds up in tile order.  Endpoints before t_0 or after t_{n-1} are
// handled by k_outside.

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

__device__ __forceinline__ bool finite_d(double x) { return fabs(x) < INFINITY; }

// value of the linear interpolant at x in segment j (exact at the samples)
__device__ __forceinline__ double power_at(const double* ts, const float* Ps, int j, double x)
{
    const double ta = ts[j], tb = ts[j + 1];
    const double pa = (double)Ps[j], pb = (double)Ps[j + 1];
    if (x == ta) return pa;
    if (x == tb) return pb;
    return pa + (pb - pa) * ((x - ta) / (tb - ta));
}

__device__ __forceinline__ double piece(const double* ts, const float* Ps, int j, double a,
                                        double b)
{
    return 0.5 * (power_at(ts, Ps, j, a) + power_at(ts, Ps, j, b)) * (b - a);
}

__device__ __forceinline__ double seg_energy(const double* ts, const float* Ps, int j)
{
    return 0.5 * ((double)Ps[j] + (double)Ps[j + 1]) * (ts[j + 1] - ts[j]);
}

// sum of whole segment energies j in [a, b) from the per-8 and per-64 sums
__device__ double full_sum(const double* ts, const float* Ps, const double* c1,
                           const double* c2, int a, int b)
{
    double acc = 0.0;
    int j = a;
    while (j < b && (j & 7)) { acc += seg_energy(ts, Ps, j); ++j; }
    while (j + 8 <= b && (j & 63)) { acc += c1[j >> 3]; j += 8; }
    while (j + 64 <= b) { acc += c2[j >> 6]; j += 64; }
    while (j + 8 <= b) { acc += c1[j >> 3]; j += 8; }
    while (j < b) { acc += seg_energy(ts, Ps, j); ++j; }
    return acc;
}

// energy of the interpolant between (xs in segment js) and (xe in segment je)
__device__ double gap_energy(const double* ts, const float* Ps, const double* c1,
                             const double* c2, double xs, int js, double xe, int je)
{
    if (js == je) return piece(ts, Ps, js, xs, xe);
    double q = piece(ts, Ps, js, xs, ts[js + 1]);
    q += full_sum(ts, Ps, c1, c2, js + 1, je);
    q += piece(ts, Ps, je, ts[je], xe);
    return q;
}

template <int NTH>
__device__ __forceinline__ double block_sum_ordered(double v, double* red)
{
    // deterministic: fixed butterfly inside each wave, then waves in order
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) red[wave] = v;
    __syncthreads();
    double tot = 0.0;
    for (int w = 0; w < NTH / 64; ++w) tot += red[w];
    __syncthreads();
    return tot;
}

}  // namespace

// ---------------------------------------------------------------------------
// main tile kernel
// ---------------------------------------------------------------------------
template <int T, int NTH>
__global__ __launch_bounds__(NTH) void k_tile(const TileParams p)
{
    constexpr int C = T / NTH;
    static_assert(C == 8, "full_sum assumes 8 segments per thread");
    static_assert(NTH % 64 == 0 && (NTH / 8) * 64 == T, "per-64 sums");
    constexpr int E = ROUND_EVENTS;
    static_assert(E <= 2 * NTH, "scan handles two events per thread");

    __shared__ double sh_t[T + 1];
    __shared__ float sh_P[T + 1];
    __shared__ double sh_c1[NTH];
    __shared__ double sh_c2[NTH / 8];
    __shared__ double ev_x[E];
    __shared__ int ev_pos[E];
    __shared__ double mg_x[E];
    __shared__ int mg_j[E];
    __shared__ int mg_d[E];
    __shared__ int mg_m[E + 1];
    __shared__ double gv[E + 1];
    __shared__ int64_t st_q[MAX_STREAMS];
    __shared__ int64_t st_len[MAX_STREAMS];
    __shared__ int64_t st_off[MAX_STREAMS + 1];
    __shared__ int st_k[MAX_STREAMS];
    __shared__ int st_take[MAX_STREAMS];
    __shared__ int st_started[MAX_STREAMS];
    __shared__ int nx_started[MAX_STREAMS];
    __shared__ double st_acc[MAX_STREAMS];
    __shared__ double nx_acc[MAX_STREAMS];
    __shared__ double sh_red[NTH / 64];
    __shared__ int sh_wsum[NTH / 64];
    __shared__ int sh_Er, sh_final, sh_m0;
    __shared__ double sh_cut;
    __shared__ double sh_rs_x;
    __shared__ int sh_rs_j;
    __shared__ unsigned sh_err;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int S = p.ss.S;
    const int cap = E / S;
    const int64_t NT = p.NT;

    const int64_t b0 = p.tile_begin + (int64_t)blockIdx.x * p.tiles_per_wg;
    const int64_t b1 = min(b0 + p.tiles_per_wg, p.tile_end);
    if (b0 >= b1) return;  // uniform over the block

    if (tid <= S) st_off[tid] = p.ss.off[tid];
    if (tid == 0) sh_err = 0u;
    __syncthreads();
    if (tid < S) st_len[tid] = 2 * (st_off[tid + 1] - st_off[tid]);
    __syncthreads();

    // cursor of each stream at the first tile: endpoints <= its start time
    // (64-ary search by one wave per stream: ~4 dependent loads)
    {
        const double tau0 = p.t[b0 * T - p.base];
        for (int a = wave; a < S; a += NTH / 64) {
            int64_t lo = 0, hi = st_len[a];
            while (hi - lo > 64) {
                const int64_t step = (hi - lo + 63) / 64;
                const int64_t pr = lo + (int64_t)(lane + 1) * step - 1;
                const bool ok = (pr < hi) && (endpoint_x(p.s, p.e, st_off[a], pr) <= tau0);
                const int c = __popcll(__ballot(ok));
                const int64_t nlo = lo + (int64_t)c * step;
                const int64_t nhi = min(hi, lo + (int64_t)(c + 1) * step - 1);
                lo = min(nlo, hi);
                hi = max(nhi, lo);
            }
            const int64_t pr = lo + lane;
            const bool ok = (pr < hi) && (endpoint_x(p.s, p.e, st_off[a], pr) <= tau0);
            const int c = __popcll(__ballot(ok));
            if (lane == 0) st_q[a] = lo + c;
        }
    }
    if (tid < S) {
        st_acc[tid] = 0.0;
        st_started[tid] = 0;
    }
    __syncthreads();

    unsigned err = 0u;

    for (int64_t b = b0; b < b1; ++b) {
        const int64_t j0 = b * T;
        const int L = (int)min((int64_t)T, p.nseg - j0);

        // ---- stage the tile's samples
        {
            const double* tg = p.t + (j0 - p.base);
            const float* Pg = p.P + (j0 - p.base);
            for (int i = tid; i <= L; i += NTH) {
                sh_t[i] = tg[i];
                sh_P[i] = Pg[i];
            }
        }
        if (tid < S) {
            p.cnt[(int64_t)tid * (NT + 1) + b] = st_q[tid];
            st_acc[tid] = 0.0;
            st_started[tid] = 0;
        }
        __syncthreads();

        // ---- segment energies: per-thread sums of 8, then sums of 64
        {
            double c1 = 0.0;
#pragma unroll
            for (int u = 0; u < C; ++u) {
                const int j = tid * C + u;
                if (j < L) {
                    const double ta = sh_t[j], tb = sh_t[j + 1];
                    const float pa = sh_P[j], pb = sh_P[j + 1];
                    if (p.validate) {
                        if (!(tb > ta) || !finite_d(ta) || !finite_d(tb)) err |= ERR_TIMESTAMPS;
                        if (!(pa >= 0.0f && pa < INFINITY) || !(pb >= 0.0f && pb < INFINITY))
                            err |= ERR_POWER;
                    }
                    c1 += 0.5 * ((double)pa + (double)pb) * (tb - ta);
                }
            }
            sh_c1[tid] = c1;
        }
        if (tid == 0) {
            sh_rs_x = sh_t[0];
            sh_rs_j = 0;
        }
        __syncthreads();
        if (tid < NTH / 8) {
            double c2 = 0.0;
#pragma unroll
            for (int u = 0; u < 8; ++u) c2 += sh_c1[tid * 8 + u];
            sh_c2[tid] = c2;
        }
        __syncthreads();
        if (tid == 0) {
            double w = 0.0;
            for (int u = 0; u < NTH / 8; ++u) w += sh_c2[u];
            p.tileW[b] = w;
        }

        const double tau_end = sh_t[L];
        double idle_acc = 0.0;

        // ---- endpoint rounds
        for (;;) {
            // window of up to `cap` endpoints per stream from its cursor
            for (int idx = tid; idx < S * cap; idx += NTH) {
                const int a = idx / cap, r = idx - a * cap;
                const int64_t q = st_q[a] + r;
                ev_x[idx] = (q < st_len[a]) ? endpoint_x(p.s, p.e, st_off[a], q) : INFINITY;
            }
            if (tid < S) st_k[tid] = cap;
            __syncthreads();
            // st_k[a]: length of the prefix of the window inside this tile
            for (int idx = tid; idx < S * cap; idx += NTH) {
                const int a = idx / cap, r = idx - a * cap;
                if (!(ev_x[idx] <= tau_end)) atomicMin(&st_k[a], r);
            }
            __syncthreads();
            if (tid == 0) {
                double cut = INFINITY;
                int full = 0, m0 = 0;
                for (int a = 0; a < S; ++a) {
                    if (st_k[a] == cap && st_q[a] + cap < st_len[a]) {
                        full = 1;
                        cut = fmin(cut, ev_x[a * cap + cap - 1]);
                    }
                    m0 += (int)(st_q[a] & 1);
                }
                sh_cut = cut;
                sh_final = !full;
                sh_m0 = m0;
            }
            __syncthreads();
            const bool fin = sh_final != 0;
            if (tid < S) st_take[tid] = st_k[tid];
            __syncthreads();
            if (!fin) {
                // a window filled up: take only endpoints <= the smallest
                // last-loaded time, so that the round holds a time-prefix
                const double cut = sh_cut;
                for (int idx = tid; idx < S * cap; idx += NTH) {
                    const int a = idx / cap, r = idx - a * cap;
                    if (r < st_k[a] && !(ev_x[idx] <= cut)) atomicMin(&st_take[a], r);
                }
                __syncthreads();
            }
            if (tid == 0) {
                int tot = 0;
                for (int a = 0; a < S; ++a) tot += st_take[a];
                if (tot == 0 && !fin) {
                    // only reachable with unsorted endpoints: force progress
                    for (int a = 0; a < S; ++a)
                        if (st_k[a] == cap && st_q[a] + cap < st_len[a]) {
                            st_take[a] = 1;
                            tot = 1;
                            break;
                        }
                    sh_err |= ERR_INTERVAL;
                }
                sh_Er = tot;
            }
            __syncthreads();
            const int Er = sh_Er;

            // segment, sample index, validation and merged position of each endpoint
            for (int idx = tid; idx < S * cap; idx += NTH) {
                const int a = idx / cap, r = idx - a * cap;
                if (r >= st_take[a]) continue;
                const double x = ev_x[idx];
                int lo = 0, hi = L + 1;
                while (lo < hi) {
                    const int mid = (lo + hi) >> 1;
                    if (sh_t[mid] < x) lo = mid + 1; else hi = mid;
                }
                const int lb = min(max(lo, 1), L);
                const int j = lb - 1;
                const int64_t q = st_q[a] + r;
                const int64_t gid = st_off[a] + (q >> 1);
                if (q & 1) {
                    if (p.end_idx) p.end_idx[gid] = j0 + lb;
                } else {
                    if (p.start_idx) p.start_idx[gid] = j0 + lb;
                }
                if (p.validate) {
                    bool bad = !finite_d(x);
                    if (q + 1 < st_len[a]) {
                        const double xn = (r + 1 < cap) ? ev_x[idx + 1]
                                                        : endpoint_x(p.s, p.e, st_off[a], q + 1);
                        if (!(x <= xn)) bad = true;
                    }
                    if (bad) err |= ERR_INTERVAL;
                }
                int pos = r;
                for (int a2 = 0; a2 < S; ++a2) {
                    if (a2 == a) continue;
                    const double* x2 = ev_x + a2 * cap;
                    int l2 = 0, h2 = st_take[a2];
                    if (a2 < a) {
                        while (l2 < h2) {
                            const int m = (l2 + h2) >> 1;
                            if (x2[m] <= x) l2 = m + 1; else h2 = m;
                        }
                    } else {
                        while (l2 < h2) {
                            const int m = (l2 + h2) >> 1;
                            if (x2[m] < x) l2 = m + 1; else h2 = m;
                        }
                    }
                    pos += l2;
                }
                pos = min(pos, Er - 1);
                ev_pos[idx] = pos;
                mg_x[pos] = x;
                mg_j[pos] = j;
                mg_d[pos] = (q & 1) ? -1 : 1;
            }
            __syncthreads();

            // concurrency in each gap: m_g = m0 + sum of +-1 before endpoint g
            {
                const int g0 = 2 * tid, g1 = 2 * tid + 1;
                const int v0 = (g0 < Er) ? mg_d[g0] : 0;
                const int v1 = (g1 < Er) ? mg_d[g1] : 0;
                int s = v0 + v1;
                for (int off = 1; off < 64; off <<= 1) {
                    const int y = __shfl_up(s, off);
                    if (lane >= off) s += y;
                }
                if (lane == 63) sh_wsum[wave] = s;
                __syncthreads();
                int wbase = 0;
                for (int w = 0; w < wave; ++w) wbase += sh_wsum[w];
                const int excl = wbase + s - (v0 + v1);
                const int m0 = sh_m0;
                if (g0 < Er) mg_m[g0] = m0 + excl;
                if (g1 < Er) mg_m[g1] = m0 + excl + v0;
                if (tid == NTH - 1) mg_m[Er] = m0 + wbase + s;
            }
            __syncthreads();

            // energy of each gap, divided among its active intervals
            const int G = Er + (fin ? 1 : 0);
            for (int g = tid; g < G; g += NTH) {
                double xs, xe;
                int js, je;
                if (g == 0) {
                    xs = sh_rs_x;
                    js = sh_rs_j;
                } else {
                    xs = mg_x[g - 1];
                    js = min(max(mg_j[g - 1], 0), L - 1);
                }
                if (g < Er) {
                    xe = mg_x[g];
                    je = min(max(mg_j[g], 0), L - 1);
                } else {
                    xe = sh_t[L];
                    je = L - 1;
                }
                const double Q = gap_energy(sh_t, sh_P, sh_c1, sh_c2, xs, js, xe, je);
                const int m = mg_m[g];
                double v = 0.0;
                if (m > 0)
                    v = p.split ? Q / (double)m : Q;
                else
                    idle_acc += Q;
                gv[g] = v;
            }
            __syncthreads();

            // interval energies: intervals that start in this round
            for (int idx = tid; idx < S * cap; idx += NTH) {
                const int a = idx / cap, r = idx - a * cap;
                if (r >= st_take[a]) continue;
                const int64_t q = st_q[a] + r;
                if (q & 1) continue;
                const int ps = ev_pos[idx];
                const int64_t gid = st_off[a] + (q >> 1);
                double acc = 0.0;
                if (r + 1 < st_take[a]) {
                    const int pe = min(ev_pos[idx + 1], G - 1);
                    for (int g = ps + 1; g <= pe; ++g) acc += gv[g];
                    p.energy[gid] = acc;
                } else {
                    for (int g = ps + 1; g < G; ++g) acc += gv[g];
                    nx_acc[a] = acc;
                    nx_started[a] = 1;
                }
            }
            // the interval each stream carried into this round
            if (tid < S) {
                const int a = tid;
                const int take = st_take[a];
                const bool active = (st_q[a] & 1) != 0;
                const bool ends_open = ((st_q[a] + take) & 1) != 0;
                if (active) {
                    double acc = 0.0;
                    if (take > 0) {
                        const int pe = min(ev_pos[a * cap], G - 1);
                        for (int g = 0; g <= pe; ++g) acc += gv[g];
                        const double Et = st_acc[a] + acc;
                        const int64_t gid = st_off[a] + (st_q[a] >> 1);
                        if (st_started[a])
                            p.energy[gid] = Et;
                        else
                            p.head[(int64_t)a * NT + b] = Et;
                        if (!ends_open) {
                            nx_acc[a] = 0.0;
                            nx_started[a] = 0;
                        }
                    } else {
                        for (int g = 0; g < G; ++g) acc += gv[g];
                        nx_acc[a] = st_acc[a] + acc;
                        nx_started[a] = st_started[a];
                    }
                } else if (!ends_open) {
                    nx_acc[a] = 0.0;
                    nx_started[a] = 0;
                }
            }
            __syncthreads();
            if (tid < S) {
                st_q[tid] += st_take[tid];
                st_acc[tid] = nx_acc[tid];
                st_started[tid] = nx_started[tid];
            }
            if (tid == 0 && Er > 0) {
                sh_rs_x = mg_x[Er - 1];
                sh_rs_j = min(max(mg_j[Er - 1], 0), L - 1);
            }
            __syncthreads();
            if (fin) break;
        }

        // ---- intervals still active at the tile's end
        if (tid < S) {
            const int a = tid;
            if (st_q[a] & 1) {
                if (st_started[a])
                    p.tail[(int64_t)a * NT + b] = st_acc[a];
                else
                    p.head[(int64_t)a * NT + b] = st_acc[a];
            }
        }
        const double idle = block_sum_ordered<NTH>(idle_acc, sh_red);
        if (tid == 0) p.tileIdle[b] = idle;
    }

    if (tid < S) {
        // where this workgroup stopped: the next workgroup must start there
        p.cnt_fin[(int64_t)tid * (NT + 1) + b1] = st_q[tid];
        if (b1 == NT) p.cnt[(int64_t)tid * (NT + 1) + NT] = st_q[tid];
    }
    if (err) atomicOr(&sh_err, err);
    __syncthreads();
    if (tid == 0 && sh_err) atomicOr(&p.status->err, sh_err);
}

// ---------------------------------------------------------------------------
// intervals whose endpoints lie in different tiles
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_cross(const FixParams p)
{
    const int64_t NT = p.NT;
    const int64_t total = (int64_t)p.ss.S * (NT + 1);
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int a = (int)(idx / (NT + 1));
        const int64_t b = idx - (int64_t)a * (NT + 1);
        const int64_t* c = p.cnt + (int64_t)a * (NT + 1);
        const int64_t c0 = c[b];
        const int64_t len = 2 * (p.ss.off[a + 1] - p.ss.off[a]);
        if (p.validate && b > p.tile_begin && b < NT && (b - p.tile_begin) % p.tiles_per_wg == 0 &&
            p.cnt_fin[(int64_t)a * (NT + 1) + b] != c0) {
            // the workgroups' endpoint ranges do not meet: some stream is unsorted
            atomicOr(&p.status->err, ERR_INTERVAL);
        }
        if (!(c0 & 1) || c0 > len) continue;            // no interval active at tile start
        if (b > 0 && c[b - 1] == c0) continue;         // not the first tile it is active at
        const int64_t gid = p.ss.off[a] + (c0 >> 1);
        double E = (b > 0) ? p.tail[(int64_t)a * NT + b - 1] : 0.0;
        for (int64_t bb = b; bb < NT && c[bb] == c0; ++bb) E += p.head[(int64_t)a * NT + bb];
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
    const int64_t* c = p.cnt + (int64_t)a * (NT + 1);
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
__global__ void k_init_status(Status* st, const double* t, int64_t n)
{
    if (threadIdx.x == 0) {
        st->err = 0u;
        st->n_inserted = 0u;
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

// whole-trace and idle energy: fixed-order reduction of the per-tile sums
__global__ __launch_bounds__(1024) void k_summary(const double* tileW, const double* tileIdle,
                                                   int64_t NT, Status* st)
{
    __shared__ double red[2][16];
    const int tid = threadIdx.x;
    const int64_t per = (NT + 1023) / 1024;
    const int64_t lo = (int64_t)tid * per, hi = min(lo + per, NT);
    double w = 0.0, z = 0.0;
    for (int64_t b = lo; b < hi; ++b) {
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
    __syncthreads();
    if (tid == 0) {
        double W = 0.0, I = 0.0;
        for (int u = 0; u < 16; ++u) {
            W += red[0][u];
            I += red[1][u];
        }
        st->trace_energy = W;
        st->idle_energy = I;
    }
}

__global__ __launch_bounds__(1024) void k_energy_total(const double* energy, int64_t m, Status* st)
{
    __shared__ double red[16];
    const int tid = threadIdx.x;
    const int64_t per = (m + 1023) / 1024;
    const int64_t lo = (int64_t)tid * per, hi = min(lo + per, m);
    double v = 0.0;
    for (int64_t i = lo; i < hi; ++i) v += energy[i];
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    if ((tid & 63) == 0) red[tid >> 6] = v;
    __syncthreads();
    if (tid == 0) {
        double s = 0.0;
        for (int u = 0; u < 16; ++u) s += red[u];
        st->attributed_energy = s;
    }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
hipError_t launch_init_status(Status* st, const double* t, int64_t n, hipStream_t stream)
{
    hipLaunchKernelGGL(k_init_status, dim3(1), dim3(64), 0, stream, st, t, n);
    return hipGetLastError();
}

hipError_t launch_tile(const TileParams& p, int grid, hipStream_t stream)
{
    hipLaunchKernelGGL((k_tile<TILE, TILE_THREADS>), dim3(grid), dim3(TILE_THREADS), 0, stream, p);
    return hipGetLastError();
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

hipError_t launch_summary(const double* tileW, const double* tileIdle, int64_t NT, Status* st,
                          hipStream_t stream)
{
    hipLaunchKernelGGL(k_summary, dim3(1), dim3(1024), 0, stream, tileW, tileIdle, NT, st);
    return hipGetLastError();
}

hipError_t launch_energy_total(const double* energy, int64_t m, Status* st, hipStream_t stream)
{
    hipLaunchKernelGGL(k_energy_total, dim3(1), dim3(1024), 0, stream, energy, m, st);
    return hipGetLastError();
}

}  // namespace mag
