// counter.hip -- per-operator energy from a delayed cumulative energy counter
// (Section 5.2, software replay mode).
//
// A reading C_j taken at t_j holds the energy used up to u_j = t_j - delay.  The
// cumulative energy C^(x) is the linear interpolant of (u_j, C_j), held at C_0
// before u_0 and at C_{n-1} after u_{n-1}.  Window i (s_i <= e_i <= s_{i+1})
// replayed its operator N_i times: E_i = (C^(e_i) - C^(s_i)) / N_i, the increase
// being the part of s_i's segment after s_i, plus the difference of the two
// readings that bound the whole segments in between, plus the part of e_i's
// segment before e_i.
//
// Work layout.  One 64-lane wave per chunk of 64 consecutive windows (lane l
// owns window 64c + l).  Chunk c owns the readings [J_c, J_{c+1}) with
// J_c = lower_bound(u, s_{64c}), J_0 = 0 and J_C = n: every reading is checked
// by exactly one wave (the J_c need not even increase for that), and for valid
// input every endpoint of the chunk's windows has its lower bound in
// [J_c, J_{c+1}].  The wave streams readings J_c .. min(J_{c+1}, n-1) through
// LDS in blocks of 256 (4 coalesced loads per lane) and resolves each endpoint
// by a binary search inside the block that holds its lower bound.  J_c comes
// from one probe of 64 readings around the position a uniform reading rate
// predicts, then a 64-ary search when the probe misses (irregular readings).
// The kernel is bound by HBM bandwidth: it reads every reading and every
// window once and writes each window's energy and indices once.

#include <hip/hip_ext.h>

#include "mag_internal.hpp"

namespace mag {
namespace {

constexpr int WAVE = 64;
constexpr int PER_LANE = CNT_BLOCK / WAVE;  // readings per lane and block
constexpr int FOLD_THREADS = 256;
constexpr int CFOLD_BLOCKS = 64;

__device__ __forceinline__ bool finite(double x) { return fabs(x) < INFINITY; }

__device__ __forceinline__ int count_true(bool p) { return __popcll(__ballot(p)); }

// lower_bound(u, x) over the whole trace for a wave-uniform x, u_j = t_j - delay.
// Terminates for any input (the candidate range shrinks every round); the
// result is the lower bound whenever u is strictly increasing.
__device__ int64_t wave_lower_bound(const CounterParams& p, double x, double u0, double un)
{
    const int k = __lane_id();
    const int64_t n = p.n;
    int64_t lo = 0, hi = n;  // the answer lies in [lo, hi]
    {
        // probe the 64 readings around the position a uniform rate predicts
        const double f = (x - u0) / (un - u0) * (double)(n - 1);
        const int64_t g = (f > 0.0) ? ((f < (double)(n - 1)) ? (int64_t)f : n - 1) : 0;
        const int64_t cnt = min((int64_t)WAVE, n);
        const int64_t w0 = max((int64_t)0, min(g - WAVE / 2, n - cnt));
        const bool in = k < cnt;
        const double uk = in ? p.t[w0 + k] - p.delay : 0.0;
        const int c = count_true(in && uk < x);
        if (c > 0) lo = w0 + c;
        if (c < cnt) hi = w0 + c;
    }
    while (lo < hi) {
        const int64_t len = hi - lo;
        if (len <= WAVE) {
            const bool in = k < len;
            const double uk = in ? p.t[lo + k] - p.delay : 0.0;
            return lo + count_true(in && uk < x);
        }
        // 64 probes spaced `step` apart, the first at lo
        const int64_t step = (len + WAVE - 1) / WAVE;
        const int64_t pos = lo + (int64_t)k * step;
        const bool in = pos < hi;
        const double uk = in ? p.t[pos] - p.delay : 0.0;
        const int c = count_true(in && uk < x);
        const int64_t lo0 = lo;
        if (c > 0) lo = lo0 + (int64_t)(c - 1) * step + 1;
        if (c < WAVE && lo0 + (int64_t)c * step < hi) hi = lo0 + (int64_t)c * step;
    }
    return lo;
}

// one endpoint: its lower bound and the readings on both sides of it
struct Endpoint {
    bool done;
    int64_t a;          // lower_bound(u, x)
    double lu, lc;      // u_{a-1}, C_{a-1} (meaningful when a >= 1)
    double hu, hc;      // u_a, C_a (meaningful when a <= n - 1)
};

// resolve x if its lower bound lies in the block [b, b + cnt) held in
// su/sc[1 .. cnt] (slot 0 holds the reading before the block)
__device__ __forceinline__ void resolve(Endpoint& q, double x, int64_t b, int cnt, double ulast,
                                        const double* su, const double* sc)
{
    if (q.done || !(x <= ulast)) return;
    int pos = 0;  // readings of the block below x
#pragma unroll
    for (int st = CNT_BLOCK / 2; st >= 1; st >>= 1)
        if (pos + st <= cnt && su[pos + st] < x) pos += st;
    pos = min(pos, cnt - 1);  // reached only by unsorted input
    q.a = b + pos;
    q.lu = su[pos];
    q.lc = sc[pos];
    q.hu = su[pos + 1];
    q.hc = sc[pos + 1];
    q.done = true;
}

// C^(e) - C^(s) from the two endpoints (s <= e)
__device__ __forceinline__ double window_increase(const Endpoint& qs, const Endpoint& qe, double s,
                                                  double e, int64_t n)
{
#pragma clang fp contract(off)
    if (qs.a == qe.a)  // one segment, or both before u_0, or both after u_{n-1}
        return (qs.a == 0 || qs.a == n) ? 0.0 : (qs.hc - qs.lc) * ((e - s) / (qs.hu - qs.lu));
    const double head = (qs.a == 0) ? 0.0 : (qs.hc - qs.lc) * ((qs.hu - s) / (qs.hu - qs.lu));
    const double mid = qe.lc - qs.hc;  // C_{a_e - 1} - C_{a_s}
    const double tail = (qe.a == n) ? 0.0 : (qe.hc - qe.lc) * ((e - qe.lu) / (qe.hu - qe.lu));
    return mid + (head + tail);
}

// workgroups are dealt to the 8 XCDs in turn: give each XCD a contiguous range
// of chunks, so that the readings two neighbouring chunks share sit in one L2
__device__ __forceinline__ int64_t xcd_block(int64_t b, int64_t G)
{
    const int64_t per = G / 8;
    return (b < 8 * per) ? (b % 8) * per + b / 8 : b;
}

__global__ __launch_bounds__(CNT_WAVES * WAVE) void k_counter(const CounterParams p)
{
    __shared__ double lds_u[CNT_WAVES][CNT_BLOCK + 1];
    __shared__ double lds_c[CNT_WAVES][CNT_BLOCK + 1];
    const int w = threadIdx.x / WAVE, k = threadIdx.x % WAVE;
    const int64_t chunk = xcd_block(blockIdx.x, gridDim.x) * CNT_WAVES + w;
    if (chunk >= p.nchunks) return;  // the whole wave
    double* su = lds_u[w];
    double* sc = lds_c[w];
    const int64_t n = p.n, m = p.m;
    const int64_t i0 = chunk * CNT_CHUNK, i = i0 + k;
    const bool live = i < m;
    const double s = live ? p.s[i] : 0.0;
    const double e = live ? p.e[i] : 0.0;
    const int32_t N = (live && p.reps) ? p.reps[i] : 1;
    const bool has_next = i0 + CNT_CHUNK < m;
    const double s_next = has_next ? p.s[i0 + CNT_CHUNK] : 0.0;
    const double u0 = p.t[0] - p.delay, un = p.t[n - 1] - p.delay;
    const int64_t Jc = (chunk == 0 || m == 0) ? 0 : wave_lower_bound(p, p.s[i0], u0, un);
    const int64_t Jn = has_next ? wave_lower_bound(p, s_next, u0, un) : n;

    uint32_t err = 0u;
    const double s_down = __shfl_down(s, 1);  // all lanes take part
    if (p.validate && live) {
        const double s_after = (k < WAVE - 1) ? s_down : s_next;  // s_{i+1}
        bool ok = finite(s) && finite(e) && s <= e && N >= 1;
        if (i + 1 < m && !(e <= s_after)) ok = false;
        if (!ok) err |= ERR_INTERVAL;
    }

    // the reading before the chunk's first one (slot 0)
    double lastu = -INFINITY, lastc = 0.0;
    if (Jc > 0) {
        lastu = p.t[Jc - 1] - p.delay;
        lastc = p.C[Jc - 1];
    }
    if (k == 0) {
        su[0] = lastu;
        sc[0] = lastc;
    }
    __builtin_amdgcn_wave_barrier();
    Endpoint qs{!live, 0, 0.0, 0.0, 0.0, 0.0}, qe{!live, 0, 0.0, 0.0, 0.0, 0.0};
    const int64_t last = min(Jn, n - 1);  // last reading streamed
    for (int64_t b = Jc; b <= last; b += CNT_BLOCK) {
        const int cnt = (int)min((int64_t)CNT_BLOCK, last + 1 - b);
        double tv[PER_LANE], cv[PER_LANE];
#pragma unroll
        for (int r = 0; r < PER_LANE; ++r) {
            const int q = k + WAVE * r;
            tv[r] = (q < cnt) ? p.t[b + q] : 0.0;
            cv[r] = (q < cnt) ? p.C[b + q] : 0.0;
        }
#pragma unroll
        for (int r = 0; r < PER_LANE; ++r) {
            const int q = k + WAVE * r;
            if (q < cnt) {
                su[q + 1] = tv[r] - p.delay;
                sc[q + 1] = cv[r];
            }
        }
        // the lanes read each other's slots: keep the compiler from moving
        // those reads above the writes (one wave's LDS operations run in order)
        __builtin_amdgcn_wave_barrier();
        if (p.validate) {
#pragma unroll
            for (int r = 0; r < PER_LANE; ++r) {
                const int q = k + WAVE * r;
                const int64_t j = b + q;
                if (q < cnt && j < Jn) {
                    const double uq = tv[r] - p.delay;
                    const bool first = (j == 0);
                    const bool ok_t = finite(tv[r]) && finite(uq) && (first || su[q] < uq);
                    const bool ok_c = finite(cv[r]) && (first || sc[q] <= cv[r]);
                    err |= (ok_t ? 0u : ERR_TIMESTAMPS) | (ok_c ? 0u : ERR_COUNTER);
                }
            }
        }
        const double ulast = su[cnt];
        resolve(qs, s, b, cnt, ulast, su, sc);
        resolve(qe, e, b, cnt, ulast, su, sc);
        lastu = ulast;
        lastc = sc[cnt];
        __builtin_amdgcn_wave_barrier();
        if (k == 0) {  // the block's last reading precedes the next block
            su[0] = lastu;
            sc[0] = lastc;
        }
        __builtin_amdgcn_wave_barrier();
    }
    // beyond the last reading streamed: for valid input only past u_{n-1}
    if (!qs.done) qs = Endpoint{true, last + 1, lastu, lastc, lastu, lastc};
    if (!qe.done) qe = Endpoint{true, last + 1, lastu, lastc, lastu, lastc};

    double inc = 0.0;
    if (live) {
        inc = window_increase(qs, qe, s, e, n);
        p.energy[i] = inc / (double)N;
        if (p.start_idx) p.start_idx[i] = qs.a;
        if (p.end_idx) p.end_idx[i] = qe.a;
    }
    const int clipped = count_true(live && (s < u0 || e > un));
#pragma unroll
    for (int off = WAVE / 2; off > 0; off >>= 1) inc += __shfl_xor(inc, off);
    const uint32_t any = (__ballot((err & ERR_TIMESTAMPS) != 0u) ? ERR_TIMESTAMPS : 0u) |
                         (__ballot((err & ERR_COUNTER) != 0u) ? ERR_COUNTER : 0u) |
                         (__ballot((err & ERR_INTERVAL) != 0u) ? ERR_INTERVAL : 0u);
    if (k == 0) {
        p.part[chunk] = make_double2(inc, (double)clipped);
        if (any) atomicOr(&p.status->err, any);
    }
}

// whole-trace figures from the per-chunk ones, and the clearing of the
// group-by state that follows
__global__ __launch_bounds__(FOLD_THREADS) void k_counter_fold(const CounterParams p,
                                                               int64_t nb_clear)
{
    const int64_t blk = blockIdx.x;
    if (blk < CFOLD_BLOCKS) {
        __shared__ double2 red[FOLD_THREADS / WAVE];
        const int64_t per = (p.nchunks + CFOLD_BLOCKS - 1) / CFOLD_BLOCKS;
        const int64_t lo = blk * per, hi = min(lo + per, p.nchunks);
        double inc = 0.0, clipped = 0.0;
        for (int64_t c = lo + threadIdx.x; c < hi; c += FOLD_THREADS) {
            const double2 v = p.part[c];
            inc += v.x;
            clipped += v.y;
        }
        for (int off = WAVE / 2; off > 0; off >>= 1) {
            inc += __shfl_xor(inc, off);
            clipped += __shfl_xor(clipped, off);
        }
        if (threadIdx.x % WAVE == 0) red[threadIdx.x / WAVE] = make_double2(inc, clipped);
        lds_barrier();
        if (threadIdx.x == 0) {
            double2 t = red[0];
            for (int u = 1; u < FOLD_THREADS / WAVE; ++u) {
                t.x += red[u].x;
                t.y += red[u].y;
            }
            if (blk == 0) {
                // the counter's whole increase; idle = that minus the windows' increases
                const double trace = p.C[p.n - 1] - p.C[0];
                p.status->trace_energy = trace;
                t.x -= trace;
            }
            if (t.x != 0.0) atomicAdd(&p.status->idle_energy, -t.x);
            if (t.y != 0.0) atomicAdd(&p.status->n_clipped, (unsigned long long)t.y);
        }
        return;
    }
    const int64_t bc = blk - CFOLD_BLOCKS;
    for (int64_t h = bc * FOLD_THREADS + threadIdx.x; h <= (int64_t)p.H;
         h += nb_clear * FOLD_THREADS) {
        reinterpret_cast<ulonglong2*>(p.table)[h] = make_ulonglong2(~0ull, ~0ull);  // empty, no id
        p.urank[h] = 0u;
    }
}

}  // namespace

hipError_t launch_counter(const CounterParams& p, hipStream_t stream, hipEvent_t ev_start,
                          hipEvent_t ev_stop)
{
    const int64_t blocks = (p.nchunks + CNT_WAVES - 1) / CNT_WAVES;
    if (ev_start || ev_stop)
        hipExtLaunchKernelGGL(k_counter, dim3((unsigned)blocks), dim3(CNT_WAVES * WAVE), 0, stream,
                              ev_start, ev_stop, 0, p);
    else
        hipLaunchKernelGGL(k_counter, dim3((unsigned)blocks), dim3(CNT_WAVES * WAVE), 0, stream, p);
    return hipGetLastError();
}

hipError_t launch_counter_fold(const CounterParams& p, hipStream_t stream)
{
    int64_t nb_clear = p.table ? ((int64_t)p.H + FOLD_THREADS) / FOLD_THREADS : 0;
    if (nb_clear > 2048) nb_clear = 2048;
    hipLaunchKernelGGL(k_counter_fold, dim3((unsigned)(CFOLD_BLOCKS + nb_clear)), dim3(FOLD_THREADS),
                       0, stream, p, nb_clear);
    return hipGetLastError();
}

}  // namespace mag
