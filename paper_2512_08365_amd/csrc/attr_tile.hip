// attr_tile.hip -- per-interval energy attribution on gfx950.
//
// The power trace is cut into tiles of T = NTH * C sample segments
// [t_j, t_{j+1}]; a persistent workgroup walks a contiguous run of tiles and
// prefetches the next tile's samples (and endpoint window) into registers
// while the current tile runs.
//
// Work inside a tile is split so that no lane ever loops over segments:
//   samples   (lane k owns segments kC .. kC+C-1): segment energies
//             S_j = (P_j + P_{j+1}) (t_{j+1} - t_j) / 2, input checks, and a
//             segmented scan of S_j that restarts after every segment holding
//             an interval endpoint ("run sums": the energy of the whole
//             segments since the last endpoint);
//   endpoints (one lane per endpoint of the round): its segment (guessed from
//             the mean sample spacing, then corrected), its sample index, its
//             position in the time-merged order of all streams;
//   gaps      (one lane per gap between consecutive endpoints): the exact
//             integral of the linear interpolant over the gap = trapezoid
//             pieces at both ends + the run sum of the whole segments between,
//             divided by the number of active intervals (equal split);
//   intervals (one lane per interval starting in the round): the sum of its
//             gaps.
// Every energy is a sum of non-negative terms; no result is a difference of
// running totals.  A tile whose endpoints exceed the LDS window is processed
// in several rounds, each a time prefix of the remaining endpoints.
//
// Intervals whose endpoints lie in different tiles leave partial energies:
// head[a][b], the piece in tile b of stream a's interval active at the tile's
// start, and tail[a][b], the piece of the interval started in tile b and still
// active at its end; k_cross adds them in tile order (attr_fix.hip).

#include "mag_internal.hpp"

namespace mag {

namespace {

__device__ __forceinline__ double endpoint_x(const double* s, const double* e, int64_t off,
                                             int64_t q)
{
    const int64_t i = off + (q >> 1);
    return (q & 1) ? e[i] : s[i];
}

// linear interpolant on [ta, tb] at x, exactly the sample values at the ends
__device__ __forceinline__ double lerp_power(double ta, double tb, double pa, double pb, double x)
{
    if (x == ta) return pa;
    if (x == tb) return pb;
    return pa + (pb - pa) * ((x - ta) / (tb - ta));
}

// number of entries <= v (le) or < v (!le) in the sorted list xs[0, n)
__device__ __forceinline__ int count_below(const double* xs, int n, double v, bool le)
{
    int lo = 0, hi = n;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        const bool go = le ? (xs[mid] <= v) : (xs[mid] < v);
        if (go) lo = mid + 1; else hi = mid;
    }
    return lo;
}

template <int NTH>
__device__ __forceinline__ double block_sum_fixed(double v, double* red)
{
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    lds_barrier();
    double tot = 0.0;
#pragma unroll
    for (int w = 0; w < NTH / 64; ++w) tot += red[w];
    lds_barrier();
    return tot;
}

}  // namespace

template <int NTH, int C, int SMAX>
__global__ __launch_bounds__(NTH) void k_tile(const TileParams p)
{
    constexpr int T = NTH * C;
    constexpr int E = ROUND_EVENTS;
    constexpr int NW = NTH / 64;
    constexpr int PER = E / NTH;  // window entries prefetched per lane
    static_assert((E & (E - 1)) == 0 && E % NTH == 0 && E <= 2 * NTH, "window layout");
    static_assert((C & (C - 1)) == 0, "C power of two");

    // samples: column tid holds the C+1 samples of lane tid's segments
    __shared__ double sh_t[C + 1][NTH];
    __shared__ float sh_P[C + 1][NTH];
    __shared__ double sh_rs[C][NTH];          // run sums per segment
    __shared__ uint32_t sh_flag[T / 32];      // segment holds a breakpoint of the round
    __shared__ double ev_x[E];                // endpoint window, stream-major
    __shared__ int ev_pos[E];                 // merged position of a window slot
    __shared__ double mg_x[E];
    __shared__ int mg_j[E];                   // segment (bits 0..30) | end flag (bit 31)
    __shared__ int mg_m[E + 1];
    __shared__ double gv[E + 1];
    __shared__ int64_t st_q[MAX_STREAMS], st_q0[MAX_STREAMS], st_len[MAX_STREAMS];
    __shared__ int64_t st_off[MAX_STREAMS + 1];
    __shared__ int st_k[MAX_STREAMS], st_take[MAX_STREAMS];
    __shared__ int st_started[MAX_STREAMS], nx_started[MAX_STREAMS];
    __shared__ double st_acc[MAX_STREAMS], nx_acc[MAX_STREAMS];
    __shared__ double red[NW];
    __shared__ int sh_wsum[NW];
    __shared__ double sh_tend;
    __shared__ unsigned sh_err;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int S = p.ss.S;
    int lcap = 0;  // window slots per stream: the largest power of two with S * cap <= E
    while ((S << (lcap + 1)) <= E) ++lcap;
    const int cap = 1 << lcap;
    const int64_t NT = p.NT;  // the last tile's successor (larger while the end is unknown)
    const int64_t LD = p.ld;
    const int64_t b0 = p.tile_begin + (int64_t)blockIdx.x * p.tiles_per_wg;
    const int64_t b1 = min(b0 + p.tiles_per_wg, p.tile_end);
    if (b0 >= b1) return;  // uniform

    if (tid <= S) st_off[tid] = p.ss.off[tid];
    if (tid < S) {
        st_k[tid] = 0;
        st_take[tid] = 0;
    }
    if (tid == 0) sh_err = 0u;
    for (int w = tid; w < T / 32; w += NTH) sh_flag[w] = 0u;
    lds_barrier();
    if (tid < S) st_len[tid] = 2 * (st_off[tid + 1] - st_off[tid]);
    lds_barrier();
    {
        // cursor of each stream at the first tile: endpoints <= its start time
        // (64-ary search, one wave per stream: about four dependent loads)
        const double tau0 = p.t[b0 * T - p.base];
        for (int a = wave; a < S; a += NW) {
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
    lds_barrier();

    // registers holding the next tile's samples of this lane (and window)
    double nt[C + 1];
    float nP[C + 1];
    double ew[PER];
    bool ew_ready = false;
    unsigned err = 0u;

    auto load_samples = [&](int64_t b) {
        const int64_t j0 = b * T;
        const int L = (int)min((int64_t)T, p.nseg - j0);
        const int cs = min(max(L - tid * C, 0), C);
        const int64_t g = j0 + (int64_t)tid * C - p.base;
        if (cs == C && p.aligned16) {
            const double2* t2 = reinterpret_cast<const double2*>(p.t + g);
            const float4* P4 = reinterpret_cast<const float4*>(p.P + g);
#pragma unroll
            for (int u = 0; u < C / 2; ++u) {
                const double2 v = t2[u];
                nt[2 * u] = v.x;
                nt[2 * u + 1] = v.y;
            }
#pragma unroll
            for (int u = 0; u < C / 4; ++u) {
                const float4 v = P4[u];
                nP[4 * u] = v.x;
                nP[4 * u + 1] = v.y;
                nP[4 * u + 2] = v.z;
                nP[4 * u + 3] = v.w;
            }
            nt[C] = p.t[g + C];
            nP[C] = p.P[g + C];
        } else {
#pragma unroll
            for (int u = 0; u <= C; ++u) {
                if (u <= cs && cs > 0) {
                    nt[u] = p.t[g + u];
                    nP[u] = p.P[g + u];
                } else {
                    nt[u] = 0.0;
                    nP[u] = 0.0f;
                }
            }
        }
    };

    load_samples(b0);
    double w_acc = 0.0, idle = 0.0;  // this lane's share of the trace and idle energy

    for (int64_t b = b0; b < b1; ++b) {
        const int64_t j0 = b * T;
        const int L = (int)min((int64_t)T, p.nseg - j0);
        const int cs = min(max(L - tid * C, 0), C);  // segments of this lane

        // ---- samples: stage, segment energies, checks; then prefetch the next tile
        double Sj[C];
        double wsum = 0.0;
#pragma unroll
        for (int u = 0; u <= C; ++u) {
            sh_t[u][tid] = nt[u];
            sh_P[u][tid] = nP[u];
        }
#pragma unroll
        for (int u = 0; u < C; ++u) {
            const double ta = nt[u], tb = nt[u + 1];
            const float pa = nP[u], pb = nP[u + 1];
            Sj[u] = 0.0;
            if (u < cs) {
                if (p.validate) {
                    if (!(tb > ta) || !(fabs(ta) < INFINITY) || !(fabs(tb) < INFINITY))
                        err |= ERR_TIMESTAMPS;
                    if (!(pa >= 0.0f && pa < INFINITY) || !(pb >= 0.0f && pb < INFINITY))
                        err |= ERR_POWER;
                }
                Sj[u] = 0.5 * ((double)pa + (double)pb) * (tb - ta);
                wsum += Sj[u];
            }
        }
        if (cs > 0 && tid * C + cs == L) sh_tend = sh_t[cs][tid];
        if (b + 1 < b1) load_samples(b + 1);  // in flight while this tile runs

        if (tid < S) {
            p.cnt[(int64_t)tid * (LD + 1) + b] = st_q[tid];
            st_q0[tid] = st_q[tid];
            st_acc[tid] = 0.0;
            st_started[tid] = 0;
        }
        if (ew_ready) {
#pragma unroll
            for (int v = 0; v < PER; ++v) ev_x[tid + v * NTH] = ew[v];
        }
        w_acc += wsum;
        lds_barrier();
        const double tau_end = sh_tend;
        const double t_begin = sh_t[0][0];
        const double inv_dt = (double)L / (tau_end - t_begin);
        double rs_x = t_begin;  // where the round's first gap starts
        int rs_j = -1;          // its segment (-1: the tile's first sample)

        // sample time / power of tile index j in [0, L]
        auto t_at = [&](int j) -> double {
            const int u = j & (C - 1), k = j / C;
            return (u == 0 && k > 0) ? sh_t[C][k - 1] : sh_t[u][k];
        };
        auto P_at = [&](int j) -> double {
            const int u = j & (C - 1), k = j / C;
            return (double)((u == 0 && k > 0) ? sh_P[C][k - 1] : sh_P[u][k]);
        };
        auto rs_at = [&](int j) -> double { return sh_rs[j & (C - 1)][j / C]; };

        for (int round = 0;; ++round) {
            // ---- endpoint window of this round
            if (!(round == 0 && ew_ready)) {
                for (int idx = tid; idx < (S << lcap); idx += NTH) {
                    const int a = idx >> lcap, r = idx & (cap - 1);
                    const int64_t q = st_q[a] + r;
                    ev_x[idx] = (q < st_len[a]) ? endpoint_x(p.s, p.e, st_off[a], q) : INFINITY;
                }
                lds_barrier();
            }
            ew_ready = false;
            // endpoints of each stream inside this tile: the window is sorted, so
            // their count is the length of its prefix
            for (int idx = tid; idx < (S << lcap); idx += NTH) {
                const bool in = ev_x[idx] <= tau_end;
                if (cap >= 64) {  // the wave lies inside one stream's window
                    const int c = __popcll(__ballot(in));
                    if (lane == 0 && c) atomicAdd(&st_k[idx >> lcap], c);
                } else if (in) {
                    atomicAdd(&st_k[idx >> lcap], 1);
                }
            }
            lds_barrier();
            // every lane derives the round's shape from the counts
            double cut = INFINITY;
            bool fin = true;
            for (int a = 0; a < S; ++a)
                if (st_k[a] == cap && st_q[a] + cap < st_len[a]) {
                    fin = false;
                    cut = fmin(cut, ev_x[(a << lcap) + cap - 1]);
                }
            if (!fin) {
                // a full window limits the round to endpoints <= cut (a time prefix)
                for (int idx = tid; idx < (S << lcap); idx += NTH) {
                    const int a = idx >> lcap, r = idx & (cap - 1);
                    const bool in = r < st_k[a] && ev_x[idx] <= cut;
                    if (cap >= 64) {
                        const int c = __popcll(__ballot(in));
                        if (lane == 0 && c) atomicAdd(&st_take[a], c);
                    } else if (in) {
                        atomicAdd(&st_take[a], 1);
                    }
                }
                lds_barrier();
                if (tid == 0) {
                    int tot = 0;
                    for (int a = 0; a < S; ++a) tot += st_take[a];
                    if (tot == 0) {  // only with unsorted endpoints: force progress
                        for (int a = 0; a < S; ++a)
                            if (st_k[a] == cap && st_q[a] + cap < st_len[a]) {
                                st_take[a] = 1;
                                break;
                            }
                        sh_err |= ERR_INTERVAL;
                    }
                }
                lds_barrier();
            }
            const int* take = fin ? st_k : st_take;
            int Er = 0, m0 = 0;
            for (int a = 0; a < S; ++a) {
                Er += take[a];
                m0 += (int)(st_q[a] & 1);
            }
            // the round's start is a breakpoint too: runs restart after it
            if (tid == 0 && rs_j >= 0) atomicOr(&sh_flag[rs_j >> 5], 1u << (rs_j & 31));

            // prefetch the next tile's endpoint window (its cursor is known now)
            if (fin && round == 0 && b + 1 < b1) {
#pragma unroll
                for (int v = 0; v < PER; ++v) {
                    const int idx = tid + v * NTH;
                    double x = INFINITY;
                    if (idx < (S << lcap)) {
                        const int a = idx >> lcap, r = idx & (cap - 1);
                        const int64_t q = st_q[a] + take[a] + r;
                        if (q < st_len[a]) x = endpoint_x(p.s, p.e, st_off[a], q);
                    }
                    ew[v] = x;
                }
                ew_ready = true;
            }

            // ---- endpoints: segment, sample index, checks, merged position
            for (int k = tid; k < Er; k += NTH) {
                int a = 0, r = k;
                while (a + 1 < S && r >= take[a]) r -= take[a++];
                const int slot = (a << lcap) + r;
                const double x = ev_x[slot];
                const int64_t q = st_q[a] + r;
                // segment j with t_j < x <= t_{j+1}: guess from the mean spacing, correct
                int j = (int)fmin(fmax((x - t_begin) * inv_dt, 0.0), (double)(L - 1));
                int steps = 0;
                while (j > 0 && t_at(j) >= x && steps < 8) {
                    --j;
                    ++steps;
                }
                while (j < L - 1 && t_at(j + 1) < x && steps < 16) {
                    ++j;
                    ++steps;
                }
                if ((t_at(j) >= x && j > 0) || (j < L - 1 && t_at(j + 1) < x)) {
                    int lo = 0, hi = L;  // first sample index >= x
                    while (lo < hi) {
                        const int mid = (lo + hi) >> 1;
                        if (t_at(mid) < x) lo = mid + 1; else hi = mid;
                    }
                    j = min(max(lo, 1), L) - 1;
                }
                const int64_t gid = st_off[a] + (q >> 1);
                if (q & 1) {
                    if (p.end_idx) p.end_idx[gid] = j0 + j + 1;
                } else {
                    if (p.start_idx) p.start_idx[gid] = j0 + j + 1;
                }
                if (p.validate) {
                    bool bad = !(fabs(x) < INFINITY);
                    if (q + 1 < st_len[a]) {
                        const double xn = (r + 1 < cap) ? ev_x[slot + 1]
                                                        : endpoint_x(p.s, p.e, st_off[a], q + 1);
                        if (!(x <= xn)) bad = true;
                    }
                    if (bad) err |= ERR_INTERVAL;
                }
                // position in the time-merged order: endpoints of the other streams
                // before x (ties: lower stream first).  Entries past a stream's take
                // lie after x, so fixed-depth searches over the whole windows,
                // interleaved across streams, give the counts.
                int pos = r;
                {
                    int c[SMAX];
#pragma unroll
                    for (int a2 = 0; a2 < SMAX; ++a2) c[a2] = 0;
                    for (int step = cap >> 1; step > 0; step >>= 1) {
#pragma unroll
                        for (int a2 = 0; a2 < SMAX; ++a2) {
                            if (a2 < S && a2 != a) {
                                const double y = ev_x[(a2 << lcap) + c[a2] + step - 1];
                                if (a2 < a ? (y <= x) : (y < x)) c[a2] += step;
                            }
                        }
                    }
#pragma unroll
                    for (int a2 = 0; a2 < SMAX; ++a2) {
                        if (a2 < S && a2 != a) {
                            const double y = ev_x[(a2 << lcap) + c[a2]];
                            if (a2 < a ? (y <= x) : (y < x)) ++c[a2];
                            pos += min(c[a2], take[a2]);
                        }
                    }
                }
                pos = min(pos, Er - 1);
                ev_pos[slot] = pos;
                mg_x[pos] = x;
                mg_j[pos] = j | ((q & 1) ? (int)0x80000000 : 0);
                atomicOr(&sh_flag[j >> 5], 1u << (j & 31));
            }
            lds_barrier();

            // ---- run sums: segmented scan of whole-segment energies, restarting
            // after every segment that holds a breakpoint (its energy is cut into
            // pieces at the breakpoints instead)
            {
                double loc[C];
                double run = 0.0;
                bool reset = false;
#pragma unroll
                for (int u = 0; u < C; ++u) {
                    const int j = tid * C + u;
                    const bool prev_flag =
                        j > 0 && ((sh_flag[(j - 1) >> 5] >> ((j - 1) & 31)) & 1u);
                    const bool self_flag = (sh_flag[j >> 5] >> (j & 31)) & 1u;
                    const double v = (self_flag || u >= cs) ? 0.0 : Sj[u];
                    if (prev_flag) {
                        run = v;
                        reset = true;
                    } else {
                        run += v;
                    }
                    loc[u] = run;
                }
                // scan of the lanes' carries (reset flag, value)
                int h = reset ? 1 : 0;
                double x = run;
                for (int off = 1; off < 64; off <<= 1) {
                    const double xo = __shfl_up(x, off);
                    const int ho = __shfl_up(h, off);
                    if (lane >= off) {
                        x = h ? x : xo + x;
                        h |= ho;
                    }
                }
                if (lane == 63) {
                    red[wave] = x;
                    sh_wsum[wave] = h;
                }
                lds_barrier();
                double px = 0.0;
#pragma unroll
                for (int w = 0; w < NW; ++w)
                    if (w < wave) px = sh_wsum[w] ? red[w] : px + red[w];
                const double incl = h ? x : px + x;
                double cin = __shfl_up(incl, 1);
                if (lane == 0) cin = px;
                bool seen = false;
#pragma unroll
                for (int u = 0; u < C; ++u) {
                    const int j = tid * C + u;
                    if (j > 0 && ((sh_flag[(j - 1) >> 5] >> ((j - 1) & 31)) & 1u)) seen = true;
                    sh_rs[u][tid] = seen ? loc[u] : cin + loc[u];
                }
            }

            // ---- concurrency in each gap: m_g = m0 + sum of +-1 before endpoint g
            {
                const int g0 = 2 * tid, g1 = 2 * tid + 1;
                const int v0 = (g0 < Er) ? ((mg_j[g0] < 0) ? -1 : 1) : 0;
                const int v1 = (g1 < Er) ? ((mg_j[g1] < 0) ? -1 : 1) : 0;
                int s = v0 + v1;
                for (int off = 1; off < 64; off <<= 1) {
                    const int y = __shfl_up(s, off);
                    if (lane >= off) s += y;
                }
                lds_barrier();  // the carries' scratch above is free again
                if (lane == 63) sh_wsum[wave] = s;
                lds_barrier();
                int wbase = 0;
                for (int w = 0; w < wave; ++w) wbase += sh_wsum[w];
                const int excl = wbase + s - (v0 + v1);
                if (g0 < Er) mg_m[g0] = m0 + excl;
                if (g1 < Er) mg_m[g1] = m0 + excl + v0;
                if (tid == NTH - 1) mg_m[Er] = m0 + wbase + s;
            }
            lds_barrier();

            // ---- gap energies, split among the active intervals
            const int G = Er + (fin ? 1 : 0);
            for (int g = tid; g < G; g += NTH) {
                double xs, xe;
                int js, je;
                if (g == 0) {
                    xs = rs_x;
                    js = rs_j;
                } else {
                    xs = mg_x[g - 1];
                    js = min(mg_j[g - 1] & 0x7fffffff, L - 1);
                }
                if (g < Er) {
                    xe = mg_x[g];
                    je = min(mg_j[g] & 0x7fffffff, L - 1);
                } else {
                    xe = tau_end;
                    je = L - 1;
                }
                double Q;
                if (js == je) {
                    const double ta = t_at(js), tb = t_at(js + 1);
                    const double pa = P_at(js), pb = P_at(js + 1);
                    Q = 0.5 * (lerp_power(ta, tb, pa, pb, xs) + lerp_power(ta, tb, pa, pb, xe)) *
                        (xe - xs);
                } else {
                    Q = 0.0;
                    if (js >= 0) {
                        const double ta = t_at(js), tb = t_at(js + 1);
                        const double pa = P_at(js), pb = P_at(js + 1);
                        Q += 0.5 * (lerp_power(ta, tb, pa, pb, xs) + pb) * (tb - xs);
                    }
                    if (je > js + 1) Q += rs_at(je - 1);
                    const double ta = t_at(je), tb = t_at(je + 1);
                    const double pa = P_at(je), pb = P_at(je + 1);
                    Q += 0.5 * (pa + lerp_power(ta, tb, pa, pb, xe)) * (xe - ta);
                }
                const int m = mg_m[g];
                double v = 0.0;
                if (m > 0)
                    v = p.split ? Q / (double)m : Q;
                else
                    idle += Q;
                gv[g] = v;
            }
            lds_barrier();

            // ---- interval energies: intervals starting in this round
            for (int k = tid; k < Er; k += NTH) {
                int a = 0, r = k;
                while (a + 1 < S && r >= take[a]) r -= take[a++];
                const int64_t q = st_q[a] + r;
                if (q & 1) continue;
                const int slot = (a << lcap) + r;
                const int ps = ev_pos[slot];
                double acc = 0.0;
                if (r + 1 < take[a]) {
                    const int pe = min(ev_pos[slot + 1], G - 1);
                    for (int g = ps + 1; g <= pe; ++g) acc += gv[g];
                    p.energy[st_off[a] + (q >> 1)] = acc;
                } else {
                    for (int g = ps + 1; g < G; ++g) acc += gv[g];
                    nx_acc[a] = acc;
                    nx_started[a] = 1;
                }
            }
            // the interval each stream carried into this round
            if (tid < S) {
                const int a = tid;
                const int ta = take[a];
                const bool active = (st_q[a] & 1) != 0;
                const bool ends_open = ((st_q[a] + ta) & 1) != 0;
                if (active) {
                    double acc = 0.0;
                    if (ta > 0) {
                        const int pe = min(ev_pos[a << lcap], G - 1);
                        for (int g = 0; g <= pe; ++g) acc += gv[g];
                        const double Et = st_acc[a] + acc;
                        if (st_started[a])
                            p.energy[st_off[a] + (st_q[a] >> 1)] = Et;
                        else
                            p.head[(int64_t)a * LD + b] = Et;
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
            // clear the breakpoint flags for the next round
            for (int w = tid; w < T / 32; w += NTH) sh_flag[w] = 0u;
            lds_barrier();
            if (tid < S) {
                st_q[tid] += take[tid];
                st_acc[tid] = nx_acc[tid];
                st_started[tid] = nx_started[tid];
            }
            lds_barrier();
            if (tid < S) {
                st_k[tid] = 0;
                st_take[tid] = 0;
            }
            if (Er > 0) {
                rs_x = mg_x[Er - 1];
                rs_j = min(mg_j[Er - 1] & 0x7fffffff, L - 1);
            }
            if (fin) break;
        }

        // ---- interval still open at the tile's end: its piece of this tile
        if (tid < S && (st_q[tid] & 1)) {
            if (st_started[tid])
                p.tail[(int64_t)tid * LD + b] = st_acc[tid];
            else
                p.head[(int64_t)tid * LD + b] = st_acc[tid];
        }
    }

    // the workgroup's trace and idle energy, kept at its first tile (others 0)
    const double Wt = block_sum_fixed<NTH>(w_acc, red);
    const double It = block_sum_fixed<NTH>(idle, red);
    for (int64_t b = b0 + tid; b < b1; b += NTH) {
        p.tileW[b] = (b == b0) ? Wt : 0.0;
        p.tileIdle[b] = (b == b0) ? It : 0.0;
    }

    if (tid < S) {
        // where this workgroup stopped: the next workgroup must start there
        p.cnt_fin[(int64_t)tid * (LD + 1) + b1] = st_q[tid];
        if (b1 == NT) p.cnt[(int64_t)tid * (LD + 1) + NT] = st_q[tid];
    }
    if (err) atomicOr(&sh_err, err);
    lds_barrier();
    if (tid == 0 && sh_err) atomicOr(&p.status->err, sh_err);
}

hipError_t launch_tile(const TileParams& p, int grid, hipStream_t stream)
{
    if (p.ss.S == 1)
        hipLaunchKernelGGL((k_tile<TILE_THREADS, SEG_PER_THREAD, 1>), dim3(grid),
                           dim3(TILE_THREADS), 0, stream, p);
    else if (p.ss.S <= 4)
        hipLaunchKernelGGL((k_tile<TILE_THREADS, SEG_PER_THREAD, 4>), dim3(grid),
                           dim3(TILE_THREADS), 0, stream, p);
    else
        hipLaunchKernelGGL((k_tile<TILE_THREADS, SEG_PER_THREAD, MAX_STREAMS>), dim3(grid),
                           dim3(TILE_THREADS), 0, stream, p);
    return hipGetLastError();
}

}  // namespace mag
