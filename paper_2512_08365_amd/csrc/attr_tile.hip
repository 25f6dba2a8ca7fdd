// attr_tile.hip -- per-interval energy attribution on gfx950.
//
// The power trace is cut into tiles of T = 64 * C sample segments
// [t_j, t_{j+1}].  One wave (a 64-lane workgroup) owns one tile at a time and
// walks a contiguous run of tiles, carrying one cursor per interval stream (the
// number of that stream's interval endpoints at or before the tile's start).
// Nothing inside a tile needs a workgroup barrier: lanes exchange data through
// wave-private LDS and ballots, so many independent waves per CU hide each
// other's memory and LDS latency.
//
// Work inside a tile:
//   samples   (lane k owns segments kC .. kC+C-1): segment energies
//             S_j = (P_j + P_{j+1}) (t_{j+1} - t_j) / 2 and the input checks;
//   endpoints (up to two per lane per round): the endpoint's segment (guessed
//             from the mean sample spacing, then corrected), its sample index,
//             its position in the time-merged order of all streams and the
//             number of intervals active just after it -- both follow from how
//             many endpoints of each other stream precede it, since a stream
//             is inside an interval exactly when its cursor is odd;
//   run sums  a segmented scan of S_j that restarts after every segment
//             holding an endpoint (the energy of the whole segments between
//             two consecutive endpoints);
//   gaps      (one lane per gap between consecutive endpoints): the exact
//             integral of the linear interpolant over the gap = trapezoid
//             pieces at both ends + the run sum between, divided by the number
//             of active intervals (equal split);
//   intervals (one lane per interval starting in the round): the sum of its
//             gaps.
// Every energy is a sum of non-negative terms; no result is a difference of
// running totals.  A tile whose endpoints overflow the per-stream window is
// processed in several rounds, each a time prefix of the remaining endpoints.
//
// Intervals whose endpoints lie in different tiles leave partial energies:
// head[a][b], the piece in tile b of stream a's interval active at the tile's
// start, and tail[a][b], the piece of the interval started in tile b and still
// active at its end; k_cross adds them in tile order (attr_fix.hip).

#include "mag_internal.hpp"

namespace mag {

namespace {

constexpr int WAVE = 64;

__device__ __forceinline__ double endpoint_x(const double* s, const double* e, int64_t off,
                                             int64_t q)
{
    const int64_t i = off + (q >> 1);
    return (q & 1) ? e[i] : s[i];
}

// The kernel's arguments, read again from the kernel-argument segment where
// they are used (scalar loads that hit the constant cache).  Loaded once at
// entry, as the compiler does for a plain parameter, they would occupy scalar
// registers for the whole kernel and spill.  The pointer is made opaque at
// every call so that no load is shared between (or hoisted out of) phases.
typedef const __attribute__((address_space(4))) TileParams* KArgs;
__device__ __forceinline__ KArgs kargs()
{
    KArgs k = (KArgs)__builtin_amdgcn_kernarg_segment_ptr();
    asm volatile("" : "+s"(k));
    return k;
}

// linear interpolant on [ta, tb] at x, exactly the sample values at the ends
__device__ __forceinline__ double lerp_power(double ta, double tb, double pa, double pb, double x)
{
    if (x == ta) return pa;
    if (x == tb) return pb;
    return pa + (pb - pa) * ((x - ta) / (tb - ta));
}

// Lanes of one wave communicate through LDS without s_barrier: a wave's LDS
// operations complete in program order, and these fences keep the compiler
// from moving memory operations across the point.
__device__ __forceinline__ void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// DPP lane moves (bound_ctrl: lanes without a source read 0)
constexpr int DPP_ROW_SHR1 = 0x111, DPP_ROW_SHR2 = 0x112, DPP_ROW_SHR4 = 0x114,
              DPP_ROW_SHR8 = 0x118, DPP_ROW_BCAST15 = 0x142, DPP_ROW_BCAST31 = 0x143,
              DPP_WAVE_SHR1 = 0x138;

template <int CTRL, int ROWS>
__device__ __forceinline__ int dpp_i32(int v)
{
    return __builtin_amdgcn_update_dpp(0, v, CTRL, ROWS, 0xf, true);
}

template <int CTRL, int ROWS>
__device__ __forceinline__ double dpp_f64(double v)
{
    const uint64_t b = (uint64_t)__double_as_longlong(v);
    const uint32_t lo = (uint32_t)dpp_i32<CTRL, ROWS>((int)(uint32_t)b);
    const uint32_t hi = (uint32_t)dpp_i32<CTRL, ROWS>((int)(uint32_t)(b >> 32));
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// one step of a segmented inclusive scan: (h, x) after (hy, y) is
// (hy | h, h ? x : y + x); lanes without a source combine with (0, 0)
template <int CTRL, int ROWS>
__device__ __forceinline__ void seg_step(int& h, double& x)
{
    const int hy = dpp_i32<CTRL, ROWS>(h);
    const double y = dpp_f64<CTRL, ROWS>(x);
    x = h ? x : y + x;
    h |= hy;
}

// inclusive segmented scan over the 64 lanes: within rows of 16, then across rows
__device__ __forceinline__ void seg_scan_wave(int& h, double& x)
{
    seg_step<DPP_ROW_SHR1, 0xf>(h, x);
    seg_step<DPP_ROW_SHR2, 0xf>(h, x);
    seg_step<DPP_ROW_SHR4, 0xf>(h, x);
    seg_step<DPP_ROW_SHR8, 0xf>(h, x);
    seg_step<DPP_ROW_BCAST15, 0xa>(h, x);
    seg_step<DPP_ROW_BCAST31, 0xc>(h, x);
}

__device__ __forceinline__ double wave_sum(double v)
{
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    return v;
}

}  // namespace

// LDS of one wave (a workgroup holds WPB independent waves)
template <int C, int SMAX>
struct WaveLds {
    static constexpr int T = WAVE * C;
    static constexpr int E = WAVE;      // endpoints per round: one per lane
    static constexpr int W = 2 * WAVE;  // window entries: two per lane
    double sh_t[C + 1][WAVE];    // column k holds the C+1 samples of lane k's segments
    float sh_P[C + 1][WAVE];
    uint32_t flag[T / 32];       // segment holds a breakpoint of the round
    int wp[T / 32 + 1];          // set flags in the words before each word
    double R[E + 2];             // run sums, by rank of the breakpoint segment they end at
    double ev_x[W];              // endpoint window, stream-major
    double mg_x[E];              // merged endpoints
    uint32_t mg_jm[E];           // segment | active-after << 16 | end flag << 31
    double gv[E + 1];            // per-gap energy share
    uint8_t ev_pos[E];           // merged position of a round slot
    int64_t st_q[SMAX], st_off[SMAX], st_len[SMAX];
    int st_take[SMAX], st_first[SMAX];  // endpoints taken this round; first round slot
    int st_started[SMAX], nx_started[SMAX];
    double st_acc[SMAX], nx_acc[SMAX];
    double st_lastx[SMAX];       // the stream's last consumed endpoint
};

template <int C, int SMAX, int WPB>
__global__ __launch_bounds__(WAVE * WPB) __attribute__((amdgpu_waves_per_eu(4))) void k_tile(
    const TileParams p)
{
    using Lds = WaveLds<C, SMAX>;
    constexpr int T = Lds::T;
    constexpr int E = Lds::E;
    constexpr int W = Lds::W;
    constexpr int NWORD = T / 32;
    static_assert((C & (C - 1)) == 0 && C >= 4 && NWORD <= WAVE && E <= 255, "tile layout");

    __shared__ Lds lds_all[WPB];
    const int lane = threadIdx.x & (WAVE - 1);
    const int wave = threadIdx.x / WAVE;
    Lds& sm = lds_all[wave];
    const int S = p.ss.S;
    int lc = 0;  // window entries per stream: the largest power of two with S * cap <= W
    while ((S << (lc + 1)) <= W) ++lc;
    const int cap = 1 << lc;
    const int nslot = S << lc;
    const int budget = cap >> 1;  // per-stream share of the round slots when they run short
    // tile indices fit 32 bits (the host caps the trace length)
    const int b0 = (int)p.tile_begin + ((int)blockIdx.x * WPB + wave) * (int)p.tiles_per_wg;
    const int b1 = min(b0 + (int)p.tiles_per_wg, (int)p.tile_end);
    if (b0 >= b1) return;  // uniform per wave; waves never wait for each other

    if (lane < S) {
        sm.st_off[lane] = p.ss.off[lane];
        sm.st_len[lane] = 2 * (p.ss.off[lane + 1] - p.ss.off[lane]);
    }
    if (lane < NWORD) sm.flag[lane] = 0u;
    wave_sync();
    {
        // cursor of each stream at the first tile: endpoints <= its start time
        // (64-ary search, about four dependent loads per stream)
        const double tau0 = p.t[(int64_t)b0 * T - p.base];
        for (int a = 0; a < S; ++a) {
            const int64_t off = sm.st_off[a];
            int64_t lo = 0, hi = sm.st_len[a];
            while (hi - lo > WAVE) {
                const int64_t step = (hi - lo + WAVE - 1) / WAVE;
                const int64_t pr = lo + (int64_t)(lane + 1) * step - 1;
                const bool ok = (pr < hi) && (endpoint_x(p.s, p.e, off, pr) <= tau0);
                const int c = __popcll(__ballot(ok));
                const int64_t nlo = lo + (int64_t)c * step;
                const int64_t nhi = min(hi, lo + (int64_t)(c + 1) * step - 1);
                lo = min(nlo, hi);
                hi = max(nhi, lo);
            }
            const int64_t pr = lo + lane;
            const bool ok = (pr < hi) && (endpoint_x(p.s, p.e, off, pr) <= tau0);
            const int c = __popcll(__ballot(ok));
            if (lane == 0) {
                const int64_t q = lo + c;
                sm.st_q[a] = q;
                sm.st_lastx[a] = (q > 0) ? endpoint_x(p.s, p.e, off, q - 1) : -INFINITY;
            }
        }
    }
    wave_sync();

    // window slot of the stream cursors (advanced by each stream's take: the
    // next tile's window)
    auto window_x = [&](int slot, bool advance) -> double {
        if (slot >= nslot) return INFINITY;
        const int a = slot >> lc, r = slot & (cap - 1);
        const int64_t q = sm.st_q[a] + (advance ? sm.st_take[a] : 0) + r;
        const KArgs k = kargs();
        return (q < sm.st_len[a]) ? endpoint_x(k->s, k->e, sm.st_off[a], q) : INFINITY;
    };
    // breakpoint segments before segment j (the run sum ending at j-1 is R[rank(j)])
    auto rank_of = [&](int j) -> int {
        const int w = j >> 5;
        return sm.wp[w] + __popc(sm.flag[w] & ((1u << (j & 31)) - 1u));
    };

    double ew[2];  // prefetched window of the next tile
    bool ew_ready = false;
    unsigned err = 0u;
    double w_acc = 0.0, idle = 0.0;  // this lane's share of the trace and idle energy

    for (int b = b0; b < b1; ++b) {
        // the lane index, opaque to the compiler within this tile: keeps per-lane
        // 64-bit addresses from being hoisted out of the tile loop (where they
        // would occupy registers for the whole kernel and spill)
        int ln = lane;
        asm volatile("" : "+v"(ln));
        const int64_t j0 = (int64_t)b * T;
        const int L = (int)min((int64_t)T, kargs()->nseg - j0);
        const int cs = min(max(L - lane * C, 0), C);  // segments of this lane

        // ---- samples: load, stage, segment energies, checks
        {
            double tv[C + 1];
            float pv[C + 1];
            const KArgs k = kargs();
            const double* tp = k->t;
            const float* Pp = k->P;
            const int64_t g = j0 + (int64_t)ln * C - k->base;
            if (cs == C && k->aligned16) {
                const double2* t2 = reinterpret_cast<const double2*>(tp + g);
                const float4* P4 = reinterpret_cast<const float4*>(Pp + g);
#pragma unroll
                for (int u = 0; u < C / 2; ++u) {
                    const double2 v = t2[u];
                    tv[2 * u] = v.x;
                    tv[2 * u + 1] = v.y;
                }
#pragma unroll
                for (int u = 0; u < C / 4; ++u) {
                    const float4 v = P4[u];
                    pv[4 * u] = v.x;
                    pv[4 * u + 1] = v.y;
                    pv[4 * u + 2] = v.z;
                    pv[4 * u + 3] = v.w;
                }
                tv[C] = tp[g + C];
                pv[C] = Pp[g + C];
            } else {
                // a lane with fewer segments repeats its last sample time with
                // zero power: the missing segments have zero width and energy
#pragma unroll
                for (int u = 0; u <= C; ++u) {
                    if (u <= cs && cs > 0) {
                        tv[u] = tp[g + u];
                        pv[u] = Pp[g + u];
                    } else {
                        tv[u] = (u > 0) ? tv[u - 1] : 0.0;
                        pv[u] = 0.0f;
                    }
                }
            }
            if (k->validate) {
                // every segment of the lane rises (the repeated last time of a
                // short lane does not), and a strictly increasing run whose ends
                // are finite is finite throughout (a NaN fails every comparison)
                int rising = 0;
#pragma unroll
                for (int u = 0; u < C; ++u) rising += (tv[u + 1] > tv[u]) ? 1 : 0;
                const bool t_ok =
                    (rising == cs) & (fabs(tv[0]) < INFINITY) & (fabs(tv[C]) < INFINITY);
                bool p_ok = true;
#pragma unroll
                for (int u = 0; u <= C; ++u) p_ok &= (pv[u] >= 0.0f) & (pv[u] < INFINITY);
                err |= (t_ok ? 0u : ERR_TIMESTAMPS) | (p_ok ? 0u : ERR_POWER);
            }
#pragma unroll
            for (int u = 0; u <= C; ++u) {
                sm.sh_t[u][lane] = tv[u];
                sm.sh_P[u][lane] = pv[u];
            }
            // segment energies (P_u + P_{u+1}) (t_{u+1} - t_u), halved once at the end
            double wl = 0.0;
#pragma unroll
            for (int u = 0; u < C; ++u)
                wl += ((double)pv[u] + (double)pv[u + 1]) * (tv[u + 1] - tv[u]);
            w_acc += 0.5 * wl;
            // computed here, while the samples are in registers (not sunk to the
            // end of the tile, which would keep them live through the rounds)
            asm volatile("" : "+v"(w_acc));
        }
        if (lane < S) {
            const KArgs k = kargs();
            k->cnt[(int64_t)ln * (k->ld + 1) + b] = sm.st_q[lane];
            sm.st_acc[lane] = 0.0;
            sm.st_started[lane] = 0;
        }
        wave_sync();

        // sample time / power of tile index j in [0, L]
        auto t_at = [&](int j) -> double {
            const int u = j & (C - 1), k = j / C;
            return (u == 0 && k > 0) ? sm.sh_t[C][k - 1] : sm.sh_t[u][k];
        };
        auto P_at = [&](int j) -> double {
            const int u = j & (C - 1), k = j / C;
            return (double)((u == 0 && k > 0) ? sm.sh_P[C][k - 1] : sm.sh_P[u][k]);
        };

        const double t_begin = sm.sh_t[0][0];
        const double tau_end = t_at(L);
        const double inv_dt = (double)L / (tau_end - t_begin);
        double rs_x = t_begin;  // where the round's first gap starts
        int rs_j = -1;          // its segment (-1: the tile's first sample)

        for (;;) {
            // ---- endpoint window of this round: entry = stream * cap + rank
            double xw[2];
            uint64_t in[2];
#pragma unroll
            for (int v = 0; v < 2; ++v) {
                xw[v] = ew_ready ? ew[v] : window_x(lane + WAVE * v, false);
                sm.ev_x[lane + WAVE * v] = xw[v];
                in[v] = __ballot(xw[v] <= tau_end);
            }
            ew_ready = false;
            wave_sync();
            // each stream's endpoints in the tile are a prefix of its (sorted)
            // window.  If they all fit the round's slots they are all taken;
            // otherwise every stream keeps at most `budget` and the round ends at
            // the earliest time a stream runs out of its share (a time prefix)
            // stream a's entries are bits [a cap, (a + 1) cap) of the 128-bit mask
            auto count_in = [&](const uint64_t* m, int a) -> int {
                if (cap > WAVE) return __popcll(m[0]) + __popcll(m[1]);  // one stream
                if (cap == WAVE) return __popcll(m[a]);                     // two streams
                const int b0 = a << lc;
                const uint64_t w = (b0 >= WAVE) ? m[1] : m[0];
                return __popcll((w >> (b0 & (WAVE - 1))) & ((1ull << cap) - 1ull));
            };
            int tot = 0;
            bool over = false;
            for (int a = 0; a < S; ++a) {
                const int ka = count_in(in, a);
                tot += ka;
                if (ka == cap && sm.st_q[a] + cap < sm.st_len[a]) over = true;
            }
            double cut = INFINITY;
            bool fin = true;
            if (over || tot > E) {
                for (int a = 0; a < S; ++a) {
                    if (count_in(in, a) > budget) {
                        fin = false;
                        cut = fmin(cut, sm.ev_x[(a << lc) + budget - 1]);
                    }
                }
            }
            uint64_t tk[2];
#pragma unroll
            for (int v = 0; v < 2; ++v) tk[v] = fin ? in[v] : (in[v] & __ballot(xw[v] <= cut));
            int Er = 0, m0 = 0;
            for (int a = 0; a < S; ++a) {
                int ta = count_in(tk, a);
                if (!fin) ta = min(ta, budget);  // endpoints equal to the cut may wait
                if (lane == 0) {
                    sm.st_take[a] = ta;
                    sm.st_first[a] = Er;
                }
                Er += ta;
                m0 += (int)(sm.st_q[a] & 1);
            }
            if (!fin && Er == 0) {
                // only with unsorted endpoints: force progress, report
                for (int a = 0; a < S; ++a) {
                    if (count_in(in, a) > budget) {
                        if (lane == 0) {
                            sm.st_take[a] = 1;
                            for (int a2 = 0; a2 < S; ++a2) sm.st_first[a2] = (a2 > a) ? 1 : 0;
                        }
                        Er = 1;
                        break;
                    }
                }
                err |= ERR_INTERVAL;
            }
            // the round's start is a breakpoint too: runs restart after it
            if (lane == 0 && rs_j >= 0) atomicOr(&sm.flag[rs_j >> 5], 1u << (rs_j & 31));
            wave_sync();

            // prefetch the next tile's window (its cursors are known now)
            if (fin && b + 1 < b1) {
#pragma unroll
                for (int v = 0; v < 2; ++v) ew[v] = window_x(lane + WAVE * v, true);
                ew_ready = true;
            }

            // round slot of this lane: stream a (the last with first[a] <= lane), rank r
            int my_a = -1, my_r = 0;
            if (lane < Er) {
                my_a = 0;
                for (int a = 1; a < S; ++a)
                    if (sm.st_first[a] <= lane) my_a = a;
                my_r = lane - sm.st_first[my_a];
            }
            const double my_x = (my_a >= 0) ? sm.ev_x[(my_a << lc) + my_r] : 0.0;

            // ---- endpoints, part 1: segment, sample index, checks, breakpoint flag
            int my_j = -1;
            if (my_a >= 0) {
                const int a = my_a, r = my_r;
                const double x = my_x;
                const int64_t q = sm.st_q[a] + r;
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
                my_j = j;
                const int64_t gid = sm.st_off[a] + (q >> 1);
                const KArgs k = kargs();
                int64_t* idx = (q & 1) ? k->end_idx : k->start_idx;
                if (idx) idx[gid] = j0 + j + 1;
                if (k->validate) {
                    // finite and not before the stream's previous endpoint
                    const double xp = (r > 0) ? sm.ev_x[(a << lc) + r - 1] : sm.st_lastx[a];
                    if (!(fabs(x) < INFINITY) || !(xp <= x)) err |= ERR_INTERVAL;
                }
                atomicOr(&sm.flag[j >> 5], 1u << (j & 31));
            }
            wave_sync();
            // set flags in the words before each word (ranks of breakpoint segments)
            if (lane < NWORD) {
                int c = __popc(sm.flag[lane]);
                for (int off = 1; off < NWORD; off <<= 1) {
                    const int y = __shfl_up(c, off);
                    if (lane >= off) c += y;
                }
                sm.wp[lane + 1] = c;
                if (lane == 0) sm.wp[0] = 0;
            }
            wave_sync();

            // ---- run sums: segmented scan of whole-segment energies (recomputed
            // from the staged samples, bit for bit as above), restarting after
            // every breakpoint segment (whose energy is cut into pieces at its
            // breakpoints instead).  The run ending just before breakpoint
            // segment j (or before the tile's last segment) is stored at rank(j).
            {
                const int j0l = lane * C;
                const uint32_t myflags = (sm.flag[j0l >> 5] >> (j0l & 31)) & ((1u << C) - 1u);
                const uint32_t nextflags =
                    (j0l + C < T) ? ((sm.flag[(j0l + C) >> 5] >> ((j0l + C) & 31)) & 1u) : 0u;
                const bool prev_lane_last =
                    lane > 0 && ((sm.flag[(j0l - 1) >> 5] >> ((j0l - 1) & 31)) & 1u);
                double loc[C];
                double run = 0.0;
                bool reset = false;
#pragma unroll
                for (int u = 0; u < C; ++u) {
                    const bool prev_flag = (u == 0) ? prev_lane_last : ((myflags >> (u - 1)) & 1u);
                    const bool self_flag = (myflags >> u) & 1u;
                    const double v =
                        (self_flag || u >= cs)
                            ? 0.0
                            : 0.5 * ((double)sm.sh_P[u][lane] + (double)sm.sh_P[u + 1][lane]) *
                                  (sm.sh_t[u + 1][lane] - sm.sh_t[u][lane]);
                    if (prev_flag) {
                        run = v;
                        reset = true;
                    } else {
                        run += v;
                    }
                    loc[u] = run;
                }
                // the lanes' carries (reset flag, value): inclusive segmented
                // scan across the wave, then shifted by one lane
                int h = reset ? 1 : 0;
                double xs = run;
                seg_scan_wave(h, xs);
                const double cin = dpp_f64<DPP_WAVE_SHR1, 0xf>(xs);
                bool seen = false;
                const uint32_t fl = myflags | (nextflags << C);
                const int rbase = rank_of(j0l);  // breakpoint segments before this lane's
#pragma unroll
                for (int u = 0; u < C; ++u) {
                    const bool prev_flag = (u == 0) ? prev_lane_last : ((myflags >> (u - 1)) & 1u);
                    if (prev_flag) seen = true;
                    const int k = j0l + u;  // this run value ends at segment k
                    const bool nxt = ((fl >> (u + 1)) & 1u) != 0;
                    if (k + 1 < L && (nxt || (k + 1 == L - 1)))
                        sm.R[rbase + __popc(myflags & ((2u << u) - 1u))] =
                            seen ? loc[u] : cin + loc[u];
                }
            }

            // ---- endpoints, part 2: merged position and the intervals active after
            {
                int take[SMAX];
                int qpar[SMAX];
#pragma unroll
                for (int a2 = 0; a2 < SMAX; ++a2) {
                    take[a2] = (a2 < S) ? sm.st_take[a2] : 0;
                    qpar[a2] = (a2 < S) ? (int)(sm.st_q[a2] & 1) : 0;
                }
                if (my_j >= 0) {
                    const double x = my_x;
                    const int a = my_a, r = my_r;
                    const int q0 = (int)(sm.st_q[a] & 1);
                    // endpoints of each other stream before x in the merged order
                    // (ties: lower stream first); entries past a stream's take lie
                    // after x, so fixed-depth searches of the whole window suffice
                    int pos = r;
                    int m_after = (q0 + r + 1) & 1;
                    int c[SMAX];
#pragma unroll
                    for (int a2 = 0; a2 < SMAX; ++a2) c[a2] = 0;
                    // (straight-line: every lane runs every step of every search)
                    for (int step = cap >> 1; step > 0; step >>= 1) {
#pragma unroll
                        for (int a2 = 0; a2 < SMAX; ++a2) {
                            const double y = sm.ev_x[(min(a2, S - 1) << lc) + c[a2] + step - 1];
                            const bool pr = (y < x) | ((a2 < a) & (y == x));
                            c[a2] += pr ? step : 0;
                        }
                    }
#pragma unroll
                    for (int a2 = 0; a2 < SMAX; ++a2) {
                        const double y = sm.ev_x[(min(a2, S - 1) << lc) + c[a2]];
                        const bool pr = (y < x) | ((a2 < a) & (y == x));
                        const int ca = min(c[a2] + (pr ? 1 : 0), take[a2]);
                        const bool other = (a2 < S) & (a2 != a);
                        pos += other ? ca : 0;
                        m_after += other ? ((qpar[a2] + ca) & 1) : 0;
                    }
                    pos = min(pos, Er - 1);
                    const int64_t q = sm.st_q[a] + r;
                    sm.ev_pos[lane] = (uint8_t)pos;
                    sm.mg_x[pos] = x;
                    sm.mg_jm[pos] = (uint32_t)my_j | ((uint32_t)m_after << 16) |
                                    ((q & 1) ? 0x80000000u : 0u);
                }
            }
            wave_sync();

            // ---- gap energies, split among the active intervals
            const int G = Er + (fin ? 1 : 0);
            for (int g = lane; g < G; g += WAVE) {
                double xs, xe;
                int js, je, m;
                if (g == 0) {
                    xs = rs_x;
                    js = rs_j;
                    m = m0;
                } else {
                    const uint32_t w = sm.mg_jm[g - 1];
                    xs = sm.mg_x[g - 1];
                    js = min((int)(w & 0xffffu), L - 1);
                    m = (int)((w >> 16) & 0x7fffu);
                }
                if (g < Er) {
                    xe = sm.mg_x[g];
                    je = min((int)(sm.mg_jm[g] & 0xffffu), L - 1);
                } else {
                    xe = tau_end;
                    je = L - 1;
                }
                // trapezoids of the interpolant: within one segment, or the piece to
                // the end of the first segment + whole segments + the piece from the
                // start of the last (straight-line code: both forms are evaluated)
                const int js0 = max(js, 0);
                const double ta_s = t_at(js0), tb_s = t_at(js0 + 1);
                const double pa_s = P_at(js0), pb_s = P_at(js0 + 1);
                const double ta_e = t_at(je), tb_e = t_at(je + 1);
                const double pa_e = P_at(je), pb_e = P_at(je + 1);
                const double px_s = lerp_power(ta_s, tb_s, pa_s, pb_s, xs);
                const double px_e = lerp_power(ta_e, tb_e, pa_e, pb_e, xe);
                const double q_in = 0.5 * (px_s + px_e) * (xe - xs);
                const double q_first = (js >= 0) ? 0.5 * (px_s + pb_s) * (tb_s - xs) : 0.0;
                const double q_mid = (je > js + 1) ? sm.R[rank_of(je)] : 0.0;
                const double q_last = 0.5 * (pa_e + px_e) * (xe - ta_e);
                const double Q = (js == je) ? q_in : (q_first + q_mid) + q_last;
                const double v = (m > 0) ? (kargs()->split ? Q / (double)m : Q) : 0.0;
                idle += (m > 0) ? 0.0 : Q;
                sm.gv[g] = v;
            }
            wave_sync();

            // ---- interval energies: intervals starting in this round
            if (my_j >= 0 && !((sm.st_q[my_a] + my_r) & 1)) {
                const int a = my_a, r = my_r;
                const int64_t q = sm.st_q[a] + r;
                const int ta = sm.st_take[a];
                const int ps = sm.ev_pos[lane];
                double acc = 0.0;
                if (r + 1 < ta) {
                    const int pe = min((int)sm.ev_pos[lane + 1], G - 1);
                    for (int g = ps + 1; g <= pe; ++g) acc += sm.gv[g];
                    kargs()->energy[sm.st_off[a] + (q >> 1)] = acc;
                } else {
                    for (int g = ps + 1; g < G; ++g) acc += sm.gv[g];
                    sm.nx_acc[a] = acc;
                    sm.nx_started[a] = 1;
                }
            }
            // the interval each stream carried into this round
            if (lane < S) {
                const int a = lane;
                const int ta = sm.st_take[a];
                const bool active = (sm.st_q[a] & 1) != 0;
                const bool ends_open = ((sm.st_q[a] + ta) & 1) != 0;
                if (active) {
                    double acc = 0.0;
                    if (ta > 0) {
                        const int pe = min((int)sm.ev_pos[sm.st_first[a]], G - 1);
                        for (int g = 0; g <= pe; ++g) acc += sm.gv[g];
                        const double Et = sm.st_acc[a] + acc;
                        const KArgs k = kargs();
                        if (sm.st_started[a])
                            k->energy[sm.st_off[a] + (sm.st_q[a] >> 1)] = Et;
                        else
                            k->head[(int64_t)(a + ln - lane) * k->ld + b] = Et;
                        if (!ends_open) {
                            sm.nx_acc[a] = 0.0;
                            sm.nx_started[a] = 0;
                        }
                    } else {
                        for (int g = 0; g < G; ++g) acc += sm.gv[g];
                        sm.nx_acc[a] = sm.st_acc[a] + acc;
                        sm.nx_started[a] = sm.st_started[a];
                    }
                } else if (!ends_open) {
                    sm.nx_acc[a] = 0.0;
                    sm.nx_started[a] = 0;
                }
            }
            if (Er > 0) {
                rs_x = sm.mg_x[Er - 1];
                rs_j = min((int)(sm.mg_jm[Er - 1] & 0xffffu), L - 1);
            }
            wave_sync();
            // commit the round; clear the breakpoint flags
            if (lane < S) {
                const int ta = sm.st_take[lane];
                if (ta > 0) sm.st_lastx[lane] = sm.ev_x[(lane << lc) + ta - 1];
                sm.st_q[lane] += ta;
                sm.st_acc[lane] = sm.nx_acc[lane];
                sm.st_started[lane] = sm.nx_started[lane];
            }
            if (lane < NWORD) sm.flag[lane] = 0u;
            wave_sync();
            if (fin) break;
        }

        // ---- interval still open at the tile's end: its piece of this tile
        if (lane < S && (sm.st_q[lane] & 1)) {
            const KArgs k = kargs();
            double* dst = sm.st_started[lane] ? k->tail : k->head;
            dst[(int64_t)ln * k->ld + b] = sm.st_acc[lane];
        }
        wave_sync();
    }

    // the wave's trace and idle energy, kept at its first tile (others 0)
    const double Wt = wave_sum(w_acc);
    const double It = wave_sum(idle);
    const KArgs k = kargs();
    for (int b = b0 + lane; b < b1; b += WAVE) {
        k->tileW[b] = (b == b0) ? Wt : 0.0;
        k->tileIdle[b] = (b == b0) ? It : 0.0;
    }
    if (lane < S) {
        // where this wave stopped: the next wave must start there
        const int LD = (int)k->ld;
        k->cnt_fin[(int64_t)lane * (LD + 1) + b1] = sm.st_q[lane];
        if (b1 == (int)k->NT) k->cnt[(int64_t)lane * (LD + 1) + b1] = sm.st_q[lane];
    }
    if (__ballot(err != 0u)) {
        unsigned e = err;
        for (int off = 32; off > 0; off >>= 1) e |= __shfl_xor(e, off);
        if (lane == 0) atomicOr(&k->status->err, e);
    }
}

namespace {

constexpr int TILE_WPB = 4;  // independent waves per workgroup

template <int SMAX>
hipError_t launch_tile_t(TileParams p, int64_t ntiles, hipStream_t stream)
{
    using K = decltype(&k_tile<SEG_PER_THREAD, SMAX, TILE_WPB>);
    const K kern = k_tile<SEG_PER_THREAD, SMAX, TILE_WPB>;
    // persistent waves: as many as can be resident at once, each over a
    // contiguous run of tiles
    static int per_cu = 0;
    if (per_cu == 0) {
        int nb = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kern, WAVE * TILE_WPB, 0) !=
                hipSuccess ||
            nb <= 0)
            nb = 2;
        per_cu = nb;
    }
    const int64_t waves = (int64_t)device_cu_count() * per_cu * TILE_WPB;
    p.tiles_per_wg = (ntiles + waves - 1) / waves;
    const int64_t runs = (ntiles + p.tiles_per_wg - 1) / p.tiles_per_wg;
    const int grid = (int)((runs + TILE_WPB - 1) / TILE_WPB);
    hipLaunchKernelGGL(kern, dim3(grid), dim3(WAVE * TILE_WPB), 0, stream, p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_tile(const TileParams& p, hipStream_t stream)
{
    const int64_t ntiles = p.tile_end - p.tile_begin;
    if (ntiles <= 0) return hipSuccess;
    if (p.ss.S == 1) return launch_tile_t<1>(p, ntiles, stream);
    if (p.ss.S <= 4) return launch_tile_t<4>(p, ntiles, stream);
    return launch_tile_t<MAX_STREAMS>(p, ntiles, stream);
}

}  // namespace mag
