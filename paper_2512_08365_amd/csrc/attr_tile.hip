// attr_tile.hip -- per-interval energy attribution on gfx950.
//
// The power trace is cut into tiles of T = 64 * C sample segments
// [t_j, t_{j+1}].  One wave (a 64-lane workgroup) owns one tile at a time and
// walks a contiguous run of tiles, carrying one cursor per interval stream (the
// number of that stream's interval endpoints at or before the tile's start).
// Nothing needs a workgroup barrier: lanes exchange data through wave-private
// LDS, ballots and DPP, so many independent waves per CU hide each other's
// memory and LDS latency.
//
// Work inside a tile:
//   samples   lane k owns segments kC .. kC+C-1: segment energies
//             S_j = (P_j + P_{j+1}) (t_{j+1} - t_j) / 2, the input checks, and
//             the tile-local prefix F_i = S_0 + ... + S_{i-1} (a per-lane
//             running sum plus a DPP scan of the lane totals), staged in LDS
//             with the samples;
//   endpoints one lane per endpoint of the round: its segment j (guessed from
//             the mean spacing, checked, binary search as the fallback), which
//             is also its sample index; the interpolated power P^(x); the
//             pieces of segment j left and right of x; its position in the
//             time order of all streams (the endpoints in earlier segments,
//             from a count histogram over the tile's segments, plus those of
//             its own segment ordered before it by direct comparison: a
//             segment index never decreases with x) and, by a scan over the
//             positions of the +1 / -1 each start / end makes, the number of
//             intervals active before it;
//   gaps      the lane of each endpoint integrates the gap from the endpoint
//             before it in time order: within one segment the trapezoid of the
//             two interpolated values; otherwise the right piece of the earlier
//             endpoint + the whole segments between (a difference of two
//             tile-local prefixes) + its own left piece; divided by the number
//             of active intervals (equal split);
//   intervals the lane of each interval's start sums the gap values up to the
//             interval's end.
// Every energy is a sum of non-negative terms.  The one difference taken, of
// two tile-local prefixes for the whole segments inside a gap, carries an
// absolute error of at most about 31 u F (u the unit roundoff, F the prefix,
// at most the tile's energy); when the difference is smaller than F / 2^14
// the whole segments are summed directly instead, so the relative error of a
// gap stays below 6e-11.
//
// A round takes at most 63 endpoints: every stream's endpoints in the tile
// when they fit, otherwise a time prefix of them; one lane is left for the
// gap from the round's last endpoint to the tile's end.
//
// Intervals whose endpoints lie in different tiles leave partial energies:
// head[a][b], the piece in tile b of stream a's interval active at the tile's
// start, and tail[a][b], the piece of the interval started in tile b and still
// active at its end; k_cross adds them in tile order (attr_fix.hip).

#include <hip/hip_ext.h>

#include <algorithm>
#include <stdlib.h>

#include "mag_internal.hpp"

namespace mag {

namespace {

constexpr int WAVE = 64;
constexpr int C = SEG_PER_THREAD;
constexpr int T = TILE;
constexpr int NCOL = WAVE + 1;  // sample columns: the tile's last sample is row 0, column 64
constexpr int WIN = 2 * WAVE;   // window entries, two per lane
constexpr int SLOTS = WAVE - 1; // endpoints per round
constexpr int64_t RUN_TILES = 16;  // most tiles one workgroup walks
static_assert(T == WAVE * C && C == 8, "tile layout");

__device__ __forceinline__ double endpoint_x(const double* s, const double* e, int64_t off,
                                             int64_t q)
{
    // endpoint q of a stream: even q = start of interval q/2, odd q = its end
    const int64_t i = off + (q >> 1);
    return (q & 1) ? e[i] : s[i];
}

// the address of endpoint q of a stream whose starts begin at byte address
// base (its ends at base + e_minus_s): s[i] for even q, e[i] for odd q, i = q/2.
// Selecting between the arrays is a mask of the byte distance between them,
// so no per-lane choice between two pointers is made
__device__ __forceinline__ uint64_t endpoint_addr(uint64_t base, int64_t e_minus_s, int64_t q)
{
    const uint32_t odd = 0u - ((uint32_t)q & 1u);  // all ones for an end
    const uint64_t d = (uint64_t)e_minus_s;
    const uint64_t dsel = ((uint64_t)((uint32_t)(d >> 32) & odd) << 32) | ((uint32_t)d & odd);
    return base + (((uint64_t)q << 2) & ~(uint64_t)7) + dsel;  // + 8 (q / 2) for q >= 0
}

// the kernel's arguments, read from the kernel-argument segment where used
// (scalar loads through the constant cache; the compiler keeps or reloads
// them as scalar-register pressure allows)
typedef const __attribute__((address_space(4))) TileParams* KArgs;
// 1/d for d >= 0 (zero gives +inf) within about an ulp: the hardware
// estimate refined by two Newton steps, far cheaper than a correctly rounded
// division; the quotients it serves (an interpolation weight, an equal share)
// need no more
__device__ __forceinline__ double recip(double d)
{
    double r = __builtin_amdgcn_rcp(d);
    double e = fma(-d, r, 1.0);
    r = fma(r, e, r);
    e = fma(-d, r, 1.0);
    r = fma(r, e, r);
    return (d > 0.0) ? r : INFINITY;
}

// the value of a window entry past the end of its stream
__device__ const double kPastEnd = INFINITY;

// a global-memory pointer argument held in scalar registers, opaque to the
// compiler: a per-lane choice between two such pointers (both taken first,
// outside the choice) stays a register select instead of becoming a per-lane
// load of the chosen argument or a branch
template <class T>
using gptr = __attribute__((address_space(1))) T*;

template <class T>
__device__ __forceinline__ gptr<T> sreg(T* v)
{
    asm volatile("" : "+s"(v));
    return (gptr<T>)v;
}

__device__ __forceinline__ KArgs kargs()
{
    return (KArgs)__builtin_amdgcn_kernarg_segment_ptr();
}

// lanes of one wave communicate through LDS without s_barrier: a wave's LDS
// operations complete in program order; the fences keep the compiler from
// moving memory operations across this point
__device__ __forceinline__ void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// DPP lane moves (bound_ctrl: lanes without a source read 0)
constexpr int DPP_ROW_SHR1 = 0x111, DPP_ROW_SHR2 = 0x112, DPP_ROW_SHR4 = 0x114,
              DPP_ROW_SHR8 = 0x118, DPP_ROW_BCAST15 = 0x142, DPP_ROW_BCAST31 = 0x143,
              DPP_WAVE_SHR1 = 0x138, DPP_WAVE_SHL1 = 0x130;

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

template <int CTRL, int ROWS>
__device__ __forceinline__ float dpp_f32(float v)
{
    return __int_as_float(dpp_i32<CTRL, ROWS>(__float_as_int(v)));
}

// inclusive scan of a non-negative double over the 64 lanes
__device__ __forceinline__ double scan_wave(double x)
{
    x += dpp_f64<DPP_ROW_SHR1, 0xf>(x);
    x += dpp_f64<DPP_ROW_SHR2, 0xf>(x);
    x += dpp_f64<DPP_ROW_SHR4, 0xf>(x);
    x += dpp_f64<DPP_ROW_SHR8, 0xf>(x);
    x += dpp_f64<DPP_ROW_BCAST15, 0xa>(x);
    x += dpp_f64<DPP_ROW_BCAST31, 0xc>(x);
    return x;
}

__device__ __forceinline__ double wave_sum(double v)
{
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    return v;
}

__device__ __forceinline__ double read_lane_f64(double v, int l)
{
    const uint64_t b = (uint64_t)__double_as_longlong(v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)b, l);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), l);
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// segment energy, one expression for every place that computes it
__device__ __forceinline__ double seg_energy(double ta, double tb, float pa, float pb)
{
    return (((double)pa + (double)pb) * (tb - ta)) * 0.5;
}

}  // namespace

// LDS of one wave
template <int SP>
struct TileLds {
    double2 tF[C][NCOL];  // {t_i, F_i} of local sample i at [i % C][i / C]
    float P[C][NCOL];
    // endpoint window: stream a's entry r at a * WS + r; once every slot lane
    // has read its entry, the segment histogram of the merge (16-bit counts,
    // then prefixes, two per word); once the round's merged positions are
    // known, entry p of the round in time order leaves its x at wx[p] and the
    // piece right of it at wx[64 + p] for the entry after it, and then wx[g]
    // holds the value of gap g (ending at entry g): its energy per active
    // interval
    double wx[WIN];
    // F at the end of the segment of the round's entry p (during the merge:
    // the x of entries sharing a segment)
    double F1[WAVE];
    // inv[p]: the entry's (segment + 1) | (1 + the change it makes to the
    // number of active intervals) << 16 | (its lane) << 24; before the merge
    // (more than 8 streams), inv[l] marks the round slot l of a stream's first
    // endpoint: (stream + 1) << 8 | l; during the merge, the (stream, rank) of
    // entries sharing a segment
    int inv[WAVE];
};

namespace {

__device__ __forceinline__ int bperm(int v, int src)
{
    return __builtin_amdgcn_ds_bpermute(src << 2, v);
}
__device__ __forceinline__ int64_t bperm64(int64_t v, int src)
{
    const uint32_t lo = (uint32_t)bperm((int)(uint32_t)v, src);
    const uint32_t hi = (uint32_t)bperm((int)(uint32_t)((uint64_t)v >> 32), src);
    return (int64_t)(((uint64_t)hi << 32) | lo);
}
__device__ __forceinline__ double bpermf(double v, int src)
{
    return __longlong_as_double(bperm64(__double_as_longlong(v), src));
}

// inclusive scans of non-negative ints over the 64 lanes
__device__ __forceinline__ int scan_add_i32(int x)
{
    x += dpp_i32<DPP_ROW_SHR1, 0xf>(x);
    x += dpp_i32<DPP_ROW_SHR2, 0xf>(x);
    x += dpp_i32<DPP_ROW_SHR4, 0xf>(x);
    x += dpp_i32<DPP_ROW_SHR8, 0xf>(x);
    x += dpp_i32<DPP_ROW_BCAST15, 0xa>(x);
    x += dpp_i32<DPP_ROW_BCAST31, 0xc>(x);
    return x;
}
__device__ __forceinline__ int scan_max_i32(int x)
{
    x = max(x, dpp_i32<DPP_ROW_SHR1, 0xf>(x));
    x = max(x, dpp_i32<DPP_ROW_SHR2, 0xf>(x));
    x = max(x, dpp_i32<DPP_ROW_SHR4, 0xf>(x));
    x = max(x, dpp_i32<DPP_ROW_SHR8, 0xf>(x));
    x = max(x, dpp_i32<DPP_ROW_BCAST15, 0xa>(x));
    x = max(x, dpp_i32<DPP_ROW_BCAST31, 0xc>(x));
    return x;
}
__device__ __forceinline__ double wave_min(double v)
{
    for (int off = 32; off > 0; off >>= 1) v = fmin(v, __shfl_xor(v, off));
    return v;
}

constexpr int log2_exact(int v) { return v <= 1 ? 0 : 1 + log2_exact(v >> 1); }

}  // namespace

namespace {

// the samples of one tile in registers (lane k: local samples kC .. kC+C).
// A whole tile of a 16-byte aligned trace is fetched one tile ahead and kept
// in the vectors the loads produce until it is processed (unpacking them
// earlier would wait for the loads right after their issue); a short tile or
// an unaligned trace is read when its tile starts.
struct SampleRegs {
    double2 pt[C / 2];
    float4 pp[C / 4];
    double ptl;  // local sample kC + C: the next lane's first (lane 63: the tile's last)
    float ppl;
};

__device__ __forceinline__ bool vector_tile(int b)
{
    const KArgs k = kargs();
    return k->aligned16 && (int64_t)b * T + T <= k->nseg;
}

__device__ __forceinline__ void sample_prefetch(SampleRegs& r, int b, int lane)
{
    const KArgs k = kargs();
    const int64_t g = (int64_t)b * T + (int64_t)lane * C - k->base;
    const double2* t2 = reinterpret_cast<const double2*>(k->t + g);
    const float4* P4 = reinterpret_cast<const float4*>(k->P + g);
#pragma unroll
    for (int u = 0; u < C / 2; ++u) r.pt[u] = t2[u];
#pragma unroll
    for (int u = 0; u < C / 4; ++u) r.pp[u] = P4[u];
    r.ptl = k->t[g + C];
    r.ppl = k->P[g + C];
}

// checks, segment energies S_j = (P_j + P_{j+1}) (t_{j+1} - t_j) / 2 and the
// tile-local prefix F (a per-lane running sum plus a DPP scan of the lane
// totals) of tile b (L segments), staged in LDS as {t, F} and P; returns the
// tile's energy (uniform)
// NC = NCOL: the tile's last sample (local index T of a whole tile) goes to
// column 64 of row 0; NC = WAVE: the arrays hold local samples 0 .. T - 1 only
// and the last sample's time and power are returned in t_end / p_end (its F is
// the returned total)
template <int NC>
__device__ __forceinline__ double sample_stage(const SampleRegs& r, int b, int L, int lane,
                                               double2 (*tF)[NC], float (*Pl)[NC],
                                               unsigned& err, double& t_end, float& p_end)
{
    const KArgs kk = kargs();
    const int64_t j0 = (int64_t)b * T;
    const int cs = min(max(L - lane * C, 0), C);  // segments of this lane
    const bool full = vector_tile(b);             // uniform: every lane has C segments
    double tv[C + 1];
    float pv[C + 1];
    if (full) {
#pragma unroll
        for (int u = 0; u < C / 2; ++u) {
            tv[2 * u] = r.pt[u].x;
            tv[2 * u + 1] = r.pt[u].y;
        }
#pragma unroll
        for (int u = 0; u < C / 4; ++u) {
            pv[4 * u] = r.pp[u].x;
            pv[4 * u + 1] = r.pp[u].y;
            pv[4 * u + 2] = r.pp[u].z;
            pv[4 * u + 3] = r.pp[u].w;
        }
        tv[C] = r.ptl;
        pv[C] = r.ppl;
    } else {
        // a lane past the tile's last sample repeats the last one it has with
        // zero power: missing segments have zero width and energy
        const int64_t g = j0 + (int64_t)lane * C - kk->base;
        const int have = min(max(L - lane * C, -1), C);  // last local sample of the lane
        double tl = 0.0;
#pragma unroll
        for (int u = 0; u <= C; ++u) {
            tv[u] = (u <= have) ? kk->t[g + u] : tl;
            pv[u] = (u <= have) ? kk->P[g + u] : 0.0f;
            tl = tv[u];
        }
    }
    if (kk->validate) {
        // every segment of the lane rises (the repeated last time of a short
        // lane does not), and a strictly increasing run whose ends are finite
        // is finite throughout (a NaN fails every comparison).  The checks
        // are collected as wave masks: the error bits are the wave's anyway
        uint64_t tbad = __ballot(!(fabs(tv[0]) < INFINITY) || !(fabs(tv[C]) < INFINITY));
        if (full) {
#pragma unroll
            for (int u = 0; u < C; ++u) tbad |= __ballot(!(tv[u + 1] > tv[u]));
        } else {
            // rising as a positive difference (the same predicate, written
            // apart from the whole-tile form above)
            int rising = 0;
#pragma unroll
            for (int u = 0; u < C; ++u) rising += (tv[u + 1] - tv[u] > 0.0) ? 1 : 0;
            tbad |= __ballot(rising != cs);
        }
        uint64_t pbad = 0;
#pragma unroll
        for (int u = 0; u <= C; ++u) pbad |= __ballot(!((pv[u] >= 0.0f) & (pv[u] < INFINITY)));
        err |= (tbad ? ERR_TIMESTAMPS : 0u) | (pbad ? ERR_POWER : 0u);
    }
    double f[C + 1];
    f[0] = 0.0;
#pragma unroll
    for (int u = 0; u < C; ++u) f[u + 1] = f[u] + seg_energy(tv[u], tv[u + 1], pv[u], pv[u + 1]);
    const double incl = scan_wave(f[C]);
    // F at the lane's first sample: the exclusive scan (lane 0 reads 0)
    const double base = dpp_f64<DPP_WAVE_SHR1, 0xf>(incl);
#pragma unroll
    for (int u = 0; u < C; ++u) {
        tF[u][lane] = make_double2(tv[u], base + f[u]);
        Pl[u][lane] = pv[u];
    }
    const double Wt = read_lane_f64(incl, WAVE - 1);
    if constexpr (NC > WAVE) {
        if (lane == WAVE - 1) {
            tF[0][WAVE] = make_double2(tv[C], Wt);
            Pl[0][WAVE] = pv[C];
        }
    }
    t_end = read_lane_f64(tv[C], WAVE - 1);
    p_end = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(pv[C]), WAVE - 1));
    return Wt;
}

}  // namespace

// SP: the number of streams rounded up to a power of two (streams S .. SP-1
// are treated as empty).  Lane a < SP holds stream a's state in registers.
template <int SP>
__global__ __launch_bounds__(WAVE) void k_tile(const TileParams p)
{
    constexpr int LSP = log2_exact(SP);
    static_assert((1 << LSP) == SP && SP <= 32, "streams");
    constexpr int LW = 7 - LSP;  // window entries per stream: WS = 2^LW
    constexpr int WS = 1 << LW;
    constexpr int B = (SLOTS >> LSP) > 0 ? (SLOTS >> LSP) : 1;  // per-stream share of a cut round
    __shared__ TileLds<SP> sm;
    const int lane = threadIdx.x;
    const int S = p.ss.S;
    // tile indices fit 32 bits (the host caps the trace length)
    const int b0 = (int)p.tile_begin + (int)blockIdx.x * (int)p.tiles_per_wg;
    const int b1 = min(b0 + (int)p.tiles_per_wg, (int)p.tile_end);
    if (b0 >= b1) return;

    // ---- stream lanes: offsets, lengths, cursors
    const bool slane = lane < S;
    const int64_t soff = slane ? p.ss.off[lane] : 0;
    const int64_t slen = slane ? 2 * (p.ss.off[lane + 1] - p.ss.off[lane]) : 0;
    int64_t sq = 0;            // endpoints of the stream consumed so far
    double slastx = -INFINITY; // the stream's last consumed endpoint
    double sacc = 0.0;         // this tile's energy of the stream's open interval so far
    int sstarted = 0;          // the open interval started in this tile
    {
        // cursor at the first tile: endpoints <= its start time.  Every stream
        // is searched at once, each by its own group of GS = 64 / SP lanes (a
        // GS-ary search: one dependent load per level for all streams)
        constexpr int GS = WAVE / SP;
        const int ga = lane / GS, gl = lane % GS;  // the lane's stream and rank in its group
        const double tau0 = p.t[(int64_t)b0 * T - p.base];
        const int64_t goff = (ga < S) ? p.ss.off[ga] : 0;
        int64_t lo = 0, hi = (ga < S) ? 2 * (p.ss.off[ga + 1] - goff) : 0;
        const uint64_t gmask = (GS == WAVE) ? ~0ull : ((1ull << (GS & 63)) - 1ull);
        for (;;) {
            const bool wide = hi - lo > GS;
            if (__ballot(wide) == 0ull) break;
            const int64_t step = wide ? (hi - lo + GS - 1) / GS : 1;
            const int64_t pr = lo + (int64_t)(gl + 1) * step - 1;
            const bool ok = wide && (pr < hi) && (endpoint_x(p.s, p.e, goff, pr) <= tau0);
            const int c = __popcll((__ballot(ok) >> (ga * GS)) & gmask);
            if (wide) {
                const int64_t nlo = lo + (int64_t)c * step;
                const int64_t nhi = min(hi, lo + (int64_t)(c + 1) * step - 1);
                lo = min(nlo, hi);
                hi = max(nhi, lo);
            }
        }
        const int64_t pr = lo + gl;
        const bool ok = (pr < hi) && (endpoint_x(p.s, p.e, goff, pr) <= tau0);
        const int64_t q = lo + __popcll((__ballot(ok) >> (ga * GS)) & gmask);
        // stream lane a takes group a's cursor, and the endpoint before it
        const int64_t qa = bperm64(q, min(lane, SP - 1) * GS);
        if (slane) {
            sq = qa;
            slastx = (qa > 0) ? endpoint_x(p.s, p.e, soff, qa - 1) : -INFINITY;
        }
    }

    // the lane's two window entries: stream, rank, and that stream's extent
    const int wa0 = lane >> LW, wa1 = (lane + WAVE) >> LW;
    const int wr0 = lane & (WS - 1), wr1 = (lane + WAVE) & (WS - 1);
    // byte address of the stream's first start (its ends lie e_minus_s further)
    const int64_t e_minus_s = (int64_t)((const char*)p.e - (const char*)p.s);
    const uint64_t wbase0 = (uint64_t)p.s + 8 * (uint64_t)bperm64(soff, wa0);
    const uint64_t wbase1 = (uint64_t)p.s + 8 * (uint64_t)bperm64(soff, wa1);
    const int64_t wlen0 = bperm64(slen, wa0), wlen1 = bperm64(slen, wa1);
    // window entry of rank r from cursor cur (+inf past the stream's end); `more`:
    // the last entry of the stream's window, with endpoints after it
    auto wload = [&](int64_t cur, int r, uint64_t base, int64_t len, bool& more) -> double {
        const int64_t q = cur + r;
        more = (r == WS - 1) && (q + 1 < len);
        // an entry past the stream's end reads +inf from device memory, so the
        // value needs no select after its load and is first waited for where
        // it is used
        const gptr<const double> ptr = (q < len)
            ? (gptr<const double>)endpoint_addr(base, e_minus_s, q)
            : (gptr<const double>)&kPastEnd;
        return *ptr;
    };
    bool em0, em1;  // `more` flags of the prefetched window
    double ew0 = wload(bperm64(sq, wa0), wr0, wbase0, wlen0, em0);
    double ew1 = wload(bperm64(sq, wa1), wr1, wbase1, wlen1, em1);

    SampleRegs sr;
    if (vector_tile(b0)) sample_prefetch(sr, b0, lane);
    // Outputs are written one round late, right after the next round's window
    // has arrived: loads complete in issue order, so a store issued between a
    // load and its use would make the use wait for the store as well.  Null:
    // nothing pending.
    gptr<int64_t> pend_idx = nullptr;  // the lane's endpoint index
    int64_t pend_idx_v = 0;
    gptr<double> pend_en = nullptr;    // an interval's energy, or a piece of it
    double pend_en_v = 0.0;
    gptr<int64_t> pend_cnt = nullptr;  // a stream's cursor at a tile's start
    int64_t pend_cnt_v = 0;
    gptr<double> pend_piece = nullptr; // a stream's open-interval piece of a tile
    double pend_piece_v = 0.0;
    auto flush = [&]() {
        if (pend_idx) *pend_idx = pend_idx_v;
        if (pend_en) *pend_en = pend_en_v;
        if (pend_cnt) *pend_cnt = pend_cnt_v;
        if (pend_piece) *pend_piece = pend_piece_v;
        pend_idx = nullptr;
        pend_en = nullptr;
        pend_cnt = nullptr;
        pend_piece = nullptr;
    };
    unsigned err = 0u;
    double idle = 0.0;    // this lane's share of the idle energy
    double w_wave = 0.0;  // the wave's trace energy (uniform)
    // 1 / lane: the equal share of a gap among mp active intervals is read
    // from lane mp (mp <= S < 64)
    const double inv_lane = (lane > 0) ? 1.0 / (double)lane : 0.0;

    for (int b = b0; b < b1; ++b) {
        const KArgs kk = kargs();
        const int64_t j0 = (int64_t)b * T;
        const int L = (int)min((int64_t)T, kk->nseg - j0);

        // ---- samples: checks, segment energies, tile-local prefix, staging
        double t_end_unused;
        float p_end_unused;
        w_wave += sample_stage(sr, b, L, lane, sm.tF, sm.P, err, t_end_unused, p_end_unused);
        if (slane) {
            pend_cnt = sreg(kk->cnt) + ((int64_t)lane * (kk->ld + 1) + b);
            pend_cnt_v = sq;
        }
        sacc = 0.0;
        sstarted = 0;
        wave_sync();
        auto tF_at = [&](int i) -> double2 { return sm.tF[i & (C - 1)][i >> 3]; };
        auto t_at = [&](int i) -> double { return sm.tF[i & (C - 1)][i >> 3].x; };
        auto P_at = [&](int i) -> double { return (double)sm.P[i & (C - 1)][i >> 3]; };
        const double t_begin = t_at(0);
        const double tau_end = t_at(L);
        const double inv_dt = (double)L * recip(tau_end - t_begin);
        // the point the round starts from (uniform): the tile's first sample,
        // later the previous round's last endpoint -- x, the piece from x to the
        // end of its segment, F at that end, (segment + 1) | active after << 16
        double rs_x = t_begin, rs_right = 0.0, rs_Fn = 0.0;
        int rs_jm = __popcll(__ballot((sq & 1) != 0)) << 16;

        bool first_round = true;
        for (;;) {
            // ---- the round's endpoints: a prefix of every stream's window
            const double xw0 = ew0, xw1 = ew1;
            sm.wx[lane] = xw0;
            sm.wx[lane + WAVE] = xw1;
            flush();  // the previous round's outputs, now that the window is here
            if (SP > 8) sm.inv[lane] = 0;  // no slot marked
            const uint64_t in0 = __ballot(xw0 <= tau_end), in1 = __ballot(xw1 <= tau_end);
            // samples of the next tile, in flight during this tile's rounds;
            // issued after the window is read, so that the wait for the window
            // loads does not wait for them (loads complete in issue order)
            if (first_round && b + 1 < b1 && vector_tile(b + 1)) sample_prefetch(sr, b + 1, lane);
            first_round = false;
            const uint64_t mo0 = __ballot(em0), mo1 = __ballot(em1);
            const int tot = __popcll(in0) + __popcll(in1);
            // stream lane a: its entries are bits [a WS, (a + 1) WS) of a 128-bit mask
            auto sbits = [&](uint64_t m0w, uint64_t m1w) -> int {
                if (WS == 2 * WAVE) return __popcll(m0w) + __popcll(m1w);
                const uint64_t w = (lane * WS >= WAVE) ? m1w : m0w;
                if (WS == WAVE) return __popcll(w);
                return __popcll((w >> ((lane * WS) & (WAVE - 1))) & ((1ull << (WS & 63)) - 1ull));
            };
            const int ka = (lane < SP) ? sbits(in0, in1) : 0;
            const bool smore = (lane < SP) && (sbits(mo0, mo1) != 0);
            const bool over = __ballot(ka == WS && smore) != 0ull;
            const bool fin = !over && tot <= SLOTS;
            wave_sync();
            int ta = ka;
            if (!fin) {
                // time prefix: each stream keeps at most B endpoints; the round
                // ends at the earliest time a stream runs out of its share
                const double cv = sm.wx[(min(lane, SP - 1) << LW) + B - 1];
                const double cut = wave_min((lane < SP && ka > B) ? cv : INFINITY);
                const uint64_t tk0 = in0 & __ballot(xw0 <= cut);
                const uint64_t tk1 = in1 & __ballot(xw1 <= cut);
                ta = (lane < SP) ? min(sbits(tk0, tk1), B) : 0;  // endpoints equal to the cut may wait
                if (__ballot(ta > 0) == 0ull) {
                    // only with unsorted or non-finite endpoints: force progress
                    ta = min(ka, B);
                    err |= ERR_INTERVAL;
                }
            }
            const int incl = scan_add_i32(ta);
            const int fa = incl - ta;
            const int Er = __builtin_amdgcn_readlane(incl, WAVE - 1);
            const int G = Er + (fin ? 1 : 0);  // gaps of the round
            if (SP > 8 && lane < SP && ta > 0) sm.inv[fa] = ((lane + 1) << 8) | fa;
            wave_sync();
            // the next round's window (this tile's next round, or the next
            // tile's first): both start at the cursors after this round
            const int64_t sqn = sq + ta;
            ew0 = wload(bperm64(sqn, wa0), wr0, wbase0, wlen0, em0);
            ew1 = wload(bperm64(sqn, wa1), wr1, wbase1, wlen1, em1);

            // ---- round slot of this lane: stream my_a, rank my_r (lane Er: the tile's end)
            const bool real = lane < Er;
            const bool pend = fin && lane == Er;
            const bool has_gap = real || pend;
            int my_a = 0, my_r = 0;
            if (SP <= 8) {
                // the stream of slot l is the last one whose first slot is <= l
                int a_l = 0, f_l = 0;
#pragma unroll
                for (int a = 1; a < SP; ++a) {
                    const int f = __builtin_amdgcn_readlane(fa, a);
                    const bool in = f <= lane;
                    a_l += in ? 1 : 0;
                    f_l = in ? f : f_l;
                }
                if (real) {
                    my_a = a_l;
                    my_r = lane - f_l;
                }
            } else {
                // each stream marked its first slot; a max-scan spreads the marks
                const int mkv = scan_max_i32(sm.inv[lane]);
                if (real) {
                    my_a = (mkv >> 8) - 1;
                    my_r = lane - (mkv & 255);
                }
            }
            const int64_t q = bperm64(sq, my_a) + my_r;
            const int64_t off_a = bperm64(soff, my_a);
            const int ta_a = bperm(ta, my_a);
            const double acc_a = bpermf(sacc, my_a);
            const int st_a = bperm(sstarted, my_a);
            const double lx_a = bpermf(slastx, my_a);
            const double x = real ? sm.wx[(my_a << LW) + my_r] : tau_end;
            const double xp = (my_r > 0) ? sm.wx[(my_a << LW) + max(my_r - 1, 0)] : lx_a;

            // ---- segment j: t_j < x <= t_{j+1}; sample index j0 + j + 1
            int j;
            {
                const int jg = (int)fmin(fmax((x - t_begin) * inv_dt, 0.0), (double)(L - 1));
                const int c0 = max(0, min(jg - 1, L - 3));
                const double u0 = t_at(c0), u1 = t_at(min(c0 + 1, L)), u2 = t_at(min(c0 + 2, L)),
                             u3 = t_at(min(c0 + 3, L));
                j = (u0 < x && x <= u1) ? c0
                  : (c0 + 1 < L && u1 < x && x <= u2) ? c0 + 1
                  : (c0 + 2 < L && u2 < x && x <= u3) ? c0 + 2 : -1;
                if (!real) j = L;
            }
            if (__ballot(j < 0) != 0ull) {
                if (j < 0) {
                    // first sample index >= x (x > t_0 of the tile for sorted input)
                    int lo = 0, hi = L;
                    while (lo < hi) {
                        const int mid = (lo + hi) >> 1;
                        if (t_at(mid) < x) lo = mid + 1; else hi = mid;
                    }
                    j = min(max(lo, 1), L) - 1;
                }
            }
            const double2 A0 = tF_at(j), A1 = tF_at(min(j + 1, L));
            const double pj = P_at(j), pj1 = P_at(min(j + 1, L));
            // interpolated power and the pieces of segment j left and right of x
            const double rh = recip(A1.x - A0.x);
            auto lerp = [&](double y) -> double {
                return (y == A1.x) ? pj1 : pj + (pj1 - pj) * ((y - A0.x) * rh);
            };
            const double ph = real ? lerp(x) : pj;
            const double left = real ? ((pj + ph) * (x - A0.x)) * 0.5 : 0.0;
            const double right = real ? ((ph + pj1) * (A1.x - x)) * 0.5 : 0.0;
            const double Fj = A0.y;  // prefix at the start of segment j (the tile's end: F_L)

            const int64_t gid = off_a + (q >> 1);
            if (real) {
                const KArgs k = kargs();
                const gptr<int64_t> ie = sreg(k->end_idx), is = sreg(k->start_idx);
                const gptr<int64_t> idx = (q & 1) ? ie : is;
                pend_idx = idx ? idx + gid : nullptr;
                pend_idx_v = j0 + j + 1;
            }
            // finite and not before the stream's previous endpoint
            if (real && kk->validate && (!(fabs(x) < INFINITY) || !(xp <= x))) err |= ERR_INTERVAL;

            // ---- merged position: the round's entries in the order of (x, stream,
            // rank).  A count histogram over the tile's segments (16-bit counts,
            // two per word, in the window's LDS, which every slot lane has read)
            // gives each entry the number of entries in earlier segments (a
            // segment index never decreases with x); the few entries that share
            // a segment order themselves by direct comparison.
            int pos = lane;
            {
                uint32_t* hist = reinterpret_cast<uint32_t*>(sm.wx);  // bin i: half i & 1 of word i >> 1
                static_assert(sizeof(sm.wx) >= T * 2, "segment histogram fits the window");
                wave_sync();  // every lane's reads of the window are done
                reinterpret_cast<uint4*>(hist)[lane] = make_uint4(0u, 0u, 0u, 0u);
                const int jj = real ? j : 0;  // the bin of a real entry (j < L <= T)
                const int sh = 16 * (jj & 1);
                uint32_t old = 0u;
                wave_sync();
                if (real) old = atomicAdd(&hist[jj >> 1], 1u << sh);
                wave_sync();
                // exclusive prefix over the bins: lane l holds bins 8l .. 8l + 7
                const uint4 hw = reinterpret_cast<const uint4*>(hist)[lane];
                const uint32_t hv[4] = {hw.x, hw.y, hw.z, hw.w};
                int run = 0;
                uint32_t pw[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int c0 = (int)(hv[u] & 0xffffu), c1 = (int)(hv[u] >> 16);
                    pw[u] = (uint32_t)run | ((uint32_t)(run + c0) << 16);
                    run += c0 + c1;
                }
                const int base = scan_add_i32(run) - run;
                const uint32_t badd = (uint32_t)base | ((uint32_t)base << 16);
                reinterpret_cast<uint4*>(hist)[lane] =
                    make_uint4(pw[0] + badd, pw[1] + badd, pw[2] + badd, pw[3] + badd);
                wave_sync();
                // entries before my segment, and in it (the next bin's prefix, or
                // the round's count after the last bin)
                const int before = (int)((hist[jj >> 1] >> sh) & 0xffffu);
                const int jn = min(jj + 1, T - 1);
                const int after = (jj + 1 < T) ? (int)((hist[jn >> 1] >> (16 * (jn & 1))) & 0xffffu) : Er;
                const int kj = after - before;
                const int o = (int)((old >> sh) & 0xffffu);  // arrival order within the segment
                const bool coll = real && kj > 1;
                int w = 0;
                if (__ballot(coll) != 0ull) {
                    // the segment's entries leave x and (stream, rank) at
                    // [before, after) of two scratch arrays, then count those
                    // ordered before them
                    const int key = (my_a << 8) | my_r;
                    if (coll) {
                        sm.F1[before + o] = x;
                        sm.inv[before + o] = key;
                    }
                    wave_sync();
                    for (int i = 0; __ballot(coll && i < kj) != 0ull; ++i) {
                        if (coll && i < kj && i != o) {
                            const double y = sm.F1[before + i];
                            const int ky = sm.inv[before + i];
                            w += (y < x || (y == x && ky < key)) ? 1 : 0;
                        }
                    }
                    wave_sync();
                }
                if (real) pos = before + w;
            }
            // the entry's segment, and the change it makes to the number of active
            // intervals (+1 a start, -1 an end, 0 the round's end) offset by 1
            const int jd = (j + 1) | ((real ? ((q & 1) ? 0 : 2) : 1) << 16);
            // each entry leaves what the entry after it in time order needs at
            // its position (the merge's reads of LDS are done: a wave's LDS
            // operations complete in order)
            if (has_gap) {
                sm.wx[pos] = x;
                sm.wx[WAVE + pos] = right;
                sm.F1[pos] = A1.y;
                sm.inv[pos] = jd | (lane << 24);
            }
            wave_sync();
            // intervals active after each position: the round's starting count
            // plus a scan of the changes in time order (lane l: position l)
            const int dl = (lane < G) ? (int)((sm.inv[lane] >> 16) & 0xff) - 1 : 0;
            const int dincl = scan_add_i32(dl);
            const int m0 = rs_jm >> 16;  // active at the round's start
            // active in the gap ending at this lane's entry: after the position before it
            const int m_gap = m0 + bperm(dincl - dl, pos);

            // ---- gap ending at this lane's entry (from the entry before it)
            double v;
            {
                // the entry before: the one at the position before, or the
                // round's starting point
                const int pp = max(pos - 1, 0);
                const double px = sm.wx[pp], pr = sm.wx[WAVE + pp], pF = sm.F1[pp];
                const int pjm = sm.inv[pp] & 0xffffff;
                const bool head_gap = (pos == 0);
                const double xpv = head_gap ? rs_x : px;
                const double pright = head_gap ? rs_right : pr;
                const double pFn = head_gap ? rs_Fn : pF;
                const int pe = head_gap ? rs_jm : pjm;
                const int pjx = (pe & 0xffff) - 1;  // segment of the entry before
                const bool same = (pjx == j);
                // both in segment j: the trapezoid of the two interpolated values
                const double q_in = ((lerp(xpv) + ph) * (x - xpv)) * 0.5;
                double whole = fmax(Fj - pFn, 0.0);
                const bool ill = has_gap && !same && (j >= pjx + 2) && (whole < Fj * 0x1p-14);
                if (__ballot(ill) != 0ull) {
                    if (ill) {
                        // the whole segments summed directly
                        double sum = 0.0;
                        for (int i = pjx + 1; i < j; ++i)
                            sum += seg_energy(t_at(i), t_at(i + 1), sm.P[i & 7][i >> 3],
                                              sm.P[(i + 1) & 7][(i + 1) >> 3]);
                        whole = sum;
                    }
                }
                const double Q = same ? q_in : (pright + whole) + left;
                const int mp = m_gap;
                // read with every lane active: a lane that is switched off
                // cannot be read across lanes
                const double inv_mp = bpermf(inv_lane, mp);
                v = (has_gap && mp > 0) ? (kk->split ? Q * inv_mp : Q) : 0.0;
                idle += (has_gap && mp == 0) ? Q : 0.0;
                if (has_gap) sm.wx[pos] = v;
            }
            wave_sync();

            // ---- interval energies: intervals starting in the round sum their
            // gaps; the interval a stream carried into the round ends at its first
            const int pos_next = dpp_i32<DPP_WAVE_SHL1, 0xf>(pos);
            const bool start = real && !(q & 1);
            const bool closes = start && (my_r + 1 < ta_a);
            const bool carried = real && (q & 1) && my_r == 0;
            const int lo = start ? pos + 1 : 0;
            const int hi = start ? (closes ? pos_next : G - 1) : (carried ? pos : -1);
            // gaps [lo, hi] summed as a difference of the round's prefix over
            // positions (lane l holds the gap ending at position l).  The
            // difference carries about 12 ulp of the prefix in rounding error;
            // where it is below 2^-16 of the prefix (that error could reach
            // 1e-10 of it) the gaps are added directly instead
            const double gl = (lane < G) ? sm.wx[lane] : 0.0;
            const double gpre = scan_wave(gl);
            const double g_hi = bpermf(gpre, max(hi, 0));
            const double g_lo = bpermf(gpre, max(lo - 1, 0));
            double acc = (hi < lo) ? 0.0 : g_hi - ((lo > 0) ? g_lo : 0.0);
            const bool direct = (hi >= lo) && !(acc >= g_hi * 0x1p-16);
            if (__ballot(direct) != 0ull) {
                double d = 0.0;
                for (int i = 0; __ballot(direct && lo + i <= hi) != 0ull; i += 2) {
                    const double y0 = sm.wx[min(lo + i, WAVE - 1)];
                    const double y1 = sm.wx[min(lo + i + 1, WAVE - 1)];
                    d += (lo + i <= hi) ? y0 : 0.0;
                    d += (lo + i + 1 <= hi) ? y1 : 0.0;
                }
                if (direct) acc = d;
            }
            if (closes || carried) {
                const KArgs k = kargs();
                const gptr<double> ph = sreg(k->head), pen = sreg(k->energy);
                pend_en = (carried && !st_a) ? (ph + (int64_t)my_a * k->ld + b) : (pen + gid);
                pend_en_v = carried ? acc_a + acc : acc;
            }
            // energy per active interval over the whole round (streams that stay
            // inside one interval through it)
            const double vall = read_lane_f64(gpre, WAVE - 1);
            // the round's last entry is where the next round starts
            if (!fin) {
                const int ll = __builtin_amdgcn_readfirstlane(sm.inv[Er - 1] >> 24);
                rs_x = read_lane_f64(x, ll);
                rs_right = read_lane_f64(right, ll);
                rs_Fn = read_lane_f64(A1.y, ll);
                rs_jm = (__builtin_amdgcn_readlane(j, ll) + 1) |
                        ((m0 + __builtin_amdgcn_readlane(dincl, WAVE - 1)) << 16);
            }
            // ---- commit the round (stream lanes)
            {
                const int last = max(fa + ta - 1, 0);  // round slot of the stream's last endpoint
                const double acc_l = bpermf(acc, last);
                const double x_l = bpermf(x, last);
                const bool open = (sqn & 1) != 0;
                if (ta > 0) {
                    sacc = open ? acc_l : 0.0;
                    sstarted = open ? 1 : 0;
                    slastx = x_l;
                } else if (sq & 1) {
                    sacc += vall;
                }
                sq = sqn;
            }
            wave_sync();
            if (fin) break;
        }

        // ---- interval still open at the tile's end: its piece of this tile
        if (slane && (sq & 1)) {
            const KArgs k = kargs();
            const gptr<double> pt_ = sreg(k->tail), ph = sreg(k->head);
            pend_piece = (sstarted ? pt_ : ph) + ((int64_t)lane * k->ld + b);
            pend_piece_v = sacc;
        }
    }
    flush();

    // the wave's trace and idle energy, at its first tile (k_fix adds them up:
    // thousands of waves adding into one address would queue at the end)
    const double It = wave_sum(idle);
    const KArgs k = kargs();
    if (lane == 0) k->part[b0] = make_double2(w_wave, It);
    if (slane) {
        // where this wave stopped: the next wave must start there
        const int LD = (int)k->ld;
        k->cnt_fin[(int64_t)lane * (LD + 1) + b1] = sq;
        if (b1 == (int)k->NT) k->cnt[(int64_t)lane * (LD + 1) + b1] = sq;
    }
    if (__ballot(err != 0u)) {
        unsigned e = err;
        for (int off = 32; off > 0; off >>= 1) e |= __shfl_xor(e, off);
        if (lane == 0) atomicOr(&k->status->err, e);
    }
}

// ---------------------------------------------------------------------------
// One stream (sequential intervals): the endpoints of a stream are already in
// time order, so a round needs no merge, no split and no per-round sums: the
// gap ending at an endpoint runs from the endpoint one lane below (the round's
// starting point for lane 0), and it is the energy of one interval (an end
// endpoint: the stream was inside an interval) or idle energy (a start).  The
// lane after the round's last endpoint takes the gap to the tile's end, the
// piece of an interval still open there.  Same outputs as k_tile: energies,
// sample indices, head/tail pieces, per-tile cursors, per-run trace and idle
// energies.
// ---------------------------------------------------------------------------
struct SeqLds {
    // local samples 0 .. T - 1 ({t, F} and P at [i % C][i / C]); a whole
    // tile's last sample (local index T) is kept in uniform registers, so
    // that a wave's LDS is exactly 10 KiB (five 2 KiB allocation blocks:
    // 16 waves per CU instead of 13)
    double2 tF[C][WAVE];
    float P[C][WAVE];
};
static_assert(sizeof(SeqLds) == 10240, "one-stream tile LDS");

__global__ __launch_bounds__(WAVE) void k_tile_seq(const TileParams p)
{
    __shared__ SeqLds sm;
    const int lane = threadIdx.x;
    const int b0 = (int)p.tile_begin + (int)blockIdx.x * (int)p.tiles_per_wg;
    const int b1 = min(b0 + (int)p.tiles_per_wg, (int)p.tile_end);
    if (b0 >= b1) return;
    const int64_t len = 2 * (p.ss.off[1] - p.ss.off[0]);  // endpoints (off[0] = 0)

    // cursor at the first tile: endpoints <= its start time (64-ary search)
    int64_t sq;
    {
        const double tau0 = p.t[(int64_t)b0 * T - p.base];
        int64_t lo = 0, hi = len;
        while (hi - lo > WAVE) {
            const int64_t step = (hi - lo + WAVE - 1) / WAVE;
            const int64_t pr = lo + (int64_t)(lane + 1) * step - 1;
            const bool ok = (pr < hi) && (endpoint_x(p.s, p.e, 0, pr) <= tau0);
            const int c = __popcll(__ballot(ok));
            const int64_t nlo = lo + (int64_t)c * step;
            const int64_t nhi = min(hi, lo + (int64_t)(c + 1) * step - 1);
            lo = min(nlo, hi);
            hi = max(nhi, lo);
        }
        const int64_t pr = lo + lane;
        const bool ok = (pr < hi) && (endpoint_x(p.s, p.e, 0, pr) <= tau0);
        sq = lo + __popcll(__ballot(ok));
    }
    // the stream's last consumed endpoint (uniform)
    double slastx = (sq > 0) ? endpoint_x(p.s, p.e, 0, sq - 1) : -INFINITY;

    // window: lane l holds endpoint sq + l; past the stream's end it reads +inf
    // from device memory, so the value needs no select after its load
    const int64_t e_minus_s = (int64_t)((const char*)p.e - (const char*)p.s);
    auto wload = [&](int64_t cur) -> double {
        const int64_t q = cur + lane;
        const gptr<const double> ptr = (q < len)
            ? (gptr<const double>)endpoint_addr((uint64_t)p.s, e_minus_s, q)
            : (gptr<const double>)&kPastEnd;
        return *ptr;
    };
    double ew = wload(sq);

    SampleRegs sr;
    if (vector_tile(b0)) sample_prefetch(sr, b0, lane);
    unsigned err = 0u;
    double idle = 0.0;    // this lane's share of the idle energy
    double w_wave = 0.0;  // the run's trace energy (uniform)

    for (int b = b0; b < b1; ++b) {
        const KArgs kk = kargs();
        const int64_t j0 = (int64_t)b * T;
        const int L = (int)min((int64_t)T, kk->nseg - j0);
        double tT;  // a whole tile's last sample: time, power and prefix (uniform)
        float pT;
        const double FT = sample_stage(sr, b, L, lane, sm.tF, sm.P, err, tT, pT);
        w_wave += FT;
        if (lane == 0) kk->cnt[b] = sq;
        // the interval open at the tile's start began in an earlier tile
        int started = 0;
        wave_sync();
        // local sample i <= L (i = T only for a whole tile; its column index
        // is wrapped so that the LDS read stays inside the arrays)
        auto tF_at = [&](int i) -> double2 {
            const double2 v = sm.tF[i & (C - 1)][(i >> 3) & (WAVE - 1)];
            return (i == T) ? make_double2(tT, FT) : v;
        };
        auto t_at = [&](int i) -> double {
            const double v = sm.tF[i & (C - 1)][(i >> 3) & (WAVE - 1)].x;
            return (i == T) ? tT : v;
        };
        auto P_at = [&](int i) -> double {
            const float v = sm.P[i & (C - 1)][(i >> 3) & (WAVE - 1)];
            return (double)((i == T) ? pT : v);
        };
        const double t_begin = t_at(0);
        const double tau_end = t_at(L);
        const double inv_dt = (double)L * recip(tau_end - t_begin);
        // where the round starts (uniform): the tile's first sample, later the
        // previous round's last endpoint -- x, its interpolated power, the
        // piece from x to the end of its segment, F at that end, its segment
        double rs_x = t_begin, rs_ph = P_at(0), rs_right = 0.0, rs_Fn = 0.0;
        int rs_j = -1;
        bool first_round = true;
        for (;;) {
            const double xw = ew;
            // the round: the window's leading entries inside the tile (63 at
            // most when they are the tile's last, so that a lane is left for
            // the gap to the tile's end)
            const uint64_t inm = __ballot(xw <= tau_end);
            const int lead = (inm == ~0ull) ? WAVE : (int)__builtin_ctzll(~inm);
            const bool fin = lead < WAVE;
            const int k = lead;
            if (first_round && b + 1 < b1 && vector_tile(b + 1)) sample_prefetch(sr, b + 1, lane);
            first_round = false;
            const int64_t sqn = sq + k;
            ew = wload(sqn);  // the next round's window

            const bool real = lane < k;
            const bool tail_lane = fin && lane == k;
            const int64_t q = sq + lane;  // the tail lane: sqn
            const double x = real ? xw : tau_end;
            // an entry that is neither inside the tile nor after its end is
            // not a number
            if (tail_lane && kk->validate && q < len && !(xw > tau_end)) err |= ERR_INTERVAL;

            // ---- segment j: t_j < x <= t_{j+1}; sample index j0 + j + 1
            int j;
            {
                const int jg = (int)fmin(fmax((x - t_begin) * inv_dt, 0.0), (double)(L - 1));
                const int c0 = max(0, min(jg - 1, L - 3));
                const double u0 = t_at(c0), u1 = t_at(min(c0 + 1, L)), u2 = t_at(min(c0 + 2, L)),
                             u3 = t_at(min(c0 + 3, L));
                j = (u0 < x && x <= u1) ? c0
                  : (c0 + 1 < L && u1 < x && x <= u2) ? c0 + 1
                  : (c0 + 2 < L && u2 < x && x <= u3) ? c0 + 2 : -1;
                if (!real) j = L;
            }
            if (__ballot(j < 0) != 0ull) {
                if (j < 0) {
                    int lo = 0, hi = L;
                    while (lo < hi) {
                        const int mid = (lo + hi) >> 1;
                        if (t_at(mid) < x) lo = mid + 1; else hi = mid;
                    }
                    j = min(max(lo, 1), L) - 1;
                }
            }
            const double2 A0 = tF_at(j), A1 = tF_at(min(j + 1, L));
            const double pj = P_at(j), pj1 = P_at(min(j + 1, L));
            const double rh = recip(A1.x - A0.x);
            const double ph = !real ? pj : (x == A1.x) ? pj1 : pj + (pj1 - pj) * ((x - A0.x) * rh);
            const double left = real ? ((pj + ph) * (x - A0.x)) * 0.5 : 0.0;
            const double right = real ? ((ph + pj1) * (A1.x - x)) * 0.5 : 0.0;
            const double Fj = A0.y;  // prefix at the start of segment j (the tile's end: F_L)
            const int64_t gid = q >> 1;
            if (real) {
                int64_t* idx = (q & 1) ? kk->end_idx : kk->start_idx;
                if (idx) idx[gid] = j0 + j + 1;
            }

            // ---- the gap ending here, from the endpoint one lane below
            double px = dpp_f64<DPP_WAVE_SHR1, 0xf>(x);
            double pph = dpp_f64<DPP_WAVE_SHR1, 0xf>(ph);
            double pright = dpp_f64<DPP_WAVE_SHR1, 0xf>(right);
            double pFn = dpp_f64<DPP_WAVE_SHR1, 0xf>(A1.y);
            int pjx = dpp_i32<DPP_WAVE_SHR1, 0xf>(j);
            if (lane == 0) {
                px = rs_x;
                pph = rs_ph;
                pright = rs_right;
                pFn = rs_Fn;
                pjx = rs_j;
            }
            // finite and not before the stream's previous endpoint
            if (real && kk->validate && (!(fabs(x) < INFINITY) || !(((lane == 0) ? slastx : px) <= x)))
                err |= ERR_INTERVAL;
            const bool has_gap = real || tail_lane;
            const bool same = (pjx == j);
            // both in segment j: the trapezoid of the two interpolated values
            const double q_in = ((pph + ph) * (x - px)) * 0.5;
            double whole = fmax(Fj - pFn, 0.0);
            const bool ill = has_gap && !same && (j >= pjx + 2) && (whole < Fj * 0x1p-14);
            if (__ballot(ill) != 0ull) {
                if (ill) {
                    // the whole segments summed directly
                    double sum = 0.0;
                    for (int i = pjx + 1; i < j; ++i)
                        sum += seg_energy(t_at(i), t_at(i + 1), (float)P_at(i), (float)P_at(i + 1));
                    whole = sum;
                }
            }
            const double Q = same ? q_in : (pright + whole) + left;
            const bool open = (q & 1) != 0;  // the gap lies inside an interval
            if (has_gap && !open) idle += Q;
            if (has_gap && open) {
                // an interval ending at this endpoint, or open at the tile's
                // end: complete when it began in this tile, else its piece here
                const bool began = (lane > 0) || started;
                if (real)
                    *(began ? &kk->energy[gid] : &kk->head[b]) = Q;
                else
                    *(began ? &kk->tail[b] : &kk->head[b]) = Q;
            }
            // ---- commit (uniform)
            if (k > 0) {
                const int ll = k - 1;
                slastx = read_lane_f64(x, ll);
                rs_x = slastx;
                rs_ph = read_lane_f64(ph, ll);
                rs_right = read_lane_f64(right, ll);
                rs_Fn = read_lane_f64(A1.y, ll);
                rs_j = __builtin_amdgcn_readlane(j, ll);
                started = (sqn & 1) ? 1 : 0;  // the last endpoint was a start
            }
            sq = sqn;
            if (fin) break;
        }
        wave_sync();
    }

    // the run's trace and idle energy, at its first tile (k_fix adds them up)
    const double It = wave_sum(idle);
    const KArgs k = kargs();
    if (lane == 0) {
        k->part[b0] = make_double2(w_wave, It);
        // where this run stopped: the next run must start there
        k->cnt_fin[b1] = sq;
        if (b1 == (int)k->NT) k->cnt[b1] = sq;
    }
    if (__ballot(err != 0u)) {
        unsigned e = err;
        for (int off = 32; off > 0; off >>= 1) e |= __shfl_xor(e, off);
        if (lane == 0) atomicOr(&k->status->err, e);
    }
}

namespace {

template <class Lds>
hipError_t launch_tile_kernel(void (*kern)(TileParams), int& per_cu, TileParams p, int64_t ntiles,
                              hipStream_t stream, hipEvent_t ev_start, hipEvent_t ev_stop)
{
    // resident waves per CU (the occupancy the runtime reports, capped by LDS)
    if (per_cu == 0) {
        int nb = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kern, WAVE, 0) != hipSuccess ||
            nb <= 0)
            nb = 8;
        // LDS is granted in 2 KiB blocks: never count on more waves than fit that way
        int dev = 0, lds = 0;
        if (hipGetDevice(&dev) == hipSuccess &&
            hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) ==
                hipSuccess &&
            lds > 0) {
            const int per_wave = (int)((sizeof(Lds) + 2047) / 2048) * 2048;
            nb = max(1, min(nb, lds / per_wave));
        }
        per_cu = nb;
    }
    // runs of at most RUN_TILES tiles: many more workgroups than fit at once,
    // so the hardware deals them out as slots free up -- workgroups of other
    // kernels (another attribution's grouping) interleave with them, and no
    // slot is left with a long run started late (measured on the A/B step of
    // the multi-stream 100M-sample workload: 16 tiles per run 0.978 ms per
    // step, 32 tiles 0.987 ms, 8 tiles no faster than 32).  A launch whose one
    // round of workgroups would take runs shorter than RUN_TILES is split in
    // two rounds of half-length runs (a 20M-sample one-stream trace: two
    // rounds of 5 tiles 0.116 ms per launch, one round of 10 0.123 ms; a
    // 32M-sample chunk keeps its one round of 16: 6.01-6.03 ms per step of the
    // long run against 6.04-6.13 ms with two rounds of 8)
    const int64_t waves = (int64_t)device_cu_count() * per_cu;
    const int64_t one_round = (ntiles + waves - 1) / waves;
    p.tiles_per_wg = one_round >= RUN_TILES
                         ? RUN_TILES
                         : std::max<int64_t>(1, (ntiles + 2 * waves - 1) / (2 * waves));
    const int64_t runs = (ntiles + p.tiles_per_wg - 1) / p.tiles_per_wg;
    if (ev_start || ev_stop)
        // timing events travel with the dispatch: no marker packets around it
        hipExtLaunchKernelGGL(kern, dim3((unsigned)runs), dim3(WAVE), 0, stream, ev_start, ev_stop,
                              0, p);
    else
        hipLaunchKernelGGL(kern, dim3((unsigned)runs), dim3(WAVE), 0, stream, p);
    return hipGetLastError();
}

template <int SP>
hipError_t launch_tile_t(const TileParams& p, int64_t ntiles, hipStream_t stream,
                         hipEvent_t ev_start, hipEvent_t ev_stop)
{
    static int per_cu = 0;
    return launch_tile_kernel<TileLds<SP>>(k_tile<SP>, per_cu, p, ntiles, stream, ev_start,
                                           ev_stop);
}

hipError_t launch_tile_seq(const TileParams& p, int64_t ntiles, hipStream_t stream,
                           hipEvent_t ev_start, hipEvent_t ev_stop)
{
    static int per_cu = 0;
    return launch_tile_kernel<SeqLds>(k_tile_seq, per_cu, p, ntiles, stream, ev_start, ev_stop);
}

}  // namespace

hipError_t launch_tile(const TileParams& p, hipStream_t stream, hipEvent_t ev_start,
                       hipEvent_t ev_stop)
{
    const int64_t ntiles = p.tile_end - p.tile_begin;
    if (ntiles <= 0) return hipSuccess;
    const int S = p.ss.S;
    if (S == 1) return launch_tile_seq(p, ntiles, stream, ev_start, ev_stop);
    if (S == 2) return launch_tile_t<2>(p, ntiles, stream, ev_start, ev_stop);
    if (S <= 4) return launch_tile_t<4>(p, ntiles, stream, ev_start, ev_stop);
    if (S <= 8) return launch_tile_t<8>(p, ntiles, stream, ev_start, ev_stop);
    if (S <= 16) return launch_tile_t<16>(p, ntiles, stream, ev_start, ev_stop);
    return launch_tile_t<32>(p, ntiles, stream, ev_start, ev_stop);
}

}  // namespace mag
