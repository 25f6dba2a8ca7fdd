/*
 * oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * The plain, slow, single-threaded CPU reference for operator-level energy
 * attribution and A/B energy comparison (Magneton, arXiv 2512.08365).  Only
 * the test suite, the package smoke check and the benchmark's CPU-baseline leg
 * may load this library.  It shares no code, header, table or constant with
 * the HIP path, and nothing in the product calls it.
 *
 * What the paper fixes, and what it leaves to a reading:
 *   - Section 5.2 (Energy Profiling) requires energy to be attributed to
 *     individual GPU kernels that run for tens to hundreds of microseconds,
 *     from a power source with microsecond resolution.  It gives no formula.
 *   - Section 4.1 makes the operator the unit that is compared between two
 *     systems; Section 2.1 (Case 1) ranks operators by energy ("top 5").
 *   - Section 6.1 detects waste from the relative energy difference between
 *     matched operators (10% threshold, 5% also works); Table
 *     "tab:energy-profiling" shows the sign convention of a relative error:
 *     (value - reference) / reference.
 * The arithmetic below is the reading this build adopts (listed, with the
 * reasons, in the design notes):
 *   - the power signal is the piecewise-linear interpolant of the samples on
 *     [t_0, t_{n-1}] and zero outside it; an interval's energy is the exact
 *     integral of that interpolant over the interval (trapezoid rule with
 *     interpolation at the interval bounds);
 *   - with equal splitting, the power at each instant is divided equally
 *     among the intervals active at that instant (half-open [s, e));
 *   - per operator key: count, sum and M2 = sum of squared deviations from
 *     the key's mean (Welford 1962, cross-checked by the two-pass formula);
 *   - diff: inner join on key, r = (E_B - E_A) / E_A, ordered by r descending
 *     then key ascending (unsigned), first k rows;
 *   - software replay mode (Section 5.2): per-operator energy from a delayed
 *     cumulative energy counter, see orc_counter_attribute.
 *
 * Numerics: every energy is a left-to-right sum of non-negative pieces, each
 * piece the trapezoid of a linear function over a sub-interval of one sample
 * segment, so no result is ever a difference of large running totals.
 * Whole-trace totals use Neumaier-compensated summation.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* status codes of this reference (kept numerically equal to the documented
   ones of the library so that tests can compare error kinds) */
enum {
    ORC_OK = 0,
    ORC_E_NULL = -1,
    ORC_E_SIZE = -2,
    ORC_E_TIMESTAMPS = -5,
    ORC_E_POWER = -6,
    ORC_E_INTERVAL = -7,
    ORC_E_STREAMS = -8,
    ORC_E_COUNTER = -13,
    ORC_E_NOMEM = -20
};

/* ------------------------------------------------------------------ */
/* textbook helpers                                                    */
/* ------------------------------------------------------------------ */

/* first index j in [0, n) with t[j] >= x, or n (std::lower_bound) */
int64_t orc_lower_bound(const double* t, int64_t n, double x)
{
    int64_t lo = 0, hi = n;
    while (lo < hi) {
        int64_t mid = lo + (hi - lo) / 2;
        if (t[mid] < x)
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo;
}

/* Neumaier (1974) compensated summation */
typedef struct {
    double s, c;
} orc_ksum;

static void ks_add(orc_ksum* k, double v)
{
    double t = k->s + v;
    if (fabs(k->s) >= fabs(v))
        k->c += (k->s - t) + v;
    else
        k->c += (v - t) + k->s;
    k->s = t;
}

static double ks_get(const orc_ksum* k) { return k->s + k->c; }

/* ------------------------------------------------------------------ */
/* the power model                                                     */
/* ------------------------------------------------------------------ */

/* value of the linear interpolant at x, with t[j] <= x <= t[j+1];
   exactly the sample value at either end of the segment */
static double power_at(const double* t, const float* P, int64_t j, double x)
{
    double pj = (double)P[j], pk = (double)P[j + 1];
    if (x == t[j])
        return pj;
    if (x == t[j + 1])
        return pk;
    return pj + (pk - pj) * ((x - t[j]) / (t[j + 1] - t[j]));
}

/* energy of the interpolant over [a, b] inside segment j: the trapezoid of a
   linear function is its exact integral */
static double piece(const double* t, const float* P, int64_t j, double a, double b)
{
    return 0.5 * (power_at(t, P, j, a) + power_at(t, P, j, b)) * (b - a);
}

/* integral of the interpolant over [a, b] (t_0 <= a, b <= t_{n-1}),
   walking the sample segments left to right and adding one piece each */
static double integral(const double* t, const float* P, int64_t n, double a, double b)
{
    double acc = 0.0;
    int64_t j;
    if (!(b > a))
        return 0.0;
    j = orc_lower_bound(t, n, a) - 1;
    if (j < 0)
        j = 0;
    for (; j < n - 1 && t[j] < b; ++j) {
        double lo = a > t[j] ? a : t[j];
        double hi = b < t[j + 1] ? b : t[j + 1];
        if (hi > lo)
            acc += piece(t, P, j, lo, hi);
    }
    return acc;
}

/* ------------------------------------------------------------------ */
/* input validation (same rules the library enforces)                  */
/* ------------------------------------------------------------------ */

int orc_validate(const double* t, const float* P, int64_t n, const double* s, const double* e,
                 int64_t m, const int64_t* offsets, int32_t n_streams)
{
    int64_t j, i;
    int32_t a;
    if (n < 2 || m < 0 || n_streams < 1)
        return ORC_E_SIZE;
    for (j = 0; j < n; ++j)
        if (!isfinite(t[j]) || (j > 0 && !(t[j] > t[j - 1])))
            return ORC_E_TIMESTAMPS;
    for (j = 0; j < n; ++j)
        if (!isfinite((double)P[j]) || P[j] < 0.0f)
            return ORC_E_POWER;
    if (offsets) {
        if (offsets[0] != 0 || offsets[n_streams] != m)
            return ORC_E_STREAMS;
        for (a = 0; a < n_streams; ++a)
            if (offsets[a + 1] < offsets[a])
                return ORC_E_STREAMS;
    }
    for (i = 0; i < m; ++i)
        if (!isfinite(s[i]) || !isfinite(e[i]) || s[i] > e[i])
            return ORC_E_INTERVAL;
    for (a = 0; a < n_streams; ++a) {
        int64_t lo = offsets ? offsets[a] : 0, hi = offsets ? offsets[a + 1] : m;
        for (i = lo + 1; i < hi; ++i)
            if (e[i - 1] > s[i])
                return ORC_E_INTERVAL; /* unsorted or overlapping within one stream */
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------ */
/* attribution                                                          */
/* ------------------------------------------------------------------ */

typedef struct {
    double time;
    int64_t id;
    int32_t open; /* 1 = interval becomes active, 0 = it stops */
} orc_event;

static int cmp_event(const void* pa, const void* pb)
{
    const orc_event* x = (const orc_event*)pa;
    const orc_event* y = (const orc_event*)pb;
    if (x->time < y->time)
        return -1;
    if (x->time > y->time)
        return 1;
    if (x->id < y->id)
        return -1;
    if (x->id > y->id)
        return 1;
    return x->open - y->open;
}

/*
 * orc_attribute: per-interval energy and sample indices.
 *   t[n] strictly increasing (s), P[n] >= 0 (W), s/e[m] interval bounds (s).
 *   offsets[n_streams+1] (may be NULL for one stream) only matter for validation.
 *   equal_split != 0: divide the power among the intervals active at each
 *   instant; 0: every interval receives the full power over its span.
 * Outputs (caller-owned host arrays): energy[m] (J), start_idx[m], end_idx[m]
 * (lower_bound of the unclipped bounds), summary[4] = {trace energy W,
 * idle energy, sum of interval energies, number of clipped intervals}.
 */
int orc_attribute(const double* t, const float* P, int64_t n, const double* s, const double* e,
                  int64_t m, const int64_t* offsets, int32_t n_streams, int32_t equal_split,
                  double* energy, int64_t* start_idx, int64_t* end_idx, double* summary)
{
    int64_t i, j, n_clipped = 0;
    orc_ksum w = {0, 0}, idle = {0, 0}, attributed = {0, 0};
    double t0, tn;
    int rc;

    if (!t || !P || (m > 0 && (!s || !e || !energy || !start_idx || !end_idx)) || !summary)
        return ORC_E_NULL;
    rc = orc_validate(t, P, n, s, e, m, offsets, n_streams);
    if (rc != ORC_OK)
        return rc;
    t0 = t[0];
    tn = t[n - 1];

    for (j = 0; j + 1 < n; ++j)
        ks_add(&w, piece(t, P, j, t[j], t[j + 1]));

    for (i = 0; i < m; ++i) {
        start_idx[i] = orc_lower_bound(t, n, s[i]);
        end_idx[i] = orc_lower_bound(t, n, e[i]);
        energy[i] = 0.0;
        if (s[i] < t0 || e[i] > tn)
            ++n_clipped;
    }

    if (!equal_split) {
        /* every interval integrates the full power over its clipped span */
        for (i = 0; i < m; ++i) {
            double a = s[i] > t0 ? s[i] : t0;
            double b = e[i] < tn ? e[i] : tn;
            energy[i] = integral(t, P, n, a, b);
        }
    }

    {
        /* sweep over interval boundaries; between two consecutive distinct
           boundary times the set of active intervals is constant.  With
           equal splitting each active interval receives 1/|A| of the energy
           of that stretch; in both modes a stretch with no active interval
           is idle energy. */
        orc_event* ev = (orc_event*)malloc(sizeof(orc_event) * (size_t)(2 * m + 1));
        int64_t* active = (int64_t*)malloc(sizeof(int64_t) * (size_t)(m + 1));
        int64_t* where = (int64_t*)malloc(sizeof(int64_t) * (size_t)(m + 1));
        int64_t n_ev = 0, n_act = 0, k;
        double cur;
        if (!ev || !active || !where) {
            free(ev);
            free(active);
            free(where);
            return ORC_E_NOMEM;
        }
        for (i = 0; i < m; ++i) {
            double a = s[i] > t0 ? s[i] : t0;
            double b = e[i] < tn ? e[i] : tn;
            if (b > a) { /* zero-length or outside spans are never active */
                ev[n_ev].time = a;
                ev[n_ev].id = i;
                ev[n_ev].open = 1;
                ++n_ev;
                ev[n_ev].time = b;
                ev[n_ev].id = i;
                ev[n_ev].open = 0;
                ++n_ev;
            }
        }
        qsort(ev, (size_t)n_ev, sizeof(orc_event), cmp_event);
        cur = t0;
        k = 0;
        while (1) {
            double next = (k < n_ev) ? ev[k].time : tn;
            if (next > cur) {
                double q = integral(t, P, n, cur, next);
                if (n_act == 0) {
                    ks_add(&idle, q);
                } else if (equal_split) {
                    int64_t u;
                    for (u = 0; u < n_act; ++u)
                        energy[active[u]] += q / (double)n_act;
                }
                cur = next;
            }
            if (k >= n_ev)
                break;
            /* apply every boundary at this instant */
            while (k < n_ev && ev[k].time == cur) {
                int64_t id = ev[k].id;
                if (ev[k].open) {
                    where[id] = n_act;
                    active[n_act++] = id;
                } else {
                    int64_t pos = where[id];
                    int64_t last = active[--n_act];
                    active[pos] = last;
                    where[last] = pos;
                }
                ++k;
            }
        }
        free(ev);
        free(active);
        free(where);
    }

    for (i = 0; i < m; ++i)
        ks_add(&attributed, energy[i]);
    summary[0] = ks_get(&w);
    summary[1] = ks_get(&idle);
    summary[2] = ks_get(&attributed);
    summary[3] = (double)n_clipped;
    return ORC_OK;
}

/* ------------------------------------------------------------------ */
/* group-by operator key                                                */
/* ------------------------------------------------------------------ */

typedef struct {
    uint64_t key;
    int64_t idx;
} orc_kv;

static int cmp_kv(const void* pa, const void* pb)
{
    const orc_kv* x = (const orc_kv*)pa;
    const orc_kv* y = (const orc_kv*)pb;
    if (x->key < y->key)
        return -1;
    if (x->key > y->key)
        return 1;
    return (x->idx > y->idx) - (x->idx < y->idx);
}

/*
 * orc_groupby: per distinct key, in ascending unsigned key order:
 *   count, sum (compensated), M2 by the two-pass definition
 *   sum_i (E_i - mean)^2 (compensated), and M2 by Welford's update applied
 *   in interval-index order (returned separately as a cross-check).
 * Output arrays must hold m rows; *n_keys receives the number written.
 */
int orc_groupby(const uint64_t* keys, const double* energy, int64_t m, uint64_t* out_keys,
                int64_t* out_count, double* out_sum, double* out_m2, double* out_m2_welford,
                int64_t* n_keys)
{
    orc_kv* kv;
    int64_t i, r = 0;
    if (m < 0)
        return ORC_E_SIZE;
    if (!n_keys || (m > 0 && (!keys || !energy || !out_keys || !out_count || !out_sum ||
                              !out_m2 || !out_m2_welford)))
        return ORC_E_NULL;
    kv = (orc_kv*)malloc(sizeof(orc_kv) * (size_t)(m + 1));
    if (!kv)
        return ORC_E_NOMEM;
    for (i = 0; i < m; ++i) {
        kv[i].key = keys[i];
        kv[i].idx = i;
    }
    qsort(kv, (size_t)m, sizeof(orc_kv), cmp_kv);
    i = 0;
    while (i < m) {
        int64_t lo = i, hi = i, u;
        orc_ksum sum = {0, 0}, sq = {0, 0};
        double mean, wmean = 0.0, wm2 = 0.0;
        while (hi < m && kv[hi].key == kv[lo].key)
            ++hi;
        for (u = lo; u < hi; ++u) {
            double x = energy[kv[u].idx];
            double d;
            ks_add(&sum, x);
            /* Welford: running mean and M2, one value at a time */
            d = x - wmean;
            wmean += d / (double)(u - lo + 1);
            wm2 += d * (x - wmean);
        }
        mean = ks_get(&sum) / (double)(hi - lo);
        for (u = lo; u < hi; ++u) {
            double d = energy[kv[u].idx] - mean;
            ks_add(&sq, d * d);
        }
        out_keys[r] = kv[lo].key;
        out_count[r] = hi - lo;
        out_sum[r] = ks_get(&sum);
        out_m2[r] = ks_get(&sq);
        out_m2_welford[r] = wm2;
        ++r;
        i = hi;
    }
    *n_keys = r;
    free(kv);
    return ORC_OK;
}

/*
 * orc_key_latency: per distinct key, in ascending unsigned key order, the
 * operator's latency: the compensated sum of its interval durations
 * ends[i] - starts[i] (unclipped bounds), each divided by reps[i] when reps
 * is given (a replay window's duration per run).  Section 6.1 weighs an
 * operator's energy difference against its performance difference; this is
 * the performance side.  Output arrays hold m rows; *n_keys receives the
 * number written.
 */
int orc_key_latency(const uint64_t* keys, const double* starts, const double* ends,
                    const int32_t* reps, int64_t m, uint64_t* out_keys, double* out_latency,
                    int64_t* n_keys)
{
    orc_kv* kv;
    int64_t i, r = 0;
    if (m < 0)
        return ORC_E_SIZE;
    if (!n_keys || (m > 0 && (!keys || !starts || !ends || !out_keys || !out_latency)))
        return ORC_E_NULL;
    kv = (orc_kv*)malloc(sizeof(orc_kv) * (size_t)(m + 1));
    if (!kv)
        return ORC_E_NOMEM;
    for (i = 0; i < m; ++i) {
        kv[i].key = keys[i];
        kv[i].idx = i;
    }
    qsort(kv, (size_t)m, sizeof(orc_kv), cmp_kv);
    i = 0;
    while (i < m) {
        int64_t lo = i, hi = i, u;
        orc_ksum sum = {0, 0};
        while (hi < m && kv[hi].key == kv[lo].key)
            ++hi;
        for (u = lo; u < hi; ++u) {
            int64_t x = kv[u].idx;
            double d = ends[x] - starts[x];
            ks_add(&sum, reps ? d / (double)reps[x] : d);
        }
        out_keys[r] = kv[lo].key;
        out_latency[r] = ks_get(&sum);
        ++r;
        i = hi;
    }
    *n_keys = r;
    free(kv);
    return ORC_OK;
}

/* ------------------------------------------------------------------ */
/* diff: join and rank                                                  */
/* ------------------------------------------------------------------ */

typedef struct {
    uint64_t key;
    double r;
    int64_t ia, ib;
} orc_row;

static int cmp_row(const void* pa, const void* pb)
{
    const orc_row* x = (const orc_row*)pa;
    const orc_row* y = (const orc_row*)pb;
    if (x->r > y->r)
        return -1;
    if (x->r < y->r)
        return 1;
    if (x->key < y->key)
        return -1;
    if (x->key > y->key)
        return 1;
    return 0;
}

/* relative energy difference of B against the baseline A */
double orc_ratio(double ea, double eb)
{
    if (ea == 0.0)
        return eb > 0.0 ? INFINITY : 0.0;
    return (eb - ea) / ea;
}

/*
 * orc_diff: inner join of two key tables (ascending keys), r = (E_B - E_A)/E_A,
 * rows ordered by r descending then key ascending; the first min(k, |join|)
 * rows are written.  counts[0..3] = {rows written, keys only in A, keys only
 * in B, |join|}.  *margin = smallest gap r_p - r_{p+1} among the first k+1
 * ordered rows (INFINITY if fewer than two).
 */
int orc_diff(const uint64_t* ka, const double* sa, const int64_t* ca, int64_t na,
             const uint64_t* kb, const double* sb, const int64_t* cb, int64_t nb, int64_t k,
             uint64_t* out_key, double* out_r, double* out_ea, double* out_eb, int64_t* out_ca,
             int64_t* out_cb, int64_t* counts, double* margin)
{
    orc_row* rows;
    int64_t ia = 0, ib = 0, nj = 0, only_a = 0, only_b = 0, u, take;
    if (na < 0 || nb < 0 || k < 0)
        return ORC_E_SIZE;
    rows = (orc_row*)malloc(sizeof(orc_row) * (size_t)(na + 1));
    if (!rows)
        return ORC_E_NOMEM;
    while (ia < na || ib < nb) {
        if (ib >= nb || (ia < na && ka[ia] < kb[ib])) {
            ++only_a;
            ++ia;
        } else if (ia >= na || kb[ib] < ka[ia]) {
            ++only_b;
            ++ib;
        } else {
            rows[nj].key = ka[ia];
            rows[nj].r = orc_ratio(sa[ia], sb[ib]);
            rows[nj].ia = ia;
            rows[nj].ib = ib;
            ++nj;
            ++ia;
            ++ib;
        }
    }
    qsort(rows, (size_t)nj, sizeof(orc_row), cmp_row);
    take = k < nj ? k : nj;
    for (u = 0; u < take; ++u) {
        out_key[u] = rows[u].key;
        out_r[u] = rows[u].r;
        out_ea[u] = sa[rows[u].ia];
        out_eb[u] = sb[rows[u].ib];
        out_ca[u] = ca[rows[u].ia];
        out_cb[u] = cb[rows[u].ib];
    }
    *margin = INFINITY;
    for (u = 0; u + 1 < nj && u < k; ++u) {
        double g = rows[u].r - rows[u + 1].r;
        if (g < *margin)
            *margin = g;
    }
    counts[0] = take;
    counts[1] = only_a;
    counts[2] = only_b;
    counts[3] = nj;
    free(rows);
    return ORC_OK;
}

/* ------------------------------------------------------------------ */
/* attribution from a cumulative energy counter (software replay mode) */
/* ------------------------------------------------------------------ */

/*
 * Section 5.2 also offers a mode without a power meter: the vendor's energy
 * interface gives a cumulative energy reading that is refreshed only at 10 to
 * 50 Hz and lags the device by up to some hundreds of milliseconds, so each
 * operator is replayed until its run is long enough for that reading to
 * settle; the per-operator energy is the reading's increase over the replay
 * window divided by the number of replays (the evaluation replays each
 * operator 1,000 times).  The paper gives no formula; the reading this build
 * adopts:
 *   - a reading C_j taken at t_j holds the energy used up to t_j - delay: the
 *     counter's points are (u_j, C_j) with u_j = t_j - delay, one fp64
 *     subtraction;
 *   - between points the cumulative energy C^(x) is the linear interpolant;
 *     before u_0 it stays at C_0 and after u_{n-1} at C_{n-1} (nothing outside
 *     the readings is attributed);
 *   - window i ran its operator N_i times: E_i = (C^(e_i) - C^(s_i)) / N_i;
 *   - windows form one sequence, s_i <= e_i <= s_{i+1} (one operator replays
 *     at a time), so that the increase outside every window is the idle
 *     energy.
 * The increase C^(y) - C^(x) is taken as the part of x's segment after x, the
 * whole segments in between (a difference of two readings) and the part of
 * y's segment before y, never as a difference of two interpolated values.
 */

/* counter increase from x to y inside segment a, u_{a-1} <= x <= y <= u_a */
static double seg_increase(const double* u, const double* C, int64_t a, double x, double y)
{
    return (C[a] - C[a - 1]) * ((y - x) / (u[a] - u[a - 1]));
}

/* C^(y) - C^(x) for x <= y */
static double counter_increase(const double* u, const double* C, int64_t n, double x, double y)
{
    int64_t a = orc_lower_bound(u, n, x), b = orc_lower_bound(u, n, y);
    double head, mid, tail;
    if (a == b) /* one segment, or both before u_0, or both after u_{n-1} */
        return (a == 0 || a == n) ? 0.0 : seg_increase(u, C, a, x, y);
    head = (a == 0) ? 0.0 : seg_increase(u, C, a, x, u[a]);
    mid = C[b - 1] - C[a];
    tail = (b == n) ? 0.0 : seg_increase(u, C, b, u[b - 1], y);
    return mid + (head + tail);
}

/* validation of a counter trace and its replay windows; u receives t - delay */
static int counter_validate(const double* t, const double* C, int64_t n, double delay,
                            const double* s, const double* e, const int32_t* reps, int64_t m,
                            double* u)
{
    int64_t j, i;
    if (n < 2 || m < 0)
        return ORC_E_SIZE;
    if (!isfinite(delay))
        return ORC_E_TIMESTAMPS;
    for (j = 0; j < n; ++j) {
        u[j] = t[j] - delay;
        if (!isfinite(t[j]) || !isfinite(u[j]) || (j > 0 && !(u[j] > u[j - 1])))
            return ORC_E_TIMESTAMPS;
    }
    for (j = 0; j < n; ++j)
        if (!isfinite(C[j]) || (j > 0 && !(C[j] >= C[j - 1])))
            return ORC_E_COUNTER;
    for (i = 0; i < m; ++i) {
        if (!isfinite(s[i]) || !isfinite(e[i]) || s[i] > e[i])
            return ORC_E_INTERVAL;
        if (i > 0 && e[i - 1] > s[i])
            return ORC_E_INTERVAL;
        if (reps && reps[i] < 1)
            return ORC_E_INTERVAL;
    }
    return ORC_OK;
}

/*
 * orc_counter_attribute: per-window operator energy from a cumulative counter.
 *   t[n] reading times (s), C[n] readings (J), delay (s), s/e[m] replay
 *   windows, reps[m] replays per window (NULL: 1 each).
 * Outputs (caller-owned host arrays): energy[m] = E_i (J per replay),
 * start_idx[m] / end_idx[m] = lower_bound of s_i / e_i among the shifted
 * times u, summary[4] = {C_{n-1} - C_0, counter increase outside every window
 * (idle), sum of E_i, windows with s_i < u_0 or e_i > u_{n-1}}.
 */
int orc_counter_attribute(const double* t, const double* C, int64_t n, double delay,
                          const double* s, const double* e, const int32_t* reps, int64_t m,
                          double* energy, int64_t* start_idx, int64_t* end_idx, double* summary)
{
    orc_ksum idle = {0, 0}, attributed = {0, 0};
    int64_t i, n_clipped = 0;
    double* u;
    int rc;
    if (!t || !C || (m > 0 && (!s || !e || !energy || !start_idx || !end_idx)) || !summary)
        return ORC_E_NULL;
    if (n < 2 || m < 0)
        return ORC_E_SIZE;
    u = (double*)malloc(sizeof(double) * (size_t)n);
    if (!u)
        return ORC_E_NOMEM;
    rc = counter_validate(t, C, n, delay, s, e, reps, m, u);
    if (rc != ORC_OK) {
        free(u);
        return rc;
    }
    for (i = 0; i < m; ++i) {
        double d = counter_increase(u, C, n, s[i], e[i]);
        start_idx[i] = orc_lower_bound(u, n, s[i]);
        end_idx[i] = orc_lower_bound(u, n, e[i]);
        energy[i] = d / (double)(reps ? reps[i] : 1);
        ks_add(&attributed, energy[i]);
        if (s[i] < u[0] || e[i] > u[n - 1])
            ++n_clipped;
        /* the gap before this window */
        ks_add(&idle, counter_increase(u, C, n, i > 0 ? e[i - 1] : -INFINITY, s[i]));
    }
    ks_add(&idle, counter_increase(u, C, n, m > 0 ? e[m - 1] : -INFINITY, INFINITY));
    summary[0] = C[n - 1] - C[0];
    summary[1] = ks_get(&idle);
    summary[2] = ks_get(&attributed);
    summary[3] = (double)n_clipped;
    free(u);
    return ORC_OK;
}
