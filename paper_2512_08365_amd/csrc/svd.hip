// svd.hip -- multi-mode SVD invariants of tensors and their matching
// (Section 4.2, "Matching Equivalent Tensors").
//
// For every non-empty proper mode subset G containing mode 0 (its complement
// gives the same spectrum), the unfolding T_(G) has the modes of G as rows and
// the others as columns.  Its singular values are the square roots of the
// eigenvalues of the Gram matrix X X^T, X the unfolding or its transpose,
// whichever has fewer rows (K = min(M, N) <= SVD_MAX_K, L = max(M, N)).
//
// k_gram: one workgroup per (task, 64 x 64 block of the upper triangle,
//   chunk of GRAM_CHUNK columns); the block's rows are staged in LDS a step
//   of columns at a time and its 16 tiles are sums of fp64 16x16x4 MFMA
//   products (fp32 data widened exactly), added into the Gram matrix (and its
//   mirror) with fp64 atomics.  The elements of X are gathered through the
//   unfolding's mixed-radix offsets.  Sides up to 32: one 32-side block;
//   sides in (64, 128]: k_gram_whole, the whole triangle per workgroup.
// k_svd_eig: one workgroup per task: Householder reduction of the Gram
//   matrix (in LDS up to side 128, else in place in global memory) to
//   tridiagonal form and its Gershgorin bounds; k_svd_count: every
//   eigenvalue by multisection on Sturm counts (the count of eigenvalues
//   below x), a wave per 16 eigenvalues, sigma = sqrt(max(lambda, 0)),
//   written in descending order.
// k_svd_match: one workgroup per tensor pair: which spectra of the two lists
//   are close, then a one-to-one pairing by augmenting paths.

#include <cfloat>

#include "mag_internal.hpp"

namespace mag {

namespace {

constexpr int GW = 64;
constexpr int EIG_THREADS = 512;

typedef double d4 __attribute__((ext_vector_type(4)));

// element offset of index x over the modes (sizes dim, strides str), the last
// mode fastest; every size and index fits 32 bits (the host checks the tensor)
__device__ __forceinline__ int64_t mode_offset(uint32_t x, int n, const int64_t* dim,
                                               const int64_t* str)
{
    int64_t off = 0;
    for (int i = n - 1; i >= 0; --i) {
        const uint32_t d = (uint32_t)dim[i];
        const uint32_t q = x / d;
        off += (int64_t)(x - q * d) * str[i];
        x = q;
    }
    return off;
}

__global__ void k_svd_clear(double* g, int64_t n)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        g[i] = 0.0;
}

// One workgroup per (task, GB x GB block of the upper triangle, chunk of
// GRAM_CHUNK columns), one wave per 16 x 16 tile of the block (GB = 64: 16
// waves; GB = 32, for unfoldings with at most 32 rows: 4 waves).  Each
// 64-column step stages the block's GB rows of each operand in LDS as fp64,
// GPER gathered elements per thread; wave w then multiplies tile
// (w / (GB/16), w % (GB/16)) from LDS with 16 MFMA steps while the next step's
// elements are in flight.  On a diagonal block the tiles below the diagonal
// are mirrors of those above: their waves only stage.  The gather runs along
// whichever side of the unfolding has unit stride (the rows when the K side's
// last mode is the tensor's last, else the columns), so 64 neighbouring
// threads read 256 contiguous bytes.
constexpr int GSTEP = 64;  // columns staged per step

template <int GB>
__global__ __launch_bounds__(GB * GB / 4) void k_gram(const SvdTask* tasks, int n_tasks,
                                                      int64_t n_items)
{
    constexpr int TPB = GB / 16;              // tiles per block side
    constexpr int THREADS = GB * GB / 4;      // one wave per tile
    constexpr int GPER = 2 * GB * GSTEP / THREADS;  // staged elements per thread and step
    // a 32-side block is the whole Gram matrix (K <= 32), its one diagonal
    // block: one operand staged, half the LDS, shorter column chunks (more
    // workgroups for the same unfoldings)
    constexpr bool ONE_BLOCK = GB == GRAM_NARROW;
    constexpr int64_t CH = ONE_BLOCK ? GRAM_CHUNK_NARROW : GRAM_CHUNK;
    __shared__ double xs[ONE_BLOCK ? 1 : 2][GSTEP][GB + 1];  // operand, [column][row], padded
    __shared__ int32_t loff[CH];
    __shared__ int64_t roff[2][GB];
    const int64_t item = blockIdx.x;
    if (item >= n_items) return;  // uniform
    int lo = 0, hi = n_tasks - 1;  // the last task whose first item is <= item
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (tasks[mid].item0 <= item) lo = mid; else hi = mid - 1;
    }
    const SvdTask& t = tasks[lo];
    const int64_t local = item - t.item0;
    const int64_t chunk = local % t.nchunk;
    int64_t pr = local / t.nchunk;
    int bi = 0, rowlen = t.nt;  // nt counts GB-row blocks here
    while (pr >= rowlen && rowlen > 0) {
        pr -= rowlen;
        ++bi;
        --rowlen;
    }
    const int bj = bi + (int)pr;
    const int tid = threadIdx.x, lane = tid % GW, wv = tid / GW;
    const int64_t b0 = chunk * CH, b1 = min(b0 + CH, t.L);
    for (int64_t q = tid; q < b1 - b0; q += THREADS)
        loff[q] = (int32_t)mode_offset((uint32_t)(b0 + q), t.nl, t.ldim, t.lstr);
    if (tid < 2 * GB) {
        const int side = tid / GB, r = tid % GB;
        const int64_t row = (int64_t)(side ? bj : bi) * GB + r;
        roff[side][r] = (row < t.K) ? mode_offset((uint32_t)row, t.nk, t.kdim, t.kstr) : -1;
    }
    // neighbouring threads take neighbouring columns unless the rows are the
    // unit-stride side (uniform)
    const bool cols_fast = t.kstr[t.nk - 1] != 1;
    __syncthreads();
    // staged element u of this thread: operand, row and column of the step
    auto slot = [&](int u, int& side, int& rr, int& c) {
        const int q = tid + u * THREADS;
        side = q / (GB * GSTEP);
        const int rem = q % (GB * GSTEP);
        rr = cols_fast ? rem / GSTEP : rem % GB;
        c = cols_fast ? rem % GSTEP : rem / GB;
    };
    // a diagonal block's two operands are the same rows: staged once (the
    // first GPER / 2 elements of every thread are operand 0's).  Measured: a
    // gain for 32-side blocks (99 -> 93 us on 64 tensors' 32 x 16384
    // unfoldings), a loss for 64-side ones (286 -> 325 us: their fetch loop
    // no longer issues its eight loads back to back), which stage both
    constexpr bool diag = ONE_BLOCK;
    float stage[GPER];
    // the tensor through a global-memory pointer (a generic one would make
    // flat loads, which the LDS waits of the products also count)
    typedef const __attribute__((address_space(1))) float* gfloat;
    const gfloat data = (gfloat)t.data;
    auto fetch = [&](int64_t s0) {
        const int cols = (int)min((int64_t)GSTEP, b1 - s0);
#pragma unroll
        for (int u = 0; u < GPER; ++u) {
            if (diag && u >= GPER / 2) break;
            int side, rr, c;
            slot(u, side, rr, c);
            const int64_t ro = roff[side][rr];
            stage[u] = (c < cols && ro >= 0) ? data[ro + loff[s0 - b0 + c]] : 0.0f;
        }
    };
    const int ti = wv / TPB, tj = wv % TPB;  // this wave's tile inside the block
    // (uniform per wave) a tile below the diagonal of a diagonal block mirrors one above
    const bool active = (bi != bj) || (ti <= tj);
    const int r = lane & 15, kq = lane >> 4;
    d4 acc = {0.0, 0.0, 0.0, 0.0};
    fetch(b0);
    for (int64_t s0 = b0; s0 < b1; s0 += GSTEP) {
#pragma unroll
        for (int u = 0; u < GPER; ++u) {
            if (diag && u >= GPER / 2) break;
            int side, rr, c;
            slot(u, side, rr, c);
            if constexpr (ONE_BLOCK)
                xs[0][c][rr] = (double)stage[u];  // fp32 widened exactly
            else
                xs[side][c][rr] = (double)stage[u];
        }
        __syncthreads();
        if (s0 + GSTEP < b1) fetch(s0 + GSTEP);  // in flight during the products
        // (two loops, so that both operands' LDS addresses stay fixed offsets)
        if constexpr (ONE_BLOCK) {
            if (active) {
#pragma unroll 4
                for (int c = 0; c < GSTEP; c += 4) {
                    const double a = xs[0][c + kq][ti * 16 + r];
                    const double b = xs[0][c + kq][tj * 16 + r];
                    acc = __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, acc, 0, 0, 0);
                }
            }
        } else if (active) {
#pragma unroll 4
            for (int c = 0; c < GSTEP; c += 4) {
                const double a = xs[0][c + kq][ti * 16 + r];
                const double b = xs[1][c + kq][tj * 16 + r];
                acc = __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, acc, 0, 0, 0);
            }
        }
        __syncthreads();  // before the next step overwrites the staged rows
    }
    if (!active) return;
    // register j of a lane holds row 4 j + lane/16, column lane%16 of the tile
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int64_t row = (int64_t)bi * GB + ti * 16 + 4 * j + kq;
        const int64_t col = (int64_t)bj * GB + tj * 16 + r;
        if (row < t.K && col < t.K && (bi != bj || row <= col)) {
            atomicAdd(&t.gram[row * t.K + col], acc[j]);
            if (row != col) atomicAdd(&t.gram[col * t.K + row], acc[j]);
        }
    }
}

// Gram sides in (64, GRAM_WHOLE]: one workgroup per (task, chunk of
// GRAM_CHUNK_WHOLE columns) makes every tile of the upper triangle.  Each
// step of WSTEP columns (11 elements per thread, the last one of some threads
// past the step and skipped; 48-column steps of 8 each: 0.223 against 0.216
// ms for 128 [4096 x 128] unfoldings, fewer MFMAs per barrier) stages the
// chunk's K rows once (the blocked kernel stages every row
// block once per block pair: three times for K = 128), and WHOLE_WAVES waves
// take WHOLE_TILES tiles each: tiles w, w + WHOLE_WAVES, ... of the upper
// triangle in row order, so that with K = 128 (36 tiles) every SIMD holds nine
// (waves are dealt to the SIMDs in turn) and every MFMA issued is a tile of
// the result; each wave's tiles are independent accumulations, interleaved.
constexpr int WHOLE_WAVES = 12;
constexpr int WHOLE_TILES = 3;
constexpr int WSTEP = 64;  // columns staged per step
constexpr int WHOLE_THREADS = WHOLE_WAVES * GW;
constexpr int WHOLE_GPER = (GRAM_WHOLE * WSTEP + WHOLE_THREADS - 1) / WHOLE_THREADS;
static_assert(WHOLE_WAVES * WHOLE_TILES >= (GRAM_WHOLE / 16) * (GRAM_WHOLE / 16 + 1) / 2,
              "every upper-triangle tile has a wave");
static_assert(WHOLE_THREADS % WSTEP == 0 && WHOLE_THREADS % GRAM_WHOLE == 0, "staging layout");

// the products of one staged step for a wave's WHOLE_TILES tiles, written
// with each k-step's operands read a step ahead (the compiler keeps a
// k-step's six reads together ahead of its three MFMAs, reusing one set of
// registers, and the SIMD's other waves cover their latency; the loop
// written without it spilled 17 registers at the 80-VGPR limit); the full unroll makes
// every LDS address a fixed offset from one register per operand
__device__ __forceinline__ void whole_products(const double (*xs)[GRAM_WHOLE + 1],
                                               const int* ti, const int* tj, int r, int kq,
                                               d4* acc)
{
    constexpr int NT = WHOLE_TILES;
    const double* pa[NT];
    const double* pb[NT];
#pragma unroll
    for (int k = 0; k < NT; ++k) {
        pa[k] = &xs[kq][ti[k] * 16 + r];
        pb[k] = &xs[kq][tj[k] * 16 + r];
    }
    double a[2][NT], b[2][NT];
#pragma unroll
    for (int k = 0; k < NT; ++k) {
        a[0][k] = pa[k][0];
        b[0][k] = pb[k][0];
    }
#pragma unroll
    for (int s = 0; s < WSTEP / 4; ++s) {
        const int cur = s & 1, nxt = cur ^ 1;
        if (s + 1 < WSTEP / 4) {
#pragma unroll
            for (int k = 0; k < NT; ++k) {
                a[nxt][k] = pa[k][(s + 1) * 4 * (GRAM_WHOLE + 1)];
                b[nxt][k] = pb[k][(s + 1) * 4 * (GRAM_WHOLE + 1)];
            }
        }
#pragma unroll
        for (int k = 0; k < NT; ++k)
            acc[k] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[cur][k], b[cur][k], acc[k], 0, 0, 0);
    }
}

// the staging and products of k_gram_whole for one gather direction: with
// COLS_FAST, 64 neighbouring threads take neighbouring columns of one row (the
// rows are not the unit-stride side), else neighbouring rows of one column.
// Thread tid stages elements u = 0..WHOLE_GPER-1 at row rr0 + u * RSTEP, column
// c0 + u * CSTEP of each step, compile-time strides, so every per-element LDS
// address is a fixed offset from one register.
template <bool COLS_FAST>
__device__ __forceinline__ void gram_whole_run(const SvdTask& t, int64_t b0, int64_t b1,
                                               double (*xs)[GRAM_WHOLE + 1],
                                               const int32_t* loff, const int32_t* roff,
                                               const int* ti, const int* tj, d4* acc)
{
    constexpr int KB = GRAM_WHOLE;
    constexpr int THREADS = WHOLE_THREADS;
    constexpr int GPER = WHOLE_GPER;
    constexpr int RSTEP = COLS_FAST ? THREADS / WSTEP : 0;
    constexpr int CSTEP = COLS_FAST ? 0 : THREADS / KB;
    const int tid = threadIdx.x, lane = tid % GW;
    const int rr0 = COLS_FAST ? tid / WSTEP : tid % KB;
    const int c0 = COLS_FAST ? tid % WSTEP : tid / KB;
    // the last element of a thread may fall past the step (GPER rounded up)
    const bool last_in = COLS_FAST ? rr0 + (GPER - 1) * RSTEP < KB : c0 + (GPER - 1) * CSTEP < WSTEP;
    typedef const __attribute__((address_space(1))) float* gfloat;
    const gfloat data = (gfloat)t.data;
    float stage[GPER];
    auto fetch = [&](int64_t s0) {
        const int cols = (int)min((int64_t)WSTEP, b1 - s0);
        const int32_t* lo = loff + (s0 - b0);  // the step's columns (chunk-local)
#pragma unroll
        for (int u = 0; u < GPER; ++u) {
            const bool in = u < GPER - 1 || last_in;
            const int c = in ? c0 + u * CSTEP : 0;
            const int ro = roff[in ? rr0 + u * RSTEP : 0];
            const int lc = lo[c];  // in the chunk's table even past its last column
            const bool ok = in && c < cols && ro >= 0;
            const float v = data[ok ? ro + lc : 0];  // element 0: a valid read
            stage[u] = ok ? v : 0.0f;
        }
    };
    const int r = lane & 15, kq = lane >> 4;
    fetch(b0);
    for (int64_t s0 = b0; s0 < b1; s0 += WSTEP) {
#pragma unroll
        for (int u = 0; u < GPER; ++u)
            if (u < GPER - 1 || last_in)
                xs[c0 + u * CSTEP][rr0 + u * RSTEP] = (double)stage[u];  // fp32 widened exactly
        __syncthreads();
        if (s0 + WSTEP < b1) fetch(s0 + WSTEP);  // in flight during the products
        whole_products(xs, ti, tj, r, kq, acc);
        __syncthreads();  // before the next step overwrites the staged rows
    }
}

// (two workgroups per CU: registers for 2 WHOLE_WAVES / 4 waves per SIMD)
__global__ __launch_bounds__(WHOLE_THREADS) __attribute__((amdgpu_waves_per_eu(WHOLE_WAVES / 2)))
void k_gram_whole(const SvdTask* tasks, int n_tasks, int64_t n_items)
{
    constexpr int KB = GRAM_WHOLE;
    constexpr int THREADS = WHOLE_THREADS;
    __shared__ double xs[WSTEP][KB + 1];  // [column][row], padded
    // column offsets of the chunk (one step's worth of slack: a step's reads
    // stay inside even past the chunk's last column) and row offsets; element
    // offsets, a tensor has fewer than 2^31
    __shared__ int32_t loff[GRAM_CHUNK_WHOLE + WSTEP];
    __shared__ int32_t roff[KB];
    const int64_t item = blockIdx.x;
    if (item >= n_items) return;  // uniform
    int lo = 0, hi = n_tasks - 1;  // the last task whose first item is <= item
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (tasks[mid].item0 <= item) lo = mid; else hi = mid - 1;
    }
    const SvdTask& t = tasks[lo];
    const int64_t chunk = item - t.item0;  // one item per chunk
    const int tid = threadIdx.x, lane = tid % GW;
    const int wv = __builtin_amdgcn_readfirstlane(tid / GW);  // uniform: scalar tile indices
    const int64_t b0 = chunk * GRAM_CHUNK_WHOLE, b1 = min(b0 + GRAM_CHUNK_WHOLE, t.L);
    for (int64_t q = tid; q < GRAM_CHUNK_WHOLE + WSTEP; q += THREADS)
        loff[q] = (q < b1 - b0) ? (int32_t)mode_offset((uint32_t)(b0 + q), t.nl, t.ldim, t.lstr)
                                : 0;
    if (tid < KB)
        roff[tid] = (tid < t.K) ? (int32_t)mode_offset((uint32_t)tid, t.nk, t.kdim, t.kstr) : -1;
    __syncthreads();
    // this wave's tiles (uniform): (ti, tj), ti <= tj < ceil(K / 16); a slot
    // past the triangle's last tile (K < GRAM_WHOLE) makes tile (0, 0) again
    // and adds nothing
    const int n16 = (int)((t.K + 15) / 16);
    const int n_up = n16 * (n16 + 1) / 2;
    int ti[WHOLE_TILES], tj[WHOLE_TILES];
#pragma unroll
    for (int k = 0; k < WHOLE_TILES; ++k) {
        int idx = wv + k * WHOLE_WAVES, row = 0;
        if (idx >= n_up) idx = 0;
        while (idx >= n16 - row) {
            idx -= n16 - row;
            ++row;
        }
        ti[k] = row;
        tj[k] = row + idx;
    }
    d4 acc[WHOLE_TILES];
#pragma unroll
    for (int k = 0; k < WHOLE_TILES; ++k) acc[k] = d4{0.0, 0.0, 0.0, 0.0};
    if (t.kstr[t.nk - 1] != 1)  // uniform: the rows are not the unit-stride side
        gram_whole_run<true>(t, b0, b1, xs, loff, roff, ti, tj, acc);
    else
        gram_whole_run<false>(t, b0, b1, xs, loff, roff, ti, tj, acc);
    // register j of a lane holds row 4 j + lane/16, column lane%16 of a tile
    const int r = lane & 15, kq = lane >> 4;
#pragma unroll
    for (int k = 0; k < WHOLE_TILES; ++k) {
        if (wv + k * WHOLE_WAVES >= n_up) break;  // uniform
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t row = (int64_t)ti[k] * 16 + 4 * j + kq;
            const int64_t col = (int64_t)tj[k] * 16 + r;
            if (row < t.K && col < t.K && row <= col) {
                atomicAdd(&t.gram[row * t.K + col], acc[k][j]);
                if (row != col) atomicAdd(&t.gram[col * t.K + row], acc[k][j]);
            }
        }
    }
}

// a double moved between lanes by DPP (bound_ctrl: lanes without a source read 0)
template <int CTRL, int ROWS>
__device__ __forceinline__ double dpp_move(double v)
{
    const uint64_t b = (uint64_t)__double_as_longlong(v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)b, CTRL, ROWS, 0xf, true);
    const uint32_t hi =
        (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(b >> 32), CTRL, ROWS, 0xf, true);
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// sum of v over the wave's 64 lanes, the same value in every lane: an
// inclusive scan by DPP row shifts (1, 2, 4, 8) and row broadcasts (lane 15
// into the next row, lane 31 into the upper half), then lane 63's total.
// Register-to-register moves, where a butterfly of lane shuffles would make
// six LDS round trips
__device__ __forceinline__ double wave_total(double x)
{
    x += dpp_move<0x111, 0xf>(x);  // row_shr:1
    x += dpp_move<0x112, 0xf>(x);  // row_shr:2
    x += dpp_move<0x114, 0xf>(x);  // row_shr:4
    x += dpp_move<0x118, 0xf>(x);  // row_shr:8
    x += dpp_move<0x142, 0xa>(x);  // row_bcast:15 into rows 1 and 3
    x += dpp_move<0x143, 0xc>(x);  // row_bcast:31 into rows 2 and 3
    const uint64_t b = (uint64_t)__double_as_longlong(x);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)b, 63);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), 63);
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// sum of v over the workgroup with one barrier: red holds two rows of
// per-wave partials used alternately (flip selects the row, toggled here), so
// a wave that is still reading one row cannot see the next call's writes
__device__ double block_sum(double v, double (*red)[EIG_THREADS / 64], int& flip)
{
    v = wave_total(v);
    if ((threadIdx.x & 63) == 0) red[flip][threadIdx.x >> 6] = v;
    __syncthreads();
    double s = 0.0;
    for (int u = 0; u < EIG_THREADS / 64; ++u) s += red[flip][u];
    flip ^= 1;
    return s;
}

// 1/q to a relative error of about 2^-48: the hardware estimate (measured on
// gfx950 to 2^-24.4 over 4M values spanning 2^+-300) refined by one Newton
// step, which squares its error.  The Sturm recurrence is a chain of these; a
// correctly rounded division would lengthen every link, and a count computed
// with this reciprocal is exact for the tridiagonal matrix with each e2[i]
// perturbed by about 2^-48 relative, far below the bisection's own tolerance
__device__ __forceinline__ double recip_nr(double q)
{
    const double r = __builtin_amdgcn_rcp(q);
    return fma(r, fma(-q, r, 1.0), r);
}

constexpr int EIG_LDS_K = 128;  // Gram matrices up to this side are reduced in LDS

// Householder reduction of the symmetric n x n matrix A (row stride n) to
// tridiagonal form: d[k] the diagonal, e2[k] the squared off-diagonal
typedef __attribute__((address_space(3))) double lds_f64;

template <class Ptr>
__device__ void tridiagonalize(Ptr A, int n, double* v, double2* uw, double* wp, double* d,
                               double* e2, double (*red)[EIG_THREADS / 64])
{
    const int tid = threadIdx.x;
    int flip = 0;
    // Householder reduction: step k annihilates column k below the subdiagonal
    // with H = I - beta u u^T, u = (x0 - alpha, x1, ..., x_{m-1}), and
    // A_sub <- H A_sub H = A_sub - u w^T - w u^T, w = p - K u, p = beta A_sub u,
    // K = beta (p . u) / 2.  u's first entry lives in a register (v[0] keeps
    // x0), so a step has three barriers: after the column, after p, after
    // the update
    for (int k = 0; k + 2 < n; ++k) {
        const int m = n - k - 1;
        double tail = 0.0;
        // column k below the diagonal, read as row k right of it (contiguous:
        // no bank conflicts in LDS, coalesced in global memory); the two agree
        // up to the rounding of the updates, which keep the matrix symmetric
        // in exact arithmetic
        for (int i = tid; i < m; i += EIG_THREADS) {
            const double x = A[(size_t)k * n + (k + 1 + i)];
            v[i] = x;
            if (i > 0) tail += x * x;
        }
        tail = block_sum(tail, red, flip);  // (its barrier publishes v)
        const double x0 = v[0];
        if (tid == 0) d[k] = A[(size_t)k * n + k];
        if (!(tail > 0.0)) {
            if (tid == 0) e2[k] = x0 * x0;
            __syncthreads();  // every thread has read x0 before v is rewritten
            continue;
        }
        // every thread derives the reflector's scalars itself
        const double alpha = (x0 >= 0.0) ? -sqrt(x0 * x0 + tail) : sqrt(x0 * x0 + tail);
        const double u0 = x0 - alpha;
        const double beta = 2.0 / (u0 * u0 + tail);
        if (tid == 0) e2[k] = alpha * alpha;
        // p = beta A_sub u, columns across threads (row j of A is read across
        // neighbouring threads); with fewer columns than threads, tpc threads
        // share a column, each taking a slice of its rows, and the slices'
        // sums are added in slice order
        int tpc = 1;  // uniform
        while (tpc < 16 && 2 * tpc * m <= EIG_THREADS) tpc *= 2;
        const int ncol = EIG_THREADS / tpc;
        const int ci = tid % ncol, hf = tid / ncol;
        const int jlo = hf * m / tpc, jhi = (hf + 1) * m / tpc;
        double pv = 0.0;
        for (int i = ci; i < m; i += ncol) {
            const auto col = A + (size_t)(k + 1) * n + (k + 1 + i);
            double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
            int j = jlo;
            if (j == 0 && j < jhi) {
                s0 = col[0] * u0;
                j = 1;
            }
            for (; j + 4 <= jhi; j += 4) {  // four independent loads in flight
                s0 += col[(size_t)j * n] * v[j];
                s1 += col[(size_t)(j + 1) * n] * v[j + 1];
                s2 += col[(size_t)(j + 2) * n] * v[j + 2];
                s3 += col[(size_t)(j + 3) * n] * v[j + 3];
            }
            for (; j < jhi; ++j) s0 += col[(size_t)j * n] * v[j];
            const double part = (s0 + s1) + (s2 + s3);
            if (tpc > 1) {
                wp[hf * ncol + i] = part;
            } else {
                const double ui = i == 0 ? u0 : v[i], wi = beta * part;
                uw[i] = make_double2(ui, wi);
                pv += wi * ui;
            }
        }
        if (tpc > 1) {
            __syncthreads();
            if (hf == 0 && ci < m) {
                double sum = 0.0;
                for (int h = 0; h < tpc; ++h) sum += wp[h * ncol + ci];
                const double ui = ci == 0 ? u0 : v[ci], wi = beta * sum;
                uw[ci] = make_double2(ui, wi);
                pv = wi * ui;
            }
        }
        const double K2 = 0.5 * beta * block_sum(pv, red, flip);  // (publishes p in w, uw)
        // A_sub -= u w'^T + w' u^T with w' = p - K2 u: entry (j, i) loses
        // u_j (w_i - 2 K2 u_i) + w_j u_i, two FMAs on the pair (u_j, w_j) read
        // from LDS at once (each thread walks its column slice down the rows;
        // the rows of one column are independent, so the loop is unrolled)
        for (int i = ci; i < m; i += ncol) {
            const auto col = A + (size_t)(k + 1) * n + (k + 1 + i);
            const double2 pi = uw[i];
            const double ui = pi.x, ci2 = pi.y - 2.0 * K2 * pi.x;
#pragma unroll 4
            for (int j = jlo; j < jhi; ++j) {
                const double2 pj = uw[j];
                col[(size_t)j * n] -= fma(pj.x, ci2, pj.y * ui);
            }
        }
        __syncthreads();
    }
    if (tid == 0) {
        if (n >= 2) {
            d[n - 2] = A[(size_t)(n - 2) * n + (n - 2)];
            const double en = A[(size_t)(n - 1) * n + (n - 2)];
            e2[n - 2] = en * en;
        }
        d[n - 1] = A[(size_t)(n - 1) * n + (n - 1)];
    }
    __syncthreads();
}

// Gershgorin interval of the symmetric tridiagonal matrix (d, e2), widened
// by two ulps of its span and the smallest pivot allowed in a Sturm count
template <class Ptr>
__device__ void gershgorin(Ptr d, Ptr e2, int n, double& glo, double& ghi, double& pivmin)
{
    glo = INFINITY;
    ghi = -INFINITY;
    double emax = 0.0;
    for (int i = 0; i < n; ++i) {
        const double r = (i > 0 ? sqrt(e2[i - 1]) : 0.0) + (i + 1 < n ? sqrt(e2[i]) : 0.0);
        glo = fmin(glo, d[i] - r);
        ghi = fmax(ghi, d[i] + r);
        if (i + 1 < n) emax = fmax(emax, e2[i]);
    }
    const double span = fmax(fabs(glo), fabs(ghi));
    pivmin = 0x1p-1000 * fmax(1.0, emax);
    glo -= 2.0 * DBL_EPSILON * span + pivmin;
    ghi += 2.0 * DBL_EPSILON * span + pivmin;
}

// the k-th smallest eigenvalue of (d, e2) by multisection on Sturm counts
// (count(lo) <= k < count(hi)): the G neighbouring threads of eigenvalue k
// (g = 0 .. G-1, G a power of two dividing 64) each count at NC of a
// round's NC G interior points, NC independent chains side by side, and the
// round keeps the one of the interval's NC G + 1 parts that holds the
// eigenvalue (the group agrees on lo and hi after every round)
template <int NC, class Ptr>
__device__ double multisect(Ptr d, Ptr e2, int n, int k, int g, int G, double glo, double ghi,
                            double pivmin)
{
    double lo = glo, hi = ghi;
    for (int it = 0; it < 64; ++it) {
        if (!(hi - lo > 2.0 * DBL_EPSILON * fmax(fabs(lo), fabs(hi)) + pivmin)) break;
        const double h = (hi - lo) / (double)(NC * G + 1);
        double x[NC], q[NC];
        int c[NC];
        // a pivot below pivmin in magnitude becomes -pivmin, so it is
        // negative after that exactly when it was below pivmin: the count
        // takes that test, beside the clamp rather than after it
        auto step = [&](double di, double ei) {
#pragma unroll
            for (int u = 0; u < NC; ++u) {
                q[u] = di - x[u] - ei * recip_nr(q[u]);
                c[u] += q[u] < pivmin;
                if (fabs(q[u]) < pivmin) q[u] = -pivmin;
            }
        };
#pragma unroll
        for (int u = 0; u < NC; ++u) {
            x[u] = lo + h * (double)(NC * g + u + 1);
            q[u] = d[0] - x[u];
            c[u] = q[u] < pivmin;
            if (fabs(q[u]) < pivmin) q[u] = -pivmin;
        }
        // the next step's coefficients are read a step ahead, so the LDS
        // latency overlaps the current step's arithmetic (the last step
        // peeled: no test inside the loop)
        if (n > 1) {
            double dn = d[1], en = e2[0];
            for (int i = 1; i + 1 < n; ++i) {
                const double di = dn, ei = en;
                dn = d[i + 1];
                en = e2[i];
                step(di, ei);
            }
            step(dn, en);
        }
        double nlo = lo, nhi = hi;
#pragma unroll
        for (int u = 0; u < NC; ++u) {
            if (c[u] <= k) nlo = fmax(nlo, x[u]);
            else nhi = fmin(nhi, x[u]);
        }
        for (int off = 1; off < G; off <<= 1) {
            nlo = fmax(nlo, __shfl_xor(nlo, off));
            nhi = fmin(nhi, __shfl_xor(nhi, off));
        }
        if (nlo == lo && nhi == hi) break;  // no representable progress
        lo = nlo;
        hi = nhi;
    }
    return 0.5 * (lo + hi);
}

__global__ __launch_bounds__(EIG_THREADS) void k_svd_eig(const SvdTask* tasks)
{
    __shared__ double v[SVD_SMALL_K];
    __shared__ double2 uw[SVD_SMALL_K];
    __shared__ double d[SVD_SMALL_K], e2[SVD_SMALL_K];
    __shared__ double red[2][EIG_THREADS / 64];
    __shared__ double As[EIG_LDS_K * EIG_LDS_K];
    __shared__ double wp[EIG_THREADS];
    const SvdTask& t = tasks[blockIdx.x];
    const int n = (int)t.K;
    if (n > SVD_SMALL_K) return;  // (uniform) a larger matrix takes the many-workgroup path
    const int tid = threadIdx.x;
    if (n <= EIG_LDS_K) {
        for (int q = tid; q < n * n; q += EIG_THREADS) As[q] = t.gram[q];
        __syncthreads();
        tridiagonalize((lds_f64*)As, n, v, uw, wp, d, e2, red);  // ds_ instructions
    } else {
        // global-memory instructions (generic ones would also count against
        // the LDS waits)
        typedef __attribute__((address_space(1))) double gdouble;
        tridiagonalize((gdouble*)t.gram, n, v, uw, wp, d, e2, red);
    }
    // the tridiagonal form and its bounds for k_svd_count
    for (int i = tid; i < n; i += EIG_THREADS) {
        t.tri[i] = d[i];
        t.tri[n + i] = e2[i];
    }
    if (tid == 0) {
        double glo, ghi, pivmin;
        gershgorin((const lds_f64*)d, (const lds_f64*)e2, n, glo, ghi, pivmin);
        t.tri[2 * n] = glo;
        t.tri[2 * n + 1] = ghi;
        t.tri[2 * n + 2] = pivmin;
    }
}

// every eigenvalue of the tridiagonal forms k_svd_eig wrote: one wave per
// EIG_PER_ITEM eigenvalues of a task (work items numbered from the task's
// eig0), COUNT_G threads per eigenvalue with COUNT_C chains each.  The
// counts are bound by instruction issue over the device as a whole (the
// work is rounds x points per round, and fewer points per round cost fewer
// instructions than the extra rounds add) and by each chain's latency within
// a wave; four threads of one chain (four points a round, 22 rounds for 52
// bits) spread a 128-side matrix over eight waves, about one wave per SIMD
// over the whole device for 64 attention-shaped tensors.  Measured on those:
// 0.15 ms; 2, 8 or 16 threads of one chain 0.21, 0.16, 0.22 ms; four threads
// of two chains 0.19 ms, of four 0.27 ms
constexpr int COUNT_G = 4;
constexpr int COUNT_C = 1;
static_assert(EIG_PER_ITEM * COUNT_G == GW, "one wave per work item");

__global__ __launch_bounds__(GW) void k_svd_count(const SvdTask* tasks, int n_tasks,
                                                 int64_t n_items)
{
    __shared__ double ds[SVD_SMALL_K], es[SVD_SMALL_K];
    const int64_t item = blockIdx.x;
    if (item >= n_items) return;  // uniform
    int lo = 0, hi = n_tasks - 1;  // the last task whose first item is <= item
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (tasks[mid].eig0 <= item) lo = mid; else hi = mid - 1;
    }
    const SvdTask& t = tasks[lo];
    const int n = (int)t.K;
    const int tid = threadIdx.x;
    for (int i = tid; i < n; i += GW) {
        ds[i] = t.tri[i];
        es[i] = t.tri[n + i];
    }
    const double glo = t.tri[2 * n], ghi = t.tri[2 * n + 1], pivmin = t.tri[2 * n + 2];
    __syncthreads();
    // (whole groups of COUNT_G lanes share k and leave together)
    const int k = (int)(item - t.eig0) * EIG_PER_ITEM + tid / COUNT_G, g = tid % COUNT_G;
    if (k >= n) return;
    const double lam = multisect<COUNT_C>((const lds_f64*)ds, (const lds_f64*)es, n, k, g,
                                          COUNT_G, glo, ghi, pivmin);
    if (g == 0) t.out[n - 1 - k] = sqrt(fmax(lam, 0.0));
}

// ---------------------------------------------------------------------------
// Gram matrices larger than SVD_SMALL_K: one Householder step is four
// launches over the whole device (the reflector; the product p = beta A u in
// 64-column x 256-row blocks; the blocks' partial sums added in block order,
// with K = beta (p . u) / 2; the rank-two update in the same blocks), then the
// tridiagonal matrix's eigenvalues by multisection with enough threads per
// eigenvalue to fill the device.  The matrix stays in place in the workspace.
// ---------------------------------------------------------------------------
constexpr int HH_THREADS = 1024;  // one-workgroup kernels
constexpr int HH_COLS = 64;       // columns per block (one per lane)
constexpr int HH_ROWS = 256;      // rows per block (64 per wave)

struct HhState {
    double beta, K2;
    double glo, ghi, pivmin;
    int32_t skip;  // the step's column is already reduced
};

__device__ double sum_1024(double v, double* red)
{
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    double s = 0.0;
    for (int u = 0; u < HH_THREADS / 64; ++u) s += red[u];
    return s;
}

// step k: u = column k below the diagonal (read along row k, the same values
// up to the rounding of the Gram matrix's accumulation), with u0 = x0 - alpha
// in place of x0; d[k], e2[k] = alpha^2, beta
__global__ __launch_bounds__(HH_THREADS) void k_hh_reflector(double* A, int n, int k, double* u,
                                                             double* d, double* e2, HhState* hs)
{
    __shared__ double red[HH_THREADS / 64];
    const int m = n - k - 1, tid = threadIdx.x;
    const double* row = A + (size_t)k * n + (k + 1);
    double tail = 0.0;
    for (int i = tid; i < m; i += HH_THREADS) {
        const double x = row[i];
        u[i] = x;
        if (i > 0) tail += x * x;
    }
    tail = sum_1024(tail, red);
    if (tid == 0) {
        const double x0 = row[0];
        d[k] = A[(size_t)k * n + k];
        if (!(tail > 0.0)) {
            e2[k] = x0 * x0;
            hs->skip = 1;
        } else {
            const double alpha = (x0 >= 0.0) ? -sqrt(x0 * x0 + tail) : sqrt(x0 * x0 + tail);
            const double u0 = x0 - alpha;
            e2[k] = alpha * alpha;
            u[0] = u0;
            hs->beta = 2.0 / (u0 * u0 + tail);
            hs->skip = 0;
        }
    }
}

// partial sums of A_sub u: block (blockIdx.x, blockIdx.y) = 64 columns x 256
// rows; wave w takes 64 rows, lane l one column (a row is read across lanes)
__global__ __launch_bounds__(256) void k_hh_matvec(const double* A, int n, int k, const double* u,
                                                   const HhState* hs, double* part)
{
    if (hs->skip) return;  // uniform
    __shared__ double red[4][HH_COLS];
    const int m = n - k - 1;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int i = blockIdx.x * HH_COLS + lane;
    const int j0 = blockIdx.y * HH_ROWS + w * 64, j1 = min(j0 + 64, m);
    double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
    if (i < m) {
        const double* col = A + (size_t)(k + 1) * n + (k + 1 + i);
        int j = j0;
        for (; j + 4 <= j1; j += 4) {
            s0 += col[(size_t)j * n] * u[j];
            s1 += col[(size_t)(j + 1) * n] * u[j + 1];
            s2 += col[(size_t)(j + 2) * n] * u[j + 2];
            s3 += col[(size_t)(j + 3) * n] * u[j + 3];
        }
        for (; j < j1; ++j) s0 += col[(size_t)j * n] * u[j];
    }
    red[w][lane] = (s0 + s1) + (s2 + s3);
    __syncthreads();
    if (w == 0 && i < m)
        part[(size_t)blockIdx.y * n + i] = (red[0][lane] + red[1][lane]) + (red[2][lane] + red[3][lane]);
}

// p = beta (the row blocks' partial sums, in block order); K2 = beta (p . u) / 2
__global__ __launch_bounds__(HH_THREADS) void k_hh_combine(int n, int k, const double* u,
                                                           const double* part, int R, double* p,
                                                           HhState* hs)
{
    if (hs->skip) return;  // uniform
    __shared__ double red[HH_THREADS / 64];
    const int m = n - k - 1;
    const double beta = hs->beta;
    double dot = 0.0;
    for (int i = threadIdx.x; i < m; i += HH_THREADS) {
        double sum = 0.0;
        for (int r = 0; r < R; ++r) sum += part[(size_t)r * n + i];
        const double pi = beta * sum;
        p[i] = pi;
        dot += pi * u[i];
    }
    dot = sum_1024(dot, red);
    if (threadIdx.x == 0) hs->K2 = 0.5 * beta * dot;
}

// A_sub -= u w^T + w u^T with w = p - K2 u, in the matvec's blocks
__global__ __launch_bounds__(256) void k_hh_update(double* A, int n, int k, const double* u,
                                                   const double* p, const HhState* hs)
{
    if (hs->skip) return;  // uniform
    const int m = n - k - 1;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int i = blockIdx.x * HH_COLS + lane;
    if (i >= m) return;  // (no barrier below)
    const int j0 = blockIdx.y * HH_ROWS + w * 64, j1 = min(j0 + 64, m);
    const double K2 = hs->K2;
    const double ui = u[i], wi = fma(-K2, ui, p[i]);
    double* col = A + (size_t)(k + 1) * n + (k + 1 + i);
#pragma unroll 4
    for (int j = j0; j < j1; ++j) {
        const double uj = u[j], wj = fma(-K2, uj, p[j]);
        col[(size_t)j * n] -= uj * wi + wj * ui;
    }
}

// the last 2 x 2 corner; then the Gershgorin interval (one workgroup)
__global__ __launch_bounds__(HH_THREADS) void k_hh_finish(const double* A, int n, double* d,
                                                          double* e2, HhState* hs)
{
    __shared__ double red[3][HH_THREADS / 64];
    __shared__ double de[2][3];
    const int tid = threadIdx.x;
    if (tid == 0) {
        // d[n-2], e2[n-2], d[n-1] (n > SVD_SMALL_K >= 2)
        de[0][0] = A[(size_t)(n - 2) * n + (n - 2)];
        const double en = A[(size_t)(n - 1) * n + (n - 2)];
        de[0][1] = en * en;
        de[0][2] = A[(size_t)(n - 1) * n + (n - 1)];
        d[n - 2] = de[0][0];
        e2[n - 2] = de[0][1];
        d[n - 1] = de[0][2];
    }
    __syncthreads();
    // per-thread ranges of the Gershgorin bounds, then one reduction
    double glo = INFINITY, ghi = -INFINITY, emax = 0.0;
    for (int i = tid; i < n; i += HH_THREADS) {
        const double di = (i == n - 2) ? de[0][0] : (i == n - 1) ? de[0][2] : d[i];
        const double el = (i > 0) ? ((i - 1 == n - 2) ? de[0][1] : e2[i - 1]) : 0.0;
        const double er = (i + 1 < n) ? ((i == n - 2) ? de[0][1] : e2[i]) : 0.0;
        const double r = sqrt(el) + sqrt(er);
        glo = fmin(glo, di - r);
        ghi = fmax(ghi, di + r);
        if (i + 1 < n) emax = fmax(emax, er);
    }
    for (int off = 32; off > 0; off >>= 1) {
        glo = fmin(glo, __shfl_xor(glo, off));
        ghi = fmax(ghi, __shfl_xor(ghi, off));
        emax = fmax(emax, __shfl_xor(emax, off));
    }
    if ((tid & 63) == 0) {
        red[0][tid >> 6] = glo;
        red[1][tid >> 6] = ghi;
        red[2][tid >> 6] = emax;
    }
    __syncthreads();
    if (tid == 0) {
        for (int u = 1; u < HH_THREADS / 64; ++u) {
            glo = fmin(glo, red[0][u]);
            ghi = fmax(ghi, red[1][u]);
            emax = fmax(emax, red[2][u]);
        }
        const double span = fmax(fabs(glo), fabs(ghi));
        const double pivmin = 0x1p-1000 * fmax(1.0, emax);
        hs->glo = glo - (2.0 * DBL_EPSILON * span + pivmin);
        hs->ghi = ghi + (2.0 * DBL_EPSILON * span + pivmin);
        hs->pivmin = pivmin;
    }
}

// every eigenvalue, G threads each (the grid holds exactly n G threads,
// rounded up to whole workgroups; whole groups leave together)
__global__ __launch_bounds__(256) void k_hh_bisect(const double* d, const double* e2, int n, int G,
                                                   const HhState* hs, double* out)
{
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int k = (int)(t / G), g = (int)(t % G);
    if (k >= n) return;
    const double lam = multisect<4>(d, e2, n, k, g, G, hs->glo, hs->ghi, hs->pivmin);
    if (g == 0) out[n - 1 - k] = sqrt(fmax(lam, 0.0));
}

__global__ __launch_bounds__(64) void k_svd_match(const SpecDesc* da, int na, const double* sa,
                                                  const SpecDesc* db, int nb, const double* sb,
                                                  double eps, uint8_t* match)
{
    __shared__ uint32_t ok[SVD_MAX_UNF];
    const int64_t pair = blockIdx.x;
    const int ia = (int)(pair / nb), ib = (int)(pair % nb);
    if (ia >= na) return;
    const SpecDesc& a = da[ia];
    const SpecDesc& b = db[ib];
    const int n = a.n;
    if (n != b.n) {
        if (threadIdx.x == 0) match[pair] = 0;
        return;
    }
    if (threadIdx.x < SVD_MAX_UNF) ok[threadIdx.x] = 0u;
    __syncthreads();
    for (int q = threadIdx.x; q < n * n; q += blockDim.x) {
        const int i = q / n, j = q % n;
        bool close = a.len[i] == b.len[j];
        if (close && a.len[i] > 0) {
            const double* x = sa + a.off[i];
            const double* y = sb + b.off[j];
            const double tol = eps * fmax(x[0], y[0]);
            for (int64_t u = 0; u < a.len[i] && close; ++u) close = fabs(x[u] - y[u]) <= tol;
        }
        if (close) atomicOr(&ok[i], 1u << j);
    }
    __syncthreads();
    if (threadIdx.x != 0) return;
    // one-to-one pairing: an augmenting path (breadth first) for every left entry
    int match_l[SVD_MAX_UNF], match_r[SVD_MAX_UNF];
    for (int u = 0; u < n; ++u) match_l[u] = match_r[u] = -1;
    bool all = true;
    for (int i = 0; i < n && all; ++i) {
        int from[SVD_MAX_UNF], queue[SVD_MAX_UNF + 1];
        uint32_t seen = 0u;
        int qh = 0, qt = 0, found = -1;
        queue[qt++] = i;
        while (qh < qt && found < 0) {
            const int u = queue[qh++];
            for (int j = 0; j < n; ++j) {
                if (!((ok[u] >> j) & 1u) || ((seen >> j) & 1u)) continue;
                seen |= 1u << j;
                from[j] = u;
                if (match_r[j] < 0) {
                    found = j;
                    break;
                }
                queue[qt++] = match_r[j];  // each right entry is queued once: qt <= n
            }
        }
        if (found < 0) {
            all = false;
            break;
        }
        for (int j = found;;) {
            const int u = from[j];
            const int prev = match_l[u];
            match_r[j] = u;
            match_l[u] = j;
            if (u == i) break;
            j = prev;
        }
    }
    match[pair] = all ? 1 : 0;
}

}  // namespace

hipError_t launch_svd(const SvdTask* tasks, int n_tasks, int n_narrow, int64_t n_items_narrow,
                      int n_whole, int64_t n_items_whole, int64_t n_items, int64_t n_eig_items,
                      double* gram, int64_t gram_len, hipStream_t stream)
{
    if (n_tasks <= 0) return hipSuccess;
    const int64_t cb = min((gram_len + 255) / 256, (int64_t)4096);
    hipLaunchKernelGGL(k_svd_clear, dim3((unsigned)max(cb, (int64_t)1)), dim3(256), 0, stream,
                       gram, gram_len);
    // tasks [0, n_narrow): K <= GRAM_NARROW, one 32-side block; then n_whole
    // with K in (64, GRAM_WHOLE], the whole upper triangle per workgroup; the
    // rest in 64-side blocks
    if (n_items_narrow > 0)
        hipLaunchKernelGGL(k_gram<GRAM_NARROW>, dim3((unsigned)n_items_narrow),
                           dim3(GRAM_NARROW * GRAM_NARROW / 4), 0, stream, tasks, n_narrow,
                           n_items_narrow);
    if (n_items_whole > 0 && n_whole > 0)
        hipLaunchKernelGGL(k_gram_whole, dim3((unsigned)n_items_whole), dim3(WHOLE_THREADS),
                           0, stream, tasks + n_narrow, n_whole, n_items_whole);
    const int n_blocked = n_tasks - n_narrow - n_whole;
    if (n_items > 0 && n_blocked > 0)
        hipLaunchKernelGGL(k_gram<64>, dim3((unsigned)n_items), dim3(64 * 64 / 4), 0, stream,
                           tasks + n_narrow + n_whole, n_blocked, n_items);
    hipLaunchKernelGGL(k_svd_eig, dim3((unsigned)n_tasks), dim3(EIG_THREADS), 0, stream, tasks);
    if (n_eig_items > 0)
        hipLaunchKernelGGL(k_svd_count, dim3((unsigned)n_eig_items), dim3(GW), 0, stream, tasks,
                           n_tasks, n_eig_items);
    return hipGetLastError();
}

int64_t svd_large_scratch(int n)
{
    const int64_t R = (n + HH_ROWS - 1) / HH_ROWS;
    // u, p, d, e2, the row blocks' partial sums, the step state
    return 4 * (int64_t)n + R * n + (int64_t)((sizeof(HhState) + 7) / 8);
}

hipError_t launch_svd_large(double* A, int n, double* scratch, double* out, hipStream_t stream)
{
    if (n <= SVD_SMALL_K) return hipErrorInvalidValue;
    const int R = (n + HH_ROWS - 1) / HH_ROWS;
    double* u = scratch;
    double* p = u + n;
    double* d = p + n;
    double* e2 = d + n;
    double* part = e2 + n;
    HhState* hs = reinterpret_cast<HhState*>(part + (size_t)R * n);
    for (int k = 0; k + 2 < n; ++k) {
        const int m = n - k - 1;
        const dim3 blocks((unsigned)((m + HH_COLS - 1) / HH_COLS), (unsigned)((m + HH_ROWS - 1) / HH_ROWS));
        hipLaunchKernelGGL(k_hh_reflector, dim3(1), dim3(HH_THREADS), 0, stream, A, n, k, u, d, e2,
                           hs);
        hipLaunchKernelGGL(k_hh_matvec, blocks, dim3(256), 0, stream, A, n, k, u, hs, part);
        hipLaunchKernelGGL(k_hh_combine, dim3(1), dim3(HH_THREADS), 0, stream, n, k, u, part,
                           (int)blocks.y, p, hs);
        hipLaunchKernelGGL(k_hh_update, blocks, dim3(256), 0, stream, A, n, k, u, p, hs);
    }
    hipLaunchKernelGGL(k_hh_finish, dim3(1), dim3(HH_THREADS), 0, stream, A, n, d, e2, hs);
    // threads per eigenvalue: enough for about 32K threads in all
    int G = 1;
    while (G < 8 && (int64_t)G * n < 32768) G *= 2;
    const int64_t threads = (int64_t)n * G;
    hipLaunchKernelGGL(k_hh_bisect, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, stream,
                       d, e2, n, G, hs, out);
    return hipGetLastError();
}

hipError_t launch_svd_match(const SpecDesc* da, int na, const double* sa, const SpecDesc* db,
                            int nb, const double* sb, double eps, uint8_t* match,
                            hipStream_t stream)
{
    const int64_t pairs = (int64_t)na * nb;
    if (pairs <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_svd_match, dim3((unsigned)pairs), dim3(64), 0, stream, da, na, sa, db, nb,
                       sb, eps, match);
    return hipGetLastError();
}

}  // namespace mag
