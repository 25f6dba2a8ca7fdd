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
//   unfolding's mixed-radix offsets.
// k_svd_eig: one workgroup per task: Householder reduction of the Gram
//   matrix (in LDS up to side 128, else in place in global memory) to
//   tridiagonal form, then every eigenvalue by multisection on Sturm counts
//   (the count of eigenvalues below x), sigma = sqrt(max(lambda, 0)), written
//   in descending order.
// k_svd_match: one workgroup per tensor pair: which spectra of the two lists
//   are close, then a one-to-one pairing by augmenting paths.

#include <cfloat>

#include "mag_internal.hpp"

namespace mag {

namespace {

constexpr int GW = 64;
constexpr int EIG_THREADS = 256;

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

// One workgroup of 16 waves per (task, 64 x 64 block of the upper triangle,
// chunk of GRAM_CHUNK columns).  Each 64-column step stages the block's 64
// rows of each operand in LDS as fp64 (one global load per element, rows
// fastest across threads, so a unit-stride row mode gives coalesced loads);
// wave w then multiplies tile (w / 4, w % 4) from LDS with 16 MFMA steps.
constexpr int GB = 64;              // block side
constexpr int GSTEP = 64;           // columns staged per step
constexpr int GTHREADS = 1024;      // 16 waves: one per 16 x 16 tile of the block

__global__ __launch_bounds__(GTHREADS) void k_gram(const SvdTask* tasks, int n_tasks,
                                                   int64_t n_items)
{
    __shared__ double xa[GSTEP][GB + 1], xb[GSTEP][GB + 1];  // [column][row], padded
    __shared__ int32_t loff[GRAM_CHUNK];
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
    int bi = 0, rowlen = t.nt;  // nt counts 64-row blocks here
    while (pr >= rowlen && rowlen > 0) {
        pr -= rowlen;
        ++bi;
        --rowlen;
    }
    const int bj = bi + (int)pr;
    const int tid = threadIdx.x, lane = tid % GW, wv = tid / GW;
    const int64_t b0 = chunk * GRAM_CHUNK, b1 = min(b0 + GRAM_CHUNK, t.L);
    for (int64_t q = tid; q < b1 - b0; q += GTHREADS)
        loff[q] = (int32_t)mode_offset((uint32_t)(b0 + q), t.nl, t.ldim, t.lstr);
    if (tid < 2 * GB) {
        const int side = tid / GB, r = tid % GB;
        const int64_t row = (int64_t)(side ? bj : bi) * GB + r;
        roff[side][r] = (row < t.K) ? mode_offset((uint32_t)row, t.nk, t.kdim, t.kstr) : -1;
    }
    __syncthreads();
    const int ti = wv / 4, tj = wv % 4;  // this wave's tile inside the block
    const int r = lane & 15, kq = lane >> 4;
    d4 acc = {0.0, 0.0, 0.0, 0.0};
    for (int64_t s0 = b0; s0 < b1; s0 += GSTEP) {
        const int cols = (int)min((int64_t)GSTEP, b1 - s0);
        // stage: element (row, column) of each operand; rows fastest
        for (int q = tid; q < 2 * GB * GSTEP; q += GTHREADS) {
            const int side = q / (GB * GSTEP), rem = q % (GB * GSTEP);
            const int c = rem / GB, rr = rem % GB;
            const int64_t ro = roff[side][rr];
            double x = 0.0;
            if (c < cols && ro >= 0) x = (double)t.data[ro + loff[s0 - b0 + c]];
            (side ? xb : xa)[c][rr] = x;
        }
        __syncthreads();
#pragma unroll 4
        for (int c = 0; c < GSTEP; c += 4) {
            const double a = xa[c + kq][ti * 16 + r];
            const double b = xb[c + kq][tj * 16 + r];
            acc = __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, acc, 0, 0, 0);
        }
        __syncthreads();  // before the next step overwrites the staged rows
    }
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

__device__ double block_sum(double v, double* red)
{
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    __syncthreads();  // earlier readers of red are done
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    double s = 0.0;
    for (int u = 0; u < EIG_THREADS / 64; ++u) s += red[u];
    return s;
}

// 1/q within about an ulp: the hardware estimate refined by two Newton steps
// (the Sturm recurrence is a chain of these; a correctly rounded division
// would lengthen every link)
__device__ __forceinline__ double recip_nr(double q)
{
    double r = __builtin_amdgcn_rcp(q);
    r = fma(r, fma(-q, r, 1.0), r);
    r = fma(r, fma(-q, r, 1.0), r);
    return r;
}

constexpr int EIG_LDS_K = 128;  // Gram matrices up to this side are reduced in LDS

// Householder reduction of the symmetric n x n matrix A (row stride n) to
// tridiagonal form: d[k] the diagonal, e2[k] the squared off-diagonal
typedef __attribute__((address_space(3))) double lds_f64;

template <class Ptr>
__device__ void tridiagonalize(Ptr A, int n, double* v, double* w, double (*w2)[EIG_THREADS / 2],
                               double* d, double* e2, double* red)
{
    const int tid = threadIdx.x;
    // Householder reduction: step k annihilates column k below the subdiagonal
    for (int k = 0; k + 2 < n; ++k) {
        const int m = n - k - 1;
        double tail = 0.0;
        for (int i = tid; i < m; i += EIG_THREADS) {
            const double x = A[(size_t)(k + 1 + i) * n + k];
            v[i] = x;
            if (i > 0) tail += x * x;
        }
        tail = block_sum(tail, red);  // (its barriers publish v)
        const double x0 = v[0];
        if (tid == 0) d[k] = A[(size_t)k * n + k];
        if (!(tail > 0.0)) {
            if (tid == 0) e2[k] = x0 * x0;
            __syncthreads();
            continue;
        }
        const double alpha = (x0 >= 0.0) ? -sqrt(x0 * x0 + tail) : sqrt(x0 * x0 + tail);
        const double v0 = x0 - alpha;
        const double beta = 2.0 / (v0 * v0 + tail);
        if (tid == 0) e2[k] = alpha * alpha;
        __syncthreads();
        if (tid == 0) v[0] = v0;
        __syncthreads();
        // p = beta A_sub v (columns by threads: row j of A is read across
        // threads); with at most half as many columns as threads, two threads
        // share a column, each taking half of the rows
        const bool split = m <= EIG_THREADS / 2;
        const int ci = split ? tid % (EIG_THREADS / 2) : tid;
        const int hf = split ? tid / (EIG_THREADS / 2) : 0;
        const int jlo = split ? hf * (m / 2) : 0, jhi = split ? (hf ? m : m / 2) : m;
        double pv = 0.0;
        for (int i = ci; i < m; i += (split ? m + 1 : EIG_THREADS)) {
            const auto col = A + (size_t)(k + 1) * n + (k + 1 + i);
            double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
            int j = jlo;
            for (; j + 4 <= jhi; j += 4) {  // four independent loads in flight
                s0 += col[(size_t)j * n] * v[j];
                s1 += col[(size_t)(j + 1) * n] * v[j + 1];
                s2 += col[(size_t)(j + 2) * n] * v[j + 2];
                s3 += col[(size_t)(j + 3) * n] * v[j + 3];
            }
            for (; j < jhi; ++j) s0 += col[(size_t)j * n] * v[j];
            const double part = beta * ((s0 + s1) + (s2 + s3));
            if (split) {
                w2[hf][i] = part;
            } else {
                w[i] = part;
                pv += part * v[i];
            }
        }
        if (split) {
            __syncthreads();
            if (hf == 0 && ci < m) {
                w[ci] = w2[0][ci] + w2[1][ci];
                pv = w[ci] * v[ci];
            }
        }
        const double K2 = 0.5 * beta * block_sum(pv, red);
        for (int i = tid; i < m; i += EIG_THREADS) w[i] -= K2 * v[i];
        __syncthreads();
        // A_sub -= v w^T + w v^T (each thread walks its columns down the rows;
        // the rows of one column are independent, so the loop is unrolled)
        for (int i = ci; i < m; i += (split ? m + 1 : EIG_THREADS)) {
            const auto col = A + (size_t)(k + 1) * n + (k + 1 + i);
            const double vi = v[i], wi = w[i];
#pragma unroll 8
            for (int j = jlo; j < jhi; ++j) col[(size_t)j * n] -= v[j] * wi + w[j] * vi;
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

__global__ __launch_bounds__(EIG_THREADS) void k_svd_eig(const SvdTask* tasks)
{
    __shared__ double v[SVD_MAX_K], w[SVD_MAX_K];
    __shared__ double d[SVD_MAX_K], e2[SVD_MAX_K];
    __shared__ double red[EIG_THREADS / 64];
    __shared__ double As[EIG_LDS_K * EIG_LDS_K];
    __shared__ double w2[2][EIG_THREADS / 2];
    const SvdTask& t = tasks[blockIdx.x];
    const int n = (int)t.K;
    const int tid = threadIdx.x;
    if (n <= EIG_LDS_K) {
        for (int q = tid; q < n * n; q += EIG_THREADS) As[q] = t.gram[q];
        __syncthreads();
        tridiagonalize((lds_f64*)As, n, v, w, w2, d, e2, red);  // ds_ instructions
    } else {
        tridiagonalize(t.gram, n, v, w, w2, d, e2, red);
    }
    // Gershgorin interval and the smallest pivot allowed in a Sturm count
    double glo = INFINITY, ghi = -INFINITY, emax = 0.0;
    for (int i = 0; i < n; ++i) {
        const double r = (i > 0 ? sqrt(e2[i - 1]) : 0.0) + (i + 1 < n ? sqrt(e2[i]) : 0.0);
        glo = fmin(glo, d[i] - r);
        ghi = fmax(ghi, d[i] + r);
        if (i + 1 < n) emax = fmax(emax, e2[i]);
    }
    const double span = fmax(fabs(glo), fabs(ghi));
    const double pivmin = 0x1p-1000 * fmax(1.0, emax);
    glo -= 2.0 * DBL_EPSILON * span + pivmin;
    ghi += 2.0 * DBL_EPSILON * span + pivmin;
    for (int k = tid; k < n; k += EIG_THREADS) {
        // the k-th smallest eigenvalue: count(lo) <= k < count(hi); each
        // round counts at four interior points (four independent Sturm
        // chains side by side) and keeps the fifth of the interval holding it
        double lo = glo, hi = ghi;
        for (int it = 0; it < 64; ++it) {
            if (!(hi - lo > 2.0 * DBL_EPSILON * fmax(fabs(lo), fabs(hi)) + pivmin)) break;
            const double h = (hi - lo) * 0.2;
            double x[4], q[4];
            int c[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                x[u] = lo + h * (double)(u + 1);
                q[u] = d[0] - x[u];
                if (fabs(q[u]) < pivmin) q[u] = -pivmin;
                c[u] = q[u] < 0.0;
            }
            for (int i = 1; i < n; ++i) {
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    q[u] = d[i] - x[u] - e2[i - 1] * recip_nr(q[u]);
                    if (fabs(q[u]) < pivmin) q[u] = -pivmin;
                    c[u] += q[u] < 0.0;
                }
            }
            double nlo = lo, nhi = hi;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                if (c[u] <= k) nlo = fmax(nlo, x[u]);
                else nhi = fmin(nhi, x[u]);
            }
            if (nlo == lo && nhi == hi) break;  // no representable progress
            lo = nlo;
            hi = nhi;
        }
        const double lam = 0.5 * (lo + hi);
        t.out[n - 1 - k] = sqrt(fmax(lam, 0.0));
    }
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

hipError_t launch_svd(const SvdTask* tasks, int n_tasks, int64_t n_items, double* gram,
                      int64_t gram_len, hipStream_t stream)
{
    if (n_tasks <= 0) return hipSuccess;
    const int64_t cb = min((gram_len + 255) / 256, (int64_t)4096);
    hipLaunchKernelGGL(k_svd_clear, dim3((unsigned)max(cb, (int64_t)1)), dim3(256), 0, stream,
                       gram, gram_len);
    if (n_items > 0)
        hipLaunchKernelGGL(k_gram, dim3((unsigned)n_items), dim3(GTHREADS), 0, stream, tasks,
                           n_tasks, n_items);
    hipLaunchKernelGGL(k_svd_eig, dim3((unsigned)n_tasks), dim3(EIG_THREADS), 0, stream, tasks);
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
