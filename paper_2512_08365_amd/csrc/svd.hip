// svd.hip -- multi-mode SVD invariants of tensors and their matching
// (Section 4.2, "Matching Equivalent Tensors").
//
// For every non-empty proper mode subset G containing mode 0 (its complement
// gives the same spectrum), the unfolding T_(G) has the modes of G as rows and
// the others as columns.  Its singular values are the square roots of the
// eigenvalues of the Gram matrix X X^T, X the unfolding or its transpose,
// whichever has fewer rows (K = min(M, N) <= SVD_MAX_K, L = max(M, N)).
//
// k_gram: one wave per (task, 16 x 16 tile pair of the upper triangle, chunk
//   of GRAM_CHUNK columns); the tile is a sum of fp64 16x16x4 MFMA products
//   over the chunk (fp32 data widened exactly), added into the Gram matrix
//   (and its mirror) with fp64 atomics.  The elements of X are gathered
//   through the unfolding's mixed-radix offsets.
// k_svd_eig: one workgroup per task: Householder reduction of the Gram
//   matrix (in place, in global memory) to tridiagonal form, then every
//   eigenvalue by bisection on Sturm counts, sigma = sqrt(max(lambda, 0)),
//   written in descending order.
// k_svd_match: one workgroup per tensor pair: which spectra of the two lists
//   are close, then a one-to-one pairing by augmenting paths.

#include <cfloat>

#include "mag_internal.hpp"

namespace mag {

namespace {

constexpr int GW = 64;
constexpr int GRAM_WAVES = 4;
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

__global__ __launch_bounds__(GW * GRAM_WAVES) void k_gram(const SvdTask* tasks, int n_tasks,
                                                          int64_t n_items)
{
    const int lane = threadIdx.x % GW;
    const int64_t item = (int64_t)blockIdx.x * GRAM_WAVES + threadIdx.x / GW;
    if (item >= n_items) return;  // the whole wave
    int lo = 0, hi = n_tasks - 1;  // the last task whose first item is <= item
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (tasks[mid].item0 <= item) lo = mid; else hi = mid - 1;
    }
    const SvdTask& t = tasks[lo];
    const int64_t local = item - t.item0;
    const int64_t chunk = local % t.nchunk;
    int64_t pr = local / t.nchunk;
    int ti = 0, rowlen = t.nt;
    while (pr >= rowlen && rowlen > 0) {
        pr -= rowlen;
        ++ti;
        --rowlen;
    }
    const int tj = ti + (int)pr;
    const int r = lane & 15, kq = lane >> 4;
    const int64_t ra = (int64_t)ti * 16 + r, rb = (int64_t)tj * 16 + r;
    const bool va = ra < t.K, vb = rb < t.K;
    const int64_t oa = va ? mode_offset((uint32_t)ra, t.nk, t.kdim, t.kstr) : 0;
    const int64_t ob = vb ? mode_offset((uint32_t)rb, t.nk, t.kdim, t.kstr) : 0;
    const int64_t b0 = chunk * GRAM_CHUNK, b1 = min(b0 + GRAM_CHUNK, t.L);
    // the chunk's column offsets, computed once by the wave's lanes together
    __shared__ int32_t loff_s[GRAM_WAVES][GRAM_CHUNK];
    int32_t* loff = loff_s[threadIdx.x / GW];
    for (int64_t q = lane; q < b1 - b0; q += GW)
        loff[q] = (int32_t)mode_offset((uint32_t)(b0 + q), t.nl, t.ldim, t.lstr);
    // the lanes read each other's entries: a wave's LDS operations complete in
    // order; the fences keep the compiler from moving the reads above the writes
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    d4 acc = {0.0, 0.0, 0.0, 0.0};
    // A operand: lane holds X[ti*16 + lane%16][b + lane/16]; B operand: lane
    // holds X[tj*16 + lane%16][b + lane/16]; the product is the Gram tile
    for (int64_t b = b0; b < b1; b += 4) {
        const int64_t bb = b + kq;
        const bool vl = bb < b1;
        const int64_t ol = vl ? (int64_t)loff[bb - b0] : 0;
        const double xa = (va && vl) ? (double)t.data[oa + ol] : 0.0;
        const double xb = (vb && vl) ? (double)t.data[ob + ol] : 0.0;
        acc = __builtin_amdgcn_mfma_f64_16x16x4f64(xa, xb, acc, 0, 0, 0);
    }
    // register j of a lane holds row 4 j + lane/16, column lane%16 of the tile
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int64_t row = (int64_t)ti * 16 + 4 * j + kq, col = (int64_t)tj * 16 + r;
        if (row < t.K && col < t.K) {
            atomicAdd(&t.gram[row * t.K + col], acc[j]);
            if (ti != tj) atomicAdd(&t.gram[col * t.K + row], acc[j]);
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

// eigenvalues of the symmetric tridiagonal (d, e) below x: Sturm count
__device__ int sturm_count(const double* d, const double* e2, int n, double x, double pivmin)
{
    int c = 0;
    double q = d[0] - x;
    if (fabs(q) < pivmin) q = -pivmin;
    c += q < 0.0;
    for (int i = 1; i < n; ++i) {
        q = d[i] - x - e2[i - 1] / q;
        if (fabs(q) < pivmin) q = -pivmin;
        c += q < 0.0;
    }
    return c;
}

constexpr int EIG_LDS_K = 128;  // Gram matrices up to this side are reduced in LDS

// Householder reduction of the symmetric n x n matrix A (row stride n) to
// tridiagonal form: d[k] the diagonal, e2[k] the squared off-diagonal
__device__ void tridiagonalize(double* A, int n, double* v, double* w, double* d, double* e2,
                               double* red)
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
        // p = beta A_sub v (columns by threads: row j of A is read across threads)
        double pv = 0.0;
        for (int i = tid; i < m; i += EIG_THREADS) {
            const double* col = A + (size_t)(k + 1) * n + (k + 1 + i);
            double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
            int j = 0;
            for (; j + 4 <= m; j += 4) {  // four independent loads in flight
                s0 += col[(size_t)j * n] * v[j];
                s1 += col[(size_t)(j + 1) * n] * v[j + 1];
                s2 += col[(size_t)(j + 2) * n] * v[j + 2];
                s3 += col[(size_t)(j + 3) * n] * v[j + 3];
            }
            for (; j < m; ++j) s0 += col[(size_t)j * n] * v[j];
            w[i] = beta * ((s0 + s1) + (s2 + s3));
            pv += w[i] * v[i];
        }
        const double K2 = 0.5 * beta * block_sum(pv, red);
        for (int i = tid; i < m; i += EIG_THREADS) w[i] -= K2 * v[i];
        __syncthreads();
        // A_sub -= v w^T + w v^T (each thread walks its columns down the rows;
        // the rows of one column are independent, so the loop is unrolled)
        for (int i = tid; i < m; i += EIG_THREADS) {
            double* col = A + (size_t)(k + 1) * n + (k + 1 + i);
            const double vi = v[i], wi = w[i];
#pragma unroll 8
            for (int j = 0; j < m; ++j) col[(size_t)j * n] -= v[j] * wi + w[j] * vi;
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
    const SvdTask& t = tasks[blockIdx.x];
    const int n = (int)t.K;
    const int tid = threadIdx.x;
    if (n <= EIG_LDS_K) {
        for (int q = tid; q < n * n; q += EIG_THREADS) As[q] = t.gram[q];
        __syncthreads();
        tridiagonalize(As, n, v, w, d, e2, red);
    } else {
        tridiagonalize(t.gram, n, v, w, d, e2, red);
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
        // the k-th smallest eigenvalue: count(lo) <= k < count(hi)
        double lo = glo, hi = ghi;
        for (int it = 0; it < 128; ++it) {
            const double mid = 0.5 * (lo + hi);
            if (!(hi - lo > 2.0 * DBL_EPSILON * fmax(fabs(lo), fabs(hi)) + pivmin) || mid == lo ||
                mid == hi)
                break;
            if (sturm_count(d, e2, n, mid, pivmin) <= k) lo = mid; else hi = mid;
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
        hipLaunchKernelGGL(k_gram, dim3((unsigned)((n_items + GRAM_WAVES - 1) / GRAM_WAVES)),
                           dim3(GW * GRAM_WAVES), 0, stream, tasks, n_tasks, n_items);
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
