// Top q eigenpairs of the subsample kernel matrix K_s by Chebyshev-filtered
// subspace iteration with Rayleigh-Ritz and locking, all in float64 on the
// device (the setup of Algorithm 1 needs sigma_1..sigma_{k+1} and
// v_1..v_k, Section 4).
//
// K_s = [k(x_ri, x_rj)] is symmetric positive semi-definite, so its
// spectrum lies in [0, sigma_1]. A block of p = q + guard orthonormal
// columns is repeatedly multiplied by T_m((K - c)/e), the degree-m
// Chebyshev polynomial of the first kind mapped so that [0, cut] goes to
// [-1, 1]: there it stays bounded by 1, above `cut` it grows like
// exp(m acosh(x)), which pulls the block towards the dominant invariant
// subspace much faster than plain powers of K when the spectrum near
// sigma_{k+1} is flat. `cut` is the smallest Ritz value of the block (an
// estimate of sigma_{p+1} from above).
//
// After each filter the block is orthonormalised (Householder QR), the
// Rayleigh-Ritz problem Q^T K Q is solved, and leading Ritz pairs whose
// residual |K v - theta v| is below tol * sigma_1 are locked: moved out of
// the block, and projected out of every later filtered block, so that they
// are not amplified again. The degree of each filter is capped so that the
// ratio between the largest and the cut's amplification stays below 1e8:
// beyond that the weaker directions of a block would sink under rounding
// of the stronger ones.
//
// The large products (K times the block, projections, rotations) are
// float64 GEMMs; the p x p Ritz problem and the QR use rocSOLVER.
#include "eigenpro.h"
#include "ep_host.h"
#include "ep_internal.h"

#include <rocblas/rocblas.h>
#include <rocsolver/rocsolver.h>

#include <algorithm>
#include <cmath>
#include <numeric>
#include <utility>
#include <vector>

namespace ep {

namespace {

__device__ inline uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// Start block: independent uniform(-1, 1) entries from a counter hash.
__global__ void __launch_bounds__(256) rand_block_kernel(double* Q, int64_t count, uint64_t seed) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= count) return;
    const uint64_t h = mix64(seed * 0x9E3779B97F4A7C15ull + (uint64_t)e + 1);
    Q[e] = (double)(h >> 11) * (2.0 / 9007199254740992.0) - 1.0;
}

// out = a (T - c Y1) - b Y0 (Y0 unused when b == 0); out may alias T.
__global__ void __launch_bounds__(256) cheb_combine_kernel(double* out, const double* T,
                                                           const double* Y1, const double* Y0,
                                                           int64_t count, double a, double c,
                                                           double b) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= count) return;
    double v = a * (T[e] - c * Y1[e]);
    if (b != 0.0) v -= b * Y0[e];
    out[e] = v;
}

// res_j = |KQ_j - theta_j Q_j| for each of the p columns (one block each).
__global__ void __launch_bounds__(256) ritz_residual_kernel(const double* KQ, const double* Q,
                                                            const double* theta, int64_t s,
                                                            double* res) {
    __shared__ double red[256];
    const int64_t j = blockIdx.x;
    const double th = theta[j];
    const double* kq = KQ + j * s;
    const double* q = Q + j * s;
    double acc = 0.0;
    for (int64_t i = threadIdx.x; i < s; i += 256) {
        const double r = kq[i] - th * q[i];
        acc = fma(r, r, acc);
    }
    red[threadIdx.x] = acc;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) res[j] = sqrt(red[0]);
}

// Descending order of an ascending eigen-decomposition of a p x p matrix:
// Wr[:, j] = W[:, p-1-j], wr[j] = w[p-1-j].
__global__ void __launch_bounds__(256) reverse_pairs_kernel(const double* W, const double* w,
                                                            int64_t p, double* Wr, double* wr) {
    const int64_t j = blockIdx.x;
    const double* src = W + (p - 1 - j) * p;
    double* dst = Wr + j * p;
    for (int64_t i = threadIdx.x; i < p; i += 256) dst[i] = src[i];
    if (threadIdx.x == 0) wr[j] = w[p - 1 - j];
}

inline unsigned nblocks(int64_t count) { return (unsigned)((count + 255) / 256); }

struct Blas {
    rocblas_handle h;
    // C (m x n) = alpha op(A) op(B) + beta C, column-major
    int gemm(bool ta, bool tb, int64_t m, int64_t n, int64_t k, double alpha, const double* A,
             int64_t lda, const double* B, int64_t ldb, double beta, double* C, int64_t ldc) {
        const rocblas_status st =
            rocblas_dgemm(h, ta ? rocblas_operation_transpose : rocblas_operation_none,
                          tb ? rocblas_operation_transpose : rocblas_operation_none,
                          (rocblas_int)m, (rocblas_int)n, (rocblas_int)k, &alpha, A,
                          (rocblas_int)lda, B, (rocblas_int)ldb, &beta, C, (rocblas_int)ldc);
        if (st != rocblas_status_success)
            return fail(EP_EDEVICE, "rocblas_dgemm returned status %d", (int)st);
        return EP_OK;
    }
};

#define EP_TRY(expr)                 \
    do {                             \
        const int rc_ = (expr);      \
        if (rc_ != EP_OK) return rc_; \
    } while (0)

}  // namespace

int subspace_topq(const double* K, int64_t s, int64_t q, const EigOpts& o, uint64_t seed,
                  rocblas_handle h, hipStream_t st, std::vector<double>& theta_out,
                  DevBuf& VL, EigStats& stats) {
    if (q < 1 || q > s) return fail(EP_EINVAL, "subspace eigensolver: need 1 <= q <= s");
    const int64_t guard = o.guard > 0 ? o.guard : round_up(std::max<int64_t>(32, q / 4), 16);
    const int64_t p = std::min<int64_t>(s, q + guard);
    const int m_max = o.max_degree > 0 ? o.max_degree : 20;
    const int max_it = o.max_iters > 0 ? o.max_iters : 100;
    const double tol = o.tol > 0 ? o.tol : 1e-11;
    const double amp_cap = 1e8;
    const size_t blk = (size_t)s * p * sizeof(double);

    DevBuf bQ, bKQ, bB[3], bH, bW, bw, bwr, bE, btau, bC, bres, binfo;
    HIP_TRY(bQ.ensure(blk));
    HIP_TRY(bKQ.ensure(blk));
    for (DevBuf& b : bB) HIP_TRY(b.ensure(blk));
    HIP_TRY(bH.ensure((size_t)p * p * sizeof(double)));
    HIP_TRY(bW.ensure((size_t)p * p * sizeof(double)));
    HIP_TRY(bw.ensure((size_t)p * sizeof(double)));
    HIP_TRY(bwr.ensure((size_t)p * sizeof(double)));
    HIP_TRY(bE.ensure((size_t)p * sizeof(double)));
    HIP_TRY(btau.ensure((size_t)p * sizeof(double)));
    HIP_TRY(bC.ensure((size_t)q * p * sizeof(double)));
    HIP_TRY(bres.ensure((size_t)p * sizeof(double)));
    HIP_TRY(binfo.ensure(sizeof(rocblas_int)));
    HIP_TRY(VL.ensure((size_t)s * q * sizeof(double)));

    double* Q = bQ.as<double>();
    double* KQ = bKQ.as<double>();
    double* pool[3] = {bB[0].as<double>(), bB[1].as<double>(), bB[2].as<double>()};
    double* Vl = VL.as<double>();
    Blas blas{h};
    rocblas_int* dinfo = binfo.as<rocblas_int>();

    int64_t nl = 0;                       // locked pairs
    int64_t pa = p;                       // active block columns
    std::vector<double> theta_l, wr(p), res(p);
    double normK = 0.0, worst = 0.0;
    int64_t matvecs = 0;

    auto product = [&](const double* Y, int64_t cols, double* out) {
        matvecs += cols;
        return blas.gemm(false, false, s, cols, s, 1.0, K, s, Y, s, 0.0, out, s);
    };
    // Y -= V_L (V_L^T Y)
    auto project = [&](double* Y, int64_t cols) -> int {
        if (nl == 0) return EP_OK;
        EP_TRY(blas.gemm(true, false, nl, cols, s, 1.0, Vl, s, Y, s, 0.0, bC.as<double>(), nl));
        return blas.gemm(false, false, s, cols, nl, -1.0, Vl, s, bC.as<double>(), nl, 1.0, Y, s);
    };
    auto orthonormalise = [&](double* Y, int64_t cols) -> int {
        rocblas_status r1 = rocsolver_dgeqrf(h, (rocblas_int)s, (rocblas_int)cols, Y,
                                             (rocblas_int)s, btau.as<double>());
        if (r1 != rocblas_status_success)
            return fail(EP_EDEVICE, "rocsolver_dgeqrf returned status %d", (int)r1);
        r1 = rocsolver_dorgqr(h, (rocblas_int)s, (rocblas_int)cols, (rocblas_int)cols, Y,
                              (rocblas_int)s, btau.as<double>());
        if (r1 != rocblas_status_success)
            return fail(EP_EDEVICE, "rocsolver_dorgqr returned status %d", (int)r1);
        return EP_OK;
    };
    auto free_buf = [&](const double* a, const double* b) -> double* {
        for (double* x : pool)
            if (x != a && x != b) return x;
        return nullptr;
    };

    // start: random orthonormal block and its product
    hipLaunchKernelGGL(rand_block_kernel, dim3(nblocks((int64_t)s * p)), dim3(256), 0, st, Q,
                       (int64_t)s * p, seed);
    HIP_TRY(hipGetLastError());
    EP_TRY(orthonormalise(Q, pa));
    EP_TRY(product(Q, pa, KQ));

    int it = 0;
    for (;;) {
        // Rayleigh-Ritz on the active block
        EP_TRY(blas.gemm(true, false, pa, pa, s, 1.0, Q, s, KQ, s, 0.0, bH.as<double>(), pa));
        const rocblas_status se =
            rocsolver_dsyevd(h, rocblas_evect_original, rocblas_fill_upper, (rocblas_int)pa,
                             bH.as<double>(), (rocblas_int)pa, bw.as<double>(), bE.as<double>(),
                             dinfo);
        if (se != rocblas_status_success)
            return fail(EP_EDEVICE, "rocsolver_dsyevd (Ritz problem) returned status %d", (int)se);
        hipLaunchKernelGGL(reverse_pairs_kernel, dim3((unsigned)pa), dim3(256), 0, st,
                           bH.as<double>(), bw.as<double>(), pa, bW.as<double>(),
                           bwr.as<double>());
        HIP_TRY(hipGetLastError());
        double* T = pool[0];
        EP_TRY(blas.gemm(false, false, s, pa, pa, 1.0, Q, s, bW.as<double>(), pa, 0.0, T, s));
        std::swap(Q, pool[0]);
        T = pool[0];
        EP_TRY(blas.gemm(false, false, s, pa, pa, 1.0, KQ, s, bW.as<double>(), pa, 0.0, T, s));
        std::swap(KQ, pool[0]);
        hipLaunchKernelGGL(ritz_residual_kernel, dim3((unsigned)pa), dim3(256), 0, st, KQ, Q,
                           bwr.as<double>(), s, bres.as<double>());
        HIP_TRY(hipGetLastError());
        rocblas_int hinfo = 0;
        HIP_TRY(hipMemcpyAsync(&hinfo, dinfo, sizeof hinfo, hipMemcpyDeviceToHost, st));
        HIP_TRY(hipMemcpyAsync(wr.data(), bwr.p, pa * sizeof(double), hipMemcpyDeviceToHost, st));
        HIP_TRY(hipMemcpyAsync(res.data(), bres.p, pa * sizeof(double), hipMemcpyDeviceToHost, st));
        HIP_TRY(hipStreamSynchronize(st));
        if (hinfo != 0) return fail(EP_ENUMERIC, "Ritz eigenproblem failed: info=%d", (int)hinfo);
        for (int64_t j = 0; j < pa; ++j)
            if (!std::isfinite(wr[j]) || !std::isfinite(res[j]))
                return fail(EP_ENUMERIC, "subspace eigensolver produced a non-finite value");
        normK = std::max(normK, std::fabs(wr[0]));
        if (nl > 0) normK = std::max(normK, std::fabs(theta_l[0]));

        // lock the leading converged pairs
        int64_t nc = 0;
        while (nc < pa && nl + nc < q && res[nc] <= tol * normK) ++nc;
        if (nl + nc < q && nc == 0 && p == s) {
            // the block is the whole space: the Ritz pairs are exact
            nc = q - nl;
        }
        if (nc > 0) {
            HIP_TRY(hipMemcpyAsync(Vl + (size_t)nl * s, Q, (size_t)nc * s * sizeof(double),
                                   hipMemcpyDeviceToDevice, st));
            for (int64_t j = 0; j < nc; ++j) {
                theta_l.push_back(wr[j]);
                worst = std::max(worst, res[j] / std::max(normK, 1e-300));
            }
            nl += nc;
            pa -= nc;
            if (nl >= q) break;
            // keep the active columns at the start of their buffers
            double* T2 = pool[0];
            HIP_TRY(hipMemcpyAsync(T2, Q + (size_t)nc * s, (size_t)pa * s * sizeof(double),
                                   hipMemcpyDeviceToDevice, st));
            std::swap(Q, pool[0]);
            T2 = pool[0];
            HIP_TRY(hipMemcpyAsync(T2, KQ + (size_t)nc * s, (size_t)pa * s * sizeof(double),
                                   hipMemcpyDeviceToDevice, st));
            std::swap(KQ, pool[0]);
            wr.erase(wr.begin(), wr.begin() + nc);
            res.erase(res.begin(), res.begin() + nc);
            wr.resize(p);
            res.resize(p);
        }
        if (++it > max_it)
            return fail(EP_ENUMERIC,
                        "subspace eigensolver: %lld of %lld pairs converged after %d iterations",
                        (long long)nl, (long long)q, max_it);

        // filter parameters: damp [0, cut], amplify above
        const double cut = wr[pa - 1];
        const double top = wr[0] + res[0];
        double c = 0.5 * cut, e = 0.5 * cut;
        int m = 1;
        if (!(cut > 1e-14 * normK)) {
            c = 0.0;                      // degenerate interval: one plain product
            e = 1.0;
        } else {
            const double xt = std::max((top - c) / e, 1.0 + 1e-12);
            m = (int)std::floor(std::acosh(amp_cap) / std::acosh(xt));
            m = std::max(1, std::min(m_max, m));
        }
        // Y1 = (K Q - c Q) / e; K Q is at hand
        double* Y0 = Q;
        double* Y1 = free_buf(nullptr, nullptr);
        hipLaunchKernelGGL(cheb_combine_kernel, dim3(nblocks((int64_t)s * pa)), dim3(256), 0, st,
                           Y1, KQ, Q, Q, (int64_t)s * pa, 1.0 / e, c, 0.0);
        HIP_TRY(hipGetLastError());
        EP_TRY(project(Y1, pa));
        for (int j = 2; j <= m; ++j) {
            double* Y2 = free_buf(Y0, Y1);
            EP_TRY(product(Y1, pa, Y2));
            hipLaunchKernelGGL(cheb_combine_kernel, dim3(nblocks((int64_t)s * pa)), dim3(256), 0,
                               st, Y2, Y2, Y1, Y0, (int64_t)s * pa, 2.0 / e, c, 1.0);
            HIP_TRY(hipGetLastError());
            EP_TRY(project(Y2, pa));
            Y0 = Y1;
            Y1 = Y2;
        }
        EP_TRY(project(Y1, pa));
        EP_TRY(orthonormalise(Y1, pa));
        // Y1 (a pool buffer) becomes Q; the old Q buffer joins the pool
        for (double*& x : pool)
            if (x == Y1) x = Q;
        Q = Y1;
        EP_TRY(product(Q, pa, KQ));
    }

    // descending order of the locked values (they are, up to rounding)
    std::vector<int64_t> order(q);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(),
                     [&](int64_t a, int64_t b) { return theta_l[a] > theta_l[b]; });
    bool sorted = true;
    for (int64_t j = 0; j < q; ++j) sorted = sorted && order[j] == j;
    if (!sorted) {
        double* T = pool[0];
        for (int64_t j = 0; j < q; ++j)
            HIP_TRY(hipMemcpyAsync(T + (size_t)j * s, Vl + (size_t)order[j] * s,
                                   s * sizeof(double), hipMemcpyDeviceToDevice, st));
        HIP_TRY(hipMemcpyAsync(Vl, T, (size_t)q * s * sizeof(double), hipMemcpyDeviceToDevice, st));
    }
    theta_out.resize(q);
    for (int64_t j = 0; j < q; ++j) theta_out[j] = theta_l[order[j]];
    HIP_TRY(hipStreamSynchronize(st));
    stats.iters = it;
    stats.matvecs = matvecs;
    stats.max_residual = worst;
    return EP_OK;
}

}  // namespace ep
