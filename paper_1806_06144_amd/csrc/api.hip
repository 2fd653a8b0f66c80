// C ABI of libeigenpro: context, argument checking, buffer management and the
// launch sequence of one EigenPro 2.0 iteration (Algorithm 1) on one GPU.
#include "eigenpro.h"
#include "ep_host.h"
#include "ep_internal.h"

#include <rocblas/rocblas.h>
#include <rocsolver/rocsolver.h>

#include <algorithm>
#include <chrono>
#include <map>
#include <mutex>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

using namespace ep;

namespace {
thread_local std::string g_err;
}  // namespace

int ep::fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

namespace {

struct TimedPair {
    hipEvent_t a, b;
};

uint64_t splitmix64(uint64_t& x) {
    uint64_t z = (x += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

}  // namespace

namespace {

// Scratch of ep_predict_noalloc: the row norms of a chunk of query rows
// followed by the partial sums of its fused pass. One copy lives on every
// device the library runs on (a file-scope device array, held until the
// process ends). In host code `scratch` names a host-side stand-in, not the
// device copy: its device address is looked up once per device
// (hipGetSymbolAddress, with that device current, when the first context is
// created there) and only that address is ever handed to kernels.
constexpr size_t kScratchFloats = size_t(16) << 20;     // 64 MiB
__device__ __align__(256) float scratch[kScratchFloats];

std::mutex g_scratch_mu;
std::map<int, float*> g_scratch_dev;    // device -> address of its scratch

// Address of the current device's scratch (looked up on first use).
int scratch_of_device(int dev, float** out) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    auto it = g_scratch_dev.find(dev);
    if (it != g_scratch_dev.end()) {
        *out = it->second;
        return EP_OK;
    }
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
        return fail(EP_EDEVICE, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    g_scratch_dev[dev] = static_cast<float*>(ptr);
    *out = static_cast<float*>(ptr);
    return EP_OK;
}

}  // namespace

struct ep_ctx {
    int device = 0;
    float* scratch = nullptr;           // this device's scratch (ep_predict_noalloc)
    hipStream_t stream = nullptr;
    const float* X = nullptr;
    int64_t n = 0, d = 0, l = 0, s = 0, k = 0;
    int64_t k_max = 0;                  // rank of the eigensystem held; k <= k_max is applied
    int kind = 0;
    float bandwidth = 1.f;
    float scale = 0.f;
    int64_t l_pad = 0, n_pad = 0, s_pad = 0, k_ld = 1;
    ep_info info{};
    std::vector<double> sigma, D;       // sigma: k_max+1 values; D: k values
    std::vector<float> Vh;              // host copy of V (s x k_max, float32 as applied)
    std::vector<double> Vh64;           // float64 eigenvectors (s x k_max): beta, Eq. 7 sums
    std::vector<int64_t> r_host;
    ep_setup_opts opts{};               // eigensolver choice of ep_setup_ex
    uint64_t seed = 0;
    bool checks = false;
    std::vector<unsigned char> seen;

    DevBuf norms, alpha, r_dev, Xs, xs_norms, V, Dk, err;
    DevBuf kpos;                        // n ints: subsample position of each row, or -1
    DevBuf ksb;                         // s x round_up(m, 64): K(X_r, X_t) captured in step 2
    // per-call scratch
    DevBuf xb, xb_norms, R, part, G, vt_part, W1, zn;

    bool timing = false;
    std::vector<TimedPair> kmv_ev, step_ev, kblk_ev, gemm_ev;
    ep_timing tsum{};

    int contract = EP_CONTRACT_AUTO;    // ep_set_contraction
    size_t block_bytes = size_t(2) << 30;
    rocblas_handle blas = nullptr;      // for the blocked form's GEMMs
    DevBuf kbuf;                        // one centre chunk's kernel block

    ~ep_ctx() {
        for (DevBuf* b : {&norms, &alpha, &r_dev, &Xs, &xs_norms, &V, &Dk, &err, &kpos, &ksb,
                          &xb, &xb_norms, &R, &part, &G, &vt_part, &W1, &zn})
            b->release();
        for (auto& p : kmv_ev) {
            (void)hipEventDestroy(p.a);
            (void)hipEventDestroy(p.b);
        }
        for (auto* v : {&step_ev, &kblk_ev, &gemm_ev})
            for (auto& p : *v) {
                (void)hipEventDestroy(p.a);
                (void)hipEventDestroy(p.b);
            }
        if (blas) rocblas_destroy_handle(blas);
    }
};

namespace {

constexpr size_t kPartBudget = size_t(2) << 30;   // bytes of split partial sums
// bytes of the captured subsample columns K(X_r, X_t); larger products run
// the separate subsample pass (and the capture must stay below 2^31 bytes,
// the reach of its buffer descriptor)
constexpr size_t kKsbBudget = (size_t(2) << 30) - 256;

int max_slices_for(int64_t rows_pad, int64_t ldw) {
    const size_t per = (size_t)rows_pad * (size_t)ldw * sizeof(float);
    return (int)std::max<size_t>(1, std::min<size_t>(256, kPartBudget / std::max<size_t>(per, 1)));
}

int record(hipStream_t s, std::vector<TimedPair>& v, bool start) {
    if (start) {
        TimedPair p;
        HIP_TRY(hipEventCreate(&p.a));
        HIP_TRY(hipEventCreate(&p.b));
        v.push_back(p);
        HIP_TRY(hipEventRecord(v.back().a, s));
    } else {
        HIP_TRY(hipEventRecord(v.back().b, s));
    }
    return EP_OK;
}

// sum_j k(q_i, c_j) W_j for all rows of Q: fused kernel + reduction target
// is the caller's; returns the slice count in *slices.
int run_kmv(ep_ctx* c, const float* Q, int64_t ldq, const float* qn, const int64_t* qid,
            int64_t nq, const float* C, int64_t ldc, const float* cn, const int64_t* cid,
            int64_t nc, const float* W, int* slices, int64_t* rows_pad, bool timed,
            bool subsample, bool capture = false) {
    *rows_pad = round_up(std::max<int64_t>(nq, 1), kBM);
    KmvPlan plan =
        kmv_plan(nq, nc, ldc, c->l_pad, c->l, c->kind, max_slices_for(*rows_pad, c->l_pad));
    *slices = plan.slices();
    HIP_TRY(c->part.ensure((size_t)plan.slices() * (size_t)(*rows_pad) * c->l_pad * sizeof(float)));
    KmvArgs a{};
    a.Q = Q;
    a.ldq = ldq;
    a.qn = qn;
    a.qid = qid;
    a.nq = nq;
    a.C = C;
    a.ldc = ldc;
    a.cn = cn;
    a.cid = cid;
    a.nc = nc;
    a.d = c->d;
    a.W = W;
    a.ldw = c->l_pad;
    a.lt = (int)(c->l_pad / kTile);
    a.out = c->part.as<float>();
    a.out_rows = *rows_pad;
    a.kind = c->kind;
    a.scale = c->scale;
    if (capture) {
        a.kpos = c->kpos.as<int>();
        a.ksb = c->ksb.as<float>();
        a.ldk = *rows_pad;
        a.s_rows = c->s;
    }
    if (timed) {
        int rc = record(c->stream, c->kmv_ev, true);
        if (rc) return rc;
    }
    HIP_TRY(kmv_launch(a, plan, c->stream, subsample));
    if (timed) {
        int rc = record(c->stream, c->kmv_ev, false);
        if (rc) return rc;
    }
    return EP_OK;
}

constexpr size_t kKBlockBudget = size_t(2) << 30;   // bytes of one chunk's kernel block

// rocBLAS handle of the context, bound to its stream.
int ensure_blas(ep_ctx* c) {
    if (!c->blas) {
        if (rocblas_create_handle(&c->blas) != rocblas_status_success) {
            c->blas = nullptr;
            return fail(EP_EDEVICE, "rocblas_create_handle failed");
        }
    }
    if (rocblas_set_stream(c->blas, c->stream) != rocblas_status_success)
        return fail(EP_EDEVICE, "rocblas_set_stream failed");
    return EP_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// Whether F = K(Q, X) alpha takes the blocked form (see ep_set_contraction).
bool use_blocked(const ep_ctx* c, const float* Q, int64_t ldq) {
    if (c->contract != EP_CONTRACT_BLOCKED) return false;
    return c->d % 4 == 0 && ldq % 4 == 0 && aligned16(Q) && aligned16(c->X);
}

// F = K(Q, X) alpha in the blocked form: per chunk of centres, the kernel
// block (kblock.hip), then float32 GEMMs (rocBLAS, column-major view:
// F^T = alpha_sub^T . block_sub^T) over sub-ranges of at most kw centres.
// The sub-range products go round robin to up to 32 partial slices of
// c->part (beta = 0 on a slice's first use), which the reduction kernels
// sum: like the fused form's centre splits, this keeps each float32
// accumulation chain near n / 32 terms instead of n.
int run_blocked(ep_ctx* c, const float* Q, int64_t ldq, const float* qn, const int64_t* qid,
                int64_t nq, int* slices, int64_t* rows_pad, bool timed) {
    hipStream_t st = c->stream;
    *rows_pad = round_up(std::max<int64_t>(nq, 1), kBM);
    const int S = std::max(1, std::min(32, max_slices_for(*rows_pad, c->l_pad)));
    const int64_t kw = std::max<int64_t>(64, round_up(ceil_div(c->n, S), 64));
    HIP_TRY(c->part.ensure((size_t)S * (*rows_pad) * c->l_pad * sizeof(float)));
    const int64_t rows256 = round_up(nq, 256);
    int64_t ldo = (int64_t)(c->block_bytes / ((size_t)rows256 * sizeof(float))) / 256 * 256;
    ldo = std::max<int64_t>(256, std::min<int64_t>(ldo, round_up(c->n, 256)));
    HIP_TRY(c->kbuf.ensure((size_t)rows256 * ldo * sizeof(float)));
    if (int rc = ensure_blas(c)) return rc;
    const size_t slice_elems = (size_t)(*rows_pad) * c->l_pad;
    int rc = EP_OK;
    int64_t sub = 0;
    if (timed && (rc = record(st, c->kmv_ev, true))) return rc;
    for (int64_t cs = 0; cs < c->n; cs += ldo) {
        const int64_t nc = std::min(ldo, c->n - cs);
        KblockArgs a{};
        a.Q = Q;
        a.ldq = ldq;
        a.qn = qn;
        a.qid = qid;
        a.nq = nq;
        a.C = c->X + cs * c->d;
        a.ldc = c->d;
        a.cn = c->norms.as<float>() + cs;
        a.cid_base = cs;
        a.nc = nc;
        a.d = c->d;
        a.kind = c->kind;
        a.scale = c->scale;
        a.out = c->kbuf.as<float>();
        a.ldo = ldo;
        if (timed && (rc = record(st, c->kblk_ev, true))) return rc;
        HIP_TRY(kblock_launch(a, st));
        if (timed && (rc = record(st, c->kblk_ev, false))) return rc;
        if (timed && (rc = record(st, c->gemm_ev, true))) return rc;
        for (int64_t k0 = 0; k0 < nc; k0 += kw, ++sub) {
            const int64_t kk = std::min(kw, nc - k0);
            const float one = 1.f, beta = sub < S ? 0.f : 1.f;
            float* out = c->part.as<float>() + (size_t)(sub % S) * slice_elems;
            const rocblas_status gs = rocblas_sgemm(
                c->blas, rocblas_operation_none, rocblas_operation_none, (rocblas_int)c->l_pad,
                (rocblas_int)nq, (rocblas_int)kk, &one,
                c->alpha.as<float>() + (cs + k0) * c->l_pad, (rocblas_int)c->l_pad,
                c->kbuf.as<float>() + k0, (rocblas_int)ldo, &beta, out, (rocblas_int)c->l_pad);
            if (gs != rocblas_status_success)
                return fail(EP_EDEVICE, "rocblas_sgemm returned status %d", (int)gs);
        }
        if (timed && (rc = record(st, c->gemm_ev, false))) return rc;
    }
    if (timed && (rc = record(st, c->kmv_ev, false))) return rc;
    *slices = (int)std::min<int64_t>(sub, S);
    return EP_OK;
}

// F = K(Q, X) alpha over all training points: blocked or fused form.
// With `capture` (fused form only) the pass also stores the kernel values of
// the subsample columns, K(X_r, X_t), in c->ksb.
int run_main_pass(ep_ctx* c, const float* Q, int64_t ldq, const float* qn, const int64_t* qid,
                  int64_t nq, int* slices, int64_t* rows_pad, bool timed, bool capture = false) {
    if (use_blocked(c, Q, ldq))
        return run_blocked(c, Q, ldq, qn, qid, nq, slices, rows_pad, timed);
    return run_kmv(c, Q, ldq, qn, qid, nq, c->X, c->d, c->norms.as<float>(), nullptr, c->n,
                   c->alpha.as<float>(), slices, rows_pad, timed, false, capture);
}

// Whether step 2 of a batch of m rows (gathered, row length d) captures the
// subsample columns for steps 4-5: fused form, vector body, and the capture
// buffer and the product's partial slices within budget.
bool capture_subsample(const ep_ctx* c, const float* xb, int64_t m) {
    return c->k > 0 && !use_blocked(c, xb, c->d) && kmv_vec(xb, c->d, c->X, c->d, c->d) &&
           (size_t)c->s * (size_t)round_up(m, kBM) * sizeof(float) <= kKsbBudget;
}

struct DeviceGuard {
    int prev = -1;
    explicit DeviceGuard(int dev) {
        if (hipGetDevice(&prev) == hipSuccess && prev != dev) (void)hipSetDevice(dev);
        else prev = -1;
    }
    ~DeviceGuard() {
        if (prev >= 0) (void)hipSetDevice(prev);
    }
};

// Top k+1 eigenpairs of K_s = [k(x_ri, x_rj)] (Algorithm 1 initialisation):
// K_s is formed in float64 on the device and solved there in float64,
// either by the full divide-and-conquer eigendecomposition or by the
// Chebyshev-filtered subspace iteration of eigsolve.hip (Section 4 needs
// only the top k+1 pairs). Fills c->sigma, c->V and the adapted kernel's
// diagonal k_G(x_ri, x_ri) at the subsample points.
int eigensystem_from_solver(ep_ctx* c) {
    const int64_t s = c->s, k = c->k, d = c->d;
    hipStream_t st = c->stream;
    const ep_setup_opts& o = c->opts;
    EigOpts eo;
    eo.max_degree = o.max_degree;
    eo.max_iters = o.max_iters;
    eo.guard = o.guard;
    eo.tol = o.tol;
    int solver = o.solver;
    if (solver == EP_SOLVER_AUTO) {
        const int64_t q = k + 1;
        const int64_t guard = o.guard > 0 ? o.guard : round_up(std::max<int64_t>(32, q / 4), 16);
        // measured crossover: the dense solve's O(s^3) wins below s ~ 16 p
        solver = (s >= 2048 && 16 * (q + guard) <= s) ? EP_SOLVER_SUBSPACE : EP_SOLVER_DENSE;
    }
    DevBuf Ks, W, E, iinfo, Vq;
    HIP_TRY(Ks.ensure((size_t)s * s * sizeof(double)));
    HIP_TRY(launch_subsample_kernel_f64(c->Xs.as<float>(), s, d, c->kind, c->bandwidth,
                                        Ks.as<double>(), st));

    rocblas_handle h = nullptr;
    if (rocblas_create_handle(&h) != rocblas_status_success)
        return fail(EP_EDEVICE, "rocblas_create_handle failed");
    struct HandleGuard {
        rocblas_handle h;
        ~HandleGuard() { rocblas_destroy_handle(h); }
    } hguard{h};
    rocblas_set_stream(h, st);

    const double* Z = nullptr;            // eigenvector columns, float64, leading dim s
    int64_t col0 = 0, col_step = 1;
    if (solver == EP_SOLVER_SUBSPACE) {
        EigStats stats;
        std::vector<double> theta;
        const int rc = subspace_topq(Ks.as<double>(), s, k + 1, eo, c->seed ^ 0x5EEDE16ull, h, st,
                                     theta, Vq, stats);
        if (rc == EP_OK) {
            c->sigma = theta;
            Z = Vq.as<double>();
            col0 = 0;
            col_step = 1;
            c->info.solver = EP_SOLVER_SUBSPACE;
            c->info.solver_iters = stats.iters;
            c->info.solver_matvecs = stats.matvecs;
            c->info.eig_residual = stats.max_residual;
        } else if (rc != EP_ENUMERIC || o.no_fallback) {
            return rc;
        } else {
            (void)hipStreamSynchronize(st);
            solver = EP_SOLVER_DENSE;     // did not converge: full solve instead
        }
    }
    if (solver == EP_SOLVER_DENSE) {
        HIP_TRY(W.ensure((size_t)s * sizeof(double)));
        HIP_TRY(E.ensure((size_t)s * sizeof(double)));
        HIP_TRY(iinfo.ensure(sizeof(rocblas_int)));
        rocblas_int* dinfo = iinfo.as<rocblas_int>();
        // eigenvalues ascending in W, eigenvectors overwrite K_s (column-major)
        const rocblas_status rs =
            rocsolver_dsyevd(h, rocblas_evect_original, rocblas_fill_upper, (rocblas_int)s,
                             Ks.as<double>(), (rocblas_int)s, W.as<double>(), E.as<double>(),
                             dinfo);
        if (rs != rocblas_status_success)
            return fail(EP_EDEVICE, "rocsolver_dsyevd returned status %d", (int)rs);
        rocblas_int hinfo = 0;
        std::vector<double> w_asc(k + 1);
        HIP_TRY(hipMemcpyAsync(&hinfo, dinfo, sizeof hinfo, hipMemcpyDeviceToHost, st));
        HIP_TRY(hipMemcpyAsync(w_asc.data(), W.as<double>() + (s - k - 1),
                               (k + 1) * sizeof(double), hipMemcpyDeviceToHost, st));
        HIP_TRY(hipStreamSynchronize(st));
        if (hinfo != 0) return fail(EP_ENUMERIC, "eigensolve failed: info=%d", (int)hinfo);
        c->sigma.assign(w_asc.rbegin(), w_asc.rend());
        // top k+1 eigenvectors are the last k+1 columns, ascending
        Z = Ks.as<double>() + (size_t)(s - k - 1) * s;
        col0 = k;
        col_step = -1;
        c->info.solver = EP_SOLVER_DENSE;
        c->info.solver_iters = 0;
        c->info.solver_matvecs = 0;
        c->info.eig_residual = 0.0;
    }
    if (!(c->sigma[k] > 0.0) || !std::isfinite(c->sigma[0]))
        return fail(EP_ENUMERIC, "sigma_{k+1} = %g is not positive", c->sigma[k]);
    HIP_TRY(launch_extract_eigvecs(Z, s, col0, col_step, s, k, c->V.as<float>(), c->k_ld, st));
    // the float64 eigenvectors on the host (row-major s x k), from which
    // beta and the rank sums of Eq. 7 are formed without float32 rounding
    c->Vh64.assign((size_t)s * k, 0.0);
    if (k > 0) {
        const double* lo = col_step > 0 ? Z + col0 * s : Z + (col0 - (k - 1)) * s;
        std::vector<double> cols((size_t)s * k);
        HIP_TRY(hipMemcpyAsync(cols.data(), lo, (size_t)s * k * sizeof(double),
                               hipMemcpyDeviceToHost, st));
        HIP_TRY(hipStreamSynchronize(st));
        for (int64_t j = 0; j < k; ++j) {
            const int64_t cj = col_step > 0 ? j : (k - 1 - j);
            for (int64_t i = 0; i < s; ++i) c->Vh64[(size_t)i * k + j] = cols[(size_t)cj * s + i];
        }
    }
    HIP_TRY(hipStreamSynchronize(st));
    return EP_OK;
}

// Eigensystem handed in by the caller (a saved setup): sigma descending,
// V row-major s x k.
int eigensystem_from_saved(ep_ctx* c, const double* sigma, const float* V) {
    const int64_t s = c->s, k = c->k;
    c->sigma.assign(sigma, sigma + k + 1);
    for (int64_t i = 0; i <= k; ++i) {
        if (!std::isfinite(c->sigma[i]) || (i > 0 && c->sigma[i] > c->sigma[i - 1]))
            return fail(EP_EINVAL, "sigma must be finite and non-increasing");
    }
    if (!(c->sigma[k] > 0.0)) return fail(EP_EINVAL, "sigma_{k+1} must be positive");
    if (k > 0 && !V) return fail(EP_EINVAL, "V is NULL");
    c->Vh64.assign((size_t)s * k, 0.0);
    for (int64_t i = 0; i < s * k; ++i) {
        if (!std::isfinite(V[i])) return fail(EP_EINVAL, "V holds a non-finite value");
        c->Vh64[(size_t)i] = V[i];
    }
    if (k > 0) {
        HIP_TRY(hipMemsetAsync(c->V.p, 0, (size_t)s * c->k_ld * sizeof(float), c->stream));
        HIP_TRY(hipMemcpy2DAsync(c->V.p, c->k_ld * sizeof(float), V, k * sizeof(float),
                                 k * sizeof(float), s, hipMemcpyHostToDevice, c->stream));
    }
    HIP_TRY(hipStreamSynchronize(c->stream));
    return EP_OK;
}

// beta(K_G) for every rank k' <= k_max at once (Section 3 Step 2 with the
// Nystrom eigenfunctions of Section 4, over the subsample points):
//   beta(k') = max_i [1 - sum_{j<k'} (sigma_j - sigma_k') V_ij^2]
//            = max_i [1 - A_i(k') + sigma_k' B_i(k')],
// A_i, B_i prefix sums of sigma_j V_ij^2 and V_ij^2.
std::vector<double> beta_all_ranks(const ep_ctx* c) {
    const int64_t s = c->s, km = c->k_max;
    std::vector<double> beta(km + 1, -1e300), A(s, 0.0), B(s, 0.0);
    for (int64_t kk = 0; kk <= km; ++kk) {
        const double floor_sigma = c->sigma[kk];
        double best = -1e300;
        for (int64_t i = 0; i < s; ++i) best = std::max(best, 1.0 - A[i] + floor_sigma * B[i]);
        beta[kk] = kk == 0 ? 1.0 : best;
        if (kk < km) {
            for (int64_t i = 0; i < s; ++i) {
                const double v = c->Vh64[(size_t)i * km + kk];
                A[i] += c->sigma[kk] * v * v;
                B[i] += v * v;
            }
        }
    }
    return beta;
}

// Make rank k (0 <= k <= k_max) the active preconditioner: D (Section 4,
// Eq. 8 with q = k+1), beta(K_G), lambda = sigma_{k+1}/s, m* = beta/lambda
// (Section 2), batch min(n, max(1, floor(m*))) and its step size.
int apply_rank(ep_ctx* c, int64_t k) {
    const int64_t s = c->s, n = c->n;
    c->k = k;
    c->D.resize(k);
    std::vector<float> dk(std::max<int64_t>(c->k_max, 1), 0.f);
    for (int64_t i = 0; i < k; ++i) {
        c->D[i] = (1.0 - c->sigma[k] / c->sigma[i]) / c->sigma[i];
        dk[i] = (float)c->D[i];
    }
    HIP_TRY(hipMemcpyAsync(c->Dk.p, dk.data(), dk.size() * sizeof(float), hipMemcpyHostToDevice,
                           c->stream));
    double beta = 1.0;
    if (k > 0) {
        beta = -1e300;
        const int64_t km = c->k_max;
        for (int64_t i = 0; i < s; ++i) {
            double acc = 0.0;
            for (int64_t j = 0; j < k; ++j) {
                const double v = c->Vh64[(size_t)i * km + j];
                acc += (c->sigma[j] - c->sigma[k]) * v * v;
            }
            beta = std::max(beta, 1.0 - acc);
        }
    }
    const double lam = c->sigma[k] / (double)s;
    const double m_star = beta / lam;
    const int64_t m = std::min<int64_t>(n, std::max<int64_t>(1, (int64_t)std::floor(m_star)));
    ep_info& I = c->info;
    I.n = n;
    I.d = c->d;
    I.l = c->l;
    I.s = s;
    I.k = k;
    I.k_max = c->k_max;
    I.sigma_1 = c->sigma[0];
    I.sigma_k1 = c->sigma[k];
    I.lambda_k1 = lam;
    I.beta = beta;
    I.m_star = m_star;
    I.m = m;
    I.eta = (double)m / (beta + (double)(m - 1) * lam);
    I.accel = 0.0;
    HIP_TRY(hipStreamSynchronize(c->stream));
    return EP_OK;
}

int do_setup(ep_ctx* c, const int64_t* sub_idx, uint64_t seed, const double* sigma_in,
             const float* V_in) {
    const int64_t n = c->n, d = c->d, s = c->s, k = c->k;
    hipStream_t st = c->stream;

    // subsample indices (Algorithm 1: fixed coordinate block r)
    c->r_host.resize(s);
    if (sub_idx) {
        std::vector<unsigned char> seen(n, 0);
        for (int64_t i = 0; i < s; ++i) {
            const int64_t v = sub_idx[i];
            if (v < 0 || v >= n) return fail(EP_EINVAL, "sub_idx[%lld]=%lld outside [0,%lld)",
                                             (long long)i, (long long)v, (long long)n);
            if (seen[v]) return fail(EP_EINVAL, "sub_idx repeats index %lld", (long long)v);
            seen[v] = 1;
            c->r_host[i] = v;
        }
    } else {
        std::vector<int64_t> perm(n);
        for (int64_t i = 0; i < n; ++i) perm[i] = i;
        uint64_t st_rng = seed;
        for (int64_t i = 0; i < s; ++i) {
            const uint64_t span = (uint64_t)(n - i);
            const int64_t j = i + (int64_t)(splitmix64(st_rng) % span);
            std::swap(perm[i], perm[j]);
            c->r_host[i] = perm[i];
        }
    }

    c->l_pad = round_up(c->l, kTile);
    c->n_pad = round_up(n, kBN);
    c->s_pad = round_up(s, kBM);
    c->k_ld = round_up(std::max<int64_t>(k, 1), 4);   // 16-byte rows for the thin products

    HIP_TRY(c->err.ensure(sizeof(int)));
    HIP_TRY(hipMemsetAsync(c->err.p, 0, sizeof(int), st));
    HIP_TRY(c->norms.ensure((size_t)c->n_pad * sizeof(float)));
    // (alpha and R serve as the weights of fused passes: kWeightTail bytes
    // after the padded rows)
    HIP_TRY(c->alpha.ensure((size_t)c->n_pad * c->l_pad * sizeof(float) + kWeightTail));
    HIP_TRY(c->r_dev.ensure((size_t)s * sizeof(int64_t)));
    HIP_TRY(c->Xs.ensure((size_t)c->s_pad * d * sizeof(float)));
    HIP_TRY(c->xs_norms.ensure((size_t)c->s_pad * sizeof(float)));
    HIP_TRY(c->V.ensure((size_t)s * c->k_ld * sizeof(float)));
    HIP_TRY(c->Dk.ensure((size_t)c->k_ld * sizeof(float)));

    HIP_TRY(launch_fill_f32(c->alpha.as<float>(), c->n_pad * c->l_pad + kWeightTail / 4, 0.f, st));
    HIP_TRY(launch_fill_f32(c->norms.as<float>(), c->n_pad, 0.f, st));
    HIP_TRY(hipMemcpyAsync(c->r_dev.p, c->r_host.data(), s * sizeof(int64_t),
                           hipMemcpyHostToDevice, st));
    {
        // subsample position of every training row (-1: not in r), which
        // lets step 2 keep the kernel values of the subsample columns
        std::vector<int32_t> kp((size_t)n, -1);
        for (int64_t i = 0; i < s; ++i) kp[(size_t)c->r_host[i]] = (int32_t)i;
        HIP_TRY(c->kpos.ensure((size_t)n * sizeof(int32_t)));
        HIP_TRY(hipMemcpy(c->kpos.p, kp.data(), (size_t)n * sizeof(int32_t),
                          hipMemcpyHostToDevice));
    }
    HIP_TRY(launch_row_norms(c->X, n, d, d, c->norms.as<float>(), st));
    HIP_TRY(launch_gather_rows(c->X, n, d, c->norms.as<float>(), c->r_dev.as<int64_t>(), s,
                               c->s_pad, c->Xs.as<float>(), c->xs_norms.as<float>(),
                               c->err.as<int>(), st));

    int rc = sigma_in ? eigensystem_from_saved(c, sigma_in, V_in) : eigensystem_from_solver(c);
    if (rc) return rc;

    int herr = 0;
    HIP_TRY(hipMemcpyAsync(&herr, c->err.p, sizeof(int), hipMemcpyDeviceToHost, st));
    c->Vh.resize((size_t)s * k);
    if (k > 0)
        HIP_TRY(hipMemcpy2DAsync(c->Vh.data(), k * sizeof(float), c->V.p, c->k_ld * sizeof(float),
                                 k * sizeof(float), s, hipMemcpyDeviceToHost, st));
    HIP_TRY(hipStreamSynchronize(st));
    if (herr) return fail(EP_EINVAL, "subsample index out of range");
    c->k_max = k;
    return apply_rank(c, k);
}

// Steps 4-5 (Algorithm 1, Eq. 8): alpha_r += coef V D V^T K(X_r, X_t) R on
// the hand-written thin products of thin_gemm.hip. With the subsample
// columns kept by step 2 (`capture`: c->ksb, s x round_up(m, kBM)) the
// product is associated in whichever order takes fewer flops:
//   G first: G = K R (s x l), W = D V^T G       2 s m l + 2 k s l
//   U first: U = V^T K (k x m), W = D U R       2 k s m + 2 k m l
// (U first wins when l > k, e.g. 1000 labels at rank 200). Otherwise the
// subsample pass of the fused kernel forms G = K(X_r, X_t) R directly.
// Then alpha_r += coef V W, added by the last product's epilogue.
int subsample_correction(ep_ctx* c, bool capture, const float* xb, const float* xbn,
                         const int64_t* t, int64_t m, const float* R, float coef) {
    hipStream_t st = c->stream;
    const int64_t s = c->s, k = c->k, L = c->l_pad, kld = c->k_ld;
    const int64_t ldk = round_up(m, kBM);
    const int groups = 1024;
    const float* V = c->V.as<float>();
    // partial slices of one product into c->part, summed (and scaled) into out
    auto product = [&](const float* A, int64_t lda, bool a_t, const float* B, int64_t ldb,
                       int64_t M, int64_t N, int64_t K, const float* Dk, float* out,
                       int64_t ldo) -> int {
        const ThinGemmPlan pl = thin_gemm_plan(M, N, K, groups);
        const int64_t slice = M * ldo;
        const bool direct = pl.chunks == 1 && !Dk;
        if (!direct) HIP_TRY(c->part.ensure((size_t)pl.chunks * slice * sizeof(float)));
        ThinGemmArgs g{};
        g.A = A;
        g.lda = lda;
        g.B = B;
        g.ldb = ldb;
        g.M = M;
        g.N = N;
        g.K = K;
        g.C = direct ? out : c->part.as<float>();
        g.ldc = ldo;
        g.slice = slice;
        HIP_TRY(thin_gemm_launch(g, pl, a_t, false, st));
        if (!direct)
            HIP_TRY(launch_sum_slices(c->part.as<float>(), pl.chunks, slice, M, N, ldo, Dk, out,
                                      ldo, st));
        return EP_OK;
    };
    int rc = EP_OK;
    HIP_TRY(c->W1.ensure((size_t)k * L * sizeof(float)));
    float* W = c->W1.as<float>();
    const double g_first = (double)s * m * L + (double)k * s * L;
    const double u_first = (double)k * s * m + (double)k * m * L;
    if (capture && u_first < g_first) {
        HIP_TRY(c->G.ensure((size_t)k * ldk * sizeof(float)));
        float* U = c->G.as<float>();
        if ((rc = product(V, kld, true, c->ksb.as<float>(), ldk, k, m, s, nullptr, U, ldk)))
            return rc;
        if ((rc = product(U, ldk, false, R, L, k, L, m, c->Dk.as<float>(), W, L))) return rc;
    } else {
        HIP_TRY(c->G.ensure((size_t)s * L * sizeof(float)));
        float* G = c->G.as<float>();
        if (capture) {
            if ((rc = product(c->ksb.as<float>(), ldk, false, R, L, s, L, m, nullptr, G, L)))
                return rc;
        } else {
            int slices = 0;
            int64_t rows_pad = 0;
            rc = run_kmv(c, c->Xs.as<float>(), c->d, c->xs_norms.as<float>(),
                         c->r_dev.as<int64_t>(), s, xb, c->d, xbn, t, m, R, &slices, &rows_pad,
                         false, true);
            if (rc) return rc;
            HIP_TRY(launch_reduce_rows(c->part.as<float>(), slices, rows_pad, L, s, L, G, L, st));
        }
        if ((rc = product(V, kld, true, G, L, k, L, s, c->Dk.as<float>(), W, L))) return rc;
    }
    // alpha_r += coef V W (depth k, one chunk; rows r are distinct)
    ThinGemmArgs g{};
    g.A = V;
    g.lda = kld;
    g.B = W;
    g.ldb = L;
    g.M = s;
    g.N = L;
    g.K = k;
    g.alpha = c->alpha.as<float>();
    g.ldalpha = L;
    g.r = c->r_dev.as<int64_t>();
    g.coef = coef;
    g.N_valid = c->l;
    ThinGemmPlan one;
    one.kc = round_up(k, 64);
    one.chunks = 1;
    one.tiles = ceil_div(s, 64) * ceil_div(L, 64);
    HIP_TRY(thin_gemm_launch(g, one, false, true, st));
    return EP_OK;
}

int ensure_step_buffers(ep_ctx* c, int64_t m) {
    const int64_t m_pad = round_up(m, kBN);
    HIP_TRY(c->xb.ensure((size_t)m_pad * c->d * sizeof(float)));
    HIP_TRY(c->xb_norms.ensure((size_t)m_pad * sizeof(float)));
    HIP_TRY(c->R.ensure((size_t)m_pad * c->l_pad * sizeof(float) + kWeightTail));
    return EP_OK;
}

}  // namespace

extern "C" {

const char* ep_last_error(void) { return g_err.c_str(); }

}  // extern "C"

namespace {

int create(ep_ctx** out, const float* X, int64_t n, int64_t d, int64_t l, int kernel,
           float bandwidth, int64_t s, int64_t k, const int64_t* sub_idx, uint64_t seed,
           void* hip_stream, ep_info* info, const double* sigma, const float* V,
           const ep_setup_opts* opts) {
    g_err.clear();
    if (!out) return fail(EP_EINVAL, "ctx out-pointer is NULL");
    *out = nullptr;
    if (!X) return fail(EP_EINVAL, "X is NULL");
    if (n < 1 || d < 1 || l < 1) return fail(EP_EINVAL, "need n, d, l >= 1");
    if (d > (int64_t(1) << 20))
        return fail(EP_EINVAL, "d = %lld exceeds 2^20 features", (long long)d);
    if (!(0 <= k && k < s && s <= n)) return fail(EP_EINVAL, "need 0 <= k < s <= n");
    if (kernel != EP_GAUSSIAN && kernel != EP_LAPLACIAN)
        return fail(EP_EINVAL, "unknown kernel id %d", kernel);
    if (!(bandwidth > 0.f) || !std::isfinite(bandwidth))
        return fail(EP_EINVAL, "bandwidth must be positive and finite");
    if (s > 46340) return fail(EP_EINVAL, "s = %lld exceeds the eigensolver's 32-bit index range",
                               (long long)s);
    if (opts) {
        if (opts->solver < EP_SOLVER_AUTO || opts->solver > EP_SOLVER_SUBSPACE)
            return fail(EP_EINVAL, "unknown solver %d", (int)opts->solver);
        if (opts->max_degree < 0 || opts->max_iters < 0 || opts->guard < 0 ||
            !(opts->tol >= 0.0) || !std::isfinite(opts->tol))
            return fail(EP_EINVAL, "setup options must be zero (default) or positive");
    }
    const auto t0 = std::chrono::steady_clock::now();
    ep_ctx* c = new (std::nothrow) ep_ctx();
    if (!c) return fail(EP_ENOMEM, "host allocation failed");
    if (hipGetDevice(&c->device) != hipSuccess) {
        delete c;
        return fail(EP_EDEVICE, "no HIP device");
    }
    if (int rc = scratch_of_device(c->device, &c->scratch)) {
        delete c;
        return rc;
    }
    c->stream = static_cast<hipStream_t>(hip_stream);
    c->X = X;
    c->n = n;
    c->d = d;
    c->l = l;
    c->s = s;
    c->k = k;
    c->kind = kernel;
    c->bandwidth = bandwidth;
    c->scale = kernel_scale(kernel, bandwidth);
    if (opts) c->opts = *opts;
    c->seed = seed;
    const int rc = do_setup(c, sub_idx, seed, sigma, V);
    if (rc != EP_OK) {
        (void)hipStreamSynchronize(c->stream);
        delete c;
        return rc;
    }
    c->info.setup_ms =
        std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
    if (info) *info = c->info;
    *out = c;
    return EP_OK;
}

}  // namespace

extern "C" {

int ep_setup(ep_ctx** out, const float* X, int64_t n, int64_t d, int64_t l, int kernel,
             float bandwidth, int64_t s, int64_t k, const int64_t* sub_idx, uint64_t seed,
             void* hip_stream, ep_info* info) {
    return create(out, X, n, d, l, kernel, bandwidth, s, k, sub_idx, seed, hip_stream, info,
                  nullptr, nullptr, nullptr);
}

int ep_setup_ex(ep_ctx** out, const float* X, int64_t n, int64_t d, int64_t l, int kernel,
                float bandwidth, int64_t s, int64_t k, const int64_t* sub_idx, uint64_t seed,
                void* hip_stream, const ep_setup_opts* opts, ep_info* info) {
    return create(out, X, n, d, l, kernel, bandwidth, s, k, sub_idx, seed, hip_stream, info,
                  nullptr, nullptr, opts);
}

int ep_restore(ep_ctx** out, const float* X, int64_t n, int64_t d, int64_t l, int kernel,
               float bandwidth, int64_t s, int64_t k, const int64_t* sub_idx,
               const double* sigma, const float* V, void* hip_stream, ep_info* info) {
    g_err.clear();
    if (!sub_idx) return fail(EP_EINVAL, "ep_restore needs the saved sub_idx");
    if (!sigma) return fail(EP_EINVAL, "ep_restore needs the saved sigma");
    return create(out, X, n, d, l, kernel, bandwidth, s, k, sub_idx, 0, hip_stream, info, sigma,
                  V, nullptr);
}

int ep_step(ep_ctx* c, const int64_t* t, int64_t m, const float* y_b, float* f_out) {
    g_err.clear();
    if (!c) return fail(EP_EINVAL, "ctx is NULL");
    if (!t || !y_b) return fail(EP_EINVAL, "t and y_b must be device pointers");
    if (m < 1 || m > c->n) return fail(EP_EINVAL, "batch size m=%lld outside [1, n]", (long long)m);
    DeviceGuard dg(c->device);
    hipStream_t st = c->stream;
    if (c->checks) {
        std::vector<int64_t> th(m);
        HIP_TRY(hipMemcpyAsync(th.data(), t, m * sizeof(int64_t), hipMemcpyDeviceToHost, st));
        HIP_TRY(hipStreamSynchronize(st));
        c->seen.assign(c->n, 0);
        for (int64_t i = 0; i < m; ++i) {
            if (th[i] < 0 || th[i] >= c->n)
                return fail(EP_EINDEX, "t[%lld]=%lld outside [0,%lld)", (long long)i,
                            (long long)th[i], (long long)c->n);
            if (c->seen[th[i]]) return fail(EP_EINDEX, "t repeats index %lld", (long long)th[i]);
            c->seen[th[i]] = 1;
        }
    }
    int rc = ensure_step_buffers(c, m);
    if (rc) return rc;
    if (c->timing) {
        rc = record(st, c->step_ev, true);
        if (rc) return rc;
    }
    const int64_t m_pad = round_up(m, kBN);
    float* xb = c->xb.as<float>();
    float* xbn = c->xb_norms.as<float>();
    float* alpha = c->alpha.as<float>();
    float* R = c->R.as<float>();

    // step 1: gather the batch
    HIP_TRY(launch_gather_rows(c->X, c->n, c->d, c->norms.as<float>(), t, m, m_pad, xb, xbn,
                               c->err.as<int>(), st));
    // step 2: F = K(X_t, X) alpha, fused; the kernel values of the
    // subsample columns are kept for steps 4-5 when the buffer allows
    int slices = 0;
    int64_t rows_pad = 0;
    const bool capture = capture_subsample(c, xb, m);
    if (capture) HIP_TRY(c->ksb.ensure((size_t)c->s * round_up(m, kBM) * sizeof(float)));
    rc = run_main_pass(c, xb, c->d, xbn, t, m, &slices, &rows_pad, c->timing, capture);
    if (rc) return rc;
    // step 3: R = F - y_b; alpha_t -= c R
    const double coef = 1.0 / (c->info.beta + (double)(m - 1) * c->info.lambda_k1);
    HIP_TRY(launch_reduce_residual(c->part.as<float>(), slices, rows_pad, c->l_pad, m, c->l, y_b,
                                   f_out, R, m_pad, alpha, c->n, t, (float)coef, st));
    if (c->k > 0) {
        rc = subsample_correction(c, capture, xb, xbn, t, m, R, (float)coef);
        if (rc) return rc;
    }
    if (c->timing) {
        rc = record(st, c->step_ev, false);
        if (rc) return rc;
    }
    return EP_OK;
}

int ep_predict(ep_ctx* c, const float* Z, int64_t n_z, float* out) {
    g_err.clear();
    if (!c) return fail(EP_EINVAL, "ctx is NULL");
    if (n_z < 0) return fail(EP_EINVAL, "n_z < 0");
    if (n_z == 0) return EP_OK;
    if (!Z || !out) return fail(EP_EINVAL, "Z and out must be device pointers");
    DeviceGuard dg(c->device);
    hipStream_t st = c->stream;
    const int64_t chunk = 32768;
    HIP_TRY(c->zn.ensure((size_t)std::min(n_z, chunk) * sizeof(float)));
    for (int64_t z0 = 0; z0 < n_z; z0 += chunk) {
        const int64_t nz = std::min(chunk, n_z - z0);
        const float* Zc = Z + z0 * c->d;
        HIP_TRY(launch_row_norms(Zc, nz, c->d, c->d, c->zn.as<float>(), st));
        int slices = 0;
        int64_t rows_pad = 0;
        int rc = run_main_pass(c, Zc, c->d, c->zn.as<float>(), nullptr, nz, &slices, &rows_pad,
                               false);
        if (rc) return rc;
        HIP_TRY(launch_reduce_rows(c->part.as<float>(), slices, rows_pad, c->l_pad, nz, c->l,
                                   out + z0 * c->l, c->l, st));
    }
    return EP_OK;
}

int ep_predict_noalloc(ep_ctx* c, const float* Z, int64_t n_z, float* out) {
    g_err.clear();
    if (!c) return fail(EP_EINVAL, "ctx is NULL");
    if (n_z < 0) return fail(EP_EINVAL, "n_z < 0");
    if (n_z == 0) return EP_OK;
    if (!Z || !out) return fail(EP_EINVAL, "Z and out must be device pointers");
    if (!c->scratch) return fail(EP_EDEVICE, "no scratch address for this device");
    DeviceGuard dg(c->device);
    hipStream_t st = c->stream;
    const int64_t L = c->l_pad;
    // Chunks of tq query tiles: the fused pass's partial slices (slices x
    // 64 tq x L floats) and the chunk's row norms (64 tq floats) must fit
    // the scratch. The slice budget per chunk is what is left after the
    // norms; tq is halved until the pass's plan fits it.
    const int64_t cap = (int64_t)kScratchFloats;
    if (kBM + (int64_t)kBM * L > cap)
        return fail(EP_EINVAL,
                    "ep_predict_noalloc: %lld label columns exceed the %zu-float scratch "
                    "(at most %lld)", (long long)c->l,
                    kScratchFloats, (long long)((cap - kBM) / kBM));
    for (int64_t z0 = 0; z0 < n_z;) {
        int64_t tq = std::min<int64_t>(ceil_div(n_z - z0, kBM), 512);
        tq = std::max<int64_t>(1, std::min<int64_t>(tq, (cap - kBM) / ((int64_t)kBM * (L + 1))));
        KmvPlan plan{};
        int64_t nq = 0, rows_pad = 0;
        for (;; tq /= 2) {
            nq = std::min<int64_t>(n_z - z0, tq * kBM);
            rows_pad = round_up(nq, kBM);
            const int64_t max_sl = (cap - rows_pad) / (rows_pad * L);
            plan = kmv_plan(nq, c->n, c->d, L, c->l, c->kind, (int)std::min<int64_t>(max_sl, 256));
            if (max_sl >= 1 && plan.slices() <= max_sl) break;
            if (tq == 1)
                return fail(EP_EINVAL,
                            "ep_predict_noalloc: the fused pass over %lld centres needs more "
                            "partial sums than the %zu-float scratch holds",
                            (long long)c->n, kScratchFloats);
        }
        float* zn = c->scratch;
        float* part = c->scratch + rows_pad;
        const float* Zc = Z + z0 * c->d;
        HIP_TRY(launch_row_norms(Zc, nq, c->d, c->d, zn, st));
        KmvArgs a{};
        a.Q = Zc;
        a.ldq = c->d;
        a.qn = zn;
        a.qid = nullptr;
        a.nq = nq;
        a.C = c->X;
        a.ldc = c->d;
        a.cn = c->norms.as<float>();
        a.cid = nullptr;
        a.nc = c->n;
        a.d = c->d;
        a.W = c->alpha.as<float>();
        a.ldw = L;
        a.lt = (int)(L / kTile);
        a.out = part;
        a.out_rows = rows_pad;
        a.kind = c->kind;
        a.scale = c->scale;
        HIP_TRY(kmv_launch(a, plan, st, false));
        HIP_TRY(launch_reduce_rows(part, plan.slices(), rows_pad, L, nq, c->l, out + z0 * c->l,
                                   c->l, st));
        z0 += nq;
    }
    return EP_OK;
}

int ep_get_alpha(ep_ctx* c, float* out) {
    g_err.clear();
    if (!c || !out) return fail(EP_EINVAL, "NULL argument");
    DeviceGuard dg(c->device);
    HIP_TRY(hipMemcpy2DAsync(out, c->l * sizeof(float), c->alpha.p, c->l_pad * sizeof(float),
                             c->l * sizeof(float), c->n, hipMemcpyDeviceToDevice, c->stream));
    return EP_OK;
}

int ep_set_alpha(ep_ctx* c, const float* in) {
    g_err.clear();
    if (!c || !in) return fail(EP_EINVAL, "NULL argument");
    DeviceGuard dg(c->device);
    HIP_TRY(hipMemcpy2DAsync(c->alpha.p, c->l_pad * sizeof(float), in, c->l * sizeof(float),
                             c->l * sizeof(float), c->n, hipMemcpyDeviceToDevice, c->stream));
    return EP_OK;
}

int ep_get_preconditioner(ep_ctx* c, double* sigma, double* D, float* V, int64_t* r) {
    g_err.clear();
    if (!c) return fail(EP_EINVAL, "ctx is NULL");
    DeviceGuard dg(c->device);
    if (sigma) std::memcpy(sigma, c->sigma.data(), (c->k + 1) * sizeof(double));
    if (D && c->k) std::memcpy(D, c->D.data(), c->k * sizeof(double));
    if (r) std::memcpy(r, c->r_host.data(), c->s * sizeof(int64_t));
    if (V && c->k) {
        // active rank k of the held V (row stride k_max)
        for (int64_t i = 0; i < c->s; ++i)
            std::memcpy(V + i * c->k, c->Vh.data() + (size_t)i * c->k_max, c->k * sizeof(float));
    }
    return EP_OK;
}

int ep_set_rank(ep_ctx* c, int64_t k) {
    g_err.clear();
    if (!c) return fail(EP_EINVAL, "ctx is NULL");
    if (k < 0 || k > c->k_max)
        return fail(EP_EINVAL, "rank %lld outside [0, %lld]", (long long)k, (long long)c->k_max);
    DeviceGuard dg(c->device);
    return apply_rank(c, k);
}

int ep_adapt(ep_ctx* c, int64_t m_G, ep_info* info) {
    g_err.clear();
    if (!c) return fail(EP_EINVAL, "ctx is NULL");
    if (m_G < 1) return fail(EP_EINVAL, "m_G must be >= 1");
    DeviceGuard dg(c->device);
    // Section 3 Step 2, Eq. 7: the largest rank whose adapted kernel has a
    // critical batch m*(k) = beta(k) s / sigma_{k+1} no larger than m_G
    const std::vector<double> beta = beta_all_ranks(c);
    int64_t best = 0;
    for (int64_t kk = 0; kk <= c->k_max; ++kk) {
        const double mstar = beta[kk] * (double)c->s / c->sigma[kk];
        if (mstar <= (double)m_G) best = kk;
    }
    int rc = apply_rank(c, best);
    if (rc) return rc;
    // Section 3 Step 3: batch m = m_G with the step size for that batch
    ep_info& I = c->info;
    I.m = std::min<int64_t>(c->n, m_G);
    I.eta = (double)I.m / (I.beta + (double)(I.m - 1) * I.lambda_k1);
    // Section 3 Claim: acceleration beta(K)/beta(K_G) * m_G / m*(k), with
    // beta(K) = 1 and m*(k) = s / sigma_1 for the original kernel
    I.accel = (1.0 / I.beta) * (double)I.m / ((double)c->s / c->sigma[0]);
    if (info) *info = I;
    return EP_OK;
}

int ep_batch_sweep(ep_ctx* c, const int64_t* ms, int count, int reps, double* ms_per_pass) {
    g_err.clear();
    if (!c) return fail(EP_EINVAL, "ctx is NULL");
    if (!ms || !ms_per_pass || count < 0 || reps < 1) return fail(EP_EINVAL, "bad arguments");
    for (int i = 0; i < count; ++i)
        if (ms[i] < 1 || ms[i] > c->n) return fail(EP_EINVAL, "batch size outside [1, n]");
    DeviceGuard dg(c->device);
    hipEvent_t e0, e1;
    HIP_TRY(hipEventCreate(&e0));
    HIP_TRY(hipEventCreate(&e1));
    int rc = EP_OK;
    for (int i = 0; i < count && rc == EP_OK; ++i) {
        const int64_t m = ms[i];
        int slices = 0;
        int64_t rows_pad = 0;
        // the step-2 pass with the first m rows of X as the batch
        rc = run_kmv(c, c->X, c->d, c->norms.as<float>(), nullptr, m, c->X, c->d,
                     c->norms.as<float>(), nullptr, c->n, c->alpha.as<float>(), &slices, &rows_pad,
                     false, false);
        if (rc) break;
        if (hipEventRecord(e0, c->stream) != hipSuccess) rc = fail(EP_EDEVICE, "event record");
        for (int r = 0; r < reps && rc == EP_OK; ++r)
            rc = run_kmv(c, c->X, c->d, c->norms.as<float>(), nullptr, m, c->X, c->d,
                         c->norms.as<float>(), nullptr, c->n, c->alpha.as<float>(), &slices,
                         &rows_pad, false, false);
        float t = 0.f;
        if (rc == EP_OK && (hipEventRecord(e1, c->stream) != hipSuccess ||
                            hipEventSynchronize(e1) != hipSuccess ||
                            hipEventElapsedTime(&t, e0, e1) != hipSuccess))
            rc = fail(EP_EDEVICE, "event timing failed");
        ms_per_pass[i] = t / reps;
    }
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    return rc;
}

int ep_batch_knee(const int64_t* ms, const double* t, int count, double tol, int64_t* m_C,
                  double* knee) {
    g_err.clear();
    if (!ms || !t || count < 2) return fail(EP_EINVAL, "need two or more batch sizes");
    if (!(tol >= 0.0 && tol < 1.0)) return fail(EP_EINVAL, "tol must be in [0, 1)");
    for (int i = 0; i < count; ++i) {
        if (ms[i] < 1 || (i > 0 && ms[i] <= ms[i - 1]))
            return fail(EP_EINVAL, "batch sizes must be positive and increasing");
        if (!(t[i] > 0.0) || !std::isfinite(t[i]))
            return fail(EP_EINVAL, "times must be positive and finite");
    }
    // Section 3 Step 1: time per iteration is flat up to the batch that
    // fills the device, then linear. Fit log t = max(log t0, log a + log m):
    // for each split j (points < j flat, >= j linear; j = 0: all linear,
    // j = count: all flat) t0 and a are the geometric means of t and t/m
    // over their parts; the split with the least squared log residual
    // gives the knee t0 / a.
    std::vector<double> lt(count), lm(count);
    for (int i = 0; i < count; ++i) {
        lt[i] = std::log(t[i]);
        lm[i] = std::log((double)ms[i]);
    }
    double best = 1e300, best_knee = (double)ms[0];
    for (int j = 0; j <= count; ++j) {
        double s0 = 0.0, s1 = 0.0;
        for (int i = 0; i < j; ++i) s0 += lt[i];
        for (int i = j; i < count; ++i) s1 += lt[i] - lm[i];
        const double l0 = j > 0 ? s0 / j : -1e300;
        const double la = j < count ? s1 / (count - j) : -1e300;
        double res = 0.0;
        for (int i = 0; i < count; ++i) {
            const double f = std::max(l0, la + lm[i]);
            res += (lt[i] - f) * (lt[i] - f);
        }
        double k;
        if (j == 0) k = (double)ms[0];
        else if (j == count) k = (double)ms[count - 1];
        else k = std::exp(l0 - la);
        if (res < best - 1e-12) {
            best = res;
            best_knee = k;
        }
    }
    const double target = (1.0 - tol) * best_knee;
    int64_t mc = 1;
    while ((double)mc < target && mc < (int64_t(1) << 40)) mc *= 2;
    mc = std::max(ms[0], std::min(ms[count - 1], mc));
    if (m_C) *m_C = mc;
    if (knee) *knee = best_knee;
    return EP_OK;
}

int ep_resource_batch(ep_ctx* c, double tol, int64_t* m_C, int64_t* m_S, int64_t* m_G) {
    g_err.clear();
    if (!c) return fail(EP_EINVAL, "ctx is NULL");
    if (!(tol >= 0.0 && tol < 1.0)) return fail(EP_EINVAL, "tol must be in [0, 1)");
    DeviceGuard dg(c->device);
    // Section 3 Step 1. m_S: batch at which the paper's memory model
    // (d + l + m) n floats fills the device; m_C: the knee of time per
    // iteration against batch size, from the medians of three sweeps.
    hipDeviceProp_t prop;
    HIP_TRY(hipGetDeviceProperties(&prop, c->device));
    const double floats = (double)prop.totalGlobalMem / 4.0;
    const int64_t ms_cap = (int64_t)(floats / (double)c->n) - c->d - c->l;
    std::vector<int64_t> grid;
    for (int64_t m = 16; m <= std::min<int64_t>(c->n, 32768); m *= 2) grid.push_back(m);
    int64_t mc = c->n;
    if (grid.size() >= 2) {
        const int sweeps = 3;
        std::vector<double> t(grid.size() * sweeps);
        for (int r = 0; r < sweeps; ++r) {
            int rc = ep_batch_sweep(c, grid.data(), (int)grid.size(), 3, t.data() + r * grid.size());
            if (rc) return rc;
        }
        std::vector<double> med(grid.size());
        for (size_t i = 0; i < grid.size(); ++i) {
            double v[3] = {t[i], t[i + grid.size()], t[i + 2 * grid.size()]};
            std::sort(v, v + 3);
            med[i] = v[1];
        }
        int rc = ep_batch_knee(grid.data(), med.data(), (int)grid.size(), tol, &mc, nullptr);
        if (rc) return rc;
    } else if (!grid.empty()) {
        mc = grid[0];
    }
    if (m_C) *m_C = mc;
    if (m_S) *m_S = std::max<int64_t>(1, ms_cap);
    if (m_G) *m_G = std::max<int64_t>(1, std::min(mc, ms_cap));
    return EP_OK;
}

int ep_get_info(ep_ctx* c, ep_info* info) {
    g_err.clear();
    if (!c || !info) return fail(EP_EINVAL, "NULL argument");
    *info = c->info;
    return EP_OK;
}

int ep_set_checks(ep_ctx* c, int on) {
    g_err.clear();
    if (!c) return fail(EP_EINVAL, "ctx is NULL");
    c->checks = on != 0;
    return EP_OK;
}

int ep_timing_enable(ep_ctx* c, int on) {
    g_err.clear();
    if (!c) return fail(EP_EINVAL, "ctx is NULL");
    DeviceGuard dg(c->device);
    HIP_TRY(hipStreamSynchronize(c->stream));
    for (auto* v : {&c->kmv_ev, &c->step_ev, &c->kblk_ev, &c->gemm_ev}) {
        for (auto& p : *v) {
            (void)hipEventDestroy(p.a);
            (void)hipEventDestroy(p.b);
        }
        v->clear();
    }
    c->tsum = ep_timing{};
    c->timing = on != 0;
    return EP_OK;
}

int ep_timing_read(ep_ctx* c, ep_timing* out) {
    g_err.clear();
    if (!c || !out) return fail(EP_EINVAL, "NULL argument");
    DeviceGuard dg(c->device);
    HIP_TRY(hipStreamSynchronize(c->stream));
    ep_timing t{};
    for (auto& p : c->kmv_ev) {
        float ms = 0.f;
        HIP_TRY(hipEventElapsedTime(&ms, p.a, p.b));
        t.kmv_ms += ms;
        t.kmv_launches += 1;
    }
    for (auto& p : c->step_ev) {
        float ms = 0.f;
        HIP_TRY(hipEventElapsedTime(&ms, p.a, p.b));
        t.step_ms += ms;
        t.steps += 1;
    }
    for (auto& p : c->kblk_ev) {
        float ms = 0.f;
        HIP_TRY(hipEventElapsedTime(&ms, p.a, p.b));
        t.kblock_ms += ms;
        t.kblock_launches += 1;
    }
    for (auto& p : c->gemm_ev) {
        float ms = 0.f;
        HIP_TRY(hipEventElapsedTime(&ms, p.a, p.b));
        t.gemm_ms += ms;
        t.gemm_launches += 1;
    }
    *out = t;
    return EP_OK;
}

int ep_set_contraction(ep_ctx* c, int mode, int64_t block_bytes) {
    g_err.clear();
    if (!c) return fail(EP_EINVAL, "ctx is NULL");
    if (mode < EP_CONTRACT_AUTO || mode > EP_CONTRACT_BLOCKED)
        return fail(EP_EINVAL, "unknown contraction mode %d", mode);
    if (block_bytes < 0) return fail(EP_EINVAL, "block_bytes < 0");
    c->contract = mode;
    c->block_bytes = block_bytes > 0 ? (size_t)block_bytes : kKBlockBudget;
    return EP_OK;
}

int ep_sync(ep_ctx* c) {
    g_err.clear();
    if (!c) return fail(EP_EINVAL, "ctx is NULL");
    DeviceGuard dg(c->device);
    HIP_TRY(hipStreamSynchronize(c->stream));
    int herr = 0;
    HIP_TRY(hipMemcpy(&herr, c->err.p, sizeof(int), hipMemcpyDeviceToHost));
    if (herr) {
        HIP_TRY(hipMemset(c->err.p, 0, sizeof(int)));
        return fail(EP_EINDEX, "a batch index was outside [0, n)");
    }
    return EP_OK;
}

void ep_destroy(ep_ctx* c) {
    if (!c) return;
    DeviceGuard dg(c->device);
    (void)hipStreamSynchronize(c->stream);
    delete c;
}

}  // extern "C"
