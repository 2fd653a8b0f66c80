// Host-side helpers shared by the library's translation units: error
// reporting, HIP call checking and a grow-only device buffer.
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstddef>

namespace ep {

// Records a printf-style message as the calling thread's last error (read
// back through ep_last_error) and returns `code`.
int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

#define HIP_TRY(expr)                                                                  \
    do {                                                                               \
        hipError_t e_ = (expr);                                                        \
        if (e_ != hipSuccess)                                                          \
            return ::ep::fail(e_ == hipErrorOutOfMemory ? EP_ENOMEM : EP_EDEVICE,      \
                              "%s: %s (%s)", #expr, hipGetErrorString(e_), __func__);  \
    } while (0)

// Grow-only device buffer. Growing frees the old allocation with hipFree,
// which waits for all work on the device first, so kernels still queued
// on the context stream never see their buffer released under them.
struct DevBuf {
    void* p = nullptr;
    size_t bytes = 0;
    DevBuf() = default;
    DevBuf(const DevBuf&) = delete;
    DevBuf& operator=(const DevBuf&) = delete;
    ~DevBuf() { release(); }
    hipError_t ensure(size_t want) {
        if (want <= bytes) return hipSuccess;
        if (p) {
            hipError_t e = hipFree(p);
            if (e != hipSuccess) return e;
            p = nullptr;
            bytes = 0;
        }
        hipError_t e = hipMalloc(&p, std::max<size_t>(want, 256));
        if (e == hipSuccess) bytes = want;
        return e;
    }
    void release() {
        if (p) (void)hipFree(p);
        p = nullptr;
        bytes = 0;
    }
    template <class T>
    T* as() const {
        return static_cast<T*>(p);
    }
};

}  // namespace ep

#include <rocblas/rocblas.h>
#include <stdint.h>
#include <vector>

namespace ep {

// Settings and outcome of the subspace eigensolver (eigsolve.hip); zero
// fields take the defaults documented with ep_setup_opts.
struct EigOpts {
    int max_degree = 0;
    int max_iters = 0;
    int64_t guard = 0;
    double tol = 0.0;
};
struct EigStats {
    int iters = 0;
    int64_t matvecs = 0;
    double max_residual = 0.0;    // max |K v - theta v| / sigma_1 over the pairs returned
};

// Top q eigenpairs of the symmetric positive semi-definite s x s float64
// matrix K (device): theta (host, descending) and V (device, s x q,
// column-major, column j for theta[j]). K is not modified. Returns EP_OK,
// EP_ENUMERIC when the iteration does not converge, EP_ENOMEM/EP_EDEVICE.
int subspace_topq(const double* K, int64_t s, int64_t q, const EigOpts& o, uint64_t seed,
                  rocblas_handle h, hipStream_t st, std::vector<double>& theta, DevBuf& V,
                  EigStats& stats);

}  // namespace ep
