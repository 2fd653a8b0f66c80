// Auxiliary kernels of the EigenPro 2.0 step on gfx950: row norms, batch
// gather, the deterministic split reduction fused with the residual and the
// batch-block update (Algorithm 1 step 3), and the float64 subsample kernel
// matrix of the initialisation.
#include "ep_internal.h"

#include <math.h>

namespace ep {

namespace {

constexpr int kGT = 64;     // tile edge of the float64 K_s kernel
constexpr int kGK = 16;     // its depth per stage

__global__ void __launch_bounds__(256) row_norms_kernel(const float* X, int64_t rows,
                                                        int64_t d, int64_t ld, float* out) {
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= rows) return;
    const float* x = X + row * ld;
    double acc = 0.0;
    for (int64_t j = lane; j < d; j += 64) {
        const double v = x[j];
        acc += v * v;
    }
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_down(acc, off, 64);
    if (lane == 0) out[row] = (float)acc;
}

__global__ void __launch_bounds__(256) gather_rows_kernel(const float* X, int64_t n, int64_t d,
                                                          const float* norms, const int64_t* idx,
                                                          int64_t m, float* out,
                                                          float* out_norms, int* err) {
    const int64_t b = blockIdx.x;
    float* o = out + b * d;
    int64_t src = -1;
    if (b < m) {
        src = idx[b];
        if (src < 0 || src >= n) {
            if (threadIdx.x == 0) atomicOr(err, 1);
            src = -1;
        }
    }
    if (src < 0) {
        for (int64_t j = threadIdx.x; j < d; j += blockDim.x) o[j] = 0.f;
        if (threadIdx.x == 0) out_norms[b] = 0.f;
        return;
    }
    const float* x = X + src * d;
    for (int64_t j = threadIdx.x; j < d; j += blockDim.x) o[j] = x[j];
    if (threadIdx.x == 0) out_norms[b] = norms[src];
}

// F = sum of partial slices; R = F - y_b; alpha[t] -= coef * R (step 3).
// Rows >= m and columns >= l of R are written as zero.
__global__ void __launch_bounds__(256) reduce_residual_kernel(
    const float* part, int slices, int64_t rows_pad, int64_t ldw, int64_t m, int64_t l,
    const float* y, float* f_out, float* R, int64_t r_rows, float* alpha, int64_t n,
    const int64_t* t, float coef) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= r_rows * ldw) return;
    const int64_t b = e / ldw;
    const int64_t c = e - b * ldw;
    if (b >= m || c >= l) {
        R[e] = 0.f;
        return;
    }
    float f = 0.f;
    for (int sl = 0; sl < slices; ++sl) f += part[((int64_t)sl * rows_pad + b) * ldw + c];
    const float r = f - y[b * l + c];
    if (f_out) f_out[b * l + c] = f;
    R[e] = r;
    const int64_t row = t[b];
    if (row >= 0 && row < n) alpha[row * ldw + c] -= coef * r;
}

__global__ void __launch_bounds__(256) reduce_rows_kernel(const float* part, int slices,
                                                          int64_t rows_pad, int64_t ldw,
                                                          int64_t rows, int64_t cols,
                                                          float* out, int64_t ldo) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= rows * cols) return;
    const int64_t b = e / cols;
    const int64_t c = e - b * cols;
    float f = 0.f;
    for (int sl = 0; sl < slices; ++sl) f += part[((int64_t)sl * rows_pad + b) * ldw + c];
    out[b * ldo + c] = f;
}

// K_s[i, j] = k(x_ri, x_rj) in float64 from direct coordinate differences.
__global__ void __launch_bounds__(256) subsample_kernel_f64(const float* Xs, int64_t s,
                                                            int64_t d, int kind, double bw,
                                                            double* Ks) {
    __shared__ double Ai[kGK][kGT + 1];
    __shared__ double Bj[kGK][kGT + 1];
    const int tid = threadIdx.x;
    const int tx = tid & 15, ty = tid >> 4;
    const int64_t i0 = (int64_t)blockIdx.y * kGT;
    const int64_t j0 = (int64_t)blockIdx.x * kGT;
    double acc[4][4] = {};
    for (int64_t k0 = 0; k0 < d; k0 += kGK) {
        for (int e = tid; e < kGK * kGT; e += 256) {
            const int ii = e / kGK, kk = e % kGK;
            const int64_t gk = k0 + kk;
            const int64_t gi = i0 + ii, gj = j0 + ii;
            Ai[kk][ii] = (gi < s && gk < d) ? (double)Xs[gi * d + gk] : 0.0;
            Bj[kk][ii] = (gj < s && gk < d) ? (double)Xs[gj * d + gk] : 0.0;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < kGK; ++kk) {
            double a[4], b[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                a[q] = Ai[kk][ty * 4 + q];
                b[q] = Bj[kk][tx * 4 + q];
            }
#pragma unroll
            for (int p = 0; p < 4; ++p)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const double df = a[p] - b[q];
                    acc[p][q] = fma(df, df, acc[p][q]);
                }
        }
        __syncthreads();
    }
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const int64_t gi = i0 + ty * 4 + p;
        if (gi >= s) continue;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int64_t gj = j0 + tx * 4 + q;
            if (gj >= s) continue;
            const double d2 = acc[p][q];
            Ks[gi * s + gj] = kind == 0 ? exp(-d2 / (2.0 * bw * bw)) : exp(-sqrt(d2) / bw);
        }
    }
}

// V[i, j] = Z[i + (col0 + j col_step) ldz]: the top-k eigenvectors in
// descending order of their eigenvalues, float32, row-major.
__global__ void __launch_bounds__(256) extract_eigvecs_kernel(const double* Z, int64_t ldz,
                                                              int64_t col0, int64_t col_step,
                                                              int64_t s, int64_t k, float* V,
                                                              int64_t ldv) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= s) return;
    for (int64_t j = 0; j < k; ++j) V[i * ldv + j] = (float)Z[i + (col0 + j * col_step) * ldz];
    for (int64_t j = k; j < ldv; ++j) V[i * ldv + j] = 0.f;
}

__global__ void __launch_bounds__(256) fill_kernel(float* p, int64_t count, float v) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e < count) p[e] = v;
}

inline unsigned blocks_for(int64_t count, int per = 256) {
    return (unsigned)((count + per - 1) / per);
}

}  // namespace

hipError_t launch_row_norms(const float* X, int64_t rows, int64_t d, int64_t ld, float* out,
                            hipStream_t s) {
    if (rows <= 0) return hipSuccess;
    hipLaunchKernelGGL(row_norms_kernel, dim3(blocks_for(rows, 4)), dim3(256), 0, s, X, rows,
                       d, ld, out);
    return hipGetLastError();
}

hipError_t launch_gather_rows(const float* X, int64_t n, int64_t d, const float* norms,
                              const int64_t* idx, int64_t m, int64_t m_pad, float* out,
                              float* out_norms, int* err, hipStream_t s) {
    if (m_pad <= 0) return hipSuccess;
    hipLaunchKernelGGL(gather_rows_kernel, dim3((unsigned)m_pad), dim3(256), 0, s, X, n, d,
                       norms, idx, m, out, out_norms, err);
    return hipGetLastError();
}

hipError_t launch_reduce_residual(const float* part, int slices, int64_t rows_pad, int64_t ldw,
                                  int64_t m, int64_t l, const float* y, float* f_out, float* R,
                                  int64_t r_rows, float* alpha, int64_t n, const int64_t* t,
                                  float coef, hipStream_t s) {
    hipLaunchKernelGGL(reduce_residual_kernel, dim3(blocks_for(r_rows * ldw)), dim3(256), 0, s,
                       part, slices, rows_pad, ldw, m, l, y, f_out, R, r_rows, alpha, n, t, coef);
    return hipGetLastError();
}

hipError_t launch_reduce_rows(const float* part, int slices, int64_t rows_pad, int64_t ldw,
                              int64_t rows, int64_t cols, float* out, int64_t ldo,
                              hipStream_t s) {
    if (rows <= 0) return hipSuccess;
    hipLaunchKernelGGL(reduce_rows_kernel, dim3(blocks_for(rows * cols)), dim3(256), 0, s, part,
                       slices, rows_pad, ldw, rows, cols, out, ldo);
    return hipGetLastError();
}

hipError_t launch_subsample_kernel_f64(const float* Xs, int64_t s, int64_t d, int kind,
                                       double bandwidth, double* Ks, hipStream_t st) {
    dim3 grid((unsigned)ceil_div(s, kGT), (unsigned)ceil_div(s, kGT));
    hipLaunchKernelGGL(subsample_kernel_f64, grid, dim3(256), 0, st, Xs, s, d, kind, bandwidth,
                       Ks);
    return hipGetLastError();
}

hipError_t launch_extract_eigvecs(const double* Z, int64_t ldz, int64_t col0, int64_t col_step,
                                  int64_t s, int64_t k, float* V, int64_t ldv, hipStream_t st) {
    hipLaunchKernelGGL(extract_eigvecs_kernel, dim3(blocks_for(s)), dim3(256), 0, st, Z, ldz,
                       col0, col_step, s, k, V, ldv);
    return hipGetLastError();
}

hipError_t launch_fill_f32(float* p, int64_t count, float v, hipStream_t st) {
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(fill_kernel, dim3(blocks_for(count)), dim3(256), 0, st, p, count, v);
    return hipGetLastError();
}

}  // namespace ep
