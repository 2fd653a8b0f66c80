// Products of steps 4-5 of Algorithm 1 (Eq. 8) on the fp32 matrix cores:
//
//   U = V^T K(X_r, X_t)      (k x m)      or   G = K(X_r, X_t) R   (s x l)
//   W = D (U R)              (k x l)           W = D (V^T G)       (k x l)
//   alpha_r += c V W                           (same)
//
// with V the s x k eigenvector block, D its diagonal scale, R the batch
// residual and K(X_r, X_t) the subsample columns kept by step 2. All are
// thin products (one side of at most a few hundred) whose depth may be long
// (s = 20000), so one kernel serves them all:
//
//   C[p] = sum over depth chunk p of A(i, kk) B(kk, j)
//
// with B row-major (depth x N) and A either row-major (M x depth) or the
// transpose of a row-major (depth x M) matrix. A workgroup of 4 waves owns
// a 64 x 64 output tile, each wave a 32 x 32 block on
// v_mfma_f32_32x32x2f32; operands are staged through LDS in 32-deep stages
// (depth-major, so a lane's operand read is one conflict-free LDS word),
// two stages deep: the next stage is fetched while the current one feeds
// the MFMAs.
// Depth is split into chunks (`kc`, one partial slice each, summed by the
// reduction kernels in slice order) so that enough workgroups exist, and
// inside a chunk the accumulation is blocked: the MFMA accumulator is
// restarted every 64 depth and added into a running sum, so no float32
// chain is longer than 32 MFMA steps plus one addition per block. (The
// component of these products along the top eigenvector sums terms that
// largely cancel; a single chain over the whole depth visibly raised the
// prediction error.)
//
// The last product's epilogue adds coef * (V W)[i, j] straight into
// alpha[r[i], j] (the rows r are distinct, so no two lanes write one
// element).
#include "ep_device.h"
#include "ep_internal.h"

namespace ep {

namespace {

constexpr int kTM = 64, kTN = 64;     // output tile
constexpr int kKS = 32;               // depth per LDS stage
constexpr int kBlk = 64;              // depth per accumulation block
constexpr int kGThreads = 256;
constexpr int kPadA = 4, kPadB = 4;   // LDS row padding (floats)

// Loads floats [j0, j0 + 4) of a row of `len` valid floats: one 16-byte load
// when all four are in range (rows 16-byte aligned), else element by element.
__device__ __forceinline__ float4 ld4(const float* row, int64_t j0, int64_t len) {
    if (j0 + 4 <= len) return *reinterpret_cast<const float4*>(row + j0);
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (j0 < len) v.x = row[j0];
    if (j0 + 1 < len) v.y = row[j0 + 1];
    if (j0 + 2 < len) v.z = row[j0 + 2];
    if (j0 + 3 < len) v.w = row[j0 + 3];
    return v;
}

template <bool A_T, bool SCATTER>
__global__ void __launch_bounds__(kGThreads) thin_gemm_kernel(ThinGemmArgs p) {
    // two LDS stages: the next stage's operands are fetched into registers
    // while the MFMAs read the current one, so one barrier per stage
    __shared__ float As[2][kKS][kTM + kPadA];
    __shared__ float Bs[2][kKS][kTN + kPadB];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int tm = (int)((p.M + kTM - 1) / kTM);
    const int tn = (int)((p.N + kTN - 1) / kTN);
    const int tile = (int)(blockIdx.x % (unsigned)(tm * tn));
    const int chunk = (int)(blockIdx.x / (unsigned)(tm * tn));
    const int64_t i0 = (int64_t)(tile / tn) * kTM;
    const int64_t j0 = (int64_t)(tile % tn) * kTN;
    const int64_t k_lo = (int64_t)chunk * p.kc;
    const int64_t k_hi = min(p.K, k_lo + p.kc);
    const int wm = wave & 1, wn = wave >> 1;

    floatx16 acc, sum;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
        acc[v] = 0.f;
        sum[v] = 0.f;
    }
    // this thread's share of a stage: two quads of A, two of B
    float4 ra[2], rb[2];
    auto fetch = [&](int64_t k0) {
        const int64_t kd = min((int64_t)kKS, k_hi - k0);   // valid depth of the stage
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            const int q = tid + e * kGThreads;
            ra[e] = make_float4(0.f, 0.f, 0.f, 0.f);
            if (A_T) {
                // A(i, kk) = A[kk * lda + i]: quad of (depth, 4 rows)
                const int kk = q / (kTM / 4), ii = 4 * (q % (kTM / 4));
                if (kk < kd) ra[e] = ld4(p.A + (k0 + kk) * p.lda + i0, ii, p.M - i0);
            } else {
                // A(i, kk) = A[i * lda + kk]: quad of (row, 4 depth)
                const int ii = q / (kKS / 4), kk = 4 * (q % (kKS / 4));
                if (i0 + ii < p.M) ra[e] = ld4(p.A + (i0 + ii) * p.lda + k0, kk, kd);
            }
            const int kk = q / (kTN / 4), jj = 4 * (q % (kTN / 4));
            rb[e] = make_float4(0.f, 0.f, 0.f, 0.f);
            if (kk < kd) rb[e] = ld4(p.B + (k0 + kk) * p.ldb + j0, jj, p.N - j0);
        }
    };
    // A tile -> As[depth][row], B tile -> Bs[depth][col]
    auto stash = [&](int buf) {
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            const int q = tid + e * kGThreads;
            if (A_T) {
                const int kk = q / (kTM / 4), ii = 4 * (q % (kTM / 4));
                *reinterpret_cast<float4*>(&As[buf][kk][ii]) = ra[e];
            } else {
                const int ii = q / (kKS / 4), kk = 4 * (q % (kKS / 4));
                As[buf][kk][ii] = ra[e].x;
                As[buf][kk + 1][ii] = ra[e].y;
                As[buf][kk + 2][ii] = ra[e].z;
                As[buf][kk + 3][ii] = ra[e].w;
            }
            const int kk = q / (kTN / 4), jj = 4 * (q % (kTN / 4));
            *reinterpret_cast<float4*>(&Bs[buf][kk][jj]) = rb[e];
        }
    };
    int in_block = 0;
    int buf = 0;
    if (k_lo < k_hi) fetch(k_lo);
    for (int64_t k0 = k_lo; k0 < k_hi; k0 += kKS, buf ^= 1) {
        // the stage written here was last read two stages ago, before the
        // previous barrier
        stash(buf);
        __syncthreads();
        if (k0 + kKS < k_hi) fetch(k0 + kKS);
        const int h = lane >> 5, r = lane & 31;
#pragma unroll
        for (int s2 = 0; s2 < kKS / 2; ++s2) {
            const float a = As[buf][2 * s2 + h][wm * 32 + r];
            const float b = Bs[buf][2 * s2 + h][wn * 32 + r];
            acc = mfma(a, b, acc);
        }
        in_block += kKS;
        if (in_block == kBlk || k0 + kKS >= k_hi) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                sum[v] += acc[v];
                acc[v] = 0.f;
            }
            in_block = 0;
        }
    }

    // element v of this lane: row acc_row(v, lane), column lane % 32
    const int64_t col = j0 + wn * 32 + (lane & 31);
    if (SCATTER) {
        if (col >= p.N_valid) return;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int64_t row = i0 + wm * 32 + acc_row(v, lane);
            if (row < p.M) p.alpha[p.r[row] * p.ldalpha + col] += p.coef * sum[v];
        }
    } else {
        if (col >= p.N) return;
        float* C = p.C + (int64_t)chunk * p.slice;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int64_t row = i0 + wm * 32 + acc_row(v, lane);
            if (row < p.M) C[row * p.ldc + col] = sum[v];
        }
    }
}

// out[i, j] = scale_i * sum_p part[p][i, j] (scale = 1 without Dk), slices
// summed in order.
__global__ void __launch_bounds__(256) sum_slices_kernel(const float* part, int slices,
                                                         int64_t slice, int64_t rows, int64_t cols,
                                                         int64_t ld, const float* Dk, float* out,
                                                         int64_t ldo) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= rows * cols) return;
    const int64_t i = e / cols, j = e - i * cols;
    float f = 0.f;
    for (int s = 0; s < slices; ++s) f += part[(int64_t)s * slice + i * ld + j];
    out[i * ldo + j] = Dk ? Dk[i] * f : f;
}

}  // namespace

ThinGemmPlan thin_gemm_plan(int64_t M, int64_t N, int64_t K, int min_groups) {
    ThinGemmPlan pl;
    const int64_t tiles = ceil_div(M, kTM) * ceil_div(N, kTN);
    // depth chunks: enough workgroups to fill the chip, chunks of whole
    // accumulation blocks and at least 256 deep
    int64_t chunks = std::max<int64_t>(1, ceil_div(min_groups, tiles));
    chunks = std::min<int64_t>(chunks, std::max<int64_t>(1, K / 256));
    chunks = std::min<int64_t>(chunks, 64);
    pl.kc = round_up(ceil_div(K, chunks), kBlk);
    pl.chunks = (int)ceil_div(K, pl.kc);
    pl.tiles = tiles;
    return pl;
}

hipError_t thin_gemm_launch(const ThinGemmArgs& a, const ThinGemmPlan& pl, bool a_t, bool scatter,
                            hipStream_t st) {
    if (a.M <= 0 || a.N <= 0) return hipSuccess;
    if ((a.lda & 3) || (a.ldb & 3) || (reinterpret_cast<uintptr_t>(a.A) & 15) ||
        (reinterpret_cast<uintptr_t>(a.B) & 15))
        return hipErrorInvalidValue;
    if (scatter && pl.chunks != 1) return hipErrorInvalidValue;
    ThinGemmArgs b = a;
    b.kc = pl.kc;
    const dim3 grid((unsigned)(pl.tiles * pl.chunks));
    if (a_t) {
        if (scatter) hipLaunchKernelGGL((thin_gemm_kernel<true, true>), grid, dim3(kGThreads), 0, st, b);
        else hipLaunchKernelGGL((thin_gemm_kernel<true, false>), grid, dim3(kGThreads), 0, st, b);
    } else {
        if (scatter) hipLaunchKernelGGL((thin_gemm_kernel<false, true>), grid, dim3(kGThreads), 0, st, b);
        else hipLaunchKernelGGL((thin_gemm_kernel<false, false>), grid, dim3(kGThreads), 0, st, b);
    }
    return hipGetLastError();
}

hipError_t launch_sum_slices(const float* part, int slices, int64_t slice, int64_t rows,
                             int64_t cols, int64_t ld, const float* Dk, float* out, int64_t ldo,
                             hipStream_t st) {
    if (rows <= 0 || cols <= 0) return hipSuccess;
    const int64_t count = rows * cols;
    hipLaunchKernelGGL(sum_slices_kernel, dim3((unsigned)ceil_div(count, 256)), dim3(256), 0, st,
                       part, slices, slice, rows, cols, ld, Dk, out, ldo);
    return hipGetLastError();
}

}  // namespace ep
