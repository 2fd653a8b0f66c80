// Internal interfaces of libeigenpro (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

namespace ep {

// Tile geometry of the fused kernel-block contraction (kmv.hip). kBN is
// also the granularity of centre splits and of the zero padding that weight
// matrices carry past their last row.
constexpr int kTile = 32;                 // MFMA 32x32 output tile edge
constexpr int kQSub = 2;                  // query sub-tiles per workgroup
constexpr int kCSub = 8;                  // centre sub-tiles per iteration
constexpr int kBM = kTile * kQSub;        // query rows per workgroup (64)
constexpr int kBN = kTile * kCSub;        // centres per iteration (256)
constexpr int kThreads = 512;             // 8 waves of 64

// Bytes every weight matrix of a fused pass carries past its last padded
// row: with three label tiles per wave one 16-byte load fetches three
// weights and drops the fourth, which can lie up to 12 bytes past the row.
constexpr int kWeightTail = 16;

inline int64_t round_up(int64_t a, int64_t b) { return (a + b - 1) / b * b; }
inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// One launch of sum_j k(q_i, c_j) W_j over a centre range, for every query
// row q_i, written as partial sums per centre split.
struct KmvArgs {
    const float* Q;        // queries, nq x d, leading dimension ldq
    int64_t ldq;
    const float* qn;       // |q_i|^2, nq entries
    const int64_t* qid;    // global row id of each query (NULL: none)
    int64_t nq;
    const float* C;        // centres, nc x d, leading dimension ldc
    int64_t ldc;
    const float* cn;       // |c_j|^2, nc entries
    const int64_t* cid;    // global row id of each centre (NULL: j itself)
    int64_t nc;
    int64_t d;
    const float* W;        // weights, >= round_up(nc, kBN) rows x ldw and
    int64_t ldw;           //   kWeightTail readable bytes after them;
                           //   rows >= nc and columns >= l are zero
    int lt;                // label tiles = ldw / 32
    float* out;            // partials [slices][out_rows][ldw]
    int64_t out_rows;      // >= round_up(nq, kBM)
    int64_t cps;           // centres per split, multiple of kBN
    int splits;
    int wl, wj;            // contraction layout: label groups x centre groups
    int kind;              // EP_GAUSSIAN / EP_LAPLACIAN
    float scale;           // exp2 argument scale (see kmv.hip)
    // Optional (vector body only): kpos[j] >= 0 marks centre j as a
    // subsample row; its kernel values k(q_i, c_j) are then also stored at
    // ksb[kpos[j] * ldk + i] (ldk >= nq rounded up to kBM, kpos[j] <
    // s_rows). NULL: none.
    const int* kpos;
    float* ksb;
    int64_t ldk;
    int64_t s_rows;        // rows of ksb; s_rows * ldk * 4 < 2^31
};

// Chooses splits / wave layout and launches; returns the number of partial
// slices written (splits * wj). Buffer sizes are the caller's duty; the
// required slice count for an (nq, nc, ldw) problem comes from kmv_plan.
struct KmvPlan {
    int splits;
    int wl, wj;
    int ltw;               // 32-label tiles per wave (compile-time variant)
    int lt16;              // > 0: 16-wide contraction on lt16 tiles of 16 labels
    int64_t cps;
    int slices() const { return splits * wj; }
};
// l: labels in use (weight columns >= l are zero, ldw >= l)
KmvPlan kmv_plan(int64_t nq, int64_t nc, int64_t ldc, int64_t ldw, int64_t l, int kind,
                 int max_slices);
// Whether a fused launch takes the vector body: d % 4 == 0 and every query
// and centre row 16-byte aligned (the staged body serves the rest).
inline bool kmv_vec(const float* Q, int64_t ldq, const float* C, int64_t ldc, int64_t d) {
    return d % 4 == 0 && (ldq & 3) == 0 && (ldc & 3) == 0 &&
           (reinterpret_cast<uintptr_t>(Q) & 15) == 0 && (reinterpret_cast<uintptr_t>(C) & 15) == 0;
}
// Launches one fused pass per block of up to 1024 label columns (kernel
// values are captured into ksb by the first only). `subsample` selects the
// entry point used for the subsample pass (same code, its own symbol in
// profiles). Capturing (kpos) needs the vector body: hipErrorInvalidValue
// otherwise.
hipError_t kmv_launch(KmvArgs a, const KmvPlan& p, hipStream_t s, bool subsample);

float kernel_scale(int kind, float bandwidth);

// One launch of out[i, j] = k(q_i, c_j) for all nq queries and a chunk of nc
// centres (kblock.hip). Rows must be 16-byte aligned and d % 4 == 0.
struct KblockArgs {
    const float* Q;        // queries, nq x d, leading dimension ldq
    int64_t ldq;
    const float* qn;       // |q_i|^2
    const int64_t* qid;    // global row id of each query (NULL: none)
    int64_t nq;
    const float* C;        // centres of the chunk, nc x d, leading dimension ldc
    int64_t ldc;
    const float* cn;       // |c_j|^2
    int64_t cid_base;      // global row id of centre 0 of the chunk
    int64_t nc;
    int64_t d;
    int kind;
    float scale;
    float* out;            // row-major, >= round_up(nq, 256) rows x ldo
    int64_t ldo;           // >= round_up(nc, 256)
};
hipError_t kblock_launch(const KblockArgs& a, hipStream_t s);

// Thin products of steps 4-5 (thin_gemm.hip):
//   C[p] = sum over depth chunk p of A(i, kk) B(kk, j), i < M, j < N,
// B row-major (K x N, ldb); A row-major (M x K, lda) or, with a_t, the
// transpose of a row-major K x M matrix (A(i, kk) = A[kk lda + i]). Partial
// slice p goes to C + p slice (row-major, ldc). With `scatter` (one depth
// chunk only) the result is added instead, times coef, into
// alpha[r[i] ldalpha + j] for j < N_valid. Leading dimensions must be
// multiples of 4 floats and A, B 16-byte aligned.
struct ThinGemmArgs {
    const float* A;
    int64_t lda;
    const float* B;
    int64_t ldb;
    int64_t M, N, K;
    int64_t kc;            // depth per chunk (set from the plan)
    float* C;
    int64_t ldc;
    int64_t slice;         // floats between partial slices
    float* alpha;          // scatter epilogue
    int64_t ldalpha;
    const int64_t* r;
    float coef;
    int64_t N_valid;
};
struct ThinGemmPlan {
    int64_t kc = 0;        // depth per chunk, a multiple of the 64-deep accumulation block
    int chunks = 1;        // partial slices
    int64_t tiles = 0;
};
// Depth chunks so that tiles x chunks reaches min_groups workgroups (each
// chunk at least 256 deep, at most 64 chunks).
ThinGemmPlan thin_gemm_plan(int64_t M, int64_t N, int64_t K, int min_groups);
hipError_t thin_gemm_launch(const ThinGemmArgs& a, const ThinGemmPlan& pl, bool a_t, bool scatter,
                            hipStream_t st);
// out[i, j] = Dk[i] * sum_p part[p slice + i ld + j] (no scale when Dk is
// NULL), for i < rows, j < cols; slices summed in order.
hipError_t launch_sum_slices(const float* part, int slices, int64_t slice, int64_t rows,
                             int64_t cols, int64_t ld, const float* Dk, float* out, int64_t ldo,
                             hipStream_t st);

// Auxiliary kernels (kernels.hip).
hipError_t launch_row_norms(const float* X, int64_t rows, int64_t d, int64_t ld,
                            float* out, hipStream_t s);
hipError_t launch_gather_rows(const float* X, int64_t n, int64_t d, const float* norms,
                              const int64_t* idx, int64_t m, int64_t m_pad,
                              float* out, float* out_norms, int* err, hipStream_t s);
// R gets r_rows rows (zero beyond m) so that it can serve as the weights of
// a fused pass whose centres are the batch rows.
hipError_t launch_reduce_residual(const float* part, int slices, int64_t rows_pad,
                                  int64_t ldw, int64_t m, int64_t l, const float* y,
                                  float* f_out, float* R, int64_t r_rows, float* alpha,
                                  int64_t n, const int64_t* t, float coef, hipStream_t s);
hipError_t launch_reduce_rows(const float* part, int slices, int64_t rows_pad,
                              int64_t ldw, int64_t rows, int64_t cols, float* out,
                              int64_t ldo, hipStream_t s);
hipError_t launch_subsample_kernel_f64(const float* Xs, int64_t s, int64_t d,
                                       int kind, double bandwidth, double* Ks,
                                       hipStream_t st);
// V[i, j] = Z[i + (col0 + j col_step) ldz] (float32, row-major, ldv) for
// j < k, zero for k <= j < ldv.
hipError_t launch_extract_eigvecs(const double* Z, int64_t ldz, int64_t col0, int64_t col_step,
                                  int64_t s, int64_t k, float* V, int64_t ldv, hipStream_t st);
hipError_t launch_fill_f32(float* p, int64_t count, float v, hipStream_t st);

}  // namespace ep
