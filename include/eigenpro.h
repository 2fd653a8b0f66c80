/*
 * eigenpro.h — C ABI of libeigenpro, an MI355X (gfx950) implementation of
 * one EigenPro 2.0 iteration (Ma & Belkin, "Kernel machines that adapt to
 * GPUs for effective large batch training", arXiv 1806.06144).
 *
 * Conventions shared by every call
 *   - Matrices are row-major float32 unless stated; "device" pointers are
 *     HIP device memory on the device that was current at ep_setup.
 *   - All work is enqueued on the stream given to ep_setup and is
 *     asynchronous unless stated. Device buffers passed in are borrowed for
 *     the duration of the call's device work: keep them alive until ep_sync
 *     (or a stream synchronisation) returns.
 *   - Return value: EP_OK (0) or a negative EP_E* code. The text of the last
 *     error of the calling thread is available from ep_last_error(). No C++
 *     exception crosses this boundary.
 *   - A context is not thread-safe: calls on one context must not overlap.
 *     Different contexts are independent.
 */
#ifndef EIGENPRO_H
#define EIGENPRO_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    EP_OK = 0,
    EP_EINVAL = -1,    /* an argument is out of its documented range        */
    EP_ENOMEM = -2,    /* a device or host allocation failed                 */
    EP_EDEVICE = -3,   /* a HIP / rocSOLVER call failed                      */
    EP_ENUMERIC = -4,  /* eigensolve failed or sigma_{k+1} <= 0              */
    EP_EINDEX = -5     /* a batch index was out of range or repeated         */
};

enum {
    EP_GAUSSIAN = 0,   /* k(x,z) = exp(-|x-z|^2 / (2 bw^2))  (Appendix B)    */
    EP_LAPLACIAN = 1   /* k(x,z) = exp(-|x-z| / bw)          (Appendix B)    */
};

typedef struct ep_ctx ep_ctx;

/* Products of setup (Algorithm 1 initialisation; Sections 3 and 4). */
typedef struct ep_info {
    int64_t n, d, l, s, k;
    double sigma_1;     /* largest eigenvalue of K_s                          */
    double sigma_k1;    /* sigma_{k+1}: level the top k eigenvalues flatten to */
    double lambda_k1;   /* sigma_{k+1} / s: top eigenvalue of the adapted
                           operator (Nystrom, Section 4)                      */
    double beta;        /* beta(K_G): max of k_G(x,x) over the s subsample
                           points (Section 3, Step 2)                         */
    double m_star;      /* beta / lambda_k1: critical batch of the adapted
                           kernel (Section 2)                                 */
    int64_t m;          /* min(n, max(1, floor(m_star)))                       */
    double eta;         /* m / (beta + (m-1) lambda_k1): step size at m; one
                           step moves each coordinate by eta/m times its
                           residual                                          */
    double setup_ms;    /* wall time of ep_setup                              */
    int64_t k_max;      /* rank of the eigensystem held (the k of ep_setup);
                           the active rank k can be lowered to any value
                           <= k_max without a new eigensolve (ep_set_rank,
                           ep_adapt)                                         */
    double accel;       /* after ep_adapt: beta(K)/beta(K_G) * m_G / m*(k),
                           the acceleration of Section 3's claim (0 before)  */
    int64_t solver;     /* eigensolver that produced sigma and V:
                           EP_SOLVER_DENSE or EP_SOLVER_SUBSPACE; 0 after
                           ep_restore (none ran)                              */
    int64_t solver_iters;   /* SUBSPACE: outer (filter + Rayleigh-Ritz)
                               iterations; 0 otherwise                        */
    int64_t solver_matvecs; /* SUBSPACE: products of K_s with a vector, in
                               total; 0 otherwise                             */
    double eig_residual;    /* SUBSPACE: max_j |K_s v_j - sigma_j v_j| /
                               sigma_1 over the k+1 pairs; 0 otherwise        */
} ep_info;

/* Eigensolvers for the top k+1 eigenpairs of K_s (ep_setup_opts.solver). */
enum {
    EP_SOLVER_AUTO = 0,     /* SUBSPACE when s >= 2048 and the block
                               (k+1+guard columns) is at most s/16; else
                               DENSE                                          */
    EP_SOLVER_DENSE = 1,    /* full divide-and-conquer eigendecomposition of
                               K_s (rocSOLVER dsyevd), O(s^3)                 */
    EP_SOLVER_SUBSPACE = 2  /* Chebyshev-filtered block subspace iteration with
                               Rayleigh-Ritz and locking, O(s^2 (k+guard))
                               per filter degree                              */
};

/* Options of ep_setup_ex; zero in any field selects its default. */
typedef struct ep_setup_opts {
    int32_t solver;      /* EP_SOLVER_*                         (AUTO)        */
    int32_t max_degree;  /* cap on the Chebyshev degree of one filter (20)    */
    int32_t max_iters;   /* outer iterations before giving up      (100)      */
    int32_t no_fallback; /* nonzero: a SUBSPACE solve that does not converge
                            returns EP_ENUMERIC; zero: DENSE runs instead     */
    int64_t guard;       /* block columns beyond k+1: max(32, (k+1)/4)
                            rounded up to a multiple of 16                    */
    double tol;          /* a Ritz pair is accepted when |K_s v - theta v| <=
                            tol * sigma_1                           (1e-11)   */
} ep_setup_opts;

/*
 * ep_setup — Algorithm 1 initialisation, Section 4 (Nystrom extension) and
 * Section 3 Steps 2-3 (beta, critical batch, step size).
 *
 *   ctx        out: new context (NULL on failure).
 *   X          device, n x d, row-major float32 training features (the
 *              kernel centres). BORROWED: never copied, must stay alive and
 *              unchanged until ep_destroy.
 *   n, d, l    centres, feature dimension, label columns; each >= 1,
 *              d <= 2^20.
 *   kernel     EP_GAUSSIAN or EP_LAPLACIAN; bandwidth > 0 and finite.
 *   s, k       subsample size and preconditioner rank, 0 <= k < s <= n.
 *              The top k+1 eigenpairs of K_s = [k(x_ri, x_rj)] are computed;
 *              the top k directions are flattened to sigma_{k+1}.
 *   sub_idx    host, s distinct indices in [0, n), or NULL to draw s
 *              indices uniformly without replacement from `seed`.
 *   hip_stream hipStream_t to enqueue all work on (NULL = default stream).
 *   info       out (may be NULL): see ep_info.
 * Sets alpha = 0. Blocks until setup is complete. K_s is formed in float64;
 * the eigensolve runs on the device in float64 with EP_SOLVER_AUTO (see
 * ep_setup_ex).
 * Errors: EP_EINVAL (ranges above, duplicate/out-of-range sub_idx),
 * EP_ENOMEM, EP_EDEVICE, EP_ENUMERIC.
 */
int ep_setup(ep_ctx** ctx, const float* X, int64_t n, int64_t d, int64_t l,
             int kernel, float bandwidth, int64_t s, int64_t k,
             const int64_t* sub_idx, uint64_t seed, void* hip_stream,
             ep_info* info);

/*
 * ep_setup_ex — ep_setup with a choice of eigensolver for K_s (Algorithm 1
 * initialisation; the Nystrom extension of Section 4 needs sigma_1 ..
 * sigma_{k+1} and v_1 .. v_k only, so the full spectrum need not be formed).
 *   opts  host, may be NULL (all defaults; then identical to ep_setup).
 * Both solvers work in float64 on K_s. SUBSPACE starts from a block drawn
 * from `seed` and accepts a pair at the residual bound opts->tol; its
 * eigenvalues agree with DENSE to that bound or better, and V D V^T (the
 * only use of the eigenvectors) is insensitive to rotations within
 * clusters of nearly equal eigenvalues. Errors: as ep_setup, plus
 * EP_EINVAL for an unknown solver or negative option, and EP_ENUMERIC when
 * SUBSPACE does not converge and no_fallback is set.
 */
int ep_setup_ex(ep_ctx** ctx, const float* X, int64_t n, int64_t d, int64_t l,
                int kernel, float bandwidth, int64_t s, int64_t k,
                const int64_t* sub_idx, uint64_t seed, void* hip_stream,
                const ep_setup_opts* opts, ep_info* info);

/*
 * ep_restore — rebuild a context from a saved setup (checkpoint / resume):
 * the same as ep_setup with the subsample and eigensystem supplied instead
 * of computed, so no eigensolver runs.
 *   sub_idx  host, the s subsample indices that were used (required).
 *   sigma    host double[k+1], descending eigenvalues of K_s (required).
 *   V        host float[s*k], row-major top-k eigenvectors, row i for
 *            sub_idx[i] (may be NULL when k = 0).
 * beta, m* and eta are recomputed from sigma and V. alpha is set to 0; use
 * ep_set_alpha to restore it. ep_get_preconditioner returns exactly these
 * three arrays. Errors: as ep_setup, plus EP_EINVAL for missing arrays,
 * non-finite or increasing sigma, sigma_{k+1} <= 0, non-finite V.
 */
int ep_restore(ep_ctx** ctx, const float* X, int64_t n, int64_t d, int64_t l,
               int kernel, float bandwidth, int64_t s, int64_t k,
               const int64_t* sub_idx, const double* sigma, const float* V,
               void* hip_stream, ep_info* info);

/*
 * ep_step — one iteration of Algorithm 1 (steps 1-5) on a batch of m points.
 *
 *   t       device int64[m]: batch indices, distinct, in [0, n).
 *   m       1 <= m <= n. The step coefficient is 1/(beta + (m-1) lambda_k1)
 *           for this call's m, so a short last batch is handled.
 *   y_b     device float32 m x l: labels of the batch rows.
 *   f_out   device float32 m x l or NULL: receives f(x_t) before the update.
 * Computes F = K(X_t, X) alpha, R = F - y_b, updates alpha_t -= c R and
 * alpha_r += c V D V^T K(X_r, X_t) R with D_i = (1 - sigma_{k+1}/sigma_i) /
 * sigma_i. K(X_r, X_t) is not recomputed: the fused step-2 pass keeps
 * those columns of the kernel block (a context buffer of s x m floats, at
 * most 2 GiB, grown on demand) as the paper reads them from its stored
 * block; past that size, with the blocked form, or for rows that are not
 * 16-byte aligned, a separate fused pass recomputes them.
 * Asynchronous. Indices outside [0, n) are not read or written
 * and make the next ep_sync return EP_EINDEX; repeated indices are
 * rejected with EP_EINDEX only when index checking is enabled
 * (ep_set_checks), since that check copies t to the host and synchronises.
 * Errors: EP_EINVAL (m out of range, NULL t / y_b), EP_EINDEX, EP_ENOMEM,
 * EP_EDEVICE.
 */
int ep_step(ep_ctx* ctx, const int64_t* t, int64_t m, const float* y_b,
            float* f_out);

/*
 * ep_predict — f(z) = sum_i alpha_i k(x_i, z) (Section 2) for each row z.
 *   Z    device float32 n_z x d.   out  device float32 n_z x l.
 * n_z >= 0 (0 is a no-op). Asynchronous.
 */
int ep_predict(ep_ctx* ctx, const float* Z, int64_t n_z, float* out);

/*
 * ep_predict_noalloc — ep_predict for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc. Same arguments and result (up to float32 summation
 * order); it calls no allocating routine. Its scratch (the row norms of a
 * chunk of Z and the partial sums of the fused pass) is a 64 MiB array that
 * the library holds once per device for the life of the process, looked up
 * when the first context is created on that device. Z is processed in
 * chunks sized to fit it; always the fused form (ep_set_contraction does
 * not apply).
 * Concurrency: every call on one device shares that device's scratch, so
 * calls that overlap on one GPU (two streams, two threads, two contexts)
 * race; serialise them. The scratch keeps the last call's contents; nothing
 * in it needs to start at zero.
 * Errors: EP_EINVAL (NULL Z / out, n_z < 0, or l so large that one 64-row
 * chunk's partial sums exceed the scratch: l > 262143), EP_EDEVICE.
 */
int ep_predict_noalloc(ep_ctx* ctx, const float* Z, int64_t n_z, float* out);

/* alpha as a dense n x l float32 device matrix (copy out / copy in).
 * Asynchronous on the context stream. */
int ep_get_alpha(ep_ctx* ctx, float* out);
int ep_set_alpha(ep_ctx* ctx, const float* in);

/* Setup products for inspection (host buffers; blocking):
 *   sigma  double[k+1] descending eigenvalues of K_s (may be NULL)
 *   D      double[k] preconditioner scales (may be NULL)
 *   V      float[s*k] row-major top-k eigenvectors, row i for r_i (may be NULL)
 *   r      int64[s] subsample indices (may be NULL) */
int ep_get_preconditioner(ep_ctx* ctx, double* sigma, double* D, float* V,
                          int64_t* r);

int ep_get_info(ep_ctx* ctx, ep_info* info);

/*
 * Resource-adaptive parameters (Section 3, Steps 1-3).
 *
 * ep_set_rank(ctx, k): make rank k (0 <= k <= info.k_max) the active
 *   preconditioner: V keeps its top k columns, D, beta(K_G), lambda =
 *   sigma_{k+1}/s, m* and the step size are recomputed from the held
 *   eigensystem (no new eigensolve). Errors: EP_EINVAL.
 * ep_adapt(ctx, m_G, info): Step 2 / Eq. 7 — choose the largest rank k <=
 *   k_max whose adapted kernel has critical batch m*(k) = beta(k) s /
 *   sigma_{k+1} <= m_G, make it active, and (Step 3) set the batch to
 *   min(n, m_G) with its step size; info.accel gets the acceleration
 *   beta(K)/beta(K_G) * m_G / m*(k) of the original kernel's m*(k) = s /
 *   sigma_1. Errors: EP_EINVAL (m_G < 1).
 * ep_batch_sweep(ctx, ms, count, reps, ms_per_pass): times the step-2
 *   fused pass (the first ms[i] rows of X as the batch, against all n
 *   centres, current alpha) for each batch size, averaged over reps launches,
 *   in ms (host array of count doubles). Synchronises. Errors: EP_EINVAL.
 * ep_resource_batch(ctx, tol, m_C, m_S, m_G): Step 1. m_S = the batch at
 *   which the paper's memory model (d + l + m) n floats fills the device's
 *   memory; m_C = the batch where time per iteration stops being flat
 *   ((d + l) m_C n ~ the device's parallel capacity): the step-2 pass is
 *   timed at power-of-two batches 16 .. min(n, 32768), three sweeps of three
 *   launches each, the median of each batch is kept, and ep_batch_knee
 *   places the knee; m_G = min(m_C, m_S). Any output may be NULL.
 *   Synchronises. Errors: EP_EINVAL (tol outside [0, 1)).
 * ep_batch_knee(ms, ms_per_pass, count, tol, m_C, knee): host only (no
 *   device work). Fits time(m) = max(t0, a m), flat then linear, to count >= 2
 *   increasing batch sizes ms and their times by least squares on log time
 *   (each split of the points into a flat and a linear part fits t0 and a
 *   as geometric means; the split with the smallest residual wins), and
 *   returns the knee t0 / a and m_C = the smallest power of two at or above
 *   (1 - tol) knee, clamped to [ms[0], ms[count-1]]. Either output may be
 *   NULL. Errors: EP_EINVAL (count < 2, ms not increasing or < 1, a time
 *   not positive and finite, tol outside [0, 1)).
 */
int ep_set_rank(ep_ctx* ctx, int64_t k);
int ep_adapt(ep_ctx* ctx, int64_t m_G, ep_info* info);
int ep_batch_sweep(ep_ctx* ctx, const int64_t* ms, int count, int reps,
                   double* ms_per_pass);
int ep_resource_batch(ep_ctx* ctx, double tol, int64_t* m_C, int64_t* m_S,
                      int64_t* m_G);
int ep_batch_knee(const int64_t* ms, const double* ms_per_pass, int count, double tol,
                  int64_t* m_C, double* knee);

/* Enable (1) / disable (0, default) host-side validation of batch indices
 * in ep_step (copies t to the host and synchronises). */
int ep_set_checks(ep_ctx* ctx, int on);

/* Timing of the dominant kernel (the fused kernel-block contraction of
 * step 2) and of whole steps, by HIP events on the context stream.
 * ep_timing_enable(ctx, 1) starts recording and clears totals;
 * ep_timing_read synchronises the stream and returns the totals in ms. */
typedef struct ep_timing {
    double kmv_ms;          /* sum over steps of the step-2 pass
                               F = K(X_t, X) alpha (one fused launch, or all
                               launches of the blocked form)               */
    int64_t kmv_launches;   /* number of step-2 passes timed               */
    double step_ms;         /* sum over ep_step calls */
    int64_t steps;
    double kblock_ms;       /* blocked form only: sum over launches of the
                               kernel-block kernel (distances -> kernel
                               values of one centre chunk)                 */
    int64_t kblock_launches;
    double gemm_ms;         /* blocked form only: sum over the contraction
                               GEMMs F += K_chunk alpha_chunk              */
    int64_t gemm_launches;
} ep_timing;
int ep_timing_enable(ep_ctx* ctx, int on);
int ep_timing_read(ep_ctx* ctx, ep_timing* out);

/* How F = K(Z, X) alpha is formed (Algorithm 1 step 2, prediction):
 *   EP_CONTRACT_FUSED    one kernel produces kernel values tile by tile in
 *                        registers and contracts them with alpha at once;
 *                        the kernel block never reaches memory.
 *   EP_CONTRACT_BLOCKED  the paper's order of work, one centre chunk at a
 *                        time: a kernel writes the chunk's kernel block
 *                        (at most block_bytes), then a GEMM adds block x
 *                        alpha chunk into F. Needs d % 4 == 0 and 16-byte aligned
 *                        rows (else the fused form runs).
 *   EP_CONTRACT_AUTO     the fused form (default). The blocked form is
 *                        slower (a little at l = 1000, several times at
 *                        small l, where its GEMM is skinny) and writes the
 *                        block to memory, so it is only taken on request.
 * Both forms give the same values up to float32 summation order. The
 * blocked form recomputes K(X_r, X_t) for steps 4-5 in a fused subsample
 * pass (see ep_step). */
enum { EP_CONTRACT_AUTO = 0, EP_CONTRACT_FUSED = 1, EP_CONTRACT_BLOCKED = 2 };
/*   block_bytes  upper bound of the blocked form's kernel-block buffer
 *                (0: 2 GiB); chunks shrink to fit it, down to 256 centres.
 * Errors: EP_EINVAL for an unknown mode or negative block_bytes. */
int ep_set_contraction(ep_ctx* ctx, int mode, int64_t block_bytes);

/* Device probe (no context): runs a register-only kernel of independent
 * fp32 MFMA chains (v_mfma_f32_32x32x2f32, two waves per SIMD on every CU)
 * on the current device and default stream, and reports the rate it
 * sustains in TFLOP/s and the shader clock during it in MHz (ratio of the
 * shader cycle counter to the 100 MHz constant counter). Blocking; about
 * 0.1 s. Either out-pointer may be NULL. Errors: EP_EDEVICE, EP_ENOMEM. */
int ep_device_probe(double* mfma_f32_tflops, double* shader_clock_mhz);

/* Wait for all work of the context; reports deferred device errors
 * (EP_EDEVICE) and out-of-range batch indices seen since the last call
 * (EP_EINDEX). */
int ep_sync(ep_ctx* ctx);

/* Free the context and everything it owns (not X). NULL is a no-op. */
void ep_destroy(ep_ctx* ctx);

/* Message for the calling thread's last error ("" if none). */
const char* ep_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* EIGENPRO_H */
