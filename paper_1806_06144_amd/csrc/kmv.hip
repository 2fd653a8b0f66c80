// Fused kernel-block contraction on gfx950:
//
//   out[q, :] = sum_j k(q, c_j) W[j, :]      (Algorithm 1 step 2: predictions
//                                              f(x_t) = sum_i alpha_i k(x_i, x_t);
//                                              steps 4-5: sum_i k(x_r, x_ti) R_i;
//                                              prediction f(z) of Section 2)
//
// with k the Gaussian or Laplacian kernel of Appendix B. The kernel block is
// produced tile by tile in registers and contracted on the spot; it never
// reaches global memory.
//
// Per workgroup (4 waves): a block of 64 query rows and a contiguous range of
// centres (one "split"), walked 64 centres at a time.
//   1. S = C_tile . Q_tile^T on fp32 MFMA (v_mfma_f32_32x32x2f32): each wave
//      owns one 32x32 sub-tile; features stream through double-buffered LDS
//      in chunks of 32.
//   2. Epilogue in registers: d2 = |q|^2 + |c|^2 - 2 S, clamped at 0; then
//      exp2(scale * d2) (Gaussian) or exp2(scale * sqrt(d2)) (Laplacian).
//      Where the query and the centre are the same training point the value
//      is set to 1 exactly (the fp32 expansion would leave it slightly below).
//   3. The kernel values go to LDS in the MFMA accumulator order, which is
//      exactly the operand order the second product needs, and
//      out^T(labels x queries) += W^T(labels x centres) . K(centres x queries)
//      runs on the same MFMA with W read straight from global memory.
// Partial sums of each split are written to their own slice and summed by a
// separate deterministic reduction.
#include "ep_internal.h"

#include <algorithm>

namespace ep {

typedef float floatx16 __attribute__((ext_vector_type(16)));

namespace {

constexpr int kDC = 32;          // features per staged chunk
constexpr int kLds = kDC + 4;    // padded LDS row (floats): conflict-free b128 reads
constexpr int kMaxLtw = 8;       // label tiles per wave (accumulator budget)

// Row, inside a 32x32 tile, of accumulator element v held by `lane` for the
// 32x32x2 f32 MFMA; the column is lane % 32. The same map gives the k index
// a lane feeds at step v when a product's K dimension is read from such an
// accumulator.
__device__ __forceinline__ int acc_row(int v, int lane) {
    return ((v >> 2) << 3) + ((lane >> 5) << 2) + (v & 3);
}

__device__ __forceinline__ floatx16 mfma(float a, float b, floatx16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float4 load4(const float* base, int64_t row, int64_t nrows,
                                        int64_t ld, int64_t col, int64_t d, bool vec) {
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (row < nrows) {
        const float* ptr = base + row * ld + col;
        if (vec && col + 3 < d) {
            v = *reinterpret_cast<const float4*>(ptr);
        } else {
            if (col < d) v.x = ptr[0];
            if (col + 1 < d) v.y = ptr[1];
            if (col + 2 < d) v.z = ptr[2];
            if (col + 3 < d) v.w = ptr[3];
        }
    }
    return v;
}

template <int KIND>
__device__ __forceinline__ float kernel_value(float d2, float scale) {
    d2 = fmaxf(d2, 0.f);
    if (KIND == 0) return __builtin_amdgcn_exp2f(scale * d2);
    return __builtin_amdgcn_exp2f(scale * __builtin_amdgcn_sqrtf(d2));
}

template <int KIND, int LTW>
__global__ void __launch_bounds__(kThreads) kmv_kernel(KmvArgs p, int vec_ok) {
    __shared__ __attribute__((aligned(16))) float xq[2][kBM][kLds];
    __shared__ __attribute__((aligned(16))) float xc[2][kBN][kLds];
    __shared__ float kb[kCSub][kQSub][16][64];
    __shared__ float s_qn[kBM];
    __shared__ float s_cn[kBN];
    __shared__ int64_t s_qid[kBM];
    __shared__ int64_t s_cid[kBN];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int64_t q0 = (int64_t)blockIdx.x * kBM;
    const int split = blockIdx.y;
    const int64_t cb = (int64_t)split * p.cps;
    const int64_t ce = min(p.nc, cb + p.cps);
    const bool vec = vec_ok != 0;

    if (tid < kBM) {
        const int64_t q = q0 + tid;
        const bool ok = q < p.nq;
        s_qn[tid] = ok ? p.qn[q] : 0.f;
        s_qid[tid] = (ok && p.qid) ? p.qid[q] : -1;
    }

    // distance sub-tile of this wave
    const int jt_s = wave >> 1;
    const int bt_s = wave & 1;
    // contraction role of this wave
    const int gl = wave % p.wl;
    const int gj = wave / p.wl;
    const bool active = wave < p.wl * p.wj;

    floatx16 facc[LTW][kQSub];
#pragma unroll
    for (int i = 0; i < LTW; ++i)
#pragma unroll
        for (int b = 0; b < kQSub; ++b)
#pragma unroll
            for (int v = 0; v < 16; ++v) facc[i][b][v] = 0.f;

    const int lr = tid >> 3;          // staged row (0..31; +32 for the second half)
    const int lc = (tid & 7) << 2;    // staged column inside the chunk
    const int64_t nchunk = (p.d + kDC - 1) / kDC;

    for (int64_t c0 = cb; c0 < ce; c0 += kBN) {
        if (tid < kBN) {
            const int64_t c = c0 + tid;
            const bool ok = c < ce;
            s_cn[tid] = ok ? p.cn[c] : 0.f;
            s_cid[tid] = ok ? (p.cid ? p.cid[c] : c) : -2;
        }
        floatx16 sacc;
#pragma unroll
        for (int v = 0; v < 16; ++v) sacc[v] = 0.f;

        float4 rq0 = load4(p.Q, q0 + lr, p.nq, p.ldq, lc, p.d, vec);
        float4 rq1 = load4(p.Q, q0 + lr + 32, p.nq, p.ldq, lc, p.d, vec);
        float4 rc0 = load4(p.C, c0 + lr, ce, p.ldc, lc, p.d, vec);
        float4 rc1 = load4(p.C, c0 + lr + 32, ce, p.ldc, lc, p.d, vec);
        *reinterpret_cast<float4*>(&xq[0][lr][lc]) = rq0;
        *reinterpret_cast<float4*>(&xq[0][lr + 32][lc]) = rq1;
        *reinterpret_cast<float4*>(&xc[0][lr][lc]) = rc0;
        *reinterpret_cast<float4*>(&xc[0][lr + 32][lc]) = rc1;
        __syncthreads();

        for (int64_t ch = 0; ch < nchunk; ++ch) {
            const int buf = (int)(ch & 1);
            const bool more = ch + 1 < nchunk;
            if (more) {
                const int64_t k1 = (ch + 1) * kDC + lc;
                rq0 = load4(p.Q, q0 + lr, p.nq, p.ldq, k1, p.d, vec);
                rq1 = load4(p.Q, q0 + lr + 32, p.nq, p.ldq, k1, p.d, vec);
                rc0 = load4(p.C, c0 + lr, ce, p.ldc, k1, p.d, vec);
                rc1 = load4(p.C, c0 + lr + 32, ce, p.ldc, k1, p.d, vec);
            }
            // Lane (row = lane%32, half h = lane/32) reads features
            // 8g+4h .. 8g+4h+3; step i of group g pairs feature 8g+i (lower
            // half) with 8g+4+i (upper half). A and B use the same map, so
            // every feature is contracted exactly once.
            const float* arow = &xc[buf][jt_s * 32 + (lane & 31)][(lane >> 5) << 2];
            const float* brow = &xq[buf][bt_s * 32 + (lane & 31)][(lane >> 5) << 2];
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const float4 a = *reinterpret_cast<const float4*>(arow + 8 * g);
                const float4 b = *reinterpret_cast<const float4*>(brow + 8 * g);
                sacc = mfma(a.x, b.x, sacc);
                sacc = mfma(a.y, b.y, sacc);
                sacc = mfma(a.z, b.z, sacc);
                sacc = mfma(a.w, b.w, sacc);
            }
            if (more) {
                *reinterpret_cast<float4*>(&xq[buf ^ 1][lr][lc]) = rq0;
                *reinterpret_cast<float4*>(&xq[buf ^ 1][lr + 32][lc]) = rq1;
                *reinterpret_cast<float4*>(&xc[buf ^ 1][lr][lc]) = rc0;
                *reinterpret_cast<float4*>(&xc[buf ^ 1][lr + 32][lc]) = rc1;
            }
            __syncthreads();
        }

        // epilogue: distances -> kernel values, stored in accumulator order
        {
            const int bl = bt_s * 32 + (lane & 31);
            const float qnb = s_qn[bl];
            const int64_t qidb = s_qid[bl];
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int jl = jt_s * 32 + acc_row(v, lane);
                float kv = kernel_value<KIND>(qnb + s_cn[jl] - 2.f * sacc[v], p.scale);
                if (qidb == s_cid[jl]) kv = 1.f;
                if (c0 + jl >= ce) kv = 0.f;
                kb[jt_s][bt_s][v][lane] = kv;
            }
        }
        __syncthreads();

        // contraction: out^T[label, q] += W[c, label] * K[c, q]
        if (active) {
            for (int jt = gj; jt < kCSub; jt += p.wj) {
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const float k0v = kb[jt][0][v][lane];
                    const float k1v = kb[jt][1][v][lane];
                    const int64_t wrow = c0 + jt * 32 + acc_row(v, lane);
                    const float* wp = p.W + wrow * p.ldw + (lane & 31);
#pragma unroll
                    for (int i = 0; i < LTW; ++i) {
                        const int lt = gl + i * p.wl;
                        if (lt < p.lt) {
                            const float a = wp[lt * 32];
                            facc[i][0] = mfma(a, k0v, facc[i][0]);
                            facc[i][1] = mfma(a, k1v, facc[i][1]);
                        }
                    }
                }
            }
        }
        // The staging barrier of the next iteration orders these kb reads
        // before the next epilogue overwrites kb.
    }

    if (active) {
        const int slice = split * p.wj + gj;
        float* o = p.out + ((int64_t)slice * p.out_rows + q0) * p.ldw;
#pragma unroll
        for (int i = 0; i < LTW; ++i) {
            const int lt = gl + i * p.wl;
            if (lt < p.lt) {
#pragma unroll
                for (int b = 0; b < kQSub; ++b) {
                    const int64_t row = b * 32 + (lane & 31);
#pragma unroll
                    for (int v = 0; v < 16; ++v)
                        o[row * p.ldw + lt * 32 + acc_row(v, lane)] = facc[i][b][v];
                }
            }
        }
    }
}

typedef void (*KmvFn)(KmvArgs, int);

template <int KIND>
KmvFn pick(int ltw) {
    switch (ltw) {
        case 1: return kmv_kernel<KIND, 1>;
        case 2: return kmv_kernel<KIND, 2>;
        case 3: return kmv_kernel<KIND, 3>;
        case 4: return kmv_kernel<KIND, 4>;
        case 5: return kmv_kernel<KIND, 5>;
        case 6: return kmv_kernel<KIND, 6>;
        case 7: return kmv_kernel<KIND, 7>;
        default: return kmv_kernel<KIND, 8>;
    }
}

KmvFn kernel_for(int kind, int ltw) { return kind == 0 ? pick<0>(ltw) : pick<1>(ltw); }

int occupancy_slots(int kind, int ltw) {
    static int cus = -1;
    if (cus < 0) {
        int dev = 0;
        hipDeviceProp_t prop;
        if (hipGetDevice(&dev) != hipSuccess || hipGetDeviceProperties(&prop, dev) != hipSuccess)
            cus = 256;
        else
            cus = prop.multiProcessorCount;
    }
    int per = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, kernel_for(kind, ltw), kThreads, 0) !=
            hipSuccess ||
        per < 1)
        per = 1;
    return per * cus;
}

}  // namespace

float kernel_scale(int kind, float bandwidth) {
    const double log2e = 1.4426950408889634;
    const double bw = bandwidth;
    if (kind == 0) return (float)(-log2e / (2.0 * bw * bw));
    return (float)(-log2e / bw);
}

KmvPlan kmv_plan(int64_t nq, int64_t nc, int64_t ldw, int kind, int max_slices) {
    KmvPlan best{};
    const int lt = (int)std::min<int64_t>(ldw / 32, 32);
    // contraction layout: fewest MFMA items on the busiest wave
    const int layouts[3][2] = {{4, 1}, {2, 2}, {1, 2}};
    int best_cost = 1 << 30;
    for (auto& lw : layouts) {
        const int wl = lw[0], wj = lw[1];
        const int ltw = (lt + wl - 1) / wl;
        if (ltw > kMaxLtw) continue;
        const int cost = ltw * (kCSub / wj);
        if (cost < best_cost) {
            best_cost = cost;
            best.wl = wl;
            best.wj = wj;
            best.ltw = ltw;
        }
    }
    const int slots = occupancy_slots(kind, best.ltw);
    const int64_t tq = ceil_div(std::max<int64_t>(nq, 1), kBM);
    const int64_t nct = ceil_div(std::max<int64_t>(nc, 1), kBN);
    // splits of the centre axis: minimise the makespan of tq * splits equal
    // workgroups over the resident slots
    int64_t best_p = 1, best_per = nct;
    double best_t = 1e300;
    for (int64_t P = 1; P <= nct && P * best.wj <= max_slices; ++P) {
        const int64_t per = ceil_div(nct, P);
        const int64_t peff = ceil_div(nct, per);
        if (peff != P) continue;
        const int64_t rounds = ceil_div(tq * peff, slots);
        const double t = (double)rounds * (double)(per + 1);
        if (t < best_t) {
            best_t = t;
            best_p = peff;
            best_per = per;
        }
    }
    best.splits = (int)best_p;
    best.cps = best_per * kBN;
    return best;
}

hipError_t kmv_launch(KmvArgs a, const KmvPlan& p, hipStream_t s) {
    a.cps = p.cps;
    a.splits = p.splits;
    a.wl = p.wl;
    a.wj = p.wj;
    const int vec_ok = ((a.ldq & 3) == 0) && ((a.ldc & 3) == 0) &&
                       ((reinterpret_cast<uintptr_t>(a.Q) & 15) == 0) &&
                       ((reinterpret_cast<uintptr_t>(a.C) & 15) == 0);
    dim3 grid((unsigned)ceil_div(std::max<int64_t>(a.nq, 1), kBM), (unsigned)p.splits);
    const int lt_total = a.lt;
    for (int t0 = 0; t0 < lt_total; t0 += 32) {
        KmvArgs b = a;
        b.W = a.W + (int64_t)t0 * 32;
        b.out = a.out + (int64_t)t0 * 32;
        b.lt = std::min(32, lt_total - t0);
        hipLaunchKernelGGL(kernel_for(a.kind, p.ltw), grid, dim3(kThreads), 0, s, b, vec_ok);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace ep
