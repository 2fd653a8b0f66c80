// Kernel block on gfx950: out[i, j] = k(q_i, c_j) for a block of queries
// and a chunk of centres (Algorithm 1 step 2 evaluates K(X_t, X); with the
// contraction F = K(X_t, X) alpha done afterwards by a plain GEMM, this is
// the paper's own order of work, one centre chunk at a time so the m x n
// block never exists whole).
//
// The distance product S = Q C^T is a large-tile fp32 MFMA GEMM:
// one workgroup = 8 waves (two per SIMD) owns a 256 x 256 output tile; each
// wave owns 64 queries x 128 centres = 2 x 4 sub-tiles of
// v_mfma_f32_32x32x2f32 with independent accumulators, so per group of 8
// features it reads 6 operand quads from LDS for 32 MFMAs. Feature chunks
// of 16 are copied from global memory straight into LDS
// (buffer_load_dwordx4 ... lds) into four rotating slots, three chunks
// ahead, with quads permuted by swz16 so that operand reads are free of
// bank conflicts. Each wave reads the first group of the next chunk before
// the barrier that ends a chunk. The epilogue applies the kernel function
// of Appendix B in registers: d2 = |q|^2 + |c|^2 - 2 S (clamped at 0),
// exp2(scale * d2) or exp2(scale * sqrt(d2)), k = 1 where the query and
// the centre are the same training point.
#include "ep_device.h"
#include "ep_internal.h"

#include <type_traits>

namespace ep {

namespace {

constexpr int kKM = 256;                // query rows per tile
constexpr int kKN = 256;                // centres per tile
constexpr int kKD = 16;                 // features per chunk (two groups of 8)
constexpr int kKRows = kKM + kKN;       // staged rows per chunk
constexpr int kKSlot = kKRows * kKD;    // floats per LDS slot (32 KB)
constexpr int kKThreads = 512;
constexpr int kKLoads = kKRows / 16 / (kKThreads / 64);   // direct loads per wave per chunk
static_assert(kKLoads == 4, "four 1 KB loads per wave and chunk");

template <int KIND>
__global__ void __launch_bounds__(kKThreads) kblock_kernel(KblockArgs p) {
    __shared__ __attribute__((aligned(16))) float xs0[kKSlot];
    __shared__ __attribute__((aligned(16))) float xs1[kKSlot];
    __shared__ __attribute__((aligned(16))) float xs2[kKSlot];
    __shared__ __attribute__((aligned(16))) float xs3[kKSlot];
    __shared__ float s_qn[kKM];
    __shared__ int64_t s_qid[kKM];
    __shared__ float s_cn[kKN];
    __shared__ int64_t s_cid[kKN];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wv = wave;
    const int tq = (int)((p.nq + kKM - 1) / kKM);
    const int ctile = (int)blockIdx.x / tq;
    const int qtile = (int)blockIdx.x - ctile * tq;
    const int64_t q0 = (int64_t)qtile * kKM;
    const int64_t c0 = (int64_t)ctile * kKN;
    const int64_t q_rows = min((int64_t)kKM, p.nq - q0);
    const int64_t c_rows = min((int64_t)kKN, p.nc - c0);
    const int nchunk = (int)((p.d + kKD - 1) / kKD);
    const int d = (int)p.d;

    if (tid < kKM) {
        const bool ok = tid < q_rows;
        s_qn[tid] = ok ? p.qn[q0 + tid] : 0.f;
        s_qid[tid] = (ok && p.qid) ? p.qid[q0 + tid] : -1;
    } else {
        const int j = tid - kKM;
        const bool ok = j < c_rows;
        s_cn[j] = ok ? p.cn[c0 + j] : 0.f;
        s_cid[j] = ok ? p.cid_base + c0 + j : -2;
    }

    // Direct loads: load i of this wave fills staged rows 16j .. 16j+15,
    // j = 4*wave + i (queries 0..255, then centres); lane L takes row
    // 16j + L/4 and stores at quad position L%4, so it fetches quad
    // (L%4) ^ swz16(row) of that row.
    const __amdgpu_buffer_rsrc_t qrs =
        make_rsrc(p.Q + q0 * p.ldq, ((q_rows - 1) * p.ldq + p.d) * 4);
    const __amdgpu_buffer_rsrc_t crs =
        make_rsrc(p.C + c0 * p.ldc, ((c_rows - 1) * p.ldc + p.d) * 4);
    int dma_voff[kKLoads], dma_col[kKLoads];
#pragma unroll
    for (int i = 0; i < kKLoads; ++i) {
        const int j = kKLoads * wv + i;
        const int r = 16 * j + (lane >> 2);
        const int q = (lane & 3) ^ swz16(r);
        dma_col[i] = 4 * q;
        dma_voff[i] = (r < kKM ? r * (int)p.ldq : (r - kKM) * (int)p.ldc) * 4 + 16 * q;
    }
    auto slot_of = [&](auto tag) -> float* {
        constexpr int S = decltype(tag)::value;
        if constexpr (S == 0) return xs0;
        else if constexpr (S == 1) return xs1;
        else if constexpr (S == 2) return xs2;
        else return xs3;
    };
    auto dma = [&](auto tag, int chunk) {
        float* base = slot_of(tag);
        const int kbase = chunk * kKD;
#pragma unroll
        for (int i = 0; i < kKLoads; ++i) {
            const int j = kKLoads * wv + i;
            const int voff = kbase + dma_col[i] < d ? dma_voff[i] : kOOB;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(j < kKM / 16 ? qrs : crs,
                                                     (lds_void*)(base + j * 16 * kKD), 16, voff,
                                                     kbase * 4, 0, 0);
        }
    };

    // Operands: lane (row = lane%32, half h = lane/32) feeds features
    // 8g+4h .. 8g+4h+3 of group g; queries are the A side (output rows),
    // centres the B side (output columns).
    const int wm = wave & 3;
    const int wn = wave >> 2;
    const int h = lane >> 5;
    const int f = swz16(lane & 31);
    const int a_off = (wm * 64 + (lane & 31)) * kKD;
    const int b_off = (kKM + wn * 128 + (lane & 31)) * kKD;
    auto rd = [&](const float* base, int off, int g) {
        return *reinterpret_cast<const float4*>(base + off + (((2 * g + h) ^ f) << 2));
    };

    floatx16 acc[2][4];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.f;

    float4 ra[2][2], rb[2][4];    // operand ring: group g in entry g % 2
    auto read_group = [&](const float* base, int g, int e) {
#pragma unroll
        for (int a = 0; a < 2; ++a) ra[e][a] = rd(base, a_off + a * 32 * kKD, g);
#pragma unroll
        for (int b = 0; b < 4; ++b) rb[e][b] = rd(base, b_off + b * 32 * kKD, g);
    };
    auto mfma_group = [&](int e) {
#pragma unroll
        for (int c = 0; c < 4; ++c)
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int b = 0; b < 4; ++b)
                    acc[a][b] = mfma(ra[e][a][c], rb[e][b][c], acc[a][b]);
    };

    // chunk `it` on slot S; its loads for chunk it+3 go to slot S+3 (mod 4),
    // whose chunk (it-1) every wave finished reading before the last barrier
    auto step = [&](auto tag, int it) {
        constexpr int S = decltype(tag)::value;
        if (it + 3 < nchunk) dma(std::integral_constant<int, (S + 3) & 3>{}, it + 3);
        const float* cur = slot_of(tag);
        const float* nxt = slot_of(std::integral_constant<int, (S + 1) & 3>{});
        read_group(cur, 1, 1);
        mfma_group(0);
        read_group(nxt, 0, 0);        // next chunk's first group (stale after the last)
        mfma_group(1);
        __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 32, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 32, 0);
        // chunk it+2 (loaded one step ago) is complete and published
        if (it + 3 < nchunk) wg_barrier<kKLoads>();
        else wg_barrier<0>();
    };

    dma(std::integral_constant<int, 0>{}, 0);
    if (nchunk > 1) dma(std::integral_constant<int, 1>{}, 1);
    if (nchunk > 2) {
        dma(std::integral_constant<int, 2>{}, 2);
        wg_barrier<kKLoads>();
    } else {
        wg_barrier<0>();
    }
    read_group(xs0, 0, 0);
    for (int it0 = 0; it0 < nchunk; it0 += 4) {
        step(std::integral_constant<int, 0>{}, it0);
        if (it0 + 1 < nchunk) step(std::integral_constant<int, 1>{}, it0 + 1);
        if (it0 + 2 < nchunk) step(std::integral_constant<int, 2>{}, it0 + 2);
        if (it0 + 3 < nchunk) step(std::integral_constant<int, 3>{}, it0 + 3);
    }

    // epilogue: kernel values, written row-major (32 consecutive centres per
    // half-wave and accumulator element)
#pragma unroll
    for (int b = 0; b < 4; ++b) {
        const int jl = wn * 128 + b * 32 + (lane & 31);
        const float cnj = s_cn[jl];
        const int64_t cidj = s_cid[jl];
        const bool col_ok = jl < c_rows;
#pragma unroll
        for (int a = 0; a < 2; ++a) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int il = wm * 64 + a * 32 + acc_row(v, lane);
                float kv = kernel_value<KIND>(s_qn[il] + cnj - 2.f * acc[a][b][v], p.scale);
                if (s_qid[il] == cidj) kv = 1.f;
                if (col_ok && il < q_rows) p.out[(q0 + il) * p.ldo + c0 + jl] = kv;
            }
        }
    }
}

}  // namespace

hipError_t kblock_launch(const KblockArgs& a, hipStream_t s) {
    if (a.nq <= 0 || a.nc <= 0) return hipSuccess;
    const int64_t tiles = ceil_div(a.nq, kKM) * ceil_div(a.nc, kKN);
    if (a.kind == 0)
        hipLaunchKernelGGL(kblock_kernel<0>, dim3((unsigned)tiles), dim3(kKThreads), 0, s, a);
    else
        hipLaunchKernelGGL(kblock_kernel<1>, dim3((unsigned)tiles), dim3(kKThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace ep
