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
// One workgroup = 8 waves (two per SIMD) owns 64 query rows and a contiguous
// range of centres (a "split"), walked 128 centres at a time:
//   1. S = C_tile . Q_tile^T on fp32 MFMA (v_mfma_f32_32x32x2f32): each wave
//      owns one 32x32 sub-tile of the 128 x 64 block. Features stream
//      through two LDS slots in chunks of 32; the global loads of a chunk are
//      issued two chunks ahead (across tile boundaries), so their latency
//      hides behind two chunks of MFMA work.
//   2. Epilogue in registers: d2 = |q|^2 + |c|^2 - 2 S, clamped at 0; then
//      exp2(scale * d2) (Gaussian) or exp2(scale * sqrt(d2)) (Laplacian).
//      Where the query and the centre are the same training point the value
//      is set to 1 exactly (the fp32 expansion would leave it slightly below).
//   3. The kernel values go to LDS in the MFMA accumulator order, which is
//      exactly the operand order the second product needs, and
//      out^T(labels x queries) += W^T(labels x centres) . K(centres x queries)
//      runs on the same MFMA with W read straight from global memory (one
//      step ahead). The label tiles are spread over the 8 waves so that the
//      accumulators of up to 1024 labels fit in 128 registers per lane.
// Partial sums of each split (and centre group, see wl/wj) are written to
// their own slice and summed by a separate deterministic reduction.
#include "ep_device.h"
#include "ep_internal.h"

#include <algorithm>
#include <type_traits>


namespace ep {

namespace {

constexpr int kRows = kBM + kBN;     // staged rows per chunk: queries, then centres
constexpr int kMaxLtw = 4;           // label tiles per wave (accumulator budget)

static_assert(kBM == 64 && kBN == 128 && kThreads == 512, "staging map assumes 64 x 128, 512");

__device__ __forceinline__ float ld1(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
}

// Features col .. col+3 (col = col_lane + col_base) of the row at byte
// offset row_off. VEC: d % 4 == 0 and rows 16-byte aligned, so the four are
// all in or all out.
template <bool VEC>
__device__ __forceinline__ float4 load_feat4(__amdgpu_buffer_rsrc_t r, int row_off, int col_lane,
                                             int col_base, int d) {
    const int col = col_lane + col_base;
    const int soff = col_base * 4;
    if (VEC) {
        const int voff = col < d ? row_off + col_lane * 4 : kOOB;
        return __builtin_bit_cast(float4,
                                  __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
    }
    const int base = row_off + col_lane * 4;
    float4 v;
    v.x = ld1(r, col < d ? base : kOOB, soff);
    v.y = ld1(r, col + 1 < d ? base + 4 : kOOB, soff);
    v.z = ld1(r, col + 2 < d ? base + 8 : kOOB, soff);
    v.w = ld1(r, col + 3 < d ? base + 12 : kOOB, soff);
    return v;
}

// LTW consecutive weights (one per virtual label tile).
template <int LTW>
__device__ __forceinline__ void load_w(__amdgpu_buffer_rsrc_t r, int voff, int soff, float* dst) {
    if (LTW == 4) {
        const float4 v = __builtin_bit_cast(
            float4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
        dst[0] = v.x;
        dst[1] = v.y;
        dst[2] = v.z;
        dst[3] = v.w;
    } else if (LTW == 2) {
        const float2 v =
            __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0));
        dst[0] = v.x;
        dst[1] = v.y;
    } else {
#pragma unroll
        for (int i = 0; i < LTW; ++i) dst[i] = ld1(r, voff == kOOB ? kOOB : voff + 4 * i, soff);
    }
}


// One thread's share of a staged chunk of DC features: NP passes of
// 512 / (DC/4) rows each over the 64 query rows then the 128 centre rows.
template <int DC>
struct Stage {
    static constexpr int kCols = DC / 4;              // float4 per staged row
    static constexpr int kRowsPerPass = kThreads / kCols;
    static constexpr int kPasses = kRows / kRowsPerPass;
    float4 v[kPasses];
};

template <int KIND, int LTW, bool VEC, int PF, int DC, bool ACC2>
__device__ __forceinline__ void kmv_body_staged(const KmvArgs& p) {
    constexpr int kLds = DC + 4;     // padded LDS row (floats): conflict-free b128 reads
    using St = Stage<DC>;
    __shared__ __attribute__((aligned(16))) float xs[2][kRows][kLds];
    __shared__ float kb[kCSub][kQSub][16][64];
    __shared__ float s_qn[kBM];
    __shared__ int64_t s_qid[kBM];
    __shared__ float s_cn[2][kBN];
    __shared__ int64_t s_cid[2][kBN];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    // query tiles run fastest: the 8 XCDs take launch slots round robin, so
    // each XCD holds a block of query tiles x centre splits whose X rows,
    // batch rows and weights it shares through its L2
    const int tq = (int)((p.nq + kBM - 1) / kBM);
    const int split = (int)blockIdx.x / tq;
    const int qtile = (int)blockIdx.x - split * tq;
    const int64_t q0 = (int64_t)qtile * kBM;
    const int64_t cb = (int64_t)split * p.cps;
    const int64_t ce = min(p.nc, cb + p.cps);
    const int64_t ntile = ce > cb ? (ce - cb + kBN - 1) / kBN : 0;
    const int nchunk = (int)((p.d + DC - 1) / DC);
    const int64_t total = ntile * nchunk;
    const int d = (int)p.d;

    if (tid < kBM) {
        const int64_t q = q0 + tid;
        const bool ok = q < p.nq;
        s_qn[tid] = ok ? p.qn[q] : 0.f;
        s_qid[tid] = (ok && p.qid) ? p.qid[q] : -1;
    }
    auto load_centre_meta = [&](int64_t tile) {
        if (tid < kBN) {
            const int64_t c = cb + tile * kBN + tid;
            const bool ok = c < ce;
            s_cn[tile & 1][tid] = ok ? p.cn[c] : 0.f;
            s_cid[tile & 1][tid] = ok ? (p.cid ? p.cid[c] : c) : -2;
        }
    };
    if (ntile > 0) load_centre_meta(0);

    const int qt_s = wave & 1;          // distance sub-tile of this wave
    const int ct_s = wave >> 1;
    const int gl = wave % p.wl;         // contraction role of this wave
    const int gj = wave / p.wl;
    // this wave's labels: a contiguous block of 32*LTW; lane m holds labels
    // lb + LTW*m + i of its LTW virtual tiles i
    const int lb = gl * LTW * kTile;
    const int lvalid = p.lt * kTile;
    const bool active = wave < p.wl * p.wj && lb < lvalid;

    floatx16 facc[LTW][kQSub];
#pragma unroll
    for (int i = 0; i < LTW; ++i)
#pragma unroll
        for (int b = 0; b < kQSub; ++b)
#pragma unroll
            for (int v = 0; v < 16; ++v) facc[i][b][v] = 0.f;
    // distance accumulator(s): with ACC2 alternate k-steps go to two
    // independent accumulators, summed in the epilogue
    floatx16 sacc, sacc2;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
        sacc[v] = 0.f;
        sacc2[v] = 0.f;
    }

    const int lr = tid / St::kCols;             // row inside a pass
    const int lc = (tid % St::kCols) * 4;       // feature inside the chunk
    const int64_t q_rows = min((int64_t)kBM, p.nq - q0);
    const __amdgpu_buffer_rsrc_t qrs =
        make_rsrc(p.Q + q0 * p.ldq, ((q_rows - 1) * p.ldq + p.d) * 4);
    // byte offset of this thread's row in each pass (query rows first)
    int row_off[St::kPasses];
#pragma unroll
    for (int ps = 0; ps < St::kPasses; ++ps) {
        const int sr = ps * St::kRowsPerPass;
        row_off[ps] = sr < kBM ? (sr + lr) * (int)p.ldq * 4 : (sr - kBM + lr) * (int)p.ldc * 4;
    }

    int64_t pf_tile = 0;                // next chunk to fetch
    int pf_ch = 0;
    auto fetch = [&](St& s) {
        const int64_t c0 = cb + pf_tile * kBN;
        const __amdgpu_buffer_rsrc_t crs =
            make_rsrc(p.C + c0 * p.ldc, ((ce - c0 - 1) * p.ldc + p.d) * 4);
        const int kbase = pf_ch * DC;
#pragma unroll
        for (int ps = 0; ps < St::kPasses; ++ps)
            s.v[ps] = load_feat4<VEC>(ps * St::kRowsPerPass < kBM ? qrs : crs, row_off[ps], lc,
                                      kbase, d);
        if (++pf_ch == nchunk) {
            pf_ch = 0;
            ++pf_tile;
        }
    };
    auto stash = [&](int slot, const St& s) {
#pragma unroll
        for (int ps = 0; ps < St::kPasses; ++ps)
            *reinterpret_cast<float4*>(&xs[slot][ps * St::kRowsPerPass + lr][lc]) = s.v[ps];
    };

    // This lane's weights for k-step (jt, v) sit in row jt*32 + acc_row(v,
    // lane) of the tile: the lane part (4 * half + column) goes in voffset,
    // the rest (jt*32 + 8*(v/4) + v%4 rows) in soffset.
    const int w_col = lb + LTW * (lane & 31);
    const int ldw4 = (int)p.ldw * 4;
    const int w_voff = w_col < lvalid ? ((lane >> 5) << 2) * ldw4 + w_col * 4 : kOOB;
    auto w_soff = [&](int jt, int v) { return (jt * 32 + ((v >> 2) << 3) + (v & 3)) * ldw4; };

    int64_t tile = 0;
    int ch = 0;
    // S += C_chunk . Q_chunk^T for the chunk staged in `slot`. Lane (row =
    // lane%32, half h = lane/32) reads features 8g+4h .. 8g+4h+3; step i of
    // group g pairs feature 8g+i (lower half) with 8g+4+i (upper half). A
    // and B use the same map, so every feature is contracted exactly once.
    auto chunk_mfma = [&](int slot) {
        const float* arow = &xs[slot][kBM + ct_s * 32 + (lane & 31)][(lane >> 5) << 2];
        const float* brow = &xs[slot][qt_s * 32 + (lane & 31)][(lane >> 5) << 2];
#pragma unroll
        for (int g = 0; g < DC / 8; ++g) {
            const float4 a = *reinterpret_cast<const float4*>(arow + 8 * g);
            const float4 b = *reinterpret_cast<const float4*>(brow + 8 * g);
            if (ACC2) {
                sacc = mfma(a.x, b.x, sacc);
                sacc2 = mfma(a.y, b.y, sacc2);
                sacc = mfma(a.z, b.z, sacc);
                sacc2 = mfma(a.w, b.w, sacc2);
            } else {
                sacc = mfma(a.x, b.x, sacc);
                sacc = mfma(a.y, b.y, sacc);
                sacc = mfma(a.z, b.z, sacc);
                sacc = mfma(a.w, b.w, sacc);
            }
        }
    };
    // After the last chunk of a tile: kernel values, then the contraction.
    auto finish_chunk = [&]() {
        if (ch == nchunk - 1) {
            // epilogue: distances -> kernel values, stored in accumulator order
            const int64_t c0 = cb + tile * kBN;
            const int bl = qt_s * 32 + (lane & 31);
            const float qnb = s_qn[bl];
            const int64_t qidb = s_qid[bl];
            const float* cn = s_cn[tile & 1];
            const int64_t* cid = s_cid[tile & 1];
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int jl = ct_s * 32 + acc_row(v, lane);
                const float dot = ACC2 ? sacc[v] + sacc2[v] : sacc[v];
                float kv = kernel_value<KIND>(qnb + cn[jl] - 2.f * dot, p.scale);
                if (qidb == cid[jl]) kv = 1.f;
                if (c0 + jl >= ce) kv = 0.f;
                kb[ct_s][qt_s][v][lane] = kv;
                sacc[v] = 0.f;
                sacc2[v] = 0.f;
            }
            if (tile + 1 < ntile) load_centre_meta(tile + 1);
            __syncthreads();

            // contraction: out^T[label, q] += W[c, label] * K[c, q], with the
            // W fragments of the next step in flight during this step's MFMAs
            if (active) {
                const __amdgpu_buffer_rsrc_t wrs =
                    make_rsrc(p.W + c0 * p.ldw, (int64_t)kBN * p.ldw * 4);
                float acur[LTW], anxt[LTW];
                load_w<LTW>(wrs, w_voff, w_soff(gj, 0), acur);
                for (int jt = gj; jt < kCSub; jt += p.wj) {
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        if (v < 15)
                            load_w<LTW>(wrs, w_voff, w_soff(jt, v + 1), anxt);
                        else if (jt + p.wj < kCSub)
                            load_w<LTW>(wrs, w_voff, w_soff(jt + p.wj, 0), anxt);
                        const float k0v = kb[jt][0][v][lane];
                        const float k1v = kb[jt][1][v][lane];
#pragma unroll
                        for (int i = 0; i < LTW; ++i) {
                            facc[i][0] = mfma(acur[i], k0v, facc[i][0]);
                            facc[i][1] = mfma(acur[i], k1v, facc[i][1]);
                        }
#pragma unroll
                        for (int i = 0; i < LTW; ++i) acur[i] = anxt[i];
                    }
                }
            }
            ++tile;
            ch = 0;
        } else {
            ++ch;
        }
        // publishes the slot staged in this step and orders this chunk's
        // reads of its slot before the next step overwrites it; also orders
        // the kb reads above before the next epilogue writes kb
        __syncthreads();
    };

    // PF register stages rotate: at step it, stage it % PF (whose chunk was
    // moved to LDS one step earlier) receives the loads of chunk it + PF,
    // and stage (it+1) % PF, loaded PF-1 steps earlier, is moved to LDS for
    // the next step.
    St st[PF];
#pragma unroll
    for (int j = 0; j < PF; ++j)
        if (j < total) fetch(st[j]);
    if (total > 0) stash(0, st[0]);
    __syncthreads();
    for (int64_t it0 = 0; it0 < total; it0 += PF) {
#pragma unroll
        for (int j = 0; j < PF; ++j) {
            const int64_t it = it0 + j;
            if (it < total) {
                const int slot = (int)(it & 1);
                if (it + PF < total) fetch(st[j]);
                chunk_mfma(slot);
                if (it + 1 < total) stash(slot ^ 1, st[(j + 1) % PF]);
                finish_chunk();
            }
        }
    }

    if (active) {
        const int slice = split * p.wj + gj;
        float* o = p.out + ((int64_t)slice * p.out_rows + q0) * p.ldw;
#pragma unroll
        for (int b = 0; b < kQSub; ++b) {
            const int64_t row = b * 32 + (lane & 31);
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int col = lb + LTW * acc_row(v, lane);
#pragma unroll
                for (int i = 0; i < LTW; ++i)
                    if (col + i < lvalid) o[row * p.ldw + col + i] = facc[i][b][v];
            }
        }
    }
}

// The same computation with the feature chunks copied from global memory
// straight into LDS (buffer_load_dwordx4 ... lds: no staging registers) into
// four rotating slots, issued three chunks ahead. Each wave reads its
// operands one group (four MFMAs) ahead, also across the barrier that ends
// a chunk (the next chunk's slot was published one barrier earlier), so its
// MFMAs do not wait for LDS after a barrier. Requires the
// VEC layout (d % 4 == 0, 16-byte aligned rows).
template <int KIND, int LTW, bool ACC2>
__device__ __forceinline__ void kmv_body_dma(const KmvArgs& p) {
    constexpr int DC = 32;                    // features per chunk (4 groups of 8)
    constexpr int kSlot = kRows * DC;         // floats per slot (24 KB)
    static_assert(kRows % 8 == 0 && kRows / 8 == 3 * (kThreads / 64), "3 loads per wave");
    __shared__ __attribute__((aligned(16))) float xs0[kSlot];
    __shared__ __attribute__((aligned(16))) float xs1[kSlot];
    __shared__ __attribute__((aligned(16))) float xs2[kSlot];
    __shared__ __attribute__((aligned(16))) float xs3[kSlot];
    __shared__ float kb[kCSub][kQSub][16][64];
    __shared__ float s_qn[kBM];
    __shared__ int64_t s_qid[kBM];
    __shared__ float s_cn[2][kBN];
    __shared__ int64_t s_cid[2][kBN];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    // wave index made visibly uniform: everything derived from it (label
    // block, centre group, weight offsets) then lives in scalar registers,
    // and buffer loads need no per-lane offset loops. Not for three label
    // tiles per wave, whose three separate weight loads the scheduler then
    // sinks next to their use (measured: a third slower).
    const int wave = LTW == 3 ? tid >> 6 : __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int tq = (int)((p.nq + kBM - 1) / kBM);
    const int split = (int)blockIdx.x / tq;
    const int qtile = (int)blockIdx.x - split * tq;
    const int64_t q0 = (int64_t)qtile * kBM;
    const int64_t cb = (int64_t)split * p.cps;
    const int64_t ce = min(p.nc, cb + p.cps);
    const int64_t ntile = ce > cb ? (ce - cb + kBN - 1) / kBN : 0;
    const int nchunk = (int)((p.d + DC - 1) / DC);
    const int64_t total = ntile * nchunk;
    const int d = (int)p.d;

    if (tid < kBM) {
        const int64_t q = q0 + tid;
        const bool ok = q < p.nq;
        s_qn[tid] = ok ? p.qn[q] : 0.f;
        s_qid[tid] = (ok && p.qid) ? p.qid[q] : -1;
    }
    auto load_centre_meta = [&](int64_t tile) {
        if (tid < kBN) {
            const int64_t c = cb + tile * kBN + tid;
            const bool ok = c < ce;
            s_cn[tile & 1][tid] = ok ? p.cn[c] : 0.f;
            s_cid[tile & 1][tid] = ok ? (p.cid ? p.cid[c] : c) : -2;
        }
    };
    if (ntile > 0) load_centre_meta(0);

    const int qt_s = wave & 1;
    const int ct_s = wave >> 1;
    const int gl = wave % p.wl;
    const int gj = wave / p.wl;
    const int lb = gl * LTW * kTile;
    const int lvalid = p.lt * kTile;
    const bool active = wave < p.wl * p.wj && lb < lvalid;

    floatx16 facc[LTW][kQSub];
#pragma unroll
    for (int i = 0; i < LTW; ++i)
#pragma unroll
        for (int b = 0; b < kQSub; ++b)
#pragma unroll
            for (int v = 0; v < 16; ++v) facc[i][b][v] = 0.f;
    floatx16 sacc, sacc2;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
        sacc[v] = 0.f;
        sacc2[v] = 0.f;
    }

    // Direct-to-LDS staging: load i (0..2) of this wave fills staged rows
    // 8j .. 8j+7, j = 3*wave + i (query rows 0..63, then centre rows), one
    // 16-byte quad per lane: lane L takes row 8j + L/8 and stores at quad
    // position L%8, i.e. it fetches quad (L%8) ^ swz(row) of that row.
    const int64_t q_rows = min((int64_t)kBM, p.nq - q0);
    const __amdgpu_buffer_rsrc_t qrs =
        make_rsrc(p.Q + q0 * p.ldq, ((q_rows - 1) * p.ldq + p.d) * 4);
    int dma_voff[3], dma_col[3];
#pragma unroll
    for (int i = 0; i < 3; ++i) {
        const int j = 3 * wv + i;
        const int r = 8 * j + (lane >> 3);
        const int q = (lane & 7) ^ swz32(r);
        dma_col[i] = 4 * q;
        dma_voff[i] = (r < kBM ? r * (int)p.ldq : (r - kBM) * (int)p.ldc) * 4 + 16 * q;
    }
    int64_t pf_tile = 0;
    int pf_ch = 0;
    auto slot_of = [&](auto tag) -> float* {
        constexpr int S = decltype(tag)::value;
        if constexpr (S == 0) return xs0;
        else if constexpr (S == 1) return xs1;
        else if constexpr (S == 2) return xs2;
        else return xs3;
    };
    auto dma = [&](auto tag) {
        float* base = slot_of(tag);
        const int64_t c0 = cb + pf_tile * kBN;
        const __amdgpu_buffer_rsrc_t crs =
            make_rsrc(p.C + c0 * p.ldc, ((ce - c0 - 1) * p.ldc + p.d) * 4);
        const int kbase = pf_ch * DC;
#pragma unroll
        for (int i = 0; i < 3; ++i) {
            const int j = 3 * wv + i;
            const int voff = kbase + dma_col[i] < d ? dma_voff[i] : kOOB;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(j < kBM / 8 ? qrs : crs,
                                                     (lds_void*)(base + j * 8 * DC), 16, voff,
                                                     kbase * 4, 0, 0);
        }
        if (++pf_ch == nchunk) {
            pf_ch = 0;
            ++pf_tile;
        }
    };

    // Operand reads: lane (row = lane%32, half h = lane/32) feeds features
    // 8g+4h .. 8g+4h+3 of group g, as in the staged body.
    const int h = lane >> 5;
    const int f = (lane & 7) ^ ((lane >> 3) & 1);     // swz of rows at multiples of 16 + lane%32
    const int a_off = (kBM + ct_s * 32 + (lane & 31)) * DC;
    const int b_off = (qt_s * 32 + (lane & 31)) * DC;
    auto rd = [&](const float* base, int off, int g) {
        return *reinterpret_cast<const float4*>(base + off + (((2 * g + h) ^ f) << 2));
    };
    auto mfma4 = [&](float4 a, float4 b) {
        if (ACC2) {
            sacc = mfma(a.x, b.x, sacc);
            sacc2 = mfma(a.y, b.y, sacc2);
            sacc = mfma(a.z, b.z, sacc);
            sacc2 = mfma(a.w, b.w, sacc2);
        } else {
            sacc = mfma(a.x, b.x, sacc);
            sacc = mfma(a.y, b.y, sacc);
            sacc = mfma(a.z, b.z, sacc);
            sacc = mfma(a.w, b.w, sacc);
        }
    };

    const int w_col = lb + LTW * (lane & 31);
    const int ldw4 = (int)p.ldw * 4;
    const int w_voff = w_col < lvalid ? ((lane >> 5) << 2) * ldw4 + w_col * 4 : kOOB;
    auto w_soff = [&](int jt, int v) { return (jt * 32 + ((v >> 2) << 3) + (v & 3)) * ldw4; };

    int64_t tile = 0;
    int ch = 0;
    float4 ra[2], rb[2];      // operand ring: group g in entry g % 2, read one group ahead
    // Contraction weights in flight: PD k-steps ahead. With few labels per
    // wave (LTW <= 2) a k-step is only 2*LTW MFMAs, too short to cover a
    // global load, so all 16 fragments of a centre sub-tile are kept in
    // flight, the first 16 issued during the tile's last chunk; with 3-4
    // label tiles two k-steps ahead (measured: 1 -> 2 gains 1.5 points of
    // peak at l = 1000, 4 no more).
    constexpr int PD = LTW <= 2 ? 16 : 2;
    float wbuf[PD][LTW];
    auto w_rsrc = [&](int64_t t) {
        return make_rsrc(p.W + (cb + t * kBN) * p.ldw, (int64_t)kBN * p.ldw * 4);
    };
    auto finish_tile = [&]() {
        const int64_t c0 = cb + tile * kBN;
        const int bl = qt_s * 32 + (lane & 31);
        const float qnb = s_qn[bl];
        const int64_t qidb = s_qid[bl];
        const float* cn = s_cn[tile & 1];
        const int64_t* cid = s_cid[tile & 1];
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int jl = ct_s * 32 + acc_row(v, lane);
            const float dot = ACC2 ? sacc[v] + sacc2[v] : sacc[v];
            float kv = kernel_value<KIND>(qnb + cn[jl] - 2.f * dot, p.scale);
            if (qidb == cid[jl]) kv = 1.f;
            if (c0 + jl >= ce) kv = 0.f;
            kb[ct_s][qt_s][v][lane] = kv;
            sacc[v] = 0.f;
            sacc2[v] = 0.f;
        }
        if (tile + 1 < ntile) load_centre_meta(tile + 1);
        wg_barrier<-1>();
        if (active) {
            const __amdgpu_buffer_rsrc_t wrs = w_rsrc(tile);
            if constexpr (PD < 16)
#pragma unroll
                for (int v = 0; v < PD; ++v) load_w<LTW>(wrs, w_voff, w_soff(gj, v), wbuf[v]);
            for (int jt = gj; jt < kCSub; jt += p.wj) {
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    float acur[LTW];
#pragma unroll
                    for (int i = 0; i < LTW; ++i) acur[i] = wbuf[v % PD][i];
                    // refill the entry with the fragment PD k-steps ahead
                    const int nv = v + PD < 16 ? v + PD : v + PD - 16;
                    const int njt = v + PD < 16 ? jt : jt + p.wj;
                    if (njt < kCSub) load_w<LTW>(wrs, w_voff, w_soff(njt, nv), wbuf[v % PD]);
                    const float k0v = kb[jt][0][v][lane];
                    const float k1v = kb[jt][1][v][lane];
#pragma unroll
                    for (int i = 0; i < LTW; ++i) {
                        facc[i][0] = mfma(acur[i], k0v, facc[i][0]);
                        facc[i][1] = mfma(acur[i], k1v, facc[i][1]);
                    }
                }
            }
        }
    };

    // One chunk on slot S: its direct loads for chunk it+3 go to slot
    // S+3 (mod 4), whose chunk (it-1) every wave finished reading before the
    // previous barrier.
    auto step = [&](auto tag, int64_t it) {
        constexpr int S = decltype(tag)::value;
        if (it + 3 < total) dma(std::integral_constant<int, (S + 3) & 3>{});
        const float* cur = slot_of(tag);
        const float* nxt = slot_of(std::integral_constant<int, (S + 1) & 3>{});
        if constexpr (PD == 16) {
            if (ch + 1 == nchunk && active) {
                const __amdgpu_buffer_rsrc_t wrs = w_rsrc(tile);
#pragma unroll
                for (int v = 0; v < 16; ++v) load_w<LTW>(wrs, w_voff, w_soff(gj, v), wbuf[v]);
            }
        }
        ra[1] = rd(cur, a_off, 1);
        rb[1] = rd(cur, b_off, 1);
        mfma4(ra[0], rb[0]);
        ra[0] = rd(cur, a_off, 2);
        rb[0] = rd(cur, b_off, 2);
        mfma4(ra[1], rb[1]);
        ra[1] = rd(cur, a_off, 3);
        rb[1] = rd(cur, b_off, 3);
        mfma4(ra[0], rb[0]);
        // first group of chunk it+1, whichever tile it belongs to (after the
        // last chunk this reads a stale slot, unused)
        ra[0] = rd(nxt, a_off, 0);
        rb[0] = rd(nxt, b_off, 0);
        mfma4(ra[1], rb[1]);
        // keep each group's reads ahead of the previous group's MFMAs (the
        // scheduler would otherwise sink them to save eight registers)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);   // 2 LDS reads
            __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);   // 4 MFMAs
        }
        if (++ch == nchunk) {
            finish_tile();
            ++tile;
            ch = 0;
        }
        // chunk it+2 (loaded one step ago) is complete in every wave and
        // published; this chunk's slot is free for the next step's loads
        if (it + 3 < total) wg_barrier<3>();
        else wg_barrier<0>();
    };

    // prologue: chunks 0..2 into slots 0..2; 0 and 1 must be visible
    if (total > 0) dma(std::integral_constant<int, 0>{});
    if (total > 1) dma(std::integral_constant<int, 1>{});
    if (total > 2) {
        dma(std::integral_constant<int, 2>{});
        wg_barrier<3>();
    } else {
        wg_barrier<0>();
    }
    ra[0] = rd(xs0, a_off, 0);
    rb[0] = rd(xs0, b_off, 0);
    for (int64_t it0 = 0; it0 < total; it0 += 4) {
        step(std::integral_constant<int, 0>{}, it0);
        if (it0 + 1 < total) step(std::integral_constant<int, 1>{}, it0 + 1);
        if (it0 + 2 < total) step(std::integral_constant<int, 2>{}, it0 + 2);
        if (it0 + 3 < total) step(std::integral_constant<int, 3>{}, it0 + 3);
    }

    if (active) {
        const int slice = split * p.wj + gj;
        float* o = p.out + ((int64_t)slice * p.out_rows + q0) * p.ldw;
#pragma unroll
        for (int b = 0; b < kQSub; ++b) {
            const int64_t row = b * 32 + (lane & 31);
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int col = lb + LTW * acc_row(v, lane);
#pragma unroll
                for (int i = 0; i < LTW; ++i)
                    if (col + i < lvalid) o[row * p.ldw + col + i] = facc[i][b][v];
            }
        }
    }
}

// Two entry points with one body, so that profiles tell the predictions pass
// (Algorithm 1 step 2, and prediction) from the subsample pass (steps 4-5).
template <int KIND, int LTW, bool VEC, int PF, int DC, bool ACC2>
__global__ void __launch_bounds__(kThreads) kmv_kernel(KmvArgs p) {
    if constexpr (VEC) kmv_body_dma<KIND, LTW, ACC2>(p);
    else kmv_body_staged<KIND, LTW, VEC, PF, DC, ACC2>(p);
}
template <int KIND, int LTW, bool VEC, int PF, int DC, bool ACC2>
__global__ void __launch_bounds__(kThreads) kmv_subsample_kernel(KmvArgs p) {
    if constexpr (VEC) kmv_body_dma<KIND, LTW, ACC2>(p);
    else kmv_body_staged<KIND, LTW, VEC, PF, DC, ACC2>(p);
}

typedef void (*KmvFn)(KmvArgs);

template <int KIND, bool VEC>
KmvFn pick(int ltw, bool sub) {
    switch (ltw) {
        case 1: return sub ? kmv_subsample_kernel<KIND, 1, VEC, 2, 32, true> : kmv_kernel<KIND, 1, VEC, 2, 32, true>;
        case 2: return sub ? kmv_subsample_kernel<KIND, 2, VEC, 2, 64, true> : kmv_kernel<KIND, 2, VEC, 2, 64, true>;
        case 3: return sub ? kmv_subsample_kernel<KIND, 3, VEC, 1, 64, false> : kmv_kernel<KIND, 3, VEC, 1, 64, false>;
        default: return sub ? kmv_subsample_kernel<KIND, 4, VEC, 1, 32, false> : kmv_kernel<KIND, 4, VEC, 1, 32, false>;
    }
}

KmvFn kernel_for(int kind, int ltw, bool vec, bool sub) {
    if (kind == 0) return vec ? pick<0, true>(ltw, sub) : pick<0, false>(ltw, sub);
    return vec ? pick<1, true>(ltw, sub) : pick<1, false>(ltw, sub);
}

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
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, kernel_for(kind, ltw, true, false),
                                                     kThreads, 0) != hipSuccess ||
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

KmvPlan kmv_plan(int64_t nq, int64_t nc, int64_t ldc, int64_t ldw, int kind, int max_slices) {
    KmvPlan best{};
    const int lt = (int)std::min<int64_t>(ldw / kTile, 32);
    // contraction layout (label groups wl x centre groups wj = 8 waves):
    // fewest MFMA steps on the busiest wave, then fewest slices
    const int layouts[3][2] = {{8, 1}, {4, 2}, {2, 4}};
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
    // workgroups over the resident slots. A split's centre rows must stay
    // below the buffer-descriptor reach kOOB (loads at kOOB must fall
    // outside every descriptor), which may force more splits than
    // max_slices asks for.
    const int64_t max_per = std::max<int64_t>(1, (int64_t)kOOB / (kBN * std::max<int64_t>(ldc, 1) * 4));
    const int64_t min_p = ceil_div(nct, max_per);
    int64_t best_p = 1, best_per = nct;
    double best_t = 1e300;
    for (int64_t P = min_p; P <= nct && (P == min_p || P * best.wj <= max_slices); ++P) {
        const int64_t per = ceil_div(nct, P);
        const int64_t peff = ceil_div(nct, per);
        if (peff != P || per > max_per) continue;
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

hipError_t kmv_launch(KmvArgs a, const KmvPlan& p, hipStream_t s, bool subsample) {
    a.cps = p.cps;
    a.splits = p.splits;
    a.wl = p.wl;
    a.wj = p.wj;
    const bool vec = (a.d % 4 == 0) && ((a.ldq & 3) == 0) && ((a.ldc & 3) == 0) &&
                     ((reinterpret_cast<uintptr_t>(a.Q) & 15) == 0) &&
                     ((reinterpret_cast<uintptr_t>(a.C) & 15) == 0);
    const int64_t tq = ceil_div(std::max<int64_t>(a.nq, 1), kBM);
    dim3 grid((unsigned)(tq * p.splits));
    const int lt_total = a.lt;
    for (int t0 = 0; t0 < lt_total; t0 += 32) {
        KmvArgs b = a;
        b.W = a.W + (int64_t)t0 * kTile;
        b.out = a.out + (int64_t)t0 * kTile;
        b.lt = std::min(32, lt_total - t0);
        hipLaunchKernelGGL(kernel_for(a.kind, p.ltw, vec, subsample), grid, dim3(kThreads), 0, s,
                           b);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace ep
