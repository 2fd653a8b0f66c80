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
// range of centres (a "split"), walked 256 centres at a time:
//   1. S = C_tile . Q_tile^T on fp32 MFMA (v_mfma_f32_16x16x4f32): each wave
//      owns 32 centres x 64 queries (2 x 4 blocks of 16 x 16 with independent
//      accumulators) of the 256 x 64 block. Its centre rows, which no other
//      wave reads, go from global memory straight into the MFMA operand
//      registers 64 features ahead; the query rows, which all waves read,
//      pass through LDS in batches of 128 (or 64) features (double
//      buffered, one barrier per batch). Rows that are not 16-byte aligned
//      take a register-staged path with 128-centre tiles and LDS for both
//      sides.
//   2. Epilogue in registers: d2 = |q|^2 + |c|^2 - 2 S, clamped at 0; then
//      exp2(scale * d2) (Gaussian) or exp2(scale * sqrt(d2)) (Laplacian).
//      Where the query and the centre are the same training point the value
//      is set to 1 exactly (the fp32 expansion would leave it slightly below).
//   3. The kernel values go to LDS in the MFMA accumulator order, which is
//      exactly the operand order the second product needs, and
//      out^T(labels x queries) += W^T(labels x centres) . K(centres x queries)
//      runs on the same MFMA with W read straight from global memory (a few
//      k-steps ahead). The label tiles are spread over the 8 waves so that
//      the accumulators of up to 1024 labels fit in 128 registers per lane.
//      Up to 160 labels the vector body contracts on tiles of 16 labels
//      instead (v_mfma_f32_16x16x4f32, no label padding beyond 15), with
//      the kernel values in LDS as [centre][query].
//   4. Optionally (kpos, step 2 of the vector body) the kernel values of the
//      centres that are subsample points are also stored, column by column,
//      so that steps 4-5 need no second pass over those m x s entries (the
//      paper reads them from its stored block).
// Partial sums of each split (and centre group, see wl/wj) are written to
// their own slice and summed by a separate deterministic reduction.
#include "ep_device.h"
#include "ep_internal.h"

#include <algorithm>
#include <type_traits>


namespace ep {

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kMaxLtw = 4;           // label tiles per wave (accumulator budget)
constexpr int kMaxLt16 = 10;         // 16-label tiles of the 16-wide contraction

// Register-staged body: 64 queries x 128 centres per iteration.
constexpr int kSCSub = 4;
constexpr int kSBN = kTile * kSCSub;
constexpr int kSRows = kBM + kSBN;   // staged rows per chunk: queries, then centres

static_assert(kBM == 64 && kThreads == 512, "staging maps assume 64 query rows, 512 threads");
static_assert(kBN == 2 * kSBN, "split granularity serves both bodies");

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

// LTW consecutive weights (one per virtual label tile). Three come from one
// 16-byte load whose fourth float (the next lane's first, or zero past the
// descriptor) is dropped: one load instead of three.
template <int LTW>
__device__ __forceinline__ void load_w(__amdgpu_buffer_rsrc_t r, int voff, int soff, float* dst) {
    if constexpr (LTW >= 3) {
        const float4 v = __builtin_bit_cast(
            float4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
        dst[0] = v.x;
        dst[1] = v.y;
        dst[2] = v.z;
        if constexpr (LTW == 4) dst[3] = v.w;
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
    static constexpr int kPasses = kSRows / kRowsPerPass;
    float4 v[kPasses];
};

template <int KIND, int LTW, bool VEC, int PF, int DC, bool ACC2>
__device__ __forceinline__ void kmv_body_staged(const KmvArgs& p) {
    constexpr int kLds = DC + 4;     // padded LDS row (floats): conflict-free b128 reads
    using St = Stage<DC>;
    __shared__ __attribute__((aligned(16))) float xs[2][kSRows][kLds];
    __shared__ float kb[kSCSub][kQSub][16][64];
    __shared__ float s_qn[kBM];
    __shared__ int64_t s_qid[kBM];
    __shared__ float s_cn[2][kSBN];
    __shared__ int64_t s_cid[2][kSBN];

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
    const int64_t ntile = ce > cb ? (ce - cb + kSBN - 1) / kSBN : 0;
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
        if (tid < kSBN) {
            const int64_t c = cb + tile * kSBN + tid;
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
        const int64_t c0 = cb + pf_tile * kSBN;
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
            const int64_t c0 = cb + tile * kSBN;
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
                    make_rsrc(p.W + c0 * p.ldw, (int64_t)kSBN * p.ldw * 4 + kWeightTail);
                float acur[LTW], anxt[LTW];
                load_w<LTW>(wrs, w_voff, w_soff(gj, 0), acur);
                for (int jt = gj; jt < kSCSub; jt += p.wj) {
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        if (v < 15)
                            load_w<LTW>(wrs, w_voff, w_soff(jt, v + 1), anxt);
                        else if (jt + p.wj < kSCSub)
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

// The same computation for rows that are 16-byte aligned (d % 4 == 0), with
// 64 x 256 tiles. Each wave's 32 centre rows are read by that wave alone, so
// they go from global memory straight into the MFMA A-operand registers (two
// 16-byte loads per lane and chunk of 16 features), issued four chunks
// ahead. The distance product runs on the 16x16x4 MFMA, whose A operand
// gives four lanes to a row: one load then covers 16 rows x 64 contiguous
// bytes (the 32x32x2 layout, two lanes per row, covers 32 rows x 32 bytes
// and measured 1.8 % slower). Only the 64 query rows, which all eight waves
// read, pass through LDS: each 64-feature part of a batch is loaded into
// registers at the start of the previous part and written to one of two
// LDS buffers at its end, so there is one workgroup barrier per batch (8 or
// 4 chunks) instead of one per chunk. (Copying both sides straight into
// shared LDS slots instead, with a barrier per chunk, reached 77 % of the
// fp32 MFMA peak at 1000 labels against 89 % for this form: the LDS slots
// cap the loads in flight, and the barriers stall both waves of a SIMD at
// once.)
constexpr int kRDC = 16;                 // features per chunk
constexpr int kRP = 4;                   // chunks in flight in the centre ring

// Chunks per batch (one barrier per batch): 8 when the feature count fills
// them, else 4 (a last batch of 8 chunks half empty costs more than the
// barriers it saves; at d = 440, 28 chunks, 2 %).
inline int batch_chunks(int64_t d) {
    const int64_t nchunk = (d + kRDC - 1) / kRDC;
    return nchunk % 8 == 0 || nchunk % 8 > 4 ? 8 : 4;
}

// LT16 = 0: contraction on 32-label tiles (32x32x2 MFMA), LTW tiles per
// wave, waves in wl label groups x wj centre groups. LT16 > 0: contraction
// on LT16 tiles of 16 labels (16x16x4 MFMA), waves in 2 query halves x 4
// centre quarters (see below); LTW is unused.
template <int KIND, int LTW, int KRB, int LT16>
__device__ __forceinline__ void kmv_body_vec(const KmvArgs& p) {
    constexpr bool k16 = LT16 > 0;
    constexpr int kRB = KRB;                 // chunks per batch
    constexpr int kRF = kRDC * kRB;          // features per batch
    constexpr int kQPR = kRF / 4;            // query quads per row and batch
    constexpr int kRowStep = kThreads / kQPR;    // rows between a thread's quads
    static_assert(kRB % kRP == 0, "the batch is staged in kRP-chunk parts");
    static_assert(kBM * kQPR == 2 * kThreads * (kRB / kRP), "two quads per thread and part");
    __shared__ __attribute__((aligned(16))) float qs[2][kBM * kRF];
    // kernel values of the tile: for the 32-wide contraction in MFMA
    // accumulator order, kb[centre sub-tile][query half][k row][lane]; for
    // the 16-wide one kb16[centre][query ^ kswz(centre)]
    __shared__ float kb[kCSub][kQSub][16][64];
    float (*kb16)[kBM] = reinterpret_cast<float (*)[kBM]>(&kb[0][0][0][0]);
    __shared__ float s_qn[kBM];
    __shared__ int64_t s_qid[kBM];
    __shared__ float s_cn[2][kBN];
    __shared__ int64_t s_cid[2][kBN];     // only with explicit centre ids
    __shared__ int s_qdiag[2][kBM];       // idem: tile position of the query's own centre
    __shared__ int s_cpos[2][kBN];        // only with kpos: subsample position or -1

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    // wave index made visibly uniform: everything derived from it (label
    // block, centre rows, weight offsets) then lives in scalar registers,
    // and buffer loads need no per-lane offset loops
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int tq = (int)((p.nq + kBM - 1) / kBM);
    const int split = (int)blockIdx.x / tq;
    const int qtile = (int)blockIdx.x - split * tq;
    const int64_t q0 = (int64_t)qtile * kBM;
    const int64_t cb = (int64_t)split * p.cps;
    const int64_t ce = min(p.nc, cb + p.cps);
    const int64_t ntile = ce > cb ? (ce - cb + kBN - 1) / kBN : 0;
    const int nchunk = (int)((p.d + kRDC - 1) / kRDC);
    const int nbt = (nchunk + kRB - 1) / kRB;            // batches per tile
    const int64_t nbatch = ntile * nbt;
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
            if (p.cid) s_cid[tile & 1][tid] = ok ? p.cid[c] : -2;
            if (p.kpos) s_cpos[tile & 1][tid] = ok ? p.kpos[c] : -1;
        }
    };
    // With explicit centre ids (the subsample pass: centres are batch rows)
    // the first wave finds, for each query, the tile position of the centre
    // that is the same training point (ids are unique on both sides), after
    // a barrier that publishes the tile's ids.
    auto find_diag = [&](int64_t tile) {
        if (tid < kBM) {
            const int64_t id = s_qid[tid];
            const int64_t* ids = s_cid[tile & 1];
            int at = -1;
#pragma unroll 8
            for (int j = 0; j < kBN; ++j) at = ids[j] == id ? j : at;
            s_qdiag[tile & 1][tid] = at;
        }
    };

    const int ct_s = wave;              // centre sub-tile of this wave (distances)
    const int gl = wave % p.wl;         // contraction role of this wave
    const int gj = wave / p.wl;
    const int lb = gl * LTW * kTile;
    const int lvalid = p.lt * kTile;
    const bool active = k16 || (wave < p.wl * p.wj && lb < lvalid);
    // 16-wide contraction: query half qh (queries 32 qh .. +31, two blocks
    // of 16), centre quarter cq (centres 64 cq .. +63 of the tile)
    const int qh = wave & 1, cq = wave >> 1;

    constexpr int kAcc32 = k16 ? 1 : LTW;
    constexpr int kAcc16 = k16 ? LT16 : 1;
    floatx16 facc[kAcc32][kQSub];
    floatx4 acc16[2][kAcc16];
    if constexpr (!k16) {
#pragma unroll
        for (int i = 0; i < LTW; ++i)
#pragma unroll
            for (int b = 0; b < kQSub; ++b)
#pragma unroll
                for (int v = 0; v < 16; ++v) facc[i][b][v] = 0.f;
    } else {
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int a = 0; a < LT16; ++a)
#pragma unroll
                for (int i = 0; i < 4; ++i) acc16[h][a][i] = 0.f;
    }
    // position of query q of centre c in kb16: the XOR keeps both the
    // epilogue's writes (centres 4 apart in one half-wave) and the
    // contraction's reads (adjacent centres) on distinct banks
    auto kswz = [](int c) { return 16 * (((c >> 2) ^ c) & 1); };
    // distances: 2 centre blocks x 4 query blocks of 16 x 16 (16x16x4 MFMA)
    floatx4 sacc[2][4];
#pragma unroll
    for (int cb = 0; cb < 2; ++cb)
#pragma unroll
        for (int qb = 0; qb < 4; ++qb)
#pragma unroll
            for (int i = 0; i < 4; ++i) sacc[cb][qb][i] = 0.f;
    const int q4 = lane >> 4;           // k slot of this lane in a 16x16x4 step

    // Query staging: thread t moves quads t and t + 512 of the batch, i.e.
    // row Q/16, features 4(Q%16) .. +3 of the batch's 64, to LDS position
    // (Q%16) ^ (row%16) of its row (rows of 64 floats; the permutation puts
    // the 16 rows that one b128 read serves on distinct banks).
    const int64_t q_rows = min((int64_t)kBM, p.nq - q0);
    const __amdgpu_buffer_rsrc_t qrs =
        make_rsrc(p.Q + q0 * p.ldq, ((q_rows - 1) * p.ldq + p.d) * 4);
    // quads tid + 512 j: rows tid/kQPR + j kRowStep, the same quad of each
    const int qst_row = tid / kQPR, qst_qq = tid % kQPR;
    const int qst_col = 4 * qst_qq;
    const int qst_voff = qst_row * (int)p.ldq * 4 + 16 * qst_qq;
    const int qst_lds = qst_row * kRF + ((qst_qq ^ (qst_row & 15)) << 2);
    const int qst_step = kRowStep * (int)p.ldq * 4;   // kRowStep rows further
    // Every load is issued on every path (out-of-range ones at kOOB, which
    // read zeros without touching memory), so that the number of loads in
    // flight is the same on all paths and the compiler's wait counts stay
    // exact instead of draining the queue. The whole row offset goes in
    // voffset: the descriptor's range check sees voffset only, so a row
    // past the tile's last one (a ragged last query tile) reads zero
    // instead of memory beyond the caller's rows.
    float4 qstage[2];
    auto qload = [&](int part, int bi, bool valid) {
        const int f0 = bi * kRF;
        const bool ok = valid && f0 + qst_col < d;
#pragma unroll
        for (int i = 0; i < 2; ++i)
            qstage[i] = __builtin_bit_cast(
                float4, __builtin_amdgcn_raw_buffer_load_b128(
                            qrs, ok ? qst_voff + (2 * part + i) * qst_step : kOOB, f0 * 4, 0));
    };
    auto qwrite = [&](int part, int buf) {
#pragma unroll
        for (int i = 0; i < 2; ++i)
            *reinterpret_cast<float4*>(&qs[buf][qst_lds + (2 * part + i) * kRowStep * kRF]) =
                qstage[i];
    };

    // Centre operands: lane (row = lane%16, k slot q4 = lane/16) of wave w
    // feeds, for centre block cb, features 4q4 .. 4q4+3 of the chunk of
    // centre 32w + 16cb + lane%16 (one 16-byte load); step i of the 16x16x4
    // MFMA pairs feature 4q4 + i of both sides, so every feature is
    // contracted exactly once.
    const int c_voff = ((ct_s * 32 + (lane & 15)) * (int)p.ldc + 4 * q4) * 4;
    const int c_blk = 16 * (int)p.ldc * 4;   // second centre block, 16 rows on
    float4 cring[kRP][2];
#pragma unroll
    for (int c = 0; c < kRP; ++c)
        cring[c][0] = cring[c][1] = make_float4(0.f, 0.f, 0.f, 0.f);
    auto centre_rsrc = [&](int64_t t) {
        const int64_t c0 = cb + t * kBN;
        return make_rsrc(p.C + c0 * p.ldc, ((ce - c0 - 1) * p.ldc + p.d) * 4);
    };
    // (row offsets in voffset, as for the queries: rows past the split's
    // end, in its ragged last tile, read zero)
    auto cload = [&](__amdgpu_buffer_rsrc_t crs, int ch, bool valid, float4* dst) {
        const int f0 = ch * kRDC;
        const bool ok = valid && f0 + 4 * q4 < d;
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
            dst[cb] = __builtin_bit_cast(
                float4, __builtin_amdgcn_raw_buffer_load_b128(crs, ok ? c_voff + cb * c_blk : kOOB,
                                                              f0 * 4, 0));
    };

    // B operand (queries) from LDS: quad 4c + q4 of row 16qb + lane%16
    const int q_base = (lane & 15) * kRF;
    const int q_swz = q4 ^ (lane & 15);
    auto rdq = [&](int buf, int c, int qb) {
        const int pos = ((4 * c) ^ q_swz) << 2;
        return *reinterpret_cast<const float4*>(&qs[buf][q_base + qb * 16 * kRF + pos]);
    };
    float4 bring[2][2];       // half e of a chunk: query blocks 2e, 2e+1
    auto mfma_half = [&](const float4* a, int e) {
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
            for (int cb = 0; cb < 2; ++cb)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    sacc[cb][2 * e + j] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                        a[cb][k], bring[e][j][k], sacc[cb][2 * e + j], 0, 0, 0);
    };

    const int w_col = lb + LTW * (lane & 31);
    const int ldw4 = (int)p.ldw * 4;
    const int w_voff = k16 ? ((lane >> 4) * (int)p.ldw + LT16 * (lane & 15)) * 4
                     : (w_col < lvalid ? ((lane >> 5) << 2) * ldw4 + w_col * 4 : kOOB);
    auto w_soff = [&](int jt, int v) { return (jt * 32 + ((v >> 2) << 3) + (v & 3)) * ldw4; };
    constexpr int PD = k16 ? 2 : (LTW <= 2 ? 16 : 2);
    constexpr int kWb = k16 ? LT16 : LTW;
    float wbuf[PD][kWb];
    // 16-wide contraction, k-step st (centres 64 cq + 4 st .. +3): lane l
    // feeds k slot l/16 (that centre's row) and, for label tile a, row
    // l%16 of the tile, i.e. label LT16 (l%16) + a: LT16 contiguous floats
    // of one weight row (16 LT16 <= ldw, so they stay in the row)
    auto load_w16 = [&](__amdgpu_buffer_rsrc_t r, int st, float* dst) {
        const int so = (64 * cq + 4 * st) * ldw4;
#pragma unroll
        for (int a = 0; a + 4 <= kWb; a += 4) {
            const float4 v = __builtin_bit_cast(
                float4, __builtin_amdgcn_raw_buffer_load_b128(r, w_voff + 4 * a, so, 0));
            dst[a] = v.x;
            dst[a + 1] = v.y;
            dst[a + 2] = v.z;
            dst[a + 3] = v.w;
        }
#pragma unroll
        for (int a = kWb & ~3; a < kWb; ++a) dst[a] = ld1(r, w_voff + 4 * a, so);
    };
    // The weight rows of a k-step sit in soffset, which the range check does
    // not see; the descriptor spans the whole padded tile (kBN rows and the
    // 16-byte tail every weight matrix carries), which the caller's weights
    // fill with zeros past their last row, so every load stays inside it.
    auto w_rsrc = [&](int64_t t) {
        const int64_t c0 = cb + t * kBN;
        return make_rsrc(p.W + c0 * p.ldw, (int64_t)kBN * p.ldw * 4 + kWeightTail);
    };
    // After the last batch of a tile: kernel values (in accumulator order,
    // which is the operand order of the second product), then
    // out^T[label, q] += W[c, label] * K[c, q] on the same MFMA.
    auto finish_tile = [&](int64_t tile) {
        const int64_t c0 = cb + tile * kBN;
        // the first weight fragments travel while the kernel values are
        // formed and published (not with four label tiles per wave, whose
        // registers are full)
        const __amdgpu_buffer_rsrc_t wrs = w_rsrc(tile);
        auto first_weights = [&]() {
#pragma unroll
            for (int v = 0; v < PD; ++v) {
                if constexpr (k16) load_w16(wrs, v, wbuf[v]);
                else load_w<LTW>(wrs, w_voff, w_soff(gj, v), wbuf[v]);
            }
        };
        if (LTW < 4 && active) first_weights();
        const float* cn = s_cn[tile & 1];
        // element i of block (cb, qb) is centre cbase + 16cb + i, query
        // 16qb + lane%16; it goes where the 32x32 contraction reads it
        const int cbase = ct_s * 32 + 4 * q4;
#pragma unroll
        for (int qb = 0; qb < 4; ++qb) {
            const int bl = qb * 16 + (lane & 15);
            const float qnb = s_qn[bl];
            int dq;
            if (p.cid) {
                dq = s_qdiag[tile & 1][bl] - cbase;
            } else {
                const int64_t rel = s_qid[bl] - c0 - cbase;
                dq = rel >= 0 && rel < 32 ? (int)rel : -1;
            }
            const int lk = 16 * (qb & 1) + (lane & 15) + 32 * (q4 & 1);
#pragma unroll
            for (int cb = 0; cb < 2; ++cb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    float kv = kernel_value<KIND>(qnb + cn[cbase + 16 * cb + i] - 2.f * sacc[cb][qb][i],
                                                  p.scale);
                    if (dq == 16 * cb + i) kv = 1.f;
                    if constexpr (k16) {
                        const int cc = cbase + 16 * cb + i;
                        kb16[cc][bl ^ kswz(cc)] = kv;
                    } else {
                        kb[ct_s][qb >> 1][8 * cb + 4 * (q4 >> 1) + i][lk] = kv;
                    }
                }
        }
        // Subsample centres (kpos >= 0): their kernel values also go to row
        // kpos of ksb, for the subsample correction. Each wave copies its
        // own 32 centres back from its block of kb, one 64-query column per
        // flagged centre (centre r of the block, query q sits at
        // kb[.][q / 32][4 (r / 8) + r % 4][q % 32 + 32 ((r / 4) % 2)]).
        if (p.kpos) {
            const int* cp = s_cpos[tile & 1] + ct_s * 32;
            uint64_t flagged = __ballot(lane < 32 && cp[lane & 31] >= 0);
            if (flagged) {
                const __amdgpu_buffer_rsrc_t ks = make_rsrc(p.ksb, (int64_t)p.s_rows * p.ldk * 4);
                const float* kcol = &kb[ct_s][lane >> 5][0][lane & 31];
                do {
                    const int r = __builtin_ctzll(flagged);
                    flagged &= flagged - 1;
                    const int pos = __builtin_amdgcn_readfirstlane(cp[r]);
                    const int cr = ct_s * 32 + r;
                    const float v =
                        k16 ? kb16[cr][lane ^ kswz(cr)]
                            : kcol[(4 * (r >> 3) + (r & 3)) * 64 + 32 * ((r >> 2) & 1)];
                    // (the store takes its data as 32 raw bits)
                    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), ks,
                                                          lane * 4, (int)((pos * p.ldk + q0) * 4), 0);
                } while (flagged);
            }
        }
        if (tile + 1 < ntile) load_centre_meta(tile + 1);
        wg_barrier<-1>();
        if (p.cid && tile + 1 < ntile) find_diag(tile + 1);
        if constexpr (k16) {
            // out^T(labels x queries) += W^T K over this wave's 64 centres,
            // four per 16x16x4 step, for its two query blocks; the kernel
            // values are read two k-steps ahead
            float kvr[2][2];
#pragma unroll
            for (int u = 0; u < 2; ++u)
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int cc = 64 * cq + 4 * u + q4;
                    kvr[u][h] = kb16[cc][(32 * qh + 16 * h + (lane & 15)) ^ kswz(cc)];
                }
#pragma unroll
            for (int st = 0; st < 16; ++st) {
                float wc[kWb];
#pragma unroll
                for (int a = 0; a < kWb; ++a) wc[a] = wbuf[st % PD][a];
                if (st + PD < 16) load_w16(wrs, st + PD, wbuf[st % PD]);
                const float kv0 = kvr[st & 1][0], kv1 = kvr[st & 1][1];
                if (st + 2 < 16) {
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        const int cc = 64 * cq + 4 * (st + 2) + q4;
                        kvr[st & 1][h] = kb16[cc][(32 * qh + 16 * h + (lane & 15)) ^ kswz(cc)];
                    }
                }
#pragma unroll
                for (int a = 0; a < kWb; ++a) {
                    acc16[0][a] = __builtin_amdgcn_mfma_f32_16x16x4f32(wc[a], kv0, acc16[0][a], 0, 0, 0);
                    acc16[1][a] = __builtin_amdgcn_mfma_f32_16x16x4f32(wc[a], kv1, acc16[1][a], 0, 0, 0);
                }
            }
        } else if (active) {
            if (LTW == 4) first_weights();
            for (int jt = gj; jt < kCSub; jt += p.wj) {
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    float acur[LTW];
#pragma unroll
                    for (int i = 0; i < LTW; ++i) acur[i] = wbuf[v % PD][i];
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
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
#pragma unroll
            for (int qb = 0; qb < 4; ++qb)
#pragma unroll
                for (int i = 0; i < 4; ++i) sacc[cb][qb][i] = 0.f;
    };

    if (ntile > 0) {
        load_centre_meta(0);
        if (p.cid) {
            __syncthreads();
            find_diag(0);
        }
        // batch 0: queries to LDS buffer 0, its first chunks to the ring
#pragma unroll
        for (int part = 0; part < kRB / kRP; ++part) {
            qload(part, 0, true);
            qwrite(part, 0);
        }
        const __amdgpu_buffer_rsrc_t crs0 = centre_rsrc(0);
#pragma unroll
        for (int c = 0; c < kRP; ++c) cload(crs0, c, c < nchunk, cring[c]);
    }
    wg_barrier<-1>();

    // the batch after the current one, whose operands are fetched meanwhile
    int64_t nx_tile = 0;
    int nx_bi = 0;
    auto advance = [&]() {
        if (++nx_bi == nbt) {
            nx_bi = 0;
            ++nx_tile;
        }
    };
    advance();
    int64_t k = 0;
    for (int64_t tile = 0; tile < ntile; ++tile) {
        for (int bi = 0; bi < nbt; ++bi, ++k) {
            const bool has_next = k + 1 < nbatch;
            const int buf = (int)(k & 1);
            const __amdgpu_buffer_rsrc_t crs_c = centre_rsrc(tile);
            const __amdgpu_buffer_rsrc_t crs_n = centre_rsrc(has_next ? nx_tile : tile);
#pragma unroll
            for (int j = 0; j < 2; ++j) bring[0][j] = rdq(buf, 0, j);
#pragma unroll
            for (int c = 0; c < kRB; ++c) {
                if (c % kRP == 0) qload(c / kRP, nx_bi, has_next);
                if (c == 0 || bi * kRB + c < nchunk) {
#pragma unroll
                    for (int j = 0; j < 2; ++j) bring[1][j] = rdq(buf, c, 2 + j);
                    mfma_half(cring[c % kRP], 0);
                    // first half of the next chunk of this batch (stale
                    // after the last, unused)
#pragma unroll
                    for (int j = 0; j < 2; ++j) bring[0][j] = rdq(buf, (c + 1) & (kRB - 1), j);
                    mfma_half(cring[c % kRP], 1);
                }
                // refill this ring entry with the chunk kRP positions on
                if (c + kRP < kRB)
                    cload(crs_c, bi * kRB + c + kRP, bi * kRB + c + kRP < nchunk, cring[c % kRP]);
                else
                    cload(crs_n, nx_bi * kRB + c + kRP - kRB,
                          has_next && nx_bi * kRB + c + kRP - kRB < nchunk, cring[c % kRP]);
                if (c % kRP == kRP - 1) qwrite(c / kRP, buf ^ 1);
            }
            wg_barrier<-1>();
            advance();
        }
        finish_tile(tile);
    }

    if constexpr (k16) {
        // element i of tile a, block h: label LT16 (4 (l/16) + i) + a,
        // query 32 qh + 16 h + l%16; slice = (split, centre quarter)
        const int slice = split * 4 + cq;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            float* o = p.out +
                       ((int64_t)slice * p.out_rows + q0 + 32 * qh + 16 * h + (lane & 15)) * p.ldw;
#pragma unroll
            for (int a = 0; a < LT16; ++a)
#pragma unroll
                for (int i = 0; i < 4; ++i) o[LT16 * (4 * q4 + i) + a] = acc16[h][a][i];
        }
    } else if (active) {
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
// KRB: chunks per batch of the vector body (unused by the staged one).
// LT16 > 0 (vector body, predictions pass only): the 16-wide contraction.
template <int KIND, int LTW, bool VEC, int PF, int DC, bool ACC2, int KRB, int LT16 = 0>
__global__ void __launch_bounds__(kThreads) kmv_kernel(KmvArgs p) {
    if constexpr (VEC) kmv_body_vec<KIND, LTW, KRB, LT16>(p);
    else kmv_body_staged<KIND, LTW, VEC, PF, DC, ACC2>(p);
}
template <int KIND, int LTW, bool VEC, int PF, int DC, bool ACC2, int KRB>
__global__ void __launch_bounds__(kThreads) kmv_subsample_kernel(KmvArgs p) {
    if constexpr (VEC) kmv_body_vec<KIND, LTW, KRB, 0>(p);
    else kmv_body_staged<KIND, LTW, VEC, PF, DC, ACC2>(p);
}

typedef void (*KmvFn)(KmvArgs);

template <int KIND, bool VEC, int KRB>
KmvFn pick(int ltw, bool sub) {
    switch (ltw) {
        case 1: return sub ? kmv_subsample_kernel<KIND, 1, VEC, 2, 32, true, KRB> : kmv_kernel<KIND, 1, VEC, 2, 32, true, KRB>;
        case 2: return sub ? kmv_subsample_kernel<KIND, 2, VEC, 2, 64, true, KRB> : kmv_kernel<KIND, 2, VEC, 2, 64, true, KRB>;
        case 3: return sub ? kmv_subsample_kernel<KIND, 3, VEC, 1, 64, false, KRB> : kmv_kernel<KIND, 3, VEC, 1, 64, false, KRB>;
        default: return sub ? kmv_subsample_kernel<KIND, 4, VEC, 1, 32, false, KRB> : kmv_kernel<KIND, 4, VEC, 1, 32, false, KRB>;
    }
}

template <int KIND, int KRB>
KmvFn pick16(int lt16) {
    switch (lt16) {
        case 1: return kmv_kernel<KIND, 1, true, 1, 64, false, KRB, 1>;
        case 2: return kmv_kernel<KIND, 1, true, 1, 64, false, KRB, 2>;
        case 3: return kmv_kernel<KIND, 1, true, 1, 64, false, KRB, 3>;
        case 4: return kmv_kernel<KIND, 1, true, 1, 64, false, KRB, 4>;
        case 5: return kmv_kernel<KIND, 1, true, 1, 64, false, KRB, 5>;
        case 6: return kmv_kernel<KIND, 1, true, 1, 64, false, KRB, 6>;
        case 7: return kmv_kernel<KIND, 1, true, 1, 64, false, KRB, 7>;
        case 8: return kmv_kernel<KIND, 1, true, 1, 64, false, KRB, 8>;
        case 9: return kmv_kernel<KIND, 1, true, 1, 64, false, KRB, 9>;
        default: return kmv_kernel<KIND, 1, true, 1, 64, false, KRB, 10>;
    }
}

// The 16-wide contraction's vector-body kernel for lt16 tiles of 16 labels
KmvFn kernel16_for(int kind, int lt16, int krb) {
    if (kind == 0) return krb == 8 ? pick16<0, 8>(lt16) : pick16<0, 4>(lt16);
    return krb == 8 ? pick16<1, 8>(lt16) : pick16<1, 4>(lt16);
}

// krb: chunks per batch of the vector body (batch_chunks), 4 or 8
KmvFn kernel_for(int kind, int ltw, bool vec, bool sub, int krb) {
    if (!vec) return kind == 0 ? pick<0, false, 4>(ltw, sub) : pick<1, false, 4>(ltw, sub);
    if (kind == 0) return krb == 8 ? pick<0, true, 8>(ltw, sub) : pick<0, true, 4>(ltw, sub);
    return krb == 8 ? pick<1, true, 8>(ltw, sub) : pick<1, true, 4>(ltw, sub);
}

int occupancy_slots(KmvFn fn) {
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
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, fn, kThreads, 0) != hipSuccess ||
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

KmvPlan kmv_plan(int64_t nq, int64_t nc, int64_t ldc, int64_t ldw, int64_t l, int kind,
                 int max_slices) {
    KmvPlan best{};
    const int lt = (int)std::min<int64_t>(ldw / kTile, 32);
    const int64_t nct = ceil_div(std::max<int64_t>(nc, 1), kBN);
    // contraction layout (label groups wl x centre groups wj = 8 waves):
    // fewest MFMA steps on the busiest wave, then fewest slices (with one
    // label tile, 1 x 8 keeps every wave busy; not for short centre ranges,
    // where its eight partial slices per split cost more than it saves)
    const int layouts[4][2] = {{8, 1}, {4, 2}, {2, 4}, {1, 8}};
    int best_cost = 1 << 30;
    for (auto& lw : layouts) {
        const int wl = lw[0], wj = lw[1];
        if (wj == 8 && nct < 64) continue;
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
    // Up to 160 labels (and with the vector body) the contraction runs on
    // ceil(l / 16) tiles of 16 labels instead: no label padding beyond 15,
    // waves as 2 query halves x 4 centre quarters. Layout and tiles per wave
    // for the 32-wide bodies that serve the same launch otherwise (staged
    // body, subsample pass) follow the same 2 x 4 split.
    const int64_t lt16 = ceil_div(std::max<int64_t>(l, 1), 16);
    best.lt16 = 0;
    if (lt16 <= kMaxLt16 && 16 * lt16 <= ldw) {
        best.lt16 = (int)lt16;
        best.wl = 2;
        best.wj = 4;
        best.ltw = (int)ceil_div(lt, 2);
    }
    const int slots = occupancy_slots(best.lt16 ? kernel16_for(kind, best.lt16, 8)
                                                : kernel_for(kind, best.ltw, true, false, 8));
    const int64_t tq = ceil_div(std::max<int64_t>(nq, 1), kBM);
    // splits of the centre axis: minimise the makespan of tq * splits equal
    // workgroups over the resident slots. A split's centre rows must stay
    // below the buffer-descriptor reach kOOB (loads at kOOB must fall
    // outside every descriptor), which may force more splits than
    // max_slices asks for.
    const int64_t max_per = std::max<int64_t>(1, (int64_t)kOOB / (kBN * std::max<int64_t>(ldc, 1) * 4));
    const int64_t min_p = ceil_div(nct, max_per);
    // Each workgroup is charged a fixed cost of `ovh` tiles on top of its
    // tiles. The first pass charges one tile; the second charges what a
    // workgroup's start-up (first operands in flight, partial sums written)
    // costs against one tile's work, 128 / (d + l) tiles, and keeps at least
    // four tiles per workgroup. Its choice is taken only when it is
    // predicted to be more than 2 % faster (for instance 240 workgroups on
    // 256 CUs become 3 full rounds).
    auto choose = [&](double ovh, int64_t min_per, int64_t& bp, int64_t& bper) {
        double bt = 1e300;
        bp = 1;
        bper = nct;
        for (int64_t P = min_p; P <= nct && (P == min_p || P * best.wj <= max_slices); ++P) {
            const int64_t per = ceil_div(nct, P);
            const int64_t peff = ceil_div(nct, per);
            if (peff != P || per > max_per || (P != min_p && per < min_per)) continue;
            const int64_t rounds = ceil_div(tq * peff, slots);
            const double t = (double)rounds * ((double)per + ovh);
            if (t < bt) {
                bt = t;
                bp = peff;
                bper = per;
            }
        }
    };
    auto cost = [&](int64_t P, int64_t per, double ovh) {
        return (double)ceil_div(tq * P, slots) * ((double)per + ovh);
    };
    const double ovh = 128.0 / (double)(std::max<int64_t>(ldc, 1) + ldw);
    int64_t p1, per1, p2, per2;
    choose(1.0, 1, p1, per1);
    choose(ovh, 4, p2, per2);
    const bool second = cost(p2, per2, ovh) < 0.98 * cost(p1, per1, ovh);
    best.splits = (int)(second ? p2 : p1);
    best.cps = (second ? per2 : per1) * kBN;
    return best;
}

hipError_t kmv_launch(KmvArgs a, const KmvPlan& p, hipStream_t s, bool subsample) {
    a.cps = p.cps;
    a.splits = p.splits;
    a.wl = p.wl;
    a.wj = p.wj;
    const bool vec = kmv_vec(a.Q, a.ldq, a.C, a.ldc, a.d);
    if (a.kpos && !vec) return hipErrorInvalidValue;
    const int64_t tq = ceil_div(std::max<int64_t>(a.nq, 1), kBM);
    dim3 grid((unsigned)(tq * p.splits));
    const int lt_total = a.lt;
    for (int t0 = 0; t0 < lt_total; t0 += 32) {
        KmvArgs b = a;
        b.W = a.W + (int64_t)t0 * kTile;
        b.out = a.out + (int64_t)t0 * kTile;
        b.lt = std::min(32, lt_total - t0);
        if (t0 > 0) b.kpos = nullptr;
        const KmvFn fn = p.lt16 > 0 && vec && !subsample && lt_total <= 32
                             ? kernel16_for(a.kind, p.lt16, batch_chunks(a.d))
                             : kernel_for(a.kind, p.ltw, vec, subsample, batch_chunks(a.d));
        hipLaunchKernelGGL(fn, grid,
                           dim3(kThreads), 0, s,
                           b);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace ep
