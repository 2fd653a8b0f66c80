// Device-side helpers shared by the MFMA kernels (kmv.hip, kblock.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ep {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void;

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

// Buffer descriptor over [base, base + bytes): loads at offsets outside it
// return zero, which provides the zero padding of ragged tiles in hardware.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const float* base, int64_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(base), (short)0, (int)bytes,
                                             0x00020000);
}
// A per-lane offset that no descriptor reaches (the host keeps every
// descriptor's extent below it: query tiles by the limit on d, centre
// ranges by the split planner): the load returns zero. Offsets are
// split into a per-lane part (voffset) and a wave-uniform part (soffset,
// held in a scalar register); a lane's voffset alone already decides
// whether it is in range.
constexpr int kOOB = 0x40000000;

template <int KIND>
__device__ __forceinline__ float kernel_value(float d2, float scale) {
    d2 = fmaxf(d2, 0.f);
    if (KIND == 0) return __builtin_amdgcn_exp2f(scale * d2);
    return __builtin_amdgcn_exp2f(scale * __builtin_amdgcn_sqrtf(d2));
}

// Position of quad q (four features) of staged row r inside its unpadded
// LDS row: q ^ swz32(r) for 32-float rows, q ^ swz16(r) for 16-float rows.
// Direct-to-LDS loads write 64 lanes x 16 bytes contiguously, so rows
// cannot be padded; permuting the quads instead puts the 8 (or 16) lanes
// that one b128 read serves together (consecutive rows, same quad) on
// distinct banks, for 32 or 64 four-byte banks alike.
__device__ __forceinline__ int swz32(int r) { return (r & 7) ^ ((r >> 3) & 1); }
__device__ __forceinline__ int swz16(int r) { return ((r >> 1) ^ (r >> 3)) & 3; }

// Workgroup barrier after this wave's LDS writes (lgkmcnt) and, with
// VM >= 0, after all but its VM most recent vector-memory operations
// (direct-to-LDS loads count there). The asm also keeps the compiler from
// moving memory operations across the barrier.
template <int VM>
__device__ __forceinline__ void wg_barrier() {
    if constexpr (VM == 0) {
        asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
    } else if constexpr (VM == 3) {
        asm volatile("s_waitcnt vmcnt(3) lgkmcnt(0)\n\ts_barrier" ::: "memory");
    } else if constexpr (VM == 4) {
        asm volatile("s_waitcnt vmcnt(4) lgkmcnt(0)\n\ts_barrier" ::: "memory");
    } else {
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    }
}

}  // namespace ep
