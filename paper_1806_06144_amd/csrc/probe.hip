// Device probe: the fp32 MFMA rate this GPU sustains and its shader clock
// while doing so. A register-only kernel runs independent chains of
// v_mfma_f32_32x32x2f32 on every SIMD (two waves per SIMD, eight
// accumulators per wave); HIP events time it, and the ratio of the shader
// cycle counter to the constant 100 MHz counter over the same loop gives
// the clock. Used to put the fused kernel's roofline fraction next to what
// the matrix units deliver in practice.
#include "eigenpro.h"
#include "ep_internal.h"

#include <string>

namespace ep {

typedef float floatx16 __attribute__((ext_vector_type(16)));

namespace {

constexpr int kChains = 8;

__global__ void __launch_bounds__(512) mfma_probe_kernel(int iters, float seed, float* sink,
                                                         unsigned long long* clocks) {
    floatx16 acc[kChains];
#pragma unroll
    for (int c = 0; c < kChains; ++c)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[c][v] = 0.f;
    const float a = seed + threadIdx.x * 1e-7f;
    const float b = seed - threadIdx.x * 1e-7f;
    const unsigned long long t0 = __builtin_amdgcn_s_memtime();
    const unsigned long long r0 = __builtin_amdgcn_s_memrealtime();
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int c = 0; c < kChains; ++c)
            acc[c] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc[c], 0, 0, 0);
    }
    const unsigned long long t1 = __builtin_amdgcn_s_memtime();
    const unsigned long long r1 = __builtin_amdgcn_s_memrealtime();
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < kChains; ++c)
#pragma unroll
        for (int v = 0; v < 16; ++v) s += acc[c][v];
    if (s == 12345.f) sink[threadIdx.x] = s;   // keeps the chains live
    if (threadIdx.x == 0 && blockIdx.x == 0) {
        clocks[0] = t1 - t0;
        clocks[1] = r1 - r0;
    }
}

}  // namespace

}  // namespace ep

extern "C" int ep_device_probe(double* mfma_f32_tflops, double* shader_clock_mhz) {
    using namespace ep;
    hipDeviceProp_t prop;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipGetDeviceProperties(&prop, dev) != hipSuccess)
        return EP_EDEVICE;
    const int blocks = prop.multiProcessorCount;   // one 8-wave block per CU
    const int iters = 20000;
    float* sink = nullptr;
    unsigned long long* clk = nullptr;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    int rc = EP_OK;
    if (hipMalloc(&sink, 512 * sizeof(float)) != hipSuccess ||
        hipMalloc(&clk, 2 * sizeof(unsigned long long)) != hipSuccess ||
        hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) {
        rc = EP_ENOMEM;
    } else {
        // warm-up, then the timed launch
        hipLaunchKernelGGL(mfma_probe_kernel, dim3(blocks), dim3(512), 0, nullptr, iters / 10,
                           1.0f, sink, clk);
        (void)hipEventRecord(e0, nullptr);
        hipLaunchKernelGGL(mfma_probe_kernel, dim3(blocks), dim3(512), 0, nullptr, iters, 1.0f,
                           sink, clk);
        (void)hipEventRecord(e1, nullptr);
        unsigned long long hc[2] = {0, 0};
        float ms = 0.f;
        if (hipEventSynchronize(e1) != hipSuccess || hipEventElapsedTime(&ms, e0, e1) != hipSuccess ||
            hipMemcpy(hc, clk, sizeof hc, hipMemcpyDeviceToHost) != hipSuccess) {
            rc = EP_EDEVICE;
        } else {
            const double flops = (double)blocks * 8 /*waves*/ * iters * kChains * 32.0 * 32.0 * 2.0 * 2.0;
            if (mfma_f32_tflops) *mfma_f32_tflops = flops / (ms * 1e-3) / 1e12;
            if (shader_clock_mhz) *shader_clock_mhz = hc[1] ? 100.0 * (double)hc[0] / (double)hc[1] : 0.0;
        }
    }
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
    if (sink) (void)hipFree(sink);
    if (clk) (void)hipFree(clk);
    return rc;
}
