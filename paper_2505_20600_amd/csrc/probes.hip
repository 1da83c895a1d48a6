// Diagnostic probes of the rates that bound the kernels of this library on the
// GPU they run on: the matrix-core issue rate, the shader clock under matrix
// load, LDS read bandwidth, and the per-CU operand stream global -> LDS
// (direct-to-LDS buffer loads) against global -> VGPRs. Each call launches,
// times with HIP events and synchronises; none is part of a denoising step.
// The workloads are synthetic (no data dependence on the values read).
#include <hip/hip_runtime.h>

#include <cstdint>

#include "common.h"
#include "step_internal.h"

namespace ms {
namespace {

constexpr int kProbeCUs = 256;
constexpr int kProbeThreads = 256;

typedef float f32x16_t __attribute__((ext_vector_type(16)));

// Eight independent accumulator chains per wave, so the issue rate (not the
// latency of one chain) bounds the loop. Lane 0 of workgroup 0 records the
// shader clock counter and the 100 MHz constant clock around the loop.
template <int KIND>
__global__ __launch_bounds__(kProbeThreads) void mfma_probe_kernel(int iters, float* out, uint64_t* clocks) {
    const int tid = threadIdx.x;
    bf16x8_t a, b;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        a[i] = (__bf16)(0.001f * (float)((tid + i) & 7));
        b[i] = (__bf16)(0.002f * (float)((tid * 3 + i) & 7));
    }
    uint64_t t0 = 0, r0 = 0;
    if (blockIdx.x == 0 && tid == 0) {
        t0 = __builtin_amdgcn_s_memtime();
        r0 = __builtin_amdgcn_s_memrealtime();
    }
    float s = 0.f;
    if constexpr (KIND == 0) {
        f32x4_t c0 = {}, c1 = {}, c2 = {}, c3 = {}, c4 = {}, c5 = {}, c6 = {}, c7 = {};
        // issued as one instruction block: the register allocator otherwise rotates the
        // four-register accumulators through copies between iterations, which serialises them
        for (int it = 0; it < iters; ++it) {
            asm volatile(
                "v_mfma_f32_16x16x32_bf16 %0, %8, %9, %0\n\t"
                "v_mfma_f32_16x16x32_bf16 %1, %8, %9, %1\n\t"
                "v_mfma_f32_16x16x32_bf16 %2, %8, %9, %2\n\t"
                "v_mfma_f32_16x16x32_bf16 %3, %8, %9, %3\n\t"
                "v_mfma_f32_16x16x32_bf16 %4, %8, %9, %4\n\t"
                "v_mfma_f32_16x16x32_bf16 %5, %8, %9, %5\n\t"
                "v_mfma_f32_16x16x32_bf16 %6, %8, %9, %6\n\t"
                "v_mfma_f32_16x16x32_bf16 %7, %8, %9, %7"
                : "+v"(c0), "+v"(c1), "+v"(c2), "+v"(c3), "+v"(c4), "+v"(c5), "+v"(c6), "+v"(c7)
                : "v"(a), "v"(b));
        }
        const f32x4_t t = (c0 + c1) + (c2 + c3) + (c4 + c5) + (c6 + c7);
        s = t[0] + t[3];
    } else {
        f32x16_t c0 = {}, c1 = {}, c2 = {}, c3 = {}, c4 = {}, c5 = {}, c6 = {}, c7 = {};
        for (int it = 0; it < iters; ++it) {
            c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c0, 0, 0, 0);
            c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c1, 0, 0, 0);
            c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c2, 0, 0, 0);
            c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c3, 0, 0, 0);
            c4 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c4, 0, 0, 0);
            c5 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c5, 0, 0, 0);
            c6 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c6, 0, 0, 0);
            c7 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c7, 0, 0, 0);
        }
        const f32x16_t t = (c0 + c1) + (c2 + c3) + (c4 + c5) + (c6 + c7);
        s = t[0] + t[15];
    }
    if (blockIdx.x == 0 && tid == 0) {
        clocks[0] = __builtin_amdgcn_s_memtime() - t0;
        clocks[1] = __builtin_amdgcn_s_memrealtime() - r0;
    }
    out[(size_t)blockIdx.x * kProbeThreads + tid] = s;
}

// Conflict-free 16-byte LDS reads: consecutive lanes read consecutive 16-byte
// chunks of a 32 KB buffer (five workgroups per CU fit), eight reads per
// iteration 4 KB apart, the window moving by one chunk per iteration.
__global__ __launch_bounds__(kProbeThreads) void lds_probe_kernel(int iters, float* out) {
    __shared__ __attribute__((aligned(16))) uint4 buf[2048];   // 32 KB
    const int tid = threadIdx.x;
    for (int i = tid; i < 2048; i += kProbeThreads) buf[i] = make_uint4(i, i * 3u, i * 5u, i * 7u);
    __syncthreads();
    uint4 acc = make_uint4(0u, 0u, 0u, 0u);
    int base = tid;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const uint4 v = buf[(base + u * 256) & 2047];
            acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
        }
        base = (base + 1) & 2047;
    }
    out[(size_t)blockIdx.x * kProbeThreads + tid] = (float)(acc.x ^ acc.y ^ acc.z ^ acc.w);
}

// Operand stream: every step moves 64 KB per workgroup (512 threads) from a
// window shared by 16 workgroups each (like GEMM operand panels) either by
// direct-to-LDS buffer loads into a two-stage LDS ring (one step in flight)
// or into VGPRs (two register sets).
template <bool DMA>
__global__ __launch_bounds__(512) void stream_probe_kernel(const uint8_t* __restrict__ src, uint32_t win, int steps,
                                                           float* out) {
    __shared__ __attribute__((aligned(1024))) uint8_t smem[2 * 65536];
    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    const uint8_t* base = src + (size_t)(blockIdx.x % 16) * win;
    const u32x4_t rs = raw_rsrc(base, win);
    const uint32_t l0 = lds_addr(smem);
    uint4 acc = make_uint4(0u, 0u, 0u, 0u);
    uint4 r0[8], r1[8];
    for (int it = 0; it < steps; ++it) {
        const uint32_t off = (uint32_t)(((uint64_t)it * 65536u) % win);   // win: a multiple of 64 KB
        if constexpr (DMA) {
            const int st = it & 1;
#pragma unroll
            for (int i = 0; i < 8; ++i)
                dma_buf16(rs, (uint32_t)((i * 8 + wave) * 1024 + lane * 16), off,
                          l0 + (uint32_t)(st * 65536 + (i * 8 + wave) * 1024));
            wait_vmcnt<0>();
            barrier_only();
            const uint4 v = *reinterpret_cast<const uint4*>(smem + st * 65536 + tid * 16);
            acc.x ^= v.x;
        } else {
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const uint4 v = *reinterpret_cast<const uint4*>(base + off + (uint32_t)(i * 512 + tid) * 16u);
                if (it & 1) r1[i] = v;
                else r0[i] = v;
            }
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const uint4 v = (it & 1) ? r0[i] : r1[i];
                acc.x ^= v.x; acc.y ^= v.y; acc.z ^= v.z; acc.w ^= v.w;
            }
        }
    }
    out[(size_t)blockIdx.x * 512 + tid] = (float)(acc.x ^ acc.y ^ acc.z ^ acc.w);
}

struct ProbeTimer {
    hipEvent_t a = nullptr, b = nullptr;
    ~ProbeTimer() {
        if (a) (void)hipEventDestroy(a);
        if (b) (void)hipEventDestroy(b);
    }
};

}  // namespace
}  // namespace ms

using namespace ms;

#define PROBE_HIP(x)                                                                                  \
    do {                                                                                              \
        hipError_t e_ = (x);                                                                          \
        if (e_ != hipSuccess) {                                                                       \
            st = ms::set_error(MS_EHIP, "%s: %s", #x, hipGetErrorString(e_));                         \
            goto done;                                                                                \
        }                                                                                             \
    } while (0)

extern "C" {

ms_status mask_probe_mfma(int32_t kind, int32_t waves_per_simd, double* tflops_out, double* clock_ghz_out) {
    if ((kind != 0 && kind != 1) || waves_per_simd < 1 || waves_per_simd > 4 || !tflops_out)
        return ms::set_error(MS_EINVAL, "need kind 0 or 1, waves_per_simd in 1..4 and tflops_out");
    ms_status st = MS_OK;
    const int blocks = kProbeCUs * waves_per_simd, iters = 20000;
    float* out = nullptr;
    uint64_t* clocks = nullptr;
    uint64_t hc[2] = {0, 0};
    float ms_ = 0.f;
    ProbeTimer t;
    PROBE_HIP(hipMalloc(&out, (size_t)blocks * kProbeThreads * sizeof(float)));
    PROBE_HIP(hipMalloc(&clocks, 2 * sizeof(uint64_t)));
    PROBE_HIP(hipEventCreate(&t.a));
    PROBE_HIP(hipEventCreate(&t.b));
    for (int rep = 0; rep < 2; ++rep) {   // the first launch warms the clocks
        PROBE_HIP(hipEventRecord(t.a, nullptr));
        if (kind == 0) hipLaunchKernelGGL(mfma_probe_kernel<0>, dim3(blocks), dim3(kProbeThreads), 0, nullptr, iters, out, clocks);
        else hipLaunchKernelGGL(mfma_probe_kernel<1>, dim3(blocks), dim3(kProbeThreads), 0, nullptr, iters, out, clocks);
        PROBE_HIP(hipGetLastError());
        PROBE_HIP(hipEventRecord(t.b, nullptr));
        PROBE_HIP(hipEventSynchronize(t.b));
    }
    PROBE_HIP(hipEventElapsedTime(&ms_, t.a, t.b));
    PROBE_HIP(hipMemcpy(hc, clocks, sizeof(hc), hipMemcpyDeviceToHost));
    {
        // 16x16x32 and 32x32x16: 16384 and 32768 FLOPs per instruction, 8 per iteration and wave
        const double per_inst = kind == 0 ? 16384.0 : 32768.0;
        const double flops = per_inst * 8.0 * iters * (double)blocks * (kProbeThreads / kWave);
        *tflops_out = flops / (ms_ * 1e-3) / 1e12;
        if (clock_ghz_out) *clock_ghz_out = hc[1] ? 0.1 * (double)hc[0] / (double)hc[1] : 0.0;
    }
done:
    if (out) (void)hipFree(out);
    if (clocks) (void)hipFree(clocks);
    return st == MS_OK ? ms::clear_error() : st;
}

ms_status mask_probe_lds(double* tbs_out) {
    if (!tbs_out) return ms::set_error(MS_EINVAL, "tbs_out is NULL");
    ms_status st = MS_OK;
    const int blocks = kProbeCUs * 8, iters = 4000;
    float* out = nullptr;
    float ms_ = 0.f;
    ProbeTimer t;
    PROBE_HIP(hipMalloc(&out, (size_t)blocks * kProbeThreads * sizeof(float)));
    PROBE_HIP(hipEventCreate(&t.a));
    PROBE_HIP(hipEventCreate(&t.b));
    for (int rep = 0; rep < 2; ++rep) {
        PROBE_HIP(hipEventRecord(t.a, nullptr));
        hipLaunchKernelGGL(lds_probe_kernel, dim3(blocks), dim3(kProbeThreads), 0, nullptr, iters, out);
        PROBE_HIP(hipGetLastError());
        PROBE_HIP(hipEventRecord(t.b, nullptr));
        PROBE_HIP(hipEventSynchronize(t.b));
    }
    PROBE_HIP(hipEventElapsedTime(&ms_, t.a, t.b));
    *tbs_out = (double)blocks * kProbeThreads * iters * 8 * 16 / (ms_ * 1e-3) / 1e12;
done:
    if (out) (void)hipFree(out);
    return st == MS_OK ? ms::clear_error() : st;
}

ms_status mask_probe_operand_stream(int32_t to_lds, double* us_per_step_out, double* tbs_out) {
    if (!us_per_step_out || !tbs_out) return ms::set_error(MS_EINVAL, "NULL output");
    ms_status st = MS_OK;
    const uint32_t win = 4u << 20;   // per stream of 16 workgroups
    const int blocks = kProbeCUs, steps = 2000;
    uint8_t* src = nullptr;
    float* out = nullptr;
    float ms_ = 0.f;
    ProbeTimer t;
    PROBE_HIP(hipMalloc(&src, (size_t)16 * win));
    PROBE_HIP(hipMemset(src, 1, (size_t)16 * win));
    PROBE_HIP(hipMalloc(&out, (size_t)blocks * 512 * sizeof(float)));
    PROBE_HIP(hipEventCreate(&t.a));
    PROBE_HIP(hipEventCreate(&t.b));
    for (int rep = 0; rep < 2; ++rep) {
        PROBE_HIP(hipEventRecord(t.a, nullptr));
        if (to_lds) hipLaunchKernelGGL(stream_probe_kernel<true>, dim3(blocks), dim3(512), 0, nullptr, src, win, steps, out);
        else hipLaunchKernelGGL(stream_probe_kernel<false>, dim3(blocks), dim3(512), 0, nullptr, src, win, steps, out);
        PROBE_HIP(hipGetLastError());
        PROBE_HIP(hipEventRecord(t.b, nullptr));
        PROBE_HIP(hipEventSynchronize(t.b));
    }
    PROBE_HIP(hipEventElapsedTime(&ms_, t.a, t.b));
    *us_per_step_out = ms_ * 1e3 / steps;
    *tbs_out = (double)blocks * steps * 65536.0 / (ms_ * 1e-3) / 1e12;
done:
    if (src) (void)hipFree(src);
    if (out) (void)hipFree(out);
    return st == MS_OK ? ms::clear_error() : st;
}

}  // extern "C"
