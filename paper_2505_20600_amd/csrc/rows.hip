// Token-wise row kernels: gather of the masked rows, the final scatter into the
// cached hidden state (Sec. 3.1: extract the masked tokens, replenish the
// unmasked ones from the cache), LayerNorm over packed rows, and the split-K
// sum of a residual projection fused with the LayerNorm that follows it.
//
// Gather and scatter are pure HBM copies: 16-byte vector loads/stores, one
// row chunk per thread, grid-stride so that any M fills the chip.
#include "common.h"
#include "kernels.h"

namespace ms {
namespace {

constexpr int kCopyThreads = 256;

__global__ __launch_bounds__(kCopyThreads) void gather_kernel(
    const uint8_t* __restrict__ x, const int32_t* __restrict__ rows, uint8_t* __restrict__ xm,
    long total, int row_vecs) {
    const long stride = (long)gridDim.x * blockDim.x;
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
        const long m = i / row_vecs;
        const int c = (int)(i - m * row_vecs);
        const long src = (long)rows[m] * row_vecs + c;
        st16(xm + (m * row_vecs + c) * 16, ld16(x + src * 16));
    }
}

// Aliased output: only the recomputed rows change.
__global__ __launch_bounds__(kCopyThreads) void scatter_masked_kernel(
    const uint8_t* __restrict__ xm, const int32_t* __restrict__ rows, uint8_t* __restrict__ y,
    long total, int row_vecs) {
    const long stride = (long)gridDim.x * blockDim.x;
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
        const long m = i / row_vecs;
        const int c = (int)(i - m * row_vecs);
        const long dst = (long)rows[m] * row_vecs + c;
        st16(y + dst * 16, ld16(xm + (m * row_vecs + c) * 16));
    }
}

// Separate output: every row of y is written once, from xm or from the cache.
__global__ __launch_bounds__(kCopyThreads) void merge_kernel(
    const uint8_t* __restrict__ xm, const int32_t* __restrict__ inv,
    const uint8_t* __restrict__ ycache, uint8_t* __restrict__ y, long total, int row_vecs) {
    const long stride = (long)gridDim.x * blockDim.x;
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
        const long r = i / row_vecs;
        const int c = (int)(i - r * row_vecs);
        const int m = inv[r];
        const uint8_t* src = m >= 0 ? xm + ((long)m * row_vecs + c) * 16 : ycache + i * 16;
        st16(y + i * 16, ld16(src));
    }
}

__global__ __launch_bounds__(kCopyThreads) void fill_kernel(uint8_t* __restrict__ p, uint8_t v, long n) {
    const long stride = (long)gridDim.x * blockDim.x;
    for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = v;
}

int copy_grid(long total) {
    long blocks = (total + kCopyThreads - 1) / kCopyThreads;
    if (blocks > 256 * 16) blocks = 256 * 16;
    return blocks < 1 ? 1 : (int)blocks;
}

// LayerNorm: one wave per row, the row held in registers (two-pass mean and
// variance in float32), 16-byte vectors. The affine parameters are loaded
// with the row, so their latency overlaps the row's.
constexpr int kLnWaves = 4;
constexpr int kLnMaxVecPerLane = 8;

template <typename T>
__device__ __forceinline__ float vec_elt(const vec16& v, int e) {
    if constexpr (sizeof(T) == 2) {
        const uint32_t w = v.w[e >> 1];
        return __uint_as_float((e & 1) ? (w & 0xffff0000u) : (w << 16));
    } else {
        return __uint_as_float(v.w[e]);
    }
}

// Normalises one row held by a wave: lane holds the 16-byte vectors c = lane
// + 64 i of the row (values v as float, affine parameters gv, bv), mean and
// variance in two passes, y = (v - mean) / sqrt(var + eps) * gamma + beta.
template <typename T, int NV>
__device__ __forceinline__ void ln_row(float (&v)[NV][16 / sizeof(T)], const vec16 (&gv)[NV],
                                       const vec16 (&bv)[NV], int lane, int nvec, int d, float eps,
                                       T* __restrict__ yr) {
    constexpr int V = 16 / sizeof(T);
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int c = lane + i * kWave;
        if (c < nvec) {
#pragma unroll
            for (int e = 0; e < V; ++e) s += v[i][e];
        }
    }
    const float mean = wave_sum(s) / d;
    float q = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int c = lane + i * kWave;
        if (c < nvec) {
#pragma unroll
            for (int e = 0; e < V; ++e) {
                const float t = v[i][e] - mean;
                q += t * t;
            }
        }
    }
    const float rstd = 1.0f / sqrtf(wave_sum(q) / d + eps);
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int c = lane + i * kWave;
        if (c < nvec) {
#pragma unroll
            for (int e = 0; e < V; e += 4) {
                float o[4];
#pragma unroll
                for (int k = 0; k < 4; ++k)
                    o[k] = (v[i][e + k] - mean) * rstd * vec_elt<T>(gv[i], e + k) + vec_elt<T>(bv[i], e + k);
                store4<T>(yr + c * V + e, o);
            }
        }
    }
}

// NV: 16-byte vectors per lane (ceil(d / (64 V))), so the row's registers
// match the width.
template <typename T, int NV>
__global__ __launch_bounds__(kLnWaves * kWave) void layernorm_kernel(
    const T* __restrict__ x, const T* __restrict__ g0, const T* __restrict__ b0,
    const T* __restrict__ g1, const T* __restrict__ b1, int m_split, T* __restrict__ y, int M,
    int d, float eps, const int32_t* __restrict__ idx) {
    constexpr int V = 16 / sizeof(T);   // elements per 16-byte vector
    const int lane = threadIdx.x % kWave;
    const int row = blockIdx.x * kLnWaves + threadIdx.x / kWave;
    if (row >= M) return;
    const T* gam = row < m_split ? g1 : g0;
    const T* bet = row < m_split ? b1 : b0;
    const int nvec = d / V;
    const T* xr = x + (long)(idx ? idx[row] : row) * d;
    vec16 xv[NV], gv[NV], bv[NV];
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int c = lane + i * kWave;
        if (c < nvec) {
            xv[i] = ld16(xr + c * V);
            gv[i] = ld16(gam + c * V);
            bv[i] = ld16(bet + c * V);
        }
    }
    float v[NV][V];
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int c = lane + i * kWave;
        if (c < nvec) {
#pragma unroll
            for (int e = 0; e < V; ++e) v[i][e] = vec_elt<T>(xv[i], e);
        }
    }
    ln_row<T, NV>(v, gv, bv, lane, nvec, d, eps, y + (long)row * d);
}

// Split-K sum of a residual projection followed by the LayerNorm that reads
// its output (Sec. 2.1: a block's attention output projection and MLP each
// add into the residual stream, which the next LayerNorm normalises). Per
// row: c = sum of the partials in split order + bias + residual, stored in T
// (the residual stream), then LayerNorm of the stored values into y. The
// arithmetic and its order are those of the separate split-K sum and
// LayerNorm kernels, so both outputs equal theirs bit for bit; the residual
// row is not read back and one launch is saved.
template <typename T, int KS, int NV>
__global__ __launch_bounds__(kLnWaves * kWave) void reduce_layernorm_kernel(
    const float* __restrict__ part, const T* __restrict__ bias, const T* __restrict__ R,
    int ldr, T* __restrict__ C, int ldc, const T* __restrict__ gam, const T* __restrict__ bet,
    T* __restrict__ y, int ldy, int M, int d, float eps) {
    constexpr int V = 16 / sizeof(T);
    const int lane = threadIdx.x % kWave;
    const int row = blockIdx.x * kLnWaves + threadIdx.x / kWave;
    if (row >= M) return;
    const int nvec = d / V;
    vec16 rv[NV], gv[NV], bv[NV];
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int c = lane + i * kWave;
        if (c < nvec) {
            rv[i] = ld16(R + (long)row * ldr + c * V);
            gv[i] = ld16(gam + c * V);
            bv[i] = ld16(bet + c * V);
        }
    }
    // the KS partials of a vector are loaded together (KS is a compile-time
    // count so that they are all in flight), then summed in split order
    float v[NV][V];
    const float* pr = part + (long)row * d;
    const long plane = (long)M * d;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int c = lane + i * kWave;
        if (c < nvec) {
#pragma unroll
            for (int e = 0; e < V; e += 4) {
                float4 p[KS];
#pragma unroll
                for (int s = 0; s < KS; ++s) p[s] = *reinterpret_cast<const float4*>(pr + s * plane + c * V + e);
                float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll
                for (int s = 0; s < KS; ++s) {
                    a0 += p[s].x; a1 += p[s].y; a2 += p[s].z; a3 += p[s].w;
                }
                v[i][e] = a0; v[i][e + 1] = a1; v[i][e + 2] = a2; v[i][e + 3] = a3;
            }
        }
    }
#pragma unroll
    for (int i = 0; i < NV; ++i) {
        const int c = lane + i * kWave;
        if (c < nvec) {
#pragma unroll
            for (int e = 0; e < V; e += 4) {
                float bb[4];
                load4<T>(bias + c * V + e, bb);
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    v[i][e + k] += bb[k];
                    v[i][e + k] += vec_elt<T>(rv[i], e + k);
                }
                T* cp = C + (long)row * ldc + c * V + e;
                if constexpr (sizeof(T) == 2) {
                    // LayerNorm takes the stored (rounded) residual values
                    uint2 o;
                    o.x = pack_bf16x2(v[i][e], v[i][e + 1]);
                    o.y = pack_bf16x2(v[i][e + 2], v[i][e + 3]);
                    *reinterpret_cast<uint2*>(cp) = o;
                    v[i][e] = __uint_as_float(o.x << 16);
                    v[i][e + 1] = __uint_as_float(o.x & 0xffff0000u);
                    v[i][e + 2] = __uint_as_float(o.y << 16);
                    v[i][e + 3] = __uint_as_float(o.y & 0xffff0000u);
                } else {
                    store4<T>(cp, &v[i][e]);
                }
            }
        }
    }
    ln_row<T, NV>(v, gv, bv, lane, nvec, d, eps, y + (long)row * ldy);
}

constexpr int kMaxReduceSplit = 8;

// Vectors per lane of a d-wide row (1..kLnMaxVecPerLane; d is validated at
// model creation).
template <typename T>
int ln_nv(int d) {
    constexpr int V = 16 / sizeof(T);
    return (d / V + kWave - 1) / kWave;
}

template <typename T, int KS, int NV>
hipError_t reduce_ln_launch_nv(const float* part, const void* bias, const void* R, int ldr, void* C, int ldc,
                               const void* g, const void* b, void* y, int ldy, int M, int d, float eps,
                               hipStream_t s) {
    dim3 grid((M + kLnWaves - 1) / kLnWaves), block(kLnWaves * kWave);
    hipLaunchKernelGGL((reduce_layernorm_kernel<T, KS, NV>), grid, block, 0, s, part,
                       static_cast<const T*>(bias), static_cast<const T*>(R), ldr, static_cast<T*>(C), ldc,
                       static_cast<const T*>(g), static_cast<const T*>(b), static_cast<T*>(y), ldy, M, d, eps);
    return hipGetLastError();
}

template <typename T, int KS>
hipError_t reduce_ln_launch(const float* part, const void* bias, const void* R, int ldr, void* C, int ldc,
                            const void* g, const void* b, void* y, int ldy, int M, int d, float eps,
                            hipStream_t s) {
    switch (ln_nv<T>(d)) {
#define MS_NV(n) case n: return reduce_ln_launch_nv<T, KS, n>(part, bias, R, ldr, C, ldc, g, b, y, ldy, M, d, eps, s);
        MS_NV(1) MS_NV(2) MS_NV(3) MS_NV(4) MS_NV(5) MS_NV(6) MS_NV(7) MS_NV(8)
#undef MS_NV
        default: return hipErrorInvalidValue;
    }
}

template <typename T, int NV>
hipError_t ln_launch_nv(const void* x, const void* g0, const void* b0, const void* g1, const void* b1,
                        int m_split, void* y, int M, int d, float eps, hipStream_t s, const int32_t* idx) {
    dim3 grid((M + kLnWaves - 1) / kLnWaves), block(kLnWaves * kWave);
    hipLaunchKernelGGL((layernorm_kernel<T, NV>), grid, block, 0, s, static_cast<const T*>(x),
                       static_cast<const T*>(g0), static_cast<const T*>(b0), static_cast<const T*>(g1),
                       static_cast<const T*>(b1), m_split, static_cast<T*>(y), M, d, eps, idx);
    return hipGetLastError();
}

template <typename T>
hipError_t ln_launch(const void* x, const void* g0, const void* b0, const void* g1, const void* b1,
                     int m_split, void* y, int M, int d, float eps, hipStream_t s, const int32_t* idx) {
    switch (ln_nv<T>(d)) {
#define MS_NV(n) case n: return ln_launch_nv<T, n>(x, g0, b0, g1, b1, m_split, y, M, d, eps, s, idx);
        MS_NV(1) MS_NV(2) MS_NV(3) MS_NV(4) MS_NV(5) MS_NV(6) MS_NV(7) MS_NV(8)
#undef MS_NV
        default: return hipErrorInvalidValue;
    }
}

template <typename T>
hipError_t reduce_ln_dispatch(int ksplit, const float* part, const void* bias, const void* R, int ldr, void* C,
                              int ldc, const void* g, const void* b, void* y, int ldy, int M, int d, float eps,
                              hipStream_t s) {
    switch (ksplit) {
#define MS_KS(n) case n: return reduce_ln_launch<T, n>(part, bias, R, ldr, C, ldc, g, b, y, ldy, M, d, eps, s);
        MS_KS(1) MS_KS(2) MS_KS(3) MS_KS(4) MS_KS(5) MS_KS(6) MS_KS(7) MS_KS(8)
#undef MS_KS
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_fill_u8(void* p, uint8_t v, size_t n, hipStream_t s) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(fill_kernel, dim3(copy_grid((long)n)), dim3(kCopyThreads), 0, s,
                       static_cast<uint8_t*>(p), v, (long)n);
    return hipGetLastError();
}

hipError_t launch_gather(const void* x, const int32_t* rows, void* xm, int M, int row_bytes,
                         hipStream_t s) {
    if (M == 0) return hipSuccess;
    const int row_vecs = row_bytes / 16;
    const long total = (long)M * row_vecs;
    hipLaunchKernelGGL(gather_kernel, dim3(copy_grid(total)), dim3(kCopyThreads), 0, s,
                       static_cast<const uint8_t*>(x), rows, static_cast<uint8_t*>(xm), total,
                       row_vecs);
    return hipGetLastError();
}

hipError_t launch_scatter(const void* xm, const int32_t* rows, const int32_t* inv,
                          const void* ycache, void* y, int M, int total_rows, int row_bytes,
                          hipStream_t s) {
    const int row_vecs = row_bytes / 16;
    if (y == ycache) {
        if (M == 0) return hipSuccess;
        const long total = (long)M * row_vecs;
        hipLaunchKernelGGL(scatter_masked_kernel, dim3(copy_grid(total)), dim3(kCopyThreads), 0,
                           s, static_cast<const uint8_t*>(xm), rows, static_cast<uint8_t*>(y),
                           total, row_vecs);
    } else {
        const long total = (long)total_rows * row_vecs;
        if (total == 0) return hipSuccess;
        hipLaunchKernelGGL(merge_kernel, dim3(copy_grid(total)), dim3(kCopyThreads), 0, s,
                           static_cast<const uint8_t*>(xm), inv,
                           static_cast<const uint8_t*>(ycache), static_cast<uint8_t*>(y), total,
                           row_vecs);
    }
    return hipGetLastError();
}

hipError_t launch_layernorm(int dtype, const void* x, const void* g0, const void* b0,
                            const void* g1, const void* b1, int m_split, void* y, int M, int d,
                            float eps, hipStream_t s, const int32_t* idx) {
    if (M == 0) return hipSuccess;
    return dtype == kBF16 ? ln_launch<bf16_t>(x, g0, b0, g1, b1, m_split, y, M, d, eps, s, idx)
                          : ln_launch<float>(x, g0, b0, g1, b1, m_split, y, M, d, eps, s, idx);
}

hipError_t launch_reduce_layernorm(int dtype, const float* part, int ksplit, const void* bias,
                                   const void* R, int ldr, void* C, int ldc, const void* g,
                                   const void* b, void* y, int ldy, int M, int d, float eps,
                                   hipStream_t s) {
    if (M == 0) return hipSuccess;
    if (ksplit < 1 || ksplit > kMaxReduceSplit) return hipErrorInvalidValue;
    return dtype == kBF16
        ? reduce_ln_dispatch<bf16_t>(ksplit, part, bias, R, ldr, C, ldc, g, b, y, ldy, M, d, eps, s)
        : reduce_ln_dispatch<float>(ksplit, part, bias, R, ldr, C, ldc, g, b, y, ldy, M, d, eps, s);
}

}  // namespace ms
