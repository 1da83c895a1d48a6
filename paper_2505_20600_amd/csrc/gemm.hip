// Row GEMMs of the block over the packed masked rows only (Table 1: the
// projections and the feed-forward scale with the masked-row count):
//
//     out[m][n] = epilogue( sum_k A[m][k] * W[n][k] + bias[n] )
//
// Both operands are K-contiguous (activations [M][K], Linear weights
// [N][K]), which is the native operand layout of the CDNA4 matrix cores.
// The weight tile is the MFMA "A" operand and the activation tile the "B"
// operand, so each lane ends up with four consecutive output columns of one
// row and the epilogue writes 4-element vectors.
//
// Epilogues: bias; bias + residual (out-projection and MLP-down); bias +
// exact GELU (MLP-up); QKV, which writes Q to its own buffer and the fresh
// K/V of each masked token straight into that token's row of the working
// K/V (the K/V cache of Fig. 7 with the masked rows replaced).
#include "common.h"
#include "kernels.h"

namespace ms {
namespace {

constexpr int kBM = 128;   // activation rows per workgroup
constexpr int kBN = 128;   // output columns per workgroup
constexpr int kThreads = 256;

template <typename T, int EPI>
__global__ __launch_bounds__(kThreads) void gemm_kernel(GemmDesc g) {
    using E = Elt<T>;
    using frag_t = typename E::frag_t;
    constexpr int BK = 128 / sizeof(T);     // one 128-byte row chunk per K step
    constexpr int V = 16 / sizeof(T);       // elements per 16-byte vector
    constexpr int LDS = BK + V;             // padded LDS row (elements): 144 bytes
    constexpr int CHUNKS = BK / V;          // 16-byte chunks per tile row (8)
    constexpr int ROWS_PER_PASS = kThreads / CHUNKS;   // 32
    constexpr int PASSES = kBM / ROWS_PER_PASS;        // 4
    __shared__ __attribute__((aligned(16))) T sA[kBM * LDS];
    __shared__ __attribute__((aligned(16))) T sW[kBN * LDS];

    const int tid = threadIdx.x;
    const int lane = tid % kWave;
    const int wave = tid / kWave;
    const int wm = wave & 1, wn = wave >> 1;
    const int n0 = blockIdx.x * kBN;
    const int m0 = blockIdx.y * kBM;
    const int M = g.M, N = g.N, K = g.K;
    const T* __restrict__ A = static_cast<const T*>(g.A);
    const T* __restrict__ W = static_cast<const T*>(g.W);

    const int lr = tid / CHUNKS;
    const int lc = tid % CHUNKS;
    vec16 ra[PASSES], rw[PASSES];
    auto gload = [&](int k0) {
#pragma unroll
        for (int i = 0; i < PASSES; ++i) {
            const int m = min(m0 + lr + ROWS_PER_PASS * i, M - 1);
            ra[i] = ld16(A + (long)m * g.lda + k0 + lc * V);
            const int n = min(n0 + lr + ROWS_PER_PASS * i, N - 1);
            rw[i] = ld16(W + (long)n * K + k0 + lc * V);
        }
    };

    f32x4_t acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    const int nk = K / BK;
    gload(0);
    for (int kt = 0; kt < nk; ++kt) {
        __syncthreads();
#pragma unroll
        for (int i = 0; i < PASSES; ++i) {
            st16(&sA[(lr + ROWS_PER_PASS * i) * LDS + lc * V], ra[i]);
            st16(&sW[(lr + ROWS_PER_PASS * i) * LDS + lc * V], rw[i]);
        }
        __syncthreads();
        if (kt + 1 < nk) gload((kt + 1) * BK);
#pragma unroll
        for (int ks = 0; ks < BK / E::kKStep; ++ks) {
            const int kk = ks * E::kKStep + (lane / 16) * E::kKPerLane;
            frag_t fw[4], fa[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                fw[i] = *reinterpret_cast<const frag_t*>(&sW[(wn * 64 + i * 16 + lane % 16) * LDS + kk]);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                fa[j] = *reinterpret_cast<const frag_t*>(&sA[(wm * 64 + j * 16 + lane % 16) * LDS + kk]);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = E::mma(fw[i], fa[j], acc[i][j]);
        }
    }

    const T* __restrict__ bias = static_cast<const T*>(g.bias);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int n = n0 + wn * 64 + i * 16 + (lane / 16) * 4;
        if (n >= N) continue;
        float bv[4];
        load4<T>(bias + n, bv);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int m = m0 + wm * 64 + j * 16 + lane % 16;
            if (m >= M) continue;
            float v[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] = acc[i][j][r] + bv[r];
            if constexpr (EPI == kEpiBiasResid) {
                float rv[4];
                load4<T>(static_cast<const T*>(g.R) + (long)m * g.ldr + n, rv);
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] += rv[r];
            }
            if constexpr (EPI == kEpiBiasGelu) {
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = 0.5f * v[r] * (1.0f + erff(v[r] * 0.70710678118654752f));
            }
            if constexpr (EPI == kEpiQKV) {
                if (n < g.d) {
                    store4<T>(static_cast<T*>(g.C) + (long)m * g.ldc + n, v);
                } else {
                    const long tok = g.rows[m];
                    store4<T>(static_cast<T*>(g.kv) + tok * 2 * g.d + (n - g.d), v);
                }
            } else {
                store4<T>(static_cast<T*>(g.C) + (long)m * g.ldc + n, v);
            }
        }
    }
}

template <typename T>
hipError_t launch_typed(const GemmDesc& g, hipStream_t s) {
    dim3 grid((g.N + kBN - 1) / kBN, (g.M + kBM - 1) / kBM), block(kThreads);
    switch (g.epilogue) {
        case kEpiBias: hipLaunchKernelGGL((gemm_kernel<T, kEpiBias>), grid, block, 0, s, g); break;
        case kEpiBiasResid: hipLaunchKernelGGL((gemm_kernel<T, kEpiBiasResid>), grid, block, 0, s, g); break;
        case kEpiBiasGelu: hipLaunchKernelGGL((gemm_kernel<T, kEpiBiasGelu>), grid, block, 0, s, g); break;
        case kEpiQKV: hipLaunchKernelGGL((gemm_kernel<T, kEpiQKV>), grid, block, 0, s, g); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(int dtype, const GemmDesc& g, hipStream_t s) {
    if (g.M == 0) return hipSuccess;
    return dtype == kBF16 ? launch_typed<bf16_t>(g, s) : launch_typed<float>(g, s);
}

}  // namespace ms
