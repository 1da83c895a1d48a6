// Host-side launchers of the maskstep kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ms {

constexpr int kQTile = 64;        // query rows per workgroup of the generic attention kernel
constexpr int kFastQTile = 128;   // query rows per workgroup of the bf16 attention kernel
constexpr int kMaxSegments = 128; // packed segments per step

enum Dtype { kF32 = 0, kBF16 = 1 };

// a1: mask -> packed rows, inverse map, segment and query-tile tables.
hipError_t launch_compact(const uint8_t* mask, int B, int N, int n_text, int dual,
                          int32_t* rows, int32_t* inv, int32_t* seg_start, int32_t* seg_req,
                          int32_t* cu_tiles, hipStream_t s);

// p[0..n) = v (device bytes).
hipError_t launch_fill_u8(void* p, uint8_t v, size_t n, hipStream_t s);

// a2: xm[m] = x[rows[m]].
hipError_t launch_gather(const void* x, const int32_t* rows, void* xm, int M, int row_bytes,
                         hipStream_t s);

// a11: y = ycache with y[rows[m]] = xm[m] (aliased: only masked rows written).
hipError_t launch_scatter(const void* xm, const int32_t* rows, const int32_t* inv,
                          const void* ycache, void* y, int M, int total_rows, int row_bytes,
                          hipStream_t s);

// a3 / a8: y[i] = LN(x[idx ? idx[i] : i]) row-wise; rows [0, m_split) use (g1, b1),
// the rest (g0, b0).
hipError_t launch_layernorm(int dtype, const void* x, const void* g0, const void* b0,
                            const void* g1, const void* b1, int m_split, void* y, int M, int d,
                            float eps, hipStream_t s, const int32_t* idx = nullptr);
// Split-K sum of a bias + residual projection into C (row stride ldc) fused
// with LayerNorm of the new C rows into y (row stride ldy), one weight set;
// part is [ksplit][M][d] float32, N = d. Same results as the split-K sum
// followed by launch_layernorm.
hipError_t launch_reduce_layernorm(int dtype, const float* part, int ksplit, const void* bias,
                                   const void* R, int ldr, void* C, int ldc, const void* g,
                                   const void* b, void* y, int ldy, int M, int d, float eps,
                                   hipStream_t s);

enum Epilogue { kEpiBias = 0, kEpiBiasResid = 1, kEpiBiasGelu = 2, kEpiQKV = 3, kEpiBiasResidMlp = 4 };

// kEpiBiasResidMlp is kEpiBiasResid for the MLP's second projection: the same
// arithmetic in its own kernel instantiation, so that traces and counters
// tell the two residual projections of a block apart.
constexpr bool epi_resid(int e) { return e == kEpiBiasResid || e == kEpiBiasResidMlp; }

struct GemmDesc {
    const void* A;      // [M][K] activations, row stride lda (elements)
    const void* W;      // [N][K] weights
    const void* bias;   // [N]
    const void* R;      // [M][N] residual (kEpiBiasResid), row stride ldr
    void* C;            // [M][N] output, row stride ldc (kEpiQKV: columns [0, d) only)
    void* kv;           // kEpiQKV: columns [d, N) of packed row m go to kv + rows[m] * kvld
    const int32_t* rows;// kEpiQKV: flat token row of each packed row
    int kvld;           // kEpiQKV: row stride of kv (elements)
    int M, N, K;
    int lda, ldr, ldc;
    int d;              // kEpiQKV: columns that go to C (d for Q|K|V, 0 for K|V only)
    int epilogue;
    int bm, bn;         // output tile (from plan_gemm)
    int stages;         // LDS stages of the bf16 main loop (0: the tile's default)
    int ksplit;         // K-range splits (1: epilogue fused in the GEMM)
    int kchunk;         // set by launch_gemm
    int group_m;        // set by launch_gemm: m-tiles per group of the tile order
    int direct_out;     // set by launch_gemm: output stored from registers, not restaged in LDS
    float* part;        // ksplit > 1: [ksplit][M][N] float32 partials
};

struct GemmPlan {
    int bm, bn, ksplit, stages;
};

// Partial buffer the split-K plans of a step may use (float32 elements):
// 5461 rows of the model width (16 MiB at d_model 768, 64 MiB at 3072), so
// the narrow row blocks whose N = d_model projections need a K split to fill
// the CUs (e.g. 2048 text rows ahead of a LayerNorm) get one at every width.
constexpr size_t gemm_part_floats(size_t d_model) { return size_t(5461) * d_model; }

// Tile shape and K split for an M x N x K product on 256 CUs.
GemmPlan plan_gemm(int dtype, int M, int N, int K, size_t part_capacity_floats);

// a4/a5/a7/a8/a9: out = epi(A W^T + bias); with ksplit > 1 only the partials
// (launch_gemm_reduce applies the epilogue). launch_gemm sets g.kchunk/ksplit.
hipError_t launch_gemm(int dtype, GemmDesc& g, hipStream_t s);
hipError_t launch_gemm_reduce(int dtype, const GemmDesc& g, hipStream_t s);

struct AttnDesc {
    const void* q;        // [M][d]
    const void* kv;       // [B][T][2][d]
    void* o;              // [M][d]
    const int32_t* seg_start;
    const int32_t* seg_req;
    const int32_t* cu_tiles;
    int nseg, T, d, hd, n_qtiles, n_heads;
    float scale_log2;     // log2(e) / sqrt(hd)
    // bf16 path: 128-row query tiles, keys split over `nsplit` workgroups of
    // `tiles_per_split` 64-key tiles; partials (O normalised by its own key
    // range's sum, in bf16, and that range's running max and sum) go to
    // part_o [nsplit][M][d] / part_ml [nsplit][M][n_heads].
    int M, n_qtiles_fast, nsplit, tiles_per_split;
    uint16_t* part_o;     // bf16
    float* part_ml;
};

// True when launch_attention uses the bf16 fast kernel for this head_dim.
bool attention_fast_path(int dtype, int hd);

// a6: attention of the packed masked queries over every key of their request
// (when the key range is split, the partials are left for launch_attention_combine).
hipError_t launch_attention(int dtype, const AttnDesc& a, hipStream_t s);

// Combine of the key-range partials (no-op when nsplit == 1).
hipError_t launch_attention_combine(int dtype, const AttnDesc& a, hipStream_t s);

}  // namespace ms
