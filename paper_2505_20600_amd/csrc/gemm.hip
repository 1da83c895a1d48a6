// Row GEMMs of the block over the packed masked rows only (Table 1: the
// projections and the feed-forward scale with the masked-row count):
//
//     out[m][n] = epilogue( sum_k A[m][k] * W[n][k] + bias[n] )
//
// Both operands are K-contiguous (activations [M][K], Linear weights
// [N][K]), the native operand layout of the CDNA4 matrix cores. The weight
// tile is the MFMA "A" operand and the activation tile the "B" operand, so
// each lane ends up with four consecutive output columns of one row; the
// QKV and plain-bias epilogues and the split-K partials first restage the
// tile through LDS so that consecutive lanes write consecutive columns.
//
// Epilogues: bias; bias + residual (out-projection and MLP-down); bias +
// erf-GELU (MLP-up, erf to 5.5e-7); QKV, which writes Q to its own buffer
// and the fresh K/V of each masked token straight into that token's row of
// the working K/V (the K/V cache of Fig. 7 with the masked rows replaced).
//
// bf16 tiles: BM x BN from 64 x 64 to 256 x 256, operands copied global ->
// LDS without staging registers into 2-4 stages of 64-deep K steps; fp32:
// 64 x 64 tiles through registers, double-buffered. The host picks tile,
// stage count and K split from a step-time table measured on MI355X; split
// workgroups write float32 partials, summed in a fixed order by a second
// kernel that applies the epilogue (or, before a LayerNorm, by the fused
// sum + LayerNorm kernel in rows.hip). Launches with more tiles than the
// CUs hold at once run persistent workgroups.
#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "common.h"
#include "kernels.h"

namespace ms {
namespace {

constexpr int kThreads = 256;
constexpr int kCUs = 256;

// erf(x) by Abramowitz & Stegun, Handbook of Mathematical Functions, formula
// 7.1.26: 1 - t (a1 + t (a2 + t (a3 + t (a4 + t a5)))) exp(-x^2), t = 1 / (1 + p|x|),
// odd in x; |error| <= 1.5e-7 (5.5e-7 evaluated in float32), far below the bf16
// rounding of the GELU output, at one reciprocal, one exponential and five FMAs.
__device__ __forceinline__ float erf_as(float x) {
    const float ax = fabsf(x);
    const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, ax, 1.0f));
    float poly = fmaf(1.061405429f, t, -1.453152027f);
    poly = fmaf(poly, t, 1.421413741f);
    poly = fmaf(poly, t, -0.284496736f);
    poly = fmaf(poly, t, 0.254829592f);
    poly *= t;
    const float e = __builtin_amdgcn_exp2f(-(ax * ax) * 1.4426950408889634f);
    return copysignf(fmaf(-poly, e, 1.0f), x);
}

template <typename T, int EPI>
__device__ __forceinline__ void epilogue_store(const GemmDesc& g, int m, int n, float v[4]) {
    const T* __restrict__ bias = static_cast<const T*>(g.bias);
    float bv[4];
    load4<T>(bias + n, bv);
#pragma unroll
    for (int r = 0; r < 4; ++r) v[r] += bv[r];
    if constexpr (epi_resid(EPI)) {
        float rv[4];
        load4<T>(static_cast<const T*>(g.R) + (long)m * g.ldr + n, rv);
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] += rv[r];
    }
    if constexpr (EPI == kEpiBiasGelu) {
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] = 0.5f * v[r] * (1.0f + erf_as(v[r] * 0.70710678118654752f));
    }
    if constexpr (EPI == kEpiQKV) {
        if (n < g.d) {
            store4<T>(static_cast<T*>(g.C) + (long)m * g.ldc + n, v);
        } else {
            const long tok = g.rows[m];
            store4<T>(static_cast<T*>(g.kv) + tok * g.kvld + (n - g.d), v);
        }
    } else {
        store4<T>(static_cast<T*>(g.C) + (long)m * g.ldc + n, v);
    }
}

// Tile of logical block id `lb` in groups of up to `gm` m-tiles: ids run over
// the m-tiles of a group first, then over n, then to the next group, so that
// the 32 consecutive ids one XCD runs at once cover a 4 x 8 block of tiles
// (12 operand slices per K step in its L2) instead of a 16 x 2 strip (18).
// Measured on MI355X against m-fastest order: -15% time on 6144x3072x3072,
// -11% on 8192x1152x4608, -2..-4% on the other large shapes, equal on small M.
// From 4096 rows on, groups of 8 m-tiles: at c4 (8 x ~860 masked rows) the
// step is 2.6% shorter, mostly in the attention that follows the QKV
// projection; below that, 4 (8 is 0.25% slower at c2).
constexpr int kGroupM = 4;
constexpr int kGroupMLarge = 8;
constexpr int kGroupLargeRows = 4096;

struct TileIdx {
    int kz, m0, n0;
};

__device__ __forceinline__ TileIdx tile_of(int lb, int tiles_m, int tiles_n, int bm, int bn, int gm) {
    const int per_k = tiles_m * tiles_n;
    const int kz = lb / per_k;
    const int r = lb - kz * per_k;
    const int group = r / (gm * tiles_n);
    const int gm0 = group * gm;
    const int gsize = min(gm, tiles_m - gm0);
    const int within = r - group * gm * tiles_n;
    return TileIdx{kz, (gm0 + within % gsize) * bm, (within / gsize) * bn};
}

template <typename T, int BM, int BN, int EPI>
__global__ __launch_bounds__(kThreads) void gemm_kernel(GemmDesc g) {
    using E = Elt<T>;
    using frag_t = typename E::frag_t;
    constexpr int BK = 128 / sizeof(T);     // one 128-byte row chunk per K step
    constexpr int V = 16 / sizeof(T);       // elements per 16-byte vector
    constexpr int LDS = BK + V;             // padded LDS row (elements): 144 bytes
    constexpr int CHUNKS = BK / V;          // 16-byte chunks per tile row (8)
    constexpr int ROWS_PER_PASS = kThreads / CHUNKS;   // 32
    constexpr int PA = BM / ROWS_PER_PASS;
    constexpr int PW = BN / ROWS_PER_PASS;
    constexpr int SM = BM / 32;             // 16-row MFMA blocks per wave (rows m)
    constexpr int SN = BN / 32;             // 16-col MFMA blocks per wave (cols n)
    __shared__ __attribute__((aligned(16))) T sA[2][BM * LDS];
    __shared__ __attribute__((aligned(16))) T sW[2][BN * LDS];

    const int tid = threadIdx.x;
    const int lane = tid % kWave;
    const int wave = tid / kWave;
    const int wm = wave & 1, wn = wave >> 1;
    const int M = g.M, N = g.N, K = g.K;
    // 1-D launch: each XCD takes a contiguous range of logical ids (k split
    // slowest), mapped to tiles in grouped order
    const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
    const int lb = xcd_logical_block(blockIdx.x, tiles_m * tiles_n * g.ksplit);
    const TileIdx ti = tile_of(lb, tiles_m, tiles_n, BM, BN, g.group_m);
    const int kz = ti.kz, m0 = ti.m0, n0 = ti.n0;
    const int kbeg = kz * g.kchunk;
    const int kend = min(K, kbeg + g.kchunk);
    const T* __restrict__ A = static_cast<const T*>(g.A);
    const T* __restrict__ W = static_cast<const T*>(g.W);

    const int lr = tid / CHUNKS;
    const int lc = tid % CHUNKS;
    vec16 ra[PA], rw[PW];
    auto gload = [&](int k0) {
#pragma unroll
        for (int i = 0; i < PA; ++i) {
            const int m = min(m0 + lr + ROWS_PER_PASS * i, M - 1);
            ra[i] = ld16(A + (long)m * g.lda + k0 + lc * V);
        }
#pragma unroll
        for (int i = 0; i < PW; ++i) {
            const int n = min(n0 + lr + ROWS_PER_PASS * i, N - 1);
            rw[i] = ld16(W + (long)n * K + k0 + lc * V);
        }
    };
    auto sstore = [&](int buf) {
#pragma unroll
        for (int i = 0; i < PA; ++i) st16(&sA[buf][(lr + ROWS_PER_PASS * i) * LDS + lc * V], ra[i]);
#pragma unroll
        for (int i = 0; i < PW; ++i) st16(&sW[buf][(lr + ROWS_PER_PASS * i) * LDS + lc * V], rw[i]);
    };

    f32x4_t acc[SN][SM];
#pragma unroll
    for (int i = 0; i < SN; ++i)
#pragma unroll
        for (int j = 0; j < SM; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    const int nk = (kend - kbeg) / BK;
    if (nk > 0) {
        gload(kbeg);
        sstore(0);
    }
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < nk) gload(kbeg + (kt + 1) * BK);
#pragma unroll
        for (int ks = 0; ks < BK / E::kKStep; ++ks) {
            const int kk = ks * E::kKStep + (lane / 16) * E::kKPerLane;
            // all activation fragments, then one weight fragment at a time
            frag_t fa[SM];
#pragma unroll
            for (int j = 0; j < SM; ++j)
                fa[j] = *reinterpret_cast<const frag_t*>(&sA[buf][(wm * (BM / 2) + j * 16 + lane % 16) * LDS + kk]);
#pragma unroll
            for (int i = 0; i < SN; ++i) {
                const frag_t fw = *reinterpret_cast<const frag_t*>(&sW[buf][(wn * (BN / 2) + i * 16 + lane % 16) * LDS + kk]);
#pragma unroll
                for (int j = 0; j < SM; ++j) acc[i][j] = E::mma(fw, fa[j], acc[i][j]);
            }
        }
        if (kt + 1 < nk) sstore(buf ^ 1);
        __syncthreads();
    }

#pragma unroll
    for (int i = 0; i < SN; ++i) {
        const int n = n0 + wn * (BN / 2) + i * 16 + (lane / 16) * 4;
        if (n >= N) continue;
#pragma unroll
        for (int j = 0; j < SM; ++j) {
            const int m = m0 + wm * (BM / 2) + j * 16 + lane % 16;
            if (m >= M) continue;
            float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
            if (g.ksplit == 1) {
                epilogue_store<T, EPI>(g, m, n, v);
            } else {
                *reinterpret_cast<float4*>(g.part + ((long)kz * M + m) * N + n) =
                    make_float4(v[0], v[1], v[2], v[3]);
            }
        }
    }
}

// bf16 main loop with direct global->LDS loads (gfx950 buffer_load_dwordx4
// ... lds, one buffer resource per tile and operand, so rows past M or N read
// as zeros) into S LDS stages, so S-1 K steps are in flight without staging
// registers.
// LDS rows are 128 bytes (one K step of 64 bf16) with their eight 16-byte
// chunks XOR-swizzled by (row >> 1) & 7: each load instruction fills 1 KB
// (8 rows) contiguously, and the 16-row MFMA fragment reads of one K chunk
// still touch 16 distinct bank groups. The copies are issued as opaque
// instructions (dma_buf16) and ordered by explicit counter waits: a compiler
// that sees them must assume each may write the stage being read and drains
// every load in flight before the first fragment read of each step.

// Waves per workgroup of the direct-to-LDS kernel: 256x256, 256x192 and
// 192x192 tiles run eight waves (2 x 4, 128 x 64, 128 x 48 or 96 x 48
// outputs each), the other tiles four (2 x 2). 192-wide tiles fill the 256
// CUs in whole waves where the projection widths are multiples of 192 and not
// of 256 (1152, 3072, 4608, 12288 columns); 192x192 holds three stages in LDS
// and quantises rows more finely than 256-row tiles.
constexpr int dl_waves(int bm, int bn) { return bm * bn >= 192 * 192 ? 8 : 4; }

template <int BM, int BN, int S, int EPI>
__global__ __launch_bounds__(kWave * dl_waves(BM, BN)) void gemm_dl_kernel(GemmDesc g) {
    static_assert(S >= 2 && S <= 4, "stages");
    constexpr int NW = dl_waves(BM, BN);
    constexpr int WM = 2, WN = NW / 2;          // wave grid: WM along m, WN along n
    using E = Elt<bf16_t>;
    using frag_t = typename E::frag_t;
    constexpr int BK = 64;
    constexpr int ROWE = 64;                    // elements per LDS row
    constexpr int IPW = (BM + BN) / (8 * NW);   // 1 KB load instructions per wave per stage
    constexpr int IA = BM / (8 * NW);           // of which for the activation tile
    constexpr int SM = BM / WM / 16;            // 16-row MFMA blocks per wave (rows m)
    constexpr int SN = BN / WN / 16;            // 16-col MFMA blocks per wave (cols n)
    static_assert(BM % (8 * NW) == 0 && BN % (8 * NW) == 0, "load split");
    // S activation stages, then S weight stages; after the main loop the
    // same LDS stages the output tile when its float32 form fits
    __shared__ __attribute__((aligned(1024))) bf16_t smem[S * (BM + BN) * ROWE];
    bf16_t* const sAb = smem;
    bf16_t* const sWb = smem + S * BM * ROWE;
    // output staging passes: the float32 tile in one pass, or in two halves
    // of its rows (the two wave rows) when only half fits
    constexpr int kLdsBytes = S * (BM + BN) * ROWE * 2;
    constexpr int kOutPasses = kLdsBytes >= BM * BN * 4 ? 1 : 2;
    static_assert(kLdsBytes * 2 >= BM * BN * 4 && WM == 2, "output staging");

    const int tid = threadIdx.x;
    const int lane = tid % kWave;
    const int wave = tid / kWave;
    const int wm = wave % WM, wn = wave / WM;
    const int M = g.M, N = g.N, K = g.K;
    const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
    const int total = tiles_m * tiles_n * g.ksplit;
    const bf16_t* __restrict__ A = static_cast<const bf16_t*>(g.A);
    const bf16_t* __restrict__ W = static_cast<const bf16_t*>(g.W);

    // Persistent when the grid is smaller than the tile count: workgroup b
    // takes physical ids b, b + grid, ... (the grid is a multiple of the XCD
    // count, so every id maps to a tile of the workgroup's own XCD).
    // Tile state: split index, tile origin, K range, and the tile's operand
    // rows as buffer resources (rows past M or N read as zeros).
    int kz, m0, n0, kbeg, nk;
    u32x4_t rA, rW;
    auto setup = [&](int hw) {
        const TileIdx ti = tile_of(xcd_logical_block(hw, total), tiles_m, tiles_n, BM, BN, g.group_m);
        kz = ti.kz; m0 = ti.m0; n0 = ti.n0;
        kbeg = kz * g.kchunk;
        nk = (min(K, kbeg + g.kchunk) - kbeg) / BK;
        rA = raw_rsrc(A + (size_t)m0 * g.lda, (uint32_t)((size_t)min(BM, M - m0) * g.lda * 2));
        rW = raw_rsrc(W + (size_t)n0 * K, (uint32_t)((size_t)min(BN, N - n0) * K * 2));
    };
    // per load instruction this lane's byte offset inside the tile's rows
    // (row * ld + swizzled chunk)
    uint32_t voff[IPW];
#pragma unroll
    for (int i = 0; i < IPW; ++i) {
        const int blk = i * NW + wave;                      // 8-row block
        const bool isA = i < IA;
        const int rloc = (isA ? blk : blk - BM / 8) * 8 + lane / 8;
        const int c = (lane % 8) ^ ((rloc >> 1) & 7);
        voff[i] = (uint32_t)((isA ? rloc * g.lda : rloc * K) + c * 8) * 2u;
    }
    // the wave's 1 KB destination of each load instruction inside a stage (bytes)
    uint32_t ldst[IPW];
#pragma unroll
    for (int i = 0; i < IPW; ++i) {
        const int blk = i * NW + wave;
        ldst[i] = i < IA ? lds_addr(sAb + blk * 512) : lds_addr(sWb + (blk - BM / 8) * 512);
    }
    constexpr uint32_t kStageA = BM * ROWE * 2, kStageW = BN * ROWE * 2;   // bytes
    auto issue = [&](int kt, int st) {
        const uint32_t k0 = (uint32_t)(kbeg + kt * BK) * 2u;
#pragma unroll
        for (int i = 0; i < IPW; ++i) {
            if (i < IA) dma_buf16(rA, voff[i], k0, ldst[i] + st * kStageA);
            else dma_buf16(rW, voff[i], k0, ldst[i] + st * kStageW);
        }
    };
    auto prologue = [&]() {
#pragma unroll
        for (int st = 0; st < S - 1; ++st)
            if (st < nk) issue(st, st);
    };

    // fragment offsets inside a stage: row r, logical chunk ks*4 + grp, swizzled by (r >> 1) & 7
    const int sw = (lane % 16) >> 1;
    const int grp = lane / 16;

    int hw = blockIdx.x;
    setup(hw);
    prologue();
    for (;;) {
    f32x4_t acc[SN][SM];
#pragma unroll
    for (int i = 0; i < SN; ++i)
#pragma unroll
        for (int j = 0; j < SM; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    for (int kt = 0; kt < nk; ++kt) {
        const int st = kt % S;
        // stage kt complete (the loads of the later stages may stay in
        // flight); the barrier also ends every wave's reads of the stage
        // refilled next, read in step kt - 1
        if (kt + S - 1 <= nk) wait_vmcnt<(S - 2) * IPW>();
        else wait_vmcnt<0>();
        barrier_only();
        // The 8-wave tiles spread this step's copies over the MFMA groups of
        // the first half step, so the matrix cores start right after the
        // barrier (measured +3..12% on their shapes); the 4-wave tiles issue
        // them at once, which keeps their shorter prefetch distance whole.
        const bool more_k = kt + S - 1 < nk;
        const int k_next = kbeg + (kt + S - 1) * BK, st_next = (kt + S - 1) % S;
        if (NW != 8 && more_k) issue(kt + S - 1, st_next);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            const int ch = ((ks * 4 + grp) ^ sw) * 8;
            frag_t fa[SM];
#pragma unroll
            for (int j = 0; j < SM; ++j)
                fa[j] = *reinterpret_cast<const frag_t*>(sAb + st * BM * ROWE + (wm * (BM / WM) + j * 16 + lane % 16) * ROWE + ch);
#pragma unroll
            for (int i = 0; i < SN; ++i) {
                const frag_t fw = *reinterpret_cast<const frag_t*>(sWb + st * BN * ROWE + (wn * (BN / WN) + i * 16 + lane % 16) * ROWE + ch);
#pragma unroll
                for (int j = 0; j < SM; ++j) acc[i][j] = E::mma(fw, fa[j], acc[i][j]);
                if (NW == 8 && ks == 0 && more_k) {
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int q = i * IPW / SN; q < (i + 1) * IPW / SN; ++q) {
                        if (q < IA) dma_buf16(rA, voff[q], (uint32_t)k_next * 2u, ldst[q] + st_next * kStageA);
                        else dma_buf16(rW, voff[q], (uint32_t)k_next * 2u, ldst[q] + st_next * kStageW);
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
        }
    }

    // Output through LDS: an MFMA block leaves each lane 4 columns of 16 rows,
    // so direct stores write 32-byte pieces of 16 rows; staged, consecutive
    // lanes write consecutive 4-column groups of one row. Float32 in LDS, so
    // the epilogue arithmetic is unchanged. The 16-byte chunks of a staged
    // row are XOR-swizzled by (row & 15), so both the 16-row writes and the
    // row-wise reads are conflict-free. Tiles too large for one pass stage
    // the rows of one wave row (BM / 2) at a time.
    // The host picks the path per launch (GemmDesc::direct_out): direct
    // stores only for the GELU epilogue of launches with few tiles per CU.
    const int hw_next = hw + (int)gridDim.x;
    const bool more = hw_next < total;
    if (EPI == kEpiBiasGelu && g.direct_out) {
        // direct stores from registers: the next tile's first stages load
        // during them (every wave is past its last read of the stages)
        const int cm0 = m0, cn0 = n0;
        if (more) {
            barrier_only();
            setup(hw_next);
            prologue();
        }
#pragma unroll
        for (int i = 0; i < SN; ++i) {
            const int n = cn0 + wn * (BN / WN) + i * 16 + grp * 4;
            if (n >= N) continue;
#pragma unroll
            for (int j = 0; j < SM; ++j) {
                const int m = cm0 + wm * (BM / WM) + j * 16 + lane % 16;
                if (m >= M) continue;
                float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
                epilogue_store<bf16_t, EPI>(g, m, n, v);
            }
        }
        if (!more) return;
        hw = hw_next;
        continue;
    }
    constexpr int CPR = BN / 4;               // 16-byte chunks per staged row
    constexpr int PR = BM / kOutPasses;       // rows per pass
    float* const sc = reinterpret_cast<float*>(smem);
#pragma unroll
    for (int pass = 0; pass < kOutPasses; ++pass) {
        __syncthreads();   // operand reads (or the previous pass's reads) are done
        if (kOutPasses == 1 || wm == pass) {
#pragma unroll
            for (int i = 0; i < SN; ++i) {
                const int nl = wn * (BN / WN) + i * 16 + grp * 4;
#pragma unroll
                for (int j = 0; j < SM; ++j) {
                    const int ml = wm * (BM / WM) + j * 16 + lane % 16 - pass * PR;
                    *reinterpret_cast<float4*>(sc + ml * BN + (((nl / 4) ^ (ml & 15)) * 4)) =
                        make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
                }
            }
        }
        __syncthreads();
        for (int idx = tid; idx < PR * CPR; idx += NW * kWave) {
            const int ml = idx / CPR, c = idx % CPR;
            const int m = m0 + pass * PR + ml, n = n0 + c * 4;
            if (m >= M || n >= N) continue;
            const float4 t = *reinterpret_cast<const float4*>(sc + ml * BN + ((c ^ (ml & 15)) * 4));
            if (g.ksplit == 1) {
                float v[4] = {t.x, t.y, t.z, t.w};
                epilogue_store<bf16_t, EPI>(g, m, n, v);
            } else {
                *reinterpret_cast<float4*>(g.part + ((long)kz * M + m) * N + n) = t;
            }
        }
    }
    if (!more) return;
    __syncthreads();   // the staging reads are done before the stages refill
    hw = hw_next;
    setup(hw);
    prologue();
    }
}

// Split-K: sum the partials in split order, then the epilogue.
template <typename T, int EPI>
__global__ __launch_bounds__(256) void gemm_reduce_kernel(GemmDesc g) {
    const long n4 = (long)g.M * g.N / 4;
    const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n4) return;
    const int m = (int)(i / (g.N / 4));
    const int n = (int)(i - (long)m * (g.N / 4)) * 4;
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    for (int s = 0; s < g.ksplit; ++s) {
        const float4 p = *reinterpret_cast<const float4*>(g.part + ((long)s * g.M + m) * g.N + n);
        v[0] += p.x; v[1] += p.y; v[2] += p.z; v[3] += p.w;
    }
    epilogue_store<T, EPI>(g, m, n, v);
}

template <typename T, int BM, int BN>
hipError_t launch_tile(const GemmDesc& g, hipStream_t s) {
    dim3 grid(((g.N + BN - 1) / BN) * ((g.M + BM - 1) / BM) * g.ksplit), block(kThreads);
    switch (g.epilogue) {
        case kEpiBias: hipLaunchKernelGGL((gemm_kernel<T, BM, BN, kEpiBias>), grid, block, 0, s, g); break;
        case kEpiBiasResid: hipLaunchKernelGGL((gemm_kernel<T, BM, BN, kEpiBiasResid>), grid, block, 0, s, g); break;
        case kEpiBiasGelu: hipLaunchKernelGGL((gemm_kernel<T, BM, BN, kEpiBiasGelu>), grid, block, 0, s, g); break;
        case kEpiQKV: hipLaunchKernelGGL((gemm_kernel<T, BM, BN, kEpiQKV>), grid, block, 0, s, g); break;
        case kEpiBiasResidMlp: hipLaunchKernelGGL((gemm_kernel<T, BM, BN, kEpiBiasResidMlp>), grid, block, 0, s, g); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// Grid of a direct-to-LDS launch: one workgroup per tile, or, past what the
// CUs hold at once, that many persistent workgroups (a multiple of the XCD
// count) looping over the tiles.
unsigned dl_grid(int resident, long tiles) {
    static const bool off = [] {   // tuning knob MS_GEMM_PERSISTENT=0: one workgroup per tile
        const char* v = std::getenv("MS_GEMM_PERSISTENT");
        return v && std::strcmp(v, "0") == 0;
    }();
    if (off || tiles <= resident) return (unsigned)tiles;
    return (unsigned)(resident - resident % kXcds);
}

template <int BM, int BN, int S, int EPI>
hipError_t launch_dl_epi(const GemmDesc& g, hipStream_t s) {
    const long tiles = (long)((g.N + BN - 1) / BN) * ((g.M + BM - 1) / BM) * g.ksplit;
    const int threads = kWave * dl_waves(BM, BN);
    static const int resident = [threads] {   // workgroups of this kernel the CUs hold at once
        int per_cu = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, gemm_dl_kernel<BM, BN, S, EPI>, threads, 0) !=
                hipSuccess || per_cu < 1)
            per_cu = 1;
        return per_cu * kCUs;
    }();
    const unsigned grid = dl_grid(resident, tiles);
    hipLaunchKernelGGL((gemm_dl_kernel<BM, BN, S, EPI>), dim3(grid), dim3(threads), 0, s, g);
    return hipGetLastError();
}

template <int BM, int BN, int S>
hipError_t launch_dl(const GemmDesc& g, hipStream_t s) {
    switch (g.epilogue) {
        case kEpiBias: return launch_dl_epi<BM, BN, S, kEpiBias>(g, s);
        case kEpiBiasResid: return launch_dl_epi<BM, BN, S, kEpiBiasResid>(g, s);
        case kEpiBiasGelu: return launch_dl_epi<BM, BN, S, kEpiBiasGelu>(g, s);
        case kEpiQKV: return launch_dl_epi<BM, BN, S, kEpiQKV>(g, s);
        case kEpiBiasResidMlp: return launch_dl_epi<BM, BN, S, kEpiBiasResidMlp>(g, s);
        default: return hipErrorInvalidValue;
    }
}

template <typename T>
hipError_t launch_reduce(const GemmDesc& g, hipStream_t s) {
    const long n4 = (long)g.M * g.N / 4;
    dim3 grid((unsigned)((n4 + 255) / 256)), block(256);
    switch (g.epilogue) {
        case kEpiBias: hipLaunchKernelGGL((gemm_reduce_kernel<T, kEpiBias>), grid, block, 0, s, g); break;
        case kEpiBiasResid: hipLaunchKernelGGL((gemm_reduce_kernel<T, kEpiBiasResid>), grid, block, 0, s, g); break;
        case kEpiBiasGelu: hipLaunchKernelGGL((gemm_reduce_kernel<T, kEpiBiasGelu>), grid, block, 0, s, g); break;
        case kEpiQKV: hipLaunchKernelGGL((gemm_reduce_kernel<T, kEpiQKV>), grid, block, 0, s, g); break;
        case kEpiBiasResidMlp: hipLaunchKernelGGL((gemm_reduce_kernel<T, kEpiBiasResidMlp>), grid, block, 0, s, g); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

// Tile and stage choice from a measured cost model. A launch whose busiest
// CU holds n workgroups of a tile and stage count costs about
// steps x a(n) + b(n) us: a(n) per 64-deep K step of the whole grid, b(n) the
// per-tile work outside the K loop (prologue, epilogue, stores). Both come
// from timing grids of n x 256 tiles (16 tile columns, GELU epilogue) at
// K = 1024 and K = 4096 on MI355X with the direct-to-LDS main loop; between
// the measured n the model interpolates linearly, past n = 48 it scales with n.
// Checked against 17 projection shapes of the workloads (M 1243..16384,
// N 1152..12288, K 768..12288): the predicted rate is within 10% of the
// measured one for the chosen tile on all but the deepest K (12288, +26%,
// same choice). Split-K multiplies the groups, divides the steps and adds the
// partial-sum pass.
namespace {
constexpr int kCostN = 13;
constexpr int kCostAt[kCostN] = {1, 2, 3, 4, 5, 6, 7, 8, 12, 16, 24, 32, 48};
struct TileCost {
    int bm, bn, stages;
    double step[kCostN];   // a(n), us per K step
    double tile[kCostN];   // b(n), us per launch
};
constexpr TileCost kCost[] = {
    {256, 256, 2, {1.353, 2.677, 3.726, 5.789, 7.043, 9.378, 11.009, 12.507, 18.991, 24.576, 34.741, 49.206, 73.895},
     {23.6, 44.1, 81.1, 79.3, 103.5, 98.8, 114.7, 172.7, 215.0, 360.7, 556.3, 541.7, 843.8}},
    {256, 192, 2, {1.056, 2.152, 3.243, 4.544, 6.230, 7.835, 9.340, 10.339, 14.877, 19.229, 30.646, 39.311, 59.356},
     {18.8, 29.5, 40.4, 47.4, 49.2, 51.8, 61.3, 82.1, 173.6, 237.3, 322.0, 447.8, 652.3}},
    {192, 192, 2, {0.897, 1.802, 2.688, 3.442, 4.039, 5.675, 6.665, 8.428, 12.631, 17.056, 25.517, 34.277, 50.877},
     {14.7, 23.3, 33.4, 54.9, 80.7, 60.6, 75.1, 59.2, 109.6, 142.3, 209.1, 273.6, 439.7}},
    {192, 192, 3, {0.918, 1.858, 2.544, 3.481, 3.979, 5.346, 6.764, 7.776, 11.618, 15.656, 23.449, 31.492, 47.153},
     {15.4, 24.3, 43.5, 53.6, 83.8, 82.1, 72.7, 77.7, 122.1, 163.2, 235.1, 299.6, 456.9}},
    {256, 128, 2, {0.865, 1.797, 2.624, 3.601, 4.574, 5.530, 6.697, 7.757, 11.686, 15.233, 23.217, 31.222, 46.550},
     {21.3, 35.0, 50.1, 62.9, 73.9, 85.7, 91.4, 100.0, 147.7, 223.4, 316.3, 421.8, 611.1}},
    {256, 128, 3, {0.885, 1.787, 2.633, 3.593, 4.522, 5.451, 6.686, 7.655, 11.689, 15.144, 23.001, 31.000, 46.451},
     {22.4, 38.8, 55.5, 69.0, 82.1, 94.1, 99.8, 110.9, 154.1, 216.6, 311.6, 410.4, 595.6}},
    {128, 128, 2, {0.667, 0.872, 1.426, 1.794, 2.263, 2.677, 3.221, 3.821, 5.954, 8.068, 11.962, 16.089, 24.757},
     {8.7, 14.0, 17.0, 19.1, 21.6, 26.4, 26.4, 29.4, 43.7, 60.3, 114.0, 158.4, 211.3}},
    {128, 128, 3, {0.574, 1.152, 1.716, 2.263, 2.870, 3.428, 4.064, 4.601, 6.858, 9.405, 14.008, 18.876, 27.324},
     {11.5, 17.8, 24.8, 31.7, 37.5, 45.0, 50.5, 57.3, 85.5, 109.5, 164.1, 223.9, 347.6}},
    {128, 128, 4, {0.515, 1.059, 1.569, 2.113, 2.627, 3.235, 3.764, 4.230, 6.562, 8.995, 13.730, 18.619, 26.798},
     {13.7, 22.4, 31.8, 40.0, 49.7, 55.6, 64.0, 75.6, 103.3, 129.4, 175.2, 232.1, 362.3}},
    {128, 64, 2, {0.575, 0.579, 0.770, 1.252, 1.319, 1.669, 2.037, 2.174, 3.349, 5.283, 8.289, 11.171, 15.806},
     {3.6, 7.2, 11.6, 11.1, 13.5, 14.1, 14.6, 16.7, 23.4, 11.7, 11.0, 15.4, 89.5}},
    {128, 64, 3, {0.411, 0.547, 0.933, 1.104, 1.489, 1.749, 2.069, 2.405, 3.661, 5.545, 8.539, 12.549, 16.871},
     {6.5, 8.6, 11.0, 12.6, 13.8, 14.7, 15.9, 17.4, 22.4, 20.0, 29.1, 22.3, 89.9}},
    {128, 64, 4, {0.372, 0.759, 1.119, 1.505, 1.865, 2.241, 2.604, 3.044, 4.527, 6.203, 9.681, 13.186, 18.494},
     {7.0, 10.7, 14.7, 17.5, 21.6, 25.4, 29.4, 32.4, 46.6, 62.4, 80.6, 102.3, 191.8}},
    {64, 128, 2, {0.592, 0.609, 0.835, 1.270, 1.357, 1.622, 1.963, 2.110, 3.356, 4.356, 7.593, 10.284, 15.445},
     {3.9, 7.8, 9.4, 10.6, 11.9, 14.1, 14.9, 16.7, 20.5, 24.6, 24.2, 26.8, 73.6}},
    {64, 128, 3, {0.444, 0.559, 0.978, 1.121, 1.507, 1.656, 2.055, 2.233, 3.550, 4.680, 8.045, 11.099, 16.777},
     {7.0, 8.7, 10.8, 12.7, 14.8, 17.9, 18.8, 22.8, 28.0, 41.7, 41.9, 48.0, 75.7}},
    {64, 128, 4, {0.404, 0.815, 1.211, 1.603, 2.021, 2.429, 2.792, 3.216, 4.830, 6.428, 9.697, 13.225, 19.503},
     {7.0, 10.8, 15.1, 18.5, 22.2, 26.5, 31.0, 33.9, 49.1, 65.3, 94.5, 120.0, 192.6}},
    {64, 64, 2, {0.512, 0.497, 0.520, 0.629, 1.065, 1.074, 1.145, 1.308, 2.322, 3.429, 5.004, 7.991, 15.165},
     {1.1, 3.0, 5.3, 7.6, 7.6, 8.8, 10.8, 10.6, 13.3, 13.8, 19.3, 11.3, 0.0}},
    {64, 64, 3, {0.303, 0.387, 0.567, 0.740, 0.883, 1.100, 1.172, 1.348, 2.152, 2.900, 4.561, 7.126, 11.196},
     {5.2, 5.3, 5.3, 7.4, 8.2, 8.6, 9.8, 10.6, 12.5, 14.5, 17.1, 7.0, 5.1}},
    {64, 64, 4, {0.287, 0.373, 0.598, 0.692, 0.939, 1.043, 1.327, 1.423, 2.106, 2.839, 4.474, 7.037, 10.639},
     {5.3, 4.7, 7.5, 8.0, 9.1, 10.8, 10.2, 12.6, 17.5, 20.5, 26.6, 25.2, 27.5}},
};

double interp(const double* v, long n) {
    if (n <= kCostAt[0]) return v[0];
    for (int i = 1; i < kCostN; ++i)
        if (n <= kCostAt[i])
            return v[i - 1] + (v[i] - v[i - 1]) * (double)(n - kCostAt[i - 1]) / (kCostAt[i] - kCostAt[i - 1]);
    return v[kCostN - 1] * (double)n / kCostAt[kCostN - 1];
}
}  // namespace

GemmPlan plan_gemm(int dtype, int M, int N, int K, size_t part_capacity_floats) {
    GemmPlan p{64, 64, 1, 2};
    if (dtype != kBF16) return p;   // fp32 path: one tile shape
    const int steps = K / 64;
    double best = 1e30;
    static const double split_scale = [] {   // tuning knob MS_GEMM_SPLIT_COST: scales the split-K pass cost
        const char* v = std::getenv("MS_GEMM_SPLIT_COST");
        return v ? std::max(0.0, std::atof(v)) : 1.0;
    }();
    for (const TileCost& c : kCost) {
        const long grp = (long)((M + c.bm - 1) / c.bm) * ((N + c.bn - 1) / c.bn);
        for (int ks = 1; ks <= 8 && ks <= steps; ++ks) {
            if (ks > 1 && (size_t)ks * M * N > part_capacity_floats) break;
            const int per = (steps + ks - 1) / ks;
            const long n = (grp * ks + kCUs - 1) / kCUs;
            double us = per * interp(c.step, n) + interp(c.tile, n);
            // partial sums: ks float planes read, one bf16 plane written, ~4 TB/s, + a launch
            if (ks > 1) us += split_scale * (2.0 + ((double)ks * 4 + 2) * M * N / 4.0e6);
            if (us < best * 0.97) {   // prefer the earlier (larger, unsplit) choice on near-ties
                best = us;
                p = GemmPlan{c.bm, c.bn, ks, c.stages};
            }
        }
    }
    if (const char* f = std::getenv("MS_GEMM_TILE")) {   // tuning override "BMxBN"
        int bm = 0, bn = 0;
        if (std::sscanf(f, "%dx%d", &bm, &bn) == 2) {
            for (const TileCost& c : kCost)
                if (c.bm == bm && c.bn == bn && c.stages == 2) p = GemmPlan{bm, bn, 1, 2};
        }
    }
    return p;
}

// Largest stage count whose LDS fits next to nothing else (160 KB per CU).
int max_stages(int bm, int bn) {
    const int per = (bm + bn) * 64 * 2;
    return std::min(4, (160 * 1024) / per);
}

hipError_t launch_gemm(int dtype, GemmDesc& g, hipStream_t s) {
    if (g.M == 0) return hipSuccess;
    const int bk = dtype == kBF16 ? 64 : 32;
    if (g.ksplit < 1) g.ksplit = 1;
    // K range per split, a multiple of the K step
    const int steps = g.K / bk;
    const int per = (steps + g.ksplit - 1) / g.ksplit;
    g.kchunk = per * bk;
    g.ksplit = (steps + per - 1) / per;
    static const int group_m = [] {   // tuning knob MS_GEMM_GROUP (tiles_m or more: m fastest)
        const char* v = std::getenv("MS_GEMM_GROUP");
        return v ? std::max(1, std::atoi(v)) : 0;
    }();
    g.group_m = group_m > 0 ? group_m : (g.M >= kGroupLargeRows ? kGroupMLarge : kGroupM);
    // Output path of the direct-to-LDS kernel: restaged through LDS (whole
    // rows per store), except the unsplit GELU epilogue of launches with fewer
    // than 8 tiles per CU, stored from registers so that the next tile's first
    // loads run under the stores. Measured per shape against the other path
    // (MI355X): residual epilogues restaged 1-6% faster or even everywhere
    // (16384x3072x3072 362 -> 339 us); GELU restaged 10% faster at
    // 16384x12288x3072 (12 tiles per CU), 1-6% slower at 2-3 (2048 and 4096 x
    // 12288 x 3072, 6855x4608x1152).
    {
        const long tiles = (long)((g.M + g.bm - 1) / std::max(1, g.bm)) * ((g.N + g.bn - 1) / std::max(1, g.bn));
        g.direct_out = g.epilogue == kEpiBiasGelu && g.ksplit == 1 && tiles < 8L * kCUs;
    }
    if (dtype != kBF16) return launch_tile<float, 64, 64>(g, s);
    // main loop: direct-to-LDS (default) or the register-staged double buffer
    // (tuning knob MS_GEMM_PIPE=staged); MS_GEMM_STAGES overrides the stage count
    static const bool staged = [] {
        const char* v = std::getenv("MS_GEMM_PIPE");
        return v && std::strcmp(v, "staged") == 0;
    }();
    // tuning knob MS_GEMM_STAGES: the stage count of every direct-to-LDS
    // launch (read per launch, so a test can take each stage variant in turn)
    const char* fs = std::getenv("MS_GEMM_STAGES");
    const int force_stages = fs ? std::atoi(fs) : 0;
    if (staged) {
        if (g.bm == 256 && g.bn == 256) return launch_tile<bf16_t, 256, 256>(g, s);
        if (g.bm == 256 && g.bn == 128) return launch_tile<bf16_t, 256, 128>(g, s);
        if (g.bm == 128 && g.bn == 128) return launch_tile<bf16_t, 128, 128>(g, s);
        if (g.bm == 128 && g.bn == 64) return launch_tile<bf16_t, 128, 64>(g, s);
        if (g.bm == 64 && g.bn == 128) return launch_tile<bf16_t, 64, 128>(g, s);
        return launch_tile<bf16_t, 64, 64>(g, s);
    }
    int st = force_stages > 0 ? force_stages : (g.stages > 0 ? g.stages : 2);
    st = std::max(2, std::min(st, max_stages(g.bm, g.bn)));
    if (g.bm == 256 && g.bn == 256) return launch_dl<256, 256, 2>(g, s);
    if (g.bm == 256 && g.bn == 192) return launch_dl<256, 192, 2>(g, s);
    if (g.bm == 192 && g.bn == 192) return st >= 3 ? launch_dl<192, 192, 3>(g, s) : launch_dl<192, 192, 2>(g, s);
    if (g.bm == 256 && g.bn == 128) return st == 3 ? launch_dl<256, 128, 3>(g, s) : launch_dl<256, 128, 2>(g, s);
    if (g.bm == 128 && g.bn == 128)
        return st == 4 ? launch_dl<128, 128, 4>(g, s) : st == 3 ? launch_dl<128, 128, 3>(g, s) : launch_dl<128, 128, 2>(g, s);
    if (g.bm == 128 && g.bn == 64)
        return st == 4 ? launch_dl<128, 64, 4>(g, s) : st == 3 ? launch_dl<128, 64, 3>(g, s) : launch_dl<128, 64, 2>(g, s);
    if (g.bm == 64 && g.bn == 128)
        return st == 4 ? launch_dl<64, 128, 4>(g, s) : st == 3 ? launch_dl<64, 128, 3>(g, s) : launch_dl<64, 128, 2>(g, s);
    return st == 4 ? launch_dl<64, 64, 4>(g, s) : st == 3 ? launch_dl<64, 64, 3>(g, s) : launch_dl<64, 64, 2>(g, s);
}

hipError_t launch_gemm_reduce(int dtype, const GemmDesc& g, hipStream_t s) {
    if (g.M == 0 || g.ksplit <= 1) return hipSuccess;
    return dtype == kBF16 ? launch_reduce<bf16_t>(g, s) : launch_reduce<float>(g, s);
}

}  // namespace ms
