// Mask compaction: the token selection of Sec. 3.1 ("extract the matrix of
// masked tokens"). One workgroup scans the uint8 masks of all requests in
// raster order and emits, in ascending token order per request, the packed
// rows, the inverse map, the segment table and the attention query-tile
// table. Masks are small (B * N bytes, a few KB to tens of KB), so a single
// 1024-thread workgroup keeps the whole scan on one CU with no inter-block
// coordination; the launch is once per mask set.
#include "common.h"
#include "kernels.h"

namespace ms {
namespace {

constexpr int kThreads = 1024;
constexpr int kPerThread = 4;   // consecutive cells per thread and chunk

// Exclusive block-wide prefix sum of `v`; also returns the block total.
__device__ int block_exclusive_scan(int v, int* s_wave, int& total) {
    const int lane = threadIdx.x % kWave;
    const int wave = threadIdx.x / kWave;
    int incl = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        int t = __shfl_up(incl, o, kWave);
        if (lane >= o) incl += t;
    }
    if (lane == kWave - 1) s_wave[wave] = incl;
    __syncthreads();
    if (wave == 0) {
        int w = lane < kThreads / kWave ? s_wave[lane] : 0;
        int wi = w;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            int t = __shfl_up(wi, o, kWave);
            if (lane >= o) wi += t;
        }
        if (lane < kThreads / kWave) s_wave[lane] = wi - w;   // exclusive per wave
        if (lane == kThreads / kWave - 1) s_wave[kThreads / kWave] = wi;
    }
    __syncthreads();
    int excl = s_wave[wave] + incl - v;
    total = s_wave[kThreads / kWave];
    __syncthreads();
    return excl;
}

__global__ __launch_bounds__(kThreads) void compact_kernel(
    const uint8_t* __restrict__ mask, int B, int N, int n_text, int dual,
    int32_t* __restrict__ rows, int32_t* __restrict__ inv, int32_t* __restrict__ seg_start,
    int32_t* __restrict__ seg_req, int32_t* __restrict__ cu_tiles) {
    __shared__ int s_count[64];
    __shared__ int s_seg[kMaxSegments + 1];
    __shared__ int s_wave[kThreads / kWave + 1];
    const int tid = threadIdx.x;
    const int T = n_text + N;
    const bool split = dual && n_text > 0;
    const int nseg = split ? 2 * B : B;

    // masked cells per request
    for (int b = 0; b < B; ++b) {
        int c = 0;
        for (int n = tid; n < N; n += kThreads) c += mask[(size_t)b * N + n] != 0;
        int tot;
        block_exclusive_scan(c, s_wave, tot);
        if (tid == 0) s_count[b] = tot;
    }
    __syncthreads();

    if (tid == 0) {
        int acc = 0, tiles = 0;
        for (int s = 0; s < nseg; ++s) {
            int b = s % B;
            int size = split ? (s < B ? n_text : s_count[b]) : n_text + s_count[b];
            s_seg[s] = acc;
            seg_start[s] = acc;
            seg_req[s] = b;
            cu_tiles[s] = tiles;
            acc += size;
            tiles += (size + kQTile - 1) / kQTile;
        }
        s_seg[nseg] = acc;
        seg_start[nseg] = acc;
        cu_tiles[nseg] = tiles;
    }
    __syncthreads();

    for (int b = 0; b < B; ++b) {
        const int text_base = s_seg[b];
        const int img_base = split ? s_seg[B + b] : s_seg[b] + n_text;
        for (int t = tid; t < n_text; t += kThreads) {
            rows[text_base + t] = b * T + t;
            inv[(size_t)b * T + t] = text_base + t;
        }
        int carry = 0;
        for (int c0 = 0; c0 < N; c0 += kThreads * kPerThread) {
            const int n0 = c0 + tid * kPerThread;
            int f[kPerThread];
            int cnt = 0;
#pragma unroll
            for (int e = 0; e < kPerThread; ++e) {
                int n = n0 + e;
                f[e] = (n < N) ? (mask[(size_t)b * N + n] != 0) : 0;
                cnt += f[e];
            }
            int tot;
            int off = block_exclusive_scan(cnt, s_wave, tot);
            int m = img_base + carry + off;
#pragma unroll
            for (int e = 0; e < kPerThread; ++e) {
                int n = n0 + e;
                if (n < N) {
                    int r = b * T + n_text + n;
                    if (f[e]) {
                        rows[m] = r;
                        inv[r] = m;
                        ++m;
                    } else {
                        inv[r] = -1;
                    }
                }
            }
            carry += tot;
        }
    }
}

}  // namespace

hipError_t launch_compact(const uint8_t* mask, int B, int N, int n_text, int dual,
                          int32_t* rows, int32_t* inv, int32_t* seg_start, int32_t* seg_req,
                          int32_t* cu_tiles, hipStream_t s) {
    hipLaunchKernelGGL(compact_kernel, dim3(1), dim3(kThreads), 0, s, mask, B, N, n_text, dual,
                       rows, inv, seg_start, seg_req, cu_tiles);
    return hipGetLastError();
}

}  // namespace ms
