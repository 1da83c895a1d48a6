/*
 * maskstep operator entry points: the block's row GEMM as a standalone call,
 * for kernel-level parity tests and tuning. The step API in maskstep.h uses
 * the same kernels.
 *
 * Table 1 of InstGenIE (arXiv 2505.20600) counts the projections XW and the
 * feed-forward (XW1)W2 as the work that shrinks with the masked-row count;
 * these are the row GEMMs computed here.
 */
#ifndef MASKSTEP_OPS_H
#define MASKSTEP_OPS_H

#include <stddef.h>
#include <stdint.h>

#include "maskstep.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    MS_EPI_BIAS = 0,        /* out = A W^T + bias */
    MS_EPI_BIAS_RESID = 1,  /* out = A W^T + bias + resid */
    MS_EPI_BIAS_GELU = 2    /* out = GELU(A W^T + bias), exact erf GELU */
} ms_epilogue;

/* out[M][N] = epilogue(A[M][K] W[N][K]^T + bias[N] (+ resid[M][N])), row-major,
 * element type `dtype` (ms_dtype), float32 accumulation, device pointers,
 * 16-byte aligned. K must be a multiple of 64 (bf16) or 32 (fp32) and N of 4.
 * tile_m x tile_n selects the output tile (256x256, 256x128, 128x128,
 * 128x64, 64x128 or 64x64; bf16 only; 0 x 0 = the planner's choice) and
 * ksplit the number of K-range splits (0 = planner's choice; > 1 needs
 * ksplit * M * N * 4 bytes of device workspace in d_ws, NULL otherwise).
 * Asynchronous on `stream`; errors as in maskstep.h, nothing enqueued on error. */
ms_status ms_linear(int32_t dtype, int32_t M, int32_t N, int32_t K, const void* A, const void* W,
                    const void* bias, const void* resid, void* out, int32_t epilogue,
                    int32_t tile_m, int32_t tile_n, int32_t ksplit, void* d_ws, size_t ws_bytes,
                    void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MASKSTEP_OPS_H */
