/*
 * maskstep — one denoising step of a diffusion-transformer block stack in
 * which only the masked (edited) tokens are recomputed, while the unmasked
 * tokens' per-layer keys/values come from a cache of an earlier inference of
 * the same image template (InstGenIE, arXiv 2505.20600: Sec. 3.1 "Mask-aware
 * attention" with Fig. 5, and the K/V-caching variant of "Alternative
 * approaches", Fig. 7; cost model in Table 1; block-wise pipelined cache
 * loading in Sec. 4.2, Fig. 8).
 *
 * C ABI over hand-written HIP kernels for gfx950 (MI355X). Plain pointers
 * and sizes only. The caller owns every buffer (device and pinned host);
 * the library allocates no device memory. Streams and events are passed as
 * `void*` and are `hipStream_t` / `hipEvent_t` of the HIP runtime the
 * caller uses (NULL = the null stream).
 *
 * Conventions
 *  - Every call returns an ms_status. Validation happens before anything is
 *    enqueued, so an error leaves no partial work. The message of the last
 *    error of the calling thread is returned by mask_last_error().
 *  - All work is asynchronous on the given streams. mask_step_init is the
 *    only call that blocks (one small device-to-host copy of the packed
 *    layout, after which it synchronizes its stream).
 *  - Element type: float32 (MS_FP32) or bfloat16 (MS_BF16, raw 16-bit
 *    storage), uniform over weights, activations and caches of one model.
 *    Accumulation is float32 in both cases.
 *  - Layouts (row-major, innermost last):
 *      hidden states        X, Y, Y_cache   [B][T][d]
 *      working K/V          kv              [B][T][2][d]   (K row then V row per token)
 *      pinned host K/V      h_kv            [B][N][2][d]   (image tokens only)
 *      mask                 uint8           [B][N]         (nonzero = masked)
 *      Linear weights       W               [out][in], bias [out]
 *    with T = n_text + N tokens per request, N = grid_h * grid_w image
 *    tokens in raster order (Sec. 2.1), head j owning columns
 *    [j*hd, (j+1)*hd) of Q, K, V and the attention output.
 *  - Packed masked rows: request-major; text tokens (always recomputed)
 *    first within a request. With a separate text weight set (dual_stream)
 *    the text rows of all requests come first, then the image rows of all
 *    requests. Each packed row m has a flat token index rows[m] = b*T + t.
 *  - Limits: d % 64 == 0; head_dim = d / n_heads, a multiple of 8, <= 128;
 *    every pointer 16-byte aligned; batch <= max_batch <= 64; tokens <= 2^20;
 *    bf16: d <= 4096 and one request's K/V block (T x 2 x d x 2 bytes) below
 *    4 GiB; fp32: d <= 2048, head_dim <= 64.
 */
#ifndef MASKSTEP_H
#define MASKSTEP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    MS_OK = 0,
    MS_EINVAL = 1,      /* null pointer, bad enum, bad layer index */
    MS_ESHAPE = 2,      /* shape outside the limits above */
    MS_EDTYPE = 3,      /* unknown element type */
    MS_EALIGN = 4,      /* pointer not 16-byte aligned */
    MS_ENOTPINNED = 5,  /* host pointer that is not pinned (page-locked) memory */
    MS_EWORKSPACE = 6,  /* workspace smaller than mask_workspace_bytes() */
    MS_ESTATE = 7,      /* call out of order (e.g. no step context) */
    MS_EHIP = 8         /* HIP runtime or launch error; message has hipGetErrorString */
} ms_status;

typedef enum { MS_FP32 = 0, MS_BF16 = 1 } ms_dtype;

/* Shape of the block stack (pre-LN transformer blocks, Sec. 3.1). */
typedef struct {
    int32_t n_layers;
    int32_t d_model;
    int32_t n_heads;
    int32_t mlp_mult;     /* feed-forward width = mlp_mult * d_model */
    int32_t grid_h, grid_w;
    int32_t n_text;       /* tokens before the image grid, always recomputed */
    int32_t dual_stream;  /* 1: text tokens use a second weight set */
    int32_t max_batch;
    int32_t dtype;        /* ms_dtype */
    float ln_eps;
} ms_model_desc;

/* One layer's parameters, device pointers of the model's element type. */
typedef struct {
    const void *ln1_g, *ln1_b;   /* [d] */
    const void *w_qkv, *b_qkv;   /* [3d][d], [3d]  (Q rows, then K, then V) */
    const void *w_o, *b_o;       /* [d][d], [d] */
    const void *ln2_g, *ln2_b;   /* [d] */
    const void *w_1, *b_1;       /* [f][d], [f] */
    const void *w_2, *b_2;       /* [d][f], [d] */
} ms_layer_weights;

typedef enum {
    MS_KV_DEVICE = 0, MS_KV_HOST_PINNED = 1,   /* K/V caching (Sec. 3.1, Fig. 7) */
    MS_Y_DEVICE = 2, MS_Y_HOST_PINNED = 3      /* Y caching (Sec. 3.1, Fig. 5 bottom) */
} ms_kv_kind;

/* Where the per-layer cache comes from.
 *  MS_KV_DEVICE:      layer[l] is a device [B][T][2][d] buffer, resident in
 *                     HBM; it is also the working buffer, so the masked rows
 *                     are overwritten with fresh K/V during the step.
 *  MS_KV_HOST_PINNED: layer[l] is a pinned host [B][N][2][d] buffer (image
 *                     tokens). slots[0..n_slots-1] are device [B][T][2][d]
 *                     buffers; the j-th cached layer of the step uses
 *                     slots[j % n_slots], and its load (on the copy stream)
 *                     waits until the compute stream has finished with the
 *                     layer that used the slot before. Across calls: with
 *                     flags & MS_KV_LOADS_AHEAD, right after a
 *                     mask_stack_forward call that streamed through the same
 *                     list of slots (any step context), a call's first loads
 *                     wait only for the blocks of that call that read their
 *                     slots (its first half of cached blocks, then all of
 *                     them), so in a run of steps the next step's loads start
 *                     under the current step's last blocks; otherwise (and
 *                     under stream capture) a call's loads wait for the
 *                     call's start on the compute stream. A caller that
 *                     writes or frees slot
 *                     buffers orders that after the calls that use them.
 *                     With n_slots >= the number of cached layers every load
 *                     starts at once (MI355X's HBM holds a whole stack's K/V
 *                     easily).
 *  MS_Y_DEVICE:       layer[l] is a device [B][N][d] buffer: block l's cached
 *                     input hidden state of the image tokens (only unmasked
 *                     rows are read). Each cached block recomputes the K/V of
 *                     the unmasked tokens from it (mask_recompute_kv) into the
 *                     workspace; half the cache bytes of the K/V kinds.
 *  MS_Y_HOST_PINNED:  layer[l] is a pinned host [B][N][d] buffer; slots are
 *                     device [B][N][d] buffers used as for MS_KV_HOST_PINNED.
 * request_layer (host-pinned kinds, may be NULL): when set, it replaces
 * layer with one pinned buffer per request and layer, entry l * B + b =
 * request b's [N][2][d] (K/V) or [N][d] (Y) cache of layer l, so that each
 * request of a continuously re-formed batch keeps its cache where it is.
 * Entries of requests that recompute nothing (no masked token, no text
 * rows) are never read and may be NULL: such a request loads no cache, in
 * either form (step-level continuous batching, Sec. 4.2 "Continuous
 * Batching": a free batch slot is a request with an empty mask). */
typedef struct {
    int32_t kind;
    const void* const* layer;   /* [n_layers] */
    int32_t n_slots;            /* host-pinned kinds only, >= 1 */
    void* const* slots;         /* [n_slots], host-pinned kinds only */
    const void* const* request_layer;   /* host-pinned kinds only: [n_layers * B] or NULL */
    int32_t flags;              /* MS_KV_* flags below, 0 for none */
} ms_kv_source;

/* flags: the caller guarantees that between this call and the previous
 * mask_stack_forward call through the same list of slots nothing else reads
 * or writes those slots (no graph replay, per-block call or kernel of its own
 * on them). The call's first loads may then start under the previous call's
 * last blocks (see MS_KV_HOST_PINNED); without it a call's loads wait for the
 * call's start on the compute stream. */
#define MS_KV_LOADS_AHEAD 1

typedef struct ms_step ms_step;   /* opaque host object, one per mask set */

typedef struct {
    int32_t batch;
    int32_t rows;        /* M: packed recomputed rows over the batch */
    int32_t n_segments;  /* packed segments (one per request, two with dual_stream) */
    int32_t n_qtiles;    /* attention query tiles */
    int32_t text_rows;   /* packed rows that use the text weight set */
    int32_t dense_prefix;/* blocks computed over every token (mask_step_set_dense_prefix) */
    int32_t copy_spans;  /* host-to-device copies one cached block's K/V load issues
                            (contiguous or strided 2-D; mask_plan_copies per recomputing
                            request, a command priced at 512 KiB of rows) */
    int64_t copy_rows;   /* image rows those copies move (>= the unmasked rows of the
                            requests that recompute anything: the plan may include masked
                            rows); bytes = rows x 2 d x elt */
    int32_t copy_spans_y;/* the same for a Y-cache load (rows of d elements: a command */
    int64_t copy_rows_y; /*  is worth twice as many rows); bytes = rows x d x elt */
} ms_step_info;

/* Bytes of device workspace a step over `batch` requests needs (worst case,
 * every token masked). Returns 0 and sets the error on an invalid description. */
size_t mask_workspace_bytes(const ms_model_desc* desc, int32_t batch);

/* Mask compaction (token selection of Sec. 3.1): from d_mask [B][N] builds,
 * inside the workspace, the ascending masked-row index of every request, the
 * inverse map and the packed-segment table, then copies the segment table to
 * the host and synchronizes `stream`. The workspace must stay valid and
 * unused by anyone else until mask_step_destroy. `*out` receives a new step
 * context. Masks are constant over the denoising steps of a request, so one
 * context serves every step of the same mask set. */
ms_status mask_step_init(ms_step** out, const ms_model_desc* desc, int32_t batch,
                         const uint8_t* d_mask, void* d_ws, size_t ws_bytes, void* stream);

/* Bytes of the device array behind mask_step_init_static (one per device). */
#define MS_STATIC_SCRATCH_BYTES ((size_t)128 << 20)

/* For callers that cannot allocate device memory (code under stream capture,
 * serving loops or harnesses that forbid allocation): mask_step_init with the
 * workspace taken from a device array of the library instead of the caller,
 * MS_STATIC_SCRATCH_BYTES (128 MiB) on each device the library runs on, held
 * from the first call on that device until the process ends. The step must
 * fit: mask_workspace_bytes(desc, batch) <= MS_STATIC_SCRATCH_BYTES (a 12-block
 * d=768 stack over 4096 tokens needs 99 MiB), else MS_EWORKSPACE and nothing
 * is done. One such context per device at a time: while one is alive, another
 * call on the same device returns MS_ESTATE; mask_step_destroy gives the array
 * back. The array keeps what the last context left in it; nothing in it needs
 * to start at zero (the compaction writes every table the step reads). Work of
 * two contexts that overlaps on one device races on the array: destroy a
 * context only after the work enqueued with it has completed. The call
 * allocates no device memory and creates no HIP object; like mask_step_init it
 * synchronizes `stream` once. Every other call takes the context as usual. */
ms_status mask_step_init_static(ms_step** out, const ms_model_desc* desc, int32_t batch,
                                const uint8_t* d_mask, void* stream);

ms_status mask_step_get_info(const ms_step* step, ms_step_info* info);

/* Device pointers into the workspace: rows [M] (flat b*T + t of each packed
 * row), inv [B*T] (packed row of a token, -1 if not recomputed), seg_start
 * [n_segments + 1] (packed offset of each segment). Valid until destroy. */
ms_status mask_step_index(const ms_step* step, const int32_t** d_rows, const int32_t** d_inv,
                          const int32_t** d_seg_start);

/* Bubble-free pipeline loading (Sec. 4.2, Alg. 1). A block may skip its
 * cache and compute every token instead; with K/V caching that is possible
 * only while every earlier block did the same (only then do the unmasked
 * tokens' hidden states exist), so the choice is a prefix: blocks [0, k)
 * over every token (no cache read, fresh K/V of all tokens in a workspace
 * buffer), blocks [k, n_layers) with the cache. mask_stack_forward follows
 * the step's current k (0 after init). The first call with k > 0 enqueues,
 * on `stream`, the construction of the every-token row layout in the
 * workspace. */
ms_status mask_step_set_dense_prefix(ms_step* step, int32_t k, void* stream);

/* Alg. 1's latency model over the prefix choices: with per-block load time
 * load_ms (cached activations of one block over the copy link), compute
 * time cached_ms (masked rows only) and full_ms (every token), a cached
 * block's load follows the previous load and its compute waits for it; a
 * full block needs no load. Returns in *k_out the prefix length with the
 * smallest modelled latency (the smallest such k on ties) and that latency
 * in *latency_ms_out (may be NULL). Host-only. */
ms_status mask_plan_dense_prefix(int32_t n_layers, double load_ms, double cached_ms, double full_ms,
                                 int32_t* k_out, double* latency_ms_out);

/* Cache-load plan of one request (block-wise loading, Sec. 4.2 and Fig. 8:
 * a cached block loads the cached rows of the unmasked image tokens only), as
 * the step context plans it for each request that recomputes rows.
 * Host-only. mask: [grid_h * grid_w] uint8 of one request, row-major on the
 * token grid, non-zero = masked. copy_cost_rows: what one copy command costs,
 * in rows of link time (the step uses 512 KiB / (2 d_model x element size)).
 * The plan is a list of copies; copy i is out[3i .. 3i+2] = (n0, w, h): image
 * rows n0 + j * grid_w + [0, w) for j < h, one strided 2-D copy when h > 1
 * (then w < grid_w), else one contiguous copy of w rows. The copies cover
 * every unmasked row and may include masked ones; the planner minimises
 * sum(copy_cost_rows + w * h) heuristically and never returns a plan costlier
 * than unmasked runs merged across gaps of at most copy_cost_rows rows.
 * *n_out receives the number of copies; MS_ESHAPE (nothing written) when it
 * exceeds cap. out: caller-owned, 3 * cap int32. */
ms_status mask_plan_copies(const uint8_t* mask, int32_t grid_h, int32_t grid_w, double copy_cost_rows,
                           int32_t* out, int32_t cap, int32_t* n_out);

/* Worker-load estimate (Sec. 4.3): linear regression models, fitted offline,
 * that map a batch's computation (FLOPs of Table 1 at the requests' mask
 * ratios) and the bytes of cached activations a block loads to latency:
 *   Comp(F) = comp_ms0 + comp_ms_per_gflop * F / 1e9    (one block)
 *   Load(B) = load_ms0 + load_ms_per_mb * B / 1e6       (one block's cache)
 * Zero work or zero bytes cost nothing (the intercepts apply only to issued
 * work). cache_bytes_per_token is what one unmasked image token's cache holds
 * per block: 2 * d_model * element size for K/V caching, d_model * element
 * size for Y caching. All fields finite and >= 0. */
typedef struct {
    double comp_ms0, comp_ms_per_gflop;
    double load_ms0, load_ms_per_mb;
    double cache_bytes_per_token;
} ms_cost_model;

/* Least-squares line y ~ intercept + slope * x over n >= 2 points with some
 * spread in x (the regression fit of Sec. 4.3), and its coefficient of
 * determination 1 - SS_res / SS_tot (1 when y is constant and fitted
 * exactly). x, y: host arrays of n doubles. r2_out may be NULL. Host-only. */
ms_status mask_fit_linear(const double* x, const double* y, int32_t n, double* intercept_out,
                          double* slope_out, double* r2_out);

/* Per-block costs of a batch and Alg. 1 over them (Sec. 4.3 with Sec. 4.2):
 * masked[b] = masked image tokens of request b (0..grid_h*grid_w; text rows,
 * when the model has them, are always recomputed). costs_out[3] receives
 * L = Load(sum of unmasked image tokens * cache_bytes_per_token),
 * C_w = Comp(sum of the cached blocks' FLOPs) and C_wo = Comp(batch * FLOPs
 * of a block over every token); *k_out and *latency_ms_out the dense prefix
 * and latency of mask_plan_dense_prefix over them. batch = 0 gives zeros.
 * Any output may be NULL. Host-only; desc is validated as for
 * mask_step_init except max_batch. */
ms_status mask_batch_cost(const ms_model_desc* desc, const ms_cost_model* model, const int32_t* masked,
                          int32_t batch, double* costs_out, int32_t* k_out, double* latency_ms_out);

/* Mask-aware request routing (Alg. 2): the cost of a worker is the
 * pipeline latency of its running batch with the new request added
 * (mask_batch_cost); the request goes to the candidate of least cost, the
 * first one on ties; candidates are the workers whose running batch holds
 * fewer than max_batch requests. running_masked holds the masked-token
 * counts of every worker's running batch back to back (worker 0's first),
 * batch_sizes[w] how many belong to worker w. *worker_out = -1 (and cost 0)
 * when no worker has room. cost_ms_out may be NULL. Host-only. */
ms_status mask_route_request(const ms_model_desc* desc, const ms_cost_model* model,
                             const int32_t* running_masked, const int32_t* batch_sizes, int32_t n_workers,
                             int32_t max_batch, int32_t request_masked, int32_t* worker_out,
                             double* cost_ms_out);

/* Row gather ("extract the matrix of masked tokens", Sec. 3.1):
 * d_xm[m] = d_x[rows[m]]; d_x [B][T][d], d_xm [M][d] (may be NULL: the
 * workspace's own packed-hidden buffer is used). */
ms_status mask_gather_rows(ms_step* step, const void* d_x, void* d_xm, void* stream);

/* One pre-LN block over the packed rows (Sec. 3.1, Fig. 5 bottom with the
 * K/V cache of Fig. 7): LN1, QKV projection whose K/V rows are written into
 * d_kv at the masked tokens, attention of the masked queries over all T keys
 * of their request in d_kv, out projection + residual, LN2, feed-forward with
 * GELU + residual. d_xm [M][d] is read and overwritten with the block output
 * (NULL: the workspace buffer). d_kv [B][T][2][d] must hold the cached K/V of
 * every unmasked token; its masked rows are overwritten. `w` points to one
 * weight set, or two (image, text) when dual_stream. `layer` is only checked
 * against n_layers. */
ms_status mask_block_forward(ms_step* step, int32_t layer, const ms_layer_weights* w,
                             void* d_xm, void* d_kv, void* stream);

/* Final scatter ("replenishing cached activations for the unmasked tokens",
 * Sec. 3.1): d_y = d_ycache with d_y[rows[m]] = d_xm[m]. d_y may equal
 * d_ycache (then only the masked rows are written). d_ycache may be NULL only
 * when every token is masked. d_xm NULL: the workspace buffer. */
ms_status mask_scatter_rows(ms_step* step, const void* d_xm, const void* d_ycache, void* d_y,
                            void* stream);

/* Block-wise cache loading (Sec. 4.2, Fig. 8 middle): enqueues on
 * `copy_stream` the host-to-device copies of layer `layer`'s cached K/V of
 * the unmasked image tokens, h_kv [B][N][2][d] (pinned) -> d_slot
 * [B][T][2][d] at rows n_text + n. Runs of unmasked tokens are merged
 * across short masked gaps (the masked rows copied that way are overwritten
 * by the block's fresh K/V afterwards, so the block must be ordered after the
 * copy). If wait_event is not NULL the copies start after it; if
 * signal_event is not NULL it is recorded after them. Nothing is copied when
 * every token is masked. */
ms_status cache_prefetch_layer(ms_step* step, int32_t layer, const void* h_kv, void* d_slot,
                               void* copy_stream, void* wait_event, void* signal_event);

/* The same block-wise loading for Y caching: the unmasked image rows of
 * layer `layer`'s cached block input, h_yin [B][N][d] (pinned) -> d_slot
 * [B][N][d] at the same rows (copy-engine copies of merged runs, as above). */
ms_status cache_prefetch_inputs(ms_step* step, int32_t layer, const void* h_yin, void* d_slot,
                                void* copy_stream, void* wait_event, void* signal_event);

/* Y caching (Sec. 3.1, Fig. 5 bottom: the unmasked tokens are replenished from
 * the cached activations): writes into the working K/V d_kv [B][T][2][d] the
 * K and V of every unmasked image token, computed from its cached block
 * input d_yin [B][N][d] with the block's LN1 and the K/V columns of its QKV
 * projection (image weight set, w[0]). Run it before mask_block_forward, which
 * then fills the masked rows. `w` as for mask_block_forward. Asynchronous on
 * `stream`; nothing is written when no token is unmasked. */
ms_status mask_recompute_kv(ms_step* step, int32_t layer, const ms_layer_weights* w, const void* d_yin,
                            void* d_kv, void* stream);

/* The whole step: gather, the n_layers blocks (the first k of them over every
 * token, see mask_step_set_dense_prefix), final scatter, with the cache (any
 * ms_kv_kind) read from HBM or streamed per layer from pinned host memory on
 * copy_stream through the slot ring, ahead of the compute stream (Fig. 8). `w` holds n_layers
 * weight sets ([n_layers][2] when dual_stream: image, text). d_x [B][T][d]
 * holds the current hidden states (only masked rows and text rows are read);
 * d_y [B][T][d] receives the output; it may equal d_ycache. With the
 * environment variable MS_SERIALIZE=1, copies run on the compute stream
 * before each block instead (the naive loading of Fig. 8 top). With
 * MS_POISON=1 (a debugging mode), every streamed slot is filled with NaN right
 * after the block that used it, so a block that read a row its own load or
 * fresh K/V did not write would produce NaN. */
ms_status mask_stack_forward(ms_step* step, const ms_layer_weights* w, const void* d_x,
                             const void* d_ycache, const ms_kv_source* kv, void* d_y,
                             void* compute_stream, void* copy_stream);

void mask_step_destroy(ms_step* step);

/* Kernel timing (tracing). Between start and stop, every launch of a
 * selected kernel class is bracketed by a pair of timing events on the
 * stream it is launched on; stop synchronizes those events and returns, per
 * class, the summed milliseconds and the launch count (arrays of
 * MS_K_COUNT entries, either may be NULL). Process-wide; up to `capacity`
 * launches are recorded, further ones are counted in `dropped`.
 * MS_K_GEMM_REDUCE (split-K partial sums) includes the LayerNorm that follows
 * a residual projection when the two run as one kernel. */
typedef enum {
    MS_K_COMPACT = 0, MS_K_GATHER = 1, MS_K_LAYERNORM = 2, MS_K_GEMM_QKV = 3,
    MS_K_ATTENTION = 4, MS_K_GEMM_OUT = 5, MS_K_GEMM_UP = 6, MS_K_GEMM_DOWN = 7,
    MS_K_SCATTER = 8, MS_K_COPY = 9, MS_K_ATTN_COMBINE = 10, MS_K_GEMM_REDUCE = 11,
    MS_K_COUNT = 12
} ms_kernel_class;

ms_status mask_profiler_start(uint32_t class_mask, int32_t capacity);
ms_status mask_profiler_stop(double* total_ms, int64_t* launches, int64_t* dropped);

/* The launches recorded between the last start and stop, in recording order:
 * kernel class, and start and end in ms relative to the first recorded start
 * (one timeline across the compute and copy streams, from the same timing
 * events). Up to `capacity` entries are written; *count receives the number
 * recorded. Valid until the next mask_profiler_start. Used to measure how much
 * of the cache-load stream (Sec. 3.2, layer-wise pipelining) runs under the
 * computation. */
ms_status mask_profiler_intervals(int32_t* cls, double* start_ms, double* end_ms, int32_t capacity,
                                  int32_t* count);

/* Diagnostic probes of the rates that bound this library's kernels on the
 * current GPU, for measurement tools (bench.py --ceilings), not for a
 * denoising step: each allocates its own small buffers, launches, times with
 * HIP events and synchronises the device. Synthetic work, no inputs.
 * mask_probe_mfma: matrix-core issue rate with eight independent accumulator
 *   chains per wave; kind 0 = v_mfma_f32_16x16x32_bf16, 1 = 32x32x16;
 *   waves_per_simd 1..4 resident at once on every CU. *tflops_out: dense bf16
 *   TFLOP/s; *clock_ghz_out (may be NULL): the shader clock during the run
 *   (clock counter against the 100 MHz constant clock).
 * mask_probe_lds: aggregate TB/s of conflict-free 16-byte LDS reads.
 * mask_probe_operand_stream: 256 workgroups of 8 waves each move 64 KB per
 *   step from a window shared by 16 of them (like GEMM operand panels),
 *   to_lds != 0: by direct-to-LDS buffer loads into a two-stage LDS ring,
 *   else into registers; *us_per_step_out and the aggregate *tbs_out. */
ms_status mask_probe_mfma(int32_t kind, int32_t waves_per_simd, double* tflops_out, double* clock_ghz_out);
ms_status mask_probe_lds(double* tbs_out);
ms_status mask_probe_operand_stream(int32_t to_lds, double* us_per_step_out, double* tbs_out);

/* Message of the calling thread's last error ("" if none). */
const char* mask_last_error(void);

/* Version of this interface: 7 (2 added Y caching's kinds and calls, 3 the
 * cost-model and routing calls, 4 the copy figures of ms_step_info and
 * mask_profiler_intervals, 5 mask_step_init_static, 6 mask_plan_copies,
 * strided 2-D cache loads and the Y-load figures of ms_step_info, 7
 * ms_kv_source.flags and the probes). */
int32_t mask_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MASKSTEP_H */
