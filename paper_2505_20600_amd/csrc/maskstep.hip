// C-ABI of the mask-aware K/V-cached step: validation, workspace carving,
// per-layer orchestration and the pinned-host cache stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <mutex>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <list>
#include <new>
#include <string>
#include <vector>

#include "../../include/maskstep.h"
#include "../../include/maskstep_ops.h"
#include "kernels.h"
#include "step_internal.h"

namespace {

constexpr int32_t kAbiVersion = 7;
constexpr int kMaxBatch = 64;
// A block's cache load is a set of host-to-device copies that covers the
// unmasked rows (copyplan.hip). Measured on MI355X from pinned host memory: a
// copy costs the copy engine ~9 us beyond its bytes (500 copies of 384 KiB
// run at 24 GB/s, 4 of 48 MiB at 57 GB/s), worth ~512 KiB at the link's
// rate, whether it is contiguous or a strided 2-D copy. Spreading the copies
// over several streams hides that cost only while no kernels run: next to the
// compute stream's GEMMs, hundreds of small copies per block crawl at 30-34
// GB/s on 1, 2 or 4 streams. The plan prices a command at 512 KiB of rows.
constexpr size_t kCopyCostBytes = 512 * 1024;

thread_local std::string g_err;

ms_status fail(ms_status st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return st;
}

ms_status ok() {
    g_err.clear();
    return MS_OK;
}

#define MS_HIP(call)                                                                    \
    do {                                                                                \
        hipError_t e_ = (call);                                                         \
        if (e_ != hipSuccess) return fail(MS_EHIP, "%s: %s", #call, hipGetErrorString(e_)); \
    } while (0)

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

struct Layout {
    size_t rows, inv, seg_start, seg_req, cu_tiles;              // masked-row packing
    size_t rows_d, inv_d, seg_start_d, seg_req_d, cu_tiles_d;    // every-token packing
    size_t ones;                                                 // all-ones mask [B][N]
    size_t u_src, u_tok;                                         // unmasked image rows (Y caching)
    size_t xm, a, q, o, h, u, kv_dense, part_o, part_ml, gemm_part, total;
};

// Attention key-range split: enough workgroups to give every CU two to three,
// bounded by the partial buffers (split count x rows <= attn_part_rows).
constexpr int kAttnTargetGroups = 640;

size_t attn_part_rows(const ms_model_desc& d, int32_t B) {
    const size_t BT = (size_t)B * ((size_t)d.n_text + (size_t)d.grid_h * d.grid_w);
    return std::max(BT, (size_t)(131072 / d.n_heads));
}

int elt_bytes(int32_t dtype) { return dtype == MS_BF16 ? 2 : 4; }

ms_status validate_desc(const ms_model_desc* d) {
    if (!d) return fail(MS_EINVAL, "model description is NULL");
    if (d->dtype != MS_FP32 && d->dtype != MS_BF16) return fail(MS_EDTYPE, "unknown dtype %d", d->dtype);
    if (d->n_layers < 1) return fail(MS_ESHAPE, "n_layers must be >= 1");
    if (d->d_model < 64 || d->d_model % 64) return fail(MS_ESHAPE, "d_model must be a positive multiple of 64");
    if (d->n_heads < 1 || d->d_model % d->n_heads) return fail(MS_ESHAPE, "d_model %% n_heads != 0");
    const int hd = d->d_model / d->n_heads;
    if (hd % 8 || hd > 128) return fail(MS_ESHAPE, "head_dim %d must be a multiple of 8 and <= 128", hd);
    if (d->dtype == MS_FP32 && hd > 64) return fail(MS_ESHAPE, "fp32 supports head_dim <= 64");
    if (d->dtype == MS_BF16 && d->d_model > 4096) return fail(MS_ESHAPE, "bf16 supports d_model <= 4096");
    if (d->dtype == MS_FP32 && d->d_model > 2048) return fail(MS_ESHAPE, "fp32 supports d_model <= 2048");
    if (d->mlp_mult < 1 || d->mlp_mult > 8) return fail(MS_ESHAPE, "mlp_mult must be in 1..8");
    if (d->grid_h < 1 || d->grid_w < 1) return fail(MS_ESHAPE, "grid must be at least 1x1");
    if (d->n_text < 0) return fail(MS_ESHAPE, "n_text must be >= 0");
    if ((int64_t)d->grid_h * d->grid_w + d->n_text > (1 << 20)) return fail(MS_ESHAPE, "too many tokens");
    // the bf16 attention addresses one request's K/V block [T][2][d] with 32-bit
    // buffer offsets, so the block must stay below 4 GiB
    if (d->dtype == MS_BF16 && 4ll * ((int64_t)d->grid_h * d->grid_w + d->n_text) * d->d_model >= (1ll << 32))
        return fail(MS_ESHAPE, "one request's K/V block (tokens x 2 x d_model x 2 bytes) must stay below 4 GiB");
    if (d->dual_stream != 0 && d->dual_stream != 1) return fail(MS_EINVAL, "dual_stream must be 0 or 1");
    if (d->max_batch < 1 || d->max_batch > kMaxBatch) return fail(MS_ESHAPE, "max_batch must be in 1..%d", kMaxBatch);
    if (!(d->ln_eps >= 0.f) || !std::isfinite(d->ln_eps)) return fail(MS_EINVAL, "ln_eps must be finite and >= 0");
    return MS_OK;
}

Layout make_layout(const ms_model_desc& d, int32_t B) {
    Layout L{};
    const size_t N = (size_t)d.grid_h * d.grid_w;
    const size_t T = (size_t)d.n_text + N;
    const size_t BT = (size_t)B * T;
    const size_t e = elt_bytes(d.dtype);
    const size_t dm = d.d_model, f = (size_t)d.mlp_mult * d.d_model;
    size_t off = 0;
    auto take = [&](size_t bytes) { size_t o = off; off = align256(off + bytes); return o; };
    L.rows = take(BT * 4);
    L.inv = take(BT * 4);
    L.seg_start = take((ms::kMaxSegments + 1) * 4);
    L.seg_req = take(ms::kMaxSegments * 4);
    L.cu_tiles = take((ms::kMaxSegments + 1) * 4);
    L.rows_d = take(BT * 4);
    L.inv_d = take(BT * 4);
    L.seg_start_d = take((ms::kMaxSegments + 1) * 4);
    L.seg_req_d = take(ms::kMaxSegments * 4);
    L.cu_tiles_d = take((ms::kMaxSegments + 1) * 4);
    L.ones = take((size_t)B * N);
    L.u_src = take((size_t)B * N * 4);
    L.u_tok = take((size_t)B * N * 4);
    L.xm = take(BT * dm * e);
    L.a = take(BT * dm * e);
    L.q = take(BT * dm * e);
    L.o = take(BT * dm * e);
    L.h = take(BT * dm * e);
    L.u = take(BT * f * e);
    L.kv_dense = take(BT * 2 * dm * e);
    L.part_o = take(attn_part_rows(d, B) * dm * 2);   // bf16
    L.part_ml = take(attn_part_rows(d, B) * (size_t)d.n_heads * 2 * 4);
    L.gemm_part = take(ms::gemm_part_floats(dm) * 4);
    L.total = off;
    return L;
}

struct Span {
    int b;              // request
    ms::CopyRect r;     // image rows r.n0 + i * grid_w + [0, r.w) for i < r.h
};

// One packed-row layout of the step: the masked rows, or every token (dense blocks).
struct Packing {
    int32_t *rows = nullptr, *inv = nullptr, *segs = nullptr, *segreq = nullptr, *cutiles = nullptr;
    std::vector<int32_t> seg_start;   // host copy
    int M = 0, nseg = 0, n_qtiles = 0, n_qtiles_fast = 0, text_rows = 0;
    int attn_nsplit = 1, attn_tps = 1;
};

// Kernel timing: event pairs around launches of the selected classes.
struct Profiler {
    std::mutex mu;
    std::atomic<bool> on{false};
    uint32_t mask = 0;
    int capacity = 0, used = 0;
    int64_t dropped = 0;
    std::vector<hipEvent_t> pool;   // 2 per recorded launch
    std::vector<int> cls;
    // intervals of the last stopped run: class, start, end (ms from the first start)
    std::vector<int> last_cls;
    std::vector<double> last_t0, last_t1;
};
Profiler g_prof;

class ProfScope {
  public:
    ProfScope(int c, hipStream_t s) : s_(s) {
        if (!g_prof.on.load(std::memory_order_relaxed) || !(g_prof.mask & (1u << c))) return;
        std::lock_guard<std::mutex> lk(g_prof.mu);
        if (g_prof.used >= g_prof.capacity) { ++g_prof.dropped; return; }
        idx_ = g_prof.used++;
        g_prof.cls[idx_] = c;
        (void)hipEventRecord(g_prof.pool[2 * idx_], s_);
    }
    ~ProfScope() {
        if (idx_ >= 0) (void)hipEventRecord(g_prof.pool[2 * idx_ + 1], s_);
    }
    ProfScope(const ProfScope&) = delete;
    ProfScope& operator=(const ProfScope&) = delete;

  private:
    hipStream_t s_;
    int idx_ = -1;
};

}  // namespace

struct ms_step {
    ms_model_desc desc;
    int B = 0, T = 0, N = 0, d = 0, f = 0, hd = 0, elt = 0;
    bool all_masked = false;
    char* ws = nullptr;
    Layout lay{};
    Packing mp;                 // masked rows
    Packing dp;                 // every token (dense-prefix blocks), built on first use
    bool dense_ready = false;
    int dense_prefix = 0;
    std::vector<Span> spans, spans_y;   // cache-load copies of one block: K/V rows, Y rows
    // unmasked image rows: index into a [B][N] input cache and flat token row (Y caching)
    int U = 0;
    std::vector<int32_t> h_usrc, h_utok;
    std::vector<hipEvent_t> ev_copied, ev_consumed;   // created on first streamed use
    uint64_t stack_calls = 0;   // mask_stack_forward calls on this context (event set parity)
    hipEvent_t ev_start = nullptr;
    int static_dev = -1;        // device whose static scratch is the workspace (mask_step_init_static)

    int M() const { return mp.M; }
    void* buf(size_t off) const { return ws + off; }
    template <typename T> T* at(size_t off) const { return reinterpret_cast<T*>(ws + off); }
};

namespace {

void destroy_events(ms_step* s) {
    for (hipEvent_t e : s->ev_copied) (void)hipEventDestroy(e);
    for (hipEvent_t e : s->ev_consumed) (void)hipEventDestroy(e);
    s->ev_copied.clear();
    s->ev_consumed.clear();
    if (s->ev_start) (void)hipEventDestroy(s->ev_start);
    s->ev_start = nullptr;
}

// Release events of a slot ring (one per device and list of slot buffers),
// recorded on the compute stream by the last call that streamed through it:
// `half` after the block that read slot h - 1 (slots [0, h) free from then
// on; h = 0 when a slot was read twice), `all` after its last cached block.
// The next call's copy stream waits on `half` before its first load and on
// `all` before its load into slot h, instead of waiting for the call's start:
// its first loads then overlap the previous step's last blocks.
struct RingRelease {
    hipEvent_t half[2] = {nullptr, nullptr}, all[2] = {nullptr, nullptr};   // by call parity
    int h = 0;
    bool recorded = false;
    uint64_t call = 0;   // the mask_stack_forward call that recorded them
    uint64_t gen = 0;    // bumped when the entry passes to another slot list
};
// Only the ring of the call right before can release a call's loads early, so
// the registry keeps a few rings per device: a caller that streams through new
// slot buffers every step takes over the least recently used entry (its
// events, never destroyed, are recorded again from then on) instead of
// growing the registry.
constexpr int kRingsPerDevice = 16;
struct RingEntry {
    int dev = 0;
    std::vector<const void*> slots;
    uint64_t last_use = 0;
    RingRelease r;
};
std::mutex g_ring_mu;
std::atomic<uint64_t> g_stack_calls{0};
std::list<RingEntry> g_rings;   // stable addresses
uint64_t g_ring_clock = 0;

ms_status ring_release(const ms_kv_source* kv, RingRelease** out, uint64_t* gen) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(MS_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
    std::vector<const void*> key(kv->slots, kv->slots + kv->n_slots);
    std::lock_guard<std::mutex> lk(g_ring_mu);
    RingEntry* hit = nullptr;
    RingEntry* lru = nullptr;
    int on_dev = 0;
    for (RingEntry& en : g_rings) {
        if (en.dev != dev) continue;
        if (en.slots == key) {
            hit = &en;
            break;
        }
        ++on_dev;
        if (!lru || en.last_use < lru->last_use) lru = &en;
    }
    if (!hit && on_dev >= kRingsPerDevice) {
        hit = lru;
        hit->slots = std::move(key);
        hit->r.recorded = false;
        ++hit->r.gen;
    } else if (!hit) {
        g_rings.emplace_back();
        hit = &g_rings.back();
        hit->dev = dev;
        hit->slots = std::move(key);
    }
    hit->last_use = ++g_ring_clock;
    RingRelease& r = hit->r;
    *gen = r.gen;
    for (int i = 0; i < 2; ++i) {
        if (!r.half[i]) {
            e = hipEventCreateWithFlags(&r.half[i], hipEventDisableTiming);
            if (e == hipSuccess) e = hipEventCreateWithFlags(&r.all[i], hipEventDisableTiming);
            if (e != hipSuccess) {
                if (r.half[i]) (void)hipEventDestroy(r.half[i]);
                r.half[i] = r.all[i] = nullptr;
                return fail(MS_EHIP, "event creation: %s", hipGetErrorString(e));
            }
        }
    }
    *out = &r;
    return MS_OK;
}

// The per-block calls touch slots outside any ring's release events: the next
// mask_stack_forward then waits for its own start again.
void forget_rings() {
    std::lock_guard<std::mutex> lk(g_ring_mu);
    for (RingEntry& en : g_rings) en.r.recorded = false;
}

ms_status ensure_events(ms_step* s, int n) {
    if (!s->ev_start) {
        hipError_t e = hipEventCreateWithFlags(&s->ev_start, hipEventDisableTiming);
        if (e != hipSuccess) {
            s->ev_start = nullptr;
            return fail(MS_EHIP, "event creation: %s", hipGetErrorString(e));
        }
    }
    while ((int)s->ev_copied.size() < n) {
        hipEvent_t a = nullptr, b = nullptr;
        hipError_t e = hipEventCreateWithFlags(&a, hipEventDisableTiming);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&b, hipEventDisableTiming);
        if (e != hipSuccess) {
            if (a) (void)hipEventDestroy(a);
            return fail(MS_EHIP, "event creation: %s", hipGetErrorString(e));
        }
        s->ev_copied.push_back(a);
        s->ev_consumed.push_back(b);
    }
    return MS_OK;
}

// Host-side tables of a packing from its segment starts: query tiles and the
// attention key-range split.
void finish_packing(Packing& p, const ms_model_desc& desc, int batch, int T, int hd) {
    p.M = p.seg_start[p.nseg];
    p.n_qtiles = 0;
    p.n_qtiles_fast = 0;
    for (int i = 0; i < p.nseg; ++i) {
        const int len = p.seg_start[i + 1] - p.seg_start[i];
        p.n_qtiles += (len + ms::kQTile - 1) / ms::kQTile;
        p.n_qtiles_fast += (len + ms::kFastQTile - 1) / ms::kFastQTile;
    }
    const int ntiles = (T + 63) / 64;
    const int base = std::max(1, p.n_qtiles_fast * desc.n_heads);
    int target = kAttnTargetGroups;
    if (const char* ev = std::getenv("MS_ATTN_SPLIT_TARGET")) target = std::max(1, std::atoi(ev));
    int ns = std::min(ntiles, std::max(1, (target + base - 1) / base));
    if (p.M > 0) ns = std::min(ns, std::max(1, (int)(attn_part_rows(desc, batch) / p.M)));
    if (!ms::attention_fast_path(desc.dtype, hd)) ns = 1;
    const int tps = (ntiles + ns - 1) / ns;
    p.attn_tps = tps;
    p.attn_nsplit = (ntiles + tps - 1) / tps;
}

// A request recomputes rows when it has a masked token or text rows (always
// recomputed). One that does not needs neither its cache nor any K/V of its
// unmasked tokens: its output is the cached hidden state.
bool request_recomputes(const ms_step* s, const uint8_t* m) {
    if (s->desc.n_text > 0) return true;
    for (int n = 0; n < s->N; ++n)
        if (m[n]) return true;
    return false;
}

bool env_flag(const char* name);

void plan_spans(ms_step* s, const std::vector<uint8_t>& mask) {
    size_t cost_bytes = kCopyCostBytes;
    if (const char* v = std::getenv("MS_COPY_GAP_BYTES")) cost_bytes = (size_t)std::atoll(v);   // tuning knob
    const bool strided = !env_flag("MS_COPY_RUNS_ONLY");
    std::vector<ms::CopyRect> rects;
    // a command's price in rows depends on the row: 2 d elements (K/V) or d (Y)
    for (int y = 0; y < 2; ++y) {
        std::vector<Span>& out = y ? s->spans_y : s->spans;
        out.clear();
        const double C = (double)cost_bytes / (double)((y ? 1ull : 2ull) * s->d * s->elt);
        for (int b = 0; b < s->B; ++b) {
            const uint8_t* m = mask.data() + (size_t)b * s->N;
            if (!request_recomputes(s, m)) continue;   // no query attends over its keys
            ms::plan_copies(m, s->desc.grid_h, s->desc.grid_w, C, strided, rects);
            for (const ms::CopyRect& r : rects) out.push_back(Span{b, r});
        }
    }
}

// The every-token packing (dense-prefix blocks): compaction of an all-ones mask.
ms_status build_dense_packing(ms_step* s, hipStream_t st) {
    if (s->dense_ready) return MS_OK;
    const bool split = s->desc.dual_stream && s->desc.n_text > 0;
    Packing& p = s->dp;
    p.rows = s->at<int32_t>(s->lay.rows_d);
    p.inv = s->at<int32_t>(s->lay.inv_d);
    p.segs = s->at<int32_t>(s->lay.seg_start_d);
    p.segreq = s->at<int32_t>(s->lay.seg_req_d);
    p.cutiles = s->at<int32_t>(s->lay.cu_tiles_d);
    p.nseg = split ? 2 * s->B : s->B;
    p.text_rows = split ? s->B * s->desc.n_text : 0;
    p.seg_start.assign(p.nseg + 1, 0);
    for (int i = 0; i < p.nseg; ++i) {
        const int len = split ? (i < s->B ? s->desc.n_text : s->N) : s->T;
        p.seg_start[i + 1] = p.seg_start[i] + len;
    }
    finish_packing(p, s->desc, s->B, s->T, s->hd);
    MS_HIP(ms::launch_fill_u8(s->buf(s->lay.ones), 1, (size_t)s->B * s->N, st));
    MS_HIP(ms::launch_compact(static_cast<const uint8_t*>(s->buf(s->lay.ones)), s->B, s->N,
                              s->desc.n_text, split ? 1 : 0, p.rows, p.inv, p.segs, p.segreq,
                              p.cutiles, st));
    s->dense_ready = true;
    return MS_OK;
}

ms_status check_weights(const ms_step* s, const ms_layer_weights* w) {
    const int nsets = (s->desc.dual_stream && s->desc.n_text > 0) ? 2 : 1;
    for (int i = 0; i < nsets; ++i) {
        const void* p[] = {w[i].ln1_g, w[i].ln1_b, w[i].w_qkv, w[i].b_qkv, w[i].w_o, w[i].b_o,
                           w[i].ln2_g, w[i].ln2_b, w[i].w_1, w[i].b_1, w[i].w_2, w[i].b_2};
        for (const void* q : p) {
            if (!q) return fail(MS_EINVAL, "weight set %d has a NULL pointer", i);
            if (!aligned16(q)) return fail(MS_EALIGN, "weight set %d has a pointer not 16-byte aligned", i);
        }
    }
    return MS_OK;
}

bool env_flag(const char* name) {
    const char* v = std::getenv(name);
    return v && v[0] && std::strcmp(v, "0") != 0;
}

// LayerNorm of a GEMM's output rows (row stride N) into y (row stride N),
// one weight set.
struct LnAfter {
    const void* g;
    const void* b;
    void* y;
};

// A projection, with the LayerNorm that reads its output when `ln` is given:
// fused into the split-K sum when the plan splits K (bias + residual
// epilogue only), else a LayerNorm launch of its own.
hipError_t run_gemm(ms_step* s, ms::GemmDesc& g, int cls, hipStream_t st, const LnAfter* ln = nullptr) {
    const ms::GemmPlan p = ms::plan_gemm(s->desc.dtype, g.M, g.N, g.K, ms::gemm_part_floats(s->d));
    g.bm = p.bm;
    g.bn = p.bn;
    g.stages = p.stages;
    g.ksplit = p.ksplit;
    g.part = static_cast<float*>(s->buf(s->lay.gemm_part));
    hipError_t e;
    {
        ProfScope prof(cls, st);
        e = ms::launch_gemm(s->desc.dtype, g, st);
    }
    if (e != hipSuccess) return e;
    if (g.ksplit > 1) {
        ProfScope prof(MS_K_GEMM_REDUCE, st);
        if (ln && ms::epi_resid(g.epilogue) && !env_flag("MS_NO_LN_FUSE"))
            return ms::launch_reduce_layernorm(s->desc.dtype, g.part, g.ksplit, g.bias, g.R, g.ldr, g.C,
                                               g.ldc, ln->g, ln->b, ln->y, g.N, g.M, g.N, s->desc.ln_eps, st);
        e = ms::launch_gemm_reduce(s->desc.dtype, g, st);
        if (e != hipSuccess) return e;
    }
    if (!ln) return hipSuccess;
    ProfScope prof(MS_K_LAYERNORM, st);
    return ms::launch_layernorm(s->desc.dtype, g.C, ln->g, ln->b, ln->g, ln->b, 0, ln->y, g.M, g.N,
                                s->desc.ln_eps, st);
}

// One block over the packed rows. `a_ready`: the scratch row buffer already
// holds LayerNorm 1 of xm (the previous block computed it); `next`: weights
// of the block that follows on the same rows, whose LayerNorm 1 this block
// then leaves in the scratch buffer.
ms_status block_forward(ms_step* s, const Packing& pk, const ms_layer_weights* w, void* xm, void* kv,
                        hipStream_t st, const ms_layer_weights* next = nullptr, bool a_ready = false) {
    if (pk.M == 0) return MS_OK;
    const int dt = s->desc.dtype;
    const bool dual = s->desc.dual_stream && s->desc.n_text > 0;
    const ms_layer_weights& wi = w[0];
    const ms_layer_weights& wt = dual ? w[1] : w[0];
    const int M = pk.M, d = s->d, f = s->f, e = s->elt;
    const int msplit = pk.text_rows;
    char* a = static_cast<char*>(s->buf(s->lay.a));
    char* q = static_cast<char*>(s->buf(s->lay.q));
    char* o = static_cast<char*>(s->buf(s->lay.o));
    char* h = static_cast<char*>(s->buf(s->lay.h));
    char* u = static_cast<char*>(s->buf(s->lay.u));
    char* x = static_cast<char*>(xm);

    if (!a_ready) {
        ProfScope p(MS_K_LAYERNORM, st);
        MS_HIP(ms::launch_layernorm(dt, x, wi.ln1_g, wi.ln1_b, wt.ln1_g, wt.ln1_b, msplit, a, M, d,
                                    s->desc.ln_eps, st));
    }
    // row ranges per weight set: text rows [0, msplit) then image rows; `nw`
    // is the next block's weight set for the same rows
    struct Range { int r0, r1; const ms_layer_weights* w; const ms_layer_weights* nw; };
    Range ranges[2] = {{0, msplit, &wt, next ? &next[dual ? 1 : 0] : nullptr},
                       {msplit, M, &wi, next}};
    for (const Range& r : ranges) {
        if (r.r1 <= r.r0) continue;
        ms::GemmDesc g{};
        g.A = a + (size_t)r.r0 * d * e;
        g.W = r.w->w_qkv;
        g.bias = r.w->b_qkv;
        g.C = q + (size_t)r.r0 * d * e;
        g.kv = kv;
        g.rows = pk.rows + r.r0;
        g.M = r.r1 - r.r0; g.N = 3 * d; g.K = d;
        g.lda = d; g.ldc = d; g.d = d; g.kvld = 2 * d;
        g.epilogue = ms::kEpiQKV;
        MS_HIP(run_gemm(s, g, MS_K_GEMM_QKV, st));
    }
    ms::AttnDesc ad{};
    ad.q = q; ad.kv = kv; ad.o = o;
    ad.seg_start = pk.segs; ad.seg_req = pk.segreq; ad.cu_tiles = pk.cutiles;
    ad.nseg = pk.nseg; ad.T = s->T; ad.d = d; ad.hd = s->hd;
    ad.n_qtiles = pk.n_qtiles; ad.n_heads = s->desc.n_heads;
    ad.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)s->hd));
    ad.M = M;
    ad.n_qtiles_fast = pk.n_qtiles_fast;
    ad.nsplit = pk.attn_nsplit;
    ad.tiles_per_split = pk.attn_tps;
    ad.part_o = static_cast<uint16_t*>(s->buf(s->lay.part_o));
    ad.part_ml = static_cast<float*>(s->buf(s->lay.part_ml));
    {
        ProfScope p(MS_K_ATTENTION, st);
        MS_HIP(ms::launch_attention(dt, ad, st));
    }
    {
        ProfScope p(MS_K_ATTN_COMBINE, st);
        MS_HIP(ms::launch_attention_combine(dt, ad, st));
    }
    for (const Range& r : ranges) {
        if (r.r1 <= r.r0) continue;
        ms::GemmDesc g{};
        g.A = o + (size_t)r.r0 * d * e; g.W = r.w->w_o; g.bias = r.w->b_o;
        g.R = x + (size_t)r.r0 * d * e; g.C = h + (size_t)r.r0 * d * e;
        g.M = r.r1 - r.r0; g.N = d; g.K = d; g.lda = d; g.ldr = d; g.ldc = d;
        g.epilogue = ms::kEpiBiasResid;
        const LnAfter ln2{r.w->ln2_g, r.w->ln2_b, a + (size_t)r.r0 * d * e};
        MS_HIP(run_gemm(s, g, MS_K_GEMM_OUT, st, &ln2));
    }
    for (const Range& r : ranges) {
        if (r.r1 <= r.r0) continue;
        ms::GemmDesc g{};
        g.A = a + (size_t)r.r0 * d * e; g.W = r.w->w_1; g.bias = r.w->b_1;
        g.C = u + (size_t)r.r0 * f * e;
        g.M = r.r1 - r.r0; g.N = f; g.K = d; g.lda = d; g.ldc = f;
        g.epilogue = ms::kEpiBiasGelu;
        MS_HIP(run_gemm(s, g, MS_K_GEMM_UP, st));
    }
    for (const Range& r : ranges) {
        if (r.r1 <= r.r0) continue;
        ms::GemmDesc g{};
        g.A = u + (size_t)r.r0 * f * e; g.W = r.w->w_2; g.bias = r.w->b_2;
        g.R = h + (size_t)r.r0 * d * e; g.C = x + (size_t)r.r0 * d * e;
        g.M = r.r1 - r.r0; g.N = d; g.K = f; g.lda = f; g.ldr = d; g.ldc = d;
        g.epilogue = ms::kEpiBiasResidMlp;
        const LnAfter ln1{r.nw ? r.nw->ln1_g : nullptr, r.nw ? r.nw->ln1_b : nullptr, a + (size_t)r.r0 * d * e};
        MS_HIP(run_gemm(s, g, MS_K_GEMM_DOWN, st, r.nw ? &ln1 : nullptr));
    }
    return MS_OK;
}

// K/V of every row of a packing from its hidden rows x: LayerNorm 1 (unless `a_ready`:
// the scratch row buffer already holds it), then the K/V columns of the QKV
// projection, written to the rows' tokens in kv [B][T][2][d]; text rows with the
// text weight set.
ms_status kv_of_rows(ms_step* s, const Packing& pk, const ms_layer_weights* w, const void* x, void* kv,
                     hipStream_t st, bool a_ready) {
    if (pk.M == 0) return MS_OK;
    const bool dual = s->desc.dual_stream && s->desc.n_text > 0;
    const ms_layer_weights& wi = w[0];
    const ms_layer_weights& wt = dual ? w[1] : w[0];
    const int d = s->d, e = s->elt, msplit = pk.text_rows;
    char* a = static_cast<char*>(s->buf(s->lay.a));
    if (!a_ready) {
        ProfScope p(MS_K_LAYERNORM, st);
        MS_HIP(ms::launch_layernorm(s->desc.dtype, x, wi.ln1_g, wi.ln1_b, wt.ln1_g, wt.ln1_b, msplit, a, pk.M, d,
                                    s->desc.ln_eps, st));
    }
    struct Range { int r0, r1; const ms_layer_weights* w; };
    const Range ranges[2] = {{0, msplit, &wt}, {msplit, pk.M, &wi}};
    for (const Range& r : ranges) {
        if (r.r1 <= r.r0) continue;
        ms::GemmDesc g{};
        g.A = a + (size_t)r.r0 * d * e;
        g.W = static_cast<const char*>(r.w->w_qkv) + (size_t)d * d * e;
        g.bias = static_cast<const char*>(r.w->b_qkv) + (size_t)d * e;
        g.kv = kv; g.rows = pk.rows + r.r0;
        g.M = r.r1 - r.r0; g.N = 2 * d; g.K = d; g.lda = d; g.ldc = 2 * d; g.d = 0; g.kvld = 2 * d;
        g.epilogue = ms::kEpiQKV;
        MS_HIP(run_gemm(s, g, MS_K_GEMM_QKV, st));
    }
    return MS_OK;
}

// Y caching (Sec. 3.1, Fig. 5 bottom): K/V of the unmasked image tokens from
// their cached block input y_in [B][N][d]: LayerNorm of the gathered rows,
// then the K/V columns of the QKV projection, written to their token rows of
// the working K/V [B][T][2][d]. Image weights (unmasked tokens are image tokens).
ms_status recompute_kv(ms_step* s, const ms_layer_weights* w, const void* y_in, void* kv, hipStream_t st) {
    if (s->U == 0) return MS_OK;
    const int d = s->d, e = s->elt;
    void* a = s->buf(s->lay.u);
    {
        ProfScope p(MS_K_LAYERNORM, st);
        MS_HIP(ms::launch_layernorm(s->desc.dtype, y_in, w->ln1_g, w->ln1_b, w->ln1_g, w->ln1_b, 0, a, s->U, d,
                                    s->desc.ln_eps, st, s->at<int32_t>(s->lay.u_src)));
    }
    ms::GemmDesc g{};
    g.A = a;
    g.W = static_cast<const char*>(w->w_qkv) + (size_t)d * d * e;
    g.bias = static_cast<const char*>(w->b_qkv) + (size_t)d * e;
    g.kv = kv; g.rows = s->at<int32_t>(s->lay.u_tok);
    g.M = s->U; g.N = 2 * d; g.K = d; g.lda = d; g.ldc = 2 * d; g.d = 0; g.kvld = 2 * d;
    g.epilogue = ms::kEpiQKV;
    MS_HIP(run_gemm(s, g, MS_K_GEMM_QKV, st));
    return MS_OK;
}

// Loads the unmasked image rows of one block's cache from pinned host memory:
// K/V rows [B][N][2][d] -> slot [B][T][2][d] at n_text + n, or (y) block
// input rows [B][N][d] -> slot [B][N][d] in place.
// One layer's host cache: a [B][N][row] buffer, or (req non-NULL) request b's
// own [N][row] buffer at req[b].
struct HostLayer {
    const void* base;
    const void* const* req;
};

ms_status prefetch(ms_step* s, HostLayer h, void* d_slot, hipStream_t cs, hipEvent_t wait, bool y = false) {
    if (wait) MS_HIP(hipStreamWaitEvent(cs, wait, 0));
    ProfScope p(MS_K_COPY, cs);
    const size_t row_bytes = (y ? 1ull : 2ull) * s->d * s->elt;
    const size_t drows = y ? (size_t)s->N : (size_t)s->T, dtext = y ? 0 : (size_t)s->desc.n_text;
    char* dst = static_cast<char*>(d_slot);
    const size_t pitch = (size_t)s->desc.grid_w * row_bytes;   // one grid row, host and device alike
    for (const Span& sp : y ? s->spans_y : s->spans) {
        const ms::CopyRect& r = sp.r;
        const char* src = h.req ? static_cast<const char*>(h.req[sp.b]) + (size_t)r.n0 * row_bytes
                                : static_cast<const char*>(h.base) + ((size_t)sp.b * s->N + r.n0) * row_bytes;
        const size_t dof = ((size_t)sp.b * drows + dtext + r.n0) * row_bytes;
        if (r.h == 1)
            MS_HIP(hipMemcpyAsync(dst + dof, src, (size_t)r.w * row_bytes, hipMemcpyHostToDevice, cs));
        else
            MS_HIP(hipMemcpy2DAsync(dst + dof, pitch, src, pitch, (size_t)r.w * row_bytes, (size_t)r.h,
                                    hipMemcpyHostToDevice, cs));
    }
    return MS_OK;
}

ms_status prefetch_signal(ms_step* s, HostLayer h, void* d_slot, hipStream_t cs, hipEvent_t wait,
                          hipEvent_t signal, bool y = false) {
    ms_status st = prefetch(s, h, d_slot, cs, wait, y);
    if (st != MS_OK) return st;
    if (signal) MS_HIP(hipEventRecord(signal, cs));
    return MS_OK;
}

ms_status check_pinned(const void* p) {
    hipPointerAttribute_t attr;
    hipError_t e = hipPointerGetAttributes(&attr, p);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(MS_ENOTPINNED, "host K/V pointer is not pinned host memory (%s)", hipGetErrorString(e));
    }
    if (attr.type != hipMemoryTypeHost)
        return fail(MS_ENOTPINNED, "host K/V pointer is not pinned host memory (memory type %d)", (int)attr.type);
    return MS_OK;
}

}  // namespace

extern "C" {

int32_t mask_abi_version(void) { return kAbiVersion; }

const char* mask_last_error(void) { return g_err.c_str(); }

size_t mask_workspace_bytes(const ms_model_desc* desc, int32_t batch) {
    if (validate_desc(desc) != MS_OK) return 0;
    if (batch < 1 || batch > desc->max_batch) {
        fail(MS_ESHAPE, "batch %d outside 1..max_batch", batch);
        return 0;
    }
    g_err.clear();
    return make_layout(*desc, batch).total;
}

ms_status mask_step_init(ms_step** out, const ms_model_desc* desc, int32_t batch,
                         const uint8_t* d_mask, void* d_ws, size_t ws_bytes, void* stream) {
    return ms::step_init(out, desc, batch, d_mask, d_ws, ws_bytes, stream, -1);
}

}  // extern "C"

namespace ms {

ms_status set_error(ms_status st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return st;
}

ms_status clear_error() {
    g_err.clear();
    return MS_OK;
}

ms_status workspace_need(const ms_model_desc* desc, int32_t batch, size_t* need) {
    ms_status st = validate_desc(desc);
    if (st != MS_OK) return st;
    if (batch < 1 || batch > desc->max_batch) return fail(MS_ESHAPE, "batch %d outside 1..max_batch", batch);
    *need = make_layout(*desc, batch).total;
    return MS_OK;
}

ms_status step_init(ms_step** out, const ms_model_desc* desc, int32_t batch, const uint8_t* d_mask,
                    void* d_ws, size_t ws_bytes, void* stream, int static_dev) {
    if (!out) return fail(MS_EINVAL, "out is NULL");
    *out = nullptr;
    ms_status st = validate_desc(desc);
    if (st != MS_OK) return st;
    if (batch < 1 || batch > desc->max_batch) return fail(MS_ESHAPE, "batch %d outside 1..max_batch", batch);
    if (!d_mask || !d_ws) return fail(MS_EINVAL, "mask or workspace is NULL");
    if (!aligned16(d_ws)) return fail(MS_EALIGN, "workspace not 16-byte aligned");
    const Layout lay = make_layout(*desc, batch);
    if (ws_bytes < lay.total)
        return fail(MS_EWORKSPACE, "workspace %zu bytes < %zu required", ws_bytes, lay.total);

    ms_step* s = new (std::nothrow) ms_step();
    if (!s) return fail(MS_EINVAL, "out of host memory");
    s->desc = *desc;
    s->B = batch;
    s->N = desc->grid_h * desc->grid_w;
    s->T = desc->n_text + s->N;
    s->d = desc->d_model;
    s->f = desc->mlp_mult * desc->d_model;
    s->hd = desc->d_model / desc->n_heads;
    s->elt = elt_bytes(desc->dtype);
    s->ws = static_cast<char*>(d_ws);
    s->lay = lay;
    s->static_dev = static_dev;
    const bool split = desc->dual_stream && desc->n_text > 0;
    Packing& p = s->mp;
    p.rows = s->at<int32_t>(lay.rows);
    p.inv = s->at<int32_t>(lay.inv);
    p.segs = s->at<int32_t>(lay.seg_start);
    p.segreq = s->at<int32_t>(lay.seg_req);
    p.cutiles = s->at<int32_t>(lay.cu_tiles);
    p.nseg = split ? 2 * batch : batch;
    p.text_rows = split ? batch * desc->n_text : 0;

    hipStream_t hs = static_cast<hipStream_t>(stream);
    // on failure the caller keeps ownership of a static scratch (static_dev)
    auto bail = [&](ms_status code) { destroy_events(s); delete s; return code; };
    hipError_t e;
    {
        ProfScope prof(MS_K_COMPACT, hs);
        e = ms::launch_compact(d_mask, batch, s->N, desc->n_text, split ? 1 : 0, p.rows, p.inv,
                               p.segs, p.segreq, p.cutiles, hs);
    }
    if (e != hipSuccess) return bail(fail(MS_EHIP, "compaction launch: %s", hipGetErrorString(e)));
    p.seg_start.assign(p.nseg + 1, 0);
    std::vector<uint8_t> hmask((size_t)batch * s->N);
    e = hipMemcpyAsync(p.seg_start.data(), p.segs, (p.nseg + 1) * sizeof(int32_t),
                       hipMemcpyDeviceToHost, hs);
    if (e == hipSuccess)
        e = hipMemcpyAsync(hmask.data(), d_mask, hmask.size(), hipMemcpyDeviceToHost, hs);
    if (e == hipSuccess) e = hipStreamSynchronize(hs);
    if (e != hipSuccess) return bail(fail(MS_EHIP, "compaction readback: %s", hipGetErrorString(e)));
    finish_packing(p, *desc, batch, s->T, s->hd);
    s->all_masked = p.M == batch * s->T;
    plan_spans(s, hmask);
    for (int b = 0; b < batch; ++b) {
        if (!request_recomputes(s, hmask.data() + (size_t)b * s->N)) continue;
        for (int n = 0; n < s->N; ++n)
            if (!hmask[(size_t)b * s->N + n]) {
                s->h_usrc.push_back(b * s->N + n);
                s->h_utok.push_back(b * s->T + desc->n_text + n);
            }
    }
    s->U = (int)s->h_usrc.size();
    if (s->U > 0) {
        e = hipMemcpyAsync(s->buf(lay.u_src), s->h_usrc.data(), s->U * sizeof(int32_t), hipMemcpyHostToDevice, hs);
        if (e == hipSuccess)
            e = hipMemcpyAsync(s->buf(lay.u_tok), s->h_utok.data(), s->U * sizeof(int32_t), hipMemcpyHostToDevice, hs);
        if (e != hipSuccess) return bail(fail(MS_EHIP, "unmasked-row upload: %s", hipGetErrorString(e)));
    }
    *out = s;
    return ok();
}

}  // namespace ms

extern "C" {

ms_status mask_step_get_info(const ms_step* s, ms_step_info* info) {
    if (!s || !info) return fail(MS_EINVAL, "NULL argument");
    info->batch = s->B;
    info->rows = s->mp.M;
    info->n_segments = s->mp.nseg;
    info->n_qtiles = s->mp.n_qtiles;
    info->text_rows = s->mp.text_rows;
    info->dense_prefix = s->dense_prefix;
    info->copy_spans = (int32_t)s->spans.size();
    info->copy_spans_y = (int32_t)s->spans_y.size();
    info->copy_rows = info->copy_rows_y = 0;
    for (const Span& sp : s->spans) info->copy_rows += (int64_t)sp.r.w * sp.r.h;
    for (const Span& sp : s->spans_y) info->copy_rows_y += (int64_t)sp.r.w * sp.r.h;
    return ok();
}

ms_status mask_step_index(const ms_step* s, const int32_t** d_rows, const int32_t** d_inv,
                          const int32_t** d_seg_start) {
    if (!s) return fail(MS_ESTATE, "no step context");
    if (d_rows) *d_rows = s->mp.rows;
    if (d_inv) *d_inv = s->mp.inv;
    if (d_seg_start) *d_seg_start = s->mp.segs;
    return ok();
}

ms_status mask_step_set_dense_prefix(ms_step* s, int32_t k, void* stream) {
    if (!s) return fail(MS_ESTATE, "no step context");
    if (k < 0 || k > s->desc.n_layers) return fail(MS_EINVAL, "dense prefix %d outside 0..n_layers", k);
    if (k > 0) {
        ms_status st = build_dense_packing(s, static_cast<hipStream_t>(stream));
        if (st != MS_OK) return st;
    }
    s->dense_prefix = k;
    return ok();
}

namespace {
// Alg. 1's clocks for the choice "first k blocks over every token, the rest with the cache":
// a full block needs no load (comp += full); a cached block's load follows the previous load
// and its compute waits for it (comp = max(load, comp) + cached). Smallest k on ties.
void plan_prefix(int32_t n_layers, double load_ms, double cached_ms, double full_ms, int32_t* k_out,
                 double* latency_out) {
    int best_k = 0;
    double best = 0.0;
    for (int k = 0; k <= n_layers; ++k) {
        double comp = 0.0, load = 0.0;
        for (int i = 0; i < n_layers; ++i) {
            if (i < k) {
                comp += full_ms;
            } else {
                load += load_ms;
                comp = std::max(load, comp) + cached_ms;
            }
        }
        if (k == 0 || comp < best - 1e-12) {
            best = comp;
            best_k = k;
        }
    }
    *k_out = best_k;
    *latency_out = best;
}

// Algorithmic FLOPs of one block for `rows` recomputed rows of a request (Table 1): the
// projections and the feed-forward (2 rows d^2 (4 + 2 mlp_mult)) and QK^T and PV over every
// token (4 rows T d). Exact in double for every model the library accepts.
double block_flops(const ms_model_desc& d, int64_t rows) {
    const double D = d.d_model;
    const double T = (double)d.n_text + (double)d.grid_h * d.grid_w;
    return 2.0 * (double)rows * D * D * (4 + 2 * d.mlp_mult) + 4.0 * (double)rows * T * D;
}

bool finite_nonneg(double v) { return std::isfinite(v) && v >= 0.0; }

ms_status check_cost_inputs(const ms_model_desc* desc, const ms_cost_model* m) {
    if (!desc || !m) return fail(MS_EINVAL, "model description or cost model is NULL");
    ms_model_desc d = *desc;
    d.max_batch = 1;   // not used by the cost model
    const ms_status st = validate_desc(&d);
    if (st != MS_OK) return st;
    if (!finite_nonneg(m->comp_ms0) || !finite_nonneg(m->comp_ms_per_gflop) || !finite_nonneg(m->load_ms0) ||
        !finite_nonneg(m->load_ms_per_mb) || !finite_nonneg(m->cache_bytes_per_token))
        return fail(MS_EINVAL, "cost model fields must be finite and >= 0");
    return MS_OK;
}

// (L, C_w, C_wo) of one block for a validated batch
void batch_block_costs(const ms_model_desc& d, const ms_cost_model& m, const int32_t* masked, int32_t n,
                       double out[3]) {
    const int32_t N = d.grid_h * d.grid_w;
    const int64_t T = (int64_t)d.n_text + N;
    double f_cached = 0.0, nbytes = 0.0;
    for (int32_t b = 0; b < n; ++b) {
        f_cached += block_flops(d, (int64_t)masked[b] + d.n_text);
        nbytes += (double)(N - masked[b]) * m.cache_bytes_per_token;
    }
    const double f_full = (double)n * block_flops(d, T);
    out[0] = nbytes == 0.0 ? 0.0 : m.load_ms0 + m.load_ms_per_mb * nbytes / 1e6;
    out[1] = f_cached == 0.0 ? 0.0 : m.comp_ms0 + m.comp_ms_per_gflop * f_cached / 1e9;
    out[2] = f_full == 0.0 ? 0.0 : m.comp_ms0 + m.comp_ms_per_gflop * f_full / 1e9;
}

double batch_latency(const ms_model_desc& d, const ms_cost_model& m, const int32_t* masked, int32_t n,
                     double costs[3], int32_t* k) {
    costs[0] = costs[1] = costs[2] = 0.0;
    *k = 0;
    if (n == 0) return 0.0;
    batch_block_costs(d, m, masked, n, costs);
    double lat = 0.0;
    plan_prefix(d.n_layers, costs[0], costs[1], costs[2], k, &lat);
    return lat;
}
}  // namespace

ms_status mask_plan_dense_prefix(int32_t n_layers, double load_ms, double cached_ms, double full_ms,
                                 int32_t* k_out, double* latency_ms_out) {
    if (n_layers < 1 || !k_out) return fail(MS_EINVAL, "need n_layers >= 1 and k_out");
    if (!(load_ms >= 0) || !(cached_ms >= 0) || !(full_ms >= 0)) return fail(MS_EINVAL, "negative or NaN cost");
    double lat = 0.0;
    plan_prefix(n_layers, load_ms, cached_ms, full_ms, k_out, &lat);
    if (latency_ms_out) *latency_ms_out = lat;
    return ok();
}

ms_status mask_plan_copies(const uint8_t* mask, int32_t grid_h, int32_t grid_w, double copy_cost_rows,
                           int32_t* out, int32_t cap, int32_t* n_out) {
    if (!mask || !n_out) return fail(MS_EINVAL, "mask and n_out must be non-NULL");
    if (grid_h < 1 || grid_w < 1 || (int64_t)grid_h * grid_w > (1 << 20))
        return fail(MS_ESHAPE, "grid %d x %d: need 1 .. 2^20 image tokens", grid_h, grid_w);
    if (!(copy_cost_rows >= 0.0) || !std::isfinite(copy_cost_rows))
        return fail(MS_EINVAL, "copy_cost_rows must be finite and >= 0");
    if (cap < 0 || (cap > 0 && !out)) return fail(MS_EINVAL, "need cap >= 0 and out when cap > 0");
    std::vector<ms::CopyRect> rects;
    ms::plan_copies(mask, grid_h, grid_w, copy_cost_rows, true, rects);
    *n_out = (int32_t)rects.size();
    if ((int64_t)rects.size() > cap) return fail(MS_ESHAPE, "the plan has %d copies, cap is %d", *n_out, cap);
    for (size_t i = 0; i < rects.size(); ++i) {
        out[3 * i] = rects[i].n0;
        out[3 * i + 1] = rects[i].w;
        out[3 * i + 2] = rects[i].h;
    }
    return ok();
}

ms_status mask_fit_linear(const double* x, const double* y, int32_t n, double* intercept_out, double* slope_out,
                          double* r2_out) {
    if (!x || !y || !intercept_out || !slope_out) return fail(MS_EINVAL, "x, y and the outputs must be non-NULL");
    if (n < 2) return fail(MS_EINVAL, "need at least two points, got %d", n);
    double xm = 0.0, ym = 0.0;
    for (int32_t i = 0; i < n; ++i) {
        if (!std::isfinite(x[i]) || !std::isfinite(y[i])) return fail(MS_EINVAL, "point %d is not finite", i);
        xm += x[i];
        ym += y[i];
    }
    xm /= n;
    ym /= n;
    double sxx = 0.0, sxy = 0.0;
    for (int32_t i = 0; i < n; ++i) {
        sxx += (x[i] - xm) * (x[i] - xm);
        sxy += (x[i] - xm) * (y[i] - ym);
    }
    if (!(sxx > 0.0)) return fail(MS_EINVAL, "x has no spread");
    const double slope = sxy / sxx;
    const double intercept = ym - slope * xm;
    double ss_res = 0.0, ss_tot = 0.0;
    for (int32_t i = 0; i < n; ++i) {
        const double r = y[i] - (intercept + slope * x[i]);
        ss_res += r * r;
        ss_tot += (y[i] - ym) * (y[i] - ym);
    }
    *intercept_out = intercept;
    *slope_out = slope;
    if (r2_out) *r2_out = ss_tot > 0.0 ? 1.0 - ss_res / ss_tot : (ss_res == 0.0 ? 1.0 : 0.0);
    return ok();
}

ms_status mask_batch_cost(const ms_model_desc* desc, const ms_cost_model* model, const int32_t* masked,
                          int32_t batch, double* costs_out, int32_t* k_out, double* latency_ms_out) {
    ms_status st = check_cost_inputs(desc, model);
    if (st != MS_OK) return st;
    if (batch < 0 || (batch > 0 && !masked)) return fail(MS_EINVAL, "need batch >= 0 and masked[batch]");
    const int32_t N = desc->grid_h * desc->grid_w;
    for (int32_t b = 0; b < batch; ++b)
        if (masked[b] < 0 || masked[b] > N) return fail(MS_EINVAL, "masked[%d] = %d outside 0..%d", b, masked[b], N);
    double costs[3];
    int32_t k = 0;
    const double lat = batch_latency(*desc, *model, masked, batch, costs, &k);
    if (costs_out) std::memcpy(costs_out, costs, sizeof costs);
    if (k_out) *k_out = k;
    if (latency_ms_out) *latency_ms_out = lat;
    return ok();
}

ms_status mask_route_request(const ms_model_desc* desc, const ms_cost_model* model, const int32_t* running_masked,
                             const int32_t* batch_sizes, int32_t n_workers, int32_t max_batch, int32_t request_masked,
                             int32_t* worker_out, double* cost_ms_out) {
    ms_status st = check_cost_inputs(desc, model);
    if (st != MS_OK) return st;
    if (!worker_out) return fail(MS_EINVAL, "worker_out is NULL");
    if (n_workers < 0 || (n_workers > 0 && !batch_sizes)) return fail(MS_EINVAL, "need n_workers >= 0 and batch_sizes");
    if (max_batch < 1) return fail(MS_EINVAL, "max_batch must be >= 1");
    const int32_t N = desc->grid_h * desc->grid_w;
    if (request_masked < 0 || request_masked > N)
        return fail(MS_EINVAL, "request masked count %d outside 0..%d", request_masked, N);
    int64_t total = 0;
    for (int32_t w = 0; w < n_workers; ++w) {
        if (batch_sizes[w] < 0) return fail(MS_EINVAL, "batch_sizes[%d] < 0", w);
        total += batch_sizes[w];
    }
    if (total > 0 && !running_masked) return fail(MS_EINVAL, "running_masked is NULL");
    for (int64_t i = 0; i < total; ++i)
        if (running_masked[i] < 0 || running_masked[i] > N)
            return fail(MS_EINVAL, "running_masked[%lld] outside 0..%d", (long long)i, N);
    int32_t best = -1;
    double best_cost = 0.0;
    std::vector<int32_t> batch;
    int64_t off = 0;
    for (int32_t w = 0; w < n_workers; ++w) {
        const int32_t nb = batch_sizes[w];
        if (nb < max_batch) {
            batch.assign(running_masked + off, running_masked + off + nb);
            batch.push_back(request_masked);
            double costs[3];
            int32_t k = 0;
            const double c = batch_latency(*desc, *model, batch.data(), (int32_t)batch.size(), costs, &k);
            if (best < 0 || c < best_cost) {
                best = w;
                best_cost = c;
            }
        }
        off += nb;
    }
    *worker_out = best;
    if (cost_ms_out) *cost_ms_out = best < 0 ? 0.0 : best_cost;
    return ok();
}

ms_status mask_gather_rows(ms_step* s, const void* d_x, void* d_xm, void* stream) {
    if (!s) return fail(MS_ESTATE, "no step context");
    if (!d_x) return fail(MS_EINVAL, "x is NULL");
    void* xm = d_xm ? d_xm : s->buf(s->lay.xm);
    if (!aligned16(d_x) || !aligned16(xm)) return fail(MS_EALIGN, "x / xm not 16-byte aligned");
    ProfScope p(MS_K_GATHER, static_cast<hipStream_t>(stream));
    MS_HIP(ms::launch_gather(d_x, s->mp.rows, xm, s->mp.M, s->d * s->elt, static_cast<hipStream_t>(stream)));
    return ok();
}

ms_status mask_block_forward(ms_step* s, int32_t layer, const ms_layer_weights* w, void* d_xm,
                             void* d_kv, void* stream) {
    if (!s) return fail(MS_ESTATE, "no step context");
    forget_rings();
    if (layer < 0 || layer >= s->desc.n_layers) return fail(MS_EINVAL, "layer %d out of range", layer);
    if (!w || !d_kv) return fail(MS_EINVAL, "weights or kv is NULL");
    void* xm = d_xm ? d_xm : s->buf(s->lay.xm);
    if (!aligned16(xm) || !aligned16(d_kv)) return fail(MS_EALIGN, "xm / kv not 16-byte aligned");
    ms_status st = check_weights(s, w);
    if (st != MS_OK) return st;
    st = block_forward(s, s->mp, w, xm, d_kv, static_cast<hipStream_t>(stream));
    return st == MS_OK ? ok() : st;
}

ms_status mask_scatter_rows(ms_step* s, const void* d_xm, const void* d_ycache, void* d_y,
                            void* stream) {
    if (!s) return fail(MS_ESTATE, "no step context");
    if (!d_y) return fail(MS_EINVAL, "y is NULL");
    if (!d_ycache && !s->all_masked) return fail(MS_EINVAL, "y_cache may be NULL only when every token is masked");
    const void* xm = d_xm ? d_xm : s->buf(s->lay.xm);
    if (!aligned16(d_y) || !aligned16(xm) || !aligned16(d_ycache)) return fail(MS_EALIGN, "pointer not 16-byte aligned");
    ProfScope p(MS_K_SCATTER, static_cast<hipStream_t>(stream));
    MS_HIP(ms::launch_scatter(xm, s->mp.rows, s->mp.inv, d_ycache, d_y, s->mp.M, s->B * s->T,
                              s->d * s->elt, static_cast<hipStream_t>(stream)));
    return ok();
}

ms_status cache_prefetch_layer(ms_step* s, int32_t layer, const void* h_kv, void* d_slot,
                               void* copy_stream, void* wait_event, void* signal_event) {
    if (!s) return fail(MS_ESTATE, "no step context");
    forget_rings();
    if (layer < 0 || layer >= s->desc.n_layers) return fail(MS_EINVAL, "layer %d out of range", layer);
    if (!h_kv || !d_slot) return fail(MS_EINVAL, "h_kv or slot is NULL");
    if (!aligned16(h_kv) || !aligned16(d_slot)) return fail(MS_EALIGN, "h_kv / slot not 16-byte aligned");
    ms_status st = check_pinned(h_kv);
    if (st != MS_OK) return st;
    st = prefetch_signal(s, HostLayer{h_kv, nullptr}, d_slot, static_cast<hipStream_t>(copy_stream),
                         static_cast<hipEvent_t>(wait_event), static_cast<hipEvent_t>(signal_event));
    return st == MS_OK ? ok() : st;
}

ms_status cache_prefetch_inputs(ms_step* s, int32_t layer, const void* h_yin, void* d_slot,
                                void* copy_stream, void* wait_event, void* signal_event) {
    if (!s) return fail(MS_ESTATE, "no step context");
    forget_rings();
    if (layer < 0 || layer >= s->desc.n_layers) return fail(MS_EINVAL, "layer %d out of range", layer);
    if (!h_yin || !d_slot) return fail(MS_EINVAL, "h_yin or slot is NULL");
    if (!aligned16(h_yin) || !aligned16(d_slot)) return fail(MS_EALIGN, "h_yin / slot not 16-byte aligned");
    ms_status st = check_pinned(h_yin);
    if (st != MS_OK) return st;
    st = prefetch_signal(s, HostLayer{h_yin, nullptr}, d_slot, static_cast<hipStream_t>(copy_stream),
                         static_cast<hipEvent_t>(wait_event), static_cast<hipEvent_t>(signal_event), true);
    return st == MS_OK ? ok() : st;
}

ms_status mask_recompute_kv(ms_step* s, int32_t layer, const ms_layer_weights* w, const void* d_yin,
                            void* d_kv, void* stream) {
    if (!s) return fail(MS_ESTATE, "no step context");
    forget_rings();
    if (layer < 0 || layer >= s->desc.n_layers) return fail(MS_EINVAL, "layer %d out of range", layer);
    if (!w || !d_kv || (!d_yin && s->U > 0)) return fail(MS_EINVAL, "NULL argument");
    if (!aligned16(d_yin) || !aligned16(d_kv)) return fail(MS_EALIGN, "pointer not 16-byte aligned");
    ms_status st = check_weights(s, w);
    if (st != MS_OK) return st;
    st = recompute_kv(s, w, d_yin, d_kv, static_cast<hipStream_t>(stream));
    return st == MS_OK ? ok() : st;
}

ms_status mask_stack_forward(ms_step* s, const ms_layer_weights* w, const void* d_x,
                             const void* d_ycache, const ms_kv_source* kv, void* d_y,
                             void* compute_stream, void* copy_stream) {
    if (!s) return fail(MS_ESTATE, "no step context");
    if (!w || !d_x || !kv || !d_y) return fail(MS_EINVAL, "NULL argument");
    if (!d_ycache && !s->all_masked) return fail(MS_EINVAL, "y_cache may be NULL only when every token is masked");
    if (kv->kind < MS_KV_DEVICE || kv->kind > MS_Y_HOST_PINNED) return fail(MS_EINVAL, "unknown kv kind %d", kv->kind);
    const bool ycache = kv->kind == MS_Y_DEVICE || kv->kind == MS_Y_HOST_PINNED;
    const bool pinned = kv->kind == MS_KV_HOST_PINNED || kv->kind == MS_Y_HOST_PINNED;
    const bool per_req = pinned && kv->request_layer;
    if (!per_req && !kv->layer) return fail(MS_EINVAL, "kv->layer is NULL");
    const int L = s->desc.n_layers;
    const int k = s->dense_prefix;
    const int wstride = s->desc.dual_stream ? 2 : 1;
    // requests whose cache is read (those with spans) need a valid host pointer per layer
    std::vector<uint8_t> reads(s->B, 0);
    for (const Span& sp : s->spans) reads[sp.b] = 1;
    for (int l = 0; l < L; ++l) {
        if (per_req) {
            for (int b = 0; b < s->B; ++b) {
                const void* q = kv->request_layer[(size_t)l * s->B + b];
                if (!reads[b]) continue;
                if (!q) return fail(MS_EINVAL, "kv->request_layer[%d * B + %d] is NULL", l, b);
                if (!aligned16(q)) return fail(MS_EALIGN, "kv->request_layer[%d * B + %d] not 16-byte aligned", l, b);
            }
        } else {
            if (!kv->layer[l]) return fail(MS_EINVAL, "kv->layer[%d] is NULL", l);
            if (!aligned16(kv->layer[l])) return fail(MS_EALIGN, "kv->layer[%d] not 16-byte aligned", l);
        }
        ms_status st = check_weights(s, w + (size_t)l * wstride);
        if (st != MS_OK) return st;
    }
    auto host_layer = [&](int l) {
        return per_req ? HostLayer{nullptr, kv->request_layer + (size_t)l * s->B} : HostLayer{kv->layer[l], nullptr};
    };
    const int n_slots = pinned ? kv->n_slots : 0;
    const uint64_t call_id = ++g_stack_calls;
    // this call's load-landed events: alternate sets, so that no event is recorded again while
    // a wait of the previous call on it may still be pending
    const int ecp = (int)(s->stack_calls++ & 1) * (pinned ? kv->n_slots : 0);
    if (pinned) {
        if (n_slots < 1 || !kv->slots) return fail(MS_EINVAL, "a pinned cache needs n_slots >= 1 device slots");
        for (int i = 0; i < n_slots; ++i) {
            if (!kv->slots[i]) return fail(MS_EINVAL, "kv->slots[%d] is NULL", i);
            if (!aligned16(kv->slots[i])) return fail(MS_EALIGN, "kv->slots[%d] not 16-byte aligned", i);
        }
        if (!s->all_masked && s->mp.M > 0 && k < L) {
            for (int b = 0; b < (per_req ? s->B : 1); ++b) {
                if (per_req && !reads[b]) continue;
                ms_status st = check_pinned(per_req ? kv->request_layer[(size_t)k * s->B + b] : kv->layer[k]);
                if (st != MS_OK) return st;
            }
        }
        ms_status st = ensure_events(s, 2 * n_slots);
        if (st != MS_OK) return st;
    }
    if (!aligned16(d_x) || !aligned16(d_y) || !aligned16(d_ycache)) return fail(MS_EALIGN, "pointer not 16-byte aligned");

    hipStream_t cs = static_cast<hipStream_t>(compute_stream);
    hipStream_t ps = static_cast<hipStream_t>(copy_stream);
    void* xm = s->buf(s->lay.xm);
    const Packing& mp = s->mp;
    if (mp.M > 0) {
        const int n_cached = L - k;
        const bool stream_cache = pinned && !s->all_masked && n_cached > 0;
        const bool serialize = stream_cache && (env_flag("MS_SERIALIZE") || ps == cs);
        const bool pipelined = stream_cache && !serialize;
        const bool poison = env_flag("MS_POISON");
        // Loads of the cached layers on the copy stream. Load j goes to slot j % n_slots and may
        // be issued once the cached block that used that slot before (j - n_slots) is launched;
        // the issue is spread over the block launches so the first kernels go out early (the
        // host stays far ahead of both streams either way).
        int issued = 0, launched = 0;
        auto allowed = [&]() { return std::min(n_cached, launched + n_slots); };
        // the copy stream must not overwrite a slot an earlier call still reads: wait for the
        // ring's release by the last call that streamed through it, else for this call's start
        RingRelease* ring = nullptr;
        uint64_t ring_gen = 0;
        int prev_h = 0;
        bool prev_known = false;
        // Under stream capture the release points of eager calls mean nothing to the replays
        // (and the replays' records are not seen here): a captured call orders its loads after
        // its own start, and the next call does the same.
        hipStreamCaptureStatus capture = hipStreamCaptureStatusNone;
        MS_HIP(hipStreamIsCapturing(cs, &capture));
        const bool capturing = capture != hipStreamCaptureStatusNone;
        if (stream_cache) {
            ms_status st = ring_release(kv, &ring, &ring_gen);
            if (st != MS_OK) return st;
            std::lock_guard<std::mutex> lk(g_ring_mu);
            // only right after the call that released the ring: a call in between
            // (a step that streams nothing) would otherwise run under the loads
            prev_known = (kv->flags & MS_KV_LOADS_AHEAD) && !capturing && ring->gen == ring_gen && ring->recorded &&
                         ring->call + 1 == call_id;
            prev_h = ring->h;
            if (capturing) ring->recorded = false;
        }
        auto issue_upto = [&](int limit) -> ms_status {
            for (; issued < limit; ++issued) {
                const int sl = issued % n_slots;
                hipEvent_t wait = issued >= n_slots ? s->ev_consumed[sl] : nullptr;
                const int pp = (int)((call_id - 1) & 1);   // the previous call's event set
                if (prev_known && issued == 0) wait = prev_h > 0 ? ring->half[pp] : ring->all[pp];
                else if (prev_known && issued == prev_h && prev_h > 0) wait = ring->all[pp];
                ms_status st = prefetch_signal(s, host_layer(k + issued), kv->slots[sl], ps, wait, s->ev_copied[ecp + sl],
                                               ycache);
                if (st != MS_OK) return st;
            }
            return MS_OK;
        };
        if (pipelined) {
            if (!prev_known) {
                MS_HIP(hipEventRecord(s->ev_start, cs));
                MS_HIP(hipStreamWaitEvent(ps, s->ev_start, 0));
            }
            ms_status st = issue_upto(std::min(allowed(), 2));
            if (st != MS_OK) return st;
        }
        // this call's release points: slots [0, h) after block h - 1, all after the last
        const int my_h = n_cached <= n_slots ? (n_cached + 1) / 2 : 0;
        bool first_ln_ready = false;   // LayerNorm 1 of block k already in the scratch rows
        if (k > 0) {
            // dense prefix, no cache read: blocks [0, k-1) over every token. Block k-1 needs every
            // token only for its K/V (block k reads the cache, and the step's output takes the
            // unmasked rows from the cached state), so it projects K/V over every token and runs
            // the rest of the block over the masked rows.
            const Packing& dp = s->dp;
            void* kvd = s->buf(s->lay.kv_dense);
            {
                ProfScope p(MS_K_GATHER, cs);
                MS_HIP(ms::launch_gather(d_x, dp.rows, xm, dp.M, s->d * s->elt, cs));
            }
            for (int l = 0; l < k - 1; ++l) {
                ms_status st = block_forward(s, dp, w + (size_t)l * wstride, xm, kvd, cs, w + (size_t)(l + 1) * wstride,
                                             l > 0);
                if (st != MS_OK) return st;
                if (pipelined && (st = issue_upto(std::min(allowed(), issued + 2))) != MS_OK) return st;
            }
            const ms_layer_weights* wl = w + (size_t)(k - 1) * wstride;
            ms_status st = kv_of_rows(s, dp, wl, xm, kvd, cs, k > 1);
            if (st != MS_OK) return st;
            // hidden states of every token back in token order, then the masked rows
            void* flat = s->buf(s->lay.o);
            {
                ProfScope p(MS_K_SCATTER, cs);
                MS_HIP(ms::launch_scatter(xm, dp.rows, dp.inv, flat, flat, dp.M, s->B * s->T,
                                          s->d * s->elt, cs));
            }
            {
                ProfScope p(MS_K_GATHER, cs);
                MS_HIP(ms::launch_gather(flat, mp.rows, xm, mp.M, s->d * s->elt, cs));
            }
            const ms_layer_weights* next = k < L ? w + (size_t)k * wstride : nullptr;
            st = block_forward(s, mp, wl, xm, kvd, cs, next, false);
            if (st != MS_OK) return st;
            if (pipelined && (st = issue_upto(std::min(allowed(), issued + 2))) != MS_OK) return st;
            first_ln_ready = next != nullptr;
        } else {
            ProfScope p(MS_K_GATHER, cs);
            MS_HIP(ms::launch_gather(d_x, mp.rows, xm, mp.M, s->d * s->elt, cs));
        }
        for (int l = k; l < L; ++l) {
            const int j = l - k;
            void* src = pinned ? nullptr : const_cast<void*>(kv->layer[l]);
            if (pinned) {
                src = kv->slots[j % n_slots];
                if (serialize) {
                    ms_status st = prefetch(s, host_layer(l), src, cs, nullptr, ycache);
                    if (st != MS_OK) return st;
                } else if (stream_cache) {
                    ms_status st = issue_upto(allowed());   // includes load j
                    if (st != MS_OK) return st;
                    MS_HIP(hipStreamWaitEvent(cs, s->ev_copied[ecp + j % n_slots], 0));
                }
            }
            // K/V variant: the cache is the working K/V; Y variant: the unmasked
            // K/V are recomputed from the cached block input into the workspace
            void* kvbuf = src;
            if (ycache) {
                kvbuf = s->buf(s->lay.kv_dense);
                ms_status st = recompute_kv(s, w + (size_t)l * wstride, src, kvbuf, cs);
                if (st != MS_OK) return st;
            }
            const ms_layer_weights* next = l + 1 < L ? w + (size_t)(l + 1) * wstride : nullptr;
            ms_status st = block_forward(s, mp, w + (size_t)l * wstride, xm, kvbuf, cs, next, l > k || first_ln_ready);
            if (st != MS_OK) return st;
            if (pinned && poison) {
                // debugging mode: the slot's contents die with its block; a later block that read a
                // row its own load or fresh K/V did not write would see NaN
                const size_t slot_bytes = (size_t)s->B * (ycache ? s->N : s->T) * (ycache ? 1 : 2) * s->d * s->elt;
                MS_HIP(ms::launch_fill_u8(src, 0xFF, slot_bytes, cs));
            }
            if (stream_cache && !capturing && (j + 1 == my_h || j + 1 == n_cached)) {
                std::lock_guard<std::mutex> lk(g_ring_mu);
                // unless another slot list has taken the entry over meanwhile
                if (ring->gen == ring_gen) {
                    if (j + 1 == my_h) MS_HIP(hipEventRecord(ring->half[call_id & 1], cs));
                    if (j + 1 == n_cached) {
                        MS_HIP(hipEventRecord(ring->all[call_id & 1], cs));
                        ring->h = my_h;
                        ring->recorded = true;
                        ring->call = call_id;
                    }
                }
            }
            if (pipelined) {
                if (j + n_slots < n_cached) MS_HIP(hipEventRecord(s->ev_consumed[j % n_slots], cs));
                launched = j + 1;
                if ((st = issue_upto(allowed())) != MS_OK) return st;
            }
        }
    }
    {
        ProfScope p(MS_K_SCATTER, cs);
        MS_HIP(ms::launch_scatter(xm, mp.rows, mp.inv, d_ycache, d_y, mp.M, s->B * s->T,
                                  s->d * s->elt, cs));
    }
    return ok();
}

void mask_step_destroy(ms_step* s) {
    if (!s) return;
    destroy_events(s);
    if (s->static_dev >= 0) ms::release_static_scratch(s->static_dev);
    delete s;
}

ms_status ms_linear(int32_t dtype, int32_t M, int32_t N, int32_t K, const void* A, const void* W,
                    const void* bias, const void* resid, void* out, int32_t epilogue,
                    int32_t tile_m, int32_t tile_n, int32_t ksplit, void* d_ws, size_t ws_bytes,
                    void* stream) {
    if (dtype != MS_FP32 && dtype != MS_BF16) return fail(MS_EDTYPE, "unknown dtype %d", dtype);
    if (M < 0 || N < 4 || K < 1 || N % 4) return fail(MS_ESHAPE, "need M >= 0, N a positive multiple of 4");
    const int bk = dtype == MS_BF16 ? 64 : 32;
    if (K % bk) return fail(MS_ESHAPE, "K must be a multiple of %d", bk);
    // the bf16 kernels address a tile's rows (up to 256 x K) with 32-bit buffer offsets
    if (dtype == MS_BF16 && (int64_t)K * 2 * 256 >= (1ll << 32)) return fail(MS_ESHAPE, "K must be below 2^23");
    if (epilogue < MS_EPI_BIAS || epilogue > MS_EPI_BIAS_GELU) return fail(MS_EINVAL, "unknown epilogue %d", epilogue);
    if (!A || !W || !bias || !out || (epilogue == MS_EPI_BIAS_RESID && !resid))
        return fail(MS_EINVAL, "NULL operand");
    if (!aligned16(A) || !aligned16(W) || !aligned16(bias) || !aligned16(out) || !aligned16(resid) ||
        !aligned16(d_ws))
        return fail(MS_EALIGN, "operand not 16-byte aligned");
    if (ksplit < 0) return fail(MS_EINVAL, "ksplit must be >= 0");
    ms::GemmPlan p = ms::plan_gemm(dtype, M, N, K, d_ws ? ws_bytes / 4 : 0);
    if (tile_m || tile_n) {
        const int ok_tiles[8][2] = {{256, 256}, {256, 192}, {192, 192}, {256, 128}, {128, 128}, {128, 64}, {64, 128}, {64, 64}};
        bool ok = false;
        for (const auto& t : ok_tiles) ok |= (t[0] == tile_m && t[1] == tile_n);
        if (!ok || (dtype == MS_FP32 && !(tile_m == 64 && tile_n == 64)))
            return fail(MS_EINVAL, "unsupported tile %dx%d", tile_m, tile_n);
        p.bm = tile_m;
        p.bn = tile_n;
        p.ksplit = 1;
        p.stages = 0;
    }
    if (ksplit > 0) p.ksplit = ksplit;
    if (p.ksplit > 1 && (!d_ws || ws_bytes < (size_t)p.ksplit * M * N * 4))
        return fail(MS_EWORKSPACE, "split-K needs %zu bytes of workspace", (size_t)p.ksplit * M * N * 4);
    if (M == 0) return ok();
    ms::GemmDesc g{};
    g.A = A; g.W = W; g.bias = bias; g.R = resid; g.C = out;
    g.M = M; g.N = N; g.K = K; g.lda = K; g.ldr = N; g.ldc = N;
    g.epilogue = epilogue == MS_EPI_BIAS ? ms::kEpiBias
               : epilogue == MS_EPI_BIAS_RESID ? ms::kEpiBiasResid : ms::kEpiBiasGelu;
    g.bm = p.bm; g.bn = p.bn; g.ksplit = p.ksplit; g.stages = p.stages;
    g.part = static_cast<float*>(d_ws);
    hipStream_t st = static_cast<hipStream_t>(stream);
    MS_HIP(ms::launch_gemm(dtype, g, st));
    MS_HIP(ms::launch_gemm_reduce(dtype, g, st));
    return ok();
}

ms_status mask_profiler_start(uint32_t class_mask, int32_t capacity) {
    if (capacity < 1 || capacity > (1 << 20)) return fail(MS_EINVAL, "capacity must be in 1..2^20");
    std::lock_guard<std::mutex> lk(g_prof.mu);
    while ((int)g_prof.pool.size() < 2 * capacity) {
        hipEvent_t e;
        hipError_t r = hipEventCreate(&e);
        if (r != hipSuccess) return fail(MS_EHIP, "hipEventCreate: %s", hipGetErrorString(r));
        g_prof.pool.push_back(e);
    }
    g_prof.cls.assign(capacity, 0);
    g_prof.capacity = capacity;
    g_prof.used = 0;
    g_prof.dropped = 0;
    g_prof.mask = class_mask;
    g_prof.on.store(true);
    return ok();
}

ms_status mask_profiler_stop(double* total_ms, int64_t* launches, int64_t* dropped) {
    std::lock_guard<std::mutex> lk(g_prof.mu);
    g_prof.on.store(false);
    std::vector<double> tot(MS_K_COUNT, 0.0);
    std::vector<int64_t> cnt(MS_K_COUNT, 0);
    g_prof.last_cls.assign(g_prof.used, 0);
    g_prof.last_t0.assign(g_prof.used, 0.0);
    g_prof.last_t1.assign(g_prof.used, 0.0);
    for (int i = 0; i < g_prof.used; ++i) {
        MS_HIP(hipEventSynchronize(g_prof.pool[2 * i + 1]));
        float ms = 0.f, a = 0.f, b = 0.f;
        MS_HIP(hipEventElapsedTime(&ms, g_prof.pool[2 * i], g_prof.pool[2 * i + 1]));
        MS_HIP(hipEventElapsedTime(&a, g_prof.pool[0], g_prof.pool[2 * i]));
        MS_HIP(hipEventElapsedTime(&b, g_prof.pool[0], g_prof.pool[2 * i + 1]));
        tot[g_prof.cls[i]] += ms;
        cnt[g_prof.cls[i]] += 1;
        g_prof.last_cls[i] = g_prof.cls[i];
        g_prof.last_t0[i] = a;
        g_prof.last_t1[i] = b;
    }
    for (int c = 0; c < MS_K_COUNT; ++c) {
        if (total_ms) total_ms[c] = tot[c];
        if (launches) launches[c] = cnt[c];
    }
    if (dropped) *dropped = g_prof.dropped;
    g_prof.used = 0;
    return ok();
}

ms_status mask_profiler_intervals(int32_t* cls, double* start_ms, double* end_ms, int32_t capacity,
                                  int32_t* count) {
    if (capacity < 0 || (capacity > 0 && (!cls || !start_ms || !end_ms))) return fail(MS_EINVAL, "NULL output");
    std::lock_guard<std::mutex> lk(g_prof.mu);
    const int n = (int)g_prof.last_cls.size();
    for (int i = 0; i < n && i < capacity; ++i) {
        cls[i] = g_prof.last_cls[i];
        start_ms[i] = g_prof.last_t0[i];
        end_ms[i] = g_prof.last_t1[i];
    }
    if (count) *count = n;
    return ok();
}

}  // extern "C"
