// Mask-aware attention (Sec. 3.1, Fig. 5): only the masked tokens are
// queried, and each query attends over the keys/values of every token of its
// request, fresh rows for masked tokens and cached rows for the others (the
// LLM-decoding analogy of that subsection). Softmax is the full, unmasked one.
//
// Workgroup = (query tile of 64 packed rows of one segment, head); four
// waves, sixteen queries each. Key/value tiles of 64 tokens are staged in
// LDS and shared by the four waves. Online softmax in float32 with exp2 and a
// log2(e)-prescaled score.
//
// MFMA orientation: the scores are computed transposed, S^T = K Q^T, so each
// lane holds one query column and four keys per 16-key subtile. That is
// exactly the per-lane data the B operand of O^T = V^T P^T needs, so the
// probabilities never leave registers; V is stored transposed in LDS so the
// A operand (V^T rows) reads contiguous keys. The pairing of MFMA K-slots to
// keys only has to agree between the two operands of one instruction, which
// it does by construction.
#include <cstdlib>

#include "common.h"
#include "kernels.h"

namespace ms {
namespace {

constexpr int kThreads = 256;
constexpr int kKeyTile = 64;

template <typename T, int HDP>
__global__ __launch_bounds__(kThreads) void attention_kernel(AttnDesc a) {
    using E = Elt<T>;
    using frag_t = typename E::frag_t;
    constexpr int V = 16 / sizeof(T);            // elements per 16-byte vector
    constexpr int KLDS = HDP + V;                // padded K row (elements)
    constexpr int VLDS = kKeyTile + V;           // padded V^T row (elements)
    constexpr int NKC = HDP / E::kKStep;         // MFMA steps over head_dim for S
    constexpr int NHS = HDP / 16;                // 16-row subtiles of O^T
    __shared__ __attribute__((aligned(16))) T sK[kKeyTile * KLDS];
    __shared__ __attribute__((aligned(16))) T sVt[HDP * VLDS];

    const int tid = threadIdx.x;
    const int lane = tid % kWave;
    const int wave = tid / kWave;
    const int grp = lane / 16;
    const int head = blockIdx.y;
    const int tile = blockIdx.x;
    const int hd = a.hd, d = a.d, T_ = a.T;

    // segment of this query tile
    int s = 0;
    while (s + 1 < a.nseg && a.cu_tiles[s + 1] <= tile) ++s;
    const int b = a.seg_req[s];
    const int row0 = a.seg_start[s] + (tile - a.cu_tiles[s]) * kQTile;
    const int row_end = a.seg_start[s + 1];
    const int qrow = row0 + wave * 16 + lane % 16;
    const bool qvalid = qrow < row_end;

    // zero the head_dim padding of the LDS tiles once; tile loads never touch it
    if (hd < HDP) {
        for (int i = tid; i < kKeyTile * (HDP - hd); i += kThreads) {
            const int r = i / (HDP - hd), c = hd + i % (HDP - hd);
            sK[r * KLDS + c] = T(0);
        }
        for (int i = tid; i < (HDP - hd) * kKeyTile; i += kThreads) {
            const int r = hd + i / kKeyTile, c = i % kKeyTile;
            sVt[r * VLDS + c] = T(0);
        }
    }

    // Q^T fragments (B operand): query = lane % 16, head_dim slots by lane group
    frag_t qf[NKC];
    const T* __restrict__ q = static_cast<const T*>(a.q);
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) {
        const int k = kc * E::kKStep + grp * E::kKPerLane;
        if constexpr (E::kKPerLane == 1) {
            qf[kc] = (qvalid && k < hd) ? q[(long)qrow * d + head * hd + k] : 0.f;
        } else {
            if (qvalid && k < hd) {
                qf[kc] = *reinterpret_cast<const frag_t*>(q + (long)qrow * d + head * hd + k);
            } else {
                vec16 z = {{0u, 0u, 0u, 0u}};
                qf[kc] = *reinterpret_cast<const frag_t*>(&z);
            }
        }
    }

    f32x4_t oacc[NHS];
#pragma unroll
    for (int h = 0; h < NHS; ++h) oacc[h] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY, l_run = 0.f;

    const T* __restrict__ kv = static_cast<const T*>(a.kv);
    const long req_base = (long)b * T_;
    const int chunks = hd / V;                     // 16-byte chunks per key row
    const int ntiles = (T_ + kKeyTile - 1) / kKeyTile;

    for (int kt = 0; kt < ntiles; ++kt) {
        const int k0 = kt * kKeyTile;
        __syncthreads();
        for (int i = tid; i < kKeyTile * chunks; i += kThreads) {
            const int kk = i / chunks, c = i % chunks;
            const int t = k0 + kk;
            vec16 kvec = {{0u, 0u, 0u, 0u}}, vvec = {{0u, 0u, 0u, 0u}};
            if (t < T_) {
                const T* src = kv + (req_base + t) * 2 * d + head * hd + c * V;
                kvec = ld16(src);
                vvec = ld16(src + d);
            }
            st16(&sK[kk * KLDS + c * V], kvec);
            const T* ve = reinterpret_cast<const T*>(&vvec);
#pragma unroll
            for (int e = 0; e < V; ++e) sVt[(c * V + e) * VLDS + kk] = ve[e];
        }
        __syncthreads();

        // S^T subtiles: keys ks*16 + 4*grp + r, query lane % 16
        float sc[4][4];
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kc = 0; kc < NKC; ++kc) {
                const int k = kc * E::kKStep + grp * E::kKPerLane;
                const frag_t kf = *reinterpret_cast<const frag_t*>(&sK[(ks * 16 + lane % 16) * KLDS + k]);
                acc = E::mma(kf, qf[kc], acc);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int t = k0 + ks * 16 + grp * 4 + r;
                sc[ks][r] = t < T_ ? acc[r] * a.scale_log2 : -INFINITY;
            }
        }

        float mx = -INFINITY;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
#pragma unroll
            for (int r = 0; r < 4; ++r) mx = fmaxf(mx, sc[ks][r]);
        mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
        mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
        const float m_new = fmaxf(m_run, mx);
        const float corr = (m_run == -INFINITY) ? 0.f : fast_exp2(m_run - m_new);
        float psum = 0.f;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                sc[ks][r] = fast_exp2(sc[ks][r] - m_new);
                psum += sc[ks][r];
            }
        l_run = l_run * corr + psum;
        m_run = m_new;
#pragma unroll
        for (int h = 0; h < NHS; ++h)
#pragma unroll
            for (int r = 0; r < 4; ++r) oacc[h][r] *= corr;

        // O^T += V^T P^T
        if constexpr (E::kKPerLane == 1) {
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int key = ks * 16 + grp * 4 + r;
#pragma unroll
                    for (int h = 0; h < NHS; ++h) {
                        const frag_t vf = sVt[(h * 16 + lane % 16) * VLDS + key];
                        oacc[h] = E::mma(vf, sc[ks][r], oacc[h]);
                    }
                }
        } else {
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                // slots 0..3: keys 32c + 4*grp + r; slots 4..7: keys 32c + 16 + 4*grp + r
                union { bf16_t u[8]; frag_t f; } pf;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    pf.u[r] = f32_to_bf16(sc[2 * c][r]);
                    pf.u[4 + r] = f32_to_bf16(sc[2 * c + 1][r]);
                }
#pragma unroll
                for (int h = 0; h < NHS; ++h) {
                    const T* row = &sVt[(h * 16 + lane % 16) * VLDS + 32 * c + 4 * grp];
                    union { uint2 w[2]; frag_t f; } vf;
                    vf.w[0] = *reinterpret_cast<const uint2*>(row);
                    vf.w[1] = *reinterpret_cast<const uint2*>(row + 16);
                    oacc[h] = E::mma(vf.f, pf.f, oacc[h]);
                }
            }
        }
    }

    float l = l_run;
    l += __shfl_xor(l, 16, kWave);
    l += __shfl_xor(l, 32, kWave);
    const float inv_l = 1.0f / l;
    if (qvalid) {
        T* __restrict__ o = static_cast<T*>(a.o);
#pragma unroll
        for (int h = 0; h < NHS; ++h) {
            const int c = h * 16 + grp * 4;
            if (c < hd) {
                float v[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = oacc[h][r] * inv_l;
                store4<T>(o + (long)qrow * d + head * hd + c, v);
            }
        }
    }
}

__device__ __forceinline__ f32x4_t mfma32(bf16x8_t a, bf16x8_t b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4_t mfma16(bf16x4_t a, bf16x4_t b, f32x4_t c) {
    typedef short s4 __attribute__((ext_vector_type(4)));
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s4, a), __builtin_bit_cast(s4, b), c, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// bf16 kernel for head_dim 64 / 72 / 128.
//
// Workgroup = 128 packed query rows of one segment x one head x one key range;
// each wave owns 32 queries (two 16-query MFMA column blocks), so every K and
// V fragment read from LDS feeds two MFMAs. Transposed scores S^T = K Q^T
// leave the probabilities in the B-operand layout of O^T = V^T P^T. K and V
// tiles of 64 keys go global -> LDS with buffer_load_dwordx4 ... lds (no
// staging registers, no VALU work to store them) into S stages, in natural
// [key][head_dim] layout;
// the PV operand V^T is read with the gfx950 transpose read
// ds_read_b64_tr_b16: within each 16-lane group, lane i receives element
// (i & 3) of the 8 bytes addressed by lane 4e + (i >> 2), e = 0..3. Each
// lane therefore addresses V[key0 + (l16 >> 2)][hd0 + 4 (l16 & 3)] and
// receives V[key0 + e][hd0 + l16], e = 0..3: four keys of one head_dim row,
// in the k-slot order of P^T. Rows of 128 / 256 bytes carry their 16-byte
// chunks XOR-swizzled by dma_swz(row) so both the K fragment reads (16 rows)
// and the transpose reads (8 rows x 32 bytes per half wave) are conflict-free;
// 144-byte rows (head_dim 72) need no swizzle. Keys past the end read as
// zeros (buffer bound). The softmax denominator comes from V^T rows of ones:
// a constant operand for head_dim 64 / 128, and for head_dim 72 the padding
// rows 72..79, whose lanes address a small LDS block of ones.
// ---------------------------------------------------------------------------

constexpr float kRescaleLog2 = 8.0f;   // softmax weights may reach 2^8 before a rescale

template <int HD>
struct DmaCfg {
    static constexpr int NK32 = HD / 32;
    static constexpr bool K16 = (HD % 32) != 0;
    static constexpr int ROWB = HD * 2;                 // bytes per K / V row
    static constexpr bool SWZ = ROWB == 128 || ROWB == 256;
    static constexpr int TILEB = kKeyTile * ROWB;       // bytes per K (or V) tile
    static constexpr int KPAD = 16;                     // past the K tile: head_dim 72 reads 8 B beyond a row
    static constexpr int STAGEB = 2 * TILEB + KPAD;     // K tile, pad, V tile
    static constexpr int INSTR = TILEB / 1024;          // 1 KB copies per tile
    static constexpr int NQ = 2 * INSTR;                // copies per stage (K then V)
    static constexpr int IPW_MIN = NQ / 4;              // copies per wave per stage (fewest)
    static constexpr int IPW_MAX = (NQ + 3) / 4;
    static constexpr bool SUM_IN_PAD = (HD % 16) != 0;
    static constexpr int NHS = (HD + 15) / 16 + (SUM_IN_PAD ? 0 : 1);
    static constexpr int NREAL = (HD + 15) / 16;        // O^T subtiles with V rows
    static_assert(TILEB % 1024 == 0, "tile copies");
};

// 16-byte chunk swizzle of a K / V row (see the kernel comment).
template <int ROWB>
__device__ __forceinline__ int dma_swz(int r) {
    if constexpr (ROWB == 128) return 2 * ((r >> 1) & 3) + ((r >> 3) & 1);
    else if constexpr (ROWB == 256) return 2 * (r & 7) + ((r >> 3) & 1);
    else return 0;
}

typedef const __attribute__((address_space(3))) uint8_t* lds_cptr;

__device__ __forceinline__ bf16x4_t ld_tr16(lds_cptr p) {
    typedef short s4 __attribute__((ext_vector_type(4)));
    const s4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s4*)(p));
    return __builtin_bit_cast(bf16x4_t, v);
}

// Workgroups per CU the register budget is set for: four for head_dim 64
// (128 VGPRs, no spills), two for 72 and 128 (whose 140 / 208 VGPRs then
// allow three and two).
constexpr int dma_occupancy(int hd) { return hd == 64 ? 4 : 2; }

template <int HD, int S>
__global__ __launch_bounds__(kThreads, dma_occupancy(HD)) void attention_dma_kernel(AttnDesc a) {
    using C = DmaCfg<HD>;
    __shared__ __attribute__((aligned(1024))) uint8_t smem[S * C::STAGEB + 16];
    const uint32_t lds0 = lds_addr(smem);
    const uint32_t ones_rel = S * C::STAGEB;            // 8 bytes of bf16 ones (head_dim 72)

    const int tid = threadIdx.x;
    const int lane = tid % kWave;
    const int wave = tid / kWave;
    const int grp = lane / 16;
    const int l16 = lane % 16;
    const int total = a.n_qtiles_fast * a.nsplit * a.n_heads;
    const int lb = xcd_logical_block(blockIdx.x, total);
    const int head = lb / (a.nsplit * a.n_qtiles_fast);
    const int split = (lb / a.n_qtiles_fast) % a.nsplit;
    const int T_ = a.T, d = a.d;

    int tile = lb % a.n_qtiles_fast, seg = 0, row0 = 0, row_end = 0;
    for (; seg < a.nseg; ++seg) {
        const int r0 = a.seg_start[seg], r1 = a.seg_start[seg + 1];
        const int nt = (r1 - r0 + kFastQTile - 1) / kFastQTile;
        if (tile < nt) { row0 = r0 + tile * kFastQTile; row_end = r1; break; }
        tile -= nt;
    }
    if (seg >= a.nseg) return;
    const int b = a.seg_req[seg];
    const int ntiles_all = (T_ + kKeyTile - 1) / kKeyTile;
    const int kt0 = split * a.tiles_per_split;
    const int kt1 = min(ntiles_all, kt0 + a.tiles_per_split);
    const int nt = max(0, kt1 - kt0);

    // constant LDS: the K pads (finite bytes for the head_dim-72 over-read) and the ones block
    if (tid < S) *reinterpret_cast<uint4*>(smem + tid * C::STAGEB + C::TILEB) = make_uint4(0u, 0u, 0u, 0u);
    if (tid == S) *reinterpret_cast<uint2*>(smem + S * C::STAGEB) = make_uint2(0x3f803f80u, 0x3f803f80u);

    // buffer resource over request b's K/V block [T][2][d]
    const u32x4_t rsrc = raw_rsrc(static_cast<const bf16_t*>(a.kv) + (long)b * T_ * 2 * d, (uint32_t)T_ * 4u * (uint32_t)d);
    // per copy of this wave: fixed per-lane global byte offset and LDS destination in a stage
    uint32_t voff[C::IPW_MAX], ldst[C::IPW_MAX];
#pragma unroll
    for (int i = 0; i < C::IPW_MAX; ++i) {
        const int q = min(i * 4 + wave, C::NQ - 1);
        const bool isV = q >= C::INSTR;
        const int pos = (q % C::INSTR) * 1024 + lane * 16;
        const int r = pos / C::ROWB;
        const int c = ((pos % C::ROWB) / 16) ^ dma_swz<C::ROWB>(r);
        voff[i] = (uint32_t)(r * 4 * d + (isV ? 2 * d : 0) + head * C::ROWB + c * 16);
        ldst[i] = __builtin_amdgcn_readfirstlane((uint32_t)((isV ? C::TILEB + C::KPAD : 0) + (q % C::INSTR) * 1024));
    }
    auto issue = [&](int kt, int st) {
        const uint32_t soff = (uint32_t)kt * kKeyTile * 4u * (uint32_t)d;
        const uint32_t sbase = lds0 + st * C::STAGEB;
#pragma unroll
        for (int i = 0; i < C::IPW_MAX; ++i)
            if (i * 4 + wave < C::NQ) dma_buf16(rsrc, voff[i], soff, sbase + ldst[i]);
    };

    // Q^T fragments (B operand)
    bf16x8_t qf[2][C::NK32 > 0 ? C::NK32 : 1];
    bf16x4_t qf16[2];
    const bf16_t* __restrict__ q = static_cast<const bf16_t*>(a.q);
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const int qrow = row0 + wave * 32 + qb * 16 + l16;
        const bool valid = qrow < row_end;
        const bf16_t* qp = q + (long)qrow * d + head * HD;
#pragma unroll
        for (int kc = 0; kc < C::NK32; ++kc) {
            vec16 v = {{0u, 0u, 0u, 0u}};
            if (valid) v = ld16(qp + kc * 32 + grp * 8);
            qf[qb][kc] = __builtin_bit_cast(bf16x8_t, v);
        }
        if constexpr (C::K16) {
            const int k = C::NK32 * 32 + grp * 4;
            uint2 v = make_uint2(0u, 0u);
            if (valid && k < HD) v = *reinterpret_cast<const uint2*>(qp + k);
            qf16[qb] = __builtin_bit_cast(bf16x4_t, v);
        }
    }

    // fragment read offsets inside a stage (bytes)
    const int fK = dma_swz<C::ROWB>(l16);
    uint32_t koff[C::NK32 > 0 ? C::NK32 : 1];
#pragma unroll
    for (int kc = 0; kc < C::NK32; ++kc) koff[kc] = l16 * C::ROWB + (((4 * kc + grp) ^ fK) * 16);
    const uint32_t koff16 = l16 * C::ROWB + C::NK32 * 64 + grp * 8;   // head_dim 72: 16-deep step
    const int rowA = 4 * grp + (l16 >> 2);
    const int fV = dma_swz<C::ROWB>(rowA);
    uint32_t voffh[C::NREAL];
#pragma unroll
    for (int h = 0; h < C::NREAL; ++h) {
        const int hd = 16 * h + 4 * (l16 & 3);
        voffh[h] = C::TILEB + C::KPAD + rowA * C::ROWB + (((hd / 8) ^ fV) * 16) + (hd % 8) * 2;
    }
    const bool ones_lane = C::SUM_IN_PAD && (16 * (C::NREAL - 1) + 4 * (l16 & 3)) >= HD;

    f32x4_t oacc[2][C::NHS];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int h = 0; h < C::NHS; ++h) oacc[qb][h] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    float m_run[2] = {-INFINITY, -INFINITY};
    const float cs = a.scale_log2;
    const bf16x8_t onesf = __builtin_bit_cast(bf16x8_t, make_uint4(0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u));

    // S^T of one tile (QK^T) into sacc, keys past T masked
    auto qk = [&](uint32_t sbase, int k0, bool tail, f32x4_t (&sacc)[2][4]) {
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) sacc[qb][ks] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
            for (int kc = 0; kc < C::NK32; ++kc) {
                const bf16x8_t kf = *reinterpret_cast<const bf16x8_t*>(smem + sbase + koff[kc] + ks * 16 * C::ROWB);
#pragma unroll
                for (int qb = 0; qb < 2; ++qb) sacc[qb][ks] = mfma32(kf, qf[qb][kc], sacc[qb][ks]);
            }
            if constexpr (C::K16) {
                const bf16x4_t kf = *reinterpret_cast<const bf16x4_t*>(smem + sbase + koff16 + ks * 16 * C::ROWB);
#pragma unroll
                for (int qb = 0; qb < 2; ++qb) sacc[qb][ks] = mfma16(kf, qf16[qb], sacc[qb][ks]);
            }
        }
        if (tail) {
#pragma unroll
            for (int qb = 0; qb < 2; ++qb)
#pragma unroll
                for (int ks = 0; ks < 4; ++ks)
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        if (k0 + ks * 16 + grp * 4 + r >= T_) sacc[qb][ks][r] = -INFINITY;
        }
    };
    // online softmax in place: sacc becomes the weights; running maxima and accumulators updated
    auto softmax = [&](f32x4_t (&sacc)[2][4]) {
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
            float mx = -INFINITY;
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
                mx = fmaxf(fmaxf(mx, fmaxf(sacc[qb][ks][0], sacc[qb][ks][1])), fmaxf(sacc[qb][ks][2], sacc[qb][ks][3]));
            mx = rows_max(mx);
            // Rescale only when some query's maximum grew by more than 2^8 (in the
            // exp2 domain): below that the stale maximum keeps the weights <= 256,
            // exact in bf16 and fp32 alike, and numerator and denominator share it.
            // This keeps the accumulators out of VALU work on almost every tile.
            const float m_new = fmaxf(m_run[qb], mx);
            if (__any((m_new - m_run[qb]) * cs > kRescaleLog2)) {
                const float corr = fast_exp2((m_run[qb] - m_new) * cs);
#pragma unroll
                for (int h = 0; h < C::NHS; ++h) oacc[qb][h] *= corr;
                m_run[qb] = m_new;
            }
            const float mc = m_run[qb] * cs;
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
#pragma unroll
                for (int r = 0; r < 4; ++r) sacc[qb][ks][r] = fast_exp2(fmaf(sacc[qb][ks][r], cs, -mc));
        }
    };
    // O^T += V^T P^T for one tile
    auto pv = [&](uint32_t sbase, f32x4_t (&sacc)[2][4]) {
        // O^T += V^T P^T; k-slots 0..3 = keys 32c + 4*grp + e, 4..7 = keys 32c + 16 + 4*grp + e
        uint32_t vbase[C::NREAL];
#pragma unroll
        for (int h = 0; h < C::NREAL; ++h) {
            vbase[h] = lds0 + sbase + voffh[h];
            asm volatile("" : "+v"(vbase[h]));   // keep the sum: offsets are added per read
        }
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            // all V^T operands of this 32-key block first, so their reads overlap
            bf16x8_t vf[C::NHS];
#pragma unroll
            for (int h = 0; h < C::NHS; ++h) {
                if (h >= C::NREAL) {
                    vf[h] = onesf;
                } else {
                    // one base address per head_dim block and tile; the key-block and
                    // second-half offsets fold into the read instructions
                    lds_cptr p0 = (lds_cptr)(uintptr_t)vbase[h] + (32 * c) * C::ROWB;
                    lds_cptr p1 = (lds_cptr)(uintptr_t)vbase[h] + (32 * c + 16) * C::ROWB;
                    if (h == C::NREAL - 1 && ones_lane) { p0 = (lds_cptr)(uintptr_t)(lds0 + ones_rel); p1 = p0; }
                    const bf16x4_t lo = ld_tr16(p0), hi = ld_tr16(p1);
                    vf[h] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
                }
            }
            bf16x8_t pf[2];
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) {
                uint4 w;
                w.x = pack_bf16x2(sacc[qb][2 * c][0], sacc[qb][2 * c][1]);
                w.y = pack_bf16x2(sacc[qb][2 * c][2], sacc[qb][2 * c][3]);
                w.z = pack_bf16x2(sacc[qb][2 * c + 1][0], sacc[qb][2 * c + 1][1]);
                w.w = pack_bf16x2(sacc[qb][2 * c + 1][2], sacc[qb][2 * c + 1][3]);
                pf[qb] = __builtin_bit_cast(bf16x8_t, w);
            }
#pragma unroll
            for (int h = 0; h < C::NHS; ++h)
#pragma unroll
                for (int qb = 0; qb < 2; ++qb) oacc[qb][h] = mfma32(vf[h], pf[qb], oacc[qb][h]);
        }
    };

    const int kfull = min(kt1, max(kt0, T_ / kKeyTile));
    auto fence_q = [&]() {
        // The Q fragments are complete here. Re-defining them through an empty asm
        // statement tells the compiler so; otherwise it makes the first MFMA of
        // every tile wait for all loads in flight, including the next prefetch.
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
#pragma unroll
            for (int kc = 0; kc < C::NK32; ++kc) asm volatile("" : "+v"(qf[qb][kc]));
            if constexpr (C::K16) asm volatile("" : "+v"(qf16[qb]));
        }
    };
    f32x4_t sa[2][4];
    // S-stage pipeline: step t reads stage t % S; tiles t + 1 .. t + S - 2 stay in flight
    for (int t = 0; t < S - 1; ++t)
        if (t < nt) issue(kt0 + t, t);
    fence_q();
    for (int t = 0; t < nt; ++t) {
        if (t + S - 1 <= nt) wait_vmcnt<(S - 2) * C::IPW_MIN>();
        else wait_vmcnt<0>();
        barrier_only();
        if (t + S - 1 < nt) issue(kt0 + t + S - 1, (t + S - 1) % S);
        const int kt = kt0 + t;
        qk((t % S) * C::STAGEB, kt * kKeyTile, kt >= kfull, sa);
        softmax(sa);
        pv((t % S) * C::STAGEB, sa);
    }

    // Output (or this key range's partial) through LDS: a lane holds 4
    // consecutive head_dim values of one query row per 16 x 16 block, so
    // direct stores write 8-byte pieces of 16 rows; staged in the (now free)
    // stage memory, each wave writes its 32 rows as row-contiguous 16-byte
    // vectors. Rows of 128 / 256 bytes XOR-swizzle their 16-byte chunks by
    // the row (head_dim 72 rows are not swizzled).
    constexpr int CH = HD / 8;                     // 16-byte chunks per row
    constexpr int SWM = C::SWZ ? (CH >= 16 ? 15 : CH - 1) : 0;
    __syncthreads();   // every wave is past its last read of the stages
    uint8_t* const so = smem + wave * 32 * C::ROWB;
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        float l;
        if constexpr (C::SUM_IN_PAD) {
            // rows 72..79 of subtile 4 are the ones rows: lane groups 2-3 hold them
            const float t0 = grp >= 2 ? oacc[qb][C::NHS - 1][0] : 0.f;
            auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(t0), __float_as_uint(t0), false, false);
            l = __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
        } else {
            l = oacc[qb][C::NHS - 1][0];
        }
        // normalised by this key range's own sum (bf16 holds it to the
        // output's precision at half the bytes of float32)
        const float inv_l = 1.0f / l;
        const int rl = qb * 16 + l16;
#pragma unroll
        for (int h = 0; h < C::NHS; ++h) {
            const int cidx = h * 16 + grp * 4;
            if (cidx < HD) {
                float v[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = oacc[qb][h][r] * inv_l;
                store4<bf16_t>(reinterpret_cast<bf16_t*>(so + rl * C::ROWB + (((cidx / 8) ^ (rl & SWM)) * 16) + (cidx % 8) * 2), v);
            }
        }
        const int qrow = row0 + wave * 32 + rl;
        if (a.nsplit > 1 && grp == 0 && qrow < row_end)
            *reinterpret_cast<float2*>(a.part_ml + 2 * (((long)split * a.M + qrow) * a.n_heads + head)) =
                make_float2(m_run[qb], l);
    }
    __syncthreads();
    bf16_t* const dst = a.nsplit == 1 ? static_cast<bf16_t*>(a.o) : a.part_o + (long)split * a.M * d;
#pragma unroll
    for (int k = lane; k < 32 * CH; k += kWave) {
        const int rl = k / CH, c = k % CH;
        const int qrow = row0 + wave * 32 + rl;
        if (qrow < row_end)
            st16(dst + (long)qrow * d + head * HD + c * 8, ld16(so + rl * C::ROWB + ((c ^ (rl & SWM)) * 16)));
    }
}

// Combine of the key-range partials, fixed split order: range s, with running
// max m_s, sum l_s and normalised output O_s, has weight l_s 2^((m_s - m) c)
// (m the largest m_s, c the log2-domain scale), and the output is the
// weighted mean of the O_s. One thread per 8 columns of a row (16-byte
// vectors); with the split count NS known at compile time every partial of
// the thread is loaded before the first is used (NS = 0: any count, loaded
// in turn). The arithmetic and its order do not depend on NS.
template <int NS>
__global__ __launch_bounds__(256) void attention_combine_kernel(AttnDesc a) {
    const long n8 = (long)a.M * a.d / 8;
    const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n8) return;
    const long m = i / (a.d / 8);
    const int col = (int)(i - m * (a.d / 8)) * 8;
    const int head = col / a.hd;
    const int ns = NS > 0 ? NS : a.nsplit;
    auto ml_of = [&](int s) { return a.part_ml + 2 * (((long)s * a.M + m) * a.n_heads + head); };
    auto po_of = [&](int s) { return a.part_o + ((long)s * a.M + m) * a.d + col; };
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    float L = 0.f;
    if constexpr (NS > 0) {
        float2 ml[NS];
        vec16 po[NS];
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            ml[s] = *reinterpret_cast<const float2*>(ml_of(s));
            po[s] = ld16(po_of(s));
        }
        float gmax = -INFINITY;
#pragma unroll
        for (int s = 0; s < NS; ++s) gmax = fmaxf(gmax, ml[s].x);
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            const float w = fast_exp2((ml[s].x - gmax) * a.scale_log2) * ml[s].y;
            L += w;
#pragma unroll
            for (int r = 0; r < 8; ++r) {
                const uint32_t u = po[s].w[r >> 1];
                acc[r] += w * __uint_as_float((r & 1) ? (u & 0xffff0000u) : (u << 16));
            }
        }
    } else {
        // any split count: chunks of 8 splits, each chunk's loads issued together
        constexpr int CH = 8;
        float gmax = -INFINITY;
        for (int s0 = 0; s0 < ns; s0 += CH) {
            float mv[CH];
#pragma unroll
            for (int j = 0; j < CH; ++j) mv[j] = s0 + j < ns ? ml_of(s0 + j)[0] : -INFINITY;
#pragma unroll
            for (int j = 0; j < CH; ++j) gmax = fmaxf(gmax, mv[j]);
        }
        for (int s0 = 0; s0 < ns; s0 += CH) {
            float2 ml[CH];
            vec16 po[CH];
#pragma unroll
            for (int j = 0; j < CH; ++j) {
                if (s0 + j < ns) {
                    ml[j] = *reinterpret_cast<const float2*>(ml_of(s0 + j));
                    po[j] = ld16(po_of(s0 + j));
                }
            }
#pragma unroll
            for (int j = 0; j < CH; ++j) {
                if (s0 + j >= ns) break;
                const float w = fast_exp2((ml[j].x - gmax) * a.scale_log2) * ml[j].y;
                L += w;
#pragma unroll
                for (int r = 0; r < 8; ++r) {
                    const uint32_t u = po[j].w[r >> 1];
                    acc[r] += w * __uint_as_float((r & 1) ? (u & 0xffff0000u) : (u << 16));
                }
            }
        }
    }
    const float inv = 1.0f / L;
#pragma unroll
    for (int r = 0; r < 8; ++r) acc[r] *= inv;
    bf16_t* o = static_cast<bf16_t*>(a.o) + m * a.d + col;
    store4<bf16_t>(o, acc);
    store4<bf16_t>(o + 4, acc + 4);
}

}  // namespace

bool attention_fast_path(int dtype, int hd) {
    return dtype == kBF16 && (hd == 64 || hd == 72 || hd == 128);
}

// bf16, head_dim 64 / 72 / 128: the fast kernel (+ combine when split). Other
// bf16 head_dims up to 128 and fp32 up to 64: the generic kernel.
hipError_t launch_attention(int dtype, const AttnDesc& a, hipStream_t s) {
    if (a.M == 0) return hipSuccess;
    if (attention_fast_path(dtype, a.hd)) {
        dim3 grid(a.n_qtiles_fast * a.n_heads * a.nsplit), block(kThreads);
        if (a.hd == 64) hipLaunchKernelGGL((attention_dma_kernel<64, 2>), grid, block, 0, s, a);
        else if (a.hd == 72) hipLaunchKernelGGL((attention_dma_kernel<72, 2>), grid, block, 0, s, a);
        else hipLaunchKernelGGL((attention_dma_kernel<128, 2>), grid, block, 0, s, a);
        return hipGetLastError();
    }
    dim3 grid(a.n_qtiles, a.n_heads), block(kThreads);
    if (dtype == kBF16) {
        if (a.hd <= 64)
            hipLaunchKernelGGL((attention_kernel<bf16_t, 64>), grid, block, 0, s, a);
        else if (a.hd <= 96)
            hipLaunchKernelGGL((attention_kernel<bf16_t, 96>), grid, block, 0, s, a);
        else if (a.hd <= 128)
            hipLaunchKernelGGL((attention_kernel<bf16_t, 128>), grid, block, 0, s, a);
        else
            return hipErrorInvalidValue;
    } else {
        if (a.hd > 64) return hipErrorInvalidValue;
        hipLaunchKernelGGL((attention_kernel<float, 64>), grid, block, 0, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_attention_combine(int dtype, const AttnDesc& a, hipStream_t s) {
    if (a.M == 0 || a.nsplit <= 1 || !attention_fast_path(dtype, a.hd)) return hipSuccess;
    const long n8 = (long)a.M * a.d / 8;
    const dim3 grid((unsigned)((n8 + 255) / 256)), block(256);
    switch (a.nsplit) {
        case 2: hipLaunchKernelGGL(attention_combine_kernel<2>, grid, block, 0, s, a); break;
        case 3: hipLaunchKernelGGL(attention_combine_kernel<3>, grid, block, 0, s, a); break;
        case 4: hipLaunchKernelGGL(attention_combine_kernel<4>, grid, block, 0, s, a); break;
        case 5: hipLaunchKernelGGL(attention_combine_kernel<5>, grid, block, 0, s, a); break;
        case 6: hipLaunchKernelGGL(attention_combine_kernel<6>, grid, block, 0, s, a); break;
        case 7: hipLaunchKernelGGL(attention_combine_kernel<7>, grid, block, 0, s, a); break;
        case 8: hipLaunchKernelGGL(attention_combine_kernel<8>, grid, block, 0, s, a); break;
        default: hipLaunchKernelGGL(attention_combine_kernel<0>, grid, block, 0, s, a); break;
    }
    return hipGetLastError();
}

}  // namespace ms
