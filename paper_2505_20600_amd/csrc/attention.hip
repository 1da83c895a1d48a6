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

// ---------------------------------------------------------------------------
// bf16 kernel for head_dim 64 / 72 / 128.
//
// Workgroup = 128 packed query rows of one segment x one head x one key range;
// each wave owns 32 queries (two 16-query MFMA column blocks), so every K and
// V fragment read from LDS feeds two MFMAs. The next 64-key K/V tile is
// fetched into registers while the current one is computed. V is written to
// LDS transposed, four keys per 8-byte store. head_dim 72 runs its QK^T
// contraction as two 32-deep steps plus one zero-padded 16-deep step.
// Softmax: the scale is folded into one FMA before exp2, probabilities are
// packed to bf16 by the hardware converter.
// ---------------------------------------------------------------------------

template <int HD>
struct FastCfg {
    static constexpr int NK32 = HD / 32;                  // 32-deep QK^T steps
    static constexpr bool K16 = (HD % 32) != 0;           // one extra 16-deep step
    static constexpr int HDQ = NK32 * 32 + (K16 ? 16 : 0);
    // O^T rows: head_dim rows, then rows of ones in V^T whose O^T rows
    // accumulate the softmax denominator (sum of the bf16 probabilities) on
    // the matrix cores. head_dim 72 uses its zero-padding rows 72..79 for it;
    // 64 and 128 get one extra 16-row subtile.
    static constexpr bool SUM_IN_PAD = (HD % 16) != 0;
    static constexpr int NHS = (HD + 15) / 16 + (SUM_IN_PAD ? 0 : 1);
    static constexpr int HDV = NHS * 16;
    static constexpr int SUMROW = SUM_IN_PAD ? HD : NHS * 16 - 16;  // first ones row
    static constexpr int KL = HDQ + 8;                    // K row stride in LDS (elements)
    static constexpr int VL = kKeyTile + 8;               // V^T row stride in LDS (elements)
    static constexpr int CH = HD / 8;                     // 16-byte chunks per key row
    static constexpr int KITEMS = kKeyTile * CH;          // K: key x chunk
    static constexpr int VITEMS = (kKeyTile / 2) * CH;    // V: key pair x chunk
    static constexpr int KPT = (KITEMS + kThreads - 1) / kThreads;
    static constexpr int VPT = (VITEMS + kThreads - 1) / kThreads;
    static_assert(HD % 8 == 0 && HD % 32 <= 16, "head_dim layout");
};

__device__ __forceinline__ f32x4_t mfma32(bf16x8_t a, bf16x8_t b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4_t mfma16(bf16x4_t a, bf16x4_t b, f32x4_t c) {
    typedef short s4 __attribute__((ext_vector_type(4)));
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s4, a), __builtin_bit_cast(s4, b), c, 0, 0, 0);
}

// Key pair held by V^T storage slot s (0..31) of a 64-key tile. The PV
// product takes, in k-slot order, keys 32c + 4g .. 32c + 4g + 3 and then
// 32c + 16 + 4g .. 32c + 16 + 4g + 3 for lane group g (the layout in which the
// transposed scores leave each lane's probabilities), so storage slots
// 16c + 4g + (0, 1) hold pairs 16c + 2g + (0, 1) and slots 16c + 4g + (2, 3)
// hold pairs 16c + 8 + 2g + (0, 1).
__device__ __forceinline__ int vt_pair_of_slot(int s) {
    const int c = s >> 4, g = (s >> 2) & 3, j = s & 3;
    return 16 * c + (j < 2 ? 2 * g + j : 8 + 2 * g + (j - 2));
}

template <int HD>
__global__ __launch_bounds__(kThreads, 2) void attention_fast_kernel(AttnDesc a) {
    using C = FastCfg<HD>;
    // two K / V^T tile buffers: the next tile is stored while the current one is read
    __shared__ __attribute__((aligned(16))) bf16_t sK[2][kKeyTile * C::KL];
    __shared__ __attribute__((aligned(16))) bf16_t sVt[2][C::HDV * C::VL];

    const int tid = threadIdx.x;
    const int lane = tid % kWave;
    const int wave = tid / kWave;
    const int grp = lane / 16;
    const int l16 = lane % 16;
    // 1-D launch, logical order head-major (head, split, query tile), placed so
    // that each XCD works on a contiguous range of heads and keeps their K/V in L2
    const int total = a.n_qtiles_fast * a.nsplit * a.n_heads;
    const int lb = xcd_logical_block(blockIdx.x, total);
    const int head = lb / (a.nsplit * a.n_qtiles_fast);
    const int split = (lb / a.n_qtiles_fast) % a.nsplit;
    const int T_ = a.T, d = a.d;

    // query tile -> segment (128-row tiles counted per segment)
    int tile = lb % a.n_qtiles_fast, seg = 0, row0 = 0, row_end = 0;
    for (; seg < a.nseg; ++seg) {
        const int r0 = a.seg_start[seg], r1 = a.seg_start[seg + 1];
        const int nt = (r1 - r0 + kFastQTile - 1) / kFastQTile;
        if (tile < nt) { row0 = r0 + tile * kFastQTile; row_end = r1; break; }
        tile -= nt;
    }
    if (seg >= a.nseg) return;   // grid larger than the tile count: nothing to do
    const int b = a.seg_req[seg];

    const int ntiles_all = (T_ + kKeyTile - 1) / kKeyTile;
    const int kt0 = split * a.tiles_per_split;
    const int kt1 = min(ntiles_all, kt0 + a.tiles_per_split);

    if constexpr (C::HDQ > HD) {
        for (int i = tid; i < 2 * kKeyTile * (C::HDQ - HD); i += kThreads) {
            const int b = i / (kKeyTile * (C::HDQ - HD)), j = i % (kKeyTile * (C::HDQ - HD));
            sK[b][(j / (C::HDQ - HD)) * C::KL + HD + j % (C::HDQ - HD)] = 0;
        }
    }
    // V^T rows past head_dim: ones from SUMROW on, zeros before (never written by tiles)
    for (int i = tid; i < 2 * (C::HDV - HD) * C::VL; i += kThreads) {
        const int b = i / ((C::HDV - HD) * C::VL), j = i % ((C::HDV - HD) * C::VL);
        sVt[b][HD * C::VL + j] = (HD + j / C::VL >= C::SUMROW) ? bf16_t(0x3f80) : bf16_t(0);
    }

    // Q^T fragments (B operand): query column l16 of block qb, head_dim slots by lane group
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

    f32x4_t oacc[2][C::NHS];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int h = 0; h < C::NHS; ++h) oacc[qb][h] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    float m_run[2] = {-INFINITY, -INFINITY};
    const float cs = a.scale_log2;

    // Every thread stages both K and V items of the next tile into its own
    // registers, with no branches around the loads, so the loads stay in
    // flight while the current tile is computed. Buffer loads: the request's
    // K/V block is the resource (bounded at its last key), each lane keeps a
    // fixed byte offset, and the tile advances through the scalar offset;
    // rows past the last key read as zeros (their scores are masked anyway).
    const auto rsrc = make_rsrc(static_cast<const bf16_t*>(a.kv) + (long)b * T_ * 2 * d,
                                (uint32_t)T_ * 2u * (uint32_t)d * 2u);
    uint32_t offk[C::KPT], offv[C::VPT][2];
#pragma unroll
    for (int j = 0; j < C::KPT; ++j) {
        const int item = min(tid + j * kThreads, C::KITEMS - 1);
        offk[j] = 2u * (uint32_t)((item / C::CH) * 2 * d + head * HD + (item % C::CH) * 8);
    }
#pragma unroll
    for (int j = 0; j < C::VPT; ++j) {
        const int item = min(tid + j * kThreads, C::VITEMS - 1);
        const int key = 2 * vt_pair_of_slot(item / C::CH);
#pragma unroll
        for (int e = 0; e < 2; ++e)
            offv[j][e] = 2u * (uint32_t)((key + e) * 2 * d + d + head * HD + (item % C::CH) * 8);
    }
    vec16 pk[C::KPT], pv[C::VPT][2];
    auto gload = [&](int kt) {
        const uint32_t soff = (uint32_t)kt * kKeyTile * 2u * (uint32_t)d * 2u;
#pragma unroll
        for (int j = 0; j < C::KPT; ++j) pk[j] = buf_ld16(rsrc, offk[j], soff);
#pragma unroll
        for (int j = 0; j < C::VPT; ++j)
#pragma unroll
            for (int e = 0; e < 2; ++e) pv[j][e] = buf_ld16(rsrc, offv[j][e], soff);
    };
    // V^T rows r hold the 64 keys as 32 key pairs in the MFMA k-slot order of
    // P^T (see vt_pair_of_slot): storage slot s holds pair vt_pair_of_slot(s),
    // placed at s ^ (8 * ((r >> 4) & 3)). Each lane's 8 keys of one PV step are
    // then one aligned 16-byte read, and the pair-packed stores of one wave
    // cover all 64 banks.
    auto sstore = [&](int buf) {
#pragma unroll
        for (int j = 0; j < C::KPT; ++j) {
            const int item = tid + j * kThreads;
            if (C::KITEMS % kThreads == 0 || item < C::KITEMS) {
                const int key = item / C::CH, c = item % C::CH;
                st16(&sK[buf][key * C::KL + c * 8], pk[j]);
            }
        }
#pragma unroll
        for (int j = 0; j < C::VPT; ++j) {
            const int item = tid + j * kThreads;
            if (C::VITEMS % kThreads == 0 || item < C::VITEMS) {
                const int kp = item / C::CH, c = item % C::CH;
                // V^T[c*8 + e][2kp .. 2kp+1] = (V[2kp][c*8+e], V[2kp+1][c*8+e])
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int r = c * 8 + e;
                    const uint32_t w = __builtin_amdgcn_perm(pv[j][1].w[e >> 1], pv[j][0].w[e >> 1],
                                                             (e & 1) ? 0x07060302u : 0x05040100u);
                    const int slot = kp ^ (8 * ((r >> 4) & 3));
                    *reinterpret_cast<uint32_t*>(&sVt[buf][r * C::VL + 2 * slot]) = w;
                }
            }
        }
    };

    // One 64-key tile: S^T = K Q^T, online softmax, O^T += V^T P^T.
    auto compute = [&](int buf, int k0, bool tail) {
        f32x4_t sacc[2][4];
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) sacc[qb][ks] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            const bf16_t* kr = &sK[buf][(ks * 16 + l16) * C::KL];
#pragma unroll
            for (int kc = 0; kc < C::NK32; ++kc) {
                const bf16x8_t kf = *reinterpret_cast<const bf16x8_t*>(kr + kc * 32 + grp * 8);
#pragma unroll
                for (int qb = 0; qb < 2; ++qb) sacc[qb][ks] = mfma32(kf, qf[qb][kc], sacc[qb][ks]);
            }
            if constexpr (C::K16) {
                const bf16x4_t kf = *reinterpret_cast<const bf16x4_t*>(kr + C::NK32 * 32 + grp * 4);
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
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
            float mx = -INFINITY;
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
                mx = fmaxf(fmaxf(mx, fmaxf(sacc[qb][ks][0], sacc[qb][ks][1])), fmaxf(sacc[qb][ks][2], sacc[qb][ks][3]));
            mx = rows_max(mx);
            const float m_new = fmaxf(m_run[qb], mx);
            // rescale the accumulators only when some query's running max grew
            if (__any(m_new > m_run[qb])) {
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
        // O^T += V^T P^T; K-slots 0..3 = keys 32c + 4*grp + r, slots 4..7 = keys 32c + 16 + 4*grp + r
#pragma unroll
        for (int c = 0; c < 2; ++c) {
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
            for (int h = 0; h < C::NHS; ++h) {
                const int x = 8 * (h & 3);   // pair-slot swizzle of rows h*16 .. h*16+15
                const bf16_t* vrow = &sVt[buf][(h * 16 + l16) * C::VL];
                const bf16x8_t vf = *reinterpret_cast<const bf16x8_t*>(vrow + 2 * ((16 * c + 4 * grp) ^ x));
#pragma unroll
                for (int qb = 0; qb < 2; ++qb) oacc[qb][h] = mfma32(vf, pf[qb], oacc[qb][h]);
            }
        }
    };

    // One barrier per tile: tile kt is read from buffer kt & 1 while tile kt+1
    // is stored into the other buffer (last read during tile kt-1, which every
    // wave finished before the previous barrier); full 64-key tiles need no
    // key masking, only a partial last tile does.
    const int kfull = min(kt1, max(kt0, T_ / kKeyTile));
    if (kt0 < kt1) {
        gload(kt0);
        sstore(kt0 & 1);
        if (kt0 + 1 < kt1) gload(kt0 + 1);
    }
    __syncthreads();
    // The Q fragments are complete here (the first tile's stores waited for
    // every earlier load). Re-defining them through an empty asm statement
    // tells the compiler so; otherwise it makes the first MFMA of every tile
    // wait for all loads in flight, including the next tile's prefetch.
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
#pragma unroll
        for (int kc = 0; kc < C::NK32; ++kc) asm volatile("" : "+v"(qf[qb][kc]));
        if constexpr (C::K16) asm volatile("" : "+v"(qf16[qb]));
    }
    for (int kt = kt0; kt < kt1; ++kt) {
        compute(kt & 1, kt * kKeyTile, kt >= kfull);
        if (kt + 1 < kt1) {
            sstore((kt + 1) & 1);
            if (kt + 2 < kt1) gload(kt + 2);
        }
        __syncthreads();
    }

#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        // denominator from the ones rows: subtile SUMROW/16, row SUMROW % 16 + 4*grp + r;
        // with the ones in the padding rows only lane groups 2-3 hold it (rows 72..79)
        float l = oacc[qb][C::SUMROW / 16][0];
        if constexpr (C::SUM_IN_PAD) {
            // lane groups 0-1 hold V rows there: zero them and add the swapped halves
            const float t = grp >= 2 ? l : 0.f;
            auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(t), __float_as_uint(t), false, false);
            l = __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
        }
        const int qrow = row0 + wave * 32 + qb * 16 + l16;
        if (qrow >= row_end) continue;
        if (a.nsplit == 1) {
            const float inv_l = 1.0f / l;
            bf16_t* op = static_cast<bf16_t*>(a.o) + (long)qrow * d + head * HD;
#pragma unroll
            for (int h = 0; h < C::NHS; ++h) {
                const int cidx = h * 16 + grp * 4;
                if (cidx < HD) {
                    float v[4];
#pragma unroll
                    for (int r = 0; r < 4; ++r) v[r] = oacc[qb][h][r] * inv_l;
                    store4<bf16_t>(op + cidx, v);
                }
            }
        } else {
            float* po = a.part_o + ((long)split * a.M + qrow) * d + head * HD;
#pragma unroll
            for (int h = 0; h < C::NHS; ++h) {
                const int cidx = h * 16 + grp * 4;
                if (cidx < HD)
                    *reinterpret_cast<float4*>(po + cidx) =
                        make_float4(oacc[qb][h][0], oacc[qb][h][1], oacc[qb][h][2], oacc[qb][h][3]);
            }
            if (grp == 0)
                *reinterpret_cast<float2*>(a.part_ml + 2 * (((long)split * a.M + qrow) * a.n_heads + head)) =
                    make_float2(m_run[qb], l);
        }
    }
}

// Combine of the key-range partials (log-sum-exp weights), fixed split order.
__global__ __launch_bounds__(256) void attention_combine_kernel(AttnDesc a) {
    const long n4 = (long)a.M * a.d / 4;
    const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n4) return;
    const long m = i / (a.d / 4);
    const int col = (int)(i - m * (a.d / 4)) * 4;
    const int head = col / a.hd;
    float gmax = -INFINITY;
    for (int s = 0; s < a.nsplit; ++s)
        gmax = fmaxf(gmax, a.part_ml[2 * (((long)s * a.M + m) * a.n_heads + head)]);
    float L = 0.f, acc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int s = 0; s < a.nsplit; ++s) {
        const float* ml = a.part_ml + 2 * (((long)s * a.M + m) * a.n_heads + head);
        const float w = fast_exp2((ml[0] - gmax) * a.scale_log2);
        L += w * ml[1];
        const float4 po = *reinterpret_cast<const float4*>(a.part_o + ((long)s * a.M + m) * a.d + col);
        acc[0] += w * po.x; acc[1] += w * po.y; acc[2] += w * po.z; acc[3] += w * po.w;
    }
    const float inv = 1.0f / L;
#pragma unroll
    for (int r = 0; r < 4; ++r) acc[r] *= inv;
    store4<bf16_t>(static_cast<bf16_t*>(a.o) + m * a.d + col, acc);
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
        if (a.hd == 64)
            hipLaunchKernelGGL((attention_fast_kernel<64>), grid, block, 0, s, a);
        else if (a.hd == 72)
            hipLaunchKernelGGL((attention_fast_kernel<72>), grid, block, 0, s, a);
        else
            hipLaunchKernelGGL((attention_fast_kernel<128>), grid, block, 0, s, a);
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
    const long n4 = (long)a.M * a.d / 4;
    hipLaunchKernelGGL(attention_combine_kernel, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace ms
