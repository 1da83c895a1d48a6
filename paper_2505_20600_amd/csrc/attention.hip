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
        const float corr = (m_run == -INFINITY) ? 0.f : exp2f(m_run - m_new);
        float psum = 0.f;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                sc[ks][r] = exp2f(sc[ks][r] - m_new);
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

}  // namespace

// bf16: head_dim up to 128 (padded to 64 / 96 / 128 in LDS and registers);
// fp32: head_dim up to 64.
hipError_t launch_attention(int dtype, const AttnDesc& a, hipStream_t s) {
    if (a.n_qtiles == 0) return hipSuccess;
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

}  // namespace ms
