// Hardware-aware lightweight group gate (Local Expert Selection, Eq. 4; Lightweight
// Group Gate Network, Eq. 5-7) and top-k selection, for gfx950.
//
// One workgroup (4 waves) takes 16 tokens. Phase 1 computes the M local and K group
// logits of those tokens with the matrix cores: gate-weight rows are the A operand,
// token rows the B operand, and each wave contracts a quarter of d. Phase 2 adds the
// four partial sums in a fixed order (deterministic). Phase 3 gives each wave four
// tokens: masked group softmax (stage 1), masked in-group softmax (stage 2), the
// product g_i = p_group^(k) * p_local,i^(k), top-k by wave shuffles with ties to the
// lower expert index, and renormalisation of the selected weights.
#include "device_common.h"
#include "internal.h"

namespace ec2moe {
namespace {

constexpr int kTok = 16;           // tokens per workgroup
constexpr int kMaxRowBlocks = 20;  // M + K <= 320 gate rows
constexpr int kMaxGroups = 160;
constexpr int kMaxTopK = 16;

__device__ __forceinline__ bool is_cand(const uint64_t* mask, int e) {
    return (mask[e >> 6] >> (e & 63)) & 1ull;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
    return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
    return v;
}

template <typename T>
__global__ __launch_bounds__(256) void gate_kernel(GateArgs p) {
    extern __shared__ float part[];  // [4 waves][rows][16 tokens], then the sums in wave 0's slot
    __shared__ float grp_max[4][kMaxGroups];
    __shared__ float grp_sum[4][kMaxGroups];
    __shared__ float grp_p[4][kMaxGroups];

    constexpr int EPC = Elem<T>::kPerChunk;
    constexpr int SLICE = 4 * EPC;  // k covered by one matrix-core step
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int g4 = lane >> 4;
    const int M = p.n_experts, K = p.n_groups, d = p.d;
    const int R = M + K;
    const int nrb = (R + 15) >> 4;
    const int t0 = blockIdx.x * kTok;

    // ---------------- phase 1: partial logits over this wave's quarter of d
    int tok = t0 + (lane & 15);
    if (tok >= p.n_tokens) tok = p.n_tokens - 1;
    const T* xrow = static_cast<const T*>(p.x) + static_cast<size_t>(tok) * d;
    const T* wl = static_cast<const T*>(p.w_local);
    const T* wg = static_cast<const T*>(p.w_global);
    const int kq = d >> 2;
    const int kbeg = wave * kq;

    f32x4 acc[kMaxRowBlocks];
#pragma unroll
    for (int rb = 0; rb < kMaxRowBlocks; ++rb) acc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int k = kbeg; k < kbeg + kq; k += SLICE) {
        const uint4 bx = ldg16(xrow + k + g4 * EPC);
#pragma unroll
        for (int rb = 0; rb < kMaxRowBlocks; ++rb) {
            if (rb < nrb) {
                const int r = rb * 16 + (lane & 15);
                uint4 aw = make_uint4(0, 0, 0, 0);
                if (r < R) {
                    const T* wrow = r < M ? wl + static_cast<size_t>(r) * d
                                          : wg + static_cast<size_t>(r - M) * d;
                    aw = ldg16(wrow + k + g4 * EPC);
                }
                acc[rb] = Mfma<T>::step(aw, bx, acc[rb]);
            }
        }
    }

    const int rows_pad = nrb * 16;
    float* mine = part + static_cast<size_t>(wave) * rows_pad * kTok;
#pragma unroll
    for (int rb = 0; rb < kMaxRowBlocks; ++rb) {
        if (rb < nrb) {
#pragma unroll
            for (int i = 0; i < 4; ++i) mine[(rb * 16 + g4 * 4 + i) * kTok + (lane & 15)] = acc[rb][i];
        }
    }
    __syncthreads();

    // ---------------- phase 2: fixed-order sum of the four partials
    const int n_el = rows_pad * kTok;
    for (int i = threadIdx.x; i < n_el; i += 256) {
        float s = part[i];
        s += part[n_el + i];
        s += part[2 * n_el + i];
        s += part[3 * n_el + i];
        part[i] = s;
    }
    __syncthreads();

    // ---------------- phase 3: two-stage softmax, fusion, top-k; 4 tokens per wave
    const float* logit = part;  // [row][token]
    const int Mk = M / K;
    for (int it = 0; it < kTok / 4; ++it) {
        const int tl = wave * (kTok / 4) + it;
        const int t = t0 + tl;

        // stage 2 statistics per group over its candidates: max and sum of exp
        for (int k = lane; k < K; k += 64) {
            float m = -INFINITY;
            for (int i = k * Mk; i < (k + 1) * Mk; ++i) {
                if (is_cand(p.mask, i)) {
                    const float l = logit[i * kTok + tl] + (p.b_local ? p.b_local[i] : 0.f);
                    m = fmaxf(m, l);
                }
            }
            float s = 0.f;
            if (m != -INFINITY) {
                for (int i = k * Mk; i < (k + 1) * Mk; ++i) {
                    if (is_cand(p.mask, i)) {
                        const float l = logit[i * kTok + tl] + (p.b_local ? p.b_local[i] : 0.f);
                        s += expf(l - m);
                    }
                }
            }
            grp_max[wave][k] = m;
            grp_sum[wave][k] = s;
        }
        __syncthreads();

        // stage 1: softmax over the groups that hold a candidate
        float lmax = -INFINITY;
        for (int k = lane; k < K; k += 64) {
            if (grp_max[wave][k] != -INFINITY) {
                const float lg = logit[(M + k) * kTok + tl] + (p.b_global ? p.b_global[k] : 0.f);
                lmax = fmaxf(lmax, lg);
            }
        }
        const float gmax = wave_max(lmax);
        float lsum = 0.f;
        for (int k = lane; k < K; k += 64) {
            if (grp_max[wave][k] != -INFINITY) {
                const float lg = logit[(M + k) * kTok + tl] + (p.b_global ? p.b_global[k] : 0.f);
                lsum += expf(lg - gmax);
            }
        }
        const float gsum = wave_sum(lsum);
        for (int k = lane; k < K; k += 64) {
            float pg = 0.f;
            if (grp_max[wave][k] != -INFINITY) {
                const float lg = logit[(M + k) * kTok + tl] + (p.b_global ? p.b_global[k] : 0.f);
                pg = expf(lg - gmax) / gsum;
            }
            grp_p[wave][k] = pg;
        }
        __syncthreads();

        // fusion, Eq. 7: g_i = p_group^(k) * p_local,i^(k); -1 marks a non-candidate
        float gv[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int i = lane + 64 * q;
            gv[q] = -1.f;
            if (i < M && is_cand(p.mask, i)) {
                const int k = i / Mk;
                const float l = logit[i * kTok + tl] + (p.b_local ? p.b_local[i] : 0.f);
                const float pl = expf(l - grp_max[wave][k]) / grp_sum[wave][k];
                gv[q] = grp_p[wave][k] * pl;
            }
            if (p.probs && t < p.n_tokens && i < M)
                p.probs[static_cast<size_t>(t) * M + i] = gv[q] < 0.f ? 0.f : gv[q];
        }

        // top-k: k rounds of a wave argmax on (g, -index)
        int sel_i[kMaxTopK];
        float sel_g[kMaxTopK];
#pragma unroll
        for (int j = 0; j < kMaxTopK; ++j) {
            sel_i[j] = 0;
            sel_g[j] = 0.f;
            if (j < p.top_k) {
                float bv = -3.f;
                int bi = 0x7fffffff;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    if (gv[q] > bv) {  // ascending index: strict > keeps the lower index on ties
                        bv = gv[q];
                        bi = lane + 64 * q;
                    }
                }
#pragma unroll
                for (int off = 32; off >= 1; off >>= 1) {
                    const float ov = __shfl_xor(bv, off);
                    const int oi = __shfl_xor(bi, off);
                    if (ov > bv || (ov == bv && oi < bi)) {
                        bv = ov;
                        bi = oi;
                    }
                }
                sel_i[j] = bi;
                sel_g[j] = bv;
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    if (lane + 64 * q == bi) gv[q] = -2.f;
            }
        }

        float denom = 1.f;
        if (p.renormalize) {
            float s = 0.f;
#pragma unroll
            for (int j = 0; j < kMaxTopK; ++j)
                if (j < p.top_k) s += sel_g[j];
            denom = s;
        }
        if (t < p.n_tokens) {
#pragma unroll
            for (int j = 0; j < kMaxTopK; ++j) {
                if (j < p.top_k && lane == j) {
                    p.topk_idx[static_cast<size_t>(t) * p.top_k + j] = sel_i[j];
                    p.topk_w[static_cast<size_t>(t) * p.top_k + j] = p.renormalize ? sel_g[j] / denom : sel_g[j];
                }
            }
        }
        __syncthreads();
    }
}

template <typename T>
hipError_t launch_gate_t(const GateArgs& a, hipStream_t s) {
    const int rows_pad = ((a.n_experts + a.n_groups + 15) / 16) * 16;
    const size_t lds = static_cast<size_t>(4) * rows_pad * kTok * sizeof(float);
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&gate_kernel<T>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize,
                                           4 * 320 * kTok * sizeof(float));
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    const int grid = (a.n_tokens + kTok - 1) / kTok;
    ProfileScope prof("gate", s);
    hipLaunchKernelGGL(gate_kernel<T>, dim3(grid), dim3(256), lds, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gate(DType dt, const GateArgs& a, hipStream_t s) {
    return dt == DType::BF16 ? launch_gate_t<bf16_t>(a, s) : launch_gate_t<float>(a, s);
}

}  // namespace ec2moe
