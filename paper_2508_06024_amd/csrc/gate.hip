// Hardware-aware lightweight group gate (Local Expert Selection, Eq. 4; Lightweight
// Group Gate Network, Eq. 5-7) and top-k selection, for gfx950.
//
// One workgroup (4 or 8 waves) takes 16 tokens. Phase 1 computes the M local and K group
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
constexpr int kMaxExperts = 256;
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

// NRB: blocks of 16 gate rows (M + K <= 16 * NRB); WAVES: waves splitting d.
template <typename T, int NRB, int WAVES>
__global__ __launch_bounds__(64 * WAVES) void gate_kernel(GateArgs p) {
    extern __shared__ float part[];  // [WAVES][NRB*16 rows][16 tokens], then the sums in wave 0's slot
    __shared__ float grp_max[WAVES][kMaxGroups];
    __shared__ float grp_sum[WAVES][kMaxGroups];
    __shared__ float grp_p[WAVES][kMaxGroups];
    __shared__ float loc[WAVES][kMaxExperts];  // a wave's biased local logits, -inf off the candidate set
    __shared__ float s_bl[kMaxExperts];        // b_local (0 if absent)
    __shared__ float s_bg[kMaxGroups];         // b_global (0 if absent)

    constexpr int EPC = Elem<T>::kPerChunk;
    constexpr int SLICE = 4 * EPC;  // k covered by one matrix-core step
    // k-slices whose loads are issued together: deep for few gate rows, shallow for many
    constexpr int U = 16 / (NRB + 1) < 1 ? 1 : (16 / (NRB + 1) > 8 ? 8 : 16 / (NRB + 1));
    constexpr int THREADS = 64 * WAVES;
    constexpr int TPW = kTok / WAVES;  // tokens per wave in the softmax phase
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int g4 = lane >> 4;
    const int M = p.n_experts, K = p.n_groups, d = p.d;
    const int R = M + K;
    const int t0 = blockIdx.x * kTok;

    // biases staged once (read by the softmax phase; the barrier after phase 1 orders them)
    for (int i = threadIdx.x; i < M; i += 64 * WAVES) s_bl[i] = p.b_local ? p.b_local[i] : 0.f;
    for (int i = threadIdx.x; i < K; i += 64 * WAVES) s_bg[i] = p.b_global ? p.b_global[i] : 0.f;

    // ---------------- phase 1: partial logits over this wave's share of d
    int tok = t0 + (lane & 15);
    if (tok >= p.n_tokens) tok = p.n_tokens - 1;
    const T* xrow = static_cast<const T*>(p.x) + static_cast<size_t>(tok) * d + g4 * EPC;
    const T* wrow[NRB];
    bool wvalid[NRB];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) {
        const int r = rb * 16 + (lane & 15);
        wvalid[rb] = r < R;
        const int rr = wvalid[rb] ? r : 0;
        wrow[rb] = (rr < M ? static_cast<const T*>(p.w_local) + static_cast<size_t>(rr) * d
                           : static_cast<const T*>(p.w_global) + static_cast<size_t>(rr - M) * d) + g4 * EPC;
    }
    const int kq = d / WAVES;
    const int kbeg = wave * kq;

    f32x4 acc[NRB];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb) acc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};

    int k = kbeg;
    for (; k + U * SLICE <= kbeg + kq; k += U * SLICE) {
        uint4 bx[U], aw[U][NRB];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            bx[u] = ldg16(xrow + k + u * SLICE);
#pragma unroll
            for (int rb = 0; rb < NRB; ++rb)
                aw[u][rb] = wvalid[rb] ? ldg16(wrow[rb] + k + u * SLICE) : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int rb = 0; rb < NRB; ++rb) acc[rb] = Mfma<T>::step(aw[u][rb], bx[u], acc[rb]);
    }
    for (; k < kbeg + kq; k += SLICE) {
        const uint4 bx = ldg16(xrow + k);
#pragma unroll
        for (int rb = 0; rb < NRB; ++rb) {
            const uint4 aw = wvalid[rb] ? ldg16(wrow[rb] + k) : make_uint4(0, 0, 0, 0);
            acc[rb] = Mfma<T>::step(aw, bx, acc[rb]);
        }
    }

    constexpr int ROWS_PAD = NRB * 16;
    constexpr int N_EL = ROWS_PAD * kTok;
    float* mine = part + static_cast<size_t>(wave) * N_EL;
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i) mine[(rb * 16 + g4 * 4 + i) * kTok + (lane & 15)] = acc[rb][i];
    __syncthreads();

    // ---------------- phase 2: fixed-order sum of the partials
    for (int i = threadIdx.x; i < N_EL; i += THREADS) {
        float sum = part[i];
#pragma unroll
        for (int w = 1; w < WAVES; ++w) sum += part[w * N_EL + i];
        part[i] = sum;
    }
    __syncthreads();

    // ---------------- phase 3: two-stage softmax, fusion, top-k; TPW tokens per wave.
    // Each wave works on its own LDS rows (loc, grp_*): wave-level ordering suffices.
    const float* logit = part;  // [row][token]
    const int Mk = M / K;
    auto wave_sync = [] {
        __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's LDS writes are done
        __builtin_amdgcn_wave_barrier();
    };
    for (int it = 0; it < TPW; ++it) {
        const int tl = wave * TPW + it;
        const int t = t0 + tl;

        // biased local logits of the candidates (lane owns experts lane + 64 q)
        float lv[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int i = lane + 64 * q;
            lv[q] = -INFINITY;
            if (i < M && is_cand(p.mask, i)) lv[q] = logit[i * kTok + tl] + s_bl[i];
            if (i < M) loc[wave][i] = lv[q];
        }
        wave_sync();

        // stage 2 statistics per group over its candidates: max and sum of exp
        for (int kk = lane; kk < K; kk += 64) {
            float m = -INFINITY;
            for (int i = kk * Mk; i < (kk + 1) * Mk; ++i) m = fmaxf(m, loc[wave][i]);
            float sum = 0.f;
            if (m != -INFINITY)
                for (int i = kk * Mk; i < (kk + 1) * Mk; ++i) {
                    const float l = loc[wave][i];
                    if (l != -INFINITY) sum += expf(l - m);
                }
            grp_max[wave][kk] = m;
            grp_sum[wave][kk] = sum;
        }
        wave_sync();

        // stage 1: softmax over the groups that hold a candidate
        float lmax = -INFINITY;
        for (int kk = lane; kk < K; kk += 64)
            if (grp_max[wave][kk] != -INFINITY) lmax = fmaxf(lmax, logit[(M + kk) * kTok + tl] + s_bg[kk]);
        const float gmax = wave_max(lmax);
        float lsum = 0.f;
        for (int kk = lane; kk < K; kk += 64)
            if (grp_max[wave][kk] != -INFINITY) lsum += expf(logit[(M + kk) * kTok + tl] + s_bg[kk] - gmax);
        const float gsum = wave_sum(lsum);
        for (int kk = lane; kk < K; kk += 64) {
            float pg = 0.f;
            if (grp_max[wave][kk] != -INFINITY) pg = expf(logit[(M + kk) * kTok + tl] + s_bg[kk] - gmax) / gsum;
            grp_p[wave][kk] = pg;
        }
        wave_sync();

        // fusion, Eq. 7: g_i = p_group^(k) * p_local,i^(k); -1 marks a non-candidate
        float gv[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int i = lane + 64 * q;
            gv[q] = -1.f;
            if (lv[q] != -INFINITY) {
                const int kk = i / Mk;
                const float pl = expf(lv[q] - grp_max[wave][kk]) / grp_sum[wave][kk];
                gv[q] = grp_p[wave][kk] * pl;
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
            float sum = 0.f;
#pragma unroll
            for (int j = 0; j < kMaxTopK; ++j)
                if (j < p.top_k) sum += sel_g[j];
            denom = sum;
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
        wave_sync();  // the next token rewrites this wave's rows
    }
}

template <typename T, int NRB, int WAVES>
hipError_t launch_waves(const GateArgs& a, hipStream_t s) {
    const size_t lds = static_cast<size_t>(WAVES) * NRB * 16 * kTok * sizeof(float);
    static bool attr_set = false;  // once per instantiation: allow the partials beside the static arrays
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&gate_kernel<T, NRB, WAVES>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    const int grid = (a.n_tokens + kTok - 1) / kTok;
    ProfileScope prof("gate", s);
    hipLaunchKernelGGL((gate_kernel<T, NRB, WAVES>), dim3(grid), dim3(64 * WAVES), lds, s, a);
    return hipGetLastError();
}

// 8 waves split d when their partial logits fit in 64 KB of LDS and d splits evenly; else 4
template <typename T, int NRB>
hipError_t launch_nrb(const GateArgs& a, hipStream_t s) {
    constexpr int SLICE = 4 * Elem<T>::kPerChunk;
    if (NRB <= 8 && a.d % (8 * SLICE) == 0) return launch_waves<T, NRB, 8>(a, s);
    return launch_waves<T, NRB, 4>(a, s);
}

template <typename T>
hipError_t launch_gate_t(const GateArgs& a, hipStream_t s) {
    switch ((a.n_experts + a.n_groups + 15) / 16) {
        case 1: return launch_nrb<T, 1>(a, s);
        case 2: return launch_nrb<T, 2>(a, s);
        case 3: return launch_nrb<T, 3>(a, s);
        case 4: return launch_nrb<T, 4>(a, s);
        case 5: return launch_nrb<T, 5>(a, s);
        case 6: return launch_nrb<T, 6>(a, s);
        case 7: case 8: return launch_nrb<T, 8>(a, s);
        case 9: case 10: case 11: case 12: return launch_nrb<T, 12>(a, s);
        case 13: case 14: case 15: case 16: return launch_nrb<T, 16>(a, s);
        default: return launch_nrb<T, kMaxRowBlocks>(a, s);
    }
}

}  // namespace

hipError_t launch_gate(DType dt, const GateArgs& a, hipStream_t s) {
    return dt == DType::BF16 ? launch_gate_t<bf16_t>(a, s) : launch_gate_t<float>(a, s);
}

}  // namespace ec2moe
