// Hardware-aware lightweight group gate (Local Expert Selection, Eq. 4; Lightweight
// Group Gate Network, Eq. 5-7) and top-k selection, for gfx950.
//
// One workgroup (4 or 8 waves) takes 16 tokens. Phase 1 computes the M local and K group
// logits of those tokens with the matrix cores: gate-weight rows are the A operand,
// token rows the B operand, and each wave contracts a quarter of d. Phase 2 adds the
// partial sums in a fixed order (deterministic). Phase 3 gives each wave its tokens:
// masked group softmax (stage 1), masked in-group softmax (stage 2), the product
// g_i = p_group^(k) * p_local,i^(k), top-k by rank (ties to the lower expert index), and
// renormalisation of the selected weights.
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

// Keeps a kernel-argument value in a scalar register: left alone, the compiler may reload
// it from the argument segment at every use, and each reload waits on that memory.
template <typename V>
__device__ __forceinline__ V pin(V v) {
    asm volatile("" : "+s"(v));
    return v;
}

// e^x with the hardware 2^x (within about 1 ulp); the gate's probabilities are float32
__device__ __forceinline__ float fast_exp(float x) { return __builtin_amdgcn_exp2f(x * 1.4426950408889634f); }

// NRB: blocks of 16 gate rows (M + K <= 16 * NRB); WAVES: waves splitting d.
template <typename T, int NRB, int WAVES>
__global__ __launch_bounds__(64 * WAVES) void gate_kernel(GateArgs p) {
    extern __shared__ float part[];  // [WAVES][NRB*16 rows][16 tokens], then the sums in wave 0's slot
    __shared__ float grp_max[WAVES][kMaxGroups];
    __shared__ float grp_sum[WAVES][kMaxGroups];
    __shared__ float grp_lg[WAVES][kMaxGroups];  // a wave's biased group logits
    __shared__ float loc[WAVES][kMaxExperts];  // a wave's biased local logits (-inf off the candidate set), then g
    __shared__ float sel_g[WAVES][kMaxTopK];
    __shared__ int sel_i[WAVES][kMaxTopK];
    __shared__ float s_bl[kMaxExperts];        // b_local (0 if absent)
    __shared__ float s_bg[kMaxGroups];         // b_global (0 if absent)
    __shared__ unsigned char s_cand[kMaxExperts];  // candidate flags of the mask

    constexpr int EPC = Elem<T>::kPerChunk;
    constexpr int SLICE = 4 * EPC;  // k covered by one matrix-core step
    // k-slices whose loads are issued together: deep for few gate rows, shallow for many
    // (U (NRB + 1) uint4 registers; the budget shrinks with more waves per SIMD)
    // (one batch covers a wave's whole share of d = 4096 with 8 waves and one row block)
    constexpr int UB = WAVES <= 8 ? 40 : 16;
    constexpr int U = UB / (NRB + 1) < 1 ? 1 : (UB / (NRB + 1) > 16 ? 16 : UB / (NRB + 1));
    constexpr int THREADS = 64 * WAVES;
    constexpr int TPW = kTok / WAVES;  // tokens per wave in the softmax phase
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int g4 = lane >> 4;
    const int M = pin(p.n_experts), K = pin(p.n_groups), d = pin(p.d);
    const int KT = pin(p.top_k);
    const int n_tokens = pin(p.n_tokens);
    const bool renormalize = pin(static_cast<int>(p.renormalize)) != 0;
    float* const probs = pin(p.probs);
    int32_t* const topk_idx = pin(p.topk_idx);
    float* const topk_w = pin(p.topk_w);
    const int R = M + K;
    const int t0 = blockIdx.x * kTok;

    // biases staged once (read by the softmax phase; the barrier after phase 1 orders them)
    for (int i = threadIdx.x; i < M; i += 64 * WAVES) {
        s_bl[i] = p.b_local ? p.b_local[i] : 0.f;
        s_cand[i] = is_cand(p.mask, i) ? 1 : 0;
    }
    for (int i = threadIdx.x; i < K; i += 64 * WAVES) s_bg[i] = p.b_global ? p.b_global[i] : 0.f;

    // ---------------- phase 1: partial logits over this wave's share of d
    int tok = t0 + (lane & 15);
    if (tok >= n_tokens) tok = n_tokens - 1;
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
    // Each wave works on its own LDS rows with wave-level ordering only. Values every lane
    // needs (group softmax, the rank order) are read back from LDS by all lanes in the
    // same order instead of cross-lane shuffles, whose latency chains dominated.
    const float* logit = part;  // [row][token]
    const int Mk = M / K;
    const int Mpad = (M + 3) & ~3;
    auto wave_sync = [] {
        __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's LDS traffic is done
        __builtin_amdgcn_wave_barrier();
    };
    for (int it = 0; it < TPW; ++it) {
        const int tl = wave * TPW + it;
        const int t = t0 + tl;
        float* gl = loc[wave];

        // biased logits: local ones of the candidates (lane owns experts lane + 64 q), group ones
        float lv[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int i = lane + 64 * q;
            lv[q] = -INFINITY;
            if (i < M && s_cand[i]) lv[q] = logit[i * kTok + tl] + s_bl[i];
            if (i < M) gl[i] = lv[q];
        }
        for (int kk = lane; kk < K; kk += 64) grp_lg[wave][kk] = logit[(M + kk) * kTok + tl] + s_bg[kk];
        wave_sync();

        // stage 2 statistics per group over its candidates: max and sum of exp
        for (int kk = lane; kk < K; kk += 64) {
            float m = -INFINITY;
            for (int i = kk * Mk; i < (kk + 1) * Mk; ++i) m = fmaxf(m, gl[i]);
            float sum = 0.f;
            if (m != -INFINITY)
                for (int i = kk * Mk; i < (kk + 1) * Mk; ++i) {
                    const float l = gl[i];
                    if (l != -INFINITY) sum += fast_exp(l - m);
                }
            grp_max[wave][kk] = m;
            grp_sum[wave][kk] = sum;
        }
        wave_sync();

        // stage 1: softmax over the groups that hold a candidate (every lane, group order)
        float gmax = -INFINITY;
        for (int kk = 0; kk < K; ++kk)
            if (grp_max[wave][kk] != -INFINITY) gmax = fmaxf(gmax, grp_lg[wave][kk]);
        float gsum = 0.f;
        for (int kk = 0; kk < K; ++kk)
            if (grp_max[wave][kk] != -INFINITY) gsum += fast_exp(grp_lg[wave][kk] - gmax);
        const float rgsum = __builtin_amdgcn_rcpf(gsum);

        // fusion, Eq. 7: g_i = p_group^(k) * p_local,i^(k); -1 marks a non-candidate
        float gv[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int i = lane + 64 * q;
            gv[q] = -1.f;
            if (lv[q] != -INFINITY) {
                const int kk = i / Mk;
                const float pg = fast_exp(grp_lg[wave][kk] - gmax) * rgsum;
                const float pl = fast_exp(lv[q] - grp_max[wave][kk]) * __builtin_amdgcn_rcpf(grp_sum[wave][kk]);
                gv[q] = pg * pl;
            }
            if (probs && t < n_tokens && i < M) probs[static_cast<size_t>(t) * M + i] = gv[q] < 0.f ? 0.f : gv[q];
        }
        wave_sync();  // every lane is done with the local logits
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int i = lane + 64 * q;
            if (i < Mpad) gl[i] = i < M ? gv[q] : -1.f;
        }
        wave_sync();

        // top-k by rank: a larger g, or an equal g at a lower index, ranks first
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int i = lane + 64 * q;
            if (gv[q] >= 0.f) {
                const float g = gv[q];
                int r = 0;
                for (int j = 0; j < Mpad; j += 4) {
                    const f32x4 o = *reinterpret_cast<const f32x4*>(gl + j);
#pragma unroll
                    for (int u = 0; u < 4; ++u) r += (o[u] > g || (o[u] == g && j + u < i)) ? 1 : 0;
                }
                if (r < KT) {
                    sel_g[wave][r] = g;
                    sel_i[wave][r] = i;
                }
            }
        }
        wave_sync();

        // slot j of the output (lane j); renormalised by the sum in slot order
        float denom = 1.f;
        if (renormalize) {
            float sum = 0.f;
            for (int j = 0; j < KT; ++j) sum += sel_g[wave][j];
            denom = sum;
        }
        if (t < n_tokens && lane < KT) {
            topk_idx[static_cast<size_t>(t) * KT + lane] = sel_i[wave][lane];
            topk_w[static_cast<size_t>(t) * KT + lane] = renormalize ? sel_g[wave][lane] / denom : sel_g[wave][lane];
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

// 8 waves split d when their partial logits fit in 64 KB of LDS and d splits evenly, else
// 4; with fewer token blocks than CUs (small batches) 16 waves shorten each wave's walk
// over d.
template <typename T, int NRB>
hipError_t launch_nrb(const GateArgs& a, hipStream_t s) {
    constexpr int SLICE = 4 * Elem<T>::kPerChunk;
    const int blocks = (a.n_tokens + kTok - 1) / kTok;
    if constexpr (NRB <= 6)
        if (blocks < 256 && a.d % (16 * SLICE) == 0) return launch_waves<T, NRB, 16>(a, s);
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
