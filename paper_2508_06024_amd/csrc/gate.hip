// Hardware-aware lightweight group gate (Local Expert Selection, Eq. 4; Lightweight
// Group Gate Network, Eq. 5-7) and top-k selection, for gfx950.
//
// One workgroup takes a tile of TT = 16 * NB tokens. Phase 1 computes the M local and K
// group logits of the tile with the matrix cores: gate-weight rows are the A operand,
// token rows the B operand, and each of the WAVES waves contracts its share of d (all
// its loads of a batch issued before the first MFMA). Phase 2 adds the partial sums in a
// fixed order (deterministic) and the biases, and sets the local logits of non-candidates
// to -inf. Phase 3 routes the tokens from the logits in LDS:
//   * regular shapes (M a multiple of 8 up to 64, each lane's M/8 experts inside one
//     group): 8 lanes per token, segmented shuffles for the two softmaxes (stage 2 inside
//     the groups, stage 1 over the groups), per-lane top-k lists of packed keys merged
//     bitonically, with an exact re-selection for keys that collide after truncation;
//   * other shapes (unequal groups, more than 64 experts, k = 16): one lane per token,
//     the group statistics in LDS and a running top-k in registers.
// Either way ties go to the lower expert index and the selected weights are renormalised
// on request.
//
// Tiles of two 16-token blocks (NB = 2) halve the gate-weight reads per token; they pay
// off when the gate has many rows and there are enough tokens to give every CU a tile.
// Small batches with a caller-given workspace split d over several workgroups per tile
// (MODE 1, partial logits to the workspace) and route in a second launch (MODE 2, the
// partials summed in split order in place of phase 1).
#include "device_common.h"
#include "internal.h"

namespace ec2moe {
namespace {

constexpr int kBlock = 16;          // tokens per MFMA block
constexpr int kMaxRowBlocks = 20;   // M + K <= 320 gate rows
constexpr int kMaxGroups = 160;
constexpr int kMaxExperts = 256;
constexpr int kChunk = 8;           // logits of one group read together in phase 3
constexpr int kSplitWaves = 4;      // waves of the split-d workgroups (small batches)
constexpr int kSplitMaxTiles = 64;  // 16-token tiles below which d is split (given a workspace)
constexpr int kMaxSplit = 32;       // d-splits per tile at most
constexpr int kSplitMinD = 2048;    // narrower gates run unsplit (the second launch costs more)
constexpr int kRouteWaves = 8;      // waves of the routing workgroups after a split (16 up to 96 rows)

// Keeps a kernel-argument value in a scalar register: left alone, the compiler may reload
// it from the argument segment at every use, and each reload waits on that memory.
template <typename V>
__device__ __forceinline__ V pin(V v) {
    asm volatile("" : "+s"(v));
    return v;
}

// e^x with the hardware 2^x (within about 1 ulp); the gate's probabilities are float32
__device__ __forceinline__ float fast_exp(float x) { return __builtin_amdgcn_exp2f(x * 1.4426950408889634f); }

// Inserts (g, i) into the descending list (sv, si) of KP entries. Candidates arrive in
// ascending index order and only a strictly larger g moves an entry down, so equal
// values keep the lower index first.
template <int KP>
__device__ __forceinline__ void topk_insert(float (&sv)[KP], int (&si)[KP], float g, int i) {
#pragma unroll
    for (int j = KP - 1; j > 0; --j) {
        const bool above = g > sv[j - 1];
        const bool here = g > sv[j];
        sv[j] = above ? sv[j - 1] : (here ? g : sv[j]);
        si[j] = above ? si[j - 1] : (here ? i : si[j]);
    }
    const bool top = g > sv[0];
    sv[0] = top ? g : sv[0];
    si[0] = top ? i : si[0];
}

// Butterfly over the lanes of an aligned segment of `width` lanes (a power of two <= 8).
__device__ __forceinline__ float seg_max(float v, int width) {
    for (int off = 1; off < width; off <<= 1) v = fmaxf(v, __shfl_xor(v, off, 8));
    return v;
}
__device__ __forceinline__ float seg_sum(float v, int width) {
    for (int off = 1; off < width; off <<= 1) v += __shfl_xor(v, off, 8);
    return v;
}

// Routing of token tl of the tile by its 8 lanes (sub-lane s holds experts s*EPL ..
// s*EPL + EPL - 1, EPL = M / 8, all in group (s*EPL) / Mk, whose LG = Mk / EPL lanes are
// aligned). Logits come from the summed, biased, masked rows in LDS; the token's fused
// probabilities are kept in the second tile-sized slot of the LDS for the outputs.
//   stage 2: group max and sum of e^(l - max), lane-local then across the group's lanes;
//   stage 1: softmax over the groups that hold a candidate, across the 8 lanes;
//   with top_groups, each lane ranks its group among the groups' logits and leaves it out
//   unless fewer than top_groups groups, or groups holding fewer than k candidates, rank
//   before it;
//   fusion (Eq. 7) and top-k: every lane keeps its experts' keys (g truncated to its
//   top 24 bits, then 255 - i) sorted, then three bitonic merges across the lanes leave
//   the token's first KP keys in every lane. Distinct truncated values order as the
//   exact ones; if two of the first k + 1 keys share their truncated g, lane 0 redoes the
//   selection exactly from the stored probabilities (ties to the lower index).
template <int KP>
__device__ __forceinline__ void route_octet(float* part, int n_el, int TT, int tl, int s, int t0, int n_tokens,
                                            int M, int Mk, int KT, bool renormalize, float* probs,
                                            int32_t* topk_idx, float* topk_w, int top_groups, const short* gcand) {
    const int EPL = M >> 3;
    const int LG = Mk / EPL;
    const int t = t0 + tl;
    const bool live = t < n_tokens;
    const float* lg = part;
    float* gb = part + n_el + static_cast<size_t>(tl) * M;  // this token's g, -1 off the candidate set
    const int i0 = s * EPL;
    const int grp = i0 / Mk;

    float v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = j < EPL ? lg[(i0 + j) * TT + tl] : -INFINITY;
    const float G = lg[(M + grp) * TT + tl];

    float m = v[0];
#pragma unroll
    for (int j = 1; j < 8; ++j) m = fmaxf(m, v[j]);
    m = seg_max(m, LG);
    const bool active = m != -INFINITY;
    float sum = 0.f;
    if (active) {
#pragma unroll
        for (int j = 0; j < 8; ++j)
            if (v[j] != -INFINITY) sum += fast_exp(v[j] - m);
    }
    sum = seg_sum(sum, LG);

    const float gmax = seg_max(active ? G : -INFINITY, 8);
    const bool leader = (s & (LG - 1)) == 0;
    const float gsum = seg_sum(leader && active ? fast_exp(G - gmax) : 0.f, 8);
    const float pg = fast_exp(G - gmax) * __builtin_amdgcn_rcpf(gsum);
    const float rs = __builtin_amdgcn_rcpf(sum);
    // Group-focused evaluation: this lane's group is kept if fewer than top_groups active groups
    // rank before it (larger logit, or equal at a lower index) or those hold fewer than k
    // candidates. Every group's logit comes from its first lane.
    bool kept = active;
    if (top_groups > 0) {
        const int K = M / Mk;
        int rank = 0, before = 0;
        for (int kk = 0; kk < K; ++kk) {
            const float Gk = __shfl(G, (kk * Mk / EPL) & 7, 8);
            const bool ak = gcand[kk] > 0;
            if (ak && (Gk > G || (Gk == G && kk < grp))) {
                ++rank;
                before += gcand[kk];
            }
        }
        kept = active && (rank < top_groups || before < KT);
    }

    uint32_t sk[KP];
#pragma unroll
    for (int j = 0; j < KP; ++j) sk[j] = 0;
    float* prow = probs && live ? probs + static_cast<size_t>(t) * M : nullptr;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        if (j < EPL) {
            const int i = i0 + j;
            float g = -1.f;
            if (kept && v[j] != -INFINITY) {
                g = pg * (fast_exp(v[j] - m) * rs);
                const uint32_t key = ((__float_as_uint(g) << 2) & 0xffffff00u) | static_cast<uint32_t>(255 - i);
#pragma unroll
                for (int q = KP - 1; q > 0; --q) sk[q] = max(sk[q], min(sk[q - 1], key));
                sk[0] = max(sk[0], key);
            }
            gb[i] = g;
            if (prow) prow[i] = g < 0.f ? 0.f : g;
        }
    }
    // merge with the lists of the lanes 1, 2, 4 apart: the elementwise max of one list and
    // the other reversed is bitonic and holds the first KP of both; sort it descending
#pragma unroll
    for (int off = 1; off < 8; off <<= 1) {
        uint32_t o[KP];
#pragma unroll
        for (int j = 0; j < KP; ++j) o[j] = __shfl_xor(sk[j], off, 8);
#pragma unroll
        for (int j = 0; j < KP; ++j) sk[j] = max(sk[j], o[KP - 1 - j]);
#pragma unroll
        for (int len = KP / 2; len >= 1; len >>= 1)
#pragma unroll
            for (int j = 0; j < KP; ++j)
                if ((j & len) == 0) {
                    const uint32_t a = sk[j], b = sk[j + len];
                    sk[j] = max(a, b);
                    sk[j + len] = min(a, b);
                }
    }
    bool amb = false;
#pragma unroll
    for (int j = 0; j + 1 < KP; ++j)
        if (j < KT && (sk[j] >> 8) == (sk[j + 1] >> 8)) amb = true;
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's probabilities are in LDS
    __builtin_amdgcn_wave_barrier();
    if (!live) return;
    int32_t* oi = topk_idx + static_cast<size_t>(t) * KT;
    float* ow = topk_w + static_cast<size_t>(t) * KT;
    if (!amb) {
        float gs[KP];
        float denom = 0.f;
#pragma unroll
        for (int j = 0; j < KP; ++j) {
            gs[j] = j < KT ? gb[255 - static_cast<int>(sk[j] & 0xffu)] : 0.f;
            if (j < KT) denom += gs[j];
        }
#pragma unroll
        for (int j = 0; j < KP; ++j)
            if (j < KT && (j & 7) == s) {
                oi[j] = 255 - static_cast<int>(sk[j] & 0xffu);
                ow[j] = renormalize ? gs[j] / denom : gs[j];
            }
        return;
    }
    if (s != 0) return;
    float sv[KP];
    int si[KP];
#pragma unroll
    for (int j = 0; j < KP; ++j) {
        sv[j] = -1.f;
        si[j] = 0;
    }
    for (int c = 0; c < M; c += 8) {
        float g[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) g[u] = gb[c + u];  // M is a multiple of 8
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (g[u] >= 0.f) topk_insert<KP>(sv, si, g[u], c + u);
    }
    float denom = 0.f;
#pragma unroll
    for (int j = 0; j < KP; ++j)
        if (j < KT) denom += sv[j];
#pragma unroll
    for (int j = 0; j < KP; ++j)
        if (j < KT) {
            oi[j] = si[j];
            ow[j] = renormalize ? sv[j] / denom : sv[j];
        }
}

// NRB: blocks of 16 gate rows (M + K <= 16 * NRB); NB: 16-token blocks per tile;
// WAVES: waves splitting d; KP: top-k list length (>= k).
// MODE 0: the whole gate for a tile. MODE 1 (small batches): phase 1 over the d-range
// blockIdx.y of p.nsplit, the waves' partials summed in order and written to p.ws
// ([tile][split][row][token]). MODE 2: phase 1 replaced by the sum of a tile's split
// partials from p.ws in split order, then phases 2 and 3.
template <typename T, int NRB, int NB, int WAVES, int KP, int MODE>
__global__ __launch_bounds__(64 * WAVES) void gate_kernel(GateArgs p) {
    constexpr int TT = kBlock * NB;
    static_assert(TT <= 64, "phase 3 gives each token one lane of wave 0");
    extern __shared__ float part[];  // [WAVES][NRB*16 rows][TT tokens]; sums land in wave 0's slot
    __shared__ float s_bl[kMaxExperts];            // b_local (0 if absent)
    __shared__ float s_bg[kMaxGroups];             // b_global (0 if absent)
    __shared__ unsigned char s_cand[kMaxExperts];  // candidate flags of the mask
    __shared__ unsigned char s_grp[kMaxExperts];   // group of each expert
    __shared__ short s_gcand[kMaxGroups];          // candidates per group

    constexpr int EPC = Elem<T>::kPerChunk;
    constexpr int SLICE = 4 * EPC;  // k covered by one matrix-core step
    // k-slices whose loads are issued together: U * (NB + NRB) 16-byte registers per lane
    constexpr int UB = WAVES <= 8 ? (NB * NRB >= 16 ? 30 : 40) : 16;  // 16 accumulator blocks: fewer in flight
    constexpr int U = UB / (NB + NRB) < 1 ? 1 : (UB / (NB + NRB) > 16 ? 16 : UB / (NB + NRB));
    constexpr int THREADS = 64 * WAVES;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int g4 = lane >> 4;
    const int M = pin(p.n_experts), K = pin(p.n_groups), d = pin(p.d);
    const int n_tokens = pin(p.n_tokens);
    const int R = M + K;
    const int Mk = M / K;
    const int t0 = blockIdx.x * TT;

    // mask and biases staged once (read by phase 2 after the first barrier)
    for (int i = threadIdx.x; i < M; i += THREADS) {
        s_bl[i] = p.b_local ? p.b_local[i] : 0.f;
        s_cand[i] = (p.mask[i >> 6] >> (i & 63)) & 1ull ? 1 : 0;
    }
    for (int kk = threadIdx.x; kk < K; kk += THREADS) {
        s_bg[kk] = p.b_global ? p.b_global[kk] : 0.f;
        int n = 0;
        for (int i = p.goff[kk]; i < p.goff[kk + 1]; ++i) {
            s_grp[i] = static_cast<unsigned char>(kk);
            n += static_cast<int>((p.mask[i >> 6] >> (i & 63)) & 1ull);
        }
        s_gcand[kk] = static_cast<short>(n);
    }

    constexpr int N_EL = NRB * 16 * TT;
    if constexpr (MODE != 2) {
    // ---------------- phase 1: partial logits over this wave's share of d
    const T* xrow[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        int tok = t0 + nb * kBlock + (lane & 15);
        if (tok >= n_tokens) tok = n_tokens - 1;
        xrow[nb] = static_cast<const T*>(p.x) + static_cast<size_t>(tok) * d + g4 * EPC;
    }
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
    const int dsplit = MODE == 1 ? d / p.nsplit : d;  // d-range of this workgroup
    const int kq = dsplit / WAVES;
    const int kbeg = (MODE == 1 ? blockIdx.y * dsplit : 0) + wave * kq;

    f32x4 acc[NRB][NB];
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[rb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

    // batches of U slices; the last batch of a wave may be partial (its missing slices
    // contribute zero products)
    const int kend = kbeg + kq;
    for (int k = kbeg; k < kend; k += U * SLICE) {
        uint4 bx[U][NB], aw[U][NRB];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const bool in = k + u * SLICE < kend;
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) bx[u][nb] = in ? ldg16(xrow[nb] + k + u * SLICE) : make_uint4(0, 0, 0, 0);
#pragma unroll
            for (int rb = 0; rb < NRB; ++rb)
                aw[u][rb] = in && wvalid[rb] ? ldg16(wrow[rb] + k + u * SLICE) : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) acc[rb][nb] = Mfma<T>::step(aw[u][rb], bx[u][nb], acc[rb][nb]);
    }

    float* mine = part + static_cast<size_t>(wave) * N_EL;
#pragma unroll
    for (int rb = 0; rb < NRB; ++rb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int i = 0; i < 4; ++i) mine[(rb * 16 + g4 * 4 + i) * TT + nb * kBlock + (lane & 15)] = acc[rb][nb][i];
    __syncthreads();
    if constexpr (MODE == 1) {
        float* out = p.ws + (static_cast<size_t>(blockIdx.x) * p.nsplit + blockIdx.y) * N_EL;
        for (int i = threadIdx.x; i < N_EL; i += THREADS) {
            float sum = part[i];
#pragma unroll
            for (int w = 1; w < WAVES; ++w) sum += part[w * N_EL + i];
            out[i] = sum;
        }
        return;
    }
    }

    if constexpr (MODE == 2) __syncthreads();  // the staged mask and biases
    // ---------------- phase 2: fixed-order sum of the partials, then the biases; local
    // logits off the candidate set become -inf (Eq. 4 applied before both softmaxes)
    for (int i = threadIdx.x; i < N_EL; i += THREADS) {
        float sum;
        if constexpr (MODE == 2) {
            // all the split partials of this logit loaded together, then added in split order
            const float* src = p.ws + static_cast<size_t>(blockIdx.x) * p.nsplit * N_EL + i;
            float v[kMaxSplit];
#pragma unroll
            for (int q = 0; q < kMaxSplit; ++q) v[q] = q < p.nsplit ? src[static_cast<size_t>(q) * N_EL] : 0.f;
            sum = v[0];
#pragma unroll
            for (int q = 1; q < kMaxSplit; ++q)
                if (q < p.nsplit) sum += v[q];
        } else {
            sum = part[i];
#pragma unroll
            for (int w = 1; w < WAVES; ++w) sum += part[w * N_EL + i];
        }
        const int r = i / TT;
        if (r < M) sum = s_cand[r] ? sum + s_bl[r] : -INFINITY;
        else if (r < R) sum += s_bg[r - M];
        part[i] = sum;
    }
    __syncthreads();

    // ---------------- phase 3
    const int KT = pin(p.top_k);
    const bool renormalize = pin(static_cast<int>(p.renormalize)) != 0;
    float* const probs = pin(p.probs);
    // Regular shapes (M a multiple of 8 up to 64, the experts of each of 8 lanes inside one
    // group, whose lanes are a power of two): 8 lanes per token.
    const int EPL = M >> 3;
    const int LG = EPL > 0 ? Mk / EPL : 0;
    const int top_groups = pin(p.top_groups);
    const bool prune = top_groups > 0 && top_groups < K;
    if (p.equal_groups && (M & 7) == 0 && M <= 64 && Mk % EPL == 0 && (LG & (LG - 1)) == 0 && KT < KP) {
        if (wave * 8 >= TT) return;
        route_octet<KP>(part, N_EL, TT, wave * 8 + (lane >> 3), lane & 7, t0, n_tokens, M, Mk, KT, renormalize,
                        probs, p.topk_idx, p.topk_w, prune ? top_groups : 0, s_gcand);
        return;
    }

    // General shapes (unequal groups and top-G groups included): one lane per token of the tile.
    if (wave != 0) return;
    const int tl = lane;
    const int t = t0 + tl;
    if (tl >= TT || t >= n_tokens) return;
    const float* lg = part;    // biased logits [row][TT], -inf off the candidate set
    float* gst = part + N_EL;  // this lane's stage-2 statistics: max at [kk][TT], sum at [K + kk][TT]
                               // (the second tile-sized slot of the LDS; N_EL >= 2 K TT since M >= K)

    // stage 2 statistics per group: max over its candidates and the sum of e^(l - max) in
    // expert order; stage 1 maximum over the groups that hold a candidate
    float gmax = -INFINITY;
    for (int kk = 0; kk < K; ++kk) {
        const int i0 = p.goff[kk];
        const int mk = p.goff[kk + 1] - i0;
        const float G = lg[(M + kk) * TT + tl];
        float m = -INFINITY, s = 0.f;
        if (mk <= kChunk) {
            float v[kChunk];
#pragma unroll
            for (int u = 0; u < kChunk; ++u) v[u] = u < mk ? lg[(i0 + u) * TT + tl] : -INFINITY;
#pragma unroll
            for (int u = 0; u < kChunk; ++u) m = fmaxf(m, v[u]);
            if (m != -INFINITY) {
#pragma unroll
                for (int u = 0; u < kChunk; ++u)
                    if (v[u] != -INFINITY) s += fast_exp(v[u] - m);
            }
        } else {
            for (int c = 0; c < mk; c += kChunk) {
                float v[kChunk];
#pragma unroll
                for (int u = 0; u < kChunk; ++u) v[u] = c + u < mk ? lg[(i0 + c + u) * TT + tl] : -INFINITY;
#pragma unroll
                for (int u = 0; u < kChunk; ++u) m = fmaxf(m, v[u]);
            }
            if (m != -INFINITY)
                for (int c = 0; c < mk; c += kChunk) {
                    float v[kChunk];
#pragma unroll
                    for (int u = 0; u < kChunk; ++u) v[u] = c + u < mk ? lg[(i0 + c + u) * TT + tl] : -INFINITY;
#pragma unroll
                    for (int u = 0; u < kChunk; ++u)
                        if (v[u] != -INFINITY) s += fast_exp(v[u] - m);
                }
        }
        gst[kk * TT + tl] = m;
        gst[(K + kk) * TT + tl] = s;
        if (m != -INFINITY) gmax = fmaxf(gmax, G);
    }
    // stage 1: softmax over the groups that hold a candidate
    float gsum = 0.f;
    for (int kk = 0; kk < K; ++kk)
        if (gst[kk * TT + tl] != -INFINITY) gsum += fast_exp(lg[(M + kk) * TT + tl] - gmax);
    const float rgsum = __builtin_amdgcn_rcpf(gsum);

    // Group-focused evaluation: keep the groups with the largest group logits (the order of
    // p_group; ties to the lower group index) until top_groups are kept and they hold at
    // least k candidates; the others leave the fusion (their statistics row becomes -inf,
    // after p_group has been formed over all of them).
    if (prune) {
        float* taken = part + 2 * N_EL;  // this lane's flags [kk][TT] (the third slot)
        for (int kk = 0; kk < K; ++kk) taken[kk * TT + tl] = 0.f;
        int kept = 0, held = 0;
        for (int n = 0; n < K && (kept < top_groups || held < KT); ++n) {
            float best = -INFINITY;
            int bk = -1;
            for (int kk = 0; kk < K; ++kk) {
                if (gst[kk * TT + tl] == -INFINITY || taken[kk * TT + tl] != 0.f) continue;
                const float G = lg[(M + kk) * TT + tl];
                if (bk < 0 || G > best) {
                    best = G;
                    bk = kk;
                }
            }
            if (bk < 0) break;
            taken[bk * TT + tl] = 1.f;
            ++kept;
            held += s_gcand[bk];
        }
        for (int kk = 0; kk < K; ++kk)
            if (taken[kk * TT + tl] == 0.f) gst[kk * TT + tl] = -INFINITY;
    }

    // Fusion (Eq. 7) of expert i of group kk: g_i = p_group^(kk) * p_local,i^(kk). The same
    // expression everywhere below, so a recomputed g has the same bits.
    auto fused = [&](int kk, float v) {
        const float pg = fast_exp(lg[(M + kk) * TT + tl] - gmax) * rgsum;
        return pg * (fast_exp(v - gst[kk * TT + tl]) * __builtin_amdgcn_rcpf(gst[(K + kk) * TT + tl]));
    };
    float* prow = probs ? probs + static_cast<size_t>(t) * M : nullptr;
    int32_t* oi = p.topk_idx + static_cast<size_t>(t) * KT;
    float* ow = p.topk_w + static_cast<size_t>(t) * KT;

    // Fast top-k: keys (g truncated to its top 24 bits, then 255 - i) kept sorted by a
    // min/max network, two instructions per slot. Distinct truncated values order as the
    // exact ones, so the result is exact unless two of the first k + 1 keys share their
    // truncated g; such tokens take the exact pass below.
    bool exact_pass = KT >= KP;
    if (!exact_pass) {
        uint32_t sk[KP];
#pragma unroll
        for (int j = 0; j < KP; ++j) sk[j] = 0;
        for (int kk = 0; kk < K; ++kk) {
            const int i0 = p.goff[kk];
            const int mk = p.goff[kk + 1] - i0;
            for (int c = 0; c < mk; c += kChunk) {
                float v[kChunk];
#pragma unroll
                for (int u = 0; u < kChunk; ++u) v[u] = c + u < mk ? lg[(i0 + c + u) * TT + tl] : -INFINITY;
                if (gst[kk * TT + tl] == -INFINITY) {  // no candidate in this group, or a group left out
                    if (prow)
                        for (int u = 0; u < kChunk && c + u < mk; ++u) prow[i0 + c + u] = 0.f;
                    continue;
                }
                const float pg = fast_exp(lg[(M + kk) * TT + tl] - gmax) * rgsum;
                const float m = gst[kk * TT + tl];
                const float rs = __builtin_amdgcn_rcpf(gst[(K + kk) * TT + tl]);
#pragma unroll
                for (int u = 0; u < kChunk; ++u) {
                    if (c + u >= mk) break;
                    const int i = i0 + c + u;
                    float g = 0.f;
                    if (v[u] != -INFINITY) {
                        g = pg * (fast_exp(v[u] - m) * rs);
                        const uint32_t key = ((__float_as_uint(g) << 2) & 0xffffff00u) | static_cast<uint32_t>(255 - i);
#pragma unroll
                        for (int j = KP - 1; j > 0; --j) sk[j] = max(sk[j], min(sk[j - 1], key));
                        sk[0] = max(sk[0], key);
                    }
                    if (prow) prow[i] = g;
                }
            }
        }
#pragma unroll
        for (int j = 0; j + 1 < KP; ++j)
            if (j < KT && (sk[j] >> 8) == (sk[j + 1] >> 8)) exact_pass = true;
        if (!exact_pass) {
            float gs[KP];
            float denom = 0.f;
#pragma unroll
            for (int j = 0; j < KP; ++j) {
                if (j < KT) {
                    const int i = 255 - static_cast<int>(sk[j] & 0xffu);
                    gs[j] = fused(s_grp[i], lg[i * TT + tl]);
                    denom += gs[j];
                    oi[j] = i;
                }
            }
#pragma unroll
            for (int j = 0; j < KP; ++j)
                if (j < KT) ow[j] = renormalize ? gs[j] / denom : gs[j];
            return;
        }
    }

    // Exact top-k: (g, i) pairs kept sorted in expert order (ties to the lower index).
    float sv[KP];
    int si[KP];
#pragma unroll
    for (int j = 0; j < KP; ++j) {
        sv[j] = -1.f;  // below every probability
        si[j] = 0;
    }
    const bool write_probs = prow && KT >= KP;  // the fast pass has written them otherwise
    for (int kk = 0; kk < K; ++kk) {
        const int i0 = p.goff[kk];
        const bool active = gst[kk * TT + tl] != -INFINITY;
        for (int i = i0; i < p.goff[kk + 1]; ++i) {
            const float v = lg[i * TT + tl];
            float g = 0.f;
            if (active && v != -INFINITY) {
                g = fused(kk, v);
                topk_insert<KP>(sv, si, g, i);
            }
            if (write_probs) prow[i] = g;
        }
    }
    float denom = 0.f;
#pragma unroll
    for (int j = 0; j < KP; ++j)
        if (j < KT) denom += sv[j];
#pragma unroll
    for (int j = 0; j < KP; ++j) {
        if (j < KT) {
            oi[j] = si[j];
            ow[j] = renormalize ? sv[j] / denom : sv[j];
        }
    }
}

template <typename T, int NRB, int NB, int WAVES, int KP, int MODE>
hipError_t launch_cfg(const GateArgs& a, hipStream_t s) {
    constexpr int TT = kBlock * NB;
    // MODE 2 keeps no per-wave partials: the logits, the routing statistics and the flags of
    // top-G pruning take three tile-sized slots
    const size_t lds = static_cast<size_t>(MODE == 2 ? 3 : WAVES) * NRB * 16 * TT * sizeof(float);
    static bool attr_set = false;  // once per instantiation: allow the partials beside the static arrays
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&gate_kernel<T, NRB, NB, WAVES, KP, MODE>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    const int grid = (a.n_tokens + TT - 1) / TT;
    ProfileScope prof(MODE == 1 ? "gate_split" : "gate", s);
    hipLaunchKernelGGL((gate_kernel<T, NRB, NB, WAVES, KP, MODE>), dim3(grid, MODE == 1 ? a.nsplit : 1),
                       dim3(64 * WAVES), lds, s, a);
    return hipGetLastError();
}

// KP > k lets the fast top-k see the (k+1)-th key; k = 16 runs the exact pass only
template <typename T, int NRB, int NB, int WAVES, int MODE = 0>
hipError_t launch_kp(const GateArgs& a, hipStream_t s) {
    if (a.top_k <= 1) return launch_cfg<T, NRB, NB, WAVES, 2, MODE>(a, s);
    if (a.top_k <= 3) return launch_cfg<T, NRB, NB, WAVES, 4, MODE>(a, s);
    if (a.top_k <= 7) return launch_cfg<T, NRB, NB, WAVES, 8, MODE>(a, s);
    return launch_cfg<T, NRB, NB, WAVES, 16, MODE>(a, s);
}

// Tile and wave split:
//   * fewer 16-token tiles than CUs (small batches): 16 waves shorten each wave's walk
//     over d (gates of at most 96 rows, whose partials fit the LDS);
//   * gates of 48..128 rows with at least two tiles per CU: 32-token tiles, 8 waves
//     (the gate weights are then read once per 32 tokens instead of per 16);
//   * otherwise 16-token tiles with 8 waves when d splits evenly, else 4.
template <typename T, int NRB>
hipError_t launch_nrb(const GateArgs& a, hipStream_t s) {
    constexpr int SLICE = 4 * Elem<T>::kPerChunk;
    const int tiles16 = (a.n_tokens + kBlock - 1) / kBlock;
    if (a.ws && a.nsplit > 1) {
        // small batch with a workspace: d split over nsplit workgroups per tile, then routing
        hipError_t e = launch_cfg<T, NRB, 1, kSplitWaves, 2, 1>(a, s);
        if (e != hipSuccess) return e;
        if constexpr (NRB <= 6) return launch_kp<T, NRB, 1, 16, 2>(a, s);  // more loads of partials in flight
        return launch_kp<T, NRB, 1, kRouteWaves, 2>(a, s);
    }
    if constexpr (NRB <= 6)
        if (tiles16 < 256 && a.d % (16 * SLICE) == 0) return launch_kp<T, NRB, 1, 16>(a, s);
    if constexpr (NRB >= 3 && NRB <= 8)
        if (tiles16 >= 512 && a.d % (8 * SLICE) == 0) return launch_kp<T, NRB, 2, 8>(a, s);
    if constexpr (NRB <= 8)
        if (a.d % (8 * SLICE) == 0) return launch_kp<T, NRB, 1, 8>(a, s);
    return launch_kp<T, NRB, 1, 4>(a, s);
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

int gate_split_count(DType dt, int n_tokens, int d) {
    const int tiles16 = (n_tokens + kBlock - 1) / kBlock;
    if (n_tokens <= 0 || tiles16 >= kSplitMaxTiles || d < kSplitMinD) return 1;
    const int slice = 4 * (dt == DType::BF16 ? Elem<bf16_t>::kPerChunk : Elem<float>::kPerChunk);
    // powers of two dividing the number of kSplitWaves-wave slices of d, up to about
    // 256 workgroups and kMaxSplit splits
    int n = 1;
    while (n < kMaxSplit && tiles16 * n * 2 <= 256 && d % (2 * n * kSplitWaves * slice) == 0) n *= 2;
    return n;
}

size_t gate_split_bytes(DType dt, int n_tokens, int d, int gate_rows) {
    const int n = gate_split_count(dt, n_tokens, d);
    if (n <= 1) return 0;
    const int nrb = (gate_rows + 15) / 16;
    const int padded = nrb <= 6 ? nrb : (nrb <= 8 ? 8 : (nrb <= 12 ? 12 : (nrb <= 16 ? 16 : kMaxRowBlocks)));
    const size_t tiles16 = (static_cast<size_t>(n_tokens) + kBlock - 1) / kBlock;
    return tiles16 * n * static_cast<size_t>(padded) * 16 * kBlock * sizeof(float);
}

}  // namespace ec2moe
