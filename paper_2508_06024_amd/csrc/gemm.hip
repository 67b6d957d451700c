// Grouped and dense "NT" GEMM on the gfx950 matrix cores.
//
//   out[p][n] = sum_k tok[row(p)][k] * w_e[n][k]     for every row p of group e
//
// Both operands are K-contiguous (token rows of the activations, rows of nn.Linear-style
// weights), which is the layout the expert networks of Eq. 1 and the codec products use.
// Groups are the per-expert segments produced by the permutation; their sizes stay on
// the device. Every workgroup counts the real tiles with a wave-parallel prefix sum over
// the segment table and maps logical tile ids to (group, m-tile, n-tile).
//
// Tile order (XCD-aware): workgroups are dispatched round-robin over the 8 XCDs, each with
// its own L2. Within a group, m-tiles go in bands of at most 8 and a band's n-tiles run in
// order with its m-tiles adjacent, so a run of consecutive logical tiles shares a few
// weight and token slabs. Each XCD walks one contiguous stretch of the logical order.
//
// Workgroup tile: TM token rows x TN weight rows, waves in a WM x WN grid. Each K-step
// moves one 128-byte slab of every tile row (64 bf16 or 32 fp32 values) into LDS, at least
// double buffered. Weight rows feed the MFMA A operand and token rows the B operand, so every
// lane ends with 4 consecutive output columns of one token row (one 8- or 16-byte store).
//
// Three mainloops:
//   * gemm_pp_kernel (bf16 256x256 tiles, K a multiple of 128, 32x32x16 MFMA): persistent
//     (one workgroup per CU, each XCD's workgroups stepping through consecutive tiles
//     together); buffer loads write the slabs straight into LDS (no register staging; two
//     slots for token rows, three for weight rows);
//     8 waves in two groups of one wave per SIMD that alternate between a phase of
//     matrix-core work and a phase of memory work, so every SIMD always has a wave
//     issuing MFMAs; the last partial round of tiles is split along K (float32 partials,
//     summed in order by a second kernel);
//   * gemm_lds_kernel (bf16 128x128 tiles, same loads and split): 4 waves that each
//     interleave their own loads, fragment reads and MFMAs;
//   * gemm_kernel (any K that is a multiple of the 16-byte chunk, bf16 or fp32): loads
//     through registers, zero-filling chunks past K; one workgroup per tile, the
//     workgroup-to-tile map rotated over the XCDs.
//
// SwiGLU epilogue: the weight tile holds TN/2 gate rows followed by the matching TN/2 up
// rows; each wave owns equal gate and up slices, so silu(gate) * up is formed in registers.
// ReLU epilogue (hidden layer of a two-layer ReLU expert): the plain store with max(v, 0)
// applied to the float32 sums before rounding, in every store path including the split-K
// reduction.
#include "device_common.h"
#include "gemm.h"

#include <algorithm>
#include <string>
#include <type_traits>

namespace ec2moe {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

// buffer_load_dwordx4 ... lds: each lane's 16 bytes land at M0 + 16 * lane
__device__ void raw_buffer_load_lds(i32x4 rsrc, lds_void* lds, int size, int voffset, int soffset, int offset,
                                    int aux) __asm("llvm.amdgcn.raw.buffer.load.lds");

namespace {

constexpr int kXcds = 8;
constexpr int kMaxSplitChunks = 32;  // K chunks of a split tail tile

struct TileInfo {
    int group;
    int64_t row0;  // first row of the tile (position in the permuted order)
    int valid;     // rows of the tile inside the group
    int nt;        // n-tile index
};

__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// s_waitcnt immediate for vmcnt(n), lgkmcnt(0) and no expcnt wait: n <= 63 (vmcnt bits 3:0 and 15:14)
constexpr int vmcnt_imm(int n) { return 0x0070 | (n & 15) | ((n >> 4) << 14); }

// Number of real tiles (uniform): sum over groups of ceil(rows_e / TM) * ntn.
template <int TM>
__device__ __forceinline__ int count_tiles(const GemmArgs& a, int ntn) {
    if (a.seg == nullptr) return uniform(static_cast<int>((a.rows + TM - 1) / TM) * ntn);
    const int lane = threadIdx.x & 63;
    int t = 0;
    for (int e0 = 0; e0 < a.n_groups; e0 += 64) {
        const int e = e0 + lane;
        int cnt = 0;
        if (e < a.n_groups) cnt = ((a.seg[e + 1] - a.seg[e] + TM - 1) / TM) * ntn;
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) cnt += __shfl_xor(cnt, off);
        t += cnt;
    }
    return uniform(t);
}

// Position of tile `local` within one group of mtiles x ntn tiles: m-tiles go in
// ceil(mtiles / 8) bands of near-equal size (4 to 8 m-tiles when there are enough); a
// band's n-tiles run in order with the band's m-tiles adjacent. A run of 32 consecutive
// tiles (one XCD's workgroups) then covers b m-tiles x 32/b n-tiles, which share
// b + 32/b slabs (11 to 12 of 64) in that XCD's L2.
__device__ __forceinline__ void band_decode(int local, int mtiles, int ntn, int& mt, int& nt) {
    const int nbands = (mtiles + 7) / 8;
    const int bsz = (mtiles + nbands - 1) / nbands;
    const int band = local / (bsz * ntn);
    const int m0 = band * bsz;
    const int bm = std::min(bsz, mtiles - m0);  // m-tiles in this band
    const int r = local - band * bsz * ntn;
    nt = r / bm;
    mt = m0 + (r - nt * bm);
}

// Tile with logical index bid (groups in order; within a group, banded as above).
template <int TM>
__device__ __forceinline__ bool tile_of(const GemmArgs& a, int ntn, int bid, TileInfo& ti) {
    if (a.seg == nullptr) {
        const int mtiles = static_cast<int>((a.rows + TM - 1) / TM);
        int mt, nt;
        band_decode(bid, mtiles, ntn, mt, nt);
        ti.group = 0;
        ti.nt = nt;
        ti.row0 = static_cast<int64_t>(mt) * TM;
        ti.valid = static_cast<int>(std::min<int64_t>(TM, a.rows - ti.row0));
        return true;
    }
    const int lane = threadIdx.x & 63;
    int base = 0;
    for (int e0 = 0; e0 < a.n_groups; e0 += 64) {
        const int e = e0 + lane;
        int lo = 0, hi = 0, cnt = 0;
        if (e < a.n_groups) {
            lo = a.seg[e];
            hi = a.seg[e + 1];
            cnt = ((hi - lo + TM - 1) / TM) * ntn;
        }
        int inc = cnt;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int v = __shfl_up(inc, off);
            if (lane >= off) inc += v;
        }
        const bool hit = e < a.n_groups && cnt > 0 && bid >= base + inc - cnt && bid < base + inc;
        const uint64_t hits = __ballot(hit);
        if (hits) {
            const int src = __ffsll(static_cast<long long>(hits)) - 1;
            const int first = base + __shfl(inc - cnt, src);
            const int glo = uniform(__shfl(lo, src));
            const int ghi = uniform(__shfl(hi, src));
            const int mtiles = (ghi - glo + TM - 1) / TM;
            const int local = uniform(bid - first);
            ti.group = uniform(e0 + src);
            int mt, nt;
            band_decode(local, mtiles, ntn, mt, nt);
            ti.nt = nt;
            ti.row0 = glo + static_cast<int64_t>(mt) * TM;
            ti.valid = std::min(TM, ghi - static_cast<int>(ti.row0));
            return true;
        }
        base += __shfl(inc, 63);
    }
    return false;
}

// XCD-aware order: workgroup p of a launch of `units` whole tiles runs logical tile
// (p % 8) * ceil(units / 8) + p / 8; -1 if p has no tile.
__device__ __forceinline__ int xcd_remap(int p, int units) {
    const int per_xcd = (units + kXcds - 1) / kXcds;
    const int j = p / kXcds;
    const int bid = (p % kXcds) * per_xcd + j;
    return (j >= per_xcd || bid >= units) ? -1 : bid;
}

// Finds the tile of this workgroup (whole tiles only); false if it has none.
template <int TM>
__device__ __forceinline__ bool find_tile(const GemmArgs& a, int ntn, TileInfo& ti) {
    const int bid = xcd_remap(blockIdx.x, count_tiles<TM>(a, ntn));
    return bid >= 0 && tile_of<TM>(a, ntn, bid, ti);
}

// Split plan of a launch with `total` tiles and `slots` workgroups resident at once: the
// tiles that fill whole rounds run whole; the tail (fewer than one round) is split into
// S chunks along K so the last round is about as wide as the machine. Chunks hold an even
// number of 64-wide slabs.
struct SplitPlan {
    int full, tail, S, chunk_slabs;
};

__host__ __device__ __forceinline__ SplitPlan split_plan(int total, int slots, int max_split, int nk) {
    SplitPlan sp;
    sp.full = slots > 0 ? total / slots * slots : total;
    sp.tail = total - sp.full;
    int S = 1;
    if (sp.tail > 0 && max_split > 1)
        // at most one split workgroup per CU: more (two 128x128 tiles fit a CU) only adds
        // partial-sum traffic (the fine-grained encoder's X V: 18.0 against 21.7 us)
        S = std::max(1, std::min(std::min(std::min(max_split, kMaxSplitChunks), std::min(slots, 256) / sp.tail),
                                 nk / 2));
    sp.S = S;
    sp.chunk_slabs = ((nk + S - 1) / S + 1) / 2 * 2;
    return sp;
}

// silu(g) = g / (1 + e^-g) with the hardware 2^x and reciprocal (each within about 1 ulp),
// e^-g = 2^(-g log2 e); a very negative g gives e^-g = inf and a zero reciprocal.
__device__ __forceinline__ float silu(float g) {
    const float e = __builtin_amdgcn_exp2f(-g * 1.4426950408889634f);
    return g * __builtin_amdgcn_rcpf(1.0f + e);
}

// Plain-store epilogue: max(v, 0) when the GEMM carries the ReLU flag (the hidden layer of
// a two-layer ReLU expert), else v. The flag is uniform over the launch.
__device__ __forceinline__ float store_act(const GemmArgs& a, float v) { return a.relu ? fmaxf(v, 0.f) : v; }
__device__ __forceinline__ f32x4 store_act(const GemmArgs& a, f32x4 v) {
    if (a.relu) {
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = fmaxf(v[i], 0.f);
    }
    return v;
}

template <typename TO>
__device__ __forceinline__ void store4(TO* dst, f32x4 v);

template <>
__device__ __forceinline__ void store4<float>(float* dst, f32x4 v) {
    *reinterpret_cast<f32x4*>(dst) = v;
}

template <>
__device__ __forceinline__ void store4<bf16_t>(bf16_t* dst, f32x4 v) {
    uint2 o;
    o.x = static_cast<uint32_t>(f32_to_bf16(v[0])) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16);
    o.y = static_cast<uint32_t>(f32_to_bf16(v[2])) | (static_cast<uint32_t>(f32_to_bf16(v[3])) << 16);
    *reinterpret_cast<uint2*>(dst) = o;
}

// LDS row (within the weight part of the tile) of fragment block ni of wave column wn.
template <int TN, int WN, int NI, bool SWIGLU>
__device__ __forceinline__ int weight_frag_row(int wn, int ni, int l16) {
    if (SWIGLU) {
        constexpr int HALF = NI / 2;
        const int part = ni < HALF ? 0 : TN / 2;
        return part + wn * (TN / 2 / WN) + (ni % HALF) * 16 + l16;
    }
    return wn * (TN / WN) + ni * 16 + l16;
}

// Writes the wave's accumulators: lane holds token row wm*(TM/WM) + mi*16 + l16 and weight
// rows 4*lg .. 4*lg+3 of each 16x16 block.
template <typename TO, int TM, int TN, int WM, int WN, int MI, int NI, bool SWIGLU>
__device__ __forceinline__ void write_tile(const GemmArgs& a, const TileInfo& ti, int wm, int wn, int lane,
                                           const f32x4 (&acc)[NI][MI]) {
    const int l16 = lane & 15;
    const int lg = lane >> 4;
    TO* out = static_cast<TO*>(a.out);
#pragma unroll
    for (int mi = 0; mi < MI; ++mi) {
        const int trow = wm * (TM / WM) + mi * 16 + l16;
        if (trow >= ti.valid) continue;
        TO* orow = out + (ti.row0 + trow) * a.ldo;
        if (SWIGLU) {
            constexpr int HALF = NI / 2;
#pragma unroll
            for (int ni = 0; ni < HALF; ++ni) {
                const int col = ti.nt * (TN / 2) + wn * (TN / 2 / WN) + ni * 16 + 4 * lg;
                f32x4 v;
#pragma unroll
                for (int i = 0; i < 4; ++i) v[i] = silu(acc[ni][mi][i]) * acc[ni + HALF][mi][i];
                if (col < a.N) store4<TO>(orow + col, v);
            }
        } else {
#pragma unroll
            for (int ni = 0; ni < NI; ++ni) {
                const int col = ti.nt * TN + wn * (TN / WN) + ni * 16 + 4 * lg;
                if (col < a.N) store4<TO>(orow + col, store_act(a, acc[ni][mi]));
            }
        }
    }
}

// Weight row (within the group's weight matrix) of tile row n.
template <int TN, bool SWIGLU>
__device__ __forceinline__ int weight_row(const GemmArgs& a, int nt, int n) {
    if (SWIGLU) return n < TN / 2 ? nt * (TN / 2) + n : a.N + nt * (TN / 2) + (n - TN / 2);
    return std::min(nt * TN + n, a.N - 1);
}

// ------------------------------------------------------------------ register-staged mainloop

// CPR: 16-byte chunks of each tile row per slab (8: 128-byte rows; 16 and 32: 256- and
// 512-byte rows, a half and a quarter as many slabs, for long K)
template <typename T, typename TO, int TM, int TN, int WM, int WN, bool SWIGLU, int CPR>
__global__ __launch_bounds__(256, 1) void gemm_kernel(GemmArgs a) {
    static_assert(WM * WN == 4, "4 waves per workgroup");
    constexpr int RPP = 256 / CPR;        // rows per load pass
    static_assert(CPR == 8 || CPR == 16 || CPR == 32, "128-, 256- or 512-byte slab rows");
    static_assert(TM % RPP == 0 && TN % RPP == 0, "tiles load whole passes");
    constexpr int EPC = Elem<T>::kPerChunk;
    constexpr int BK = CPR * EPC;         // elements per slab row
    constexpr int MI = TM / WM / 16;      // token blocks per wave
    constexpr int NI = TN / WN / 16;      // weight blocks per wave
    constexpr int TOK_PASSES = TM / RPP;
    constexpr int W_PASSES = TN / RPP;
    constexpr int NOUT = SWIGLU ? TN / 2 : TN;
    constexpr int ROWS = TM + TN;
    static_assert(!SWIGLU || NI % 2 == 0, "SwiGLU waves hold matching gate/up blocks");

    __shared__ uint4 lds[2][ROWS * CPR];

    const int ntn = (a.N + NOUT - 1) / NOUT;
    TileInfo ti;
    if (!find_tile<TM>(a, ntn, ti)) return;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave % WM;
    const int wn = wave / WM;
    const int K = a.K;

    // ---- global load addressing: thread -> (chunk c, rows rr + RPP i)
    const int c = tid % CPR;
    const int rr = tid / CPR;
    const T* tok = static_cast<const T*>(a.tok);
    const T* wbase = static_cast<const T*>(a.w) + static_cast<int64_t>(ti.group) * a.w_group_stride;
    uint32_t tok_off[TOK_PASSES];
    uint32_t w_off[W_PASSES];
#pragma unroll
    for (int i = 0; i < TOK_PASSES; ++i) {
        const int r = std::min(rr + RPP * i, ti.valid - 1);
        const int64_t p = ti.row0 + r;
        const int64_t src = a.row_index ? a.row_index[p] : p;
        tok_off[i] = static_cast<uint32_t>(src * K + c * EPC);
    }
#pragma unroll
    for (int i = 0; i < W_PASSES; ++i) {
        const int wrow = weight_row<TN, SWIGLU>(a, ti.nt, rr + RPP * i);
        w_off[i] = static_cast<uint32_t>(static_cast<int64_t>(wrow) * K + c * EPC);
    }

    uint4 stage_t[TOK_PASSES];
    uint4 stage_w[W_PASSES];
    // chunks past K (a K that is not a whole number of slabs) load zeros on both sides
    auto load_global = [&](int ks) {
        const uint32_t k0 = static_cast<uint32_t>(ks) * BK;
        const bool in_k = static_cast<int>(k0) + c * EPC < K;
#pragma unroll
        for (int i = 0; i < TOK_PASSES; ++i) stage_t[i] = in_k ? ldg16(tok + tok_off[i] + k0) : make_uint4(0, 0, 0, 0);
#pragma unroll
        for (int i = 0; i < W_PASSES; ++i) stage_w[i] = in_k ? ldg16(wbase + w_off[i] + k0) : make_uint4(0, 0, 0, 0);
    };
    auto store_lds = [&](int buf) {
#pragma unroll
        for (int i = 0; i < TOK_PASSES; ++i) {
            const int row = rr + RPP * i;
            lds[buf][row * CPR + (c ^ (row & (CPR - 1)))] = stage_t[i];
        }
#pragma unroll
        for (int i = 0; i < W_PASSES; ++i) {
            const int row = TM + rr + RPP * i;
            lds[buf][row * CPR + (c ^ (row & (CPR - 1)))] = stage_w[i];
        }
    };

    const int l16 = lane & 15;
    const int lg = lane >> 4;
    int frag_t[MI];
    int frag_w[NI];
#pragma unroll
    for (int mi = 0; mi < MI; ++mi) frag_t[mi] = wm * (TM / WM) + mi * 16 + l16;
#pragma unroll
    for (int ni = 0; ni < NI; ++ni) frag_w[ni] = TM + weight_frag_row<TN, WN, NI, SWIGLU>(wn, ni, l16);

    f32x4 acc[NI][MI];
#pragma unroll
    for (int ni = 0; ni < NI; ++ni)
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) acc[ni][mi] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int nk = (K + BK - 1) / BK;
    load_global(0);
    store_lds(0);
    __syncthreads();
    for (int ks = 0; ks < nk; ++ks) {
        const int cur = ks & 1;
        if (ks + 1 < nk) load_global(ks + 1);
#pragma unroll
        for (int s = 0; s < CPR / 4; ++s) {
            const int ch = 4 * s + lg;
            uint4 bt[MI];
            uint4 aw[NI];
#pragma unroll
            for (int mi = 0; mi < MI; ++mi) {
                const int row = frag_t[mi];
                bt[mi] = lds[cur][row * CPR + (ch ^ (row & (CPR - 1)))];
            }
#pragma unroll
            for (int ni = 0; ni < NI; ++ni) {
                const int row = frag_w[ni];
                aw[ni] = lds[cur][row * CPR + (ch ^ (row & (CPR - 1)))];
            }
#pragma unroll
            for (int ni = 0; ni < NI; ++ni)
#pragma unroll
                for (int mi = 0; mi < MI; ++mi) acc[ni][mi] = Mfma<T>::step(aw[ni], bt[mi], acc[ni][mi]);
        }
        if (ks + 1 < nk) store_lds(cur ^ 1);
        __syncthreads();
    }

    write_tile<TO, TM, TN, WM, WN, MI, NI, SWIGLU>(a, ti, wm, wn, lane, acc);
}

// ------------------------------------------------------------------ direct-to-LDS mainloop

__device__ __forceinline__ i32x4 buffer_rsrc(const void* base, uint32_t bytes) {
    const uint64_t p = reinterpret_cast<uint64_t>(base);
    i32x4 r;
    r[0] = uniform(static_cast<int>(static_cast<uint32_t>(p)));
    r[1] = uniform(static_cast<int>(static_cast<uint32_t>(p >> 32)));
    r[2] = uniform(static_cast<int>(bytes));
    r[3] = 0x00020000;  // raw (untyped, unswizzled) buffer of the gfx9 family
    return r;
}

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

// Writes a wave's 32x32-block accumulators. After v_mfma_f32_32x32x16 with weight rows as A
// and token rows as B, lane l holds token row (l % 32) of the block and, in register r,
// weight row 8*(r/4) + 4*(l/32) + r%4: four runs of 4 consecutive output columns.
template <typename TO, int TM, int TN, int WM, int WN, int MI, int NI, bool SWIGLU>
__device__ __forceinline__ void write_tile32(const GemmArgs& a, const TileInfo& ti, int wm, int wn, int lane,
                                             const f32x16 (&acc)[NI][MI]) {
    const int l32 = lane & 31;
    const int lh = lane >> 5;
    TO* out = static_cast<TO*>(a.out);
#pragma unroll
    for (int mi = 0; mi < MI; ++mi) {
        const int trow = wm * (TM / WM) + mi * 32 + l32;
        if (trow >= ti.valid) continue;
        TO* orow = out + (ti.row0 + trow) * a.ldo;
        if (SWIGLU) {
            constexpr int HALF = NI / 2;
#pragma unroll
            for (int ni = 0; ni < HALF; ++ni) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int col = ti.nt * (TN / 2) + wn * (TN / 2 / WN) + ni * 32 + 8 * q + 4 * lh;
                    f32x4 v;
#pragma unroll
                    for (int i = 0; i < 4; ++i) v[i] = silu(acc[ni][mi][4 * q + i]) * acc[ni + HALF][mi][4 * q + i];
                    if (col < a.N) store4<TO>(orow + col, v);
                }
            }
        } else {
#pragma unroll
            for (int ni = 0; ni < NI; ++ni) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int col = ti.nt * TN + wn * (TN / WN) + ni * 32 + 8 * q + 4 * lh;
                    f32x4 v;
#pragma unroll
                    for (int i = 0; i < 4; ++i) v[i] = store_act(a, acc[ni][mi][4 * q + i]);
                    if (col < a.N) store4<TO>(orow + col, v);
                }
            }
        }
    }
}

// Writes a wave's 16x16-block accumulators. After v_mfma_f32_16x16x32 with weight rows as A
// and token rows as B, lane l holds token row (l % 16) of the block and, in register r,
// weight row 4*(l/16) + r: a run of 4 consecutive output columns.
template <typename TO, int TM, int TN, int WM, int WN, int MI, int NI, bool SWIGLU>
__device__ __forceinline__ void write_tile16(const GemmArgs& a, const TileInfo& ti, int wm, int wn, int lane,
                                             const f32x4 (&acc)[NI][MI]) {
    const int l16 = lane & 15;
    const int lg = lane >> 4;
    TO* out = static_cast<TO*>(a.out);
#pragma unroll
    for (int mi = 0; mi < MI; ++mi) {
        const int trow = wm * (TM / WM) + mi * 16 + l16;
        if (trow >= ti.valid) continue;
        TO* orow = out + (ti.row0 + trow) * a.ldo;
        if (SWIGLU) {
            constexpr int HALF = NI / 2;
#pragma unroll
            for (int ni = 0; ni < HALF; ++ni) {
                const int col = ti.nt * (TN / 2) + wn * (TN / 2 / WN) + ni * 16 + 4 * lg;
                f32x4 v;
#pragma unroll
                for (int i = 0; i < 4; ++i) v[i] = silu(acc[ni][mi][i]) * acc[ni + HALF][mi][i];
                if (col < a.N) store4<TO>(orow + col, v);
            }
        } else {
#pragma unroll
            for (int ni = 0; ni < NI; ++ni) {
                const int col = ti.nt * TN + wn * (TN / WN) + ni * 16 + 4 * lg;
                f32x4 v;
#pragma unroll
                for (int i = 0; i < 4; ++i) v[i] = store_act(a, acc[ni][mi][i]);
                if (col < a.N) store4<TO>(orow + col, v);
            }
        }
    }
}

// Workgroups of the large-tile kernel resident at once on the chip: 256 CUs, and as many
// workgroups per CU as its LDS stages allow (one 256x256 tile, two 128x128 tiles).
constexpr int kCUs = 256;
template <int TM, int TN>
__host__ __device__ constexpr int gemm_slots() {
    return kCUs * ((160 * 1024) / (2 * (TM + TN) * 128));
}

// bf16 mainloop on 32x32x16 matrix-core blocks (a full-rate bf16 MFMA shape on gfx950; the
// 256x256 ping-pong kernel below uses 16x16x32, which holds a higher clock under load).
//
// K advances in slabs of 64 (one 128-byte row per tile row) through two LDS stages; the
// buffer loads of slab ks + 1 fly while slab ks is consumed. Each stage is its own LDS
// object and the K loop is unrolled by two, so every access names its stage at compile
// time (fragment reads of one stage then need not wait for loads landing in the other).
// LDS rows are 8 chunks of 16 bytes, chunk c of row r stored at c ^ ((r >> 1) & 7): a
// 16-lane group of ds_read_b128 reading one chunk of 16 consecutive rows touches all 64
// banks once, and the buffer loads write 1 KB contiguous runs.
// Within a slab of 4 k-steps, fragment reads run one k-step ahead of the MFMAs; the
// MFMAs of a slab's last k-step are deferred past the next barrier, where they cover the
// latency of the next slab's first reads.
template <int TM, int TN, int WM, int WN, bool SWIGLU, typename TO>
__global__ __launch_bounds__(64 * WM * WN, 1) void gemm_lds_kernel(GemmArgs a) {
    constexpr int NW = WM * WN;                // waves per workgroup
    static_assert(NW == 4 || NW == 8, "4 or 8 waves per workgroup");
    constexpr int MI = TM / WM / 32;           // token blocks of 32 per wave
    constexpr int NI = TN / WN / 32;           // weight blocks of 32 per wave
    constexpr int NOUT = SWIGLU ? TN / 2 : TN;
    constexpr int ROWS = TM + TN;
    constexpr int RB = 128;                    // bytes per tile row per slab (64 bf16)
    constexpr int STAGE = ROWS * RB;
    constexpr int WROWS = ROWS / NW;           // tile rows loaded by each wave
    constexpr int LOADS = WROWS / 8;           // 8-row load instructions per wave per slab
    static_assert(MI >= 1 && NI >= 1, "wave tile of at least one 32x32 block");
    static_assert(WROWS % 8 == 0 && TM % WROWS == 0, "each wave loads only token or only weight rows");
    static_assert(!SWIGLU || NI % 2 == 0, "SwiGLU waves hold matching gate/up blocks");

    __shared__ __attribute__((aligned(1024))) char lds0[STAGE];
    __shared__ __attribute__((aligned(1024))) char lds1[STAGE];

    const int ntn = (a.N + NOUT - 1) / NOUT;
    const int K = a.K;
    const int nk_all = K / 64;  // even: K is a multiple of 128 on this path
    constexpr int P = gemm_slots<TM, TN>();  // workgroups of the launch, all resident at once
    constexpr int XW = P / kXcds;            // workgroups on each XCD
    const SplitPlan sp = split_plan(count_tiles<TM>(a, ntn), P, a.part ? a.max_split : 1, nk_all);
    const int rounds = sp.full / P;
    const int p = blockIdx.x;

    // Persistent loop. Whole rounds first: workgroup p runs on XCD p % 8, and in round r
    // takes logical tile (p % 8) * (rounds * XW) + r * XW + p / 8, so the XW workgroups of
    // one XCD step together through consecutive tiles (m-tiles of one weight slab adjacent)
    // and share their slabs in that XCD's L2 while they are at the same K. Then at most one
    // unit of the tail (a whole tile, or one K chunk of a split tile).
    for (int it = 0; it <= rounds; ++it) {
    int bid, chunk = 0;
    bool split = false;
    if (it < rounds) {
        bid = (p % kXcds) * (rounds * XW) + it * XW + p / kXcds;
    } else {
        if (p >= sp.tail * sp.S) break;
        bid = sp.full + p / sp.S;
        chunk = p % sp.S;
        split = sp.S > 1;
    }
    TileInfo ti;
    if (!tile_of<TM>(a, ntn, bid, ti)) break;
    const int kb = split ? chunk * sp.chunk_slabs : 0;                  // first slab of this unit
    const int nk = split ? std::min(nk_all, kb + sp.chunk_slabs) - kb : nk_all;

    // Lane-derived addresses are rebuilt every tile from an opaque copy of the thread id:
    // hoisted out of the tile loop they would stay live through the mainloop and spill.
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int lane = tid & 63;
    const int wave = uniform(tid >> 6);
    const int wm = wave % WM;
    const int wn = wave / WM;
    const uint32_t row_bytes = static_cast<uint32_t>(K) * 2u;
    // this wave's rows [wave * WROWS, (wave + 1) * WROWS) are all token rows or all weight rows
    const bool tok_wave = wave * WROWS < TM;
    const bf16_t* wgrp = static_cast<const bf16_t*>(a.w) + static_cast<int64_t>(ti.group) * a.w_group_stride;
    const i32x4 rs = tok_wave ? buffer_rsrc(a.tok, static_cast<uint32_t>(a.src_rows) * row_bytes)
                              : buffer_rsrc(wgrp, static_cast<uint32_t>(a.w_rows) * row_bytes);

    // one load instruction fills 8 rows: lane -> (row lane / 8, LDS chunk lane % 8), which
    // holds logical chunk (lane % 8) ^ ((row >> 1) & 7); the swizzle is applied on the
    // global side
    uint32_t voff[LOADS];
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
        const int row = wave * WROWS + i * 8 + (lane >> 3);
        const uint32_t chunk_off = static_cast<uint32_t>(((lane & 7) ^ ((row >> 1) & 7)) * 16);
        if (tok_wave) {
            const int r = std::min(row, ti.valid - 1);
            const int64_t p = ti.row0 + r;
            const int64_t src = a.row_index ? a.row_index[p] : p;
            voff[i] = static_cast<uint32_t>(src) * row_bytes + chunk_off;
        } else {
            voff[i] = static_cast<uint32_t>(weight_row<TN, SWIGLU>(a, ti.nt, row - TM)) * row_bytes + chunk_off;
        }
    }
    auto issue_slab = [&](int ks, char* stage) {
        const int soff = (kb + ks) * RB;
#pragma unroll
        for (int i = 0; i < LOADS; ++i) {
            lds_void* dst = reinterpret_cast<lds_void*>(
                reinterpret_cast<uintptr_t>(stage + (wave * WROWS + i * 8) * RB));
            raw_buffer_load_lds(rs, dst, 16, static_cast<int>(voff[i]), soff, 0, 0);
        }
    };

    // fragment rows: lane l feeds row (l % 32) of each 32-row block with logical chunk
    // (2 s + l / 32) of k-step s; blocks start at multiples of 32, so the swizzle depends on
    // the lane only. Block offsets are compile-time and fold into the read's immediate.
    const int l32 = lane & 31;
    const int lh = lane >> 5;
    const int sw = (l32 >> 1) & 7;
    constexpr int WTOK = TM / WM;                       // token rows per wave
    constexpr int WW = SWIGLU ? TN / 2 / WN : TN / WN;  // weight rows per wave (per half)
    int off_t[4], off_w[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        const int ch = ((2 * s + lh) ^ sw) * 16;
        off_t[s] = (wm * WTOK + l32) * RB + ch;
        off_w[s] = (TM + wn * WW + l32) * RB + ch;
    }
    auto wblk = [](int ni) constexpr {
        if (SWIGLU) {
            constexpr int HALF = NI / 2;
            return (ni < HALF ? 0 : TN / 2) + (ni % HALF) * 32;
        }
        return ni * 32;
    };

    f32x16 acc[NI][MI];
#pragma unroll
    for (int ni = 0; ni < NI; ++ni)
#pragma unroll
        for (int mi = 0; mi < MI; ++mi)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[ni][mi][r] = 0.f;

    auto mma = [&](const uint4 (&fa)[NI], const uint4 (&fb)[MI]) {
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
#pragma unroll
            for (int mi = 0; mi < MI; ++mi)
                acc[ni][mi] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, fa[ni]),
                                                                     __builtin_bit_cast(bf16x8, fb[mi]),
                                                                     acc[ni][mi], 0, 0, 0);
    };
    uint4 pa[NI], pb[MI];  // k-step 3 fragments of the previous slab, consumed after the barrier

    // Program order of a slab: k-step 0 reads, the next slab's buffer loads (other stage),
    // then [previous slab's k-step 3 | k-step 0 | 1 | 2] MFMAs with reads of k-steps 1, 2, 3
    // placed one group ahead; k-step 3's MFMAs wait for the next slab.
    auto slab = [&](const char* base, char* refill, bool prefetch, int ks_next, bool pending) {
        uint4 fa[3][NI], fb[3][MI];
        auto read_step = [&](int s, uint4 (&ra)[NI], uint4 (&rb)[MI]) {
#pragma unroll
            for (int ni = 0; ni < NI; ++ni) ra[ni] = *reinterpret_cast<const uint4*>(base + off_w[s] + wblk(ni) * RB);
#pragma unroll
            for (int mi = 0; mi < MI; ++mi) rb[mi] = *reinterpret_cast<const uint4*>(base + off_t[s] + mi * 32 * RB);
        };
        read_step(0, fa[0], fb[0]);
        if (prefetch) issue_slab(ks_next, refill);
        read_step(1, fa[1], fb[1]);
        if (pending) mma(pa, pb);
        read_step(2, fa[2], fb[2]);
        mma(fa[0], fb[0]);
        read_step(3, pa, pb);
        mma(fa[1], fb[1]);
        mma(fa[2], fb[2]);

        constexpr int RD = NI + MI;                 // fragment reads per k-step
        constexpr int MF = NI * MI / RD;            // MFMAs before each read
        constexpr int REST = NI * MI - MF * RD;
        static_assert(MF >= 1, "an MFMA for every read of the next k-step");
        __builtin_amdgcn_sched_group_barrier(0x100, RD, 0);
        if (prefetch) __builtin_amdgcn_sched_group_barrier(0x020, LOADS, 0);
        if (pending) {
#pragma unroll
            for (int i = 0; i < RD; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x008, MF, 0);
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            }
            if (REST) __builtin_amdgcn_sched_group_barrier(0x008, REST, 0);
        } else {
            __builtin_amdgcn_sched_group_barrier(0x100, RD, 0);
        }
#pragma unroll
        for (int g = 0; g < 2; ++g) {
#pragma unroll
            for (int i = 0; i < RD; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x008, MF, 0);
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            }
            if (REST) __builtin_amdgcn_sched_group_barrier(0x008, REST, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, NI * MI, 0);
    };

    // Before consuming a slab: its loads have landed (vmcnt(0): they are the only ones
    // outstanding) and this wave's LDS reads have all returned; the barrier then makes every
    // wave's loads visible and guarantees that no wave still reads the stage about to be
    // refilled. A bare s_barrier: __syncthreads() would add a fence with the same waits.
    auto sync = [&]() {
        __builtin_amdgcn_s_waitcnt(0x0070);  // vmcnt(0) expcnt(7) lgkmcnt(0)
        asm volatile("s_barrier" ::: "memory");
    };

    if (nk > 0) {  // nk is even (whole chunks of an even number of slabs)
        issue_slab(0, lds0);
        sync();
        slab(lds0, lds1, true, 1, false);
        for (int ks = 1; ks + 1 < nk; ks += 2) {
            sync();
            slab(lds1, lds0, true, ks + 1, true);
            sync();
            slab(lds0, lds1, true, ks + 2, true);
        }
        sync();
        slab(lds1, lds0, false, 0, true);
        mma(pa, pb);
    }

    if (split) {
        // raw float32 partial tile [TM][TN] (weight rows in tile order) of this K chunk
        float* part = a.part + static_cast<int64_t>(p) * TM * TN;
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) {
            const int trow = wm * WTOK + mi * 32 + l32;
#pragma unroll
            for (int ni = 0; ni < NI; ++ni) {
                const int wrow = wn * WW + wblk(ni);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    f32x4 v;
#pragma unroll
                    for (int i = 0; i < 4; ++i) v[i] = acc[ni][mi][4 * q + i];
                    *reinterpret_cast<f32x4*>(part + trow * TN + wrow + 8 * q + 4 * lh) = v;
                }
            }
        }
        continue;
    }
    write_tile32<TO, TM, TN, WM, WN, MI, NI, SWIGLU>(a, ti, wm, wn, lane, acc);
    }
}

// 8-wave ping-pong mainloop for the 256x256 tile. Waves 0-3 (group 0, token loaders) and
// waves 4-7 (group 1, weight loaders) sit one per SIMD each; the groups alternate between a
// compute phase (the 64 products of one slab, at raised priority) and a memory phase
// (fragment reads of the next slab, buffer loads), with a workgroup barrier between phases,
// so on every SIMD one wave issues MFMAs while the other waits on memory.
//   group 0, slab s: issue token rows of slab s+1 | read slab s | barrier | MFMA slab s |
//                    wait own loads | barrier
//   group 1, slab s: MFMA slab s-1 | barrier | issue weight rows of slab s+2 into the slot of
//                    slab s-1, read slab s | wait loads of slab s+1 | barrier
// Token rows sit in two 32 KB slots and weight rows in three, so that every slot is refilled
// only after a barrier that follows the last read of it by any wave (with two combined
// stages the weight rows of slab s+2 had to go into the stage of slab s, which the other
// group could still be reading).
// The products are v_mfma_f32_16x16x32_bf16: on random bf16 operands the chip sustains
// 1.92 PFLOP/s with them against 1.72 with 32x32x16 (the same flops through a quarter of
// the accumulator traffic per instruction), so the power-bound clock stays higher. A wave
// holds 4 x 8 blocks of 16 x 16 (128 accumulators); the memory phase reads both k-steps'
// token fragments and k-step 0's weight fragments, and k-step 1's weight fragments are read
// during the products of k-step 0 (into the registers of the block just consumed). Those
// late reads stay behind the same barriers: a group's products of slab s read the weight
// slot of slab s before the barrier after which slab s+3 refills it, and after the last
// slab every path waits at a barrier before any slot is written again.
template <bool SWIGLU, typename TO>
__global__ __launch_bounds__(512, 1) void gemm_pp_kernel(GemmArgs a) {
    constexpr int TM = 256, TN = 256, WM = 4, WN = 2, NW = 8;
    constexpr int MI = TM / WM / 16;           // 4 token blocks of 16 per wave
    constexpr int NI = TN / WN / 16;           // 8 weight blocks of 16 per wave
    constexpr int NOUT = SWIGLU ? TN / 2 : TN;
    constexpr int ROWS = TM + TN;
    constexpr int RB = 128;
    constexpr int SLOT = TM * RB;              // 32 KB: the token rows, or the weight rows, of one slab
    static_assert(TM == TN, "token and weight slots of one size");
    constexpr int WROWS = ROWS / NW;           // 64
    constexpr int LOADS = WROWS / 8;           // 8
    static_assert(2 * LOADS < 64, "vmcnt immediate");

    // one LDS object per slot (each named at compile time where it is read, so a wait before
    // a fragment read covers only the loads into that slot): 160 KB in all
    __shared__ __attribute__((aligned(1024))) char t0[SLOT];
    __shared__ __attribute__((aligned(1024))) char t1[SLOT];
    __shared__ __attribute__((aligned(1024))) char w0[SLOT];
    __shared__ __attribute__((aligned(1024))) char w1[SLOT];
    __shared__ __attribute__((aligned(1024))) char w2[SLOT];

    const int ntn = (a.N + NOUT - 1) / NOUT;
    const int K = a.K;
    const int nk_all = K / 64;
    constexpr int P = gemm_slots<TM, TN>();
    constexpr int XW = P / kXcds;
    const SplitPlan sp = split_plan(count_tiles<TM>(a, ntn), P, a.part ? a.max_split : 1, nk_all);
    const int rounds = sp.full / P;
    const int p = blockIdx.x;

    for (int it = 0; it <= rounds; ++it) {
    int bid, chunk = 0;
    bool split = false;
    if (it < rounds) {
        bid = (p % kXcds) * (rounds * XW) + it * XW + p / kXcds;
    } else {
        if (p >= sp.tail * sp.S) break;
        bid = sp.full + p / sp.S;
        chunk = p % sp.S;
        split = sp.S > 1;
    }
    TileInfo ti;
    if (!tile_of<TM>(a, ntn, bid, ti)) break;
    const int kb = split ? chunk * sp.chunk_slabs : 0;
    const int nk = split ? std::min(nk_all, kb + sp.chunk_slabs) - kb : nk_all;

    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int lane = tid & 63;
    const int wave = uniform(tid >> 6);
    const int wm = wave % WM;
    const int wn = wave / WM;                 // also the group
    const uint32_t row_bytes = static_cast<uint32_t>(K) * 2u;
    const bool tok_wave = wave * WROWS < TM;  // group 0
    const bf16_t* wgrp = static_cast<const bf16_t*>(a.w) + static_cast<int64_t>(ti.group) * a.w_group_stride;
    const i32x4 rs = tok_wave ? buffer_rsrc(a.tok, static_cast<uint32_t>(a.src_rows) * row_bytes)
                              : buffer_rsrc(wgrp, static_cast<uint32_t>(a.w_rows) * row_bytes);
    uint32_t voff[LOADS];
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
        const int row = wave * WROWS + i * 8 + (lane >> 3);
        const uint32_t chunk_off = static_cast<uint32_t>(((lane & 7) ^ ((row >> 1) & 7)) * 16);
        if (tok_wave) {
            const int r = std::min(row, ti.valid - 1);
            const int64_t pr = ti.row0 + r;
            const int64_t src = a.row_index ? a.row_index[pr] : pr;
            voff[i] = static_cast<uint32_t>(src) * row_bytes + chunk_off;
        } else {
            voff[i] = static_cast<uint32_t>(weight_row<TN, SWIGLU>(a, ti.nt, row - TM)) * row_bytes + chunk_off;
        }
    }
    // this wave's rows of a slab into a token or weight slot (rows 64 (wave & 3) .. + 63 of it)
    auto issue_slab = [&](int ks, char* slot) {
        const int soff = (kb + ks) * RB;
#pragma unroll
        for (int i = 0; i < LOADS; ++i) {
            lds_void* dst = reinterpret_cast<lds_void*>(
                reinterpret_cast<uintptr_t>(slot + ((wave & 3) * WROWS + i * 8) * RB));
            raw_buffer_load_lds(rs, dst, 16, static_cast<int>(voff[i]), soff, 0, 0);
        }
    };

    // 16x16x32 blocks: lane l feeds row l % 16 of a block with the 8 k of logical chunk
    // 4 s + l / 16 of k-step s (two k-steps of 32 per slab); blocks start at multiples of 16
    // rows, so the swizzle depends on the lane only
    const int l16 = lane & 15;
    const int lg = lane >> 4;
    const int sw = (l16 >> 1) & 7;
    constexpr int WTOK = TM / WM;
    constexpr int WW = SWIGLU ? TN / 2 / WN : TN / WN;
    int off_t[2], off_w[2];
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        const int ch = ((4 * s + lg) ^ sw) * 16;
        off_t[s] = (wm * WTOK + l16) * RB + ch;  // in a token slot
        off_w[s] = (wn * WW + l16) * RB + ch;    // in a weight slot
    }
    auto wblk = [](int ni) constexpr {
        if (SWIGLU) {
            constexpr int HALF = NI / 2;
            return (ni < HALF ? 0 : TN / 2) + (ni % HALF) * 16;
        }
        return ni * 16;
    };

    f32x4 acc[NI][MI];
#pragma unroll
    for (int ni = 0; ni < NI; ++ni)
#pragma unroll
        for (int mi = 0; mi < MI; ++mi)
#pragma unroll
            for (int r = 0; r < 4; ++r) acc[ni][mi][r] = 0.f;

    // one slab of fragments: both k-steps of the token rows, one k-step of the weight rows
    // at a time (k-step 1's are read by mma_slab_w)
    uint4 fa[NI], fb[2][MI];
    auto read_slab = [&](const char* tslot, const char* wslot) {
#pragma unroll
        for (int ni = 0; ni < NI; ++ni) fa[ni] = *reinterpret_cast<const uint4*>(wslot + off_w[0] + wblk(ni) * RB);
#pragma unroll
        for (int s = 0; s < 2; ++s)
#pragma unroll
            for (int mi = 0; mi < MI; ++mi) fb[s][mi] = *reinterpret_cast<const uint4*>(tslot + off_t[s] + mi * 16 * RB);
    };
    auto mma_slab_w = [&](const char* wslot) {
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int ni = 0; ni < NI; ++ni) {
#pragma unroll
            for (int mi = 0; mi < MI; ++mi)
                acc[ni][mi] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, fa[ni]),
                                                                     __builtin_bit_cast(bf16x8, fb[0][mi]),
                                                                     acc[ni][mi], 0, 0, 0);
            fa[ni] = *reinterpret_cast<const uint4*>(wslot + off_w[1] + wblk(ni) * RB);
        }
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
#pragma unroll
            for (int mi = 0; mi < MI; ++mi)
                acc[ni][mi] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, fa[ni]),
                                                                     __builtin_bit_cast(bf16x8, fb[1][mi]),
                                                                     acc[ni][mi], 0, 0, 0);
        // k-step 0 with a read after every block's products, then k-step 1: each read has the
        // rest of k-step 0 (28 products or more) to land
#pragma unroll
        for (int ni = 0; ni < NI; ++ni) {
            __builtin_amdgcn_sched_group_barrier(0x008, MI, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, NI * MI, 0);
        __builtin_amdgcn_s_setprio(0);
    };
    auto barrier = [&]() {
        __builtin_amdgcn_sched_barrier(0);
        asm volatile("s_barrier" ::: "memory");
        __builtin_amdgcn_sched_barrier(0);
    };

    if (nk > 0) {  // nk is even and the same for every wave
        if (tok_wave) {
            issue_slab(0, t0);
            issue_slab(1, t1);
            __builtin_amdgcn_s_waitcnt(0x0070 | LOADS);  // own rows of slab 0 landed
        } else {
            issue_slab(0, w0);
            issue_slab(1, w1);
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(LOADS));  // own rows of slab 0 landed
        }
        barrier();
        // slab s: tokens in slot s % 2, weights in slot s % 3 (the loops run six slabs a turn)
        if (tok_wave) {
            auto slab0 = [&](const char* tcur, char* tnxt, const char* wcur, int s) {
                if (s >= nk) return;
                if (s >= 1 && s + 1 < nk) issue_slab(s + 1, tnxt);
                read_slab(tcur, wcur);
                __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
                barrier();
                mma_slab_w(wcur);
                __builtin_amdgcn_sched_barrier(0);
                __builtin_amdgcn_s_waitcnt(0x0070);  // token rows of slab s+1 landed
                barrier();
            };
            for (int s = 0; s < nk; s += 6) {
                slab0(t0, t1, w0, s);
                slab0(t1, t0, w1, s + 1);
                slab0(t0, t1, w2, s + 2);
                slab0(t1, t0, w0, s + 3);
                slab0(t0, t1, w1, s + 4);
                slab0(t1, t0, w2, s + 5);
            }
        } else {
            // The slot refilled in step s holds slab s - 1, whose last reads (this group's) were
            // done before the previous barrier: no wave can still be reading it.
            auto slab1 = [&](const char* tcur, const char* wcur, char* wfree, int s) {
                if (s >= nk) return;
                if (s > 0) mma_slab_w(wfree);  // slab s - 1, whose weights sit in the slot refilled next
                barrier();
                // the refill goes out before this group's fragment reads: a longer lead for the
                // weight rows, which come from HBM (gate-up 1589 -> 1567 us, down 773 -> 760 us
                // on the Mixtral-shaped layer; issuing it before the barrier instead, at the end of
                // the products, delays the barrier: 1658 and 822 us)
                if (s + 2 < nk) issue_slab(s + 2, wfree);
                read_slab(tcur, wcur);
                __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
                if (s + 2 < nk) __builtin_amdgcn_s_waitcnt(vmcnt_imm(LOADS));  // weight rows of slab s+1 landed
                else __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
                barrier();
            };
            for (int s = 0; s < nk; s += 6) {
                slab1(t0, w0, w2, s);
                slab1(t1, w1, w0, s + 1);
                slab1(t0, w2, w1, s + 2);
                slab1(t1, w0, w2, s + 3);
                slab1(t0, w1, w0, s + 4);
                slab1(t1, w2, w1, s + 5);
            }
            const int last = (nk - 1) % 3;
            mma_slab_w(last == 0 ? w0 : last == 1 ? w1 : w2);
        }
    }

    if (split) {
        // raw float32 partial tile [TM][TN] (weight rows in tile order) of this K chunk; lane l
        // holds, per block, weight rows 4 (l / 16) .. + 3 of token row l % 16
        float* part = a.part + static_cast<int64_t>(p) * TM * TN;
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) {
            const int trow = wm * WTOK + mi * 16 + l16;
#pragma unroll
            for (int ni = 0; ni < NI; ++ni) {
                const int wrow = wn * WW + wblk(ni) + 4 * lg;
                *reinterpret_cast<f32x4*>(part + trow * TN + wrow) = acc[ni][mi];
            }
        }
        barrier();  // the weight loaders' last products read their slot: no refill before this
        continue;
    }
    if constexpr (sizeof(TO) == 4) {
        write_tile16<TO, TM, TN, WM, WN, MI, NI, SWIGLU>(a, ti, wm, wn, lane, acc);
        barrier();  // the weight loaders' last products read their slot: no refill before this
    } else {
        // The finished tile is staged in LDS as bf16 rows (every slot is free after the last
        // slab) so that the global stores are whole rows: 16 bytes per lane, 128-byte lines.
        // Staged row r holds its 16-byte chunk c at c ^ (r % OCH).
        constexpr int OROW = NOUT * 2;   // bytes per staged row
        constexpr int OCH = OROW / 16;   // 16-byte chunks per row
        constexpr int RPS = SLOT / OROW;  // rows per 32 KB slot (128 for SwiGLU, 64 otherwise)
        static_assert(TM <= 4 * RPS && WTOK <= RPS && RPS % WTOK == 0, "staged tile fits four slots");
        auto ost = [&](int i) -> char* { return i == 0 ? t0 : i == 1 ? t1 : i == 2 ? w0 : w1; };
        // this wave's rows wm * 64 .. wm * 64 + 63 lie in one slot
        char* wst = ost(wm * WTOK / RPS) + (wm * WTOK % RPS) * OROW;
        // without SwiGLU the staged rows also fill two weight slots, one of which the weight
        // loaders' last products may still be reading
        if constexpr (!SWIGLU) barrier();
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) {
            const int r = mi * 16 + l16;  // row within this wave's 64
            const int sr = wm * WTOK + r;  // row within the tile (swizzle key)
            constexpr int NB = SWIGLU ? NI / 2 : NI;
#pragma unroll
            for (int ni = 0; ni < NB; ++ni) {
                float v[4];
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    v[e] = SWIGLU ? silu(acc[ni][mi][e]) * acc[ni + NB][mi][e] : store_act(a, acc[ni][mi][e]);
                bf16x4 o;
#pragma unroll
                for (int e = 0; e < 4; ++e) o[e] = static_cast<__bf16>(v[e]);
                // columns 4 lg .. + 3 of the block: half lg % 2 of 8-column chunk lg / 2
                const int col = wn * (NOUT / WN) + ni * 16 + 8 * (lg >> 1);
                const int ch = (col / 8) ^ (sr % OCH);
                *reinterpret_cast<bf16x4*>(wst + r * OROW + ch * 16 + (lg & 1) * 8) = o;
            }
        }
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
        barrier();
        // whole rows back out: ROWS_PER_INSTR rows of OCH lanes per instruction
        constexpr int RPI = 64 / OCH;
        constexpr int NINSTR = TM / NW / RPI;
        TO* out = static_cast<TO*>(a.out);
#pragma unroll
        for (int j = 0; j < NINSTR; ++j) {
            const int r = wave * (TM / NW) + j * RPI + lane / OCH;  // tile row
            const int c = lane % OCH;
            const char* src = ost(r / RPS) + (r % RPS) * OROW + ((c ^ (r % OCH)) * 16);
            const uint4 v = *reinterpret_cast<const uint4*>(src);
            const int col = ti.nt * NOUT + c * 8;
            if (r < ti.valid && col < a.N) *reinterpret_cast<uint4*>(out + (ti.row0 + r) * a.ldo + col) = v;
        }
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): staged rows read before the slots refill
        barrier();
    }
    }
}

// Sums the float32 partial tiles of the split tail in chunk order and applies the
// epilogue (store, ReLU store, or silu(gate) * up) of the large-tile kernel. One workgroup per
// (tail tile, 16 rows); every thread owns a run of 4 output columns per pass and issues
// the loads of up to 16 chunks (8 of each half with SwiGLU) before adding them in order.
template <int TM, int TN, bool SWIGLU, typename TO>
__global__ __launch_bounds__(256) void gemm_split_reduce_kernel(GemmArgs a) {
    constexpr int NOUT = SWIGLU ? TN / 2 : TN;
    const int ntn = (a.N + NOUT - 1) / NOUT;
    const SplitPlan sp = split_plan(count_tiles<TM>(a, ntn), gemm_slots<TM, TN>(), a.max_split, a.K / 64);
    if (sp.S <= 1) return;
    constexpr int ROWS = 16;
    constexpr int QUADS = NOUT / 4;                  // float4 column runs per row
    constexpr int KB = SWIGLU ? 8 : 16;              // chunks loaded together
    const int t = blockIdx.x / (TM / ROWS);
    if (t >= sp.tail) return;
    TileInfo ti;
    if (!tile_of<TM>(a, ntn, sp.full + t, ti)) return;
    const float* tile_part = a.part + static_cast<int64_t>(t) * sp.S * TM * TN;
    const int r0 = (blockIdx.x % (TM / ROWS)) * ROWS;
    for (int i = threadIdx.x; i < ROWS * QUADS; i += 256) {
        const int r = r0 + i / QUADS;
        const int c = (i % QUADS) * 4;
        if (r >= ti.valid) continue;
        // chunks in order, KB (SwiGLU: twice KB / 2) loads in flight at a time
        f32x4 sg = f32x4{0.f, 0.f, 0.f, 0.f}, su = sg;
        for (int k0 = 0; k0 < sp.S; k0 += KB) {
            f32x4 g[KB], u[KB];
#pragma unroll
            for (int k = 0; k < KB; ++k) {
                if (k0 + k < sp.S) {
                    const float* src = tile_part + static_cast<int64_t>(k0 + k) * TM * TN + r * TN + c;
                    g[k] = *reinterpret_cast<const f32x4*>(src);
                    if (SWIGLU) u[k] = *reinterpret_cast<const f32x4*>(src + TN / 2);
                }
            }
#pragma unroll
            for (int k = 0; k < KB; ++k) {
                if (k0 + k < sp.S) {
                    sg = k0 + k == 0 ? g[k] : sg + g[k];
                    if (SWIGLU) su = k0 + k == 0 ? u[k] : su + u[k];
                }
            }
        }
        TO* orow = static_cast<TO*>(a.out) + (ti.row0 + r) * a.ldo;
        if (SWIGLU) {
            f32x4 v;
#pragma unroll
            for (int q = 0; q < 4; ++q) v[q] = silu(sg[q]) * su[q];
            if (ti.nt * NOUT + c < a.N) store4<TO>(orow + ti.nt * NOUT + c, v);
        } else {
            const int col = ti.nt * TN + c;
            if (col < a.N) store4<TO>(orow + col, store_act(a, sg));
        }
    }
}

// ------------------------------------------------------------------ dispatch

template <int TM, int TN, bool SWIGLU>
int64_t grid_size(const GemmArgs& a) {
    constexpr int NOUT = SWIGLU ? TN / 2 : TN;
    const int64_t ntn = (a.N + NOUT - 1) / NOUT;
    const int64_t mtiles = a.seg ? (a.rows + TM - 1) / TM + a.n_groups : (a.rows + TM - 1) / TM;
    return (mtiles * ntn + kXcds - 1) / kXcds * kXcds;
}

template <typename T, typename TO, int TM, int TN, int WM, int WN, bool SWIGLU, int CPR = 8>
hipError_t run(const GemmArgs& a, hipStream_t s) {
    const int64_t grid = grid_size<TM, TN, SWIGLU>(a);
    if (grid == 0) return hipSuccess;
    ProfileScope prof(a.name ? a.name : "gemm", s);
    hipLaunchKernelGGL((gemm_kernel<T, TO, TM, TN, WM, WN, SWIGLU, CPR>), dim3(static_cast<unsigned>(grid)),
                       dim3(256), 0, s, a);
    return hipGetLastError();
}

template <int TM, int TN, int WM, int WN, bool SWIGLU, typename TO>
hipError_t run_lds(const GemmArgs& a, hipStream_t s) {
    if (grid_size<TM, TN, SWIGLU>(a) == 0) return hipSuccess;
    const bool can_split = a.part != nullptr && a.max_split > 1;
    // persistent: one workgroup per resident slot, each looping over its tiles
    const int64_t grid = gemm_slots<TM, TN>();
    {
        ProfileScope prof(a.name ? a.name : "gemm", s);
        if constexpr (TM == 256 && TN == 256 && WM * WN == 8)
            hipLaunchKernelGGL((gemm_pp_kernel<SWIGLU, TO>), dim3(static_cast<unsigned>(grid)), dim3(512), 0, s, a);
        else
            hipLaunchKernelGGL((gemm_lds_kernel<TM, TN, WM, WN, SWIGLU, TO>), dim3(static_cast<unsigned>(grid)),
                               dim3(64 * WM * WN), 0, s, a);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !can_split) return e;
    // The tile count of a dense launch is known here: the reduction gets one workgroup per
    // (tail tile, 16 rows), or no launch without a split tail. Grouped launches count their
    // tiles on the device: a workgroup for every tail tile that can be split (a split needs
    // two chunks per tail tile within 256 workgroups: at most 128 tail tiles), the surplus
    // leaving at once.
    int64_t rgrid = static_cast<int64_t>(std::min(gemm_slots<TM, TN>(), 128)) * (TM / 16);
    if (a.seg == nullptr) {
        constexpr int NOUT = SWIGLU ? TN / 2 : TN;
        const int64_t tiles = (a.rows + TM - 1) / TM * ((a.N + NOUT - 1) / NOUT);
        const SplitPlan sp = split_plan(static_cast<int>(tiles), gemm_slots<TM, TN>(), a.max_split, a.K / 64);
        if (sp.S <= 1) return hipSuccess;
        rgrid = static_cast<int64_t>(sp.tail) * (TM / 16);
    }
    std::string rname = std::string(a.name ? a.name : "gemm") + "_tail";
    ProfileScope prof(rname.c_str(), s);
    hipLaunchKernelGGL((gemm_split_reduce_kernel<TM, TN, SWIGLU, TO>), dim3(static_cast<unsigned>(rgrid)), dim3(256),
                       0, s, a);
    return hipGetLastError();
}

// Tile choice. The bf16 direct-to-LDS path (K a multiple of 128) takes the largest tile
// whose rows are mostly occupied; its split-K tail supplies parallelism for few tiles.
// Otherwise the register-staged kernel, with the largest tile that still gives two
// workgroups per CU.
enum class Tile { Big, Mid, Small };

Tile choose_tile(const GemmArgs& a, bool swiglu, bool lds) {
    auto tiles = [&](int tm, int tn) {
        const int nout = swiglu ? tn / 2 : tn;
        const int64_t mt = (a.rows + tm - 1) / tm + (a.seg ? a.n_groups : 0);
        return mt * ((a.N + nout - 1) / nout);
    };
    const int64_t avg_rows = a.seg ? a.rows / std::max(1, a.n_groups) : a.rows;
    if (lds) {
        // the 256x256 tile whenever it fills at least one round of the machine (short K
        // included: the codec's rank-r products run 1.6x faster on it than on 128x128 tiles)
        if (avg_rows >= 256 && tiles(256, 256) >= gemm_slots<256, 256>()) return Tile::Big;
        // long K and only a few 128x128 tiles (the encoder's X V for a handful of tokens): the
        // split-K tail of the 128x128 kernel spreads K over up to 32 workgroups per tile
        if (tiles(128, 128) * 4 <= gemm_slots<128, 128>() && a.K >= 2048) return Tile::Mid;
        // a few slabs of K and too few big tiles (the decoder's V_hat Z^T; grouped products
        // up to K = 1024 such as the input layer of the 4 x 256-token ReLU experts, K = 768):
        // the small register-staged tile fills the machine without a split (2.5x and 1.5x
        // faster than a split 128x128 tile there). Grouped products whose experts fill
        // 128-row tiles, with at least a round of them (the 16-expert SwiGLU layer's gate-up,
        // K = 1024: 51 against 71 us), stay on the 128x128 tile.
        const bool mid_fills = avg_rows >= 128 && tiles(128, 128) >= gemm_slots<128, 128>();
        if (a.K <= 256 || (a.seg && a.K <= 1024 && !mid_fills)) return Tile::Small;
        if (avg_rows >= 64) return Tile::Mid;
        return Tile::Small;
    }
    if (avg_rows >= 256 && tiles(256, 256) >= 512) return Tile::Big;
    if (avg_rows >= 64 && tiles(128, 128) >= 512) return Tile::Mid;
    return Tile::Small;
}

template <typename T, typename TO, bool SWIGLU>
hipError_t dispatch(const GemmArgs& a, hipStream_t s) {
    constexpr bool kLdsPath = sizeof(T) == 2;
    const bool lds_ok = kLdsPath && a.K % 128 == 0;
    switch (choose_tile(a, SWIGLU, lds_ok)) {
        case Tile::Big:
            if constexpr (kLdsPath)
                if (lds_ok) return run_lds<256, 256, 4, 2, SWIGLU, TO>(a, s);
            return run<T, TO, 256, 256, 2, 2, SWIGLU>(a, s);
        case Tile::Mid:
            if constexpr (kLdsPath)
                if (lds_ok) return run_lds<128, 128, 2, 2, SWIGLU, TO>(a, s);
            return run<T, TO, 128, 128, 2, 2, SWIGLU>(a, s);
        // the small tile streams its whole K a slab at a time: wider slab rows (fewer slabs) for
        // long K, e.g. the 64-expert ReLU layer's output layer (K = 3072): 38.2 against 48.9 us
        // with 256-byte rows, the decode workload's gate-up (K = 4096): 181 against 187 us with
        // 512-byte rows; short K keeps 128-byte rows (K = 768: 19.9 against 22.9 us)
        default:
            if (a.K >= 4096) return run<T, TO, 32, 128, 1, 4, SWIGLU, 32>(a, s);
            if (a.K >= 2048) return run<T, TO, 32, 128, 1, 4, SWIGLU, 16>(a, s);
            return run<T, TO, 32, 128, 1, 4, SWIGLU, 8>(a, s);
    }
}

}  // namespace

size_t gemm_split_scratch_bytes() {
    return std::max(static_cast<size_t>(gemm_slots<256, 256>()) * 256 * 256,
                    static_cast<size_t>(gemm_slots<128, 128>()) * 128 * 128) * sizeof(float);
}

hipError_t launch_gemm(DType dt, Epilogue epi, OutType ot, const GemmArgs& args, hipStream_t s) {
    const bool sw = epi == Epilogue::SwiGLU;
    GemmArgs a = args;
    a.relu = epi == Epilogue::ReLU ? 1 : 0;
    if (dt == DType::BF16) {
        if (sw) return dispatch<bf16_t, bf16_t, true>(a, s);
        if (ot == OutType::F32) return dispatch<bf16_t, float, false>(a, s);
        return dispatch<bf16_t, bf16_t, false>(a, s);
    }
    if (sw) return dispatch<float, float, true>(a, s);
    return dispatch<float, float, false>(a, s);
}

}  // namespace ec2moe
