// Grouped and dense "NT" GEMM on the gfx950 matrix cores.
//
//   out[p][n] = sum_k tok[row(p)][k] * w_e[n][k]     for every row p of group e
//
// Both operands are K-contiguous (token rows of the activations, rows of nn.Linear-style
// weights), which is the layout the expert networks of Eq. 1 and the codec products use.
// Groups are the per-expert segments produced by the permutation; their sizes stay on
// the device. The grid is sized for the upper bound sum_e ceil(n_e / TM) <= ceil(rows/TM)
// + groups, and every workgroup finds its (expert, m-tile, n-tile) with a wave-parallel
// prefix sum over the segment table; surplus workgroups exit.
//
// Workgroup tile: TM token rows x TN weight rows, 4 waves in a WM x WN grid. Each K-step
// moves one 128-byte slab of every tile row (64 bf16 or 32 fp32 values) global -> LDS,
// double-buffered so the next slab's loads are in flight during the matrix-core work on
// the current one. LDS rows are 8 chunks of 16 bytes stored at chunk ^ (row & 7), which
// keeps both the 16-byte stores and the 16-byte fragment reads free of bank conflicts.
// Weight rows feed the MFMA A operand and token rows the B operand, so every lane ends
// with 4 consecutive output columns of one token row (one 8- or 16-byte store).
//
// SwiGLU epilogue: the weight tile holds TN/2 gate rows followed by the matching TN/2 up
// rows; each wave owns equal gate and up slices, so silu(gate) * up is formed in registers.
#include "device_common.h"
#include "internal.h"

#include <algorithm>

namespace ec2moe {
namespace {

struct TileInfo {
    int group;
    int64_t row0;  // first row of the tile (position in the permuted order)
    int valid;     // rows of the tile inside the group
    int nt;        // n-tile index
};

// Finds the tile of this workgroup; false if the workgroup has no tile.
template <int TM>
__device__ __forceinline__ bool find_tile(const GemmArgs& a, int ntn, TileInfo& ti) {
    const int bid = blockIdx.x;
    if (a.seg == nullptr) {
        const int64_t mtiles = (a.rows + TM - 1) / TM;
        if (bid >= mtiles * ntn) return false;
        const int64_t mt = bid % mtiles;
        ti.group = 0;
        ti.nt = static_cast<int>(bid / mtiles);
        ti.row0 = mt * TM;
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
            const int glo = __shfl(lo, src);
            const int ghi = __shfl(hi, src);
            const int mtiles = (ghi - glo + TM - 1) / TM;
            const int local = bid - first;
            ti.group = e0 + src;
            ti.nt = local / mtiles;
            const int mt = local - ti.nt * mtiles;
            ti.row0 = glo + static_cast<int64_t>(mt) * TM;
            ti.valid = std::min(TM, ghi - static_cast<int>(ti.row0));
            return true;
        }
        base += __shfl(inc, 63);
    }
    return false;
}

__device__ __forceinline__ float silu(float g) { return g / (1.0f + expf(-g)); }

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

template <typename T, typename TO, int TM, int TN, int WM, int WN, bool SWIGLU>
__global__ __launch_bounds__(256, 1) void gemm_kernel(GemmArgs a) {
    static_assert(WM * WN == 4, "4 waves per workgroup");
    static_assert(TM % 32 == 0 && TN % 32 == 0, "tiles load 32 rows per pass");
    constexpr int EPC = Elem<T>::kPerChunk;
    constexpr int BK = 8 * EPC;           // elements per 128-byte slab row
    constexpr int MI = TM / WM / 16;      // token blocks per wave
    constexpr int NI = TN / WN / 16;      // weight blocks per wave
    constexpr int TOK_PASSES = TM / 32;
    constexpr int W_PASSES = TN / 32;
    constexpr int NOUT = SWIGLU ? TN / 2 : TN;
    constexpr int ROWS = TM + TN;
    static_assert(!SWIGLU || NI % 2 == 0, "SwiGLU waves hold matching gate/up blocks");

    __shared__ uint4 lds[2][ROWS * 8];

    const int ntn = (a.N + NOUT - 1) / NOUT;
    TileInfo ti;
    if (!find_tile<TM>(a, ntn, ti)) return;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave % WM;
    const int wn = wave / WM;
    const int K = a.K;

    // ---- global load addressing: thread -> (chunk c, rows rr + 32 i)
    const int c = tid & 7;
    const int rr = tid >> 3;
    const T* tok = static_cast<const T*>(a.tok);
    const T* wbase = static_cast<const T*>(a.w) + static_cast<int64_t>(ti.group) * a.w_group_stride;
    uint32_t tok_off[TOK_PASSES];
    uint32_t w_off[W_PASSES];
#pragma unroll
    for (int i = 0; i < TOK_PASSES; ++i) {
        const int r = std::min(rr + 32 * i, ti.valid - 1);
        const int64_t p = ti.row0 + r;
        const int64_t src = a.row_index ? a.row_index[p] : p;
        tok_off[i] = static_cast<uint32_t>(src * K + c * EPC);
    }
#pragma unroll
    for (int i = 0; i < W_PASSES; ++i) {
        const int n = rr + 32 * i;
        int wrow;
        if (SWIGLU) {
            wrow = n < TN / 2 ? ti.nt * (TN / 2) + n : a.N + ti.nt * (TN / 2) + (n - TN / 2);
        } else {
            wrow = std::min(ti.nt * TN + n, a.N - 1);
        }
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
            const int row = rr + 32 * i;
            lds[buf][row * 8 + (c ^ (row & 7))] = stage_t[i];
        }
#pragma unroll
        for (int i = 0; i < W_PASSES; ++i) {
            const int row = TM + rr + 32 * i;
            lds[buf][row * 8 + (c ^ (row & 7))] = stage_w[i];
        }
    };

    // ---- fragment rows of this wave
    const int l16 = lane & 15;
    const int lg = lane >> 4;
    int frag_t[MI];
    int frag_w[NI];
#pragma unroll
    for (int mi = 0; mi < MI; ++mi) frag_t[mi] = wm * (TM / WM) + mi * 16 + l16;
#pragma unroll
    for (int ni = 0; ni < NI; ++ni) {
        int wr;
        if (SWIGLU) {
            constexpr int HALF = NI / 2;
            const int part = ni < HALF ? 0 : TN / 2;
            wr = part + wn * (TN / 2 / WN) + (ni % HALF) * 16 + l16;
        } else {
            wr = wn * (TN / WN) + ni * 16 + l16;
        }
        frag_w[ni] = TM + wr;
    }

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
        for (int s = 0; s < 2; ++s) {
            const int ch = 4 * s + lg;
            uint4 bt[MI];
            uint4 aw[NI];
#pragma unroll
            for (int mi = 0; mi < MI; ++mi) {
                const int row = frag_t[mi];
                bt[mi] = lds[cur][row * 8 + (ch ^ (row & 7))];
            }
#pragma unroll
            for (int ni = 0; ni < NI; ++ni) {
                const int row = frag_w[ni];
                aw[ni] = lds[cur][row * 8 + (ch ^ (row & 7))];
            }
#pragma unroll
            for (int ni = 0; ni < NI; ++ni)
#pragma unroll
                for (int mi = 0; mi < MI; ++mi) acc[ni][mi] = Mfma<T>::step(aw[ni], bt[mi], acc[ni][mi]);
        }
        if (ks + 1 < nk) store_lds(cur ^ 1);
        __syncthreads();
    }

    // ---- epilogue: lane holds token row frag_t[mi] (col l16 of the MFMA output) and
    // weight rows 4*lg .. 4*lg+3 of each block
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
                store4<TO>(orow + col, v);
            }
        } else {
#pragma unroll
            for (int ni = 0; ni < NI; ++ni) {
                const int col = ti.nt * TN + wn * (TN / WN) + ni * 16 + 4 * lg;
                if (col < a.N) store4<TO>(orow + col, acc[ni][mi]);
            }
        }
    }
}

template <typename T, typename TO, int TM, int TN, int WM, int WN, bool SWIGLU>
hipError_t run(const GemmArgs& a, hipStream_t s) {
    constexpr int NOUT = SWIGLU ? TN / 2 : TN;
    const int ntn = (a.N + NOUT - 1) / NOUT;
    int64_t mtiles = a.seg ? (a.rows + TM - 1) / TM + a.n_groups : (a.rows + TM - 1) / TM;
    const int64_t grid = mtiles * ntn;
    if (grid == 0) return hipSuccess;
    ProfileScope prof(a.name ? a.name : "gemm", s);
    hipLaunchKernelGGL((gemm_kernel<T, TO, TM, TN, WM, WN, SWIGLU>), dim3(static_cast<unsigned>(grid)), dim3(256), 0,
                       s, a);
    return hipGetLastError();
}

// Tile choice: the largest tile that still gives at least two workgroups per CU.
enum class Tile { Big, Mid, Small };

Tile choose_tile(const GemmArgs& a, bool swiglu) {
    auto tiles = [&](int tm, int tn) {
        const int nout = swiglu ? tn / 2 : tn;
        const int64_t mt = (a.rows + tm - 1) / tm + (a.seg ? a.n_groups : 0);
        return mt * ((a.N + nout - 1) / nout);
    };
    const int64_t avg_rows = a.seg ? a.rows / std::max(1, a.n_groups) : a.rows;
    if (avg_rows >= 256 && tiles(256, 256) >= 512) return Tile::Big;
    if (avg_rows >= 64 && tiles(128, 128) >= 512) return Tile::Mid;
    return Tile::Small;
}

template <typename T, typename TO, bool SWIGLU>
hipError_t dispatch(const GemmArgs& a, hipStream_t s) {
    switch (choose_tile(a, SWIGLU)) {
        case Tile::Big: return run<T, TO, 256, 256, 2, 2, SWIGLU>(a, s);
        case Tile::Mid: return run<T, TO, 128, 128, 2, 2, SWIGLU>(a, s);
        default: return run<T, TO, 32, 128, 1, 4, SWIGLU>(a, s);
    }
}

}  // namespace

hipError_t launch_gemm(DType dt, Epilogue epi, OutType ot, const GemmArgs& a, hipStream_t s) {
    const bool sw = epi == Epilogue::SwiGLU;
    if (dt == DType::BF16) {
        if (sw) return dispatch<bf16_t, bf16_t, true>(a, s);
        if (ot == OutType::F32) return dispatch<bf16_t, float, false>(a, s);
        return dispatch<bf16_t, bf16_t, false>(a, s);
    }
    if (sw) return dispatch<float, float, true>(a, s);
    return dispatch<float, float, false>(a, s);
}

}  // namespace ec2moe
