// Kernels of the low-rank codec (Encoder-Decoder based on Low-Rank Compression) for gfx950:
// a tiled transpose; the fused encoder of bf16 layers (P = X V and its share of Z = U^T P in
// one workgroup per 64 x 64 tile of P); the contraction Z = U^T P of the other shapes at
// float32 accuracy (P = X V in float32; bfloat16 U on the bf16 matrix cores with P split in
// three bf16 planes, float32 U on the float32 matrix cores); the in-order reduction of the
// partial sums over token tiles or chunks; the small-batch encoder and decoder (at most 64
// tokens per slice, float32 throughout); the decoder's first product W = V_hat bf16(Z)^T of
// bf16 layers in one launch; and the float32 -> bfloat16 rounding of Z for the decoder's
// other shapes. U_hat W^T, and X V outside the fused encoder, run on the matrix-core GEMM.
#include "device_common.h"
#include "internal.h"

#include <algorithm>
#include <string>

namespace ec2moe {
namespace {

template <typename T>
__device__ __forceinline__ float ld(const void* p, int64_t i) {
    return Elem<T>::to_f32(static_cast<const T*>(p)[i]);
}

// dst[c][r] = src[r][c] through 64x64 tiles in LDS; 16-byte global loads and stores
// (rows and cols multiples of 16 / sizeof(T), both pointers 16-byte aligned). The LDS row
// pitch is an odd number of 4-byte words, so a column walk hits distinct banks.
template <typename T>
__global__ __launch_bounds__(256) void transpose_kernel(const T* __restrict__ src, int rows, int cols,
                                                        T* __restrict__ dst) {
    constexpr int EPC = 16 / static_cast<int>(sizeof(T));  // elements per 16-byte chunk
    constexpr int CPR = 64 / EPC;                           // chunks per 64-element tile row
    __shared__ T tile[64][64 + 4 / sizeof(T)];
    const int c0 = blockIdx.x * 64, r0 = blockIdx.y * 64;
    for (int i = threadIdx.x; i < 64 * CPR; i += 256) {
        const int r = i / CPR, ch = i % CPR;
        const int gr = r0 + r, gc = c0 + ch * EPC;
        if (gr < rows && gc < cols) {
            const uint4 v = *reinterpret_cast<const uint4*>(src + static_cast<int64_t>(gr) * cols + gc);
            const T* e = reinterpret_cast<const T*>(&v);
#pragma unroll
            for (int j = 0; j < EPC; ++j) tile[r][ch * EPC + j] = e[j];
        }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < 64 * CPR; i += 256) {
        const int oc = i / CPR, ch = i % CPR;  // output row c0 + oc, output columns r0 + ch * EPC ..
        const int gc = c0 + oc, gr = r0 + ch * EPC;
        if (gc < cols && gr < rows) {
            uint4 v;
            T* e = reinterpret_cast<T*>(&v);
#pragma unroll
            for (int j = 0; j < EPC; ++j) e[j] = tile[ch * EPC + j][oc];
            *reinterpret_cast<uint4*>(dst + static_cast<int64_t>(gc) * rows + gr) = v;
        }
    }
}

constexpr int kUtpT = 64;   // tokens per LDS stage
constexpr int kUtpC = 64;   // columns of P per workgroup
constexpr int kUtpUP = 272;  // LDS pitch of the staged U rows (floats; 272 % 64 = 16: the four
                             // 16-lane groups of a read fall on disjoint banks)
constexpr int kUtpPP = 80;   // LDS pitch of the staged P rows (80 % 64 = 16)

// One token chunk of Z = U^T P: part[s][r][c] = sum over t in chunk s of U[t][r] P[t][c], for
// the 64 columns c0.. of this workgroup and all r_h <= 256 rows (blockIdx.z: the slice, whose
// P rows, partials and Z follow the previous slice's), on the float32 matrix cores
// (v_mfma_f32_16x16x4f32: lane l feeds A[l % 16][l / 16] and B[l / 16][l % 16] and holds
// D[4 (l / 16) + i][l % 16]). Each stage loads 64 token rows of U (converted to float32) and of
// P with 16-byte loads into LDS; rows past the chunk are zero. Wave w owns rows w*64 .. w*64+63.
template <typename TU>
__global__ __launch_bounds__(256) void utp_kernel(UtpArgs g) {
    __shared__ float Us[kUtpT * kUtpUP];
    __shared__ float Ps[kUtpT * kUtpPP];
    constexpr int EPC = 16 / static_cast<int>(sizeof(TU));
    const int c0 = blockIdx.x * kUtpC;
    const int tb = blockIdx.y * g.tc;
    const float* pin_ = g.p + static_cast<int64_t>(blockIdx.z) * g.T * g.rw;
    const int te = min(g.T, tb + g.tc);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int l16 = lane & 15, lg = lane >> 4;
    const int rbase = wave * 64;
    // Waves whose 64 rows all lie past r_h have nothing to compute. In the last active wave
    // the U columns r_h .. (its end) stay zero: its blocks past r_h (and P columns past r_w)
    // multiply zeros, which keeps its matrix-core sequence free of branches; their outputs
    // are not stored.
    const bool active = rbase < g.rh;
    const int zc = ((g.rh + 63) & ~63) - g.rh;
    for (int i = threadIdx.x; i < kUtpT * zc; i += 256) {
        const int r = i / zc, c = g.rh + i % zc;
        Us[r * kUtpUP + c] = 0.f;
    }
    f32x4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    const TU* u = static_cast<const TU*>(g.u);
    for (int t0 = tb; t0 < te; t0 += kUtpT) {
        const int nt = min(kUtpT, te - t0);
        // U rows (rh / EPC chunks per row, at most 8 chunks per thread) and P rows (16 chunks
        // of 4 floats per row, 4 per thread): all loads of the stage issue before the LDS stores
        const int ucpr = g.rh / EPC;
        constexpr int UPT = kUtpT * (256 / EPC) / 256;
        uint4 uq[UPT];
#pragma unroll
        for (int j = 0; j < UPT; ++j) {
            const int i = threadIdx.x + 256 * j;
            const int r = i / ucpr, ch = i % ucpr;
            uq[j] = make_uint4(0, 0, 0, 0);
            if (i < kUtpT * ucpr && r < nt)
                uq[j] = *reinterpret_cast<const uint4*>(u + static_cast<int64_t>(t0 + r) * g.rh + ch * EPC);
        }
        constexpr int PPT = kUtpT * 16 / 256;
        f32x4 pq[PPT];
#pragma unroll
        for (int j = 0; j < PPT; ++j) {
            const int i = threadIdx.x + 256 * j;
            const int r = i / 16, c = c0 + (i % 16) * 4;
            pq[j] = f32x4{0.f, 0.f, 0.f, 0.f};
            if (r < nt && c < g.rw) pq[j] = *reinterpret_cast<const f32x4*>(pin_ + static_cast<int64_t>(t0 + r) * g.rw + c);
        }
#pragma unroll
        for (int j = 0; j < UPT; ++j) {
            const int i = threadIdx.x + 256 * j;
            if (i < kUtpT * ucpr) {
                const int r = i / ucpr, ch = i % ucpr;
                const TU* e = reinterpret_cast<const TU*>(&uq[j]);
#pragma unroll
                for (int q = 0; q < EPC; q += 4)
                    *reinterpret_cast<f32x4*>(Us + r * kUtpUP + ch * EPC + q) =
                        f32x4{Elem<TU>::to_f32(e[q]), Elem<TU>::to_f32(e[q + 1]), Elem<TU>::to_f32(e[q + 2]),
                              Elem<TU>::to_f32(e[q + 3])};
            }
        }
#pragma unroll
        for (int j = 0; j < PPT; ++j) {
            const int i = threadIdx.x + 256 * j;
            *reinterpret_cast<f32x4*>(Ps + (i / 16) * kUtpPP + (i % 16) * 4) = pq[j];
        }
        __syncthreads();
        auto kstep = [&](int k) {
            float a[4], b[4];
#pragma unroll
            for (int rb = 0; rb < 4; ++rb) a[rb] = Us[(k + lg) * kUtpUP + rbase + rb * 16 + l16];
#pragma unroll
            for (int cb = 0; cb < 4; ++cb) b[cb] = Ps[(k + lg) * kUtpPP + cb * 16 + l16];
#pragma unroll
            for (int rb = 0; rb < 4; ++rb)
#pragma unroll
                for (int cb = 0; cb < 4; ++cb)
                    acc[rb][cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[rb], b[cb], acc[rb][cb], 0, 0, 0);
        };
        if (active && nt == kUtpT) {
#pragma unroll
            for (int k = 0; k < kUtpT; k += 4) kstep(k);
        } else if (active) {
            const int nk = (nt + 3) & ~3;
            for (int k = 0; k < nk; k += 4) kstep(k);
        }
        __syncthreads();
    }
    float* part = g.part + (static_cast<int64_t>(blockIdx.z) * gridDim.y + blockIdx.y) * g.rh * g.rw;
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
#pragma unroll
        for (int cb = 0; cb < 4; ++cb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int r = rbase + rb * 16 + 4 * lg + i;
                const int c = c0 + cb * 16 + l16;
                if (r < g.rh && c < g.rw) part[static_cast<int64_t>(r) * g.rw + c] = acc[rb][cb][i];
            }
}

// Z = U^T P with bfloat16 U on the bfloat16 matrix cores at float32 accuracy. Each float32
// value of P is split exactly into three bfloat16 values, p = hi + mid + lo up to 2^-27 |p|
// (hi = bf16(p), mid = bf16(p - hi), lo = bf16(p - hi - mid); each difference is exact in
// float32), and the three products with U, all exact in float32, are accumulated in
// float32: the same order of accuracy as a float32 contraction, at 3/16 of its matrix-core
// cost. Tokens are the contraction axis, so a stage of 64 tokens is staged transposed in
// LDS: U^T as [r][t] rows (an 8x8 register transpose of 16-byte loads) and each plane of P
// as [c][t] rows, 128 bytes per row with the GEMM's chunk swizzle (chunk i of row R at
// i ^ ((R >> 1) & 7)). Wave w owns rows 64 w .. 64 w + 63 of this workgroup's 64 columns:
// 2 x 2 blocks of v_mfma_f32_32x32x16_bf16 (lane l: column l % 32 of a block, rows
// 8 (q / 4) + 4 (l / 32) + q % 4 in register q). Tokens past the chunk are zero in every
// operand. Partials per token chunk as in utp_kernel.
constexpr int kU3T = 64;  // tokens per LDS stage
constexpr int kU3C = 64;  // columns of P per workgroup

__device__ __forceinline__ uint32_t bf16_pair(uint4 a, uint4 b, int j) {
    const uint32_t wa = (&a.x)[j >> 1] >> (16 * (j & 1));
    const uint32_t wb = (&b.x)[j >> 1] >> (16 * (j & 1));
    return (wa & 0xffffu) | (wb << 16);
}

__global__ __launch_bounds__(256) void utp3_kernel(UtpArgs g) {
    __shared__ __attribute__((aligned(1024))) char lds_u[256 * 128];      // U^T [r][64 tokens]
    __shared__ __attribute__((aligned(1024))) char lds_p[3 * kU3C * 128];  // P^T planes [3][c][64 tokens]
    const int c0 = blockIdx.x * kU3C;
    const int tb = blockIdx.y * g.tc;
    const int te = min(g.T, tb + g.tc);
    const float* ps = g.p + static_cast<int64_t>(blockIdx.z) * g.T * g.rw;
    const bf16_t* u = static_cast<const bf16_t*>(g.u);
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int l32 = lane & 31, lh = lane >> 5;
    const int sw = (l32 >> 1) & 7;
    const int rbase = wave * 64;
    const bool active = rbase < g.rh;
    const int rgroups = ((g.rh + 63) & ~63) / 8;  // 8-row groups of U^T staged (zeros past r_h)

    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;

    // Per stage each thread holds at most one U item (8 tokens x 8 rows: 8 * rgroups <= 256)
    // and one P item (8 tokens x 2 columns). The next stage's loads are issued before this
    // stage's matrix-core work, so they fly while it runs.
    const bool has_u = tid < 8 * rgroups;
    const int urg = tid % rgroups, utg = tid / rgroups;
    const int pcg = tid % 32, ptg = tid / 32;
    const int pc = c0 + pcg * 2;
    uint4 rowv[8];
    float2 pv[8];
    auto load_stage = [&](int t0) {
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int t = t0 + utg * 8 + q;
            rowv[q] = (has_u && t < te && urg * 8 < g.rh) ? ldg16(u + static_cast<int64_t>(t) * g.rh + urg * 8)
                                                          : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int t = t0 + ptg * 8 + q;
            pv[q] = (t < te && pc < g.rw) ? *reinterpret_cast<const float2*>(ps + static_cast<int64_t>(t) * g.rw + pc)
                                          : make_float2(0.f, 0.f);
        }
    };
    if (tb < te) load_stage(tb);
    for (int t0 = tb; t0 < te; t0 += kU3T) {
        // U^T rows r0 .. r0 + 7, 8 tokens of group utg: an 8 x 8 transpose in registers
        if (has_u) {
            const int r0 = urg * 8;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int R = r0 + j;
                const uint4 o = make_uint4(bf16_pair(rowv[0], rowv[1], j), bf16_pair(rowv[2], rowv[3], j),
                                           bf16_pair(rowv[4], rowv[5], j), bf16_pair(rowv[6], rowv[7], j));
                *reinterpret_cast<uint4*>(lds_u + R * 128 + ((utg ^ ((R >> 1) & 7)) * 16)) = o;
            }
        }
        // P^T planes: columns pc, pc + 1, each value split into hi, mid, lo
#pragma unroll
        for (int cc = 0; cc < 2; ++cc) {
            uint32_t hw[4], mw[4], lw[4];
#pragma unroll
            for (int q = 0; q < 8; q += 2) {
                uint32_t hb[2], mb[2], lb[2];
#pragma unroll
                for (int e = 0; e < 2; ++e) {
                    const float v = cc ? pv[q + e].y : pv[q + e].x;
                    const uint16_t h = f32_to_bf16(v);
                    const float r1 = v - bf16_to_f32(h);
                    const uint16_t m = f32_to_bf16(r1);
                    const float r2 = r1 - bf16_to_f32(m);
                    hb[e] = h;
                    mb[e] = m;
                    lb[e] = f32_to_bf16(r2);
                }
                hw[q / 2] = hb[0] | (hb[1] << 16);
                mw[q / 2] = mb[0] | (mb[1] << 16);
                lw[q / 2] = lb[0] | (lb[1] << 16);
            }
            const int R = pcg * 2 + cc;
            const int off = R * 128 + ((ptg ^ ((R >> 1) & 7)) * 16);
            *reinterpret_cast<uint4*>(lds_p + 0 * kU3C * 128 + off) = make_uint4(hw[0], hw[1], hw[2], hw[3]);
            *reinterpret_cast<uint4*>(lds_p + 1 * kU3C * 128 + off) = make_uint4(mw[0], mw[1], mw[2], mw[3]);
            *reinterpret_cast<uint4*>(lds_p + 2 * kU3C * 128 + off) = make_uint4(lw[0], lw[1], lw[2], lw[3]);
        }
        __syncthreads();
        if (t0 + kU3T < te) load_stage(t0 + kU3T);
        if (active) {
#pragma unroll
            for (int s = 0; s < kU3T / 16; ++s) {
                const int ch = ((2 * s + lh) ^ sw) * 16;
                uint4 a[2], b[3][2];
#pragma unroll
                for (int rb = 0; rb < 2; ++rb) a[rb] = *reinterpret_cast<const uint4*>(lds_u + (rbase + rb * 32 + l32) * 128 + ch);
#pragma unroll
                for (int j = 0; j < 3; ++j)
#pragma unroll
                    for (int cb = 0; cb < 2; ++cb)
                        b[j][cb] = *reinterpret_cast<const uint4*>(lds_p + (j * kU3C + cb * 32 + l32) * 128 + ch);
#pragma unroll
                for (int j = 0; j < 3; ++j)
#pragma unroll
                    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
                        for (int cb = 0; cb < 2; ++cb)
                            acc[rb][cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                                __builtin_bit_cast(bf16x8, a[rb]), __builtin_bit_cast(bf16x8, b[j][cb]), acc[rb][cb], 0, 0,
                                0);
            }
        }
        __syncthreads();
    }
    if (!active) return;
    float* part = g.part + (static_cast<int64_t>(blockIdx.z) * gridDim.y + blockIdx.y) * g.rh * g.rw;
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
#pragma unroll
            for (int q = 0; q < 16; ++q) {
                const int r = rbase + rb * 32 + 8 * (q / 4) + 4 * lh + (q % 4);
                const int c = c0 + cb * 32 + l32;
                if (r < g.rh && c < g.rw) part[static_cast<int64_t>(r) * g.rw + c] = acc[rb][cb][q];
            }
}

// ------------------------------------------------------------------ fused encoder (bf16 layers)
//
// One workgroup per (64-token tile, 64-column tile) of P = X V: the tile's products over the
// whole model width (no split along it), then at once its share of Z = U^T P,
//   part[s][tt][r][c] = sum over the tile's 64 tokens t of U[t][r] P[t][c],
// which split_reduce_kernel adds over the token tiles in order. X and V (as stored, [w][r_w])
// stream through a ring of four LDS stages of 128 model columns (32 KB: 64 token rows of 256
// bytes, and the 128 rows of V for those model columns, 128 bytes each: the tile's 64 columns)
// filled by buffer_load ... lds, so three stages are in flight while one is consumed. V's
// operand fragments need 8 consecutive model columns per lane, which run down the staged
// rows: the gfx950 transposing LDS read (ds_read_b64_tr_b16) gathers them, 4 rows at a time. Eight waves: wave w computes the 32x32 block (w & 1, (w >> 1) & 1) of the
// P tile over the even (w < 4) or odd (w >= 4) 16-column steps of each stage; the two halves
// are added once at the end. The P tile is then split exactly into three bf16 planes
// (hi + mid + lo) and, with U^T, staged in LDS for the bf16 matrix cores, as in utp3_kernel.
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

}  // namespace

// buffer_load_dwordx4 ... lds: each lane's 16 bytes land at M0 + 16 * lane
__device__ void raw_buffer_load_lds(i32x4 rsrc, lds_void* lds, int size, int voffset, int soffset, int offset,
                                    int aux) __asm("llvm.amdgcn.raw.buffer.load.lds");

namespace {

__device__ __forceinline__ i32x4 enc_rsrc(const void* base, uint32_t bytes) {
    const uint64_t p = reinterpret_cast<uint64_t>(base);
    i32x4 r;
    r[0] = __builtin_amdgcn_readfirstlane(static_cast<int>(static_cast<uint32_t>(p)));
    r[1] = __builtin_amdgcn_readfirstlane(static_cast<int>(static_cast<uint32_t>(p >> 32)));
    r[2] = __builtin_amdgcn_readfirstlane(static_cast<int>(bytes));
    r[3] = 0x00020000;  // raw (untyped, unswizzled) buffer of the gfx9 family
    return r;
}

constexpr int kEncT = 64;                            // tokens per tile
constexpr int kEncC = 64;                            // columns of P per tile
constexpr int kEncK = 128;                           // model columns per LDS stage
constexpr int kEncRing = 4;                          // LDS stages
constexpr int kEncRow = kEncK * 2;                   // bytes per staged row
constexpr int kEncStage = (kEncT + kEncC) * kEncRow;  // 32 KB
constexpr int kEncLoads = 4;                         // DMA instructions per wave per stage

// gfx950 transposing LDS read of 16-bit data: in each group of 16 lanes, lane i reads the 8 bytes
// at its address (elements S[i][0..3]) and receives S[4 e + i / 4][i % 4] in element e
typedef short i16x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint2 lds_read_tr16(const char* p) {
    const i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) i16x4*)(const_cast<char*>(p)));
    return __builtin_bit_cast(uint2, v);
}

__global__ __launch_bounds__(512, 1) void encode_fused_kernel(EncArgs a) {
    // one LDS object per ring slot, each named at compile time where it is read, so the wait
    // before a fragment read only covers the DMA into that slot
    __shared__ __attribute__((aligned(1024))) char lds0[kEncStage];
    __shared__ __attribute__((aligned(1024))) char lds1[kEncStage];
    __shared__ __attribute__((aligned(1024))) char lds2[kEncStage];
    __shared__ __attribute__((aligned(1024))) char lds3[kEncStage];
    static_assert(kEncT * kEncRow == kEncK * kEncC * 2, "token rows and V rows fill equal halves of a stage");
    const int ct_n = a.rw / kEncC, tt_n = a.h / kEncT;
    const int n = ct_n * tt_n * a.slices;
    const int g = blockIdx.x;
    int ct, tts;
    if (n % (8 * ct_n) == 0) {
        // the column tiles of one token tile run on one XCD (workgroups go round-robin over the
        // eight): X rows are fetched into that XCD's L2 once for all of them
        const int q = g / 8;
        ct = q % ct_n;
        tts = g % 8 + 8 * (q / ct_n);
    } else {
        ct = g % ct_n;
        tts = g / ct_n;
    }
    const int s = tts / tt_n, tt = tts % tt_n;

    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l32 = lane & 31, lh = lane >> 5;
    const uint32_t row_bytes = static_cast<uint32_t>(a.w) * 2u;

    // U^T staging items (8 tokens x 8 rows of U^T each), loaded first: their loads are older
    // than every DMA load, so the counted waits of the ring also cover them
    const int rgroups = ((a.rh + 63) & ~63) / 8;
    const bool has_u = tid < 8 * rgroups;
    const int urg = tid % rgroups, utg = tid / rgroups;
    uint4 rowv[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        const int t = tt * kEncT + utg * 8 + q;
        rowv[q] = has_u && urg * 8 < a.rh ? ldg16(static_cast<const bf16_t*>(a.u) + static_cast<int64_t>(t) * a.rh + urg * 8)
                                           : make_uint4(0, 0, 0, 0);
    }

    // DMA, 1 KB per instruction: waves 0..3 fill token rows 16 w .. 16 w + 15 of the stage's first
    // half (four rows of 256 bytes per instruction; chunk c of row R sits at c ^ (R % 16)), waves
    // 4..7 V rows 32 (w - 4) .. + 31 of its second half (eight rows of 128 bytes per instruction;
    // chunk c of V row k sits at c ^ 2 (k % 4)); both swizzles are applied on the global side
    const bool tok_wave = wave < 4;
    const uint32_t vrow_bytes = static_cast<uint32_t>(a.rw) * 2u;
    const i32x4 rs = tok_wave
        ? enc_rsrc(static_cast<const bf16_t*>(a.x) + (static_cast<int64_t>(s) * a.h + static_cast<int64_t>(tt) * kEncT) * a.w,
                   kEncT * row_bytes)
        : enc_rsrc(a.v, static_cast<uint32_t>(a.w) * vrow_bytes);
    const int sstep = tok_wave ? kEncRow : kEncK * static_cast<int>(vrow_bytes);  // bytes per stage
    uint32_t voff[kEncLoads];
#pragma unroll
    for (int j = 0; j < kEncLoads; ++j) {
        if (tok_wave) {
            const int row = 16 * wave + 4 * j + (lane >> 4);
            voff[j] = static_cast<uint32_t>(row) * row_bytes + static_cast<uint32_t>(((lane & 15) ^ (row & 15)) * 16);
        } else {
            const int k = 32 * (wave - 4) + 8 * j + (lane >> 3);
            voff[j] = static_cast<uint32_t>(k) * vrow_bytes + static_cast<uint32_t>(ct * kEncC * 2) +
                      static_cast<uint32_t>(((lane & 7) ^ (2 * (k & 3))) * 16);
        }
    }
    auto issue = [&](int st, char* slot) {
        char* base = slot + 16 * wave * kEncRow;
#pragma unroll
        for (int j = 0; j < kEncLoads; ++j)
            raw_buffer_load_lds(rs, reinterpret_cast<lds_void*>(reinterpret_cast<uintptr_t>(base + 4 * j * kEncRow)), 16,
                                static_cast<int>(voff[j]), st * sstep, 0, 0);
    };

    // fragments: A = column 32 wn + l32 of P (V's column ct * 64 + 32 wn + l32), model columns
    // 16 (2 q + kh) + 8 lh .. + 7 of the stage in k-step q; B = token row 32 wm + l32, the 16
    // bytes of logical chunk 2 (2 q + kh) + lh. A transposing read by the 16 lanes of a group
    // (g = lane / 16, i = lane % 16) takes 8 bytes from V row k0 + i / 4 at columns
    // mb + 4 (i % 4) .. + 3 and hands lane i the 4 rows k0 .. k0 + 3 of column mb + i; here
    // k0 = 16 (2 q + kh) + 8 (g / 2) + 4 h for the halves h = 0, 1 of the lane's 8 model columns
    // and mb = 32 wn + 16 (g % 2), so lane l gets column 32 wn + l % 32 as the product needs
    const int wm = wave & 1, wn = (wave >> 1) & 1, kh = wave >> 2;
    const int rb = 32 * wm + l32;
    const int gi = lane & 15, gg = lane >> 4;
    const int chv = 4 * wn + 2 * (gg & 1) + ((gi & 3) >> 1);  // 16-byte chunk of the V row
    const int offv = kEncT * kEncRow + ((chv ^ (2 * (gi >> 2))) * 16) + (gi & 1) * 8;
    int offa[4][2], offb[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int ch = 2 * (2 * q + kh) + lh;
#pragma unroll
        for (int h = 0; h < 2; ++h) offa[q][h] = offv + (16 * (2 * q + kh) + 8 * (gg >> 1) + 4 * h + (gi >> 2)) * 128;
        offb[q] = rb * kEncRow + ((ch ^ (rb & 15)) * 16);
    }
    f32x16 acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;

    const int ns = a.w / kEncK;
    auto step = [&](int st, const char* cur, char* refill) {
        if (st >= ns) return;
        const int later = min(kEncRing - 2, ns - 1 - st);  // stages issued after this one
        if (later >= 2) __builtin_amdgcn_s_waitcnt(0x0070 | (2 * kEncLoads));
        else if (later == 1) __builtin_amdgcn_s_waitcnt(0x0070 | kEncLoads);
        else __builtin_amdgcn_s_waitcnt(0x0070);
        // every wave's loads of this stage are in LDS, and every wave is done with the previous
        // stage, whose slot is refilled next (a bare barrier: __syncthreads would also wait for
        // the loads still in flight)
        __builtin_amdgcn_sched_barrier(0);
        asm volatile("s_barrier" ::: "memory");
        __builtin_amdgcn_sched_barrier(0);
        if (st + kEncRing - 1 < ns) issue(st + kEncRing - 1, refill);
        uint4 fa[4], fb[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const uint2 lo = lds_read_tr16(cur + offa[q][0]), hi = lds_read_tr16(cur + offa[q][1]);
            fa[q] = make_uint4(lo.x, lo.y, hi.x, hi.y);
            fb[q] = *reinterpret_cast<const uint4*>(cur + offb[q]);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q)
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, fa[q]), __builtin_bit_cast(bf16x8, fb[q]),
                                                          acc, 0, 0, 0);
    };
    if (ns > 0) issue(0, lds0);
    if (ns > 1) issue(1, lds1);
    if (ns > 2) issue(2, lds2);
    for (int st = 0; st < ns; st += kEncRing) {
        step(st, lds0, lds3);
        step(st + 1, lds1, lds0);
        step(st + 2, lds2, lds1);
        step(st + 3, lds3, lds2);
    }

    // the odd-step half of each block is added to the even-step half
    __syncthreads();
    float* red = reinterpret_cast<float*>(lds0);
    if (kh == 1) {
#pragma unroll
        for (int r = 0; r < 16; ++r) red[((wave - 4) * 16 + r) * 64 + lane] = acc[r];
    }
    char* lds_u = lds1;  // U^T [r][64 tokens], 128-byte rows (32 KB)
    char* lds_p = lds2;  // P^T planes [3][64 columns][64 tokens] (24 KB)
    __syncthreads();
    if (kh == 0) {
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[r] += red[(wave * 16 + r) * 64 + lane];
        // lane holds token j = 32 wm + l32 and, in register r, column i = 32 wn + 8 (r / 4) + 4 lh + r % 4
        const int j = 32 * wm + l32;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int i = 32 * wn + 8 * (r / 4) + 4 * lh + (r % 4);
            const float v = acc[r];
            const uint16_t hi = f32_to_bf16(v);
            const float r1 = v - bf16_to_f32(hi);
            const uint16_t mid = f32_to_bf16(r1);
            const uint16_t lo = f32_to_bf16(r1 - bf16_to_f32(mid));
            const int off = i * 128 + (((j >> 3) ^ ((i >> 1) & 7)) * 16) + (j & 7) * 2;
            *reinterpret_cast<uint16_t*>(lds_p + 0 * kEncC * 128 + off) = hi;
            *reinterpret_cast<uint16_t*>(lds_p + 1 * kEncC * 128 + off) = mid;
            *reinterpret_cast<uint16_t*>(lds_p + 2 * kEncC * 128 + off) = lo;
        }
    }
    if (has_u) {
        const int r0 = urg * 8;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int R = r0 + j;
            const uint4 o = make_uint4(bf16_pair(rowv[0], rowv[1], j), bf16_pair(rowv[2], rowv[3], j),
                                       bf16_pair(rowv[4], rowv[5], j), bf16_pair(rowv[6], rowv[7], j));
            *reinterpret_cast<uint4*>(lds_u + R * 128 + ((utg ^ ((R >> 1) & 7)) * 16)) = o;
        }
    }
    __syncthreads();

    // Z share: wave w owns rows 64 (w & 3) .. + 63 of U^T P and the 32 columns 32 (w >> 2) ..
    const int rbase = 64 * (wave & 3), cb = wave >> 2;
    if (rbase >= a.rh) return;
    f32x16 z[2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) z[i][r] = 0.f;
    const int sw = (l32 >> 1) & 7;
#pragma unroll
    for (int q = 0; q < kEncT / 16; ++q) {
        const int ch = ((2 * q + lh) ^ sw) * 16;
        uint4 ua[2], pb[3];
#pragma unroll
        for (int i = 0; i < 2; ++i) ua[i] = *reinterpret_cast<const uint4*>(lds_u + (rbase + 32 * i + l32) * 128 + ch);
#pragma unroll
        for (int pl = 0; pl < 3; ++pl) pb[pl] = *reinterpret_cast<const uint4*>(lds_p + (pl * kEncC + 32 * cb + l32) * 128 + ch);
#pragma unroll
        for (int pl = 0; pl < 3; ++pl)
#pragma unroll
            for (int i = 0; i < 2; ++i)
                z[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, ua[i]), __builtin_bit_cast(bf16x8, pb[pl]),
                                                               z[i], 0, 0, 0);
    }
    float* part = a.part + (static_cast<int64_t>(s) * tt_n + tt) * a.rh * a.rw;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            const int r = rbase + 32 * i + 8 * (q / 4) + 4 * lh + (q % 4);
            const int c = ct * kEncC + 32 * cb + l32;
            if (r < a.rh) part[static_cast<int64_t>(r) * a.rw + c] = z[i][q];
        }
}

// ------------------------------------------------------------------ small batches (h <= 64 tokens)
//
// With a few dozen tokens per slice the codec's products are tiny, and the launches of the
// general path cost more than their work. Three launches do the whole round trip with float32
// arithmetic throughout (exact products for bf16 layers), Z and U_hat Z kept in float32:
//   enc_small_partial: part[s][kc][t][c] = sum over the 64 model columns k of chunk kc of
//                      X[s][t][k] V[k][c] (one workgroup per chunk, 16 columns of P and slice);
//   enc_small_finish:  P[t][c] = the chunk partials added in a fixed order (the even and the
//                      odd chunks each in order, then the two sums), then
//                      Z[s] = U^T P (one workgroup per 2 columns of Z and slice);
//   dec_small:         Y = U_hat Z[s] (h x r_w), then X_hat[s][t][j] = sum_c Y[t][c] V_hat[j][c] for 32
//                      model columns j per workgroup, rounded once to the layer dtype.
constexpr int kSmallT = 64;   // tokens per slice at most
constexpr int kSmallK = 64;   // model columns per encoder chunk
constexpr int kSmallPC = 16;  // columns of P per partial workgroup
constexpr int kSmallZC = 2;   // columns of Z per finishing workgroup
constexpr int kSmallJ = 32;   // model columns per decoder workgroup

template <typename T>
__device__ __forceinline__ void load_chunk_f32(const T* src, float* dst) {
    const uint4 v = ldg16(src);
    const T* e = reinterpret_cast<const T*>(&v);
#pragma unroll
    for (int i = 0; i < Elem<T>::kPerChunk; ++i) dst[i] = Elem<T>::to_f32(e[i]);
}

template <typename T>
__global__ __launch_bounds__(256) void enc_small_partial_kernel(const T* __restrict__ x, const T* __restrict__ v,
                                                                int h, int w, int rw, float* __restrict__ part) {
    constexpr int EPC = Elem<T>::kPerChunk;
    __shared__ float xs[kSmallT][kSmallK + 1];
    __shared__ float vs[kSmallK][kSmallPC];
    const int kc = blockIdx.x, c0 = blockIdx.y * kSmallPC, s = blockIdx.z, nkc = gridDim.x;
    const int k0 = kc * kSmallK;
    const T* xsl = x + static_cast<int64_t>(s) * h * w;
    for (int e = threadIdx.x; e < h * (kSmallK / EPC); e += 256) {
        const int t = e / (kSmallK / EPC), q = (e % (kSmallK / EPC)) * EPC;
        load_chunk_f32(xsl + static_cast<int64_t>(t) * w + k0 + q, &xs[t][q]);
    }
    for (int e = threadIdx.x; e < kSmallK * (kSmallPC / EPC); e += 256) {
        const int k = e / (kSmallPC / EPC), q = (e % (kSmallPC / EPC)) * EPC;
        load_chunk_f32(v + static_cast<int64_t>(k0 + k) * rw + c0 + q, &vs[k][q]);
    }
    __syncthreads();
    float* out = part + (static_cast<int64_t>(s) * nkc + kc) * h * rw;
    for (int o = threadIdx.x; o < h * kSmallPC; o += 256) {
        const int t = o / kSmallPC, c = o % kSmallPC;
        float acc = 0.f;
#pragma unroll 16
        for (int k = 0; k < kSmallK; ++k) acc = fmaf(xs[t][k], vs[k][c], acc);
        out[static_cast<int64_t>(t) * rw + c0 + c] = acc;
    }
}

template <typename T>
__global__ __launch_bounds__(256) void enc_small_finish_kernel(const float* __restrict__ part, const T* __restrict__ u,
                                                               int h, int rh, int rw, int nkc, float* __restrict__ z) {
    constexpr int RUNS = 256 / (kSmallT * kSmallZC);  // interleaved runs of chunks per element (2)
    __shared__ float red[RUNS][kSmallT * kSmallZC];
    __shared__ float ps[kSmallT][kSmallZC];
    __shared__ float us[kSmallT][kSmallT + 1];
    const int c0 = blockIdx.x * kSmallZC, s = blockIdx.y;
    const float* src = part + static_cast<int64_t>(s) * nkc * h * rw;
    const int e = threadIdx.x % (kSmallT * kSmallZC), run = threadIdx.x / (kSmallT * kSmallZC);
    const int t = e / kSmallZC, c = e % kSmallZC;
    float acc = 0.f;
    if (t < h) {
        const float* col = src + static_cast<int64_t>(t) * rw + c0 + c;
        // chunks run, run + RUNS, ... in order, 16 loads in flight at a time
        for (int q0 = run; q0 < nkc; q0 += 16 * RUNS) {
            float vq[16];
#pragma unroll
            for (int q = 0; q < 16; ++q) {
                const int ch = q0 + q * RUNS;
                vq[q] = ch < nkc ? col[static_cast<int64_t>(ch) * h * rw] : 0.f;
            }
#pragma unroll
            for (int q = 0; q < 16; ++q)
                if (q0 + q * RUNS < nkc) acc += vq[q];
        }
    }
    red[run][e] = acc;
    for (int i = threadIdx.x; i < h * rh; i += 256) us[i / rh][i % rh] = Elem<T>::to_f32(u[i]);
    __syncthreads();
    if (threadIdx.x < kSmallT * kSmallZC && t < h) {
        float sum = red[0][e];
#pragma unroll
        for (int r = 1; r < RUNS; ++r) sum += red[r][e];
        ps[t][c] = sum;
    }
    __syncthreads();
    float* zs = z + static_cast<int64_t>(s) * rh * rw;
    for (int o = threadIdx.x; o < rh * kSmallZC; o += 256) {
        const int i = o / kSmallZC, cc = o % kSmallZC;
        float zacc = 0.f;
        for (int tt = 0; tt < h; ++tt) zacc = fmaf(us[tt][i], ps[tt][cc], zacc);
        zs[static_cast<int64_t>(i) * rw + c0 + cc] = zacc;
    }
}

template <typename T>
__global__ __launch_bounds__(256) void dec_small_kernel(const float* __restrict__ z, const T* __restrict__ u_hat,
                                                        const T* __restrict__ v_hat, int h, int w, int rh, int rw,
                                                        T* __restrict__ x_hat) {
    constexpr int EPC = Elem<T>::kPerChunk;
    constexpr int TG = 256 / kSmallJ;      // token groups (8)
    constexpr int TPT = kSmallT / TG;      // tokens per thread at most (8)
    constexpr int PRE = 32 / EPC;          // V_hat chunks loaded before the first barrier (32 columns)
    __shared__ float zs[kSmallT][256];          // Z [r_h][r_w]
    __shared__ float uh[kSmallT][kSmallT + 1];  // U_hat [h][r_h]
    __shared__ float ys[kSmallT][256];          // Y = U_hat Z [h][r_w]
    const int j0 = blockIdx.x * kSmallJ, s = blockIdx.y;
    const int j = j0 + (threadIdx.x % kSmallJ), tg = threadIdx.x / kSmallJ;
    const T* vrow = v_hat + static_cast<int64_t>(j) * rw;
    // the first columns of this thread's V_hat row, loaded while Y is formed
    uint4 vpre[PRE];
#pragma unroll
    for (int q = 0; q < PRE; ++q) vpre[q] = q * EPC < rw ? ldg16(vrow + q * EPC) : make_uint4(0, 0, 0, 0);
    const float* zsl = z + static_cast<int64_t>(s) * rh * rw;
    for (int e = threadIdx.x; e < rh * rw; e += 256) zs[e / rw][e % rw] = zsl[e];
    for (int e = threadIdx.x; e < h * rh; e += 256) uh[e / rh][e % rh] = Elem<T>::to_f32(u_hat[e]);
    __syncthreads();
    for (int o = threadIdx.x; o < h * rw; o += 256) {
        const int t = o / rw, c = o % rw;
        float acc = 0.f;
        for (int i = 0; i < rh; ++i) acc = fmaf(uh[t][i], zs[i][c], acc);
        ys[t][c] = acc;
    }
    __syncthreads();
    float acc[TPT];
#pragma unroll
    for (int q = 0; q < TPT; ++q) acc[q] = 0.f;
    auto columns = [&](int c, const uint4& raw) {
        const T* e = reinterpret_cast<const T*>(&raw);
#pragma unroll
        for (int q = 0; q < TPT; ++q) {
            const int t = tg + TG * q;
            if (t < h) {
#pragma unroll
                for (int i = 0; i < EPC; ++i) acc[q] = fmaf(ys[t][c + i], Elem<T>::to_f32(e[i]), acc[q]);
            }
        }
    };
#pragma unroll
    for (int q = 0; q < PRE; ++q)
        if (q * EPC < rw) columns(q * EPC, vpre[q]);
    for (int c = PRE * EPC; c < rw; c += EPC) columns(c, ldg16(vrow + c));
    T* out = x_hat + static_cast<int64_t>(s) * h * w;
#pragma unroll
    for (int q = 0; q < TPT; ++q) {
        const int t = tg + TG * q;
        if (t < h) out[static_cast<int64_t>(t) * w + j] = Elem<T>::from_f32(acc[q]);
    }
}

// ------------------------------------------------------------------ decoder, X_hat = U_hat Wt^T (bf16)
//
// X_hat[t][j] = sum_i U_hat[t][i] Wt[j][i] over K = r_h (128 or 256), rounded to bfloat16: a
// rank-r_h expansion whose cost is its 2-byte output. A workgroup owns a band of 128 tokens and a
// run of 64-column chunks of X_hat. Each of its four waves holds the U_hat operand fragments of its
// 32 tokens in registers for the whole run; the chunks' Wt rows (64 x r_h, K-contiguous) stream
// through two LDS buffers by buffer_load ... lds. A chunk's results wait in registers (packed to
// bf16) and are stored after the next chunk's loads have landed, so the stores drain during that
// chunk's products instead of under the wait for its loads (the wait is vmcnt(0): loads and stores
// are not counted in order with each other). Two workgroups per CU overlap each other's waits.
// Wt is the A operand of v_mfma_f32_16x16x32_bf16 with its rows permuted: operand row m = 4 g + e
// of block b is column 16 g + 4 b + e of the chunk, so a lane's 16 results of one token are 16
// consecutive columns. Each wave passes its 32 x 64 results through 4 KB of LDS so that every
// store instruction writes 8 whole 128-byte row pieces (16-byte pieces spread over 16 rows per
// instruction: 8% slower). Staged Wt row R keeps its 16-byte chunk c at c ^ ex_swz(R), which
// spreads the 16 rows read by one group of lanes over distinct banks; the output staging keeps
// piece p of row r at p ^ (r % 8).
constexpr int kExT = 128;  // tokens per band: four waves of 32
constexpr int kExC = 64;   // columns of X_hat per chunk

__device__ __forceinline__ int ex_swz(int r) { return (r & 3) | (((r >> 4) & 3) << 2); }

template <int RH>
__global__ __launch_bounds__(256, 2) void expand_kernel(const bf16_t* __restrict__ u_hat, const bf16_t* __restrict__ wt,
                                                       int w, int cpw, bf16_t* __restrict__ x_hat) {
    constexpr int ROWB = RH * 2;         // bytes per Wt row
    constexpr int CHB = kExC * ROWB;     // bytes per chunk
    constexpr int CPR = ROWB / 16;       // 16-byte pieces per row
    constexpr int RPI = 1024 / ROWB;     // rows per DMA instruction (1 KB)
    constexpr int NLD = CHB / 1024 / 4;  // DMA instructions per wave per chunk
    constexpr int KS = RH / 32;          // k-steps
    __shared__ __attribute__((aligned(1024))) char buf0[CHB];
    __shared__ __attribute__((aligned(1024))) char buf1[CHB];
    __shared__ __attribute__((aligned(1024))) char ostage[4 * 32 * kExC * 2];
    const int nch = w / kExC;
    const int nranges = (nch + cpw - 1) / cpw;
    const int band = blockIdx.x / nranges;
    const int c0 = (blockIdx.x % nranges) * cpw, c1 = min(c0 + cpw, nch);

    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l16 = lane & 15, g = lane >> 4;

    // U_hat fragments: token 32 wave + 16 n + l16 of the band, k-run 8 g of step s
    uint4 fb[2][KS];
    const bf16_t* urow = u_hat + (static_cast<int64_t>(band) * kExT + 32 * wave + l16) * RH + 8 * g;
#pragma unroll
    for (int n = 0; n < 2; ++n)
#pragma unroll
        for (int s = 0; s < KS; ++s) fb[n][s] = ldg16(urow + 16 * n * RH + 32 * s);

    // DMA: instruction j of the wave fills bytes 1024 (NLD wave + j) .. + 1023 of a buffer, i.e.
    // row R = RPI (NLD wave + j) + lane / CPR, position lane % CPR
    const i32x4 rs = enc_rsrc(wt, static_cast<uint32_t>(w) * ROWB);
    uint32_t voff[NLD];
#pragma unroll
    for (int j = 0; j < NLD; ++j) {
        const int R = RPI * (NLD * wave + j) + lane / CPR;
        voff[j] = static_cast<uint32_t>(R * ROWB + (((lane % CPR) ^ ex_swz(R)) * 16));
    }
    auto issue = [&](int c, char* buf) {
        char* base = buf + 1024 * NLD * wave;
#pragma unroll
        for (int j = 0; j < NLD; ++j)
            raw_buffer_load_lds(rs, reinterpret_cast<lds_void*>(reinterpret_cast<uintptr_t>(base + 1024 * j)), 16,
                                static_cast<int>(voff[j]), c * CHB, 0, 0);
    };
    // A fragments: operand row l16 of block b is chunk row 16 (l16 / 4) + 4 b + l16 % 4
    int rowoff[4], rsw[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
        const int R = 16 * (l16 >> 2) + 4 * b + (l16 & 3);
        rowoff[b] = R * ROWB;
        rsw[b] = ex_swz(R);
    }
    // output staging of the wave (32 rows of 128 bytes); store q of a lane: row 8 q + lane / 8 of the
    // wave's tokens, columns 8 (lane % 8) .. + 7 of the chunk
    char* ost = ostage + wave * (32 * kExC * 2);
    bf16_t* orow = x_hat + (static_cast<int64_t>(band) * kExT + 32 * wave + (lane >> 3)) * w + 8 * (lane & 7);

    // the previous chunk's results, read back from the staging in store order (named values, not
    // an array: an array read by the deferred stores was kept in scratch memory)
    uint4 p0, p1, p2, p3;
    const int64_t w8 = static_cast<int64_t>(8) * w;
    auto store_pending = [&](int c) {
        bf16_t* dst = orow + c * kExC;
        *reinterpret_cast<uint4*>(dst) = p0;
        *reinterpret_cast<uint4*>(dst + w8) = p1;
        *reinterpret_cast<uint4*>(dst + 2 * w8) = p2;
        *reinterpret_cast<uint4*>(dst + 3 * w8) = p3;
    };
    if (c0 < c1) issue(c0, buf0);
    for (int c = c0; c < c1; ++c) {
        const bool odd = (c - c0) & 1;
        const char* cur = odd ? buf1 : buf0;
        char* nxt = odd ? buf0 : buf1;
        // this chunk's rows are in LDS (and the stores issued before its products are done);
        // after the barrier every wave is done reading the other buffer, which is refilled next
        __builtin_amdgcn_s_waitcnt(0x0070);
        __builtin_amdgcn_sched_barrier(0);
        asm volatile("s_barrier" ::: "memory");
        __builtin_amdgcn_sched_barrier(0);
        if (c + 1 < c1) issue(c + 1, nxt);
        if (c > c0) store_pending(c - 1);
        f32x4 acc[2][4];
#pragma unroll
        for (int n = 0; n < 2; ++n)
#pragma unroll
            for (int b = 0; b < 4; ++b) acc[n][b] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            uint4 fa[4];
#pragma unroll
            for (int b = 0; b < 4; ++b) fa[b] = *reinterpret_cast<const uint4*>(cur + rowoff[b] + (((4 * s + g) ^ rsw[b]) * 16));
#pragma unroll
            for (int n = 0; n < 2; ++n)
#pragma unroll
                for (int b = 0; b < 4; ++b)
                    acc[n][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, fa[b]),
                                                                         __builtin_bit_cast(bf16x8, fb[n][s]), acc[n][b], 0, 0, 0);
        }
        // lane: token 16 n + l16 of the wave, columns 16 g + 4 b + e of the chunk, i.e. pieces 2 g and
        // 2 g + 1 of staged row 16 n + l16; hardware round-to-nearest-even (v_cvt_pk_bf16_f32)
#pragma unroll
        for (int n = 0; n < 2; ++n) {
            bf16x8 o0, o1;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                o0[e] = static_cast<__bf16>(acc[n][0][e]);
                o0[4 + e] = static_cast<__bf16>(acc[n][1][e]);
                o1[e] = static_cast<__bf16>(acc[n][2][e]);
                o1[4 + e] = static_cast<__bf16>(acc[n][3][e]);
            }
            const int r = 16 * n + l16;
            *reinterpret_cast<bf16x8*>(ost + r * 128 + (((2 * g) ^ (r & 7)) * 16)) = o0;
            *reinterpret_cast<bf16x8*>(ost + r * 128 + (((2 * g + 1) ^ (r & 7)) * 16)) = o1;
        }
        // the wave's staging writes are done before its lanes read each other's pieces (the
        // staging is the wave's own: no other wave touches it)
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
        __builtin_amdgcn_wave_barrier();
        // row 8 q + lane / 8 has (row % 8) = lane / 8 for every q
        const int rpos = ((lane & 7) ^ (lane >> 3)) * 16 + (lane >> 3) * 128;
        p0 = *reinterpret_cast<const uint4*>(ost + rpos);
        p1 = *reinterpret_cast<const uint4*>(ost + rpos + 8 * 128);
        p2 = *reinterpret_cast<const uint4*>(ost + rpos + 16 * 128);
        p3 = *reinterpret_cast<const uint4*>(ost + rpos + 24 * 128);
        // the reads are done before the next chunk's staging writes
        __builtin_amdgcn_s_waitcnt(0xC07F);
        __builtin_amdgcn_wave_barrier();
    }
    if (c0 < c1) store_pending(c1 - 1);
}

// ------------------------------------------------------------------ decoder, W = V_hat Z^T (bf16)
//
// Wt[s][j][i] = sum_c V_hat[j][c] * bf16(Z[s][i][c]), rounded to bfloat16: the first product of
// the decoder with the rounding of Z folded into the staging (one launch instead of a rounding
// pass and a GEMM). A workgroup owns 64 rows j of V_hat and 64 rows i of Z: it loads both
// blocks whole with coalesced 16-byte loads (all of a thread's loads in flight at once), Z
// rounded to bf16 on the way into LDS, and each of its four waves computes one 32 x 32 block
// on v_mfma_f32_32x32x16_bf16 over K = r_w <= 256, Z as the A operand (lane l: row l % 32,
// k-run 8 (l / 32) of each 16-wide step) and V_hat as the B operand, so that a lane's results
// are four runs of four consecutive i of one row j: 8-byte stores.
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
constexpr int kVztT = 64;                // rows j and rows i per workgroup
constexpr int kVztPitch = 256 * 2 + 16;  // LDS bytes per staged row (r_w <= 256, 16 bytes of skew)

__global__ __launch_bounds__(256) void vzt_kernel(const float* __restrict__ z, const bf16_t* __restrict__ v_hat,
                                                  int w, int rh, int rw, bf16_t* __restrict__ wt) {
    __shared__ __attribute__((aligned(16))) char zs[kVztT * kVztPitch];
    __shared__ __attribute__((aligned(16))) char vs[kVztT * kVztPitch];
    const int j0 = blockIdx.x * kVztT, i0 = blockIdx.y * kVztT, s = blockIdx.z;
    const int pitch = rw * 2 + 16;
    // Z: 64 rows of r_w / 4 four-float chunks, thread t loading chunk t % 64 of rows t / 64 + 4 q;
    // V_hat: 64 rows of r_w / 8 eight-bf16 chunks, chunk t % 32 of rows t / 32 + 8 q
    // (no integer division in the address arithmetic; lanes past r_w idle)
    constexpr int ZQ = kVztT / 4, VQ = kVztT / 8;
    const int zc = threadIdx.x & 63, zr0 = threadIdx.x >> 6;
    const int vc = threadIdx.x & 31, vr0 = threadIdx.x >> 5;
    const bool zon = zc < rw / 4, von = vc < rw / 8;
    f32x4 zr[ZQ];
    uint4 vr[VQ];
#pragma unroll
    for (int q = 0; q < ZQ; ++q) {
        const int i = std::min(i0 + zr0 + 4 * q, rh - 1);  // rows past r_h repeat the last (not stored)
        if (zon) zr[q] = *reinterpret_cast<const f32x4*>(z + (static_cast<int64_t>(s) * rh + i) * rw + 4 * zc);
    }
#pragma unroll
    for (int q = 0; q < VQ; ++q)
        if (von) vr[q] = ldg16(v_hat + static_cast<int64_t>(j0 + vr0 + 8 * q) * rw + 8 * vc);
    if (zon) {
#pragma unroll
        for (int q = 0; q < ZQ; ++q) {
            bf16x4 o;  // hardware round-to-nearest-even (v_cvt_pk_bf16_f32)
#pragma unroll
            for (int e = 0; e < 4; ++e) o[e] = static_cast<__bf16>(zr[q][e]);
            *reinterpret_cast<bf16x4*>(zs + (zr0 + 4 * q) * pitch + 8 * zc) = o;
        }
    }
    if (von) {
#pragma unroll
        for (int q = 0; q < VQ; ++q) *reinterpret_cast<uint4*>(vs + (vr0 + 8 * q) * pitch + 16 * vc) = vr[q];
    }
    __syncthreads();
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int l32 = lane & 31, lh = lane >> 5;
    const int wi = wave >> 1, wj = wave & 1;
    const char* arow = zs + (32 * wi + l32) * pitch + 16 * lh;
    const char* brow = vs + (32 * wj + l32) * pitch + 16 * lh;
    f32x16 acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
    // all fragments read before the products (16 k-steps at most)
    const int nk = rw / 16;
    uint4 fa[16], fb[16];
#pragma unroll
    for (int k = 0; k < 16; ++k)
        if (k < nk) {
            fa[k] = *reinterpret_cast<const uint4*>(arow + 32 * k);
            fb[k] = *reinterpret_cast<const uint4*>(brow + 32 * k);
        }
#pragma unroll
    for (int k = 0; k < 16; ++k)
        if (k < nk)
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, fa[k]), __builtin_bit_cast(bf16x8, fb[k]),
                                                         acc, 0, 0, 0);
    // lane: row j of Wt, columns i0 + 32 wi + 8 q + 4 lh + e of acc[4 q + e]
    const int j = j0 + 32 * wj + l32;
    bf16_t* out = wt + (static_cast<int64_t>(s) * w + j) * rh;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int i = i0 + 32 * wi + 8 * q + 4 * lh;
        if (i < rh) {  // r_h is a multiple of 4: the run of four is whole
            bf16x4 o;
#pragma unroll
            for (int e = 0; e < 4; ++e) o[e] = static_cast<__bf16>(acc[4 * q + e]);
            *reinterpret_cast<bf16x4*>(out + i) = o;
        }
    }
}

// dst[i] = round-to-nearest-even bfloat16 of src[i], four elements per thread (n a multiple of 4)
__global__ __launch_bounds__(256) void f32_to_bf16_kernel(const float* __restrict__ src, int64_t n,
                                                          bf16_t* __restrict__ dst) {
    for (int64_t i = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * 4; i < n;
         i += static_cast<int64_t>(gridDim.x) * 256 * 4) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(src + i);
        uint2 o;
        o.x = static_cast<uint32_t>(f32_to_bf16(v[0])) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16);
        o.y = static_cast<uint32_t>(f32_to_bf16(v[2])) | (static_cast<uint32_t>(f32_to_bf16(v[3])) << 16);
        *reinterpret_cast<uint2*>(dst + i) = o;
    }
}

// Decoder set-up for n slices at once: Z rounded to bfloat16 (when zb is given), and the
// segment offsets and row maps of the two grouped products (slice s owns rows s*w .. of
// V_hat Z^T, gathered from row p - s*w of V_hat, and rows s*h .. of X_hat, from row p - s*h
// of U_hat).
__global__ __launch_bounds__(256) void codec_prep_kernel(const float* __restrict__ z, int64_t nz,
                                                         bf16_t* __restrict__ zb, int n, int w, int h,
                                                         int32_t* __restrict__ seg_w, int32_t* __restrict__ rows_w,
                                                         int32_t* __restrict__ seg_h, int32_t* __restrict__ rows_h) {
    const int64_t tid = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * 256;
    if (zb)
        for (int64_t i = tid * 4; i < nz; i += stride * 4) {
            const f32x4 v = *reinterpret_cast<const f32x4*>(z + i);
            uint2 o;
            o.x = static_cast<uint32_t>(f32_to_bf16(v[0])) | (static_cast<uint32_t>(f32_to_bf16(v[1])) << 16);
            o.y = static_cast<uint32_t>(f32_to_bf16(v[2])) | (static_cast<uint32_t>(f32_to_bf16(v[3])) << 16);
            *reinterpret_cast<uint2*>(zb + i) = o;
        }
    for (int64_t i = tid; i < static_cast<int64_t>(n) * w; i += stride) rows_w[i] = static_cast<int32_t>(i % w);
    for (int64_t i = tid; i < static_cast<int64_t>(n) * h; i += stride) rows_h[i] = static_cast<int32_t>(i % h);
    for (int64_t i = tid; i <= n; i += stride) {
        seg_w[i] = static_cast<int32_t>(i * w);
        seg_h[i] = static_cast<int32_t>(i * h);
    }
}

template <typename TO>
__device__ __forceinline__ void put4(TO* dst, f32x4 v) {
#pragma unroll
    for (int i = 0; i < 4; ++i) dst[i] = Elem<TO>::from_f32(v[i]);
}

// out[i] = sum over p of part[p][i] (deterministic): four groups of threads each add a quarter
// of the partials in order with up to 16 loads in flight, and the group sums are added in
// group order. A workgroup owns 64 runs of four consecutive elements (mn a multiple of 4);
// blockIdx.y is the slice (its partials and outputs follow the previous slice's).
template <typename TO>
__global__ __launch_bounds__(256) void split_reduce_kernel(const float* __restrict__ part, int64_t mn, int splits,
                                                           TO* __restrict__ out) {
    __shared__ f32x4 grp[4][64];
    part += static_cast<int64_t>(blockIdx.y) * splits * mn;
    out += static_cast<int64_t>(blockIdx.y) * mn;
    const int col = threadIdx.x & 63, g = threadIdx.x >> 6;
    const int per = (splits + 3) / 4;
    const int p0 = g * per, p1 = min(splits, p0 + per);
    for (int64_t base = static_cast<int64_t>(blockIdx.x) * 256; base < mn; base += static_cast<int64_t>(gridDim.x) * 256) {
        const int64_t i = base + col * 4;
        f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f};
        if (i < mn) {
            for (int q = p0; q < p1; q += 16) {
                f32x4 v[16];
#pragma unroll
                for (int j = 0; j < 16; ++j)
                    if (q + j < p1) v[j] = *reinterpret_cast<const f32x4*>(part + (q + j) * mn + i);
#pragma unroll
                for (int j = 0; j < 16; ++j)
                    if (q + j < p1) s += v[j];
            }
        }
        grp[g][col] = s;
        __syncthreads();
        if (g == 0 && i < mn) put4<TO>(out + i, ((grp[0][col] + grp[1][col]) + grp[2][col]) + grp[3][col]);
        __syncthreads();
    }
}

}  // namespace

hipError_t launch_transpose(DType dt, const void* src, int rows, int cols, void* dst, hipStream_t s) {
    dim3 grid((cols + 63) / 64, (rows + 63) / 64);
    ProfileScope prof("transpose", s);
    if (dt == DType::BF16)
        hipLaunchKernelGGL(transpose_kernel<bf16_t>, grid, dim3(256), 0, s, static_cast<const bf16_t*>(src), rows,
                           cols, static_cast<bf16_t*>(dst));
    else
        hipLaunchKernelGGL(transpose_kernel<float>, grid, dim3(256), 0, s, static_cast<const float*>(src), rows,
                           cols, static_cast<float*>(dst));
    return hipGetLastError();
}

hipError_t launch_utp(DType udt, const UtpArgs& g, hipStream_t s) {
    const int chunks = (g.T + g.tc - 1) / g.tc;
    dim3 grid((g.rw + kUtpC - 1) / kUtpC, chunks, g.slices);
    static_assert(kUtpC == kU3C, "both contractions tile P by the same column blocks");
    {
        ProfileScope prof("codec_utp", s);
        if (udt == DType::BF16) hipLaunchKernelGGL(utp3_kernel, grid, dim3(256), 0, s, g);
        else hipLaunchKernelGGL(utp_kernel<float>, grid, dim3(256), 0, s, g);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t mn = static_cast<int64_t>(g.rh) * g.rw;
    const int rgrid = static_cast<int>(std::min<int64_t>((mn + 255) / 256, 4096));
    ProfileScope prof("codec_utp_reduce", s);
    hipLaunchKernelGGL(split_reduce_kernel<float>, dim3(rgrid, g.slices), dim3(256), 0, s, g.part, mn, chunks, g.z);
    return hipGetLastError();
}

bool encode_fused_ok(DType dt, int h, int w, int rh, int rw) {
    return dt == DType::BF16 && h > 0 && h % kEncT == 0 && rw % kEncC == 0 && w % kEncK == 0 && rh <= 256;
}

hipError_t launch_encode_fused(const EncArgs& a, float* z, hipStream_t s) {
    const int tt_n = a.h / kEncT;
    {
        ProfileScope prof("codec_encode", s);
        hipLaunchKernelGGL(encode_fused_kernel, dim3((a.rw / kEncC) * tt_n * a.slices), dim3(512), 0, s, a);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t mn = static_cast<int64_t>(a.rh) * a.rw;
    const int rgrid = static_cast<int>(std::min<int64_t>((mn + 255) / 256, 4096));
    ProfileScope prof("codec_utp_reduce", s);
    hipLaunchKernelGGL(split_reduce_kernel<float>, dim3(rgrid, a.slices), dim3(256), 0, s, a.part, mn, tt_n, z);
    return hipGetLastError();
}

bool codec_small_ok(int h, int w, int rh, int rw) {
    return h > 0 && h <= kSmallT && rh <= kSmallT && rw <= 256 && rw % kSmallPC == 0 && w % kSmallK == 0 &&
           w % kSmallJ == 0;
}

size_t codec_small_part_floats(int h, int w, int rw, int slices) {
    return static_cast<size_t>(slices) * (w / kSmallK) * h * rw;
}

hipError_t launch_encode_small(DType dt, const void* x, const void* u, const void* v, int h, int w, int rh, int rw,
                               int slices, float* part, float* z, hipStream_t s) {
    const int nkc = w / kSmallK;
    {
        ProfileScope prof("codec_encode_part", s);
        const dim3 grid(nkc, rw / kSmallPC, slices);
        if (dt == DType::BF16)
            hipLaunchKernelGGL(enc_small_partial_kernel<bf16_t>, grid, dim3(256), 0, s,
                               static_cast<const bf16_t*>(x), static_cast<const bf16_t*>(v), h, w, rw, part);
        else
            hipLaunchKernelGGL(enc_small_partial_kernel<float>, grid, dim3(256), 0, s,
                               static_cast<const float*>(x), static_cast<const float*>(v), h, w, rw, part);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    ProfileScope prof("codec_encode_finish", s);
    if (dt == DType::BF16)
        hipLaunchKernelGGL(enc_small_finish_kernel<bf16_t>, dim3(rw / kSmallZC, slices), dim3(256), 0, s, part,
                           static_cast<const bf16_t*>(u), h, rh, rw, nkc, z);
    else
        hipLaunchKernelGGL(enc_small_finish_kernel<float>, dim3(rw / kSmallZC, slices), dim3(256), 0, s, part,
                           static_cast<const float*>(u), h, rh, rw, nkc, z);
    return hipGetLastError();
}

hipError_t launch_decode_small(DType dt, const float* z, const void* u_hat, const void* v_hat, int h, int w, int rh,
                               int rw, int slices, void* x_hat, hipStream_t s) {
    ProfileScope prof("codec_decode", s);
    if (dt == DType::BF16)
        hipLaunchKernelGGL(dec_small_kernel<bf16_t>, dim3(w / kSmallJ, slices), dim3(256), 0, s, z,
                           static_cast<const bf16_t*>(u_hat), static_cast<const bf16_t*>(v_hat), h, w, rh, rw,
                           static_cast<bf16_t*>(x_hat));
    else
        hipLaunchKernelGGL(dec_small_kernel<float>, dim3(w / kSmallJ, slices), dim3(256), 0, s, z,
                           static_cast<const float*>(u_hat), static_cast<const float*>(v_hat), h, w, rh, rw,
                           static_cast<float*>(x_hat));
    return hipGetLastError();
}

hipError_t launch_codec_prep(const float* z, int64_t nz, void* zb, int n, int w, int h, int32_t* seg_w,
                             int32_t* rows_w, int32_t* seg_h, int32_t* rows_h, hipStream_t s) {
    const int64_t work = std::max<int64_t>({nz / 4, static_cast<int64_t>(n) * std::max(w, h), n + 1});
    const int grid = static_cast<int>(std::min<int64_t>((work + 255) / 256, 4096));
    ProfileScope prof("codec_prep", s);
    hipLaunchKernelGGL(codec_prep_kernel, dim3(grid), dim3(256), 0, s, z, nz, static_cast<bf16_t*>(zb), n, w, h,
                       seg_w, rows_w, seg_h, rows_h);
    return hipGetLastError();
}

bool vzt_ok(DType dt, int w, int rh, int rw) {
    return dt == DType::BF16 && w % kVztT == 0 && rh > 0 && rh % 4 == 0 && rw > 0 && rw % 16 == 0 && rw <= 256;
}

hipError_t launch_vzt(const float* z, const void* v_hat, int w, int rh, int rw, int slices, void* wt, hipStream_t s) {
    ProfileScope prof("codec_vzt", s);
    hipLaunchKernelGGL(vzt_kernel, dim3(w / kVztT, (rh + kVztT - 1) / kVztT, slices), dim3(256), 0, s, z,
                       static_cast<const bf16_t*>(v_hat), w, rh, rw, static_cast<bf16_t*>(wt));
    return hipGetLastError();
}

bool expand_ok(DType dt, int h, int w, int rh) {
    return dt == DType::BF16 && h > 0 && h % kExT == 0 && w > 0 && w % kExC == 0 && (rh == 128 || rh == 256);
}

hipError_t launch_expand(const void* u_hat, const void* wt, int h, int w, int rh, void* x_hat, hipStream_t s) {
    // about two workgroups per CU: the chunk runs are as short as that allows
    const int64_t bands = h / kExT, nch = w / kExC;
    const int cpw = static_cast<int>(std::max<int64_t>(1, (bands * nch + 511) / 512));
    const int64_t grid = bands * ((nch + cpw - 1) / cpw);
    ProfileScope prof("codec_uw", s);
    if (rh == 256)
        hipLaunchKernelGGL(expand_kernel<256>, dim3(static_cast<unsigned>(grid)), dim3(256), 0, s,
                           static_cast<const bf16_t*>(u_hat), static_cast<const bf16_t*>(wt), w, cpw, static_cast<bf16_t*>(x_hat));
    else
        hipLaunchKernelGGL(expand_kernel<128>, dim3(static_cast<unsigned>(grid)), dim3(256), 0, s,
                           static_cast<const bf16_t*>(u_hat), static_cast<const bf16_t*>(wt), w, cpw, static_cast<bf16_t*>(x_hat));
    return hipGetLastError();
}

hipError_t launch_f32_to_bf16(const float* src, int64_t n, void* dst, hipStream_t s) {
    const int grid = static_cast<int>(std::min<int64_t>((n / 4 + 255) / 256, 4096));
    ProfileScope prof("codec_z_bf16", s);
    hipLaunchKernelGGL(f32_to_bf16_kernel, dim3(grid), dim3(256), 0, s, src, n, static_cast<bf16_t*>(dst));
    return hipGetLastError();
}

}  // namespace ec2moe
