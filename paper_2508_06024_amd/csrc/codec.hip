// Helpers of the low-rank codec (Encoder-Decoder based on Low-Rank Compression) for
// gfx950: a tiled transpose, and a float32-accumulating GEMM for the small products
// whose operands must stay in float32 (U^T (X V) with X V in float32, Z V_hat^T with Z
// in float32). The large products X V and U_hat W run on the matrix-core GEMM.
//
// small_gemm: C[m][n] = sum_k A(m,k) B(k,n) with arbitrary element strides, 64x64 output
// tile per workgroup, 4x4 outputs per thread, k split into `splits` parts written to a
// float32 partial buffer and summed in part order by a second kernel (deterministic).
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

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kT = 64;    // output tile (64 x 64 per workgroup, one 32 x 32 block per wave)
constexpr int kBK = 32;   // k per LDS stage
constexpr int kPitch = 97;  // LDS row pitch in floats: odd, so 32 consecutive k rows hit distinct banks

// C[m][n] = sum_k A(m,k) B(k,n) on the float32 matrix cores (v_mfma_f32_32x32x2f32).
// Operands are staged to LDS as [k][m] and [k][n] from any global layout (reads walk the
// contiguous direction); lane l then feeds row/column l % 32 at k = l / 32 of each step.
template <typename TA, typename TB>
__global__ __launch_bounds__(256) void small_gemm_kernel(SmallGemmArgs g) {
    __shared__ float As[kBK * kPitch];
    __shared__ float Bs[kBK * kPitch];
    const int m0 = blockIdx.x * kT, n0 = blockIdx.y * kT;
    const int split = blockIdx.z;
    const int kper = (g.K + g.splits - 1) / g.splits;
    const int kbeg = split * kper;
    const int kend = std::min(g.K, kbeg + kper);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave & 1, wn = wave >> 1;
    const bool a_k_fast = g.a_sk == 1;
    const bool b_k_fast = g.b_sk == 1;
    f32x16 acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
    constexpr int PER = kT * kBK / 256;  // elements of each operand per thread per stage
    for (int k0 = kbeg; k0 < kend; k0 += kBK) {
        // all loads of the stage first, then the LDS stores
        float va[PER], vb[PER];
        int ia[PER], ib[PER];
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            const int e = threadIdx.x + 256 * j;
            int mm, kk;
            if (a_k_fast) { kk = e % kBK; mm = e / kBK; } else { mm = e % kT; kk = e / kT; }
            // clamped, unconditional loads (all in flight together); out-of-range lanes select 0
            const int m = m0 + mm, k = k0 + kk;
            const float a_v = ld<TA>(g.a, min(m, g.M - 1) * g.a_sm + min(k, kend - 1) * g.a_sk);
            va[j] = (m < g.M && k < kend) ? a_v : 0.f;
            ia[j] = kk * kPitch + mm;
            int nn, kb;
            if (b_k_fast) { kb = e % kBK; nn = e / kBK; } else { nn = e % kT; kb = e / kT; }
            const int n = n0 + nn, kq = k0 + kb;
            const float b_v = ld<TB>(g.b, min(kq, kend - 1) * g.b_sk + min(n, g.N - 1) * g.b_sn);
            vb[j] = (n < g.N && kq < kend) ? b_v : 0.f;
            ib[j] = kb * kPitch + nn;
        }
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            As[ia[j]] = va[j];
            Bs[ib[j]] = vb[j];
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < kBK; kk += 2) {
            const float av = As[(kk + (lane >> 5)) * kPitch + wm * 32 + (lane & 31)];
            const float bv = Bs[(kk + (lane >> 5)) * kPitch + wn * 32 + (lane & 31)];
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, acc, 0, 0, 0);
        }
        __syncthreads();
    }
    // lane l holds C[m0 + wm*32 + 8*(r/4) + 4*(l/32) + r%4][n0 + wn*32 + l%32]
    float* part = g.part + static_cast<int64_t>(split) * g.M * g.N;
    const int n = n0 + wn * 32 + (lane & 31);
    if (n < g.N) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int m = m0 + wm * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            if (m < g.M) part[static_cast<int64_t>(m) * g.N + n] = acc[r];
        }
    }
}

template <typename TO>
__device__ __forceinline__ void put4(TO* dst, f32x4 v) {
#pragma unroll
    for (int i = 0; i < 4; ++i) dst[i] = Elem<TO>::from_f32(v[i]);
}

// out[i] = sum over p of part[p][i], in p order (deterministic); four elements per thread
// (mn a multiple of 4), the loads of up to 8 partials in flight at once.
template <typename TO>
__global__ __launch_bounds__(256) void split_reduce_kernel(const float* __restrict__ part, int64_t mn, int splits,
                                                           TO* __restrict__ out) {
    for (int64_t i = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * 4; i < mn;
         i += static_cast<int64_t>(gridDim.x) * 256 * 4) {
        f32x4 s = *reinterpret_cast<const f32x4*>(part + i);
        for (int p0 = 1; p0 < splits; p0 += 8) {
            f32x4 v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (p0 + j < splits) v[j] = *reinterpret_cast<const f32x4*>(part + (p0 + j) * mn + i);
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (p0 + j < splits) s += v[j];
        }
        put4<TO>(out + i, s);
    }
}

template <typename TA, typename TB>
hipError_t small_gemm_t(const SmallGemmArgs& g, hipStream_t s) {
    dim3 grid((g.M + kT - 1) / kT, (g.N + kT - 1) / kT, g.splits);
    {
        ProfileScope prof(g.name ? g.name : "small_gemm", s);
        hipLaunchKernelGGL((small_gemm_kernel<TA, TB>), grid, dim3(256), 0, s, g);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t mn = static_cast<int64_t>(g.M) * g.N;
    const int rgrid = static_cast<int>(std::min<int64_t>((mn / 4 + 255) / 256, 4096));
    std::string rname = std::string(g.name ? g.name : "small_gemm") + "_reduce";
    ProfileScope prof(rname.c_str(), s);
    if (g.out_dt == DType::BF16)
        hipLaunchKernelGGL(split_reduce_kernel<bf16_t>, dim3(rgrid), dim3(256), 0, s, g.part, mn, g.splits,
                           static_cast<bf16_t*>(g.out));
    else
        hipLaunchKernelGGL(split_reduce_kernel<float>, dim3(rgrid), dim3(256), 0, s, g.part, mn, g.splits,
                           static_cast<float*>(g.out));
    return hipGetLastError();
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

hipError_t launch_small_gemm(const SmallGemmArgs& g, hipStream_t s) {
    const bool ab = g.a_dt == DType::BF16, bb = g.b_dt == DType::BF16;
    if (ab && bb) return small_gemm_t<bf16_t, bf16_t>(g, s);
    if (ab) return small_gemm_t<bf16_t, float>(g, s);
    if (bb) return small_gemm_t<float, bf16_t>(g, s);
    return small_gemm_t<float, float>(g, s);
}

}  // namespace ec2moe
