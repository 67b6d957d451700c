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

template <typename T>
__global__ __launch_bounds__(256) void transpose_kernel(const T* __restrict__ src, int rows, int cols,
                                                        T* __restrict__ dst) {
    __shared__ T tile[32][33];
    const int c0 = blockIdx.x * 32, r0 = blockIdx.y * 32;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 32 x 8
    for (int i = ty; i < 32; i += 8) {
        const int r = r0 + i, c = c0 + tx;
        if (r < rows && c < cols) tile[i][tx] = src[static_cast<int64_t>(r) * cols + c];
    }
    __syncthreads();
    for (int i = ty; i < 32; i += 8) {
        const int c = c0 + i, r = r0 + tx;
        if (r < rows && c < cols) dst[static_cast<int64_t>(c) * rows + r] = tile[tx][i];
    }
}

constexpr int kT = 64;   // output tile
constexpr int kBK = 16;  // k per LDS stage

template <typename TA, typename TB>
__global__ __launch_bounds__(256) void small_gemm_kernel(SmallGemmArgs g) {
    __shared__ float As[kBK][kT + 4];
    __shared__ float Bs[kBK][kT + 4];
    const int m0 = blockIdx.x * kT, n0 = blockIdx.y * kT;
    const int split = blockIdx.z;
    const int kper = (g.K + g.splits - 1) / g.splits;
    const int kbeg = split * kper;
    const int kend = std::min(g.K, kbeg + kper);
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    float acc[4][4] = {};
    const bool a_k_fast = g.a_sk == 1;
    const bool b_k_fast = g.b_sk == 1;
    for (int k0 = kbeg; k0 < kend; k0 += kBK) {
        for (int i = threadIdx.x; i < kT * kBK; i += 256) {
            // A tile [kBK][kT]: walk memory-contiguous direction fastest
            int mm, kk;
            if (a_k_fast) { mm = i / kBK; kk = i % kBK; } else { kk = i / kT; mm = i % kT; }
            const int m = m0 + mm, k = k0 + kk;
            As[kk][mm] = (m < g.M && k < kend) ? ld<TA>(g.a, m * g.a_sm + k * g.a_sk) : 0.f;
            int nn, kb;
            if (b_k_fast) { nn = i / kBK; kb = i % kBK; } else { kb = i / kT; nn = i % kT; }
            const int n = n0 + nn, kq = k0 + kb;
            Bs[kb][nn] = (n < g.N && kq < kend) ? ld<TB>(g.b, kq * g.b_sk + n * g.b_sn) : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < kBK; ++kk) {
            float av[4], bv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) av[i] = As[kk][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) bv[j] = Bs[kk][tx * 4 + j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
        }
        __syncthreads();
    }
    float* part = g.part + static_cast<int64_t>(split) * g.M * g.N;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int m = m0 + ty * 4 + i;
        if (m >= g.M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int n = n0 + tx * 4 + j;
            if (n < g.N) part[static_cast<int64_t>(m) * g.N + n] = acc[i][j];
        }
    }
}

template <typename TO>
__global__ __launch_bounds__(256) void split_reduce_kernel(const float* __restrict__ part, int64_t mn, int splits,
                                                           TO* __restrict__ out) {
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < mn;
         i += static_cast<int64_t>(gridDim.x) * 256) {
        float s = part[i];
        for (int p = 1; p < splits; ++p) s += part[p * mn + i];
        out[i] = Elem<TO>::from_f32(s);
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
    const int rgrid = static_cast<int>(std::min<int64_t>((mn + 255) / 256, 4096));
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
    dim3 grid((cols + 31) / 32, (rows + 31) / 32);
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
