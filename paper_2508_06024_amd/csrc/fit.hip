// Data-free fitting of the codec projections (Encoder-Decoder based on Low-Rank
// Compression, Eq. 8 with lambda = 0) for gfx950: the kernels that the matrix-core GEMM
// does not cover. The fit is subspace iteration on the Gram matrices of the calibration
// slices (the products run on the GEMM); every iterate is orthonormalised by CholeskyQR2
// (Yamamoto et al., 2015): G = Y^T Y, G = R^T R, Q = Y R^-1, twice. The Gram matrix and
// its Cholesky factor are float64, so the factorisation holds for condition numbers of Y
// up to about 1e7 (float32 would fail near 4e3); the second pass restores the
// orthogonality the float32 product Y R^-1 loses.
#include "device_common.h"
#include "internal.h"

#include <algorithm>

namespace ec2moe {
namespace {

constexpr int kGramB = 64;  // output block of the Gram kernel
constexpr int kGramT = 32;  // rows of Y staged per step

// g[i][j] = sum over t of y[t][i] * y[t][j] (i, j < r) in float64, rows in order (the
// matrix is exactly symmetric: both triangles add the same products in the same order).
// One workgroup per 64x64 block; thread (a, b) owns the 4x4 entries 4a.., 4b...
__global__ __launch_bounds__(256) void gram64_kernel(const float* __restrict__ y, int n, int r,
                                                     double* __restrict__ g) {
    __shared__ double ys_i[kGramT][kGramB];
    __shared__ double ys_j[kGramT][kGramB];
    const int i0 = blockIdx.x * kGramB, j0 = blockIdx.y * kGramB;
    const int a = threadIdx.x / 16, b = threadIdx.x % 16;
    double acc[4][4] = {};
    for (int t0 = 0; t0 < n; t0 += kGramT) {
        for (int e = threadIdx.x; e < kGramT * kGramB; e += 256) {
            const int t = e / kGramB, c = e % kGramB;
            const bool rowok = t0 + t < n;
            ys_i[t][c] = rowok && i0 + c < r ? static_cast<double>(y[static_cast<int64_t>(t0 + t) * r + i0 + c]) : 0.0;
            ys_j[t][c] = rowok && j0 + c < r ? static_cast<double>(y[static_cast<int64_t>(t0 + t) * r + j0 + c]) : 0.0;
        }
        __syncthreads();
        for (int t = 0; t < kGramT; ++t) {
            double vi[4], vj[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                vi[q] = ys_i[t][4 * a + q];
                vj[q] = ys_j[t][4 * b + q];
            }
#pragma unroll
            for (int p = 0; p < 4; ++p)
#pragma unroll
                for (int q = 0; q < 4; ++q) acc[p][q] = fma(vi[p], vj[q], acc[p][q]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int p = 0; p < 4; ++p)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int i = i0 + 4 * a + p, j = j0 + 4 * b + q;
            if (i < r && j < r) g[static_cast<int64_t>(i) * r + j] = acc[p][q];
        }
}

// Cholesky factor of g (r x r, float64, symmetric positive definite): g = R^T R with R
// upper triangular, overwriting g's upper triangle (right-looking, one step per column),
// then R^-1 by back substitution, one column per thread. Writes rinv_t[n][k] = R^-1[k][n]
// in float32 (the weight layout of the GEMM for Y R^-1). A pivot that is not positive
// sets *status to 1 and is replaced by 1, so the outputs stay finite; reset: *status = 0
// first. One workgroup.
__global__ __launch_bounds__(1024) void chol_inv_kernel(double* __restrict__ g, int r, float* __restrict__ rinv_t,
                                                        double* __restrict__ rinv, int32_t* __restrict__ status,
                                                        int reset) {
    __shared__ double piv;
    __shared__ int bad;
    if (threadIdx.x == 0) bad = 0;
    for (int k = 0; k < r; ++k) {
        if (threadIdx.x == 0) {
            double d = g[static_cast<int64_t>(k) * r + k];
            if (!(d > 0.0)) {
                bad = 1;
                d = 1.0;
            }
            piv = sqrt(d);
            g[static_cast<int64_t>(k) * r + k] = piv;
        }
        __syncthreads();
        for (int j = k + 1 + threadIdx.x; j < r; j += blockDim.x) g[static_cast<int64_t>(k) * r + j] /= piv;
        __syncthreads();
        // trailing update of the upper triangle: g[i][j] -= R[k][i] R[k][j], k < i <= j
        const int m = r - k - 1;
        const int64_t cnt = static_cast<int64_t>(m) * m;
        for (int64_t e = threadIdx.x; e < cnt; e += blockDim.x) {
            const int i = k + 1 + static_cast<int>(e / m), j = k + 1 + static_cast<int>(e % m);
            if (j >= i) g[static_cast<int64_t>(i) * r + j] -= g[static_cast<int64_t>(k) * r + i] * g[static_cast<int64_t>(k) * r + j];
        }
        __syncthreads();
    }
    // R^-1 column c: R x = e_c, x_i = (delta_ic - sum_{l > i} R[i][l] x_l) / R[i][i], i = c .. 0
    for (int c = threadIdx.x; c < r; c += blockDim.x) {
        for (int i = r - 1; i > c; --i) rinv[static_cast<int64_t>(i) * r + c] = 0.0;
        for (int i = c; i >= 0; --i) {
            double s = i == c ? 1.0 : 0.0;
            for (int l = i + 1; l <= c; ++l) s -= g[static_cast<int64_t>(i) * r + l] * rinv[static_cast<int64_t>(l) * r + c];
            rinv[static_cast<int64_t>(i) * r + c] = s / g[static_cast<int64_t>(i) * r + i];
        }
        for (int i = 0; i < r; ++i) rinv_t[static_cast<int64_t>(c) * r + i] = static_cast<float>(rinv[static_cast<int64_t>(i) * r + c]);
    }
    if (threadIdx.x == 0 && status) {
        if (reset) *status = bad;
        else if (bad) *status = 1;
    }
}

// xu[t][s*w + j] = x[s][t][j]: the mode-1 unfolding of c slices [c][h][w] (16-byte chunks)
template <typename T>
__global__ __launch_bounds__(256) void unfold_kernel(const T* __restrict__ x, int c, int h, int w, T* __restrict__ xu) {
    constexpr int EPC = 16 / static_cast<int>(sizeof(T));
    const int64_t chunks = static_cast<int64_t>(c) * h * (w / EPC);
    for (int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; e < chunks;
         e += static_cast<int64_t>(gridDim.x) * 256) {
        const int64_t row = e / (w / EPC);  // s * h + t
        const int j = static_cast<int>(e % (w / EPC)) * EPC;
        const int s = static_cast<int>(row / h), t = static_cast<int>(row % h);
        *reinterpret_cast<uint4*>(xu + static_cast<int64_t>(t) * c * w + static_cast<int64_t>(s) * w + j) =
            *reinterpret_cast<const uint4*>(x + row * w + j);
    }
}

}  // namespace

hipError_t launch_gram64(const float* y, int n, int r, double* g, hipStream_t s) {
    dim3 grid((r + kGramB - 1) / kGramB, (r + kGramB - 1) / kGramB);
    ProfileScope prof("fit_gram", s);
    hipLaunchKernelGGL(gram64_kernel, grid, dim3(256), 0, s, y, n, r, g);
    return hipGetLastError();
}

hipError_t launch_chol_inv(double* g, int r, float* rinv_t, double* rinv, int32_t* status, bool reset, hipStream_t s) {
    ProfileScope prof("fit_chol", s);
    hipLaunchKernelGGL(chol_inv_kernel, dim3(1), dim3(1024), 0, s, g, r, rinv_t, rinv, status, reset ? 1 : 0);
    return hipGetLastError();
}

hipError_t launch_unfold(DType dt, const void* x, int c, int h, int w, void* xu, hipStream_t s) {
    const int64_t chunks = static_cast<int64_t>(c) * h * w * static_cast<int64_t>(elem_bytes(dt)) / 16;
    const int grid = static_cast<int>(std::min<int64_t>((chunks + 255) / 256, 4096));
    ProfileScope prof("fit_unfold", s);
    if (dt == DType::BF16)
        hipLaunchKernelGGL(unfold_kernel<bf16_t>, dim3(grid), dim3(256), 0, s, static_cast<const bf16_t*>(x), c, h, w,
                           static_cast<bf16_t*>(xu));
    else
        hipLaunchKernelGGL(unfold_kernel<float>, dim3(grid), dim3(256), 0, s, static_cast<const float*>(x), c, h, w,
                           static_cast<float*>(xu));
    return hipGetLastError();
}

}  // namespace ec2moe
