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

// part[z][i][j] = sum over the rows t of chunk z of y[t][i] * y[t][j] (i, j < r) in float64,
// rows in order (both triangles add the same products in the same order, so the sum is
// exactly symmetric). One workgroup per (64x64 block, chunk of tc rows); thread (a, b) owns
// the 4x4 entries 4a.., 4b...
__global__ __launch_bounds__(256) void gram64_kernel(const float* __restrict__ y, int n, int r, int tc,
                                                     double* __restrict__ part) {
    __shared__ double ys_i[kGramT][kGramB];
    __shared__ double ys_j[kGramT][kGramB];
    const int i0 = blockIdx.x * kGramB, j0 = blockIdx.y * kGramB;
    const int a = threadIdx.x / 16, b = threadIdx.x % 16;
    const int tb = blockIdx.z * tc, te = min(n, tb + tc);
    double* g = part + static_cast<int64_t>(blockIdx.z) * r * r;
    double acc[4][4] = {};
    for (int t0 = tb; t0 < te; t0 += kGramT) {
        for (int e = threadIdx.x; e < kGramT * kGramB; e += 256) {
            const int t = e / kGramB, c = e % kGramB;
            const bool rowok = t0 + t < te;
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

// g[e] = sum over chunks z in order of part[z][e] (e < r*r)
__global__ __launch_bounds__(256) void gram_reduce_kernel(const double* __restrict__ part, int chunks, int64_t rr,
                                                          double* __restrict__ g) {
    for (int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; e < rr;
         e += static_cast<int64_t>(gridDim.x) * 256) {
        double v = part[e];
        for (int z = 1; z < chunks; ++z) v += part[z * rr + e];
        g[e] = v;
    }
}

constexpr int kPanel = 32;  // columns per panel of the blocked Cholesky factor and inverse

// Cholesky factor of g (r x r, float64, symmetric positive definite, r <= 256): g = R^T R
// with R upper triangular, overwriting g's upper triangle, then R^-1 (rinv, float64) and
// rinv_t[n][k] = R^-1[k][n] in float32 (the weight layout of the GEMM for Y R^-1). A pivot
// that is not positive sets *status to 1 and is replaced by 1, so the outputs stay finite;
// reset: *status = 0 first. One workgroup; blocked by panels of 32 columns:
//   factor: per panel, the diagonal block in LDS (column steps), the panel rows by
//   forward substitution (a thread per column), then the rank-32 update of the trailing
//   upper triangle from the panel kept in LDS;
//   inverse: the diagonal blocks' inverses in LDS, then X_ij = -X_ii (sum_k R_ik X_kj) for
//   the blocks above the diagonal, block column by block column, rows upward.
__global__ __launch_bounds__(256) void chol_inv_kernel(double* __restrict__ g, int r, float* __restrict__ rinv_t,
                                                        double* __restrict__ rinv, int32_t* __restrict__ status,
                                                        int reset) {
    __shared__ double dl[kPanel][kPanel + 1];
    __shared__ double pl[kPanel][256];  // the panel rows of R right of the diagonal block
    __shared__ double piv;
    __shared__ int bad;
    const int tid = threadIdx.x;
    auto G = [&](int i, int j) -> double& { return g[static_cast<int64_t>(i) * r + j]; };
    auto X = [&](int i, int j) -> double& { return rinv[static_cast<int64_t>(i) * r + j]; };
    if (tid == 0) bad = 0;
    for (int p0 = 0; p0 < r; p0 += kPanel) {
        const int pb = min(kPanel, r - p0), pe = p0 + pb, m = r - pe;
        for (int e = tid; e < pb * pb; e += blockDim.x) dl[e / pb][e % pb] = G(p0 + e / pb, p0 + e % pb);
        __syncthreads();
        for (int k = 0; k < pb; ++k) {
            if (tid == 0) {
                double d = dl[k][k];
                if (!(d > 0.0)) {
                    bad = 1;
                    d = 1.0;
                }
                piv = sqrt(d);
                dl[k][k] = piv;
            }
            __syncthreads();
            for (int j = k + 1 + tid; j < pb; j += blockDim.x) dl[k][j] /= piv;
            __syncthreads();
            for (int e = tid; e < pb * pb; e += blockDim.x) {
                const int i = e / pb, j = e % pb;
                if (i > k && j >= i) dl[i][j] -= dl[k][i] * dl[k][j];
            }
            __syncthreads();
        }
        for (int e = tid; e < pb * pb; e += blockDim.x) {
            const int i = e / pb, j = e % pb;
            if (j >= i) G(p0 + i, p0 + j) = dl[i][j];
        }
        // panel rows: R_d^T x = g[p0:pe][j] for each column j right of the block
        for (int c = tid; c < m; c += blockDim.x) {
            const int j = pe + c;
            double x[kPanel];
#pragma unroll
            for (int i = 0; i < kPanel; ++i) {
                if (i < pb) {
                    double v = G(p0 + i, j);
#pragma unroll
                    for (int l = 0; l < i; ++l) v -= dl[l][i] * x[l];
                    x[i] = v / dl[i][i];
                    G(p0 + i, j) = x[i];
                    pl[i][c] = x[i];
                }
            }
        }
        __syncthreads();
        // trailing update of the upper triangle: g[i][j] -= sum_l R[l][i] R[l][j], pe <= i <= j
        for (int64_t e = tid; e < static_cast<int64_t>(m) * m; e += blockDim.x) {
            const int i = static_cast<int>(e / m), j = static_cast<int>(e % m);
            if (j < i) continue;
            double v = G(pe + i, pe + j);
            for (int l = 0; l < pb; ++l) v -= pl[l][i] * pl[l][j];
            G(pe + i, pe + j) = v;
        }
        __syncthreads();
    }
    // R^-1: zero below the diagonal, then the diagonal blocks (back substitution in LDS)
    for (int64_t e = tid; e < static_cast<int64_t>(r) * r; e += blockDim.x) {
        const int i = static_cast<int>(e / r), j = static_cast<int>(e % r);
        if (i > j) X(i, j) = 0.0;
    }
    for (int p0 = 0; p0 < r; p0 += kPanel) {
        const int pb = min(kPanel, r - p0);
        __syncthreads();
        for (int e = tid; e < pb * pb; e += blockDim.x) dl[e / pb][e % pb] = G(p0 + e / pb, p0 + e % pb);
        __syncthreads();
        for (int c = tid; c < pb; c += blockDim.x) {  // column c of the block's inverse
            double x[kPanel];
#pragma unroll
            for (int i = kPanel - 1; i >= 0; --i) {
                if (i < pb) {
                    double v = i == c ? 1.0 : 0.0;
#pragma unroll
                    for (int l = i + 1; l < kPanel; ++l)
                        if (l <= c) v -= dl[i][l] * x[l];
                    x[i] = i <= c ? v / dl[i][i] : 0.0;
                    X(p0 + i, p0 + c) = x[i];
                }
            }
        }
    }
    __syncthreads();
    // off-diagonal blocks: X_ij = -X_ii * sum_{k = i+1 .. j} R_ik X_kj; the blocks of R and X
    // of each term staged in LDS, every thread accumulating 4 entries of the 32x32 block
    constexpr int EPT = kPanel * kPanel / 256;  // entries per thread (blockDim 256)
    const int nb = (r + kPanel - 1) / kPanel;
    for (int bj = 1; bj < nb; ++bj) {
        const int j0 = bj * kPanel, jb = min(kPanel, r - j0);
        for (int bi = bj - 1; bi >= 0; --bi) {
            const int i0 = bi * kPanel;  // full panel (only the last block can be short)
            double acc[EPT] = {};
            for (int kb = bi + 1; kb <= bj; ++kb) {
                const int k0 = kb * kPanel, kw = min(kPanel, r - k0);
                __syncthreads();
                for (int e = tid; e < kPanel * kPanel; e += blockDim.x) {
                    const int a = e / kPanel, l = e % kPanel;
                    dl[a][l] = l < kw ? G(i0 + a, k0 + l) : 0.0;           // R_{i, kb}
                    pl[a][l] = a < kw && l < jb ? X(k0 + a, j0 + l) : 0.0;  // X_{kb, j} (row a, column l)
                }
                __syncthreads();
#pragma unroll
                for (int q = 0; q < EPT; ++q) {
                    const int e = tid + q * 256, a = e / kPanel, b = e % kPanel;
                    double v = acc[q];
                    for (int l = 0; l < kPanel; ++l) v += dl[a][l] * pl[l][b];
                    acc[q] = v;
                }
            }
            __syncthreads();
            for (int e = tid; e < kPanel * kPanel; e += blockDim.x) {
                const int a = e / kPanel, l = e % kPanel;
                dl[a][l] = X(i0 + a, i0 + l);  // X_{i, i}
            }
#pragma unroll
            for (int q = 0; q < EPT; ++q) {
                const int e = tid + q * 256;
                pl[e / kPanel][e % kPanel] = acc[q];  // the sum S, row a, column b
            }
            __syncthreads();
#pragma unroll
            for (int q = 0; q < EPT; ++q) {
                const int e = tid + q * 256, a = e / kPanel, b = e % kPanel;
                if (b < jb) {
                    double v = 0.0;
                    for (int l = a; l < kPanel; ++l) v -= dl[a][l] * pl[l][b];
                    X(i0 + a, j0 + b) = v;
                }
            }
        }
    }
    __syncthreads();
    for (int64_t e = tid; e < static_cast<int64_t>(r) * r; e += blockDim.x) {
        const int n = static_cast<int>(e / r), k = static_cast<int>(e % r);
        rinv_t[e] = static_cast<float>(X(k, n));
    }
    if (tid == 0 && status) {
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

int gram64_chunks(int n, int r) {
    const int blocks = ((r + kGramB - 1) / kGramB) * ((r + kGramB - 1) / kGramB);
    const int want = std::max(1, 256 / blocks);  // about one workgroup per CU
    const int tc = std::max(kGramT, (n + want - 1) / want);
    return (n + tc - 1) / tc;
}

hipError_t launch_gram64(const float* y, int n, int r, double* part, double* g, hipStream_t s) {
    const int chunks = gram64_chunks(n, r);
    const int tc = (n + chunks - 1) / chunks;
    dim3 grid((r + kGramB - 1) / kGramB, (r + kGramB - 1) / kGramB, chunks);
    {
        ProfileScope prof("fit_gram", s);
        hipLaunchKernelGGL(gram64_kernel, grid, dim3(256), 0, s, y, n, r, tc, part);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t rr = static_cast<int64_t>(r) * r;
    ProfileScope prof("fit_gram_reduce", s);
    hipLaunchKernelGGL(gram_reduce_kernel, dim3(static_cast<unsigned>(std::min<int64_t>((rr + 255) / 256, 1024))),
                       dim3(256), 0, s, part, chunks, rr, g);
    return hipGetLastError();
}

hipError_t launch_chol_inv(double* g, int r, float* rinv_t, double* rinv, int32_t* status, bool reset, hipStream_t s) {
    ProfileScope prof("fit_chol", s);
    hipLaunchKernelGGL(chol_inv_kernel, dim3(1), dim3(256), 0, s, g, r, rinv_t, rinv, status, reset ? 1 : 0);
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
