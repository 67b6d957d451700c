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

// Cholesky factor and triangular inverse of one r x r float64 Gram matrix (r <= 256, a
// multiple of 16) in one workgroup of 512 threads, with the matrix held in registers:
// thread (ti, tj) = (tid / 32, tid % 32) owns the entries (16 a + ti, 32 b + tj) of the
// blocks (a, b) that meet the upper triangle (a <= 2 b + 1: 72 of the 128 blocks, 144
// registers). Each of the 2 r steps publishes one row (and column) through LDS, double
// buffered by the parity of the step, so one barrier per step suffices; every thread then
// applies the step to its entries with multipliers that are zero where the step changes
// nothing, so the update is branch-free. The steps run in four phases of 64; a phase
// leaves out, at compile time, the blocks that none of its steps can change.
//   factor (right-looking, a rank-1 update per column): with d = A[k][k],
//     A[i][j] -= A[k][i] A[k][j] / d for i, j > k, and row k becomes R[k][j] = A[k][j] / sqrt(d)
//     for j >= k (zero left of the diagonal); a pivot that is not positive sets the status
//     and is replaced by 1;
//   inverse (Gauss-Jordan elimination on R, in place; the triangle is preserved): with
//     q = 1 / R[k][k], A[i][j] -= A[i][k] q A[k][j] for i < k < j, column k above the
//     diagonal becomes -A[i][k] q, and row k becomes q A[k][j] (q on the diagonal).
// Outputs rinv_t[n][k] = R^-1[k][n] in float32 (the weight layout of the GEMM for Y R^-1).
constexpr int kCholThreads = 512;
constexpr int kCholRB = 16;  // row blocks: row 16 a + ti
constexpr int kCholCB = 8;   // column blocks: column 32 b + tj

__host__ __device__ constexpr bool chol_kept(int a, int b) { return a <= 2 * b + 1; }

// 1 / sqrt(d) and 1 / p for d, p > 0 (the pivots): the hardware estimates refined by two
// Newton steps each, to within a few units in the last place of float64
__device__ __forceinline__ double rsqrt64(double d) {
    double y = __builtin_amdgcn_rsq(d);
    const double h = 0.5 * d;
#pragma unroll
    for (int n = 0; n < 2; ++n) y = y * fma(-h * y, y, 1.5);
    return y;
}
__device__ __forceinline__ double rcp64(double p) {
    double q = __builtin_amdgcn_rcp(p);
#pragma unroll
    for (int n = 0; n < 2; ++n) q = fma(q, fma(-p, q, 1.0), q);
    return q;
}

// Reads the published values of a step: cols[b] = crow[32 b + tj] and rows[a] = rrow[16 a + ti],
// every read issued before any is used.
__device__ __forceinline__ void lds_step(const double* crow, const double* rrow, int tj, int ti,
                                         double (&cols)[kCholCB], double (&rows)[kCholRB]) {
#pragma unroll
    for (int b = 0; b < kCholCB; ++b) cols[b] = crow[32 * b + tj];
#pragma unroll
    for (int a = 0; a < kCholRB; ++a) rows[a] = rrow[16 * a + ti];
#pragma unroll
    for (int b = 0; b < kCholCB; ++b) asm volatile("" : "+v"(cols[b]));
#pragma unroll
    for (int a = 0; a < kCholRB; ++a) asm volatile("" : "+v"(rows[a]));
}

struct CholLds {
    double row[2][256];
    double col[2][256];
    int bad;
};

// Steps k in [64 P, 64 P + 64) of the factor. Row blocks a < 4 P hold finished rows and
// column blocks b < 2 P only entries left of every pivot of the phase: neither changes.
template <int P>
__device__ __forceinline__ void chol_factor_phase(double (&m)[kCholRB][kCholCB], CholLds& sh, int r, int ti, int tj,
                                                  int tid) {
    constexpr int A0 = 4 * P, B0 = 2 * P;
    const int kend = min(r, 64 * P + 64);
    for (int k = 64 * P; k < kend; ++k) {
        const int ak = k >> 4, buf = k & 1;
        if (ti == (k & 15)) {
#pragma unroll
            for (int a = A0; a < kCholRB; ++a)
                if (a == ak) {
#pragma unroll
                    for (int b = B0; b < kCholCB; ++b)
                        if (chol_kept(a, b)) sh.row[buf][32 * b + tj] = m[a][b];
                }
        }
        __syncthreads();
        double d = sh.row[buf][k];
        double v[kCholCB], ur[kCholRB];
        lds_step(sh.row[buf], sh.row[buf], tj, ti, v, ur);
        if (!(d > 0.0)) {
            d = 1.0;
            if (tid == 0) sh.bad = 1;
        }
        const double inv_s = rsqrt64(d), inv_d = inv_s * inv_s, sd = d * inv_s;
        double vm[kCholCB];
#pragma unroll
        for (int b = B0; b < kCholCB; ++b) vm[b] = 32 * b + tj > k ? v[b] : 0.0;
#pragma unroll
        for (int a = A0; a < kCholRB; ++a) {
            const double u = 16 * a + ti > k ? ur[a] * inv_d : 0.0;
#pragma unroll
            for (int b = B0; b < kCholCB; ++b)
                if (chol_kept(a, b)) m[a][b] = fma(-u, vm[b], m[a][b]);
        }
        if (ti == (k & 15)) {
#pragma unroll
            for (int a = A0; a < kCholRB; ++a)
                if (a == ak) {
#pragma unroll
                    for (int b = 0; b < kCholCB; ++b)
                        if (chol_kept(a, b)) {
                            const int j = 32 * b + tj;
                            m[a][b] = j == k ? sd : (j > k ? v[b] * inv_s : 0.0);
                        }
                }
        }
    }
}

// Steps k in [64 P, 64 P + 64) of the inverse. Row blocks a > 4 P + 3 lie below every pivot
// of the phase and column blocks b < 2 P left of it: neither changes.
template <int P>
__device__ __forceinline__ void chol_inverse_phase(double (&m)[kCholRB][kCholCB], CholLds& sh, int r, int ti, int tj) {
    constexpr int A1 = 4 * P + 4, B0 = 2 * P;
    const int kend = min(r, 64 * P + 64);
    for (int k = 64 * P; k < kend; ++k) {
        const int ak = k >> 4, bk = k >> 5, buf = k & 1;
        if (ti == (k & 15)) {
#pragma unroll
            for (int a = 0; a < A1; ++a)
                if (a == ak) {
#pragma unroll
                    for (int b = B0; b < kCholCB; ++b)
                        if (chol_kept(a, b)) sh.row[buf][32 * b + tj] = m[a][b];
                }
        }
        if (tj == (k & 31)) {
#pragma unroll
            for (int b = B0; b < kCholCB; ++b)
                if (b == bk) {
#pragma unroll
                    for (int a = 0; a < A1; ++a)
                        if (chol_kept(a, b)) sh.col[buf][16 * a + ti] = m[a][b];
                }
        }
        __syncthreads();
        const double p = sh.row[buf][k];
        double rq[kCholCB], cr[kCholRB];
        lds_step(sh.row[buf], sh.col[buf], tj, ti, rq, cr);
        const double q = rcp64(p);
        double rqm[kCholCB];
#pragma unroll
        for (int b = B0; b < kCholCB; ++b) rqm[b] = 32 * b + tj > k ? rq[b] * q : 0.0;
#pragma unroll
        for (int a = 0; a < A1; ++a) {
            const double c = 16 * a + ti < k ? cr[a] : 0.0;
#pragma unroll
            for (int b = B0; b < kCholCB; ++b)
                if (chol_kept(a, b)) m[a][b] = fma(-c, rqm[b], m[a][b]);
        }
        if (tj == (k & 31)) {
#pragma unroll
            for (int b = B0; b < kCholCB; ++b)
                if (b == bk) {
#pragma unroll
                    for (int a = 0; a < A1; ++a)
                        if (chol_kept(a, b)) m[a][b] = 16 * a + ti < k ? -cr[a] * q : m[a][b];
                }
        }
        if (ti == (k & 15)) {
#pragma unroll
            for (int a = 0; a < A1; ++a)
                if (a == ak) {
#pragma unroll
                    for (int b = B0; b < kCholCB; ++b)
                        if (chol_kept(a, b)) {
                            const int j = 32 * b + tj;
                            m[a][b] = j == k ? q : (j > k ? rq[b] * q : m[a][b]);
                        }
                }
        }
    }
}

__global__ __launch_bounds__(kCholThreads, 1) void chol_inv_kernel(const double* __restrict__ g, int r,
                                                                   float* __restrict__ rinv_t,
                                                                   int32_t* __restrict__ status, int reset) {
    __shared__ CholLds sh;
    const int tid = threadIdx.x;
    const int ti = tid >> 5, tj = tid & 31;
    double m[kCholRB][kCholCB];

    // the upper triangle of g; zeros below it and outside r (also in the published rows)
#pragma unroll
    for (int a = 0; a < kCholRB; ++a)
#pragma unroll
        for (int b = 0; b < kCholCB; ++b)
            if (chol_kept(a, b)) {
                const int i = 16 * a + ti, j = 32 * b + tj;
                m[a][b] = i <= j && i < r && j < r ? g[static_cast<int64_t>(i) * r + j] : 0.0;
            }
    for (int e = tid; e < 2 * 256; e += kCholThreads) {
        (&sh.row[0][0])[e] = 0.0;
        (&sh.col[0][0])[e] = 0.0;
    }
    if (tid == 0) sh.bad = 0;
    __syncthreads();

    chol_factor_phase<0>(m, sh, r, ti, tj, tid);
    chol_factor_phase<1>(m, sh, r, ti, tj, tid);
    chol_factor_phase<2>(m, sh, r, ti, tj, tid);
    chol_factor_phase<3>(m, sh, r, ti, tj, tid);
    chol_inverse_phase<0>(m, sh, r, ti, tj);
    chol_inverse_phase<1>(m, sh, r, ti, tj);
    chol_inverse_phase<2>(m, sh, r, ti, tj);
    chol_inverse_phase<3>(m, sh, r, ti, tj);

    // entries below the diagonal of a kept block hold leftovers of the factor's updates
#pragma unroll
    for (int a = 0; a < kCholRB; ++a)
#pragma unroll
        for (int b = 0; b < kCholCB; ++b) {
            const int i = 16 * a + ti, j = 32 * b + tj;
            if (i < r && j < r)
                rinv_t[static_cast<int64_t>(j) * r + i] = chol_kept(a, b) && i <= j ? static_cast<float>(m[a][b]) : 0.f;
        }
    __syncthreads();
    if (tid == 0 && status) {
        if (reset) *status = sh.bad;
        else if (sh.bad) *status = 1;
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

hipError_t launch_chol_inv(const double* g, int r, float* rinv_t, int32_t* status, bool reset, hipStream_t s) {
    ProfileScope prof("fit_chol", s);
    hipLaunchKernelGGL(chol_inv_kernel, dim3(1), dim3(kCholThreads), 0, s, g, r, rinv_t, status, reset ? 1 : 0);
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
