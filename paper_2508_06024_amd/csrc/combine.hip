// Weighted combine of the expert outputs, Eq. 1, for gfx950:
//   y[t] = sum_{j<k} w[t][j] * y_perm[inv_perm[t*k + j]]
// One wave per token; each lane owns 16-byte chunks of the row, accumulates the k slots in
// float32 in slot order and rounds once. Memory-bound: reads k rows, writes one. Few
// tokens (decode-sized batches) also split the row over blockIdx.y, so that enough waves
// have loads in flight.
#include "device_common.h"
#include "internal.h"

namespace ec2moe {
namespace {

constexpr int kMaxK = 16;
constexpr int kTokPerBlock = 4;  // one wave per token

// B chunks of 16 bytes per lane per batch, with all B*k row loads issued before the sums;
// NT: loads and stores with the streaming cache policy
template <typename T, int KMAX, int B, bool NT>
__global__ __launch_bounds__(64 * kTokPerBlock) void combine_kernel(const T* __restrict__ y_perm, const int32_t* __restrict__ inv_perm,
                                                      const float* __restrict__ w, int n_tokens, int top_k, int d,
                                                      T* __restrict__ y) {
    constexpr int EPC = Elem<T>::kPerChunk;
    const int lane = threadIdx.x & 63;
    const int t = blockIdx.x * kTokPerBlock + (threadIdx.x >> 6);
    if (t >= n_tokens) return;
    // slot j's position and weight, loaded by lane j and broadcast
    int my_pos = -1;
    float my_w = 0.f;
    if (lane < top_k) {
        my_pos = inv_perm[static_cast<int64_t>(t) * top_k + lane];
        my_w = w[static_cast<int64_t>(t) * top_k + lane];
    }
    int pos[KMAX];
    float wt[KMAX];
#pragma unroll
    for (int j = 0; j < KMAX; ++j) {
        pos[j] = __shfl(my_pos, j);
        wt[j] = __shfl(my_w, j);
    }
    const int chunks = d / EPC;
    const int per = chunks / gridDim.y;  // chunks of this row range (gridDim.y divides chunks)
    const int cbeg = blockIdx.y * per, cend = cbeg + per;
    for (int c0 = cbeg + lane; c0 < cend; c0 += 64 * B) {
        uint4 v[B][KMAX];
#pragma unroll
        for (int b = 0; b < B; ++b)
#pragma unroll
            for (int j = 0; j < KMAX; ++j) {
                const int c = c0 + 64 * b;
                v[b][j] = (j < top_k && pos[j] >= 0 && c < cend)
                              ? (NT ? ldg16_nt(y_perm + static_cast<int64_t>(pos[j]) * d + c * EPC)
                                    : ldg16(y_perm + static_cast<int64_t>(pos[j]) * d + c * EPC))
                              : make_uint4(0, 0, 0, 0);
            }
#pragma unroll
        for (int b = 0; b < B; ++b) {
            const int c = c0 + 64 * b;
            if (c >= cend) break;
            float acc[EPC];
#pragma unroll
            for (int i = 0; i < EPC; ++i) acc[i] = 0.f;
#pragma unroll
            for (int j = 0; j < KMAX; ++j) {
                if (j < top_k && pos[j] >= 0) {
                    const T* ve = reinterpret_cast<const T*>(&v[b][j]);
#pragma unroll
                    for (int i = 0; i < EPC; ++i) acc[i] += wt[j] * Elem<T>::to_f32(ve[i]);
                }
            }
            uint4 o;
            T* oe = reinterpret_cast<T*>(&o);
#pragma unroll
            for (int i = 0; i < EPC; ++i) oe[i] = Elem<T>::from_f32(acc[i]);
            if (NT) stg16_nt(y + static_cast<int64_t>(t) * d + c * EPC, o);
            else stg16(y + static_cast<int64_t>(t) * d + c * EPC, o);
        }
    }
}

template <typename T, int KMAX, int B, bool NT>
void launch_k(const void* y_perm, const int32_t* inv_perm, const float* w, int n_tokens, int top_k, int d, void* y,
              hipStream_t s) {
    const int grid = (n_tokens + kTokPerBlock - 1) / kTokPerBlock;
    // row ranges of at least 64 chunks while the token waves number fewer than 1024
    const int chunks = d / Elem<T>::kPerChunk;
    int ysplit = 1;
    while (n_tokens * ysplit * 2 <= 1024 && chunks % (ysplit * 2) == 0 && chunks / (ysplit * 2) >= 64) ysplit *= 2;
    hipLaunchKernelGGL((combine_kernel<T, KMAX, B, NT>), dim3(grid, ysplit), dim3(64 * kTokPerBlock), 0, s,
                       static_cast<const T*>(y_perm), inv_perm, w, n_tokens, top_k, d, static_cast<T*>(y));
}

template <typename T>
void launch_t(const void* y_perm, const int32_t* inv_perm, const float* w, int n_tokens, int top_k, int d, void* y,
              hipStream_t s) {
    // four to eight row loads in flight per lane: more (longer batches) measured slower, e.g.
    // 18.7 against 15.9 us for 8 against 2 chunks per slot at k = 2, 4096 tokens of 4096.
    // From k = 5 on, the streaming cache policy: in the layer (expert outputs just written by
    // the down GEMM) 40.7 against 43.7 us at k = 6, 8192 tokens of 2048; no difference at k = 2.
    if (top_k <= 2) launch_k<T, 2, 2, false>(y_perm, inv_perm, w, n_tokens, top_k, d, y, s);
    else if (top_k <= 4) launch_k<T, 4, 1, false>(y_perm, inv_perm, w, n_tokens, top_k, d, y, s);
    else if (top_k <= 8) launch_k<T, 8, 1, true>(y_perm, inv_perm, w, n_tokens, top_k, d, y, s);
    else launch_k<T, kMaxK, 1, true>(y_perm, inv_perm, w, n_tokens, top_k, d, y, s);
}

}  // namespace

hipError_t launch_combine(DType dt, const void* y_perm, const int32_t* inv_perm, const float* w, int n_tokens,
                          int top_k, int d, void* y, hipStream_t s) {
    if (n_tokens == 0) return hipSuccess;
    ProfileScope prof("combine", s);
    if (dt == DType::BF16)
        launch_t<bf16_t>(y_perm, inv_perm, w, n_tokens, top_k, d, y, s);
    else
        launch_t<float>(y_perm, inv_perm, w, n_tokens, top_k, d, y, s);
    return hipGetLastError();
}

}  // namespace ec2moe
