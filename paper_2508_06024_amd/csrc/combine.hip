// Weighted combine of the expert outputs, Eq. 1, for gfx950:
//   y[t] = sum_{j<k} w[t][j] * y_perm[inv_perm[t*k + j]]
// One workgroup per token; each thread owns 16-byte chunks of the row, accumulates the k
// slots in float32 in slot order and rounds once. Memory-bound: reads k rows, writes one.
#include "device_common.h"
#include "internal.h"

namespace ec2moe {
namespace {

constexpr int kMaxK = 16;

template <typename T>
__global__ __launch_bounds__(256) void combine_kernel(const T* __restrict__ y_perm,
                                                      const int32_t* __restrict__ inv_perm,
                                                      const float* __restrict__ w, int top_k, int d,
                                                      T* __restrict__ y) {
    constexpr int EPC = Elem<T>::kPerChunk;
    const int t = blockIdx.x;
    int pos[kMaxK];
    float wt[kMaxK];
#pragma unroll
    for (int j = 0; j < kMaxK; ++j) {
        pos[j] = -1;
        wt[j] = 0.f;
        if (j < top_k) {
            pos[j] = inv_perm[static_cast<int64_t>(t) * top_k + j];
            wt[j] = w[static_cast<int64_t>(t) * top_k + j];
        }
    }
    const int chunks = d / EPC;
    for (int c = threadIdx.x; c < chunks; c += 256) {
        float acc[EPC];
#pragma unroll
        for (int i = 0; i < EPC; ++i) acc[i] = 0.f;
#pragma unroll
        for (int j = 0; j < kMaxK; ++j) {
            if (j < top_k && pos[j] >= 0) {
                const uint4 v = ldg16(y_perm + static_cast<int64_t>(pos[j]) * d + c * EPC);
                const T* ve = reinterpret_cast<const T*>(&v);
#pragma unroll
                for (int i = 0; i < EPC; ++i) acc[i] += wt[j] * Elem<T>::to_f32(ve[i]);
            }
        }
        uint4 o;
        T* oe = reinterpret_cast<T*>(&o);
#pragma unroll
        for (int i = 0; i < EPC; ++i) oe[i] = Elem<T>::from_f32(acc[i]);
        stg16(y + static_cast<int64_t>(t) * d + c * EPC, o);
    }
}

}  // namespace

hipError_t launch_combine(DType dt, const void* y_perm, const int32_t* inv_perm, const float* w, int n_tokens,
                          int top_k, int d, void* y, hipStream_t s) {
    if (n_tokens == 0) return hipSuccess;
    ProfileScope prof("combine", s);
    if (dt == DType::BF16)
        hipLaunchKernelGGL(combine_kernel<bf16_t>, dim3(n_tokens), dim3(256), 0, s,
                           static_cast<const bf16_t*>(y_perm), inv_perm, w, top_k, d, static_cast<bf16_t*>(y));
    else
        hipLaunchKernelGGL(combine_kernel<float>, dim3(n_tokens), dim3(256), 0, s,
                           static_cast<const float*>(y_perm), inv_perm, w, top_k, d, static_cast<float*>(y));
    return hipGetLastError();
}

}  // namespace ec2moe
