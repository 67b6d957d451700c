// Device-side helpers shared by the gfx950 kernels: element types, bfloat16 rounding,
// 16-byte vectors and the matrix-core step used by every contraction.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ec2moe {

// bfloat16 is carried as its 16-bit pattern; arithmetic is done in float32.
struct bf16_t {
    uint16_t bits;
};

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Round to nearest even; NaN stays NaN (quiet).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return static_cast<uint16_t>(u >> 16);
}

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));  // accumulators of a 32x32 matrix-core block

// Element traits: how many elements fill one 16-byte chunk and how a chunk of the
// token operand and a chunk of the weight operand feed the 16x16 matrix core.
template <typename T>
struct Elem;

template <>
struct Elem<bf16_t> {
    static constexpr int kPerChunk = 8;
    __device__ static float to_f32(bf16_t v) { return bf16_to_f32(v.bits); }
    __device__ static bf16_t from_f32(float f) { return bf16_t{f32_to_bf16(f)}; }
};

template <>
struct Elem<float> {
    static constexpr int kPerChunk = 4;
    __device__ static float to_f32(float v) { return v; }
    __device__ static float from_f32(float f) { return f; }
};

// One 16x16 output block, contraction over one "k-slice": the four lane groups of the
// wave (lanes 16g..16g+15) each bring one 16-byte chunk of their row. Both operands use
// the same (lane group, element) -> k assignment, so the sum covers the slice exactly once.
//   a: chunk of the row this lane feeds as matrix A (output rows  = lane % 16 after MFMA)
//   b: chunk of the row this lane feeds as matrix B (output cols  = lane % 16)
// Output: lane l holds D[4*(l/16) + i][l % 16], i = 0..3.
template <typename T>
struct Mfma;

template <>
struct Mfma<bf16_t> {
    __device__ static __forceinline__ f32x4 step(uint4 a, uint4 b, f32x4 c) {
        bf16x8 av = __builtin_bit_cast(bf16x8, a);
        bf16x8 bv = __builtin_bit_cast(bf16x8, b);
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, c, 0, 0, 0);
    }
};

template <>
struct Mfma<float> {
    // four 16x16x4 steps: element i of every lane's chunk forms the i-th step
    __device__ static __forceinline__ f32x4 step(uint4 a, uint4 b, f32x4 c) {
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
        return c;
    }
};

__device__ __forceinline__ uint4 ldg16(const void* p) {
    return *reinterpret_cast<const uint4*>(p);
}

__device__ __forceinline__ void stg16(void* p, uint4 v) {
    *reinterpret_cast<uint4*>(p) = v;
}

// 16-byte load and store with the non-temporal (streaming) cache policy: for data read or
// written once, so that it does not displace lines that are reused.
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ldg16_nt(const void* p) {
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
    return make_uint4(v[0], v[1], v[2], v[3]);
}

__device__ __forceinline__ void stg16_nt(void* p, uint4 v) {
    const u32x4_t w = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(w, reinterpret_cast<u32x4_t*>(p));
}

}  // namespace ec2moe
