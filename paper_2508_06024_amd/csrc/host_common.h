// Host-side basics shared by every launcher: element types and the kernel timing scope.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ec2moe {

enum class DType : int32_t { F32 = 0, BF16 = 1 };

inline size_t elem_bytes(DType t) { return t == DType::F32 ? 4 : 2; }

// ---------------------------------------------------------------- kernel timing
// Brackets a launch with events when profiling is on (see ec2moe_profile_enable).
struct ProfileScope {
    ProfileScope(const char* name, hipStream_t s);
    ~ProfileScope();
    int slot;
    hipStream_t stream;
};

}  // namespace ec2moe
