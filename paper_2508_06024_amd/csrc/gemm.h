// Interface of the grouped / dense matrix-core GEMM (gemm.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "host_common.h"

namespace ec2moe {

// ---------------------------------------------------------------- grouped / dense GEMM
// out[p][n] = sum_k tok[row(p)][k] * w_e[n][k] for every row p of group e, where
// row(p) = row_index ? row_index[p] : p and w_e = w + e * w_group_stride.
// SwiGLU mode: weight rows 0..N-1 are the gate branch and N..2N-1 the up branch; the
// output is silu(gate) * up with N columns. ReLU mode: out = max(sum, 0).
enum class Epilogue : int { Store = 0, SwiGLU = 1, ReLU = 2 };
enum class OutType : int { Same = 0, F32 = 1 };

struct GemmArgs {
    const void* tok;          // [rows][K]
    const int32_t* row_index; // gather map or null
    const void* w;            // [groups][Nw][K]
    int64_t w_group_stride;   // elements between consecutive groups' weights
    const int32_t* seg;       // [groups+1] device segment offsets, or null (dense: one group)
    int n_groups;
    int64_t rows;             // total rows (upper bound for grouped; exact for dense)
    int64_t src_rows;         // rows of the token matrix `tok` (gather targets are below this)
    int64_t w_rows;           // rows of one group's weight matrix
    int K;
    int N;                    // output columns
    void* out;                // [rows][N]
    int64_t ldo;              // output row stride (elements)
    const char* name;         // kernel name for the timing record
    // split-K tail (bf16 large-tile path): tiles beyond the last whole round of `slots`
    // resident workgroups are split along K into at most max_split chunks whose float32
    // partial tiles go to `part` and are summed in chunk order by a second kernel.
    // part == nullptr or max_split <= 1 disables the split.
    float* part;              // [slots][TM][TN] float32 scratch
    int max_split;
    int relu;                 // set by launch_gemm from the epilogue: plain stores take max(v, 0)
};
// Bytes of `part` scratch the large-tile GEMM may use (0 if it cannot split).
size_t gemm_split_scratch_bytes();
hipError_t launch_gemm(DType dt, Epilogue epi, OutType ot, const GemmArgs& a, hipStream_t s);

}  // namespace ec2moe
