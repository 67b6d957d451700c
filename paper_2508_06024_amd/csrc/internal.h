// Host-side interface between the C ABI (api.cpp) and the kernel launchers (*.hip).
// Launchers assume validated arguments; they return the HIP error of the launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "ec2moe.h"

namespace ec2moe {

enum class DType : int32_t { F32 = 0, BF16 = 1 };

// Records the detail of a failing call for ec2moe_last_error() and returns st (api.cpp).
ec2moe_status report_error(ec2moe_status st, const char* detail);

inline size_t elem_bytes(DType t) { return t == DType::F32 ? 4 : 2; }

// ---------------------------------------------------------------- kernel timing
// Brackets a launch with events when profiling is on (see ec2moe_profile_enable).
struct ProfileScope {
    ProfileScope(const char* name, hipStream_t s);
    ~ProfileScope();
    int slot;
    hipStream_t stream;
};

// ---------------------------------------------------------------- gate
struct GateArgs {
    const void* x;
    const void* w_global;
    const float* b_global;
    const void* w_local;
    const float* b_local;
    int32_t* topk_idx;
    float* topk_w;
    float* probs;
    int n_tokens, d, n_experts, n_groups, top_k;
    bool renormalize;
    uint64_t mask[4];
    int top_groups;    // > 0: keep the top_groups groups of largest p_group (more while < k candidates)
    int equal_groups;  // goff[k] = k * M / K
    int32_t goff[161]; // group k = experts goff[k] .. goff[k + 1] - 1 (K <= 160)
};
hipError_t launch_gate(DType dt, const GateArgs& a, hipStream_t s);

// ---------------------------------------------------------------- permutation
// Work split of the permutation kernels: assignments are processed in chunks of
// kPermChunk; per-chunk counts live in the workspace.
constexpr int kPermChunk = 1024;
inline int perm_chunks(int64_t n_assign) { return static_cast<int>((n_assign + kPermChunk - 1) / kPermChunk); }

hipError_t launch_permute(const int32_t* topk_idx, int64_t n_assign, int top_k, int n_experts,
                          int32_t* chunk_counts /*[chunks][M]*/, int32_t* seg_offsets,
                          int32_t* perm_src, int32_t* inv_perm, hipStream_t s);
// x_perm[r] = x[perm_src[r]] for r < *seg_end (device scalar: the last segment offset); zeros beyond
hipError_t launch_gather_rows(DType dt, const void* x, int64_t n_src, const int32_t* perm_src,
                              const int32_t* seg_end, int64_t n_rows, int d, void* x_perm, hipStream_t s);

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

// ---------------------------------------------------------------- combine
hipError_t launch_combine(DType dt, const void* y_perm, const int32_t* inv_perm, const float* w,
                          int n_tokens, int top_k, int d, void* y, hipStream_t s);

// ---------------------------------------------------------------- codec helpers
// dst[c][r] = src[r][c] for a rows x cols matrix
hipError_t launch_transpose(DType dt, const void* src, int rows, int cols, void* dst, hipStream_t s);

// Z[s][r][c] = sum_t U[t][r] P[s][t][c] (r < rh, c < rw, t < T, s < slices): float32
// partial sums over token chunks of tc rows go to part ([slices][ceil(T / tc)][rh][rw]
// float32), then are added in chunk order into z ([slices][rh][rw]; deterministic). U has
// the layer dtype, P and Z are float32. rh <= 256; rh and rw are multiples of 16; every row
// is 16-byte aligned.
struct UtpArgs {
    const void* u;
    const float* p;
    int T, rh, rw, tc, slices;
    float* part;
    float* z;
};
hipError_t launch_utp(DType udt, const UtpArgs& g, hipStream_t s);
// Decoder set-up of n slices: zb = bfloat16(z) (nz elements, a multiple of 4; skipped when zb is
// null); seg_w[s] = s*w, rows_w[p] = p % w, seg_h[s] = s*h, rows_h[p] = p % h (s <= n).
hipError_t launch_codec_prep(const float* z, int64_t nz, void* zb, int n, int w, int h, int32_t* seg_w,
                             int32_t* rows_w, int32_t* seg_h, int32_t* rows_h, hipStream_t s);
// dst = bfloat16(src) with round-to-nearest-even, n a multiple of 4
hipError_t launch_f32_to_bf16(const float* src, int64_t n, void* dst, hipStream_t s);

}  // namespace ec2moe
