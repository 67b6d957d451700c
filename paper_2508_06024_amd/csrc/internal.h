// Host-side interface between the C ABI (api.cpp) and the kernel launchers (*.hip).
// Launchers assume validated arguments; they return the HIP error of the launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "ec2moe.h"
#include "gemm.h"
#include "host_common.h"

namespace ec2moe {

// Records the detail of a failing call for ec2moe_last_error() and returns st (api.cpp).
ec2moe_status report_error(ec2moe_status st, const char* detail);

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
    float* ws;         // split-d partials of small batches, or null
    int nsplit;        // d-splits per tile (> 1 only with ws)
    int top_groups;    // > 0: keep the top_groups groups of largest p_group (more while < k candidates)
    int equal_groups;  // goff[k] = k * M / K
    int32_t goff[161]; // group k = experts goff[k] .. goff[k + 1] - 1 (K <= 160)
};
hipError_t launch_gate(DType dt, const GateArgs& a, hipStream_t s);
// d-splits per 16-token tile for a small batch (1: no split) and the workspace bytes of the
// split partials (0 when there is no split)
int gate_split_count(DType dt, int n_tokens, int d);
size_t gate_split_bytes(DType dt, int n_tokens, int d, int gate_rows);

// ---------------------------------------------------------------- permutation
// Work split of the permutation kernels: assignments are processed in chunks of
// kPermChunk; per-chunk counts live in the workspace.
constexpr int kPermChunk = 1024;
inline int perm_chunks(int64_t n_assign) { return static_cast<int>((n_assign + kPermChunk - 1) / kPermChunk); }

// The library's own per-device count array (1 MiB) for callers that pass no workspace:
// *counts receives the current device's copy (looked up once per device). Calls that
// overlap on one device share it and race.
constexpr int kPermStaticCountWords = 1 << 18;
hipError_t permute_static_counts(int32_t** counts);

hipError_t launch_permute(const int32_t* topk_idx, int64_t n_assign, int top_k, int n_experts,
                          int32_t* chunk_counts /*[chunks][M]*/, int32_t* seg_offsets,
                          int32_t* perm_src, int32_t* inv_perm, hipStream_t s);
// x_perm[r] = x[perm_src[r]] for r < *seg_end (device scalar: the last segment offset); zeros beyond
hipError_t launch_gather_rows(DType dt, const void* x, int64_t n_src, const int32_t* perm_src,
                              const int32_t* seg_end, int64_t n_rows, int d, void* x_perm, hipStream_t s);

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
// Fused encoder of bf16 layers: part[s][tt][r][c] = U^T (X V) over 64-token tiles tt (X [slices][h][w],
// V [w][r_w], U [h][r_h]), then z[s] = sum over tt in order. Applies when encode_fused_ok();
// part holds slices * (h / 64) * r_h * r_w floats.
struct EncArgs {
    const void* x;   // bf16
    const void* v;   // bf16
    const void* u;   // bf16
    float* part;
    int h, w, rh, rw, slices;
};
bool encode_fused_ok(DType dt, int h, int w, int rh, int rw);
// Small batches (h <= 64 tokens per slice, r_h <= 64): the encoder in two launches through
// part (codec_small_part_floats floats) and the decoder in one, in float32 throughout.
bool codec_small_ok(int h, int w, int rh, int rw);
size_t codec_small_part_floats(int h, int w, int rw, int slices);
hipError_t launch_encode_small(DType dt, const void* x, const void* u, const void* v, int h, int w, int rh, int rw,
                               int slices, float* part, float* z, hipStream_t s);
hipError_t launch_decode_small(DType dt, const float* z, const void* u_hat, const void* v_hat, int h, int w, int rh,
                               int rw, int slices, void* x_hat, hipStream_t s);
hipError_t launch_encode_fused(const EncArgs& a, float* z, hipStream_t s);
// Decoder set-up of n slices: zb = bfloat16(z) (nz elements, a multiple of 4; skipped when zb is
// null); seg_w[s] = s*w, rows_w[p] = p % w, seg_h[s] = s*h, rows_h[p] = p % h (s <= n).
hipError_t launch_codec_prep(const float* z, int64_t nz, void* zb, int n, int w, int h, int32_t* seg_w,
                             int32_t* rows_w, int32_t* seg_h, int32_t* rows_h, hipStream_t s);
// ---------------------------------------------------------------- codec fitting
// g = y^T y in float64 (y [n][r] float32, g [r][r]) through per-chunk partials part
// ([gram64_chunks(n, r)][r][r] float64) added in chunk order
int gram64_chunks(int n, int r);
hipError_t launch_gram64(const float* y, int n, int r, double* part, double* g, hipStream_t s);
// g = R^T R (Cholesky, float64, r <= 256 a multiple of 16; g is read only) and
// rinv_t[n][k] = (R^-1)[k][n] in float32. *status: 1 if a pivot was not positive (set to 0
// first when reset).
hipError_t launch_chol_inv(const double* g, int r, float* rinv_t, int32_t* status, bool reset, hipStream_t s);
// xu [h][c*w] = the slices [c][h][w] side by side (w a multiple of 16 bytes)
hipError_t launch_unfold(DType dt, const void* x, int c, int h, int w, void* xu, hipStream_t s);

// dst = bfloat16(src) with round-to-nearest-even, n a multiple of 4
hipError_t launch_f32_to_bf16(const float* src, int64_t n, void* dst, hipStream_t s);
// Decoder product Wt[s] = V_hat bf16(Z[s])^T [w][r_h] in one launch for bf16 layers
// (w a multiple of 64, r_h of 4, r_w of 16 and at most 256); vzt_ok tells whether the shape qualifies.
bool vzt_ok(DType dt, int w, int rh, int rw);
hipError_t launch_vzt(const float* z, const void* v_hat, int w, int rh, int rw, int slices, void* wt, hipStream_t s);
// Decoder product X_hat = U_hat Wt^T [h][w] (bf16, one slice) in one launch: U_hat [h][r_h], Wt [w][r_h],
// h a multiple of 128, w of 64, r_h 128 or 256; expand_ok tells whether the shape qualifies.
bool expand_ok(DType dt, int h, int w, int rh);
hipError_t launch_expand(const void* u_hat, const void* wt, int h, int w, int rh, void* x_hat, hipStream_t s);


}  // namespace ec2moe
