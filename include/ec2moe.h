/*
 * ec2moe.h - C ABI of the MI355X (gfx950) library for the data-parallel hot path of
 * EC2MoE (arXiv 2508.06024): the group-gated Mixture-of-Experts layer forward and the
 * low-rank encoder/decoder applied to hidden states at the end-cloud pipeline cut.
 *
 * Conventions for every call
 *   - Tensor pointers are DEVICE pointers unless marked [host]. Tensors are dense and
 *     row-major, 16-byte aligned. Element type: the descriptor's dtype (float32 or
 *     bfloat16 bit patterns) unless the type says otherwise; biases, gate weights out,
 *     codec Z and probabilities are always float32; indices are int32.
 *   - The caller owns every buffer, including the workspace; the library keeps no
 *     pointer after a call returns and allocates nothing on these paths. Host arrays
 *     (descriptors, the candidate mask) are read during the call only. Outputs must
 *     not alias inputs.
 *   - Calls are stream-ordered and asynchronous on the given hipStream_t (0 = the null
 *     stream); the library never synchronises. Results are deterministic: the same
 *     inputs on the same GPU give bit-identical outputs.
 *   - All validation happens on the host before any launch. On any error nothing is
 *     launched and no output is written; ec2moe_last_error() returns the detail
 *     (thread-local). No C++ exception crosses this interface.
 *   - Supported shapes: d_model and ffn_hidden multiples of 128, 1 <= top_k <= 16,
 *     n_experts <= 256, n_experts + n_groups <= 320, n_groups <= n_experts (and
 *     dividing it for the gate without group sizes; the calls after the gate never
 *     read the group structure);
 *     codec ranks r_h, r_w multiples of 16 and at most 256, w a multiple of 128.
 *     Others return EC2MOE_ERR_UNSUPPORTED. n_tokens == 0 is valid and launches nothing.
 */
#ifndef EC2MOE_H
#define EC2MOE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { EC2MOE_F32 = 0, EC2MOE_BF16 = 1 } ec2moe_dtype;

typedef enum {
    EC2MOE_OK = 0,
    EC2MOE_ERR_INVALID_ARGUMENT = 1,   /* null pointer, bad dimension, misalignment, bad mask bits */
    EC2MOE_ERR_UNSUPPORTED = 2,        /* valid but outside the supported shapes listed above */
    EC2MOE_ERR_TOO_FEW_CANDIDATES = 3, /* fewer candidate experts than top_k */
    EC2MOE_ERR_WORKSPACE_TOO_SMALL = 4,
    EC2MOE_ERR_HIP = 5                 /* a HIP launch or runtime call failed */
} ec2moe_status;

/* flags of ec2moe_moe_desc */
#define EC2MOE_GATE_RENORMALIZE 1u /* selected gate weights are divided by their sum (Eq. 1:
                                      the gate weights of a token sum to 1); else raw g */
#define EC2MOE_EXPERT_RELU 2u      /* expert networks are two-layer ReLU feed-forward layers,
                                      E(x) = W_out relu(W_in x), as in the Switch Transformer
                                      base model of the paper's experiments (Experimental
                                      Setup); else SwiGLU. Changes the layout of w_gate_up. */

/* Shape of one MoE layer call: T tokens of width d, M experts in K contiguous equal
 * groups (group k = experts [k*M/K, (k+1)*M/K)), expert hidden width H, top-k routing. */
typedef struct {
    int32_t n_tokens;   /* T */
    int32_t d_model;    /* d */
    int32_t n_experts;  /* M */
    int32_t n_groups;   /* K */
    int32_t top_k;      /* k */
    int32_t ffn_hidden; /* H */
    ec2moe_dtype dtype; /* of x, gate weights, expert weights and y (an int-sized enum) */
    uint32_t flags;     /* OR of EC2MOE_GATE_RENORMALIZE, EC2MOE_EXPERT_RELU, or 0 */
} ec2moe_moe_desc;

/* Shape of the codec: n_slices blocks X[c] of h x w (h = tokens, w = model width),
 * projected to r_h x r_w. */
typedef struct {
    int32_t n_slices; /* c */
    int32_t h;
    int32_t w;
    int32_t r_h;
    int32_t r_w;
    ec2moe_dtype dtype; /* of x, x_hat and the projections (an int-sized enum) */
} ec2moe_codec_desc;

/*
 * Hardware-aware lightweight group gate (Local Expert Selection, Eq. 4; Lightweight
 * Group Gate Network, Eq. 5-7) followed by top-k selection.
 *   cand_mask [host] ceil(M/64) words: bit e of word e/64 set <=> expert e is in the
 *             candidate set E_local. Bits at or above M must be clear.
 *   x         [T][d]
 *   w_global  [K][d], b_global [K] float32 or NULL (zero): stage-1 group gate, Eq. 6
 *   w_local   [M][d], b_local  [M] float32 or NULL (zero): the K stacked group gates
 *             W_k (rows k*M/K .. (k+1)*M/K - 1), Eq. 5
 *   topk_idx  [T][k] int32 out: selected experts, descending fused probability
 *             g_i = p_group^(k) * p_local,i^(k) (Eq. 7); exact ties -> lower index.
 *   topk_w    [T][k] float32 out: g of the selected experts, renormalised to sum 1
 *             when EC2MOE_GATE_RENORMALIZE is set.
 *   probs     [T][M] float32 out or NULL: the full fused distribution g (0 for
 *             non-candidates).
 * Non-candidates get no probability; a group with no candidate leaves the group softmax.
 * Errors: EC2MOE_ERR_TOO_FEW_CANDIDATES if popcount(mask) < k.
 */
ec2moe_status ec2moe_group_gate(const ec2moe_moe_desc* desc, const uint64_t* cand_mask,
                                const void* x, const void* w_global, const float* b_global,
                                const void* w_local, const float* b_local,
                                int32_t* topk_idx, float* topk_w, float* probs,
                                hipStream_t stream);

/* Options of ec2moe_group_gate_ex. */
typedef struct {
    int32_t top_groups;         /* G > 0: group-focused evaluation (the closing remark of the
                                   Lightweight Group Gate Network section): per token only the
                                   groups ranked first by p_group (ties to the lower group
                                   index) keep their experts; more groups are kept in that
                                   order while the kept ones hold fewer than k candidates.
                                   p_group stays the softmax over every group with a candidate;
                                   left-out experts get g = 0. 0 (or G >= K): every group, Eq. 7. */
    const int32_t* group_sizes; /* [host] K group sizes M_k >= 1 summing to M (Eq. 5: M = sum
                                   of M_k), group k = the next M_k experts; NULL: K equal
                                   groups (K must divide M). Read during the call only. */
    void* workspace;            /* [device] or NULL: scratch of ec2moe_gate_workspace_size bytes
                                   (16-byte aligned, no initial contents) that lets a small
                                   batch split d over more workgroups; NULL runs unsplit.
                                   Calls that overlap on one workspace race. */
    size_t workspace_bytes;     /* size of workspace; an error if below the required size */
} ec2moe_gate_opts;

/* Gate workspace bytes for this descriptor (0: the batch is large enough to run unsplit,
 * and the gate ignores a workspace). */
ec2moe_status ec2moe_gate_workspace_size(const ec2moe_moe_desc* desc, size_t* bytes /*[host]*/);

/*
 * ec2moe_group_gate with options (opts may be NULL: the same as ec2moe_group_gate).
 * Unequal groups relax the rule that K divides M. The candidate set must still hold at
 * least k experts. Logits of every group are computed either way (the gate reads X once;
 * the pruning changes which experts may be selected, not the memory traffic).
 */
ec2moe_status ec2moe_group_gate_ex(const ec2moe_moe_desc* desc, const ec2moe_gate_opts* opts,
                                   const uint64_t* cand_mask, const void* x, const void* w_global,
                                   const float* b_global, const void* w_local, const float* b_local,
                                   int32_t* topk_idx, float* topk_w, float* probs, hipStream_t stream);

/* Workspace bytes needed by ec2moe_permute, ec2moe_expert_ffn and ec2moe_moe_forward
 * for this descriptor (a superset for all three). */
ec2moe_status ec2moe_moe_workspace_size(const ec2moe_moe_desc* desc, size_t* bytes /*[host]*/);

/*
 * Dispatch of tokens to experts (the routing step between the gate and the expert
 * networks of Eq. 1): assignments a = t*k + j are sorted stably by topk_idx.
 *   topk_idx    [T][k] int32 in [0, M)
 *   seg_offsets [M+1] int32 out: expert e owns positions [seg[e], seg[e+1])
 *   perm_src    [T*k] int32 out: token of each position (ascending inside a segment)
 *   inv_perm    [T*k] int32 out: position of each assignment
 *   x, x_perm   [T][d] in, [T*k][d] out: gathered rows; both NULL to skip the gather
 *   ws          workspace of ec2moe_moe_workspace_size bytes
 */
ec2moe_status ec2moe_permute(const ec2moe_moe_desc* desc, const int32_t* topk_idx,
                             const void* x, int32_t* seg_offsets, int32_t* perm_src,
                             int32_t* inv_perm, void* x_perm, void* ws, size_t ws_bytes,
                             hipStream_t stream);

/*
 * ec2moe_permute without a workspace, for callers that cannot allocate (code under HIP
 * graph capture, serving loops, harnesses that forbid allocation). The same kernels and
 * results as ec2moe_permute; the per-chunk expert counts of inputs above 8192 assignments
 * go to an array the library holds on each GPU (1 MiB, kept until the process ends, looked
 * up on the first call on that device; this call allocates nothing). Every count it reads
 * is written first in the same call, so the array needs no clearing.
 *   Limit: ceil(T*k / 1024) * n_experts <= 262144 (e.g. 1,048,576 assignments over 256
 *   experts); larger inputs return EC2MOE_ERR_UNSUPPORTED before any launch.
 *   Calls that overlap on one GPU (other streams, other threads) share the array and race:
 *   order them, or use ec2moe_permute with a workspace each.
 */
ec2moe_status ec2moe_permute_noalloc(const ec2moe_moe_desc* desc, const int32_t* topk_idx,
                                     const void* x, int32_t* seg_offsets, int32_t* perm_src,
                                     int32_t* inv_perm, void* x_perm, hipStream_t stream);

/*
 * The expert networks E_i of Eq. 1 on permuted rows:
 *   y_perm[p] = E_e(x[perm_src[p]]) for every position p of segment e.
 * Default: SwiGLU feed-forward layers, E(x) = W_down (silu(W_gate x) * (W_up x)),
 *   w_gate_up [M][2H][d] (rows 0..H-1 gate branch, H..2H-1 up branch);
 *   act [T*k][H] out or NULL: silu(gate) * up in the layer dtype.
 * With EC2MOE_EXPERT_RELU: two-layer ReLU feed-forward layers, E(x) = W_down relu(W_in x),
 *   w_gate_up [M][H][d] holding W_in; act [T*k][H] out or NULL: relu(W_in x).
 * Both: x [T][d]; seg_offsets [M+1], perm_src [T*k] as from ec2moe_permute;
 *   w_down [M][d][H]; y_perm [T*k][d] out.
 * Intermediates are accumulated in float32 and rounded once to the layer dtype.
 */
ec2moe_status ec2moe_expert_ffn(const ec2moe_moe_desc* desc, const void* x,
                                const int32_t* seg_offsets, const int32_t* perm_src,
                                const void* w_gate_up, const void* w_down, void* act,
                                void* y_perm, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Weighted combine, Eq. 1: y[t] = sum_{j<k} topk_w[t][j] * y_perm[inv_perm[t*k+j]],
 * accumulated in float32 in slot order j = 0..k-1 and rounded once.
 *   y_perm [T*k][d], inv_perm [T*k] int32, topk_w [T][k] float32, y [T][d] out.
 */
ec2moe_status ec2moe_combine(const ec2moe_moe_desc* desc, const void* y_perm,
                             const int32_t* inv_perm, const float* topk_w, void* y,
                             hipStream_t stream);

/*
 * Sparse MoE layer output, Eq. 1, for given routing: permute, expert networks,
 * combine. y[t] = sum_j topk_w[t][j] * E_{topk_idx[t][j]}(x[t]).
 *   x [T][d]; topk_idx [T][k] int32 in [0, M); topk_w [T][k] float32;
 *   w_gate_up [M][2H][d] (SwiGLU) or [M][H][d] (EC2MOE_EXPERT_RELU); w_down [M][d][H];
 *   y [T][d] out; ws of ec2moe_moe_workspace_size bytes.
 * Routing may come from ec2moe_group_gate on other hidden states (the end-cloud split:
 * route on X, run the experts on the reconstruction X_hat).
 */
ec2moe_status ec2moe_moe_forward(const ec2moe_moe_desc* desc, const void* x,
                                 const int32_t* topk_idx, const float* topk_w,
                                 const void* w_gate_up, const void* w_down, void* y,
                                 void* ws, size_t ws_bytes, hipStream_t stream);

/* Workspace bytes needed by ec2moe_lowrank_encode and ec2moe_lowrank_decode. */
ec2moe_status ec2moe_lowrank_workspace_size(const ec2moe_codec_desc* desc,
                                            size_t* bytes /*[host]*/);

/*
 * Low-rank encoder (Encoder-Decoder based on Low-Rank Compression): Z = U^T X V per slice.
 *   x [c][h][w]; u [h][r_h]; v [w][r_w]; z [c][r_h][r_w] float32 out.
 * X V is accumulated in float32 and kept in float32 for the product with U^T.
 */
ec2moe_status ec2moe_lowrank_encode(const ec2moe_codec_desc* desc, const void* x,
                                    const void* u, const void* v, float* z, void* ws,
                                    size_t ws_bytes, hipStream_t stream);

/*
 * Low-rank decoder: X_hat = U_hat Z V_hat^T per slice, with the decoder's own
 * ("inverse") projections.
 *   z [c][r_h][r_w] float32; u_hat [h][r_h]; v_hat [w][r_w]; x_hat [c][h][w] out.
 * The small product Z V_hat^T is accumulated in float32 and rounded to the layer dtype
 * before the h x w product, which accumulates in float32.
 */
ec2moe_status ec2moe_lowrank_decode(const ec2moe_codec_desc* desc, const float* z,
                                    const void* u_hat, const void* v_hat, void* x_hat,
                                    void* ws, size_t ws_bytes, hipStream_t stream);

/* Static description of a status code. */
const char* ec2moe_status_string(ec2moe_status status);

/* Detail of the last failing call on this thread ("" if none). */
const char* ec2moe_last_error(void);

/*
 * Kernel timing. While enabled, every kernel the library launches is bracketed by two
 * HIP events recorded on its launch stream (timing-only events, created without the
 * system-scope memory fence on record). ec2moe_profile_collect waits for the
 * recorded events, writes up to max_entries per-kernel totals (name, launches, total
 * milliseconds) in first-launch order, sets *n_out, and clears the record.
 */
typedef struct {
    char name[48];
    int64_t launches;
    double total_ms;
} ec2moe_kernel_stat;

ec2moe_status ec2moe_profile_enable(int32_t enable);
ec2moe_status ec2moe_profile_collect(ec2moe_kernel_stat* out, int32_t max_entries,
                                     int32_t* n_out);
/*
 * Restrict the timing to kernels named `name` (the names ec2moe_profile_collect
 * reports, e.g. "expert_gate_up"); NULL records every kernel again. The string is
 * copied. Lets a caller time one kernel without event records around the others.
 */
ec2moe_status ec2moe_profile_select(const char* name);

/* Workspace bytes needed by ec2moe_lowrank_fit. */
ec2moe_status ec2moe_lowrank_fit_workspace_size(const ec2moe_codec_desc* desc, size_t* bytes /*[host]*/);

/*
 * Data-free fitting of the codec projections (Encoder-Decoder based on Low-Rank
 * Compression, Eq. 8 with lambda = 0: the reconstruction loss alone). The target is the
 * truncated higher-order SVD of the calibration slices: U spans the r_h leading left
 * singular vectors of [X_1 ... X_c], V the r_w leading ones of [X_1^T ... X_c^T] (for one
 * slice, the truncated SVD of X, the Eckart-Young minimiser of ||X - U U^T X V V^T||).
 * Computed by subspace iteration on the Gram matrices A = sum X_s X_s^T and B = sum
 * X_s^T X_s, starting from the given blocks and orthonormalising every iterate (the
 * positive-diagonal QR, by CholeskyQR2 with a float64 Gram matrix and factor).
 *   x [c][h][w] calibration slices (layer dtype; c*h a multiple of 8);
 *   omega_u [h][r_h], omega_v [w][r_w] float32 start blocks of full column rank (random,
 *   drawn by the caller); iters >= 0 (at most 64) steps: the columns converge to the
 *   leading subspaces at the rate of the spectral gap;
 *   u [h][r_h], v [w][r_w] out, layer dtype, orthonormal columns (to the layer precision);
 *   status device int32 out or NULL: 0, or 1 if a Cholesky pivot was not positive (a start
 *   block or data of rank below r: the outputs are then not orthonormal);
 *   ws of ec2moe_lowrank_fit_workspace_size bytes (two float32 Gram matrices of the larger
 *   of h and w, among others).
 */
ec2moe_status ec2moe_lowrank_fit(const ec2moe_codec_desc* desc, const void* x, const float* omega_u,
                                 const float* omega_v, int32_t iters, void* u, void* v, int32_t* status,
                                 void* ws, size_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------- host planner
 * Producers of the candidate mask and of the end/cloud placement of pipeline tasks, run
 * on the host (no GPU work, no stream). The paper leaves the capability function H, the
 * complexity matching function f and their thresholds open; the forms below are this
 * library's stated choices. All arrays are [host]; nothing is kept after a call.
 */

/* Device state S_device (Eq. 2): available compute, memory, power budget and network
 * bandwidth, each >= 0 in the caller's units. */
typedef struct {
    double cpu, mem, power, bandwidth;
} ec2moe_device_state;

typedef struct {
    double w_cpu, w_mem, w_power, w_bandwidth; /* H (Eq. 3): T_capability = w_cpu cpu + w_mem mem +
                                                  w_power power + w_bandwidth bandwidth, weights >= 0 */
    double epsilon;      /* tolerance of Eq. 4, >= 0 */
    double max_fraction; /* cap on |E_local| / M in [0, 1] (Parameter Selection caps the candidate
                            set at 40% of the experts); 1 = no cap */
} ec2moe_selection_params;

/*
 * Hardware-aware local expert selection (Local Expert Selection, Eq. 2-4) with the
 * matching function f(V_i, T) = V_i / T_capability: E_local = { i : f <= epsilon };
 * when more than floor(max_fraction * M) experts qualify, the ones of smallest f are kept
 * (equal f: the lower index). T_capability <= 0 selects nothing.
 *   complexity [M] values V_i >= 0; mask_out ceil(M/64) words (bit i set <=> i selected,
 *   bits >= M clear), the format of ec2moe_group_gate's candidate mask; n_selected out.
 *   1 <= M <= 256. Errors: EC2MOE_ERR_INVALID_ARGUMENT for NULL pointers, negative or
 *   non-finite inputs, M out of range.
 */
ec2moe_status ec2moe_select_candidates(const ec2moe_device_state* state, const ec2moe_selection_params* params,
                                       const double* complexity, int32_t n_experts, uint64_t* mask_out,
                                       int32_t* n_selected);

typedef struct {
    double alpha;       /* Eq. 9: weight of execution time (1 - alpha: of communication), in [0, 1] */
    double beta;        /* Eq. 11: priority threshold for local execution */
    double epsilon;     /* Eq. 10: guard of the priority's denominator, > 0 */
    double t_end;       /* Eq. 11: computation threshold T_end of the end device */
    double load_end;    /* initial Load_end */
    double load_cloud;  /* initial Load_cloud */
    double speed_end;   /* ExecTime = C / speed_end on the end device, > 0 */
    double speed_cloud; /* ExecTime = C / speed_cloud in the cloud, > 0 */
} ec2moe_schedule_params;

/*
 * Route-aware heuristic pipeline scheduling (Eq. 9-11), greedy: tasks are taken in
 * descending priority P = C / (Comm + epsilon) (equal P: the lower index); a task runs on
 * the end device iff Load_end + C <= T_end and P >= beta, and then Load_end grows by C;
 * otherwise it runs in the cloud and Load_cloud grows by C. The objective of Eq. 9 is
 * sum over tasks (in index order) of alpha ExecTime + (1 - alpha) Comm, with ExecTime
 * = C / speed of the chosen side and Comm counted for cloud tasks only (a task run on
 * the end device transmits nothing).
 *   complexity, comm [n_tasks] values >= 0; location [n_tasks] out: 0 end, 1 cloud;
 *   order [n_tasks] out or NULL: the tasks in processing order; summary [3] out or
 *   NULL: objective, final Load_end, final Load_cloud. n_tasks == 0 is valid.
 * Errors: EC2MOE_ERR_INVALID_ARGUMENT for NULL pointers, negative or non-finite inputs,
 * parameters out of range.
 */
ec2moe_status ec2moe_schedule_tasks(const ec2moe_schedule_params* params, const double* complexity,
                                    const double* comm, int32_t n_tasks, int32_t* location, int32_t* order,
                                    double* summary);

#ifdef __cplusplus
}
#endif

#endif /* EC2MOE_H */
